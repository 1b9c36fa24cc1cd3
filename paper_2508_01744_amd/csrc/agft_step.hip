// agft_step.hip -- batched AGFT decide-and-update step for CDNA4 (gfx950).
//
// One workgroup per tuner instance.  Each arm's record (theta_k and the
// packed upper factor S_k of A_k^{-1}) is read by a group of G = d/2 lanes:
// lane j of the group owns factor columns j and d-1-j (d+1 elements
// together) and theta_{2j}, theta_{2j+1}, so it forms two complete entries
// of v = S^T x_t and two terms of theta^T x_t on its own, and the group only
// sums two numbers at the end.  A record's main part is contiguous in HBM
// and its short tail sits beside the tails of the other arms of its block
// (Rec below): for every load instruction the G lanes of a group read G x 16
// contiguous bytes of one record and a wavefront covers whole cache lines,
// and rewriting one arm touches a handful of cache lines instead of one line
// per 16-byte piece.
//
// Per step and instance (Sec. 4.2-4.4):
//   0. read the instance's words, mask, context and reward, all in one
//      memory round trip; with the switch to exploitation on, feed the
//      previous reward to the instance's Page-Hinkley test and switch when
//      the rewards are stable;
//   1. fetch the record of the previous decision's arm (its update waits);
//      with the paper's pruning rules on, drop arms by their reward counts
//      and means; list the other arms in play (in the action space, not
//      pruned);
//   2. every listed arm: m = theta^T x_t, w^2 = |S^T x_t|^2,
//      UCB = m + alpha_t w, LCB = m - alpha_t w  (Eq. 1); an exploiting
//      instance reads only a contiguous copy of theta and scores m (Eq. 2);
//   3. fold the previous decision's reward into its arm: Eq. 3-5 as a
//      square-root rank-1 update of S (below) plus the matching theta
//      update, in LDS while the stream's first pass is in flight; the
//      updated arm is scored on x_t from LDS in the same operation order as
//      the stream, and its record is written back at the end of the step;
//   4. pruning when due (drop UCB_k < max_j LCB_j), argmax with ties to the
//      lowest arm index; refinement of the action space when due; epilogue.
//
// Square-root update.  Eq. 3 adds x x^T to A, so P = A^{-1} changes by the
// Sherman-Morrison identity P' = P - P x x^T P / (1 + x^T P x).  With P = S S^T
// (S upper triangular) and f = S^T x, P' = S M M^T S^T where M is the upper
// triangular factor of I - f f^T / alpha_d, alpha_j = 1 + f_0^2 + ... + f_j^2
// (alpha_{-1} = 1):
//   M_jj = sqrt(alpha_{j-1} / alpha_j),  M_ij = -f_i f_j / sqrt(alpha_{j-1} alpha_j), i < j,
// so S' = S M column by column:
//   S'_ij = M_jj S_ij - f_j / sqrt(alpha_{j-1} alpha_j) * sum_{i<=k<j} f_k S_ik.
// Eq. 4-5 combine into theta' = theta + g (r - x^T theta) with the gain
// g = P x / (1 + x^T P x) = S f / alpha_{d-1}.
// This is the triangular square-root covariance update of sequential
// estimation (Carlson's form); its fp32 error grows with the square root of
// the condition number of A rather than with the condition number itself.

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <type_traits>

#include "agft.h"
#include "agft_env_math.h"

namespace {

constexpr uint32_t kMagic = 0x54464741u;  // "AGFT"
constexpr int kWave = 64;
constexpr int kMaxK = 1024;
constexpr int kMaxWords = kMaxK / 32;
constexpr int kMaxWaves = 16;
constexpr size_t kAlign = 256;

// Header at the start of the state buffer (256 bytes).
struct alignas(16) StateHeader {
    uint32_t magic;
    uint32_t version;
    int32_t B, K, d, chunks, mask_words, pending;
    int64_t t;
    float lambda, alpha0;
    int32_t alpha_sched, prune_rule, prune_period;
    int32_t exploit;      // 1: the buffer holds the theta copy of the switch
    int32_t tail_floats;  // record layout: floats per lane slice of a tail
    int32_t stats_kept;   // 1: the per-arm reward counts and sums are maintained
    uint32_t reserved[44];
};
static_assert(sizeof(StateHeader) == 256, "header is 256 bytes");

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Record geometry for context dimension D: G lanes per arm, each owning
// D + 3 positions (D + 1 factor elements and two theta entries).  Positions
// 0..D-1 of every lane form the arm's main part (D/4 float4 chunks per
// lane, lane-interleaved); positions D..D+2 its tail, TF floats per lane.
// NB = 64/D arms make a block: their main parts, then their tails, so that
// every main part starts on a 128-byte line.  With TF = 3 records carry no
// padding (608 bytes at D = 16) and the NB tails fill three whole lines,
// but half of them straddle two; with TF = 4 each tail slice is padded to
// a chunk and every tail sits in one line.  An instance's arms take
// ceil(K/NB) blocks.
template <int D, int TF>
struct Rec {
    static constexpr int G = D / 2;              // lanes per arm
    static constexpr int P = D + 1;              // factor elements per lane
    static constexpr int MQ = D / 4;             // main chunks per lane
    static constexpr int S = MQ + 1;             // register slots per lane (the last holds the tail)
    static constexpr int MAIN = G * MQ;          // main chunks per arm
    static constexpr int TAIL = G * TF / 4;      // tail chunks per arm
    static constexpr int R = MAIN + TAIL;        // chunks per record
    static constexpr int NB = 32 / G;            // arms per block
    static constexpr int BLK = NB * R;           // chunks per block
    static constexpr int NSE = D * (D + 1) / 2;  // packed factor elements
    static constexpr int CAN = D + NSE;          // canonical floats: theta, then packed S
};

int chunks_for(int d, int tf) { return (d / 2) * (d / 4) + (d / 2) * tf / 4; }
int block_arms(int d) { return 64 / d; }
// float4 chunks of one instance's arm records: whole blocks
size_t instance_chunks(int K, int d, int tf) {
    const int nb = block_arms(d);
    return (size_t)((K + nb - 1) / nb) * nb * chunks_for(d, tf);
}

// Packed column-major index of S_ij (i <= j) within the factor part.
__host__ __device__ constexpr int packed(int i, int j) { return j * (j + 1) / 2 + i; }

// Canonical index (theta_0..theta_{D-1}, then packed S) of position e of
// lane j's slice of a record; -1 for padding.
__host__ __device__ constexpr int canon(int D, int j, int e) {
    return e <= j ? D + packed(e, j)
         : e <= D ? D + packed(D - e, D - 1 - j)
         : e == D + 1 ? 2 * j
         : e == D + 2 ? 2 * j + 1
         : -1;
}

// Chunk c of arm k's record, as an offset (in chunks) from the instance's
// first block: chunks 0..MAIN-1 are the main part, the rest the tail.
__host__ __device__ constexpr size_t rec_chunk(int D, int TF, int k, int c) {
    const int G = D / 2, NB = 64 / D, MAIN = G * (D / 4), TAIL = G * TF / 4;
    const size_t blk = (size_t)(k / NB) * NB * (MAIN + TAIL);
    return c < MAIN ? blk + (size_t)(k % NB) * MAIN + c
                    : blk + (size_t)NB * MAIN + (size_t)(k % NB) * TAIL + (c - MAIN);
}

// Canonical index of component q of record chunk c; -1 for padding.
__host__ __device__ constexpr int canon_chunk(int D, int TF, int c, int q) {
    const int G = D / 2, MAIN = G * (D / 4);
    if (c < MAIN) return canon(D, c % G, 4 * (c / G) + q);
    const int t = 4 * (c - MAIN) + q;   // tail float: lane t/TF, position D + t%TF
    return t % TF < 3 ? canon(D, t / TF, D + t % TF) : -1;
}

// Float offset, within an arm's record (chunks in record order), of factor
// element S_ij (i <= j) and of theta_i: column j < G sits in lane slice j at
// position i, column j >= G in slice D-1-j at position D-i; theta_i at
// position D+1+(i%2) of slice i/2.  Positions below D are component e%4 of
// main chunk (e/4)*G + slice, the others tail float TF*slice + (e-D).
template <int D, int TF>
__host__ __device__ constexpr int rec_pos_S(int i, int jc) {
    constexpr int G = D / 2, MAIN = G * (D / 4);
    const bool first = jc < G;
    const int sl = first ? jc : D - 1 - jc;
    const int e = first ? i : D - i;
    return e < D ? 4 * ((e >> 2) * G + sl) + (e & 3) : 4 * MAIN + TF * sl + (e - D);
}
template <int D, int TF>
__host__ __device__ constexpr int rec_pos_theta(int i) {
    constexpr int G = D / 2, MAIN = G * (D / 4);
    return 4 * MAIN + TF * (i >> 1) + 1 + (i & 1);
}

// The two offset functions above invert canon_chunk: checked at compile time
// for every record layout the kernels are built for.
template <int D, int TF>
constexpr bool rec_pos_consistent() {
    for (int jc = 0; jc < D; ++jc)
        for (int i = 0; i <= jc; ++i) {
            const int pos = rec_pos_S<D, TF>(i, jc);
            if (canon_chunk(D, TF, pos / 4, pos % 4) != D + packed(i, jc)) return false;
        }
    for (int i = 0; i < D; ++i) {
        const int pos = rec_pos_theta<D, TF>(i);
        if (canon_chunk(D, TF, pos / 4, pos % 4) != i) return false;
    }
    return true;
}
static_assert(rec_pos_consistent<8, 3>() && rec_pos_consistent<8, 4>() && rec_pos_consistent<16, 3>() &&
                  rec_pos_consistent<16, 4>() && rec_pos_consistent<32, 3>() && rec_pos_consistent<32, 4>(),
              "record offsets of the update disagree with the record layout");

// The update walks the factor RP rows apart from one pass to the next.  For
// RP a multiple of 4, row r0 + ps*RP of column jc sits at a fixed per-lane
// base plus ps steps of +G*RP floats (top-down slices, columns < G) or
// -G*RP (bottom-up slices), except row 0 of a bottom-up column, which is its
// slice's tail float; theta_i, RP/2 slices further per pass, moves by TF*RP/2.
// So each pass costs one add of address arithmetic.  Checked at compile time
// against rec_pos_S for every lane and pass of the kernels' shapes.
template <int D, int TF, int RP>
struct RowWalk {
    static constexpr int G = D / 2, MAIN = G * (D / 4);
    static constexpr bool kLinear = RP % 4 == 0;
    __host__ __device__ static constexpr int step(int jc) { return jc < G ? G * RP : -G * RP; }
    __host__ __device__ static constexpr int base(int r0, int jc) {
        const int sl = jc < G ? jc : D - 1 - jc;
        const int e = jc < G ? r0 : D - r0;
        return 4 * ((e >> 2) * G + sl) + (e & 3);
    }
    __host__ __device__ static constexpr int tail(int jc) { return 4 * MAIN + TF * (D - 1 - jc); }
    __host__ __device__ static constexpr int pos(int r0, int jc, int ps) {
        return ps == 0 && r0 == 0 && jc >= G ? tail(jc) : base(r0, jc) + ps * step(jc);
    }
};

template <int D, int TF, int RP>
constexpr bool row_walk_consistent() {
    if constexpr (!RowWalk<D, TF, RP>::kLinear) return true;
    for (int jc = 0; jc < D; ++jc)
        for (int r0 = 0; r0 < RP && r0 < D; ++r0)
            for (int ps = 0; r0 + ps * RP < D; ++ps) {
                const int i = r0 + ps * RP;
                if (i <= jc && RowWalk<D, TF, RP>::pos(r0, jc, ps) != rec_pos_S<D, TF>(i, jc)) return false;
                if (rec_pos_theta<D, TF>(r0) + ps * TF * (RP / 2) != rec_pos_theta<D, TF>(i)) return false;
            }
    return true;
}
// rows per pass: (64 / D) segments per wavefront times 1 or 4 wavefronts
static_assert(row_walk_consistent<8, 3, 8>() && row_walk_consistent<8, 4, 8>() && row_walk_consistent<8, 3, 32>() &&
                  row_walk_consistent<8, 4, 32>() && row_walk_consistent<16, 3, 4>() && row_walk_consistent<16, 4, 4>() &&
                  row_walk_consistent<16, 3, 16>() && row_walk_consistent<16, 4, 16>() &&
                  row_walk_consistent<32, 3, 8>() && row_walk_consistent<32, 4, 8>(),
              "the update's row walk matches the record layout");

// Column j and row i of packed element e.
__device__ inline void unpack(int e, int &i, int &j) {
    int c = 0;
    while ((c + 1) * (c + 2) / 2 <= e) ++c;
    j = c;
    i = e - c * (c + 1) / 2;
}

// Per-instance block of 32-bit words: previous action, active-arm count,
// non-finite-input count, mode (-1 exploring, else the round exploitation
// began), the Page-Hinkley state (n, mean, m+, min m+, m-, min m-), the round
// of its last alarm, its last margin, the action space (lo, hi, stride), the
// top-two score gap of the last decision that dumped its scores, then the
// stashed context.  Kept together so the epilogue
// writes one or two lines per instance.
constexpr int kInstAprev = 0, kInstKact = 1, kInstBad = 2, kInstMode = 3, kInstPh = 4,
              kInstPhLast = 10, kInstPhMargin = 11, kInstLo = 12, kInstHi = 13, kInstStride = 14,
              kInstGap = 15, kInstX = 16;

int inst_words(int d) { return (kInstX + d + 15) / 16 * 16; }

struct Layout {
    size_t arms, mask, inst, stats, theta, total;
};

// Arms an instance may have in play: K, or with the refinement the larger of
// the coarse grid and the window.
int arms_in_play(const agft_config &c) {
    if (!c.refine) return c.K;
    const int coarse = (c.K - 1) / c.refine_stride + 1, window = 2 * c.refine_half + 1;
    const int k = coarse > window ? coarse : window;
    return k < c.K ? k : c.K;
}

// Bytes an exploring instance streams per step, at most: theta and the
// packed factor of every arm in play.
size_t explore_bytes(const agft_config &c) {
    return (size_t)arms_in_play(c) * 4 * (size_t)(c.d + c.d * (c.d + 1) / 2);
}

// Record layout: packed tails (TF = 3) where an exploring instance streams
// more than 16 KB per step, or more than 8 KB when every step streams every
// record (no pruning rule, no refinement, no switch to exploitation), so
// that the stream moves no padding; padded tails (TF = 4) otherwise, where
// the update's one-record read and write-back weigh more than the stream
// and a tail that straddles two lines costs more than its padding.
// Measured on MI355X (step kernel, packed / padded tails): K=128 d=16
// B=65,536 (76 KB) 853 / 889 us, the same with exploitation 827 / 845 us,
// K=256 d=32 B=1,024 (560 KB) 92.0 / 93.0 us, K=128 d=16 B=65,536 with the
// refinement (13 KB) 186 / 176 us, with the refinement, the rules and the
// switch 190 / 179 us; K=64 d=8 B=4,096 (11 KB) over the whole horizon
// 12.85 / 13.25 us without pruning, 11.6 / 11.25 us with rules 1-8,
// 10.45 / 10.45 us with the refinement, 10.5 / 10.4 us with the switch.
int tail_floats(const agft_config &c) {
    const size_t bytes = explore_bytes(c);
    return bytes > 16384 || (bytes > 8192 && c.prune_rule == 0 && !c.refine && !c.exploit) ? 3 : 4;
}

// The per-arm reward counts and sums are read only by the paper's rules 2-8
// and by the refinement's statistical anchor; without those the update
// skips them (their one-line store per instance and step costs 1.4% of the
// step at K=128 d=16 B=65,536) and they stay at zero.
bool stats_kept(const agft_config &c) { return (c.prune_rule & 14) != 0 || c.refine != 0; }

// theta copy [B][K][d] only with the switch to exploitation (0 bytes otherwise)
Layout layout_for(const agft_config &c) {
    Layout L;
    const size_t b = (size_t)c.B, k = (size_t)c.K;
    const size_t kw = (k + 31) / 32;
    size_t off = sizeof(StateHeader);
    L.arms = off;  off = align_up(off + b * instance_chunks(c.K, c.d, tail_floats(c)) * 16);
    L.mask = off;  off = align_up(off + b * kw * 4);
    L.inst = off;  off = align_up(off + b * (size_t)inst_words(c.d) * 4);
    L.stats = off; off = align_up(off + b * k * 8);
    L.theta = off; off = align_up(off + (c.exploit ? b * k * (size_t)c.d * 4 : 0));
    L.total = off;
    return L;
}

// Dynamic LDS of the step kernel: UCB and LCB per arm, then the arm list.
size_t step_lds_bytes(int K) { return ((size_t)K * (2 * 4 + 2) + 15) / 16 * 16; }

// Workgroup width (wavefronts); one workgroup per instance, looping over its
// arms in passes of 64*w/(d/2).  The step is a chain of dependent phases per
// instance, so narrow workgroups (more instances in flight per CU, cheaper
// barriers) win unless each instance streams many bytes.  The bytes per
// step are estimated from the arms in play (with the refinement, at most the
// larger of the coarse grid and the window) times what each costs (the
// record, or the theta copy once instances exploit): one wavefront up to
// 16 KB, four beyond.  Measured on MI355X with padded 640-byte records
// (step kernel, us, w = 1 / 2 / 4; with the packed blocks, w = 2 stayed
// 2-3% slower than w = 4 at K=128 d=16):
//   K=64 d=8 B=4,096 (12 KB):              21 / 25 / 30
//   K=128 d=16 B=65,536 (80 KB):           895 / 892 / 882
//   the same, exploitation (8 KB):         595 / 602 / 672
//   the same, refinement (13 KB):          190 / 231 / 376
//   K=256 d=32 B=1,024 (590 KB):           31 / 29 / 29
//   the same, exploitation (32 KB):        43 / 34 / 31
int waves_for(const agft_config &c) {
    const size_t bytes = c.exploit ? (size_t)arms_in_play(c) * 4 * c.d : explore_bytes(c);
    return bytes <= 16384 ? 1 : 4;
}

// Before round ph_min_rounds no instance can have switched to exploitation,
// so with the switch on, those steps take the width of an exploring
// instance.  Measured on MI355X (us per step over the whole horizon, one
// width throughout / exploring width before the first possible switch):
// K=128 d=16 B=65,536 566.2 / 557.9, the same with rules 2-8 570.8 / 565.1,
// B=16,384 82.6 / 81.5.
int waves_at(const agft_config &c, int64_t t) {
    if (c.exploit && t < c.ph_min_rounds) return explore_bytes(c) <= 16384 ? 1 : 4;
    return waves_for(c);
}

// Whether the update of the previous decision's arm runs before the stream
// (its first pass lands meanwhile and the chain gets shorter) rather than
// after it: always, except at d = 32 where an instance streams more than
// 16 KB, since there the longer update holds back the second pass (the
// kernel still runs it before the stream at a step whose list of arms fits
// in one pass).
// Measured on MI355X (step kernel, before / after the stream): K=64 d=8
// B=4,096 19.1 / 20.5 us; K=128 d=16 B=65,536 853 / 857 us, B=16,384 218.4 /
// 220.8 us; K=256 d=32 B=1,024 92.4 / 91.7 us.
bool early_update(const agft_config &c) { return c.d < 32 || explore_bytes(c) <= 16384; }

// Per-lane slice of the Eq. 1 terms from the S chunks of one record slice:
// va, vb = the two owned entries of S^T x, m = the two owned theta terms.
// xa/xb hold x_e (e <= j) and x_{D-e} (e > j) for this lane's positions.
template <int D>
__device__ __forceinline__ void slice_terms(const float *f, const float *xa, const float *xb,
                                            float xt0, float xt1, float &m, float &w2) {
    float va = 0.0f, vb = 0.0f;
#pragma unroll
    for (int e = 0; e <= D; ++e) {
        va = fmaf(f[e], xa[e], va);
        vb = fmaf(f[e], xb[e], vb);
    }
    m = fmaf(f[D + 2], xt1, f[D + 1] * xt0);
    w2 = fmaf(vb, vb, va * va);
}

// v of another lane of the same row, through a DPP lane pattern.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the G lanes of an aligned group (G = 2, 4, 8, 16), every lane
// ending with the same total: pairs within quads, then the two pairs of a
// quad, then mirrored half rows (8 lanes) and mirrored rows (16 lanes), each
// step a DPP add on the vector unit.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
    static_assert(G == 1 || G == 2 || G == 4 || G == 8 || G == 16, "group of 1..16 lanes");
    if constexpr (G >= 2) v += dpp<0xB1>(v);    // quad_perm [1,0,3,2]
    if constexpr (G >= 4) v += dpp<0x4E>(v);    // quad_perm [2,3,0,1]
    if constexpr (G >= 8) v += dpp<0x141>(v);   // row_half_mirror
    if constexpr (G >= 16) v += dpp<0x140>(v);  // row_mirror
    return v;
}

// Parameters of the paper's pruning rules (bits 2, 4, 8 of the rule mask).
struct Heuristics {
    int32_t mask;          // rule bits 2 | 4 | 8 in use
    int32_t ext_rounds, ext_min_n;
    float ext_thr;
    int32_t hist_after, hist_min_n;
    float hist_kappa;
    int32_t hist_min_arms, cascade_k;
};

// Bits of word w of the action space lo <= k <= hi, (hi - k) % stride == 0.
__device__ inline uint32_t space_bits(int w, int lo, int hi, int stride) {
    const int k0 = 32 * w;
    const int first = lo > k0 ? lo - k0 : 0;
    const int last = hi < k0 + 31 ? hi - k0 : 31;
    if (last < first) return 0u;
    const uint32_t range = last - first == 31 ? 0xffffffffu : ((1u << (last - first + 1)) - 1u) << first;
    if (stride == 1) return range;
    uint32_t grid = 0u;   // positions congruent to hi modulo the stride
    for (int b = (hi - k0) % stride; b < 32; b += stride) grid |= 1u << b;
    return range & grid;
}

// Refinement of the action space after this step's decision (Sec. 4.4).
struct Refine {
    int32_t now;          // refinement due at this step
    int32_t stat;         // statistical anchor (before maturity), else predictive
    int32_t half, min_n;  // window half-width in arms; samples for the statistical anchor
};

// Switch to greedy exploitation after a Page-Hinkley test finds the
// reward sequence stable (Sec. 4.2, Eq. 2).
struct Exploit {
    int32_t on;
    float delta, lambda;
    int32_t window, min_rounds;
};

struct StepArgs {
    float4 *arms;
    uint32_t *mask;
    int32_t *inst;        // [B][IW] per-instance blocks
    int2 *stats;          // [B][K] rewards folded in, their sum (fp32 bits)
    float *theta;         // [B][K][D] copy of theta (exploitation on), else nullptr
    Heuristics h;
    Exploit e;
    Refine rf;
    int64_t t;            // decisions made before this step
    StateHeader *hdr;
    const float *ctx;     // [B][D] or nullptr (flush)
    const float *reward;  // [B] or nullptr
    int32_t *action;      // [B] or nullptr
    float *scores;        // [B][2][K] or nullptr
    int32_t B, K, KW, IW;
    int32_t apply_update;  // a decision is pending
    int32_t prune_now;
    int32_t prune_reset;   // rule 1 starts again from the whole action space (non-sticky)
    int32_t early_update;  // fold the previous reward in before the stream
    int32_t keep_stats;    // maintain the per-arm reward counts and sums
    float alpha;
    int64_t t_next;        // t after this call (header bookkeeping)
};

// Streaming load that bypasses cache retention: every record is read once
// per step and the state of a large batch is many times the cache size.
typedef float nt_f4 __attribute__((ext_vector_type(4)));
// three floats at 4-byte alignment (a record tail slice)
typedef float nt_f3 __attribute__((ext_vector_type(3))) __attribute__((aligned(4)));
__device__ __forceinline__ float4 ld_nt(const float4 *p) {
    const nt_f4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_f4 *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

// The one record per instance that the update gathers and writes back takes
// the same non-temporal hint only for d = 16.  Measured per step against
// ordinary accesses: d = 16, -0.9% (65,536 x 128) and -0.4% (16,384 x 128);
// d = 8, +5% (4,096 x 64); d = 32, +3% (1,024 x 256).
template <int D>
__device__ __forceinline__ float4 ld_record(const float4 *p) {
    if constexpr (D == 16) return ld_nt(p);
    else return *p;
}
template <int D>
__device__ __forceinline__ void st_record(float4 *p, float x, float y, float z, float w) {
    if constexpr (D == 16) __builtin_nontemporal_store(nt_f4{x, y, z, w}, reinterpret_cast<nt_f4 *>(p));
    else *p = make_float4(x, y, z, w);
}

// Element `idx` of a register array indexed by a lane-varying value
// (an unrolled select, so the array stays in registers).
template <int N>
__device__ __forceinline__ float pick(const float *v, int idx) {
    float out = 0.0f;
#pragma unroll
    for (int q = 0; q < N; ++q) out = (idx == q) ? v[q] : out;
    return out;
}

struct BestPair {
    float v;
    int k;
};

__device__ inline BestPair better(BestPair a, BestPair b) {
    if (b.v > a.v || (b.v == a.v && b.k < a.k)) return b;
    return a;
}

// Partner value for step s (0..5) of a 64-lane butterfly: quad pairs, quads,
// mirrored half rows, mirrored rows (all DPP, within rows of 16 lanes), then
// rows 16 and 32 lanes apart.  After the six steps of an associative and
// commutative op every lane holds the same result.
template <int STEP>
__device__ __forceinline__ int partner(int v) {
    if constexpr (STEP == 0) return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
    else if constexpr (STEP == 1) return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
    else if constexpr (STEP == 2) return __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
    else if constexpr (STEP == 3) return __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
    else if constexpr (STEP == 4) return __shfl_xor(v, 16);
    else return __shfl_xor(v, 32);
}
template <int STEP>
__device__ __forceinline__ float partner(float v) { return __int_as_float(partner<STEP>(__float_as_int(v))); }

template <class T, class Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
    v = op(v, partner<0>(v));
    v = op(v, partner<1>(v));
    v = op(v, partner<2>(v));
    v = op(v, partner<3>(v));
    v = op(v, partner<4>(v));
    return op(v, partner<5>(v));
}

__device__ __forceinline__ BestPair wave_best(BestPair b) {
    auto step = [&](BestPair o) { b = better(b, o); };
    step(BestPair{partner<0>(b.v), partner<0>(b.k)});
    step(BestPair{partner<1>(b.v), partner<1>(b.k)});
    step(BestPair{partner<2>(b.v), partner<2>(b.k)});
    step(BestPair{partner<3>(b.v), partner<3>(b.k)});
    step(BestPair{partner<4>(b.v), partner<4>(b.k)});
    step(BestPair{partner<5>(b.v), partner<5>(b.k)});
    return b;
}

// Inclusive prefix sum within aligned segments of SEG lanes (8, 16 or 32):
// DPP shifts within rows of 16 lanes (zero-filled at row edges), masked at
// the edges of 8-lane segments; for 32 lanes, the first row's total is then
// added to the second row of each half-wavefront.
template <int SEG>
__device__ __forceinline__ float segment_scan(float v, int lane) {
    static_assert(SEG == 8 || SEG == 16 || SEG == 32, "segments of 8, 16 or 32 lanes");
    auto shr = [](float x, auto ctrl) {
        return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), decltype(ctrl)::value,
                                                          0xF, 0xF, true));
    };
    const int pos = lane & 7;
    float s = shr(v, std::integral_constant<int, 0x111>{});    // row_shr:1
    v += (SEG > 8 || pos >= 1) ? s : 0.0f;
    s = shr(v, std::integral_constant<int, 0x112>{});          // row_shr:2
    v += (SEG > 8 || pos >= 2) ? s : 0.0f;
    s = shr(v, std::integral_constant<int, 0x114>{});          // row_shr:4
    v += (SEG > 8 || pos >= 4) ? s : 0.0f;
    if constexpr (SEG >= 16) v += shr(v, std::integral_constant<int, 0x118>{});   // row_shr:8
    if constexpr (SEG == 32)
        v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xA, 0xF, false));  // row_bcast:15
    return v;
}

// Sum over the 64/SEG segments of a wavefront: every lane ends with the
// total of its column (lane % SEG) over the segments.
template <int SEG>
__device__ __forceinline__ float segment_colsum(float v) {
    if constexpr (SEG == 8) v += dpp<0x128>(v);   // row_ror:8, the other half row
    if constexpr (SEG <= 16) v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

// Workgroup-wide reductions through one LDS slot per wavefront (a
// one-wavefront workgroup needs neither the slots nor the barriers).
template <class T, class Op>
__device__ T block_reduce(T v, T *red, int lane, int wave, int nwave, Op op) {
    v = wave_reduce(v, op);
    if (nwave == 1) return v;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    T out = red[0];
    for (int w = 1; w < nwave; ++w) out = op(out, red[w]);
    __syncthreads();
    return out;
}

// Wavefronts per SIMD the register allocation must allow (the kernel's W).
// At d = 16 with packed tails (instances that stream more than 16 KB, four
// wavefronts each) the code the compiler gives at six (75 registers) beats
// the one squeezed into seven (72): step kernel 842 vs 848 us at K=128
// B=65,536, 211.7 vs 212.8 us at B=16,384.  Seven wins everywhere else:
// with the paper's rules 2-8, whose pass over the arm statistics gains from
// more instances in flight (918.6 vs 885.2 us at K=128 B=65,536, 186.4 vs
// 177.8 us at B=16,384), and with padded tails (one wavefront per instance):
// 173.6 vs 183.1 us with the refinement, rules and switch, 48.6 vs 49.8 us
// with the refinement alone.
int occupancy_for(const agft_config &c, int tail) {
    if (c.d == 32) return 4;
    return c.d == 16 && tail == 3 && !(c.prune_rule & 14) ? 6 : 7;
}

// Workgroups per compute unit for four-wavefront workgroups at six
// wavefronts per SIMD (d = 16, packed tails, no rules 2-8): 4, enforced by
// the launch's LDS request.  There the chain of phases per instance is short
// beside its stream, and four instances per compute unit keep enough of the
// stream in flight to hold the HBM rate, while more interleave more
// concurrent streams and lose rate.  Measured on MI355X (step kernel, us, at
// 6 / 5 / 4 / 3 workgroups per compute unit): K=128 d=16 B=65,536 823.6 /
// 819.5 / 807.8 / 858.0, B=16,384 199.0 / 197.5 / 197.1 / 209.4.  Not with
// the paper's rules 2-8, whose pass over the arm statistics needs the
// instances in flight (K=128 d=16 B=65,536: 827.7 uncapped, 852.6 at 5,
// 911.1 at 4), nor for one-wavefront workgroups, whose steps are short
// chains with little to stream.
int cu_workgroups_for(int waves, int simd_waves) { return waves == 4 && simd_waves == 6 ? 4 : 0; }

// ENV: the simulator's environment responds in the epilogue (agft_sim_step):
// once the decision is known, the first lanes of wavefront 0 run the
// instance's next window with it, writing the reward and the next context in
// place of the ones read.  The word each of those lanes prefetches costs a
// register: at d = 16 the seven-wavefront form gets six, to fit without
// spilling.
template <int D, int TF, int W, int NW, bool ENV>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(ENV && D == 16 && W > 6 ? W - 1 : W)))
void agft_step_kernel(StepArgs p, agft_env_detail::EnvArgs env) {
    using R = Rec<D, TF>;
    constexpr int G = R::G, S = R::S;
    constexpr int NQ = (R::R + kWave - 1) / kWave;   // update-record chunks per thread (>= 64 threads)
    const int inst = blockIdx.x;
    const int tid = threadIdx.x;
    constexpr int nthr = NW * kWave;   // the launch's workgroup width, fixed per instantiation
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    constexpr int nwave = NW;
    const int K = p.K;
    const int KW = p.KW;
    const int j = tid % G;           // slot of this lane within its arm's group
    const int grp = tid / G;         // group index within the workgroup
    const int apw = nthr / G;        // arms per pass of the workgroup
    const size_t inst_chunks = (size_t)((K + R::NB - 1) / R::NB) * R::BLK;
    const float4 *recs = p.arms + (size_t)inst * inst_chunks;

    // the previous decision's record before and after its update, chunks in
    // record order (the layout of the arm's record in HBM)
    __shared__ float4 s_old4[R::R];
    __shared__ float4 s_new4[R::R];
    float *s_old = reinterpret_cast<float *>(s_old4);
    float *s_new = reinterpret_cast<float *>(s_new4);
    __shared__ float s_fpart[NW][D];   // per-wavefront partial sums of f = S^T xp
    // per-arm scores and the list of arms to stream, sized by K at launch
    // (step_lds_bytes) so that small arm counts leave room for more workgroups
    extern __shared__ float s_arm[];
    float *s_ucb = s_arm;
    float *s_lcb = s_arm + K;
    short *s_list = reinterpret_cast<short *>(s_arm + 2 * K);
    __shared__ uint32_t s_mask[kMaxWords];
    __shared__ int s_nlist;
    __shared__ float s_red_v[kMaxWaves];
    __shared__ int s_red_k[kMaxWaves];
    __shared__ int s_red_n[kMaxWaves];
    __shared__ uint32_t s_mask2[kMaxWords];
    __shared__ uint32_t s_raw[kMaxWords];   // arms no rule has removed (the global mask words)
    __shared__ float s_red_v2[kMaxWaves];
    __shared__ int s_red_k2[kMaxWaves];

    __shared__ float s_xp[D];   // context of the previous decision, for the update
    __shared__ int2 s_stu;      // its arm's reward count and sum

    const bool decide = p.ctx != nullptr;
    int32_t *blk = p.inst + (size_t)inst * p.IW;
    // Everything the step reads before it knows the previous decision's arm is
    // requested at once, so that the prologue waits for one memory round trip
    // rather than one per item (the vector loads first: the compiler's waits
    // for the addresses of later ones would hold them back behind the scalar
    // loads).  Vector loads, by wavefront 0: the environment's state of the
    // instance (for the epilogue), the instance's mask words and the previous
    // decision's context; at D = 32 also the context, by every wavefront.
    // Scalar loads: the instance's first sixteen words, the reward and, up
    // to D = 16, the context.
    __shared__ uint32_t s_envw[ENV ? 32 : 1];
    uint32_t env_pre = 0u;
    if constexpr (ENV)
        if (wave == 0) env_pre = agft_env_detail::env_prefetch(env, inst, lane);
    const int lane_d = lane < D ? lane : 0;   // clamped element index
    const uint32_t *mask_at = p.mask + (size_t)inst * KW + (lane < KW ? lane : 0);
    const float *xp_at = reinterpret_cast<const float *>(blk + kInstX) + lane_d;
    uint32_t raw_word = 0u;
    float xp_word = 0.0f;
    if (wave == 0) {
        raw_word = *mask_at;
        xp_word = *xp_at;
    }
    const int4 *blk4 = reinterpret_cast<const int4 *>(blk);
    const int4 wa = blk4[0], wb = blk4[1], wc = blk4[2], wd = blk4[3];
    // (no branch around the reward either: without a pending decision the
    // block's first word stands in for it, unused)
    const float r_in = *(p.apply_update ? p.reward + inst : reinterpret_cast<const float *>(blk));
    // The context, without a branch: a flush reads the block's own words in
    // its place, and nothing uses them (x_ok is false, so no arm is listed,
    // scored or stashed).  Non-finite test on the exponent bits (both
    // operands of the and evaluated: a short-circuit branch would hold back
    // the loads after it).  Up to D = 16 the context comes by scalar loads;
    // at D = 32 lane l < D reads element l and the selectors below take the
    // values from the lanes, so that 32 scalar registers are not held while
    // the loads are in flight (they would push the scalar loads apart).
    const float *xi = decide ? p.ctx + (size_t)inst * D : reinterpret_cast<const float *>(blk);
    float x[D];
    float x_lane;   // element `lane` of the context, lanes < D
    bool x_ok;
    if constexpr (D <= 16) {
        uint32_t nonfinite = 0u;
#pragma unroll
        for (int q = 0; q < D; ++q) {
            x[q] = xi[q];
            nonfinite |= (__float_as_uint(x[q]) & 0x7f800000u) == 0x7f800000u ? 1u : 0u;
        }
        x_ok = decide & (nonfinite == 0u);
        x_lane = pick<D>(x, lane);
    } else {
        x_lane = xi[lane_d];
        x_ok = decide & (__ballot((__float_as_uint(x_lane) & 0x7f800000u) == 0x7f800000u) == 0ull);
#pragma unroll
        for (int q = 0; q < D; ++q) x[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x_lane), q));
    }

    // The context also waits in LDS for its later readers (the exploiting
    // stream and the stash in the epilogue).
    __shared__ float s_x[D];
    if (wave == 0 && lane < D) s_x[lane] = x_lane;
    // This lane's selectors of x: xa_e = x_e for e <= j, xb_e = x_{D-e} for e > j.
    float xa[D + 1], xb[D + 1];
#pragma unroll
    for (int e = 0; e <= D; ++e) {
        xa[e] = e <= j ? x[e] : 0.0f;
        xb[e] = (e > j && e >= 1) ? x[D - e < 0 ? 0 : D - e] : 0.0f;
    }
    const float xt0 = pick<D>(x, 2 * j), xt1 = pick<D>(x, 2 * j + 1);
    const int a_prev = p.apply_update ? wa.x : -1;   // word kInstAprev
    const bool has_prev = a_prev >= 0 && a_prev < K;
    // (taken back to a scalar register: the select leaves it in a vector one)
    const float r = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(has_prev ? r_in : 0.0f)));
    const bool upd = has_prev && isfinite(r);
    const int a_upd = upd ? a_prev : -1;

    // Page-Hinkley test on the instance's rewards and the switch to greedy
    // exploitation (uniform scalar code, single precision, fixed order).
    static_assert(kInstMode == 3 && kInstPh == 4 && kInstPhLast == 10 && kInstPhMargin == 11 && kInstLo == 12 &&
                      kInstHi == 13 && kInstStride == 14,
                  "word order of the instance block");
    int mode = p.e.on ? wa.w : -1;
    float ph[6] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int ph_last = 0;
    float ph_margin = 0.0f;
    if (p.e.on) {
        ph[0] = __int_as_float(wb.x);
        ph[1] = __int_as_float(wb.y);
        ph[2] = __int_as_float(wb.z);
        ph[3] = __int_as_float(wb.w);
        ph[4] = __int_as_float(wc.x);
        ph[5] = __int_as_float(wc.y);
        ph_last = wc.z;
        ph_margin = __int_as_float(wc.w);
        if (upd && mode < 0) {
            ph[0] = ph[0] + 1.0f;
            ph[1] = ph[1] + (r - ph[1]) / ph[0];
            ph[2] = ph[2] + ((r - ph[1]) - p.e.delta);
            ph[3] = fminf(ph[3], ph[2]);
            ph[4] = ph[4] + ((ph[1] - r) - p.e.delta);
            ph[5] = fminf(ph[5], ph[4]);
            const float up = ph[2] - ph[3], dn = ph[4] - ph[5];
            ph_margin = p.e.lambda - (up > dn ? up : dn);
            if (up > p.e.lambda || dn > p.e.lambda) {
                ph_last = (int)p.t;
#pragma unroll
                for (int q = 0; q < 6; ++q) ph[q] = 0.0f;
            }
        }
        if (mode < 0 && x_ok && p.t >= p.e.min_rounds && p.t - ph_last >= p.e.window) mode = (int)p.t;
    }
    const bool greedy = mode >= 0;
    // The block's words 3..11 after this step, parked in LDS by the lanes that
    // store them at the end (so they hold no registers through the stream; every
    // wave has read the old words before any lane writes the new ones).
    __shared__ int s_phw[kInstPhMargin + 1 - kInstMode];
    const bool ph_lane = p.e.on && tid >= kInstMode && tid <= kInstPhMargin;
    if (ph_lane)
        s_phw[tid - kInstMode] = tid == kInstMode ? mode
                               : tid == kInstPhLast ? ph_last
                               : tid == kInstPhMargin ? __float_as_int(ph_margin)
                               : __float_as_int(pick<6>(ph, tid - kInstPh));

    // the arms in play: not removed by a pruning rule, inside the action space;
    // at a rule-1 step of the non-sticky reading, every arm of the space
    const int sp_lo = wd.x, sp_hi = wd.y;
    const int sp_st = wd.z > 1 ? wd.z : 1;
    const bool reset = p.prune_reset && !greedy && x_ok;
    if (wave == 0 && lane < KW) {
        s_raw[lane] = raw_word;
        s_mask[lane] = (reset ? 0xffffffffu : raw_word) & space_bits(lane, sp_lo, sp_hi, sp_st);
    }
    if (upd && wave == 0 && lane < D) s_xp[lane] = xp_word;

    // Record of the previous decision's arm, requested once its index is
    // known (after the LDS stores above, which would otherwise wait for it
    // too) and staged in LDS before the stream.  Its reward count and sum
    // are fetched with it, so that the end of the step only stores them.
    float4 old_chunk[NQ];
    int2 st_upd = make_int2(0, 0);
    if (upd) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int c = tid + q * nthr;
            if (c < R::R) old_chunk[q] = ld_record<D>(recs + rec_chunk(D, TF, a_upd, c));
        }
        if (p.keep_stats && tid == 0) st_upd = p.stats[(size_t)inst * K + a_upd];
    }

    // The paper's pruning rules (Sec. 4.3) on the arms active at step start,
    // with the previous decision's reward already counted.
    if (p.h.mask != 0 && x_ok) {
        __syncthreads();
        const int2 *st = p.stats + (size_t)inst * K;
        const Heuristics &h = p.h;
        auto act0 = [&](int k) { return ((s_mask[k >> 5] >> (k & 31)) & 1u) != 0; };
        // means to s_lcb, counts to s_ucb (as int bits); both are rewritten by the stream
        int q = 0;
        float qsum = 0.0f, qbest = -INFINITY;
        for (int k = tid; k < K; k += nthr) {
            const int2 v = st[k];
            int n = v.x;
            float rs = __int_as_float(v.y);
            if (k == a_upd) {
                n += 1;
                rs += r;
            }
            const float mean = n > 0 ? rs / (float)n : 0.0f;
            s_lcb[k] = mean;
            s_ucb[k] = __int_as_float(n);
            if (act0(k) && n >= h.hist_min_n) {
                ++q;
                qsum += mean;
                qbest = fmaxf(qbest, mean);
            }
        }
        auto fsum = [](float a, float b) { return a + b; };
        auto fmx = [](float a, float b) { return fmaxf(a, b); };
        auto isum = [](int a, int b) { return a + b; };
        auto imx = [](int a, int b) { return a > b ? a : b; };
        q = block_reduce(q, s_red_n, lane, wave, nwave, isum);
        qsum = block_reduce(qsum, s_red_v, lane, wave, nwave, fsum);
        qbest = block_reduce(qbest, s_red_v, lane, wave, nwave, fmx);
        const bool hist_on = (h.mask & 4) && p.t >= h.hist_after && q >= h.hist_min_arms && q > 0;
        float sigma = 0.0f;
        if (hist_on) {
            const float mu = qsum / (float)q;
            float acc = 0.0f;
            for (int k = tid; k < K; k += nthr) {
                const int n = __float_as_int(s_ucb[k]);
                if (act0(k) && n >= h.hist_min_n) acc += (s_lcb[k] - mu) * (s_lcb[k] - mu);
            }
            acc = block_reduce(acc, s_red_v, lane, wave, nwave, fsum);
            sigma = sqrtf(acc / (float)q);
        }
        auto gone = [&](int k) {
            if (!act0(k)) return false;
            const int n = __float_as_int(s_ucb[k]);
            const float mean = s_lcb[k];
            if ((h.mask & 2) && p.t < h.ext_rounds && n >= h.ext_min_n && mean < h.ext_thr) return true;
            if (hist_on && n >= h.hist_min_n && h.hist_kappa * sigma - (qbest - mean) < 0.0f) return true;
            return false;
        };
        int kstar = -1;
        if (h.mask & 8) {
            for (int k = tid; k < K; k += nthr)
                if (k < h.cascade_k && gone(k)) kstar = k > kstar ? k : kstar;
            kstar = block_reduce(kstar, s_red_n, lane, wave, nwave, imx);
        }
        int left = 0;
        for (int base = 0; base < K; base += nthr) {
            const int k = base + tid;
            const bool stay = k < K && act0(k) && !gone(k) && !(k < kstar);
            left += stay ? 1 : 0;
            const unsigned long long bal = __ballot(stay);
            const int w0 = (base + wave * kWave) >> 5;
            if (lane == 0 && w0 < KW) s_mask2[w0] = (uint32_t)(bal & 0xffffffffull);
            if (lane == 0 && w0 + 1 < KW) s_mask2[w0 + 1] = (uint32_t)(bal >> 32);
        }
        left = block_reduce(left, s_red_n, lane, wave, nwave, isum);
        if (left == 0) {
            // keep the best mean reward among the arms that had rewards, else the first arm
            BestPair bk{-INFINITY, 0x7fffffff};
            int first = 0x7fffffff;
            for (int k = tid; k < K; k += nthr)
                if (act0(k)) {
                    first = k < first ? k : first;
                    if (__float_as_int(s_ucb[k]) > 0) bk = better(bk, BestPair{s_lcb[k], k});
                }
            bk = wave_best(bk);
            first = wave_reduce(first, [](int a, int b) { return a < b ? a : b; });
            if (lane == 0) {
                s_red_v[wave] = bk.v;
                s_red_k[wave] = bk.k;
                s_red_n[wave] = first;
            }
            __syncthreads();
            if (tid == 0) {
                BestPair all{s_red_v[0], s_red_k[0]};
                int f0 = s_red_n[0];
                for (int w = 1; w < nwave; ++w) {
                    all = better(all, BestPair{s_red_v[w], s_red_k[w]});
                    f0 = s_red_n[w] < f0 ? s_red_n[w] : f0;
                }
                const int keep = all.k != 0x7fffffff ? all.k : f0;
                if (keep < K) s_mask2[keep >> 5] |= 1u << (keep & 31);
            }
        }
        __syncthreads();
        if (wave == 0 && lane < KW) {
            const uint32_t w = s_mask2[lane];
            const uint32_t removed = s_mask[lane] & ~w;
            if (removed != 0u) {
                s_raw[lane] &= ~removed;
                p.mask[(size_t)inst * KW + lane] = s_raw[lane];
            }
            s_mask[lane] = w;
        }
        __syncthreads();
    }

    // Active arms other than the one being updated, in index order: one arm
    // per lane, 64 at a time, each placed by the count of active lanes below
    // it in the wavefront's ballot.
    if (wave == 0) {
        int placed = 0;
        for (int k0 = 0; k0 < K; k0 += kWave) {
            const int k = k0 + lane;
            const bool on = x_ok && k < K && k != a_upd && ((s_mask[k >> 5] >> (k & 31)) & 1u) != 0u;
            const unsigned long long bal = __ballot(on);
            if (on) s_list[placed + __popcll(bal & ((1ull << lane) - 1ull))] = (short)k;
            placed += __popcll(bal);
        }
        if (lane == 0) s_nlist = placed;
    }

    // The previous decision's record, fetched at kernel start, goes to LDS now,
    // so that it holds no registers through the stream.
    if (upd) {
        if (tid == 0) s_stu = st_upd;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int c = tid + q * nthr;
            if (c < R::R) s_old4[c] = old_chunk[q];
        }
    }
    __syncthreads();

    const int nlist = s_nlist;
    // Stream buffers: two sets of S slots per lane, used in turn, so that one
    // pass is scored while the next one's loads are in flight: the lane's
    // main chunks, then its three tail floats.  The first pass is issued now
    // and lands while the update below runs.
    float4 buf_a[S], buf_b[S];
    auto fetch = [&](int k, float4 *dst) {
        const float4 *blk = recs + (size_t)(k / R::NB) * R::BLK;
        const float4 *src = blk + (k % R::NB) * R::MAIN + j;
#pragma unroll
        for (int sidx = 0; sidx < R::MQ; ++sidx) dst[sidx] = ld_nt(src + sidx * G);
        const float *tail = reinterpret_cast<const float *>(blk + R::NB * R::MAIN + (k % R::NB) * R::TAIL) + TF * j;
        const nt_f3 t = __builtin_nontemporal_load(reinterpret_cast<const nt_f3 *>(tail));
        dst[R::MQ] = make_float4(t.x, t.y, t.z, 0.0f);
    };
    auto list_at = [&](int slot) { return slot < nlist ? (int)s_list[slot] : -1; };
    int k_a = -1;
    if (!greedy) {
        k_a = list_at(grp);
        if (k_a >= 0) fetch(k_a, buf_a);
    }

    // ---- square-root rank-1 update of the previous decision's arm ----
    // Run while the stream's first pass is in flight, or after the stream
    // (early_update on the host decides which, and the kernel runs it early
    // whenever the whole list fits in the first pass), in LDS; the updated
    // record is written back as the kernel's last act (write_back below).
    auto update = [&]() {
        if (upd) {
            // Lane l of every wavefront takes column j = l % D of one row per
            // pass (row segments of D lanes; a pass of the workgroup covers RP
            // rows), so that the column sums and the row prefix sums below are
            // segment-wide DPP reductions instead of D-step loops on one lane.
            constexpr int SEGS = kWave / D, RP = NW * SEGS, NP = (D + RP - 1) / RP;
            const int jc = lane % D, seg = lane / D;
            const int r0 = wave * SEGS + seg;   // this lane's row in pass 0
            using Walk = RowWalk<D, TF, RP>;
            const int wbase = Walk::base(r0, jc), wstep = Walk::step(jc), wtail = Walk::tail(jc);
            const int tbase = rec_pos_theta<D, TF>(r0 < D ? r0 : 0);
            auto pos_S = [&](int ps, int i) {
                if constexpr (Walk::kLinear) return ps == 0 && r0 == 0 && jc >= G ? wtail : wbase + ps * wstep;
                else return rec_pos_S<D, TF>(i, jc);
            };
            // f_j = sum_{i<=j} S_ij xp_i: this lane's rows, then the other
            // segments of the wavefront, then the other wavefronts
            float fj = 0.0f;
#pragma unroll
            for (int ps = 0; ps < NP; ++ps) {
                const int i = ps * RP + r0;
                if (i < D && i <= jc) fj = fmaf(s_old[pos_S(ps, i)], s_xp[i], fj);
            }
            fj = segment_colsum<D>(fj);
            if constexpr (NW > 1) {
                if (seg == 0) s_fpart[wave][jc] = fj;
                __syncthreads();
                fj = s_fpart[0][jc];
#pragma unroll
                for (int w = 1; w < NW; ++w) fj += s_fpart[w][jc];
            }
            // alpha_j = 1 + f_0^2 + ... + f_j^2 (prefix over the segment) and the
            // column coefficients of M; alpha_{d-1} from the segment's last lane
            const float incl = segment_scan<D>(fj * fj, lane);
            const float al = 1.0f + incl;
            const float al_prev = 1.0f + (incl - fj * fj);
            const float ca = sqrtf(al_prev / al), cb = fj / sqrtf(al_prev * al);
            const float al_last = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(al), D - 1));
            // prediction error r - xp^T theta
            float pred = lane < D ? s_xp[lane] * s_old[rec_pos_theta<D, TF>(lane)] : 0.0f;
            pred = wave_reduce(pred, [](float a, float b) { return a + b; });
            const float err = r - pred;
            // row i of S' = S M:  S'_ij = ca_j S_ij - cb_j g_ij with g_ij the
            // exclusive prefix sum of f_q S_iq along the row; its total is
            // (S f)_i, so the gain is that total / alpha_{d-1} (one reciprocal
            // for all rows: theta carries a 1e-3 tolerance, orders of
            // magnitude above the ulp this gives away)
            const float inv_al = 1.0f / al_last;
#pragma unroll
            for (int ps = 0; ps < NP; ++ps) {
                const int i = ps * RP + r0;
                const bool in_row = i < D && i <= jc;
                const int pos = pos_S(ps, i < D ? i : 0);
                const float sij = in_row ? s_old[pos] : 0.0f;
                const float q = fj * sij;
                const float qi = segment_scan<D>(q, lane);
                if (in_row) s_new[pos] = ca * sij - cb * (qi - q);
                if (i < D && jc == D - 1) {
                    const int tp = tbase + ps * TF * (RP / 2);
                    s_new[tp] = fmaf(qi * inv_al, err, s_old[tp]);
                }
            }
            // padded tails: the fourth float of each lane slice's tail stays 0
            if constexpr (TF == 4)
                if (tid < G) s_new[4 * R::MAIN + 4 * tid + 3] = 0.0f;
            __syncthreads();
        } else if (has_prev && tid == 0) {
            blk[kInstBad] += 1;
        }
    };
    // The updated record, its theta copy and its reward count and sum go out
    // last.  Loads and stores share one completion counter on this
    // architecture, and the compiler's waits for the stream's loads do not
    // follow paths: a store issued before a wait for a load is waited for too,
    // so stores in the middle of the step would hold up the rest of it by
    // their full latency.
    auto write_back = [&]() {
        if (upd) {
            float4 *dst = p.arms + (size_t)inst * inst_chunks;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int c = tid + q * nthr;
                if (c < R::R) {
                    const float4 v = s_new4[c];
                    st_record<D>(dst + rec_chunk(D, TF, a_upd, c), v.x, v.y, v.z, v.w);
                }
            }
            if (p.theta != nullptr && tid < D / 4) {
                float4 *tdst = reinterpret_cast<float4 *>(p.theta + ((size_t)inst * K + a_upd) * D);
                tdst[tid] = make_float4(s_new[rec_pos_theta<D, TF>(4 * tid)], s_new[rec_pos_theta<D, TF>(4 * tid + 1)],
                                        s_new[rec_pos_theta<D, TF>(4 * tid + 2)], s_new[rec_pos_theta<D, TF>(4 * tid + 3)]);
            }
            if (p.keep_stats && tid == 0)
                p.stats[(size_t)inst * K + a_upd] =
                    make_int2(s_stu.x + 1, __float_as_int(__int_as_float(s_stu.y) + r));
        }
    };
    // The updated arm, scored on x_t from LDS exactly as the stream scores a
    // record from HBM (same slices, same operation order).  With the early
    // update it runs right after it, while the stream's first pass is in
    // flight, instead of after the stream on the step's critical path.
    auto score_updated = [&]() {
        if (upd && x_ok && wave == 0) {
            float f[4 * S];
#pragma unroll
            for (int sidx = 0; sidx < R::MQ; ++sidx) {
                const float4 c4 = s_new4[sidx * G + j];
                f[4 * sidx] = c4.x;
                f[4 * sidx + 1] = c4.y;
                f[4 * sidx + 2] = c4.z;
                f[4 * sidx + 3] = c4.w;
            }
            const float *tl = s_new + 4 * R::MAIN + TF * j;
            f[4 * R::MQ] = tl[0];
            f[4 * R::MQ + 1] = tl[1];
            f[4 * R::MQ + 2] = tl[2];
            f[4 * R::MQ + 3] = 0.0f;
            float m, w2;
            slice_terms<D>(f, xa, xb, xt0, xt1, m, w2);
            m = group_sum<G>(m);
            w2 = group_sum<G>(w2);
            if (lane == 0) {
                const float w = sqrtf(w2);
                s_ucb[a_upd] = greedy ? m : fmaf(p.alpha, w, m);
                s_lcb[a_upd] = greedy ? m : fmaf(-p.alpha, w, m);
            }
        }
    };
    // An exploiting instance has no pass in flight.  Where the whole list fits
    // in the first pass, no later pass can wait behind the update.
    const bool early = (p.early_update || nlist <= apw) && !greedy;
    if (early) {
        update();
        score_updated();
    }

    // ---- scoring of every listed arm (Eq. 1), two passes in flight ----
    if (greedy) {
        // Eq. 2: only theta_k^T x_t, read from the contiguous theta copy by
        // groups of D/4 lanes (one float4 each)
        constexpr int GT = D / 4;
        const int jt = tid % GT, gt = tid / GT, apt = nthr / GT;
        const float x0 = s_x[4 * jt], x1 = s_x[4 * jt + 1];
        const float x2 = s_x[4 * jt + 2], x3 = s_x[4 * jt + 3];
        const float4 *th = reinterpret_cast<const float4 *>(p.theta + (size_t)inst * K * D);
        // UT passes' loads are issued before any of them is used, so that an
        // instance waits for about one load latency per UT passes (three at
        // d = 16 with seven wavefronts per SIMD, where four would spill).
        // The explicit wait first (gfx9 encoding: vmcnt 0 only) clears the
        // loads of the prologue, all consumed by now, from the compiler's
        // count: otherwise a register they targeted, reused in the loop,
        // would make it wait for every load in flight in each pass.
        constexpr int UT = D == 16 && W >= 7 ? 3 : 4;
        __builtin_amdgcn_s_waitcnt(0x0F70);
        for (int base = 0; base < nlist; base += UT * apt) {
            int kc[UT];
            float4 v[UT];
#pragma unroll
            for (int u = 0; u < UT; ++u) {
                const int slot = base + u * apt + gt;
                kc[u] = slot < nlist ? s_list[slot] : -1;
                v[u] = kc[u] >= 0 ? ld_nt(th + (size_t)kc[u] * GT + jt) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
#pragma unroll
            for (int u = 0; u < UT; ++u) {
                float m = kc[u] >= 0 ? fmaf(v[u].w, x3, fmaf(v[u].z, x2, fmaf(v[u].y, x1, v[u].x * x0))) : 0.0f;
                m = group_sum<GT>(m);
                if (kc[u] >= 0 && jt == 0) {
                    s_ucb[kc[u]] = m;
                    s_lcb[kc[u]] = m;
                }
            }
        }
    } else {
        auto score = [&](const float4 *c4, int k) {
            float f[4 * S];
#pragma unroll
            for (int sidx = 0; sidx < S; ++sidx) {
                f[4 * sidx + 0] = c4[sidx].x;
                f[4 * sidx + 1] = c4[sidx].y;
                f[4 * sidx + 2] = c4[sidx].z;
                f[4 * sidx + 3] = c4[sidx].w;
            }
            float m, w2;
            slice_terms<D>(f, xa, xb, xt0, xt1, m, w2);
            if (k < 0) {
                m = 0.0f;
                w2 = 0.0f;
            }
            m = group_sum<G>(m);
            w2 = group_sum<G>(w2);
            if (k >= 0 && j == 0) {
                const float w = sqrtf(w2);
                s_ucb[k] = fmaf(p.alpha, w, m);
                s_lcb[k] = fmaf(-p.alpha, w, m);
            }
        };
        for (int base = 0; base < nlist; base += 2 * apw) {
            const int k_b = list_at(base + apw + grp);
            if (k_b >= 0) fetch(k_b, buf_b);
            score(buf_a, k_a);
            if (base + apw >= nlist) break;
            k_a = list_at(base + 2 * apw + grp);
            if (k_a >= 0) fetch(k_a, buf_a);
            score(buf_b, k_b);
        }
    }

    if (!early) {
        update();
        score_updated();
    }

    if (!decide) {
        if (tid == 0) {
            blk[kInstAprev] = -1;
            if (inst == 0) p.hdr->pending = 0;
        }
        if (ph_lane) blk[tid] = s_phw[tid - kInstMode];
        write_back();
        return;
    }

    if (!x_ok) {
        if (p.scores != nullptr) {
            float *sc = p.scores + (size_t)inst * 2 * K;
            for (int q = tid; q < K; q += nthr) {
                sc[q] = -INFINITY;
                sc[K + q] = -INFINITY;
            }
        }
        if (tid == 0) {
            blk[kInstBad] += 1;
            blk[kInstAprev] = -1;
            if (p.action != nullptr) p.action[inst] = -1;
            if (inst == 0) {
                p.hdr->t = p.t_next;
                p.hdr->pending = 1;
            }
        }
        if (ph_lane) blk[tid] = s_phw[tid - kInstMode];
        if constexpr (ENV)
            if (wave == 0) agft_env_detail::env_epilogue(env, inst, -1, lane, env_pre, s_envw);
        write_back();
        return;
    }
    __syncthreads();

    // ---- pruning and argmax over the scores in LDS ----
    auto is_active = [&](int k) { return k < K && ((s_mask[k >> 5] >> (k & 31)) & 1u) != 0; };
    float lstar = -INFINITY;
    const bool prune_now = p.prune_now && !greedy;
    if (prune_now) {
        float l = -INFINITY;
        for (int k = tid; k < K; k += nthr)
            if (is_active(k)) l = fmaxf(l, s_lcb[k]);
        l = wave_reduce(l, [](float a, float b) { return fmaxf(a, b); });
        if (lane == 0) s_red_v[wave] = l;
        __syncthreads();
        for (int w = 0; w < nwave; ++w) lstar = fmaxf(lstar, s_red_v[w]);
        __syncthreads();
    }
    BestPair b{-INFINITY, 0x7fffffff};
    BestPair sb{-INFINITY, 0x7fffffff};   // statistical refinement anchor
    const bool stat_anchor = p.rf.now && p.rf.stat;
    int n = 0;
    float *sc = p.scores != nullptr ? p.scores + (size_t)inst * 2 * K : nullptr;
    float top1 = -INFINITY, top2 = -INFINITY;   // two largest kept scores (with the dump only)
    for (int base = 0; base < K; base += nthr) {
        const int k = base + tid;
        const bool act = is_active(k);
        const float u = act ? s_ucb[k] : -INFINITY;
        const bool keep = act && !(u < lstar);
        n += __popcll(__ballot(keep));   // uniform over the wavefront
        if (keep) {
            b = better(b, BestPair{u, k});
            if (sc != nullptr) {
                top2 = fmaxf(top2, fminf(top1, u));
                top1 = fmaxf(top1, u);
            }
            if (stat_anchor) {
                // best mean reward among the arms with enough rewards (this
                // step's update already counted: the updated arm's count and
                // sum are written back only at the end of the step)
                const int2 v = k == a_upd ? make_int2(s_stu.x + 1, __float_as_int(__int_as_float(s_stu.y) + r))
                                          : p.stats[(size_t)inst * K + k];
                if (v.x >= p.rf.min_n) sb = better(sb, BestPair{__int_as_float(v.y) / (float)v.x, k});
            }
        }
        if (sc != nullptr && k < K) {
            sc[k] = u;
            sc[K + k] = act ? s_lcb[k] : -INFINITY;
        }
        if (prune_now) {
            // clear the arms rule 1 removed from the global words (non-sticky:
            // the words become exactly this step's removals, all other arms set)
            const unsigned long long bal = __ballot(keep);
            const int w0 = (base + wave * kWave) >> 5;
            uint32_t *mwo = p.mask + (size_t)inst * KW;
            auto all_arms = [&](int w) {
                return K - 32 * w >= 32 ? 0xffffffffu : (1u << (K - 32 * w)) - 1u;
            };
            if (lane == 0 && w0 < KW) {
                const uint32_t from = reset ? all_arms(w0) : s_raw[w0];
                s_raw[w0] = from & ~(s_mask[w0] & ~(uint32_t)(bal & 0xffffffffull));
                mwo[w0] = s_raw[w0];
            }
            if (lane == 0 && w0 + 1 < KW) {
                const uint32_t from = reset ? all_arms(w0 + 1) : s_raw[w0 + 1];
                s_raw[w0 + 1] = from & ~(s_mask[w0 + 1] & ~(uint32_t)(bal >> 32));
                mwo[w0 + 1] = s_raw[w0 + 1];
            }
        }
    }
    b = wave_best(b);
    if (stat_anchor) sb = wave_best(sb);
    __shared__ float s_top[kMaxWaves][2];
    if (sc != nullptr) {
        // the two largest of a pair of (largest, second) pairs
        auto merge = [&](float o1, float o2) {
            top2 = fmaxf(fminf(top1, o1), fmaxf(top2, o2));
            top1 = fmaxf(top1, o1);
        };
        merge(partner<0>(top1), partner<0>(top2));
        merge(partner<1>(top1), partner<1>(top2));
        merge(partner<2>(top1), partner<2>(top2));
        merge(partner<3>(top1), partner<3>(top2));
        merge(partner<4>(top1), partner<4>(top2));
        merge(partner<5>(top1), partner<5>(top2));
        if (lane == 0) {
            s_top[wave][0] = top1;
            s_top[wave][1] = top2;
        }
    }
    // a one-wavefront workgroup has its results in every lane already
    if constexpr (NW > 1) {
        if (lane == 0) {
            s_red_v[wave] = b.v;
            s_red_k[wave] = b.k;
            s_red_n[wave] = n;
            s_red_v2[wave] = sb.v;
            s_red_k2[wave] = sb.k;
        }
        __syncthreads();
    }
    if (wave == 0) {
        // every lane of wavefront 0 reduces the per-wave results, then the
        // lanes write the instance block (action, count, context) at once
        BestPair best = b;
        int cnt = n;
        if constexpr (NW > 1) {
            best = BestPair{s_red_v[0], s_red_k[0]};
            cnt = s_red_n[0];
            for (int w = 1; w < nwave; ++w) {
                best = better(best, BestPair{s_red_v[w], s_red_k[w]});
                cnt += s_red_n[w];
            }
        }
        const int a = best.k == 0x7fffffff ? -1 : best.k;
        // refinement after the decision: a window of 2*half+1 arms around the
        // anchor, every arm at full resolution, from the next step on
        int anchor = -1;
        if (p.rf.now && a >= 0) {
            if (p.rf.stat) {
                BestPair sbest = sb;
                if constexpr (NW > 1) {
                    sbest = BestPair{s_red_v2[0], s_red_k2[0]};
                    for (int w = 1; w < nwave; ++w) sbest = better(sbest, BestPair{s_red_v2[w], s_red_k2[w]});
                }
                anchor = sbest.k == 0x7fffffff ? -1 : sbest.k;
            } else {
                anchor = a;
            }
        }
        const int nlo = anchor - p.rf.half > 0 ? anchor - p.rf.half : 0;
        const int nhi = anchor + p.rf.half < K - 1 ? anchor + p.rf.half : K - 1;
        if (anchor >= 0) {
            // arms in play in the new space
            int c2 = lane < KW ? __popc(s_raw[lane] & space_bits(lane, nlo, nhi, 1)) : 0;
            c2 = wave_reduce(c2, [](int a, int c) { return a + c; });
            cnt = c2;
        }
        if (lane == 0) {
            if (p.action != nullptr) p.action[inst] = a;
            if (inst == 0) {
                p.hdr->t = p.t_next;
                p.hdr->pending = 1;
            }
        }
        if (lane == kInstAprev) blk[kInstAprev] = a;
        if (lane == kInstKact) blk[kInstKact] = cnt;
        if (sc != nullptr && lane == kInstGap) {
            float t1 = top1, t2 = top2;   // one wavefront: already merged in every lane
            if constexpr (NW > 1) {
                t1 = s_top[0][0];
                t2 = s_top[0][1];
            }
            for (int w = 1; w < nwave; ++w) {
                t2 = fmaxf(fminf(t1, s_top[w][0]), fmaxf(t2, s_top[w][1]));
                t1 = fmaxf(t1, s_top[w][0]);
            }
            blk[kInstGap] = __float_as_int(t1 - t2);   // +inf with one kept arm
        }
        if (anchor >= 0 && lane >= kInstLo && lane <= kInstStride)
            blk[lane] = lane == kInstLo ? nlo : (lane == kInstHi ? nhi : 1);
        if (ph_lane) blk[tid] = s_phw[tid - kInstMode];
        if (lane >= kInstX && lane < kInstX + D)
            reinterpret_cast<float *>(blk)[lane] = s_x[lane - kInstX];
        // the context and reward read at the start are dead by now: the
        // environment's response overwrites them in place
        if constexpr (ENV) agft_env_detail::env_epilogue(env, inst, a, lane, env_pre, s_envw);
    }
    write_back();
}

// ---- initialisation and export ----

struct InitArgs {
    float4 *arms;
    uint32_t *mask;
    int32_t *inst;
    int2 *stats;
    float4 *theta;        // [B][K][d/4] or nullptr
    StateHeader *hdr;
    StateHeader h;
    int32_t B, K, KW, d, C, IW;
    int32_t tf;           // tail floats per lane slice
    int32_t stride0;      // stride of the starting action space
    float inv_sqrt_lambda;
};

__global__ void agft_init_kernel(InitArgs p) {
    const size_t gtid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t gsz = (size_t)gridDim.x * blockDim.x;
    // every chunk of every block, the arms past K of the last block zeroed
    const int nb = 64 / p.d, main = (p.d / 2) * (p.d / 4), tail = (p.d / 2) * p.tf / 4;
    const int blk = nb * p.C;
    const size_t ic = (size_t)((p.K + nb - 1) / nb) * blk;
    for (size_t idx = gtid; idx < (size_t)p.B * ic; idx += gsz) {
        const int o = (int)(idx % ic % blk);
        const int k = (int)(idx % ic / blk) * nb + (o < nb * main ? o / main : (o - nb * main) / tail);
        const int c = o < nb * main ? o % main : main + (o - nb * main) % tail;
        float v[4];
        for (int q = 0; q < 4; ++q) {
            const int ci = k < p.K ? canon_chunk(p.d, p.tf, c, q) : -1;
            v[q] = 0.0f;
            if (ci >= p.d) {
                int i, col;
                unpack(ci - p.d, i, col);
                if (i == col) v[q] = p.inv_sqrt_lambda;
            }
        }
        p.arms[idx] = make_float4(v[0], v[1], v[2], v[3]);
    }
    const size_t nmask = (size_t)p.B * p.KW;
    for (size_t idx = gtid; idx < nmask; idx += gsz) {
        const int w = (int)(idx % p.KW);
        const int rem = p.K - 32 * w;
        p.mask[idx] = rem >= 32 ? 0xffffffffu : ((1u << rem) - 1u);
    }
    for (size_t idx = gtid; idx < (size_t)p.B * p.K; idx += gsz) p.stats[idx] = make_int2(0, 0);
    if (p.theta != nullptr)
        for (size_t idx = gtid; idx < (size_t)p.B * p.K * (p.d / 4); idx += gsz)
            p.theta[idx] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (size_t idx = gtid; idx < (size_t)p.B * p.IW; idx += gsz) {
        const int w = (int)(idx % p.IW);
        const int hi = p.K - 1;
        const int kact0 = (hi - 0) / p.stride0 + 1;   // arms on the starting grid
        p.inst[idx] = w == kInstAprev || w == kInstMode ? -1
                    : w == kInstKact ? kact0
                    : w == kInstPhMargin ? 0x7f800000   // +inf: no test yet
                    : w == kInstHi ? hi
                    : w == kInstStride ? p.stride0
                    : 0;
    }
    if (gtid == 0) *p.hdr = p.h;
}

template <int D, int TF>
__global__ void agft_export_kernel(const float4 *arms, int B, int K, float *theta, float *ainv) {
    using R = Rec<D, TF>;
    const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (size_t)B * K) return;
    float can[R::CAN];
    const float4 *rec = arms + (gid / K) * ((size_t)((K + R::NB - 1) / R::NB) * R::BLK);
    const int k = (int)(gid % K);
    for (int c = 0; c < R::R; ++c) {
        const float4 v = rec[rec_chunk(D, TF, k, c)];
        const float vv[4] = {v.x, v.y, v.z, v.w};
        for (int q = 0; q < 4; ++q) {
            const int ci = canon_chunk(D, TF, c, q);
            if (ci >= 0) can[ci] = vv[q];
        }
    }
    if (theta != nullptr)
        for (int i = 0; i < D; ++i) theta[gid * D + i] = can[i];
    if (ainv != nullptr) {
        const float *S = can + D;
        for (int r = 0; r < D; ++r)
            for (int c = 0; c < D; ++c) {
                float acc = 0.0f;
                for (int jc = (r > c ? r : c); jc < D; ++jc) acc = fmaf(S[packed(r, jc)], S[packed(c, jc)], acc);
                ainv[(gid * D + r) * D + c] = acc;
            }
    }
}

}  // namespace

// ---- C ABI ----

struct agft_handle {
    agft_config cfg;
    Layout lay;
    char *base;
    hipStream_t stream;
    int64_t t;
    int pending;
};

namespace {

bool config_ok(const agft_config *c) {
    if (c == nullptr) return false;
    if (c->B < 1 || c->K < 1 || c->K > kMaxK) return false;
    if (!std::isfinite(c->lambda) || !(c->lambda > 0.0f)) return false;
    if (!std::isfinite(c->alpha0) || c->alpha0 < 0.0f) return false;
    if (c->alpha_sched != 0 && c->alpha_sched != 1) return false;
    if (c->prune_rule < 0 || c->prune_rule > 15) return false;
    if (c->prune_period < 1) return false;
    if (c->prune_sticky != 0 && c->prune_sticky != 1) return false;
    if ((c->prune_rule & 2) && (c->ext_rounds < 0 || c->ext_min_n < 1 || !std::isfinite(c->ext_thr)))
        return false;
    if ((c->prune_rule & 4) && (c->hist_after < 0 || c->hist_min_n < 1 || c->hist_min_arms < 1 ||
                                !std::isfinite(c->hist_kappa) || c->hist_kappa < 0.0f))
        return false;
    if ((c->prune_rule & 8) && (c->cascade_k < 0 || c->cascade_k > c->K)) return false;
    if (c->exploit != 0 && c->exploit != 1) return false;
    if (c->refine != 0 && c->refine != 1) return false;
    if (c->refine && (c->refine_period < 1 || c->refine_stride < 1 || c->refine_half < 0 ||
                      c->refine_mature < 0 || c->refine_min_n < 1))
        return false;
    if (c->exploit && (!std::isfinite(c->ph_delta) || !std::isfinite(c->ph_lambda) || c->ph_lambda < 0.0f ||
                       c->ph_window < 0 || c->ph_min_rounds < 0))
        return false;
    if ((c->flags & ~AGFT_ADOPT_STATE) != 0) return false;
    return true;
}

// Context dimensions the kernels are built for; a non-sticky rule 1 only on
// its own (the paper's rules 2-8 remove arms for good, and one mask cannot
// hold both kinds of removal).
bool supported(const agft_config *c) {
    return (c->d == 8 || c->d == 16 || c->d == 32) && (c->prune_sticky || !(c->prune_rule & 14));
}

int hip_status(hipError_t e) { return e == hipSuccess ? AGFT_OK : AGFT_E_HIP; }

StateHeader make_header(const agft_config *c) {
    StateHeader h;
    std::memset(&h, 0, sizeof(h));
    h.magic = kMagic;
    h.version = AGFT_ABI_VERSION;
    h.B = c->B;
    h.K = c->K;
    h.d = c->d;
    h.chunks = chunks_for(c->d, tail_floats(*c));
    h.tail_floats = tail_floats(*c);
    h.stats_kept = stats_kept(*c) ? 1 : 0;
    h.mask_words = (c->K + 31) / 32;
    h.pending = 0;
    h.t = 0;
    h.lambda = c->lambda;
    h.alpha0 = c->alpha0;
    h.alpha_sched = c->alpha_sched;
    h.prune_rule = c->prune_rule;
    h.prune_period = c->prune_period;
    h.exploit = c->exploit;
    return h;
}

template <class T>
T *at(char *base, size_t off) {
    return reinterpret_cast<T *>(base + off);
}
// agft_sim_step runs the environment in the step kernel's epilogue up to
// this many instances, and launches the step and environment kernels above.
constexpr int kFusedMaxB = 8192;

// Dynamic LDS that caps a kernel at `cap` workgroups per compute unit: a
// 1/cap share of the unit's LDS less the kernel's static LDS, lowered in
// 512-byte steps until the occupancy calculator admits exactly cap
// workgroups (allocation granules round a request up).  Worked out once per
// kernel and device; a share the calculator does not confirm, or below what
// the kernel needs, leaves the launch uncapped.  Only host queries, no
// allocation; the error of a failed query is cleared so that the launch's
// own error check does not see it.
constexpr int kMaxDevices = 64;
template <int D, int TF, int W, int NW, bool ENV>
std::atomic<int64_t> *capped_lds_cache() {
    static std::atomic<int64_t> cache[kMaxDevices];   // 0: not worked out; else bytes + 1
    return cache;
}

size_t capped_lds(const void *kernel, int threads, size_t need, int cap, std::atomic<int64_t> *cache) {
    if (cap <= 0) return need;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return need;
    }
    if (dev < 0 || dev >= kMaxDevices) return need;
    int64_t v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int64_t dyn = 0;   // 0: uncapped
        int per_cu = 0;
        hipFuncAttributes fa;
        bool failed = hipDeviceGetAttribute(&per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
                          hipSuccess ||
                      hipFuncGetAttributes(&fa, kernel) != hipSuccess;
        if (!failed && per_cu > 0) {
            const int64_t max_dyn = 64 * 1024 - (int64_t)fa.sharedSizeBytes;
            for (int64_t d = (per_cu / cap - (int64_t)fa.sharedSizeBytes) / 16 * 16; d >= (int64_t)need && d > 0;
                 d -= 512) {
                if (d > max_dyn) continue;
                int blocks = 0;
                if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, threads, (size_t)d) != hipSuccess) {
                    failed = true;
                    break;
                }
                if (blocks == cap) {
                    dyn = d;
                    break;
                }
                if (blocks > cap) break;
            }
        }
        if (failed) (void)hipGetLastError();
        v = dyn + 1;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    // (a share worked out for a smaller need than this launch's is not used)
    return v > 1 && (size_t)(v - 1) >= need ? (size_t)(v - 1) : need;
}

// The step kernel for one or four wavefronts per workgroup (the two widths
// waves_for chooses), each compiled for its width.
template <int D, int TF, int W, bool ENV>
void launch_width(int waves, int cap, unsigned grid, size_t lds, hipStream_t stream, const StepArgs &p,
                  const agft_env_detail::EnvArgs &e) {
    if (waves == 1) {
        hipLaunchKernelGGL((agft_step_kernel<D, TF, W, 1, ENV>), dim3(grid), dim3(kWave), lds, stream, p, e);
    } else {
        lds = capped_lds(reinterpret_cast<const void *>(&agft_step_kernel<D, TF, W, 4, ENV>), 4 * kWave, lds, cap,
                         capped_lds_cache<D, TF, W, 4, ENV>());
        hipLaunchKernelGGL((agft_step_kernel<D, TF, W, 4, ENV>), dim3(grid), dim3(4 * kWave), lds, stream, p, e);
    }
}

// One decision for every instance of handle h (and, with env, the
// environment's response): arguments checked by the caller.
int launch_step(agft_handle *h, const float *d_ctx, const float *d_reward, int32_t *d_action, float *d_scores,
                const agft_env_detail::EnvArgs *env) {
    const agft_config &c = h->cfg;
    StepArgs p;
    p.arms = at<float4>(h->base, h->lay.arms);
    p.mask = at<uint32_t>(h->base, h->lay.mask);
    p.inst = at<int32_t>(h->base, h->lay.inst);
    p.stats = at<int2>(h->base, h->lay.stats);
    p.theta = c.exploit ? at<float>(h->base, h->lay.theta) : nullptr;
    p.h.mask = c.prune_rule & 14;
    p.h.ext_rounds = c.ext_rounds;
    p.h.ext_min_n = c.ext_min_n;
    p.h.ext_thr = c.ext_thr;
    p.h.hist_after = c.hist_after;
    p.h.hist_min_n = c.hist_min_n;
    p.h.hist_kappa = c.hist_kappa;
    p.h.hist_min_arms = c.hist_min_arms;
    p.h.cascade_k = c.cascade_k;
    p.t = h->t;
    p.e.on = c.exploit;
    p.e.delta = c.ph_delta;
    p.e.lambda = c.ph_lambda;
    p.e.window = c.ph_window;
    p.e.min_rounds = c.ph_min_rounds;
    p.rf.now = (c.refine && d_ctx != nullptr && h->t > 0 && h->t % c.refine_period == 0) ? 1 : 0;
    p.rf.stat = h->t < c.refine_mature ? 1 : 0;
    p.rf.half = c.refine_half;
    p.rf.min_n = c.refine_min_n;
    p.hdr = at<StateHeader>(h->base, 0);
    p.ctx = d_ctx;
    p.reward = d_reward;
    p.action = d_ctx != nullptr ? d_action : nullptr;
    p.scores = d_ctx != nullptr ? d_scores : nullptr;
    p.B = c.B;
    p.K = c.K;
    p.KW = (c.K + 31) / 32;
    p.IW = inst_words(c.d);
    p.apply_update = h->pending;
    const int64_t t = h->t;
    p.prune_now = (d_ctx != nullptr && (c.prune_rule & 1) && t > 0 && t % c.prune_period == 0) ? 1 : 0;
    p.prune_reset = p.prune_now && !c.prune_sticky ? 1 : 0;
    p.alpha = c.alpha_sched == 0 ? c.alpha0 : (float)((double)c.alpha0 / std::sqrt((double)t + 1.0));
    p.t_next = d_ctx != nullptr ? t + 1 : t;
    agft_launch_shape shape;
    agft_launch_shape_for(&c, &shape);
    const int waves = waves_at(c, t);
    p.early_update = shape.early_update;
    p.keep_stats = stats_kept(c) ? 1 : 0;
    if (waves != 1 && waves != 4) return AGFT_E_UNSUPPORTED;
    const unsigned grid = (unsigned)c.B;
    const size_t lds = step_lds_bytes(c.K);
    const bool packed_tails = shape.tail_floats == 3;
    hipStream_t s = h->stream;
    agft_env_detail::EnvArgs e{};
    if (env != nullptr) e = *env;
    // The simulator's single launch runs uncapped: the environment's
    // response at the end of each workgroup wants more instances in flight
    // (K=128 d=16, us per fused step, uncapped / at 4, measured when larger
    // batches took the single launch too: B=65,536 881.5 / 891.0, B=16,384
    // 211.9 / 218.0).
    const int cap = env != nullptr ? 0 : cu_workgroups_for(waves, shape.simd_waves);
#define AGFT_LAUNCH(D_, TF_, W_)                                                       \
    (env != nullptr ? launch_width<D_, TF_, W_, true>(waves, cap, grid, lds, s, p, e) \
                    : launch_width<D_, TF_, W_, false>(waves, cap, grid, lds, s, p, e))
    switch (c.d) {
        case 8:
            if (packed_tails) AGFT_LAUNCH(8, 3, 7);
            else AGFT_LAUNCH(8, 4, 7);
            break;
        case 16:
            if (packed_tails && shape.simd_waves == 6) AGFT_LAUNCH(16, 3, 6);
            else if (packed_tails) AGFT_LAUNCH(16, 3, 7);
            else AGFT_LAUNCH(16, 4, 7);
            break;
        case 32:
            if (packed_tails) AGFT_LAUNCH(32, 3, 4);
            else AGFT_LAUNCH(32, 4, 4);
            break;
        default: return AGFT_E_UNSUPPORTED;
    }
#undef AGFT_LAUNCH
    if (hipGetLastError() != hipSuccess) return AGFT_E_HIP;
    if (d_ctx != nullptr) {
        h->t = t + 1;
        h->pending = 1;
    } else {
        h->pending = 0;
    }
    return AGFT_OK;
}

}  // namespace

extern "C" {

size_t agft_state_bytes(const agft_config *cfg) {
    if (!config_ok(cfg) || !supported(cfg)) return 0;
    return layout_for(*cfg).total;
}

int agft_create(const agft_config *cfg, void *d_state, size_t nbytes, void *stream, agft_handle **out) {
    if (out == nullptr) return AGFT_E_INVAL;
    *out = nullptr;
    if (!config_ok(cfg) || d_state == nullptr) return AGFT_E_INVAL;
    if (!supported(cfg)) return AGFT_E_UNSUPPORTED;
    if (reinterpret_cast<uintptr_t>(d_state) % kAlign != 0) return AGFT_E_INVAL;
    const Layout lay = layout_for(*cfg);
    if (nbytes < lay.total) return AGFT_E_INVAL;
    agft_handle *h = new (std::nothrow) agft_handle;
    if (h == nullptr) return AGFT_E_INVAL;
    h->cfg = *cfg;
    h->lay = lay;
    h->base = static_cast<char *>(d_state);
    h->stream = static_cast<hipStream_t>(stream);
    h->t = 0;
    h->pending = 0;
    const StateHeader want = make_header(cfg);
    if (cfg->flags & AGFT_ADOPT_STATE) {
        StateHeader got;
        hipError_t e = hipMemcpyAsync(&got, d_state, sizeof(got), hipMemcpyDeviceToHost, h->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
        if (e != hipSuccess) {
            delete h;
            return AGFT_E_HIP;
        }
        if (got.magic != kMagic || got.version != want.version || got.B != want.B || got.K != want.K ||
            got.d != want.d || got.chunks != want.chunks || got.tail_floats != want.tail_floats ||
            got.stats_kept != want.stats_kept ||
            got.exploit != want.exploit || got.t < 0 ||
            (got.pending != 0 && got.pending != 1)) {
            delete h;
            return AGFT_E_STATE;
        }
        h->t = got.t;
        h->pending = got.pending;
        *out = h;
        return AGFT_OK;
    }
    InitArgs a;
    a.arms = at<float4>(h->base, lay.arms);
    a.mask = at<uint32_t>(h->base, lay.mask);
    a.inst = at<int32_t>(h->base, lay.inst);
    a.stats = at<int2>(h->base, lay.stats);
    a.theta = cfg->exploit ? at<float4>(h->base, lay.theta) : nullptr;
    a.hdr = at<StateHeader>(h->base, 0);
    a.h = want;
    a.B = cfg->B;
    a.K = cfg->K;
    a.KW = (cfg->K + 31) / 32;
    a.d = cfg->d;
    a.tf = tail_floats(*cfg);
    a.C = chunks_for(cfg->d, a.tf);
    a.IW = inst_words(cfg->d);
    a.stride0 = cfg->refine ? cfg->refine_stride : 1;
    a.inv_sqrt_lambda = (float)(1.0 / std::sqrt((double)cfg->lambda));
    const size_t work = (size_t)cfg->B * a.C * cfg->K;
    size_t blocks = (work + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(agft_init_kernel, dim3((unsigned)blocks), dim3(256), 0, h->stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        delete h;
        return AGFT_E_HIP;
    }
    *out = h;
    return AGFT_OK;
}

int agft_step(agft_handle *h, const float *d_ctx, const float *d_reward, int32_t *d_action, float *d_scores) {
    if (h == nullptr) return AGFT_E_INVAL;
    if (h->pending && d_reward == nullptr) return AGFT_E_STATE;
    return launch_step(h, d_ctx, d_reward, d_action, d_scores, nullptr);
}

int agft_sim_step(agft_handle *h, const agft_env_config *env_cfg, void *d_env, size_t env_nbytes,
                  const int32_t *d_arrivals, const float *d_noise, float *d_ctx, float *d_reward,
                  int32_t *d_action, float *d_scores) {
    using namespace agft_env_detail;
    if (h == nullptr || !env_config_ok(env_cfg)) return AGFT_E_INVAL;
    if (env_cfg->B != h->cfg.B || env_cfg->K != h->cfg.K || env_cfg->d != h->cfg.d) return AGFT_E_INVAL;
    if (d_env == nullptr || d_arrivals == nullptr || d_noise == nullptr || d_ctx == nullptr ||
        d_reward == nullptr || d_action == nullptr)
        return AGFT_E_INVAL;
    if (reinterpret_cast<uintptr_t>(d_ctx) % 16 != 0) return AGFT_E_INVAL;
    if (reinterpret_cast<uintptr_t>(d_env) % agft_env_detail::kAlign != 0 || env_nbytes < env_layout(env_cfg->B).total)
        return AGFT_E_INVAL;
    if (h->t >= env_cfg->T) return AGFT_E_STATE;   // the draws end at window T
    // Large batches take the step kernel and then the environment kernel:
    // there the epilogue's per-instance stores to the environment's
    // structure-of-arrays state cost more than the launch they save.
    // Measured on MI355X (us per simulator step over the whole horizon,
    // fused / two launches): K=128 d=16 B=65,536 879 / 814, B=16,384 211 /
    // 201; K=64 d=8 B=4,096 16.1 / 18.5; K=256 d=32 B=1,024 23.4 / 27.1.
    if (h->cfg.B > kFusedMaxB) {
        const int64_t t = h->t;
        const int rc = launch_step(h, d_ctx, d_reward, d_action, d_scores, nullptr);
        if (rc != AGFT_OK) return rc;
        return agft_env_step(env_cfg, d_env, env_nbytes, (int32_t)t, d_action, d_arrivals, d_noise, d_reward, d_ctx,
                             h->stream);
    }
    EnvArgs e = make_args(env_cfg, d_env);
    e.arrivals = d_arrivals;
    e.noise = d_noise;
    e.action = d_action;
    e.reward = d_reward;
    e.ctx = d_ctx;
    e.w = (int32_t)h->t + 1;
    const double tau = env_cfg->T > 1 ? (double)h->t / (double)(env_cfg->T - 1) : 0.0;
    e.scale = (float)(1.0 + (double)env_cfg->drift * tau);
    e.reset = 0;
    return launch_step(h, d_ctx, d_reward, d_action, d_scores, &e);
}

int agft_launch_shape_for(const agft_config *cfg, agft_launch_shape *out) {
    if (out == nullptr || !config_ok(cfg)) return AGFT_E_INVAL;
    if (!supported(cfg)) return AGFT_E_UNSUPPORTED;
    out->waves = waves_for(*cfg);
    out->tail_floats = tail_floats(*cfg);
    out->simd_waves = occupancy_for(*cfg, out->tail_floats);
    out->early_update = early_update(*cfg) ? 1 : 0;
    out->cu_workgroups = cu_workgroups_for(out->waves, out->simd_waves);
    return AGFT_OK;
}

int agft_get_state(const agft_handle *h, agft_state_view *out) {
    if (h == nullptr || out == nullptr) return AGFT_E_INVAL;
    out->t = h->t;
    out->pending = h->pending;
    out->B = h->cfg.B;
    out->K = h->cfg.K;
    out->d = h->cfg.d;
    out->tail_floats = tail_floats(h->cfg);
    out->chunks = chunks_for(h->cfg.d, out->tail_floats);
    out->block_arms = block_arms(h->cfg.d);
    out->mask_words = (h->cfg.K + 31) / 32;
    out->arms = h->base + h->lay.arms;
    out->mask = at<uint32_t>(h->base, h->lay.mask);
    out->inst = at<int32_t>(h->base, h->lay.inst);
    out->inst_words = inst_words(h->cfg.d);
    out->stats = at<int32_t>(h->base, h->lay.stats);
    out->theta = h->cfg.exploit ? at<float>(h->base, h->lay.theta) : nullptr;
    return AGFT_OK;
}

int agft_export(agft_handle *h, float *d_theta, float *d_ainv) {
    if (h == nullptr) return AGFT_E_INVAL;
    if (d_theta == nullptr && d_ainv == nullptr) return AGFT_OK;
    const agft_config &c = h->cfg;
    const size_t n = (size_t)c.B * c.K;
    const dim3 grid((unsigned)((n + 127) / 128)), block(128);
    const float4 *arms = at<float4>(h->base, h->lay.arms);
    const bool packed_tails = tail_floats(c) == 3;
    switch (c.d) {
        case 8:
            if (packed_tails) hipLaunchKernelGGL((agft_export_kernel<8, 3>), grid, block, 0, h->stream, arms, c.B, c.K, d_theta, d_ainv);
            else hipLaunchKernelGGL((agft_export_kernel<8, 4>), grid, block, 0, h->stream, arms, c.B, c.K, d_theta, d_ainv);
            break;
        case 16:
            if (packed_tails) hipLaunchKernelGGL((agft_export_kernel<16, 3>), grid, block, 0, h->stream, arms, c.B, c.K, d_theta, d_ainv);
            else hipLaunchKernelGGL((agft_export_kernel<16, 4>), grid, block, 0, h->stream, arms, c.B, c.K, d_theta, d_ainv);
            break;
        case 32:
            if (packed_tails) hipLaunchKernelGGL((agft_export_kernel<32, 3>), grid, block, 0, h->stream, arms, c.B, c.K, d_theta, d_ainv);
            else hipLaunchKernelGGL((agft_export_kernel<32, 4>), grid, block, 0, h->stream, arms, c.B, c.K, d_theta, d_ainv);
            break;
        default: return AGFT_E_UNSUPPORTED;
    }
    return hip_status(hipGetLastError());
}

int agft_set_stream(agft_handle *h, void *stream) {
    if (h == nullptr) return AGFT_E_INVAL;
    h->stream = static_cast<hipStream_t>(stream);
    return AGFT_OK;
}

int agft_destroy(agft_handle *h) {
    delete h;
    return AGFT_OK;
}

const char *agft_strerror(int code) {
    switch (code) {
        case AGFT_OK: return "ok";
        case AGFT_E_INVAL: return "invalid argument";
        case AGFT_E_UNSUPPORTED: return "unsupported configuration";
        case AGFT_E_STATE: return "call not valid in the current state";
        case AGFT_E_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

int agft_abi_version(void) { return AGFT_ABI_VERSION; }

}  // extern "C"
