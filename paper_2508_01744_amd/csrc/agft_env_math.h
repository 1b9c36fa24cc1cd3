// agft_env_math.h -- internal to libagft: the synthetic serving
// environment's per-instance closed form (stated in agft_sim.h) and its
// state layout, shared by the environment kernel and by the step kernel's
// fused simulator epilogue.
#ifndef AGFT_ENV_MATH_H
#define AGFT_ENV_MATH_H

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "agft_sim.h"

namespace agft_env_detail {

constexpr size_t kAlign = 256;
constexpr int kZ = 7;      // raw features per window
constexpr int kZLags = 4;  // z_t .. z_{t-3}
constexpr int kRLags = 3;  // rho_t .. rho_{t-2}

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct EnvLayout {
    size_t q, cap, f, zh, rh, total;
};

inline EnvLayout env_layout(int B) {
    EnvLayout L;
    const size_t b = (size_t)B;
    size_t off = 0;
    L.q = off;   off = align_up(off + b * 4);
    L.cap = off; off = align_up(off + b * 4);
    L.f = off;   off = align_up(off + b * 4);
    L.zh = off;  off = align_up(off + b * kZLags * kZ * 4);
    L.rh = off;  off = align_up(off + b * kRLags * 4);
    L.total = off;
    return L;
}

struct EnvArgs {
    int32_t *q;
    int32_t *cap;
    float *f;
    float *zh;  // [kZLags][kZ][B], lag 0 = most recent
    float *rh;  // [kRLags][B]
    const int32_t *arrivals;
    const float *noise;
    const int32_t *action;
    float *reward;
    float *ctx;
    int32_t B, K, d, w;  // window index
    float scale;         // 1 + drift * tau of this window
    float P0, c, l0, a, b, lat_min, f_lo, f_hi, f_init, tpot_div;
    int32_t svc_lo, svc_hi, svc_init, q_cap, run_cap;
    float mu[kZ], inv_sd[kZ];
    int32_t reset;
};

__device__ inline float arm_clock(const EnvArgs &p, int k) {
    if (p.K == 1) return p.f_hi;
    return p.f_lo + (p.f_hi - p.f_lo) * (float)k / (float)(p.K - 1);
}

__device__ inline int arm_capacity(const EnvArgs &p, int k) {
    if (p.K == 1) return p.svc_hi;
    const long long num = (long long)p.svc_lo * (p.K - 1) + (long long)(p.svc_hi - p.svc_lo) * k;
    const long long den = p.K - 1;
    return (int)((2 * num + den) / (2 * den));
}

// The closed form of one window: from the queue q, capacity cap and clock f
// in force and the decision a (-1 or out of range: the previous clock), the
// window's state (queue, capacity, clock), reward rho and features z.
struct Window {
    int q, cap;
    float f, rho;
    float z[kZ];
};

__device__ __forceinline__ Window env_window(const EnvArgs &p, int q, int cap, float f, int a, int n, float eta) {
    if (a >= 0 && a < p.K) {
        f = arm_clock(p, a);
        cap = arm_capacity(p, a);
    }
    const float nf = (float)n;
    const float bw = p.b * p.scale, cw = p.c * p.scale;
    const float lat = fmaxf(p.lat_min, p.l0 * (p.a + bw * nf / f) + eta);
    const float power = p.P0 + cw * f * f * f;
    const float lat_ref = p.l0 * (p.a + bw * nf);
    Window o;
    o.rho = -(power * lat * lat) / ((p.P0 + cw) * lat_ref * lat_ref);
    int qn = q + n - cap;
    qn = qn < 0 ? 0 : qn;
    qn = qn > p.q_cap ? p.q_cap : qn;
    int running = qn + n;
    running = running > p.run_cap ? p.run_cap : running;
    const float capf = (float)cap;
    const float ttft = lat * (1.0f + (float)qn / capf);
    const float raw[kZ] = {nf, log1pf((float)qn), (float)running, logf(ttft), lat / p.tpot_div,
                           fminf(1.0f, nf / capf), f};
#pragma unroll
    for (int j = 0; j < kZ; ++j) o.z[j] = (raw[j] - p.mu[j]) * p.inv_sd[j];
    o.q = qn;
    o.cap = cap;
    o.f = f;
    return o;
}

// One instance's window run at the clock of action a: state update, reward
// and the next context, which goes to xs (d/4 float4 slots).
__device__ __forceinline__ void env_instance(const EnvArgs &p, int i, int a, float4 *xs) {
    const size_t B = (size_t)p.B;
    const int n = p.arrivals[(size_t)p.w * B + i];
    const float eta = p.noise[(size_t)p.w * B + i];
    const Window wnd = p.reset ? env_window(p, 0, p.svc_init, p.f_init, -1, n, eta)
                               : env_window(p, p.q[i], p.cap[i], p.f[i], a, n, eta);
    const float rho = wnd.rho;
    const int qn = wnd.q, cap = wnd.cap;
    const float f = wnd.f;
    float z[kZ];
#pragma unroll
    for (int j = 0; j < kZ; ++j) z[j] = wnd.z[j];

    float zl[kZLags][kZ];
    float rl[kRLags];
    if (p.reset) {
#pragma unroll
        for (int l = 0; l < kZLags; ++l)
#pragma unroll
            for (int j = 0; j < kZ; ++j) zl[l][j] = z[j];
#pragma unroll
        for (int l = 0; l < kRLags; ++l) rl[l] = rho;
    } else {
#pragma unroll
        for (int l = kZLags - 1; l > 0; --l)
#pragma unroll
            for (int j = 0; j < kZ; ++j) zl[l][j] = p.zh[((size_t)(l - 1) * kZ + j) * B + i];
#pragma unroll
        for (int j = 0; j < kZ; ++j) zl[0][j] = z[j];
#pragma unroll
        for (int l = kRLags - 1; l > 0; --l) rl[l] = p.rh[(size_t)(l - 1) * B + i];
        rl[0] = rho;
        p.reward[i] = rho;
    }
#pragma unroll
    for (int l = 0; l < kZLags; ++l)
#pragma unroll
        for (int j = 0; j < kZ; ++j) p.zh[((size_t)l * kZ + j) * B + i] = zl[l][j];
#pragma unroll
    for (int l = 0; l < kRLags; ++l) p.rh[(size_t)l * B + i] = rl[l];
    p.q[i] = qn;
    p.cap[i] = cap;
    p.f[i] = f;

    float x[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) x[k] = 0.0f;
    x[0] = 1.0f;
#pragma unroll
    for (int j = 0; j < kZ; ++j) x[1 + j] = zl[0][j];
    if (p.d == 16) {
#pragma unroll
        for (int j = 0; j < kZ; ++j) x[8 + j] = zl[1][j];
        x[15] = rl[0];
    } else if (p.d == 32) {
#pragma unroll
        for (int l = 1; l < kZLags; ++l)
#pragma unroll
            for (int j = 0; j < kZ; ++j) x[1 + l * kZ + j] = zl[l][j];
#pragma unroll
        for (int l = 0; l < kRLags; ++l) x[29 + l] = rl[l];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
        if (4 * q < p.d) xs[q] = make_float4(x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]);
}

// The same window for instance i spread over the first 32 lanes of a
// wavefront (the step kernel's epilogue).  Each lane prefetches one word of
// the instance's state early (env_prefetch), so that the epilogue only
// computes and stores: lanes 0-4 the queue, capacity, clock, arrivals and
// latency noise, lane 8 + 7(l-1) + j feature j of lag l-1 (l = 1..3, the
// lags to be shifted one place), lanes 30 and 31 rewards of lags 0 and 1.
// Lane e < d then writes element e of the next context: with this numbering
// a shifted feature or reward sits in the lane of its place in the context.
__device__ __forceinline__ uint32_t env_prefetch(const EnvArgs &p, int i, int lane) {
    const size_t B = (size_t)p.B, w = (size_t)p.w;
    const void *src = nullptr;
    if (lane == 0) src = p.q + i;
    else if (lane == 1) src = p.cap + i;
    else if (lane == 2) src = p.f + i;
    else if (lane == 3) src = p.arrivals + w * B + i;
    else if (lane == 4) src = p.noise + w * B + i;
    else if (lane >= 8 && lane < 8 + (kZLags - 1) * kZ) src = p.zh + (size_t)(lane - 8) * B + i;
    else if (lane == 30 || lane == 31) src = p.rh + (size_t)(lane - 30) * B + i;
    return src != nullptr ? *static_cast<const uint32_t *>(src) : 0u;
}

// s_w: 32 words of LDS private to the calling wavefront; a: the decision.
// Every lane of the wavefront calls it.
__device__ __forceinline__ void env_epilogue(const EnvArgs &p, int i, int a, int lane, uint32_t pre,
                                             uint32_t *s_w) {
    const size_t B = (size_t)p.B;
    if (lane < 32) s_w[lane] = pre;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane == 0) {
        const Window wnd = env_window(p, (int)s_w[0], (int)s_w[1], __uint_as_float(s_w[2]), a, (int)s_w[3],
                                      __uint_as_float(s_w[4]));
        p.q[i] = wnd.q;
        p.cap[i] = wnd.cap;
        p.f[i] = wnd.f;
        p.reward[i] = wnd.rho;
        p.rh[i] = wnd.rho;
#pragma unroll
        for (int j = 0; j < kZ; ++j) {
            p.zh[(size_t)j * B + i] = wnd.z[j];
            s_w[1 + j] = __float_as_uint(wnd.z[j]);
        }
        s_w[0] = __float_as_uint(1.0f);
        s_w[p.d == 16 ? 15 : 29] = __float_as_uint(wnd.rho);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // lags move one place; the next context leaves as d contiguous words
    if (lane >= 8 && lane < 8 + (kZLags - 1) * kZ) p.zh[(size_t)(lane - 8 + kZ) * B + i] = __uint_as_float(pre);
    if (lane == 30 || lane == 31) p.rh[(size_t)(lane - 29) * B + i] = __uint_as_float(pre);
    if (lane < p.d) {
        const bool own = lane >= 8 && !(p.d == 16 && lane == 15) && lane != 29;
        p.ctx[(size_t)i * p.d + lane] = own ? __uint_as_float(pre) : __uint_as_float(s_w[lane]);
    }
}

// Validation and kernel arguments of a configuration (agft_env.hip).
bool env_config_ok(const agft_env_config *c);
EnvArgs make_args(const agft_env_config *c, void *d_env);

}  // namespace agft_env_detail

#endif  // AGFT_ENV_MATH_H
