// agft_env.hip -- synthetic serving environment of the batched tuner, one
// thread per instance.  The closed form is stated in agft_sim.h.  Per-instance
// state is kept structure-of-arrays so that a wavefront's 64 instances read
// and write contiguous words; the exogenous draws are time-major [T+1][B]
// for the same reason.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "agft.h"
#include "agft_sim.h"

namespace {

constexpr size_t kAlign = 256;
constexpr int kZ = 7;      // raw features per window
constexpr int kZLags = 4;  // z_t .. z_{t-3}
constexpr int kRLags = 3;  // rho_t .. rho_{t-2}

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct EnvLayout {
    size_t q, cap, f, zh, rh, total;
};

EnvLayout env_layout(int B) {
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

constexpr int kEnvThreads = 256;

// One instance's window: state update, reward and the next context, which
// goes to xs (d/4 float4 slots).
__device__ __forceinline__ void env_instance(const EnvArgs &p, int i, float4 *xs) {
    const size_t B = (size_t)p.B;
    int q, cap;
    float f;
    if (p.reset) {
        q = 0;
        cap = p.svc_init;
        f = p.f_init;
    } else {
        q = p.q[i];
        cap = p.cap[i];
        f = p.f[i];
        const int a = p.action[i];
        if (a >= 0 && a < p.K) {
            f = arm_clock(p, a);
            cap = arm_capacity(p, a);
        }
    }
    const int n = p.arrivals[(size_t)p.w * B + i];
    const float eta = p.noise[(size_t)p.w * B + i];
    const float nf = (float)n;
    const float bw = p.b * p.scale, cw = p.c * p.scale;
    const float lat = fmaxf(p.lat_min, p.l0 * (p.a + bw * nf / f) + eta);
    const float power = p.P0 + cw * f * f * f;
    const float lat_ref = p.l0 * (p.a + bw * nf);
    const float rho = -(power * lat * lat) / ((p.P0 + cw) * lat_ref * lat_ref);
    int qn = q + n - cap;
    qn = qn < 0 ? 0 : qn;
    qn = qn > p.q_cap ? p.q_cap : qn;
    int running = qn + n;
    running = running > p.run_cap ? p.run_cap : running;
    const float capf = (float)cap;
    const float ttft = lat * (1.0f + (float)qn / capf);
    const float raw[kZ] = {nf, log1pf((float)qn), (float)running, logf(ttft), lat / p.tpot_div,
                           fminf(1.0f, nf / capf), f};
    float z[kZ];
#pragma unroll
    for (int j = 0; j < kZ; ++j) z[j] = (raw[j] - p.mu[j]) * p.inv_sd[j];

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

// One thread per instance.  Each context goes through LDS so that the
// block's contexts (contiguous in the output) leave as whole-line float4
// stores rather than d strided words per thread.
__global__ __launch_bounds__(kEnvThreads) void agft_env_kernel(EnvArgs p) {
    __shared__ float4 s_ctx[kEnvThreads * 32 / 4];
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < p.B) env_instance(p, i, s_ctx + threadIdx.x * (p.d / 4));
    __syncthreads();
    const int i0 = blockIdx.x * blockDim.x;
    const int n = p.B - i0 < (int)blockDim.x ? p.B - i0 : (int)blockDim.x;
    float4 *dst = reinterpret_cast<float4 *>(p.ctx + (size_t)i0 * p.d);
    for (int c = threadIdx.x; c < n * p.d / 4; c += blockDim.x) dst[c] = s_ctx[c];
}

bool env_config_ok(const agft_env_config *c) {
    if (c == nullptr) return false;
    if (c->B < 1 || c->K < 1 || c->K > 1024 || c->T < 1) return false;
    if (c->d != 8 && c->d != 16 && c->d != 32) return false;
    if (!(c->lat_min > 0.0f) || !(c->f_lo > 0.0f) || !(c->f_hi >= c->f_lo) || !(c->f_init > 0.0f))
        return false;
    if (!(c->tpot_div > 0.0f)) return false;
    if (c->svc_lo < 1 || c->svc_hi < c->svc_lo || c->svc_init < 1) return false;
    if (c->q_cap < 0 || c->run_cap < 0) return false;
    for (int j = 0; j < kZ; ++j)
        if (!(c->sd[j] > 0.0f) || !std::isfinite(c->mu[j])) return false;
    const float vals[] = {c->P0, c->c, c->l0, c->a, c->b, c->drift};
    for (float v : vals)
        if (!std::isfinite(v)) return false;
    return true;
}

EnvArgs make_args(const agft_env_config *c, void *d_env) {
    const EnvLayout L = env_layout(c->B);
    char *base = static_cast<char *>(d_env);
    EnvArgs p;
    p.q = reinterpret_cast<int32_t *>(base + L.q);
    p.cap = reinterpret_cast<int32_t *>(base + L.cap);
    p.f = reinterpret_cast<float *>(base + L.f);
    p.zh = reinterpret_cast<float *>(base + L.zh);
    p.rh = reinterpret_cast<float *>(base + L.rh);
    p.B = c->B;
    p.K = c->K;
    p.d = c->d;
    p.P0 = c->P0;
    p.c = c->c;
    p.l0 = c->l0;
    p.a = c->a;
    p.b = c->b;
    p.lat_min = c->lat_min;
    p.f_lo = c->f_lo;
    p.f_hi = c->f_hi;
    p.f_init = c->f_init;
    p.tpot_div = c->tpot_div;
    p.svc_lo = c->svc_lo;
    p.svc_hi = c->svc_hi;
    p.svc_init = c->svc_init;
    p.q_cap = c->q_cap;
    p.run_cap = c->run_cap;
    for (int j = 0; j < kZ; ++j) {
        p.mu[j] = c->mu[j];
        p.inv_sd[j] = (float)(1.0 / (double)c->sd[j]);
    }
    return p;
}

int launch(const EnvArgs &p, void *stream) {
    const unsigned blocks = (unsigned)((p.B + kEnvThreads - 1) / kEnvThreads);
    hipLaunchKernelGGL(agft_env_kernel, dim3(blocks), dim3(kEnvThreads), 0, static_cast<hipStream_t>(stream), p);
    return hipGetLastError() == hipSuccess ? AGFT_OK : AGFT_E_HIP;
}

}  // namespace

extern "C" {

size_t agft_env_state_bytes(const agft_env_config *cfg) {
    if (!env_config_ok(cfg)) return 0;
    return env_layout(cfg->B).total;
}

int agft_env_reset(const agft_env_config *cfg, void *d_env, size_t nbytes, const int32_t *d_arrivals,
                   const float *d_noise, float *d_ctx, void *stream) {
    if (!env_config_ok(cfg)) return AGFT_E_INVAL;
    if (d_env == nullptr || d_arrivals == nullptr || d_noise == nullptr || d_ctx == nullptr)
        return AGFT_E_INVAL;
    if (reinterpret_cast<uintptr_t>(d_ctx) % 16 != 0) return AGFT_E_INVAL;
    if (reinterpret_cast<uintptr_t>(d_env) % kAlign != 0 || nbytes < env_layout(cfg->B).total)
        return AGFT_E_INVAL;
    EnvArgs p = make_args(cfg, d_env);
    p.arrivals = d_arrivals;
    p.noise = d_noise;
    p.action = nullptr;
    p.reward = nullptr;
    p.ctx = d_ctx;
    p.w = 0;
    p.scale = 1.0f;
    p.reset = 1;
    return launch(p, stream);
}

int agft_env_step(const agft_env_config *cfg, void *d_env, size_t nbytes, int32_t t,
                  const int32_t *d_action, const int32_t *d_arrivals, const float *d_noise,
                  float *d_reward, float *d_ctx, void *stream) {
    if (!env_config_ok(cfg)) return AGFT_E_INVAL;
    if (d_env == nullptr || d_action == nullptr || d_arrivals == nullptr || d_noise == nullptr ||
        d_reward == nullptr || d_ctx == nullptr)
        return AGFT_E_INVAL;
    if (reinterpret_cast<uintptr_t>(d_ctx) % 16 != 0) return AGFT_E_INVAL;
    if (reinterpret_cast<uintptr_t>(d_env) % kAlign != 0 || nbytes < env_layout(cfg->B).total)
        return AGFT_E_INVAL;
    if (t < 0 || t >= cfg->T) return AGFT_E_INVAL;
    EnvArgs p = make_args(cfg, d_env);
    p.arrivals = d_arrivals;
    p.noise = d_noise;
    p.action = d_action;
    p.reward = d_reward;
    p.ctx = d_ctx;
    p.w = t + 1;
    const double tau = cfg->T > 1 ? (double)t / (double)(cfg->T - 1) : 0.0;
    p.scale = (float)(1.0 + (double)cfg->drift * tau);
    p.reset = 0;
    return launch(p, stream);
}

}  // extern "C"
