// agft_env.hip -- synthetic serving environment of the batched tuner, one
// thread per instance.  The closed form is stated in agft_sim.h.  Per-instance
// state is kept structure-of-arrays so that a wavefront's 64 instances read
// and write contiguous words; the exogenous draws are time-major [T+1][B]
// for the same reason.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "agft.h"
#include "agft_env_math.h"

namespace agft_env_detail {
constexpr int kEnvThreads = 256;

// One thread per instance.  Each context goes through LDS so that the
// block's contexts (contiguous in the output) leave as whole-line float4
// stores rather than d strided words per thread.
__global__ __launch_bounds__(kEnvThreads) void agft_env_kernel(EnvArgs p) {
    __shared__ float4 s_ctx[kEnvThreads * 32 / 4];
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < p.B) env_instance(p, i, p.reset ? -1 : p.action[i], s_ctx + threadIdx.x * (p.d / 4));
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

namespace {

int launch(const EnvArgs &p, void *stream) {
    const unsigned blocks = (unsigned)((p.B + kEnvThreads - 1) / kEnvThreads);
    hipLaunchKernelGGL(agft_env_kernel, dim3(blocks), dim3(kEnvThreads), 0, static_cast<hipStream_t>(stream), p);
    return hipGetLastError() == hipSuccess ? AGFT_OK : AGFT_E_HIP;
}

}  // namespace
}  // namespace agft_env_detail

using namespace agft_env_detail;

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
