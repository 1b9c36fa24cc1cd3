/*
 * agft_sim.h -- C ABI of the synthetic serving environment that drives the
 * batched AGFT tuner on the GPU (one thread per tuner instance).
 *
 * The paper's controller reads live serving metrics and measures energy and
 * latency over each sampling window (Sec. 4.1, Sec. 4.2).  Here each instance
 * is a closed-form model of a serving node: per window w, with arrivals n,
 * latency noise eta and normalised clock f of the chosen arm,
 *
 *   latency = max(lat_min, l0 (a + b_w n / f) + eta),   power = P0 + c_w f^3,
 *   EDP     = power * latency^2                    (energy x delay, Sec. 2.3),
 *   reward  = -EDP / EDP_ref,  EDP_ref = (P0 + c_w)(l0 (a + b_w n))^2,
 *   queue   = min(q_cap, max(0, queue + n - cap))  (integer service capacity cap),
 *   running = min(run_cap, queue + n),  TTFT = latency (1 + queue / cap),
 *   TPOT    = latency / tpot_div,  util = min(1, n / cap),
 *   z       = ([n, log1p(queue), running, log(TTFT), TPOT, util, f] - mu) / sd,
 *
 * where b_w, c_w = b, c scaled by (1 + drift * t / (T - 1)) in the window of
 * decision t, and cap = round(svc_lo + (svc_hi - svc_lo) k / (K - 1)) for arm
 * k (svc_init for the warm-up window 0, run at f_init).  The context of
 * decision t is [1, z_t] (d = 8), [1, z_t, z_{t-1}, rho_t] (d = 16) or
 * [1, z_t, z_{t-1}, z_{t-2}, z_{t-3}, rho_t, rho_{t-1}, rho_{t-2}] (d = 32),
 * rho_w being the reward of window w and windows before 0 repeating window 0.
 * The reward of decision t is rho_{t+1}.
 *
 * Memory, streams and errors follow agft.h: caller-owned device buffers, no
 * allocation, work only enqueued on the given stream, negative status codes
 * (the AGFT_E_* values) on invalid arguments.
 */
#ifndef AGFT_SIM_H
#define AGFT_SIM_H

#include <stddef.h>
#include <stdint.h>

#include "agft.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct agft_env_config {
    int32_t B;        /* instances, >= 1 */
    int32_t K;        /* arms, 1..1024 (arm k runs at f_lo + (f_hi - f_lo) k / (K - 1)) */
    int32_t d;        /* context features: 8, 16 or 32 */
    int32_t T;        /* decisions per run, >= 1; exogenous arrays cover windows 0..T */
    float P0, c;      /* power model */
    float l0, a, b;   /* latency model */
    float lat_min;    /* latency floor, > 0 */
    float f_lo, f_hi; /* normalised clock range of the arm grid, 0 < f_lo <= f_hi */
    float f_init;     /* clock of the warm-up window, > 0 */
    float tpot_div;   /* TPOT = latency / tpot_div, > 0 */
    float drift;      /* relative growth of b and c over the run (0 = stationary) */
    int32_t svc_lo, svc_hi, svc_init; /* integer service capacities, >= 1 */
    int32_t q_cap, run_cap;           /* queue and concurrency caps, >= 0 */
    float mu[7], sd[7];               /* feature normalisation, sd > 0 */
} agft_env_config;

/* Bytes of device state for cfg (256-byte aligned regions); 0 if invalid. */
size_t agft_env_state_bytes(const agft_env_config *cfg);

/*
 * Run the warm-up window 0 for every instance and write the first context.
 * d_env       [agft_env_state_bytes] device buffer, 256-byte aligned, caller-owned.
 * d_arrivals  int32 [T+1][B] arrivals per window (time-major), device.
 * d_noise     fp32 [T+1][B] latency noise per window, device.
 * d_ctx       fp32 [B][d] out: x_0, 16-byte aligned.
 * stream      hipStream_t (NULL = null stream).
 */
int agft_env_reset(const agft_env_config *cfg, void *d_env, size_t nbytes, const int32_t *d_arrivals,
                   const float *d_noise, float *d_ctx, void *stream);

/*
 * Run window t+1 at the clock of decision t (0 <= t < T) for every instance.
 * d_action    int32 [B]: a_t (-1 keeps the previous clock).
 * d_reward    fp32 [B] out: reward of decision t.
 * d_ctx       fp32 [B][d] out: x_{t+1}, 16-byte aligned.
 */
int agft_env_step(const agft_env_config *cfg, void *d_env, size_t nbytes, int32_t t,
                  const int32_t *d_action, const int32_t *d_arrivals, const float *d_noise,
                  float *d_reward, float *d_ctx, void *stream);

/*
 * One decision of tuner h followed by the environment's response: the same
 * results as
 *   agft_step(h, d_ctx, d_reward, d_action, d_scores);
 *   agft_env_step(env_cfg, d_env, env_nbytes, t, d_action, d_arrivals, d_noise,
 *                 d_reward, d_ctx, stream of h);
 * with t the decisions h had made before the call (the decision step of
 * Sec. 4.2 followed by the measured window of Sec. 4.1).  Up to 8,192
 * instances in a single launch, each instance's environment running in the
 * step's epilogue once its decision is known, without the second launch and
 * its wait; beyond that as the two calls above, which are faster there.
 * In place: d_ctx holds x_t on entry and x_{t+1} on return, d_reward r_{t-1}
 * (read only when a decision is pending) and then r_t.  Enqueued on h's stream.
 * env_cfg must describe the same B, K, d as h; d_env as in agft_env_step.
 * d_ctx [B][d] fp32 (16-byte aligned), d_reward [B] fp32, d_action [B] int32:
 * device, non-NULL.  d_scores [B][2][K] or NULL, as in agft_step.
 * AGFT_E_INVAL for NULL or mismatched arguments, AGFT_E_STATE when the
 * exogenous draws end before this decision's window (t >= env_cfg->T).
 */
int agft_sim_step(agft_handle *h, const agft_env_config *env_cfg, void *d_env, size_t env_nbytes,
                  const int32_t *d_arrivals, const float *d_noise, float *d_ctx, float *d_reward,
                  int32_t *d_action, float *d_scores);

#ifdef __cplusplus
}
#endif

#endif /* AGFT_SIM_H */
