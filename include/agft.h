/*
 * agft.h -- C ABI of the batched AGFT tuner step on AMD Instinct MI355X (gfx950).
 *
 * One call of agft_step advances B independent tuner instances by one
 * decision of AGFT's contextual-bandit frequency selector (Sec. 4.2): it
 * folds the previous decision's reward into that arm's model (Eq. 3-5),
 * scores every active frequency arm on the new context with the linear upper
 * confidence bound (Eq. 1), applies the action-space pruning rule when due
 * (motivated in Sec. 4.3), and returns the argmax arm per instance.
 *
 * Memory: the caller owns every device buffer (state, contexts, rewards,
 * actions, score dumps); the library owns only the small host-side handle.
 * No entry point allocates or frees device memory.  Every entry point only
 * enqueues work on the handle's HIP stream and returns without waiting,
 * except agft_create with AGFT_ADOPT_STATE, which reads the buffer's header
 * back synchronously.  A handle is not thread-safe; use one handle per
 * stream.  Calls launch on the calling thread's current HIP device: make
 * the device of the handle's stream and buffers current before each call.
 *
 * Errors: every int-returning call returns AGFT_OK (0) or a negative code;
 * arguments are validated before anything is enqueued.  A device fault of
 * earlier work surfaces as AGFT_E_HIP from a later call.
 *
 * Model kept per (instance i, arm k), in fp32:
 *   theta_k = A_k^{-1} b_k                      (Eq. 5)
 *   S_k     upper triangular with S_k S_k^T = A_k^{-1}
 * where A_k = lambda I + sum x x^T (Eq. 3) and b_k = sum r x (Eq. 4) over
 * the decisions that chose arm k.  The rank-1 change of A_k^{-1} that Eq. 3
 * implies (the Sherman-Morrison identity) is applied to the factor S_k in
 * square-root form, which keeps fp32 scores within 1e-5 of exact arithmetic
 * where the plain inverse update drifts by 1e-3 over thousands of updates.
 */
#ifndef AGFT_H
#define AGFT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AGFT_ABI_VERSION 6

enum agft_status {
    AGFT_OK = 0,
    AGFT_E_INVAL = -1,       /* NULL pointer, size or value out of range */
    AGFT_E_UNSUPPORTED = -2, /* well-formed but not supported (d not in {8,16,32}, a
                                non-sticky rule 1 beside rules 2-8) */
    AGFT_E_STATE = -3,       /* call not valid now (missing reward, adopted
                                buffer that does not match the configuration) */
    AGFT_E_HIP = -4          /* HIP runtime error, including earlier device faults */
};

/* agft_config.flags */
#define AGFT_ADOPT_STATE 0x1u /* resume from the state already in the buffer */

typedef struct agft_config {
    int32_t B;            /* independent tuner instances, >= 1 */
    int32_t K;            /* frequency arms per instance (the set F of Eq. 1), 1..1024 */
    int32_t d;            /* context features per decision (x_t, Sec. 4.1): 8, 16 or 32 */
    float lambda;         /* ridge prior, A_k(0) = lambda I: finite, > 0 */
    float alpha0;         /* exploration weight of Eq. 1: finite, >= 0 */
    int32_t alpha_sched;  /* 0: alpha_t = alpha0; 1: alpha_t = alpha0 / sqrt(t + 1) */
    int32_t prune_rule;   /* bit mask of pruning rules; every rule removes arms for good
                             (rule 1 unless prune_sticky is 0):
                             1  confidence bounds: at steps t > 0 with
                                t % prune_period == 0, an active arm k goes when
                                UCB_k < max_j LCB_j over the active arms j, with that
                                step's context and alpha_t, before the argmax;
                             2  extreme-frequency pruning (Sec. 4.3): while
                                t < ext_rounds, an active arm with at least
                                ext_min_n rewards averaging below ext_thr goes;
                             4  historical pruning (Sec. 4.3): once t >= hist_after,
                                among the active arms with at least hist_min_n
                                rewards (if there are hist_min_arms of them), an arm
                                goes when the best of their mean rewards exceeds its
                                own by more than hist_kappa times the population
                                standard deviation of those means;
                             8  cascade pruning (Sec. 4.3): when rule 2 or 4 removes
                                an arm with index < cascade_k (clock below half of
                                the top clock), every lower arm goes too.
                             Rules 2-8 act on the arms active when the step starts,
                             after the previous reward is folded in, before scoring;
                             if they would leave no arm, the arm with the best mean
                             reward (lowest index on ties) stays. */
    int32_t prune_period; /* period of rule 1; >= 1 */
    int32_t prune_sticky; /* 1: rule 1 removes arms for good, like the paper's own rules
                             (Sec. 4.3); 0: rule 1 is re-evaluated at each of its steps
                             over the whole action space (every arm of it scored, the
                             kept set {k : UCB_k >= max_j LCB_j} replacing the previous
                             one), so an arm removed once can come back.  0 is supported
                             with rule 1 alone (prune_rule 0 or 1; AGFT_E_UNSUPPORTED
                             beside rules 2-8).  Must be 0 or 1: a zero-filled
                             configuration gets the non-sticky reading. */
    uint32_t flags;       /* 0 or AGFT_ADOPT_STATE */
    /* parameters of rules 2, 4, 8 (read only when the rule's bit is set) */
    int32_t ext_rounds;    /* >= 0 */
    int32_t ext_min_n;     /* >= 1 */
    float ext_thr;         /* finite */
    int32_t hist_after;    /* >= 0 */
    int32_t hist_min_n;    /* >= 1 */
    float hist_kappa;      /* finite, >= 0 */
    int32_t hist_min_arms; /* >= 1 */
    int32_t cascade_k;     /* 0..K */
    /* switch to greedy exploitation (Sec. 4.2, Eq. 2): 0 off, 1 on.  Every
       reward folded in feeds a two-sided Page-Hinkley test in single precision
       (running mean rbar; m+ += (r - rbar) - ph_delta, m- += (rbar - r) - ph_delta;
       an alarm when m+ - min m+ or m- - min m- exceeds ph_lambda, after which the
       test restarts).  Once t >= ph_min_rounds and no alarm came in the last
       ph_window rounds, the instance exploits for good: a_t = argmax over the
       active arms of theta_k^T x_t (reported as both UCB and LCB), reading only
       the contiguous copy of theta that the state holds when this is on (4*d
       bytes per arm, against 4*(d + d(d+1)/2) for a whole record); rule 1 is not
       applied; updates go on.  A buffer adopted with AGFT_ADOPT_STATE must have
       been made with the same setting. */
    int32_t exploit;
    float ph_delta;        /* finite */
    float ph_lambda;       /* finite, >= 0 */
    int32_t ph_window;     /* >= 0 */
    int32_t ph_min_rounds; /* >= 0 */
    /* mixed-maturity refinement of the action space (Sec. 4.4): 0 off, 1 on.
       The action space is lo <= k <= hi with (hi - k) % stride == 0, minus the
       arms a pruning rule removed; it starts as the coarse grid lo = 0,
       hi = K-1, stride = refine_stride (stride 1 when off).  At a step t > 0
       with t % refine_period == 0 that decides, after the decision, an anchor
       is taken among the arms of the space that survived the step's pruning:
       before round refine_mature the best mean reward among the arms with at
       least refine_min_n rewards (lowest index on ties; none qualifying: no
       change), from then on the arm just chosen.  From the next step the
       space is the full-resolution window [anchor - refine_half,
       anchor + refine_half] clipped to [0, K-1].  Models persist for every
       arm whether in the space or not. */
    int32_t refine;
    int32_t refine_period; /* >= 1 */
    int32_t refine_stride; /* >= 1 */
    int32_t refine_half;   /* >= 0 */
    int32_t refine_mature; /* >= 0 */
    int32_t refine_min_n;  /* >= 1 */
} agft_config;

typedef struct agft_handle agft_handle;

/* Device pointers into the state buffer and the handle's counters. */
typedef struct agft_state_view {
    int64_t t;          /* decisions made so far */
    int32_t pending;    /* 1 while the last decision awaits its reward */
    int32_t B, K, d;
    int32_t chunks;     /* float4 chunks per arm record: (d/2)*(d/4) + (d/2)*TF/4 */
    int32_t block_arms; /* arms per block of records: NB = 64/d */
    int32_t tail_floats;/* TF, floats per lane slice of a record tail: 3 (packed, no
                           padding) when an exploring instance streams more than
                           16 KB of records per step (arms in play * 4 * (d +
                           d(d+1)/2) bytes), or more than 8 KB with no pruning
                           rule, refinement or switch to exploitation; else 4
                           (one float of padding per slice, so that no tail
                           straddles two 128-byte lines) */
    int32_t mask_words; /* uint32 words per instance in the action-set mask: ceil(K/32) */
    void *arms;         /* float4 records, instance i's at chunk i * ceil(K/NB)*NB*chunks.
                           Arm k sits in block k/NB (NB*chunks chunks), slot r = k%NB.
                           A block holds the NB main parts (M = (d/2)*(d/4) chunks each,
                           slot r at chunk r*M), then the NB tails (T = (d/2)*TF/4
                           chunks each, slot r at chunk NB*M + r*T).  Every record has
                           G = d/2 lane slices of d+3 positions:
                             e = 0..j:      S_{e,j}            (column j of S)
                             e = j+1..d:    S_{d-e, d-1-j}     (column d-1-j, bottom up)
                             e = d+1, d+2:  theta_{2j}, theta_{2j+1}
                           with S upper triangular, S S^T = A^{-1}.  Positions e < d of
                           slice j are component e%4 of main chunk (e/4)*G + j;
                           positions d..d+2 are tail floats TF*j .. TF*j+2 (with
                           TF = 4, float TF*j+3 is 0).  Slots past K in the last
                           block hold zeros. */
    uint32_t *mask;     /* [B][mask_words]: bit k%32 of word k/32 set = arm k not
                           removed by a pruning rule (the action space is apart; with
                           a non-sticky rule 1, the arms its last evaluation kept and
                           every arm it did not score) */
    int32_t *inst;      /* [B][inst_words] per-instance block of 32-bit words:
                           [0] last decision (-1: none), [1] arms in play (in the
                           action space and not removed by a rule),
                           [2] non-finite contexts or rewards met,
                           [3] -1 while exploring, else the round exploitation began,
                           [4..9] Page-Hinkley n, mean, m+, min m+, m-, min m- (fp32),
                           [10] round of its last alarm, [11] its last margin (fp32),
                           [12] [13] [14] action space lo, hi, stride,
                           [15] top-two gap of the last decision made with a score
                           dump (d_scores non-NULL): the largest score of the arms
                           kept by pruning minus the second largest (fp32; 0 at a
                           tie, +inf with one arm kept; the argmax margin of Eq. 1,
                           or of Eq. 2 once exploiting),
                           [16 .. 16+d) context of the last decision (fp32) */
    int32_t inst_words; /* words per instance block: 16 + d rounded up to 16 */
    int32_t *stats;     /* [B][K][2] per arm: [0] rewards folded in (int32),
                           [1] their sum (fp32 bits).  Maintained only when a rule
                           that reads them is on (prune_rule bits 2, 4, 8, or
                           refine); otherwise they stay 0. */
    float *theta;       /* [B][K][d] copy of theta_k (Eq. 5), kept in step with the
                           records, which exploiting instances read in their place;
                           NULL when cfg.exploit is 0 */
} agft_state_view;

/* Bytes of device state for cfg (a 256-byte header, then the arm records,
 * the masks, the instance blocks, the arm statistics and, with cfg.exploit,
 * the theta copy of agft_state_view, each region 256-byte aligned); 0 if cfg
 * is invalid. */
size_t agft_state_bytes(const agft_config *cfg);

/*
 * Bind a handle to the caller's state buffer d_state (nbytes >= agft_state_bytes,
 * 256-byte aligned) and HIP stream (a hipStream_t; NULL = the null stream).
 * Without AGFT_ADOPT_STATE, enqueues the initialisation: S_k = I / sqrt(lambda),
 * theta_k = 0, every arm active, t = 0.  With it, reads the buffer's header
 * back (synchronously) and resumes from its t; the header must match cfg
 * (dimensions, record layout, the switch, and whether the per-arm reward
 * statistics are maintained), else AGFT_E_STATE.
 * *out receives the handle; on error *out is set to NULL.
 */
int agft_create(const agft_config *cfg, void *d_state, size_t nbytes, void *stream,
                agft_handle **out);

/*
 * One decision for all B instances (Sec. 4.2):
 *   1. if a decision is pending, fold its reward d_reward[i] into the chosen
 *      arm with the stored context (Eq. 3-5; a non-finite reward skips this);
 *   2. score every active arm on d_ctx (Eq. 1): UCB and LCB;
 *   3. at pruning steps, apply the pruning rule;
 *   4. d_action[i] = lowest-index active arm with the largest UCB (-1 when
 *      the context holds a non-finite value: no decision, no update next step);
 *   5. remember d_ctx and the action for the next call; t += 1.
 * d_ctx     [B][d] fp32, device.  NULL = flush: apply step 1 only, no decision.
 * d_reward  [B] fp32, device: reward of the previous decision; must be non-NULL
 *           when a decision is pending (AGFT_E_STATE otherwise), else ignored.
 * d_action  [B] int32, device, or NULL.
 * d_scores  [B][2][K] fp32, device, or NULL: UCB (row 0) and LCB (row 1) of
 *           every arm active before this step's pruning, -inf for the others;
 *           with it the step also leaves the top-two gap of its decision in
 *           word 15 of each instance block (agft_state_view.inst).
 */
int agft_step(agft_handle *h, const float *d_ctx, const float *d_reward, int32_t *d_action,
              float *d_scores);

/* How agft_step launches the step kernel for cfg (host-only, no device
 * call): one workgroup per instance.  The five fields follow from the
 * configuration alone: the bytes an exploring instance streams per step
 * (arms in play times 4(d + d(d+1)/2)) choose the record layout, with the
 * switch the bytes an exploiting instance streams choose the workgroup
 * width, d, the layout and the pruning rules choose the register target
 * and where the update runs, and the width with the register target the
 * cap on workgroups per compute unit. */
typedef struct agft_launch_shape {
    int32_t waves;        /* wavefronts per workgroup: 1 up to 16 KB streamed per
                             instance, 4 beyond (with the switch: the exploiting
                             instance's bytes; agft_step's steps before round
                             ph_min_rounds, when no instance can exploit yet,
                             take the exploring instance's width) */
    int32_t simd_waves;   /* wavefronts per SIMD the kernel's registers allow */
    int32_t tail_floats;  /* record layout, as agft_state_view.tail_floats */
    int32_t early_update; /* 1: the rank-1 update runs while the stream's first pass
                             is in flight; 0: after the stream */
    int32_t cu_workgroups;  /* workgroups per compute unit agft_step's launch admits
                               (its LDS request caps them there); 0: no cap.
                               agft_sim_step's single launch is uncapped. */
} agft_launch_shape;

/* Fill *out for cfg.  AGFT_E_INVAL if cfg is invalid or out is NULL,
 * AGFT_E_UNSUPPORTED for a context dimension other than 8, 16, 32 or a
 * non-sticky rule 1 beside rules 2-8. */
int agft_launch_shape_for(const agft_config *cfg, agft_launch_shape *out);

/* Fill *out with device pointers into the state and the handle's counters. */
int agft_get_state(const agft_handle *h, agft_state_view *out);

/*
 * Materialise the model for inspection: d_theta [B][K][d] = theta_k (Eq. 5)
 * and d_ainv [B][K][d][d] = A_k^{-1} = S_k S_k^T.  Either may be NULL.
 */
int agft_export(agft_handle *h, float *d_theta, float *d_ainv);

/* Enqueue later work of this handle on another HIP stream. */
int agft_set_stream(agft_handle *h, void *stream);

/* Release the host handle (the state buffer stays the caller's). NULL is a no-op. */
int agft_destroy(agft_handle *h);

/* Static text for a status code. */
const char *agft_strerror(int code);

/* AGFT_ABI_VERSION of the loaded library. */
int agft_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AGFT_H */
