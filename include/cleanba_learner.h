/*
 * cleanba_learner.h -- C-ABI of the MI355X (gfx950) learner-update library.
 *
 * One learner update of Cleanba's PPO / IMPALA on one GPU's share of the batch
 * (Huang et al., "Cleanba: A Reproducible and Efficient Distributed Reinforcement
 * Learning Platform", Algorithm 1 learning phase, Appendix A objective, Appendix B
 * hyperparameter tables): the IMPALA-ResNet forward and backward over uint8 Atari
 * frames, GAE or V-trace targets, the PPO clipped-surrogate or IMPALA policy-gradient
 * loss with value and entropy terms, global-norm gradient clipping and Adam.
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory      Every array pointer is caller-owned DEVICE memory unless marked "host".
 *             The library never allocates, frees or retains caller pointers; workspaces
 *             are caller-allocated and sized by the *_workspace_bytes queries.
 * Streams     Every call enqueues its kernels on `stream` and returns without waiting.
 *             The returned status covers argument validation (done on the host before
 *             any HIP call) and launch errors; it does not report kernel completion.
 * Outputs     Outputs are overwritten, never accumulated into.
 * Layout      Row-major, innermost index last. Rollout arrays are time-major [T, E] with
 *             the env index fastest; flattened row = t*E + e (Algorithm 1 flattens the
 *             batch this way). Frames are NHWC uint8 [*, H, W, C].
 * Parameters  One flat float32 buffer holding 36 tensors in the order that
 *             impala_param_layout() reports: per stage the entry conv (w, b) then the
 *             four residual convs (w, b); then dense, logits, value (w, b). Conv weights
 *             are HWIO [3,3,Cin,Cout]; dense weights are [in, out].
 * Precision   IMPALA_PREC_BF16: bf16 matrix-core operands and stored activations with
 *             float32 accumulation. IMPALA_PREC_FP32: float32 throughout (validation).
 *             Logits, values, losses, gradients and optimiser state are float32 in both.
 * Errors      Non-zero status on failure; impala_last_error() returns a message for the
 *             calling thread. Non-finite numbers propagate; adam_step flags them.
 * Determinism No floating-point atomics: every reduction runs in a fixed order, so a
 *             call repeated on the same inputs returns bit-identical outputs.
 * Threads     Calls may run concurrently from several host threads on different streams
 *             when their workspaces and outputs are distinct (the actor-learner pipeline
 *             does this); the library keeps no state between calls besides a per-device
 *             occupancy cache and adam_step_noalloc's buffer. The per-launch profiler of
 *             cleanba_profile.h is the exception: one host thread.
 */
#ifndef CLEANBA_LEARNER_H
#define CLEANBA_LEARNER_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Network shape. The paper's agents use "IMPALA's ResNet" (Section 5): per stage a 3x3
 * SAME conv, a 3x3 stride-2 SAME max-pool and two residual blocks x + conv(relu(conv(relu(x)))),
 * then ReLU, flatten (H, W, C), dense + ReLU, and policy / value heads.
 * Supported: in_c == 4; ch[i] in {16, 32, 64} with ch[0] <= ch[1] <= ch[2];
 * 1 <= in_h, in_w <= 128; 1 <= hidden <= 4096; 1 <= num_actions <= 64. */
typedef struct impala_net {
    int32_t in_h, in_w, in_c;
    int32_t ch[3];
    int32_t hidden;
    int32_t num_actions;
} impala_net_t;

typedef enum { IMPALA_PREC_BF16 = 0, IMPALA_PREC_FP32 = 1 } impala_prec_t;

typedef enum {
    IMPALA_OK = 0,
    IMPALA_EINVAL = -1,       /* bad argument (null pointer, bad size, inconsistent shape) */
    IMPALA_EWORKSPACE = -2,   /* workspace smaller than the matching *_workspace_bytes */
    IMPALA_EUNSUPPORTED = -3, /* valid but unsupported shape (see impala_net_t) */
    IMPALA_EHIP = -4          /* a HIP launch reported an error */
} impala_status_t;

typedef struct impala_tensor_desc {
    char name[32];   /* e.g. "s1.res0.conv1.w", "dense.b" */
    int64_t offset;  /* in floats, into the flat parameter buffer */
    int32_t ndim;
    int32_t shape[4];
} impala_tensor_desc_t;

/* Number of float32 parameters (1,094,115 for (16,32,32)/256/18 at 84x84x4); -1 if the
 * shape is invalid. */
int64_t impala_param_count(const impala_net_t* net);

/* Writes up to `cap` tensor descriptors (36 for a valid net) and returns the number of
 * tensors, or a negative status. `out` is host memory. */
int impala_param_layout(const impala_net_t* net, impala_tensor_desc_t* out, int cap);

/* Workspace bytes for impala_cnn_fwd / impala_cnn_bwd / impala_actor_step on n_frames
 * frames. training != 0 sizes the saved activations the backward pass reads. 0 on error. */
size_t impala_workspace_bytes(const impala_net_t* net, int64_t n_frames, impala_prec_t prec,
                              int training);

/* Message describing the last error on the calling thread ("" if none). */
const char* impala_last_error(void);

/* Forward pass: logits [n, A] and value [n] of frames obs[row_idx[i]] (or obs[i] when
 * row_idx is NULL; gathering the minibatch rows of Algorithm 1 in the first conv's load).
 * obs: uint8 [*, H, W, C]; row_idx: int32 [n] or NULL, every entry a row of obs (0 <= r <
 * rows of obs; the call cannot check this without reading device memory, and an entry outside
 * the buffer makes the kernels read outside it). Pixels are scaled by 1/255.
 * training != 0 keeps the activations in `ws` for a following impala_cnn_bwd with the same
 * (params, obs, row_idx, n, ws). */
impala_status_t impala_cnn_fwd(const impala_net_t* net, impala_prec_t prec, const float* params,
                               const uint8_t* obs, const int32_t* row_idx, int64_t n, void* ws,
                               size_t ws_bytes, int training, float* logits, float* value,
                               hipStream_t stream);

/* Backward pass ("back-propagate" in Algorithm 1): the flat float32 gradient
 * grads [param_count] of sum(dlogits * logits) + sum(dvalue * value) w.r.t. every parameter,
 * reading the activations a training-mode impala_cnn_fwd left in `ws` (in bf16 mode also
 * its bf16 copy of the dense weights, so `params` must be the forward's).
 * dlogits: [n, A]; dvalue: [n]. */
impala_status_t impala_cnn_bwd(const impala_net_t* net, impala_prec_t prec, const float* params,
                               const uint8_t* obs, const int32_t* row_idx, int64_t n, void* ws,
                               size_t ws_bytes, const float* dlogits, const float* dvalue,
                               float* grads, hipStream_t stream);

/* Generalised advantage estimation for PPO (the advantage estimator of J^CLIP, Appendix A;
 * computed once per learning phase in Algorithm 1):
 *   delta_t = r_t + gamma (1 - d_{t+1}) V_{t+1} - V_t,  A_t = delta_t + gamma lambda (1 - d_{t+1}) A_{t+1},
 *   R_t = A_t + V_t, with d_T = next_done, V_T = next_value, A_T = 0.
 * d_t = 1 means s_t starts a new episode (Algorithm 1 caches d_t before stepping).
 * rewards, values, adv, ret: float [T, E]; dones: uint8 [T, E]; next_value: float [E];
 * next_done: uint8 [E]. */
impala_status_t gae_advantages(int32_t T, int32_t E, const float* rewards, const float* values,
                               const uint8_t* dones, const float* next_value,
                               const uint8_t* next_done, float gamma, float lambda, float* adv,
                               float* ret, hipStream_t stream);

/* V-trace targets for IMPALA (Appendix B points to rlax's vtrace_td_error_and_advantage;
 * Espeholt et al. 2018, Sec. 4.1). With is_t = exp(target_logp - behav_logp),
 * gamma_t = gamma (1 - d_{t+1}), rho_t = min(rho_bar, is_t), c_t = lambda min(c_bar, is_t):
 *   vs_t = V_t + rho_t (r_t + gamma_t V_{t+1} - V_t) + gamma_t c_t (vs_{t+1} - V_{t+1}),
 *   pg_adv_t = min(pg_rho_bar, is_t) (r_t + gamma_t (lambda vs_{t+1} + (1 - lambda) V_{t+1}) - V_t),
 * with vs_T = V_T = bootstrap_value. All float arrays [T, E] except bootstrap_value [E];
 * dones uint8 [T, E]; next_done uint8 [E]. */
impala_status_t vtrace_targets(int32_t T, int32_t E, const float* behav_logp,
                               const float* target_logp, const float* rewards, const float* values,
                               const uint8_t* dones, const float* bootstrap_value,
                               const uint8_t* next_done, float gamma, float lambda, float rho_bar,
                               float c_bar, float pg_rho_bar, float* vs, float* pg_adv,
                               hipStream_t stream);

/* PPO loss and its gradient over a minibatch of m rows (Appendix A's J^CLIP and joint
 * objective; Algorithm 1: normalise advantages, L = -L^pi + c1 L^V - c2 L^S):
 *   A_hat = (adv - mean) / (std + 1e-8) over the minibatch (population std) if norm_adv,
 *   r = exp(log pi(a) - old_logp), pg = max(-A_hat r, -A_hat clip(r, 1-eps, 1+eps)),
 *   L = mean(pg) + vf_coef * 0.5 mean((V - ret)^2) - ent_coef mean(entropy).
 * logits, dlogits: [m, A]; value, old_logp, adv, ret, dvalue: [m]; actions: int32 [m].
 * stats (device, float [8]): [L, policy, value, entropy, approx_kl, clipfrac, adv mean,
 * adv std].
 * ws: optional device scratch of loss_workspace_bytes(m) bytes (NULL: none). With it the rows
 * are spread over many workgroups in one pass over the logits; without it, up to 16384 rows
 * run in one workgroup, and larger minibatches keep their partial sums in dvalue's memory
 * and pass over the logits twice. Every output is the same bit for bit either way. */
size_t loss_workspace_bytes(int64_t m);
impala_status_t ppo_loss_grad(int64_t m, int32_t A, const float* logits, const float* value,
                              const int32_t* actions, const float* old_logp, const float* adv,
                              const float* ret, int32_t norm_adv, float clip_eps, float vf_coef,
                              float ent_coef, float* dlogits, float* dvalue, float* stats, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/* IMPALA loss and its gradient over m rows (Appendix B's IMPALA table):
 *   L = pg_coef mean(-pg_adv log pi(a)) + vf_coef * 0.5 mean((V - vs)^2) - ent_coef mean(H).
 * Shapes and ws as ppo_loss_grad; stats: [L, policy, value, entropy, mean pg_adv, mean vs, 0, 0]. */
impala_status_t impala_loss_grad(int64_t m, int32_t A, const float* logits, const float* value,
                                 const int32_t* actions, const float* vs, const float* pg_adv,
                                 float pg_coef, float vf_coef, float ent_coef, float* dlogits,
                                 float* dvalue, float* stats, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* Global-norm clip then Adam over the flat buffers (Algorithm 1: clip the gradient norm,
 * step the optimiser; Appendix B: Adam epsilon 1e-5):
 *   n = ||g||_2; g <- g * (max_grad_norm / n) if max_grad_norm > 0 and n > max_grad_norm;
 *   m <- b1 m + (1-b1) g; v <- b2 v + (1-b2) g^2;
 *   p <- p - lr (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps).
 * step is 1-based. params, m, v are updated in place; grads is read only.
 * stats (device, float [2] or NULL): [pre-clip norm, 1 if the norm is not finite].
 * ws: device scratch of adam_workspace_bytes() bytes for the norm's partial sums. */
size_t adam_workspace_bytes(int64_t n_params);
impala_status_t adam_step(int64_t n_params, float* params, const float* grads, float* m, float* v,
                          int32_t step, float lr, float beta1, float beta2, float eps,
                          float max_grad_norm, float* stats, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/* adam_step without a workspace, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same kernels
 * and results as adam_step (bit for bit), with the norm's partial sums in a buffer the library
 * holds on each GPU it runs on (8 KB per device, kept until the process ends). It calls no
 * allocating routine. Calls that overlap on one GPU share that buffer and race: order them on
 * one stream, or use adam_step with a workspace each. Arguments and errors as adam_step;
 * IMPALA_EINVAL if the partial sums would outgrow the buffer (they never do: their count is
 * capped at 1024 for every n_params), IMPALA_EHIP if the buffer's address cannot be found. */
impala_status_t adam_step_noalloc(int64_t n_params, float* params, const float* grads, float* m,
                                  float* v, int32_t step, float lr, float beta1, float beta2,
                                  float eps, float max_grad_norm, float* stats, hipStream_t stream);

/* Global-norm clip then RMSprop over the flat buffers (Algorithm 1: clip the gradient norm,
 * step the optimiser; Appendix B's IMPALA table: RMSprop with epsilon 0.01, decay 0.99):
 *   g as adam_step's clip;  nu <- decay nu + (1 - decay) g^2;  p <- p - lr g / sqrt(nu + eps).
 * The paper does not place epsilon. Reading: inside the square root, with nu starting at zero,
 * the convention of optax's RMSprop (the paper's learner is written in JAX).
 * params and nu are updated in place (nu zero before the first step); grads is read only.
 * stats (device, float [2] or NULL) and ws (rmsprop_workspace_bytes()) as adam_step.
 * EINVAL for n_params < 0, decay outside [0, 1) or eps < 0. */
size_t rmsprop_workspace_bytes(int64_t n_params);
impala_status_t rmsprop_step(int64_t n_params, float* params, const float* grads, float* nu,
                             float lr, float decay, float eps, float max_grad_norm, float* stats,
                             void* ws, size_t ws_bytes, hipStream_t stream);

typedef enum { LEARNER_PPO = 0, LEARNER_IMPALA = 1 } learner_algo_t;
typedef enum { LEARNER_OPT_ADAM = 0, LEARNER_OPT_RMSPROP = 1 } learner_opt_t;

/* One learning phase's hyperparameters (Appendix A nomenclature; Appendix B values). */
typedef struct learner_cfg {
    int32_t algo;             /* learner_algo_t */
    int32_t prec;             /* impala_prec_t */
    int32_t T, E;             /* num_steps, local_num_envs */
    int32_t update_epochs;    /* PPO; IMPALA takes each minibatch once */
    int32_t num_minibatches;  /* PPO: row minibatches; IMPALA: env blocks (divides E) */
    int32_t minibatch_size;   /* PPO m; num_minibatches * m <= T * E */
    int32_t norm_adv;         /* PPO: normalise advantages per minibatch */
    float gamma, lambda;      /* discount; GAE lambda / V-trace lambda */
    float clip_eps;           /* PPO epsilon */
    float vf_coef, ent_coef;  /* c1, c2 */
    float pg_coef;            /* IMPALA policy-gradient weight */
    float rho_bar, c_bar, pg_rho_bar; /* IMPALA importance-weight clips */
    float lr, beta1, beta2, adam_eps;
    float max_grad_norm;      /* omega; <= 0 disables clipping */
    int32_t optimizer;        /* learner_opt_t: Adam (Appendix B's PPO table) or RMSprop (its
                                 IMPALA table) */
    float rms_decay, rms_eps; /* RMSprop (Appendix B: 0.99, 0.01) */
} learner_cfg_t;

/* The rollout one learning phase consumes (Algorithm 1's D plus the bootstrap state). */
typedef struct rollout {
    const uint8_t* obs;        /* PPO: [T*E, H, W, C]; IMPALA: [(T+1)*E, H, W, C], rows
                                  T*E.. are the bootstrap frames s_next */
    const int32_t* actions;    /* [T*E] */
    const float* behav_logp;   /* [T*E] log-prob of the action under the behaviour policy */
    const float* rewards;      /* [T, E] */
    const uint8_t* dones;      /* [T, E] */
    const float* values;       /* PPO: [T, E] behaviour values; IMPALA: unused (NULL) */
    const float* next_value;   /* PPO: [E] v(s_next); IMPALA: unused (NULL) */
    const uint8_t* next_done;  /* [E] */
} rollout_t;

/* Workspace bytes for learner_step with this net and cfg; 0 on error. */
size_t learner_workspace_bytes(const impala_net_t* net, const learner_cfg_t* cfg);

/* One learning phase. PPO: GAE once, then for epoch j and minibatch k the rows
 * perm[j*T*E + k*m .. +m]: forward, loss, backward, clip, optimiser step (step incremented
 * per update). IMPALA: for minibatch k, the env block [k*E/N, (k+1)*E/N) (N = num_minibatches;
 * V-trace runs along time, so a minibatch keeps whole trajectories): forward over its T*E/N
 * rollout frames and E/N bootstrap frames, target log-probs, V-trace, loss over the rollout
 * rows, backward (bootstrap rows get no gradient), clip, optimiser step.
 * params, m, v: float [param_count], updated in place (RMSprop: v holds its nu, m is unused and
 * may be NULL). step: HOST int32, 1-based count of
 * updates done so far (incremented). perm: int32 [update_epochs, T*E] (PPO; NULL for IMPALA),
 * every entry in [0, T*E) (not checked: it indexes the frames and the rollout arrays on the
 * device; each row of perm is normally a permutation).
 * stats: float [n_updates, 8] (n_updates = update_epochs * num_minibatches for PPO,
 * num_minibatches for IMPALA) rows [L, policy, value, entropy, approx_kl or mean pg_adv,
 * clipfrac or mean vs, pre-clip grad norm, nonfinite]. */
impala_status_t learner_step(const impala_net_t* net, const learner_cfg_t* cfg,
                             const rollout_t* rollout, float* params, float* m, float* v,
                             int32_t* step, const int32_t* perm, void* ws, size_t ws_bytes,
                             float* stats, hipStream_t stream);

/* Actor inference (Algorithm 1: a_t ~ pi(.|s_t) and v_t = v(s_t)): forward on n frames,
 * then Gumbel-max sampling a = argmax_j(z_j + gumbel_j) with ties to the lowest index, and
 * log pi(a). gumbel: float [n, A] caller-drawn standard Gumbel noise. actions: int32 [n];
 * logp, value: float [n]; logits: float [n, A] or NULL. ws: impala_workspace_bytes(net, n,
 * prec, 0) bytes, plus n*A*4 rounded up to a multiple of 256 when logits is NULL (the logits
 * are then kept there). */
impala_status_t impala_actor_step(const impala_net_t* net, impala_prec_t prec, const float* params,
                                  const uint8_t* obs, int64_t n, const float* gumbel, void* ws,
                                  size_t ws_bytes, int32_t* actions, float* logp, float* value,
                                  float* logits, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* CLEANBA_LEARNER_H */
