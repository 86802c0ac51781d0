/*
 * cleanba_layers.h -- layer-level entry points of the learner-update library.
 *
 * Each call runs one step of the IMPALA-ResNet forward or backward pass (the network the
 * paper trains with, Section 5) on activations in the library's storage type:
 * IMPALA_PREC_BF16 stores activations as bf16 bit patterns (uint16, round to nearest even)
 * and computes on bf16 matrix cores with float32 accumulation; IMPALA_PREC_FP32 stores
 * and computes in float32. Weights and weight gradients are float32 HWIO [3,3,cin,cout].
 * Conventions (memory, streams, errors, determinism) are those of cleanba_learner.h.
 * Supported channel pairs are those the network uses: cin == 4 for uint8 frames, else
 * cin, cout in {16, 32, 64} with cin <= cout (cin == cout when x_mode is IMPALA_X_RELU).
 */
#ifndef CLEANBA_LAYERS_H
#define CLEANBA_LAYERS_H

#include "cleanba_learner.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    IMPALA_X_PLAIN = 0,  /* x as stored */
    IMPALA_X_RELU = 1,   /* relu(x), applied while loading */
    IMPALA_X_U8 = 2      /* uint8 frames obs[row_idx[i]] (row_idx may be NULL), cin == 4;
                            the convolution sum is scaled by 1/255 */
} impala_x_mode_t;

/* y = conv3x3_same(X, w) + bias [+ add], X = x, relu(x) or frames/255 per x_mode.
 * x: [n, H, W, cin]; bias: float [cout] or NULL; add: [n, H, W, cout] or NULL;
 * y: [n, H, W, cout]. */
impala_status_t impala_conv3x3_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W,
                                   int32_t cin, int32_t cout, const void* x, int32_t x_mode,
                                   const int32_t* row_idx, const float* w, const float* bias,
                                   const void* add, void* y, hipStream_t stream);

/* A stage's entry (conv, then max-pool; Section 5's IMPALA-ResNet) in one pass, bf16 only:
 * y = maxpool3x3s2_same(conv3x3_same(X, w) + bias), arg as impala_maxpool_fwd. The
 * full-resolution conv output is rounded to bf16 and pooled without being stored, so y and
 * arg equal those of impala_conv3x3_fwd followed by impala_maxpool_fwd.
 * x_mode: IMPALA_X_PLAIN or IMPALA_X_U8. x: [n, H, W, cin]; y (bf16) and arg (uint8):
 * [n, ceil(H/2), ceil(W/2), cout]. IMPALA_PREC_FP32 returns IMPALA_EUNSUPPORTED. */
impala_status_t impala_conv3x3_pool_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W,
                                        int32_t cin, int32_t cout, const void* x, int32_t x_mode,
                                        const int32_t* row_idx, const float* w, const float* bias,
                                        void* y, uint8_t* arg, hipStream_t stream);

/* One residual block of Section 5's IMPALA-ResNet in one pass, bf16 only (C = 16 or 32):
 * t = conv3x3_same(relu(x), w1) + b1 and y = x + conv3x3_same(relu(t), w2) + b2. t is
 * rounded to bf16 before conv2 reads it, so t and y equal those of two impala_conv3x3_fwd
 * calls (IMPALA_X_RELU, the second with add = x); t is returned for the backward pass.
 * x, t, y: [n, H, W, C] bf16; w1, w2: float HWIO [3,3,C,C]; b1, b2: float [C] or NULL.
 * Other precisions or channel counts return IMPALA_EUNSUPPORTED. */
impala_status_t impala_resblock_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                   const void* x, const float* w1, const float* b1, const float* w2,
                                   const float* b2, void* t, void* y, hipStream_t stream);

/* Input gradient of y = conv3x3_same(x, w): dx = conv3x3_same^T(dy, w), then
 * dx *= (mask > 0) if mask is not NULL, then dx += add if add is not NULL.
 * dy: [n, H, W, cout]; mask, add, dx: [n, H, W, cin]. */
impala_status_t impala_conv3x3_dgrad(impala_prec_t prec, int64_t n, int32_t H, int32_t W,
                                     int32_t cin, int32_t cout, const void* dy, const float* w,
                                     const void* mask, const void* add, void* dx,
                                     hipStream_t stream);

/* Weight and bias gradient: dw[ky][kx][ci][co] = sum over pixels of X_pad[h+ky][w+kx][ci]
 * dy[h][w][co] (X per x_mode; with uint8 frames the sum is scaled by 1/255), db[co] = sum dy.
 * dw: float [3,3,cin,cout]; db: float [cout]; ws: device scratch of
 * impala_conv3x3_wgrad_workspace_bytes() bytes. */
size_t impala_conv3x3_wgrad_workspace_bytes(impala_prec_t prec, int32_t H, int32_t W, int32_t cin,
                                            int32_t cout);
impala_status_t impala_conv3x3_wgrad(impala_prec_t prec, int64_t n, int32_t H, int32_t W,
                                     int32_t cin, int32_t cout, const void* x, int32_t x_mode,
                                     const int32_t* row_idx, const void* dy, float* dw, float* db,
                                     void* ws, size_t ws_bytes, hipStream_t stream);

/* The whole backward pass of y = conv3x3_same(X, w) + bias in one pass, bf16 only, with
 * X = x (IMPALA_X_PLAIN) or relu(x) (IMPALA_X_RELU); Algorithm 1's back-propagation through
 * one convolution of Section 5's IMPALA-ResNet:
 *   dx = conv3x3_same^T(G, w), then dx *= (x > 0) when x_mode is IMPALA_X_RELU, then
 *   dx += add if add is not NULL;
 *   dw, db as impala_conv3x3_wgrad with the same x and x_mode and gradient G.
 * G = dy when pool_arg is NULL. Otherwise the conv feeds a stage's max-pool (a stage entry)
 * and dy is the gradient at the pool output, [n, ceil(H/2), ceil(W/2), cout], with pool_arg
 * its argmax as impala_maxpool_fwd returns it; G is then the pool's input gradient, formed
 * on chip exactly as impala_maxpool_bwd forms and rounds it.
 * dy (or G) and x are staged on chip once and both gradients are formed from them, so the
 * result equals impala_maxpool_bwd (with pool_arg), impala_conv3x3_dgrad (mask = x) and
 * impala_conv3x3_wgrad.
 * dy: [n, H, W, cout] or pooled as above; x, add, dx: [n, H, W, cin] (all bf16); w: float
 * HWIO [3,3,cin,cout]; dw: float [3,3,cin,cout]; db: float [cout] (both overwritten); ws:
 * device scratch of impala_conv3x3_bwd_workspace_bytes() bytes. Supported: IMPALA_X_RELU
 * without pool_arg with cin == cout in {16, 32}; IMPALA_X_PLAIN without add for (cin, cout)
 * in {(16,16), (16,32), (32,32)}; anything else returns IMPALA_EUNSUPPORTED. */
size_t impala_conv3x3_bwd_workspace_bytes(impala_prec_t prec, int32_t cin, int32_t cout);
impala_status_t impala_conv3x3_bwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t cin,
                                   int32_t cout, const void* dy, const uint8_t* pool_arg, const void* x,
                                   int32_t x_mode, const float* w, const void* add, void* dx, float* dw,
                                   float* db, void* ws, size_t ws_bytes, hipStream_t stream);

/* The backward pass of one residual block of Section 5's IMPALA-ResNet in one pass, bf16
 * only (C = 16 or 32), Algorithm 1's back-propagation through the block that impala_resblock_fwd
 * computes: with t = conv3x3_same(relu(x), wa) + ba, y = x + conv3x3_same(relu(t), wb) + bb
 * (wa, wb are that call's w1, w2) and dy the gradient at y:
 *   dt = conv3x3_same^T(dy, wb) * (t > 0), rounded to bf16;
 *   dx = conv3x3_same^T(dt, wa) * (x > 0) + dy;
 *   dwb, dbb as impala_conv3x3_wgrad of relu(t) against dy; dwa, dba of relu(x) against dt.
 * The result equals impala_conv3x3_bwd for the second conv (IMPALA_X_RELU with x = t)
 * followed by impala_conv3x3_bwd for the first (IMPALA_X_RELU with add = dy); dt never
 * leaves the chip. dy, t, x, dx: [n, H, W, C] bf16 (dx must not overlap the inputs); wa, wb:
 * float HWIO [3,3,C,C]; dwa, dwb: float [3,3,C,C] and dba, dbb: float [C] (all overwritten);
 * ws: device scratch of impala_resblock_bwd_workspace_bytes() bytes. Other precisions or
 * channel counts return IMPALA_EUNSUPPORTED. */
size_t impala_resblock_bwd_workspace_bytes(impala_prec_t prec, int32_t C);
impala_status_t impala_resblock_bwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                    const void* dy, const void* t, const void* x, const float* wa,
                                    const float* wb, void* dx, float* dwa, float* dba, float* dwb,
                                    float* dbb, void* ws, size_t ws_bytes, hipStream_t stream);

/* Backward of the first stage entry of Section 5's IMPALA-ResNet, y = maxpool3x3s2_same(
 * conv3x3_same(frames / 255, w) + bias), in one pass, bf16 only (Algorithm 1's
 * back-propagation; the frames need no input gradient): the max-pool's input gradient
 * dC (as impala_maxpool_bwd forms it, rounded to bf16) is built on chip from the gradient
 * at the pool output and the pool argmax, and feeds the weight gradient directly, so the
 * result equals impala_maxpool_bwd followed by impala_conv3x3_wgrad (IMPALA_X_U8).
 * obs: uint8 frames; frame i is obs[row_idx[i]] (row_idx may be NULL), [*, H, W, 4].
 * dpool (bf16) and arg (uint8): [n, ceil(H/2), ceil(W/2), cout]. dw: float [3,3,4,cout];
 * db: float [cout] (both overwritten). ws: device scratch of
 * impala_conv3x3_pool_wgrad_u8_workspace_bytes() bytes. cout must be 16 or 32, else
 * IMPALA_EUNSUPPORTED (as for IMPALA_PREC_FP32). */
size_t impala_conv3x3_pool_wgrad_u8_workspace_bytes(impala_prec_t prec, int32_t cout);
impala_status_t impala_conv3x3_pool_wgrad_u8(impala_prec_t prec, int64_t n, int32_t H, int32_t W,
                                             int32_t cout, const uint8_t* obs, const int32_t* row_idx,
                                             const void* dpool, const uint8_t* arg, float* dw, float* db,
                                             void* ws, size_t ws_bytes, hipStream_t stream);

/* 3x3 stride-2 SAME max-pool with XLA's padding split (pad_lo = P/2) and -inf padding.
 * x: [n, H, W, C]; y: [n, ceil(H/2), ceil(W/2), C]; arg: uint8, same shape as y, the
 * row-major window index 0..8 of the first maximum. C % 4 == 0, C <= 256. */
impala_status_t impala_maxpool_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                   const void* x, void* y, uint8_t* arg, hipStream_t stream);

/* Max-pool input gradient: dx[cell] = sum of dy over the windows whose argmax is the cell. */
impala_status_t impala_maxpool_bwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                   const uint8_t* arg, const void* dy, void* dx,
                                   hipStream_t stream);

/* Where a training-mode impala_cnn_fwd on n_frames frames (workspace laid out by
 * impala_workspace_bytes(net, n_frames, prec, 1)) leaves the activations that impala_cnn_bwd
 * reads, so a caller can inspect them or replace them between the two calls: the backward
 * pass (Algorithm 1's back-propagation) then differentiates the network at the activations it
 * finds there, taking every ReLU decision from the stored x and t and every max-pool routing
 * from the stored argmax. Tests use this to evaluate the backward pass at a reference
 * forward's activations.
 * Regions, each frame-major ([n_frames, ...], frame i at offset + i * bytes / n_frames):
 *   "s<k>.arg"  uint8 [n, ceil(H_k/2), ceil(W_k/2), C_k]  stage k's max-pool argmax, the
 *               row-major window index 0..8 as impala_maxpool_fwd returns it;
 *   "s<k>.x0"   the pooled output of stage k (input of its residual block 0);
 *   "s<k>.x1", "s<k>.x2"  the outputs of residual blocks 0 and 1 (x2 feeds stage k+1's
 *               entry conv, or for k = 2 the flatten);
 *   "s<k>.t0", "s<k>.t1"  the inner activation t = conv(relu(x)) + b of blocks 0 and 1;
 *   "h"         [n, hidden], the dense layer's output after its ReLU;
 *   "s<k>.conv" (IMPALA_PREC_FP32 only) [n, H_k, W_k, C_k], the stage entry's conv output
 *               before pooling (the bf16 path pools on chip and never stores it).
 * x, t, h and conv are bf16 bit patterns in IMPALA_PREC_BF16 and float32 otherwise; stage k
 * reads [H_k, W_k] (the frame for k = 0, halved, rounded up, per stage). The first stage's
 * input is the uint8 frames themselves, read through row_idx. Writes `cap` descriptors at most
 * into `out` (host memory) and returns the number of regions (19 bf16, 22 float32), or a
 * negative status. */
typedef enum { IMPALA_DT_U8 = 0, IMPALA_DT_BF16 = 1, IMPALA_DT_F32 = 2 } impala_dtype_t;
typedef struct impala_activation_desc {
    char name[32];
    int64_t offset;    /* bytes from the start of the workspace */
    int64_t bytes;     /* bytes of the region's n_frames frames */
    int32_t dtype;     /* impala_dtype_t */
    int32_t ndim;
    int64_t shape[4];  /* [n_frames, H, W, C] or [n_frames, hidden] */
} impala_activation_desc_t;
int impala_activation_layout(const impala_net_t* net, impala_prec_t prec, int64_t n_frames,
                             impala_activation_desc_t* out, int cap);

/* Log-probability of given actions under given logits, the target log-probs that V-trace
 * reads (log pi(a_t|s_t) in Espeholt et al.'s importance weights, which Appendix B's rlax
 * V-trace takes): logp[i] = log_softmax(logits[i])[actions[i]], NaN where actions[i] is
 * outside [0, A). logits: float [n, A]; actions: int32 [n]; logp: float [n]. */
impala_status_t impala_action_logp(int64_t n, int32_t A, const float* logits, const int32_t* actions,
                                   float* logp, hipStream_t stream);

/* Gumbel-max sampling on given logits: actions[i] = argmax_j (logits[i][j] + gumbel[i][j])
 * (float32 sums, ties to the lowest index) and logp[i] = log_softmax(logits[i])[actions[i]]. */
impala_status_t impala_gumbel_sample(int64_t n, int32_t A, const float* logits,
                                     const float* gumbel, int32_t* actions, float* logp,
                                     hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* CLEANBA_LAYERS_H */
