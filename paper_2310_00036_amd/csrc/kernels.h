// Internal launch interface between the host orchestration and the gfx950 kernels.
// Every launcher validates nothing (the C-ABI layer does) and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "prof.h"

namespace cb {

enum Prec { BF16 = 0, FP32 = 1 };
enum InMode { IN_PLAIN = 0, IN_RELU = 1, IN_U8 = 2 };

// ---- 3x3 SAME convolution as implicit GEMM (forward, and input-gradient with flip=1)
struct ConvArgs {
    const void* x;          // input activations [n, H, W, cin] (storage type) or uint8 frames
    const int32_t* row_idx; // uint8 mode: frame i reads obs row row_idx[i] (NULL: i)
    const float* w;         // float32 HWIO weights of the forward conv
    const float* bias;      // [cout] or NULL
    const void* add;        // [n, H, W, cout] added after the mask, or NULL
    const void* mask;       // [n, H, W, cout]: output kept where mask > 0, or NULL
    void* y;                // [n, H, W, cout] (conv3x3_pool: the pooled [n, OH, OW, cout])
    uint8_t* arg;           // conv3x3_pool: argmax of each pooled value (0..8), else unused
    int n, H, W;
    float scale;            // multiplies the sum before the bias (1/255 for uint8 frames)
};
// flip = 0: y = conv(x, w) (cin, cout are the forward conv's channels).
// flip = 1: y = conv^T(x, w), the adjoint w.r.t. the forward input; here x has the forward
//           conv's output channels (cin argument = forward cout) and y its input channels.
hipError_t conv3x3(int prec, int cin, int cout, int mode, int flip, const ConvArgs& a,
                   hipStream_t s);
bool conv3x3_supported(int cin, int cout, int mode, int flip);
// bf16 only: y = maxpool3x3s2(conv(x, w) + b) with its argmax (as maxpool_fwd), the conv
// output kept in LDS; OH = (H+1)/2, OW = (W+1)/2. Modes IN_U8 and IN_PLAIN.
hipError_t conv3x3_pool(int cin, int cout, int mode, const ConvArgs& a, hipStream_t s);

// Tile of the conv + max-pool kernel (conv_pool_fast): bands of PTH pooled rows.
struct CpTile {
    int PTH, nbands, ntiles, OH, OW, ph, pw, THmax;
    int raw_off, win_off, win_guard, key_off;   // LDS layout (bytes)
    float inv_OW;
};
bool conv_pool_fast_supported(int cin, int cout, int mode);
hipError_t conv_pool_fast(int cin, int cout, int mode, const ConvArgs& a, hipStream_t s);

// ---- a whole residual block, bf16 forward: t = conv1(relu(x)) + b1 (stored),
//      y = x + conv2(relu(t)) + b2; all tensors [n, H, W, C], weights float32 HWIO [3,3,C,C].
struct ResBlockArgs {
    const void* x; const float* w1; const float* b1; const float* w2; const float* b2;
    void* t; void* y;
    int n, H, W;
};
bool resblock_fwd_supported(int C);
hipError_t resblock_fwd(int C, const ResBlockArgs& a, hipStream_t s);

// ---- weight gradient of a 3x3 SAME conv (deterministic split over pixels)
struct WgradArgs {
    const void* x;          // forward input (storage type or uint8 frames)
    const int32_t* row_idx;
    const void* dy;         // [n, H, W, cout] gradient at the conv output
    float* dw;              // float32 HWIO [3,3,cin,cout]
    float* db;              // float32 [cout]
    float* partial;         // workspace, wgrad_partial_floats() floats
    int n, H, W;
    float scale;            // applied to dw (1/255 for uint8 frames)
};
size_t wgrad_partial_floats(int prec, int cin, int cout, int H, int W);
hipError_t conv3x3_wgrad(int prec, int cin, int cout, int mode, const WgradArgs& a,
                         hipStream_t s);
bool wgrad_supported(int cin, int cout, int mode);

// ---- whole backward pass of one 3x3 SAME conv (bf16): input gradient and weight gradient
//      from one staging of dy and x. Forward: y = conv(X, w) + b, X = relu(x) (IN_RELU) or x.
// A weight-gradient partial sum deferred to the next kernel on the stream: nparts float32
// partials (stride pstride floats) laid out [mt*(NB+1) + nb][co 16][col 16] (NB = 9*cin/16
// column blocks, 3 for uint8 frames; the last block holds the bias sums), to be scattered to
// HWIO dw (times scale) and db. nparts == 0: none.
struct PendingReduce {
    const float* partial;
    float* dw; float* db;
    int nparts, pstride, cin, cout, u8;
    float scale;
};
// Launches the standalone fixed-order reduce of a pending partial sum (no-op if none).
hipError_t flush_pending_reduce(const PendingReduce& r, hipStream_t s);

// ---- backward of a whole residual block, t = conv_a(relu(x)) + b_a, y = x + conv_b(relu(t)) + b_b
// (bf16): dx = conv_a^T(conv_b^T(dy) * [t > 0]) * [x > 0] + dy and both weight gradients
struct ResBwdArgs {
    const void* dy;         // [n, H, W, C] gradient at the block output
    const void* t;          // [n, H, W, C] conv_a's output as the forward stored it
    const void* x;          // [n, H, W, C] block input
    const float* wa; const float* wb;   // float32 HWIO [3,3,C,C]
    void* dx;               // [n, H, W, C]
    float* dwa; float* dba; float* dwb; float* dbb;
    float* partial;         // workspace, resblock_bwd_partial_floats() floats
    int n, H, W;
    PendingReduce pend, pend2;   // earlier launches' partials, summed by this kernel first
};
struct RbbTile {
    int TH, nbands, ntiles;
    int dy_off, t_off, x_off, dt_off;   // LDS byte offsets; 64 zero bytes at offset 0
    int tx_guard;                       // t / x windows: byte offset of the rear guard pixel
    int dt_bytes;                       // dt window bytes
    int pset;                           // floats per partial set (one per conv)
    float inv_W;
};
bool resblock_bwd_supported(int C);
bool resblock_bwd_preferred(int C, int H, int W);   // over two fused conv backward launches
size_t resblock_bwd_partial_floats(int C);
// out[0] / out[1]: conv_b's / conv_a's weight-gradient partials, left for a later launch to sum
hipError_t resblock_bwd(int C, const ResBwdArgs& a, hipStream_t s, PendingReduce out[2]);

struct ConvBwdArgs {
    const void* dy;         // [n, H, W, cout] bf16; with arg: the max-pool output gradient
                            // [n, ceil(H/2), ceil(W/2), cout] of the pool this conv feeds
    const uint8_t* arg;     // that pool's argmax (same shape), or NULL: dy is the conv's own
    const void* x;          // [n, H, W, cin] bf16, the forward input as stored
    const float* w;         // float32 HWIO [3,3,cin,cout]
    const void* add;        // [n, H, W, cin] added to dx, or NULL
    void* dx;               // [n, H, W, cin]: conv^T(dy) * (x > 0 if IN_RELU) + add
    float* dw;              // float32 HWIO [3,3,cin,cout]
    float* db;              // float32 [cout]
    float* partial;         // workspace, conv3x3_bwd_partial_floats() floats
    int n, H, W;
    PendingReduce pend, pend2;   // earlier launches' partials, summed by this kernel first
};
struct CbTile {
    int TH, FR, nbands, ntiles;
    int dy_off, x_off;            // LDS byte offsets; 64 zero bytes at offset 0
    int x_guard;                  // x window: byte offset of its rear guard pixel
    int dp_off, ag_off, PR;       // pooled gradient / argmax rows in LDS (PR rows), pooled input
    int OH, OW, ph, pw, BH, BW;   // max-pool geometry (2x2 block grid BH x BW)
    float inv_W, inv_TW, inv_TH, inv_TR, inv_BW;
};
bool conv3x3_bwd_supported(int cin, int cout, int mode, int add, int pooled);
size_t conv3x3_bwd_partial_floats(int cin, int cout);
// deferred: when non-NULL the launch's own partial sum is not reduced; it is described there
// for a later launch (conv3x3_bwd / pool_wgrad_u8 via .pend, or flush_pending_reduce).
hipError_t conv3x3_bwd(int cin, int cout, int mode, const ConvBwdArgs& a, hipStream_t s,
                       PendingReduce* deferred = nullptr);
// Fixed-order sum of nparts bf16 weight-gradient partials laid out [mt*(NB+1) + nb]
// [co 16][col 16] (the last column block holds the bias sums), scattered to HWIO dw (times
// scale) and db. NB = 9*cin/16 column blocks of 16 input channels of one tap; for uint8
// frames (cin == 4) NB = 3 blocks of 4 taps x 4 channels.
hipError_t wgrad_reduce_tr(int cin, int cout, const float* partial, int nparts, float* dw, float* db,
                           float scale, hipStream_t s);

// ---- backward of the first stage entry, bf16: y = maxpool(conv3x3(frames / 255) + b); the
//      max-pool backward feeds the conv's weight gradient on chip (the frames need no input
//      gradient). Equals maxpool_bwd followed by conv3x3_wgrad(IN_U8).
struct PoolWgArgs {
    const uint8_t* obs;     // frames [*, H, W, 4]; frame i is obs[row_idx[i]] (NULL: i)
    const int32_t* row_idx;
    const void* dp;         // [n, OH, OW, cout] bf16 gradient at the pool output
    const uint8_t* arg;     // [n, OH, OW, cout] pool argmax (0..8)
    float* dw;              // float32 HWIO [3,3,4,cout]
    float* db;              // float32 [cout]
    float* partial;         // workspace, pool_wgrad_u8_partial_floats() floats
    int n, H, W;
    PendingReduce pend, pend2;   // earlier launches' partials, summed by this kernel first
};
struct PwTile {
    int TB, nbands, ntiles;         // 2x2 pixel-block rows per band
    int OH, OW, ph, pw, BH, BW;     // pool geometry (padded-coordinate block grid BH x BW)
    int raw_off, win_off, win_guard, dp_off, arg_off, dc_off;   // LDS layout (bytes)
};
bool pool_wgrad_u8_supported(int cout);
size_t pool_wgrad_u8_partial_floats(int cout);
hipError_t pool_wgrad_u8(int cout, const PoolWgArgs& a, hipStream_t s);

// ---- 3x3 stride-2 SAME max-pool (XLA padding split), first-max argmax in 0..8
hipError_t maxpool_fwd(int prec, int n, int H, int W, int C, const void* x, void* y,
                       uint8_t* arg, hipStream_t s);
hipError_t maxpool_bwd(int prec, int n, int H, int W, int C, const uint8_t* arg, const void* dy,
                       void* dx, hipStream_t s);

// ---- GEMM D[m][n] = sum_k A(m,k) B(k,n) on MFMA, output out[n*ld + m]
struct GemmArgs {
    const void* a; int a_f32; int a_kcontig; int64_t lda;   // A(m,k) = a[m*lda+k] or a[k*lda+m]
    const void* b; int b_f32; int b_kcontig; int64_t ldb;   // B(k,n) = b[n*ldb+k] or b[k*ldb+n]
    int b_relu;                                             // relu(B) on load
    int M, N, K;
    // epilogue (applied after the split-K sum): v = sum*alpha + bias; relu; mask; store
    float alpha;
    const float* bias1; const float* bias2;                 // bias for m < msplit / m >= msplit
    int relu;
    const void* mask; int64_t ldmask;                       // storage type, keep where > 0
    void* out1; int64_t ld1; int out1_f32;                  // rows m < msplit
    void* out2; int64_t ld2; int out2_f32;                  // rows m >= msplit (index m - msplit)
    int msplit;
    float* partial;                                         // split-K workspace (or NULL)
    size_t partial_floats;                                  // its capacity
};
// Floats of split-K workspace a GEMM of this shape uses at most.
size_t gemm_partial_floats(int M, int N, int K);
// The launcher splits K so the grid covers the chip, within a.partial_floats.
hipError_t gemm(int prec, const GemmArgs& a, hipStream_t s);

// y[i] = bf16(x[i]) (round to nearest even); y 4-byte aligned.
hipError_t cast_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s);

// ---- policy-logit and value heads (float32 FMAs; h and dh in the storage type)
struct HeadsArgs {
    const void* h;      // [n][J] dense-layer output (after relu), storage type
    const float* wl;    // [J][A] logit weights
    const float* bl;    // [A]
    const float* wv;    // [J] value weights
    const float* bv;    // [1]
    int64_t n; int J, A;
};
// logits [n][A] and value [n], float32.
hipError_t heads_fwd(int prec, const HeadsArgs& a, float* logits, float* value, hipStream_t s);
// dh [n][J] (storage type) = (dz W^T) * (h > 0) with dz = [dlogits | dvalue]; the head weight
// and bias gradients and the dense bias gradient (column sums of dh as stored) are
// overwritten. `partial` holds heads_bwd_partial_floats(n, J, A) floats.
hipError_t heads_bwd(int prec, const HeadsArgs& a, const float* dlogits, const float* dvalue, void* dh,
                     float* dwl, float* dbl, float* dwv, float* dbv, float* db_dense, float* partial,
                     size_t partial_floats, hipStream_t s);
size_t heads_bwd_partial_floats(int64_t n, int J, int A);

// ---- loss, targets, optimiser
hipError_t gae(int T, int E, const float* r, const float* v, const uint8_t* d, const float* nv,
               const uint8_t* nd, float gamma, float lam, float* adv, float* ret, hipStream_t s);
hipError_t vtrace(int T, int E, const float* mu, const float* pi, const float* r, const float* v,
                  const uint8_t* d, const float* bv, const uint8_t* nd, float gamma, float lam,
                  float rho_bar, float c_bar, float pg_rho_bar, float* vs, float* pg,
                  hipStream_t s);
// Losses without a workspace. stats [8] holds the advantage statistics (entries 6, 7) between
// launches; above 16384 rows dv holds the per-workgroup partial sums until the gradients are
// written there.
hipError_t ppo_loss(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                    const float* old_logp, const float* adv, const float* ret,
                    const int32_t* rows, int norm_adv, float clip, float vf, float ent,
                    float* dz, float* dv, float* stats, hipStream_t s);
hipError_t impala_loss(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                       const float* vs, const float* pg, float pgc, float vf, float ent,
                       float* dz, float* dv, float* stats, hipStream_t s);
// The same results (bit-identical) over many workgroups, for callers with a workspace of
// loss_ws_bytes(m) bytes (the advantage statistics and the per-row loss terms, or above 16384
// rows the per-workgroup partial sums).
size_t loss_ws_bytes(int64_t m);
hipError_t ppo_loss_ws(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                       const float* old_logp, const float* adv, const float* ret, const int32_t* rows,
                       int norm_adv, float clip, float vf, float ent, float* dz, float* dv, float* stats,
                       void* ws, hipStream_t s, const float* ms_pre = nullptr);
// PPO advantage mean / std of nmb minibatches of m rows each (minibatch u: rows + (u / per) *
// stride2 + (u % per) * stride) into ms[2u], ms[2u + 1], in one launch; ppo_loss_ws takes
// minibatch u's pair as ms_pre (bit-identical to the statistics it forms itself) where
// ppo_adv_stats_batched(m).
bool ppo_adv_stats_batched(int64_t m);
hipError_t ppo_adv_stats(int64_t m, int nmb, const float* adv, const int32_t* rows, int64_t stride, int per,
                         int64_t stride2, float* ms, hipStream_t s);
hipError_t impala_loss_ws(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                          const float* vs, const float* pg, float pgc, float vf, float ent, float* dz,
                          float* dv, float* stats, void* ws, hipStream_t s);
// IMPALA minibatch gather (env block [e0, e0 + Eb) of a [T, E] rollout): rows [(T+1)*Eb]
// rollout row indices (the last Eb are the bootstrap frames), act, mu, r, d [T*Eb], nd [Eb].
struct EnvBlock {
    int32_t* rows; int32_t* act; float* mu; float* r; uint8_t* d; uint8_t* nd;
};
hipError_t env_block_gather(int T, int E, int e0, int Eb, const int32_t* act, const float* mu, const float* r,
                            const uint8_t* d, const uint8_t* nd, const EnvBlock& b, hipStream_t s);
hipError_t action_logp(int64_t m, int A, const float* z, const int32_t* act, float* logp,
                       hipStream_t s);
hipError_t gumbel_max(int64_t m, int A, const float* z, const float* g, int32_t* act,
                      float* logp, hipStream_t s);
size_t adam_partial_floats(int64_t n);
// The allocation-free optimiser's per-device norm-partial buffer (a file-scope device array):
// its size, and its address on the current device (looked up once per device).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(float** out);
// omb1 = 1 - b1, omb2 = 1 - b2, bc1 = 1 - b1^t, bc2 = 1 - b2^t, all formed in double.
enum { OPT_ADAM = 0, OPT_RMSPROP = 1 };
// Adam: b1, b2, omb1 = 1 - b1, omb2 = 1 - b2 (formed in double), bc1 = 1 - b1^t, bc2 = 1 - b2^t.
// RMSprop: b2 = decay, omb2 = 1 - decay; m unused; v holds nu.
struct OptArgs {
    int64_t n;
    float* p; const float* g; float* m; float* v;
    float lr, b1, b2, omb1, omb2, bc1, bc2, eps, max_norm;
    // optional bf16 mirror of p[mir_off, mir_off + mir_len): mir[i - mir_off] = bf16(p[i]) as
    // updated (the copy the bf16 forward's dense GEMMs read); NULL for none
    uint16_t* mir; int64_t mir_off, mir_len;
};
// Global-norm clip then one optimiser step; stats [2] = [pre-clip norm, nonfinite] or NULL.
hipError_t clip_opt_step(int opt, const OptArgs& a, float* stats, float* partial, hipStream_t s);
// Largest dynamic LDS allocation per workgroup on the current device (bytes).
size_t lds_limit();
// Workgroups of kernel `fn` (with `threads` threads and `lds` bytes of dynamic LDS) that are
// resident at once on the whole current device; sizes persistent grids (cached).
int resident_blocks(const void* fn, int threads, size_t lds);

// ---- achievable MFMA throughput: `blocks` workgroups of 4 waves, each wave `iters` rounds of
// 8 independent 16x16x32 bf16 MFMAs on register operands; one float per thread to `sink`
hipError_t mfma_probe(int blocks, int iters, float* sink, hipStream_t s);
int64_t mfma_probe_flop(int blocks, int iters);

}  // namespace cb
