// IMPALA-ResNet forward / backward launch sequences on one stream.
//
// Network (the "IMPALA's ResNet" the paper trains with, Section 5): for each of three
// stages, conv3x3 -> maxpool3x3/2 -> 2 x [x + conv(relu(conv(relu(x))))]; then relu,
// flatten (H, W, C), dense + relu, and the policy-logit / value heads.
//
// Saved for the backward pass (all frame-major, `cap` frames): every stage's pre-pool
// conv output (only its pool argmax is read back), the pool argmax, the three residual
// stream tensors x0..x2 and the two inner activations t0, t1 per stage, and the dense
// output h. The backward pass reads the residual inputs with relu applied on load, so no
// relu'd copies are stored.
#include <algorithm>
#include <cstring>

#include "kernels.h"
#include "plan.h"

namespace cb {

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

std::string check_net(const impala_net_t* net) {
    if (!net) return "net is NULL";
    if (net->in_c != 4) return "in_c must be 4 (stacked uint8 frames)";
    if (net->in_h < 1 || net->in_h > 128 || net->in_w < 1 || net->in_w > 128)
        return "in_h and in_w must be in [1, 128]";
    for (int i = 0; i < 3; ++i) {
        const int c = net->ch[i];
        if (c != 16 && c != 32 && c != 64) return "stage channels must be 16, 32 or 64";
        if (i > 0 && c < net->ch[i - 1]) return "stage channels must be non-decreasing";
    }
    if (net->hidden < 1 || net->hidden > 4096) return "hidden must be in [1, 4096]";
    if (net->num_actions < 1 || net->num_actions > 64) return "num_actions must be in [1, 64]";
    return "";
}

ParamOffsets param_offsets(const impala_net_t& net) {
    ParamOffsets o;
    int64_t off = 0;
    int cin = net.in_c, h = net.in_h, w = net.in_w;
    for (int s = 0; s < 3; ++s) {
        const int c = net.ch[s];
        for (int k = 0; k < 5; ++k) {
            const int ci = k == 0 ? cin : c;
            o.conv_w[s][k] = off; off += int64_t(9) * ci * c;
            o.conv_b[s][k] = off; off += c;
        }
        cin = c;
        h = (h + 1) / 2;
        w = (w + 1) / 2;
    }
    const int64_t flat = int64_t(h) * w * net.ch[2];
    o.dense_w = off; off += flat * net.hidden;
    o.dense_b = off; off += net.hidden;
    o.logits_w = off; off += int64_t(net.hidden) * net.num_actions;
    o.logits_b = off; off += net.num_actions;
    o.value_w = off; off += net.hidden;
    o.value_b = off; off += 1;
    o.total = off;
    return o;
}

NetPlan make_plan(const impala_net_t& net, int prec, int64_t cap, int training) {
    NetPlan p;
    std::memset(&p, 0, sizeof(p));
    p.net = net;
    p.prec = prec;
    p.es = prec == BF16 ? 2 : 4;
    p.cap = cap;
    p.training = training;
    p.H[0] = net.in_h; p.W[0] = net.in_w; p.C[0] = net.in_c;
    for (int s = 0; s < 3; ++s) {
        p.H[s + 1] = (p.H[s] + 1) / 2;
        p.W[s + 1] = (p.W[s] + 1) / 2;
        p.C[s + 1] = net.ch[s];
    }
    p.flat = p.H[3] * p.W[3] * p.C[3];
    p.hidden = net.hidden;
    p.A = net.num_actions;
    p.po = param_offsets(net);

    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t o = off; off += align256(bytes); return o; };
    int64_t maxact = std::max<int64_t>(p.hidden, p.flat);
    for (int s = 0; s < 3; ++s) {
        const int64_t conv_el = int64_t(p.H[s]) * p.W[s] * p.C[s + 1];
        const int64_t pool_el = int64_t(p.H[s + 1]) * p.W[s + 1] * p.C[s + 1];
        maxact = std::max(maxact, conv_el);
        p.c[s] = take(prec == BF16 ? 0 : size_t(cap * conv_el) * p.es);   // bf16 pools on chip
        p.idx[s] = take(size_t(cap * pool_el));
        for (int k = 0; k < 3; ++k) p.x[s][k] = take(size_t(cap * pool_el) * p.es);
        for (int k = 0; k < 2; ++k) p.t[s][k] = take(size_t(cap * pool_el) * p.es);
    }
    p.h = take(size_t(cap) * p.hidden * p.es);
    p.wdb = take(prec == BF16 ? size_t(p.flat) * p.hidden * 2 : 0);
    // split-K / column-sum / weight-gradient partials, shared by the launches in turn. The
    // GEMM launcher never splits beyond this capacity, so the sizing only affects speed.
    size_t sc = 0;
    for (int64_t nn = cap; nn >= 1; nn = nn > 64 ? nn / 2 : 0) {
        sc = std::max(sc, gemm_partial_floats(p.hidden, int(nn), p.flat));
        if (training) {
            sc = std::max(sc, heads_bwd_partial_floats(nn, p.hidden, p.A));
            sc = std::max(sc, gemm_partial_floats(p.hidden, p.flat, int(nn)));
            sc = std::max(sc, gemm_partial_floats(p.flat, int(nn), p.hidden));
        }
    }
    if (training) {
        for (int k = 0; k < 3; ++k) p.g[k] = take(size_t(cap * maxact) * p.es);
        for (int s = 0; s < 3; ++s) {
            sc = std::max(sc, wgrad_partial_floats(prec, p.C[s], p.C[s + 1], p.H[s], p.W[s]));
            sc = std::max(sc, wgrad_partial_floats(prec, p.C[s + 1], p.C[s + 1], p.H[s + 1], p.W[s + 1]));
            if (prec == BF16) {
                if (s == 0) sc = std::max(sc, pool_wgrad_u8_partial_floats(p.C[1]));
                sc = std::max(sc, conv3x3_bwd_partial_floats(p.C[s], p.C[s + 1]));
                sc = std::max(sc, conv3x3_bwd_partial_floats(p.C[s + 1], p.C[s + 1]));
                sc = std::max(sc, resblock_bwd_partial_floats(p.C[s + 1]));
            }
        }
    }
    // the trunk backward's fused kernels defer each weight-gradient reduce to the next launch,
    // alternating between two partial buffers: the second one follows the shared scratch
    size_t sc2 = 0;
    if (training && prec == BF16)
        for (int s = 0; s < 3; ++s) {
            if (s == 0) sc2 = std::max(sc2, pool_wgrad_u8_partial_floats(p.C[1]));
            sc2 = std::max(sc2, conv3x3_bwd_partial_floats(p.C[s], p.C[s + 1]));
            sc2 = std::max(sc2, conv3x3_bwd_partial_floats(p.C[s + 1], p.C[s + 1]));
            sc2 = std::max(sc2, resblock_bwd_partial_floats(p.C[s + 1]));
        }
    p.scratch_floats = sc;
    p.scratch_bytes = (sc + sc2) * sizeof(float);
    p.scratch = take(p.scratch_bytes);
    p.total = off;
    return p;
}

#define CB_TRY(x)                          \
    do {                                   \
        hipError_t e_ = (x);               \
        if (e_ != hipSuccess) return e_;   \
    } while (0)

hipError_t run_forward(const NetPlan& p, const float* params, const uint8_t* obs,
                       const int32_t* row_idx, int64_t n, char* ws, float* logits, float* value,
                       hipStream_t s, bool dense_bf16_ready) {
    if (n <= 0) return hipSuccess;
    const ParamOffsets& po = p.po;
    for (int st = 0; st < 3; ++st) {
        ConvArgs a{};
        a.x = st == 0 ? static_cast<const void*>(obs) : static_cast<const void*>(ws + p.x[st - 1][2]);
        a.row_idx = st == 0 ? row_idx : nullptr;
        a.w = params + po.conv_w[st][0];
        a.bias = params + po.conv_b[st][0];
        a.n = int(n); a.H = p.H[st]; a.W = p.W[st];
        a.scale = st == 0 ? 1.f / 255.f : 1.f;
        if (p.prec == BF16) {
            // conv and pool in one pass: the full-resolution output stays on chip
            a.y = ws + p.x[st][0];
            a.arg = reinterpret_cast<uint8_t*>(ws + p.idx[st]);
            CB_TRY(conv3x3_pool(p.C[st], p.C[st + 1], st == 0 ? IN_U8 : IN_PLAIN, a, s));
        } else {
            a.y = ws + p.c[st];
            CB_TRY(conv3x3(p.prec, p.C[st], p.C[st + 1], st == 0 ? IN_U8 : IN_PLAIN, 0, a, s));
            CB_TRY(maxpool_fwd(p.prec, int(n), p.H[st], p.W[st], p.C[st + 1], ws + p.c[st], ws + p.x[st][0],
                               reinterpret_cast<uint8_t*>(ws + p.idx[st]), s));
        }
        const int C = p.C[st + 1];
        for (int r = 0; r < 2; ++r) {
            if (p.prec == BF16 && resblock_fwd_supported(C)) {
                // the whole block in one pass: t and y written, x read once
                ResBlockArgs rb{};
                rb.x = ws + p.x[st][r];
                rb.w1 = params + po.conv_w[st][1 + 2 * r]; rb.b1 = params + po.conv_b[st][1 + 2 * r];
                rb.w2 = params + po.conv_w[st][2 + 2 * r]; rb.b2 = params + po.conv_b[st][2 + 2 * r];
                rb.t = ws + p.t[st][r]; rb.y = ws + p.x[st][r + 1];
                rb.n = int(n); rb.H = p.H[st + 1]; rb.W = p.W[st + 1];
                CB_TRY(resblock_fwd(C, rb, s));
                continue;
            }
            ConvArgs b{};
            b.x = ws + p.x[st][r]; b.w = params + po.conv_w[st][1 + 2 * r];
            b.bias = params + po.conv_b[st][1 + 2 * r]; b.y = ws + p.t[st][r];
            b.n = int(n); b.H = p.H[st + 1]; b.W = p.W[st + 1]; b.scale = 1.f;
            CB_TRY(conv3x3(p.prec, C, C, IN_RELU, 0, b, s));
            ConvArgs c{};
            c.x = ws + p.t[st][r]; c.w = params + po.conv_w[st][2 + 2 * r];
            c.bias = params + po.conv_b[st][2 + 2 * r]; c.add = ws + p.x[st][r];
            c.y = ws + p.x[st][r + 1];
            c.n = int(n); c.H = p.H[st + 1]; c.W = p.W[st + 1]; c.scale = 1.f;
            CB_TRY(conv3x3(p.prec, C, C, IN_RELU, 0, c, s));
        }
    }
    // dense: h[i][j] = relu(b[j] + sum_k relu(x)[i][k] W[k][j])
    // bf16: the dense weights are cast once per pass (or were written by the optimiser step
    // that produced them), so both dense GEMMs read bf16 operands
    const bool wbf = p.prec == BF16;
    if (wbf && !dense_bf16_ready) CB_TRY(cast_bf16(params + po.dense_w, reinterpret_cast<uint16_t*>(ws + p.wdb),
                              int64_t(p.flat) * p.hidden, s));
    GemmArgs d{};
    d.a = wbf ? static_cast<const void*>(ws + p.wdb) : static_cast<const void*>(params + po.dense_w);
    d.a_f32 = !wbf; d.a_kcontig = 0; d.lda = p.hidden;
    d.b = ws + p.x[2][2]; d.b_f32 = p.prec == FP32; d.b_kcontig = 1; d.ldb = p.flat; d.b_relu = 1;
    d.M = p.hidden; d.N = int(n); d.K = p.flat;
    d.alpha = 1.f; d.bias1 = params + po.dense_b; d.relu = 1;
    d.out1 = ws + p.h; d.ld1 = p.hidden; d.out1_f32 = p.prec == FP32; d.msplit = p.hidden;
    d.partial = reinterpret_cast<float*>(ws + p.scratch); d.partial_floats = p.scratch_bytes / sizeof(float);
    CB_TRY(gemm(p.prec, d, s));
    // heads: logits[i][a] = bl[a] + sum_j h[i][j] Wl[j][a]; value[i] = bv + sum_j h[i][j] Wv[j]
    HeadsArgs hd{ws + p.h, params + po.logits_w, params + po.logits_b, params + po.value_w,
                 params + po.value_b, n, p.hidden, p.A};
    CB_TRY(heads_fwd(p.prec, hd, logits, value, s));
    return hipSuccess;
}

hipError_t run_backward(const NetPlan& p, const float* params, const uint8_t* obs,
                        const int32_t* row_idx, int64_t n, char* ws, const float* dlogits,
                        const float* dvalue, float* grads, hipStream_t s) {
    const ParamOffsets& po = p.po;
    if (n <= 0) return fill_zero(grads, po.total, s);
    const int A = p.A;
    const int st_f32 = p.prec == FP32;
    float* scratch = reinterpret_cast<float*>(ws + p.scratch);
    char* G[3] = {ws + p.g[0], ws + p.g[1], ws + p.g[2]};

    // heads: dh = (dz Wh^T) * (h > 0), the head weight / bias gradients and the dense bias
    // gradient (column sums of dh) from one pass over h
    HeadsArgs hd{ws + p.h, params + po.logits_w, params + po.logits_b, params + po.value_w,
                 params + po.value_b, n, p.hidden, A};
    CB_TRY(heads_bwd(p.prec, hd, dlogits, dvalue, G[0], grads + po.logits_w, grads + po.logits_b,
                     grads + po.value_w, grads + po.value_b, grads + po.dense_b, scratch,
                     p.scratch_bytes / sizeof(float), s));
    // dense weight gradient: dWd[k][j] = sum_i relu(x)[i][k] dh[i][j]
    GemmArgs dw{};
    dw.a = G[0]; dw.a_f32 = st_f32; dw.a_kcontig = 0; dw.lda = p.hidden;
    dw.b = ws + p.x[2][2]; dw.b_f32 = st_f32; dw.b_kcontig = 0; dw.ldb = p.flat; dw.b_relu = 1;
    dw.M = p.hidden; dw.N = p.flat; dw.K = int(n); dw.alpha = 1.f;
    dw.out1 = grads + po.dense_w; dw.ld1 = p.hidden; dw.out1_f32 = 1; dw.msplit = p.hidden;
    dw.partial = scratch; dw.partial_floats = p.scratch_bytes / sizeof(float);
    CB_TRY(gemm(p.prec, dw, s));
    // dense input gradient: dx[i][k] = (sum_j Wd[k][j] dh[i][j]) * (x[i][k] > 0)
    // bf16: the forward pass left the bf16 copy of the same dense weights in the workspace
    const bool wbf = p.prec == BF16;
    GemmArgs dg{};
    dg.a = wbf ? static_cast<const void*>(ws + p.wdb) : static_cast<const void*>(params + po.dense_w);
    dg.a_f32 = !wbf; dg.a_kcontig = 1; dg.lda = p.hidden;
    dg.b = G[0]; dg.b_f32 = st_f32; dg.b_kcontig = 1; dg.ldb = p.hidden;
    dg.M = p.flat; dg.N = int(n); dg.K = p.hidden; dg.alpha = 1.f;
    dg.mask = ws + p.x[2][2]; dg.ldmask = p.flat;
    dg.out1 = G[1]; dg.ld1 = p.flat; dg.out1_f32 = st_f32; dg.msplit = p.flat;
    dg.partial = scratch; dg.partial_floats = p.scratch_bytes / sizeof(float);
    CB_TRY(gemm(p.prec, dg, s));

    int gy = 1;
    auto others = [](int k, int& a, int& b) { a = (k + 1) % 3; b = (k + 2) % 3; };
    // fused conv backward launches: each one's weight-gradient reduce runs at the start of the
    // next fused launch (or a standalone reduce before any other launch), the partials
    // alternating between two buffers
    // (a residual block's backward leaves two: one per conv)
    float* pbuf[2] = {scratch, scratch + p.scratch_floats};
    PendingReduce pend[2] = {};
    int pb = 0;
    auto fused_bwd = [&](int ci, int co, int mode, ConvBwdArgs c) -> hipError_t {
        c.partial = pbuf[pb];
        c.pend = pend[0];
        c.pend2 = pend[1];
        PendingReduce nx{};
        const hipError_t e = conv3x3_bwd(ci, co, mode, c, s, &nx);
        pend[0] = nx;
        pend[1].nparts = 0;
        pb ^= 1;
        return e;
    };
    auto flush = [&]() -> hipError_t {
        hipError_t e = flush_pending_reduce(pend[0], s);
        if (e == hipSuccess) e = flush_pending_reduce(pend[1], s);
        pend[0].nparts = 0;
        pend[1].nparts = 0;
        return e;
    };
    for (int st = 2; st >= 0; --st) {
        const int C = p.C[st + 1], Hs = p.H[st + 1], Ws = p.W[st + 1];
        for (int r = 1; r >= 0; --r) {
            int fa, fb;
            others(gy, fa, fb);
            const int k0 = 1 + 2 * r, k1 = 2 + 2 * r;
            if (p.prec == BF16 && resblock_bwd_preferred(C, Hs, Ws)) {
                // the whole block in one pass: dt stays on chip
                ResBwdArgs rb{};
                rb.dy = G[gy]; rb.t = ws + p.t[st][r]; rb.x = ws + p.x[st][r];
                rb.wa = params + po.conv_w[st][k0]; rb.wb = params + po.conv_w[st][k1]; rb.dx = G[fa];
                rb.dwa = grads + po.conv_w[st][k0]; rb.dba = grads + po.conv_b[st][k0];
                rb.dwb = grads + po.conv_w[st][k1]; rb.dbb = grads + po.conv_b[st][k1];
                rb.partial = pbuf[pb]; rb.pend = pend[0]; rb.pend2 = pend[1];
                rb.n = int(n); rb.H = Hs; rb.W = Ws;
                CB_TRY(resblock_bwd(C, rb, s, pend));
                pb ^= 1;
                gy = fa;
                continue;
            }
            if (p.prec == BF16 && conv3x3_bwd_supported(C, C, IN_RELU, 1, 0)) {
                // each conv's input and weight gradients from one staging of its dy and input
                ConvBwdArgs c1{};
                c1.dy = G[gy]; c1.x = ws + p.t[st][r]; c1.w = params + po.conv_w[st][k1]; c1.dx = G[fa];
                c1.dw = grads + po.conv_w[st][k1]; c1.db = grads + po.conv_b[st][k1];
                c1.n = int(n); c1.H = Hs; c1.W = Ws;
                CB_TRY(fused_bwd(C, C, IN_RELU, c1));
                ConvBwdArgs c0{};
                c0.dy = G[fa]; c0.x = ws + p.x[st][r]; c0.w = params + po.conv_w[st][k0]; c0.add = G[gy];
                c0.dx = G[fb]; c0.dw = grads + po.conv_w[st][k0]; c0.db = grads + po.conv_b[st][k0];
                c0.n = int(n); c0.H = Hs; c0.W = Ws;
                CB_TRY(fused_bwd(C, C, IN_RELU, c0));
                gy = fb;
                continue;
            }
            // y = x + conv1(relu(t)) + b1 with t = conv0(relu(x)) + b0
            CB_TRY(flush());
            WgradArgs w1{};
            w1.x = ws + p.t[st][r]; w1.dy = G[gy]; w1.dw = grads + po.conv_w[st][k1];
            w1.db = grads + po.conv_b[st][k1]; w1.partial = scratch;
            w1.n = int(n); w1.H = Hs; w1.W = Ws; w1.scale = 1.f;
            CB_TRY(conv3x3_wgrad(p.prec, C, C, IN_RELU, w1, s));
            ConvArgs d1{};
            d1.x = G[gy]; d1.w = params + po.conv_w[st][k1]; d1.mask = ws + p.t[st][r]; d1.y = G[fa];
            d1.n = int(n); d1.H = Hs; d1.W = Ws; d1.scale = 1.f;
            CB_TRY(conv3x3(p.prec, C, C, IN_PLAIN, 1, d1, s));
            WgradArgs w0{};
            w0.x = ws + p.x[st][r]; w0.dy = G[fa]; w0.dw = grads + po.conv_w[st][k0];
            w0.db = grads + po.conv_b[st][k0]; w0.partial = scratch;
            w0.n = int(n); w0.H = Hs; w0.W = Ws; w0.scale = 1.f;
            CB_TRY(conv3x3_wgrad(p.prec, C, C, IN_RELU, w0, s));
            ConvArgs d0{};
            d0.x = G[fa]; d0.w = params + po.conv_w[st][k0]; d0.mask = ws + p.x[st][r];
            d0.add = G[gy]; d0.y = G[fb];
            d0.n = int(n); d0.H = Hs; d0.W = Ws; d0.scale = 1.f;
            CB_TRY(conv3x3(p.prec, C, C, IN_PLAIN, 1, d0, s));
            gy = fb;
        }
        int fa, fb;
        others(gy, fa, fb);
        if (st == 0 && p.prec == BF16 && pool_wgrad_u8_supported(C)) {
            // max-pool backward on chip, feeding the frames' conv weight gradient
            PoolWgArgs pa{};
            pa.obs = obs; pa.row_idx = row_idx; pa.dp = G[gy];
            pa.arg = reinterpret_cast<const uint8_t*>(ws + p.idx[0]);
            pa.dw = grads + po.conv_w[0][0]; pa.db = grads + po.conv_b[0][0]; pa.partial = pbuf[pb];
            pa.n = int(n); pa.H = p.H[0]; pa.W = p.W[0];
            pa.pend = pend[0];   // the previous fused launch's reduces run first in this kernel
            pa.pend2 = pend[1];
            pend[0].nparts = 0;
            pend[1].nparts = 0;
            CB_TRY(pool_wgrad_u8(C, pa, s));
            continue;
        }
        if (st > 0 && p.prec == BF16 && conv3x3_bwd_supported(p.C[st], C, IN_PLAIN, 0, 1)) {
            // the stage entry's max-pool backward, input and weight gradients in one pass: the
            // full-resolution conv-output gradient is formed on chip from the pooled one
            ConvBwdArgs ce{};
            ce.dy = G[gy]; ce.arg = reinterpret_cast<const uint8_t*>(ws + p.idx[st]);
            ce.x = ws + p.x[st - 1][2]; ce.w = params + po.conv_w[st][0]; ce.dx = G[fa];
            ce.dw = grads + po.conv_w[st][0]; ce.db = grads + po.conv_b[st][0];
            ce.n = int(n); ce.H = p.H[st]; ce.W = p.W[st];
            CB_TRY(fused_bwd(p.C[st], C, IN_PLAIN, ce));
            gy = fa;
            continue;
        }
        CB_TRY(flush());
        CB_TRY(maxpool_bwd(p.prec, int(n), p.H[st], p.W[st], C,
                           reinterpret_cast<const uint8_t*>(ws + p.idx[st]), G[gy], G[fa], s));
        WgradArgs we{};
        we.x = st == 0 ? static_cast<const void*>(obs) : static_cast<const void*>(ws + p.x[st - 1][2]);
        we.row_idx = st == 0 ? row_idx : nullptr;
        we.dy = G[fa]; we.dw = grads + po.conv_w[st][0]; we.db = grads + po.conv_b[st][0];
        we.partial = scratch; we.n = int(n); we.H = p.H[st]; we.W = p.W[st];
        we.scale = st == 0 ? 1.f / 255.f : 1.f;
        CB_TRY(conv3x3_wgrad(p.prec, p.C[st], C, st == 0 ? IN_U8 : IN_PLAIN, we, s));
        if (st > 0) {
            ConvArgs de{};
            de.x = G[fa]; de.w = params + po.conv_w[st][0]; de.y = G[fb];
            de.n = int(n); de.H = p.H[st]; de.W = p.W[st]; de.scale = 1.f;
            CB_TRY(conv3x3(p.prec, p.C[st], C, IN_PLAIN, 1, de, s));
            gy = fb;
        }
    }
    CB_TRY(flush());
    return hipSuccess;
}

}  // namespace cb
