// 3x3 stride-2 SAME max-pool over NHWC activations, as the IMPALA-ResNet stages use.
// Padding follows XLA's SAME split: P = max((out-1)*2 + 3 - in, 0), pad_lo = P/2, and the
// padded cells never win (they behave as -inf). The forward pass also writes the argmax
// (0..8, row-major window order, first maximum wins) so the backward pass can route each
// window's gradient with a gather: every input cell sums the gradients of the (at most
// 2x2) windows whose argmax it is, in a fixed order -- no atomics.
//
// One thread handles VEC consecutive channels (8 in bf16 when the channel count allows, else
// 4) of one output cell (forward) or of a 2x2 block of input cells (backward); grid rows are
// frames, so in-frame indices stay 32-bit and divide exactly by a reciprocal multiply. These kernels are bound by
// vector-ALU issue as much as by HBM, so the index math is kept minimal.
#include "common.h"
#include "kernels.h"

namespace cb {

struct PoolGeom {
    int H, W, C, OH, OW, ph, pw, CG;   // CG = C / VEC channel groups
    float inv_CG, inv_W, inv_OW, inv_BW;   // inv_BW = 1 / ceil((W + pw) / 2)
};

static inline PoolGeom pool_geom(int H, int W, int C, int vec) {
    PoolGeom g;
    g.H = H; g.W = W; g.C = C;
    g.OH = (H + 1) / 2; g.OW = (W + 1) / 2;
    const int PH = (g.OH - 1) * 2 + 3 - H, PW = (g.OW - 1) * 2 + 3 - W;
    g.ph = (PH > 0 ? PH : 0) / 2;
    g.pw = (PW > 0 ? PW : 0) / 2;
    g.CG = C / vec;
    g.inv_CG = 1.f / float(g.CG); g.inv_W = 1.f / float(W); g.inv_OW = 1.f / float(g.OW);
    g.inv_BW = 1.f / float((W + g.pw + 1) / 2);
    return g;
}

template <class T, int VEC>
CB_DEV void loadv(const T* p, float* v) {
    if constexpr (VEC == 8) {
        const uint4 u = *reinterpret_cast<const uint4*>(p);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) { v[2 * j] = __uint_as_float(w[j] << 16); v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u); }
    } else {
        load4(p, v);
    }
}

template <class T, int VEC>
CB_DEV void storev(T* p, const float* v) {
    if constexpr (VEC == 8) {
        *reinterpret_cast<uint4*>(p) = make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]),
                                                  pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
    } else {
        store4(p, v[0], v[1], v[2], v[3]);
    }
}

template <class T, int VEC>
__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                          uint8_t* __restrict__ arg, PoolGeom g) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= g.OH * g.OW * g.CG) return;
    const int q = qdiv(t, g.inv_CG), c = (t - q * g.CG) * VEC;
    const int oh = qdiv(q, g.inv_OW), ow = q - oh * g.OW;
    const int64_t n = blockIdx.y;
    const T* xf = x + n * g.H * g.W * g.C + c;
    float best[VEC];
    int bi[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) { best[j] = 0.f; bi[j] = -1; }
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
        const int h = oh * 2 + dy - g.ph;
        if (h < 0 || h >= g.H) continue;
#pragma unroll
        for (int dx = 0; dx < 3; ++dx) {
            const int w = ow * 2 + dx - g.pw;
            if (w < 0 || w >= g.W) continue;
            float v[VEC];
            loadv<T, VEC>(xf + uint32_t(h * g.W + w) * g.C, v);
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (bi[j] < 0 || v[j] > best[j]) { best[j] = v[j]; bi[j] = dy * 3 + dx; }
        }
    }
    const uint32_t o = uint32_t(q) * g.C + c;
    const int64_t fo = n * g.OH * g.OW * g.C;
    storev<T, VEC>(y + fo + o, best);
    uint32_t a[VEC / 4];
#pragma unroll
    for (int k = 0; k < VEC / 4; ++k)
        a[k] = uint32_t(bi[4 * k]) | (uint32_t(bi[4 * k + 1]) << 8) | (uint32_t(bi[4 * k + 2]) << 16) |
               (uint32_t(bi[4 * k + 3]) << 24);
    if constexpr (VEC == 8) *reinterpret_cast<uint2*>(arg + fo + o) = make_uint2(a[0], a[1]);
    else *reinterpret_cast<uint32_t*>(arg + fo + o) = a[0];
}

// Backward as a gather over 2x2 input blocks: block (i, j) holds the cells with padded
// coordinates (2i + a, 2j + b), a, b in {0, 1}, and only the windows (i-1 | i, j-1 | j) reach
// it (window (oh, ow) covers padded rows 2oh..2oh+2 and columns 2ow..2ow+2). Every lane runs
// the same four windows, so nothing diverges; each cell adds its windows in (oh, ow) order.
template <class T, int VEC>
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const uint8_t* __restrict__ arg,
                                                          const T* __restrict__ dy,
                                                          T* __restrict__ dx, PoolGeom g) {
    const int BH = (g.H + g.ph + 1) >> 1, BW = (g.W + g.pw + 1) >> 1;
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= BH * BW * g.CG) return;
    const int blk = qdiv(t, g.inv_CG), c = (t - blk * g.CG) * VEC;
    const int i = qdiv(blk, g.inv_BW), j = blk - i * BW;
    const int64_t n = blockIdx.y;
    const uint8_t* af = arg + n * g.OH * g.OW * g.C + c;
    const T* df = dy + n * g.OH * g.OW * g.C + c;
    float a00[VEC], a01[VEC], a10[VEC], a11[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) { a00[e] = 0.f; a01[e] = 0.f; a10[e] = 0.f; a11[e] = 0.f; }
    // The four windows; one outside the pooled grid reads a clamped window with its argmax
    // bytes forced to 0xff, which matches no cell. No branches, so the loads overlap.
    const bool up = i >= 1, left = j >= 1, down = i < g.OH, right = j < g.OW;
    const int ohs[2] = {up ? i - 1 : 0, down ? i : g.OH - 1};
    const int ows[2] = {left ? j - 1 : 0, right ? j : g.OW - 1};
    const bool ok[4] = {up && left, up && right, down && left, down && right};
    uint32_t ka[4][VEC / 4];
    float v[4][VEC];
#pragma unroll
    for (int wdw = 0; wdw < 4; ++wdw) {
        const uint32_t o = uint32_t(ohs[wdw >> 1] * g.OW + ows[wdw & 1]) * g.C;
        if constexpr (VEC == 8) {
            const uint2 u = *reinterpret_cast<const uint2*>(af + o);
            ka[wdw][0] = ok[wdw] ? u.x : 0xffffffffu;
            ka[wdw][1] = ok[wdw] ? u.y : 0xffffffffu;
        } else {
            const uint32_t u = *reinterpret_cast<const uint32_t*>(af + o);
            ka[wdw][0] = ok[wdw] ? u : 0xffffffffu;
        }
        loadv<T, VEC>(df + o, v[wdw]);
    }
    // cell <- window: a00 <- (i-1,j-1):8, (i-1,j):6, (i,j-1):2, (i,j):0; a01 <- (i-1,j):7, (i,j):1;
    // a10 <- (i,j-1):5, (i,j):3; a11 <- (i,j):4 -- each in (oh, ow) order
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
        uint32_t k[4];
#pragma unroll
        for (int wdw = 0; wdw < 4; ++wdw) k[wdw] = (ka[wdw][e >> 2] >> (8 * (e & 3))) & 0xffu;
        a00[e] += k[0] == 8 ? v[0][e] : 0.f;
        a00[e] += k[1] == 6 ? v[1][e] : 0.f;
        a00[e] += k[2] == 2 ? v[2][e] : 0.f;
        a00[e] += k[3] == 0 ? v[3][e] : 0.f;
        a01[e] += k[1] == 7 ? v[1][e] : 0.f;
        a01[e] += k[3] == 1 ? v[3][e] : 0.f;
        a10[e] += k[2] == 5 ? v[2][e] : 0.f;
        a10[e] += k[3] == 3 ? v[3][e] : 0.f;
        a11[e] += k[3] == 4 ? v[3][e] : 0.f;
    }
    T* xf = dx + n * g.H * g.W * g.C + c;
    const int h0 = 2 * i - g.ph, w0 = 2 * j - g.pw;
    const bool r0 = h0 >= 0, r1 = h0 + 1 < g.H, c0 = w0 >= 0, c1 = w0 + 1 < g.W;
    const int o = (h0 * g.W + w0) * g.C;   // negative at a top / left border; each sum below is
                                           // formed before it offsets the pointer, and only
                                           // for cells inside the frame
    if (r0 && c0) storev<T, VEC>(xf + o, a00);
    if (r0 && c1) storev<T, VEC>(xf + (o + g.C), a01);
    if (r1 && c0) storev<T, VEC>(xf + (o + g.W * g.C), a10);
    if (r1 && c1) storev<T, VEC>(xf + (o + (g.W + 1) * g.C), a11);
}

// Frames per launch: grid rows are frames (at most 65535 per launch).
constexpr int64_t kPoolFrames = 65535;

template <class T, int VEC>
static hipError_t pool_fwd_launch(int64_t n, int H, int W, int C, const T* x, T* y, uint8_t* arg,
                                  hipStream_t s) {
    const PoolGeom g = pool_geom(H, W, C, VEC);
    const int per = g.OH * g.OW * g.CG;
    for (int64_t n0 = 0; n0 < n; n0 += kPoolFrames) {
        const int64_t nn = n - n0 < kPoolFrames ? n - n0 : kPoolFrames;
        const int64_t in0 = n0 * H * W * C, out0 = n0 * g.OH * g.OW * C;
        hipLaunchKernelGGL((maxpool_fwd_kernel<T, VEC>), dim3(unsigned((per + 255) / 256), unsigned(nn)),
                           dim3(256), 0, s, x + in0, y + out0, arg + out0, g);
    }
    return hipGetLastError();
}

template <class T, int VEC>
static hipError_t pool_bwd_launch(int64_t n, int H, int W, int C, const uint8_t* arg, const T* dy, T* dx,
                                  hipStream_t s) {
    const PoolGeom g = pool_geom(H, W, C, VEC);
    const int per = ((H + g.ph + 1) / 2) * ((W + g.pw + 1) / 2) * g.CG;
    for (int64_t n0 = 0; n0 < n; n0 += kPoolFrames) {
        const int64_t nn = n - n0 < kPoolFrames ? n - n0 : kPoolFrames;
        const int64_t in0 = n0 * H * W * C, out0 = n0 * g.OH * g.OW * C;
        hipLaunchKernelGGL((maxpool_bwd_kernel<T, VEC>), dim3(unsigned((per + 255) / 256), unsigned(nn)),
                           dim3(256), 0, s, arg + out0, dy + out0, dx + in0, g);
    }
    return hipGetLastError();
}

hipError_t maxpool_fwd(int prec, int n, int H, int W, int C, const void* x, void* y, uint8_t* arg,
                       hipStream_t s) {
    if (n <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return cb_key("pool_fwd", prec, std::to_string(C) + "/" + cb_dims(H, W)); });
    if (prec == BF16) {
        const uint16_t* xs = static_cast<const uint16_t*>(x);
        uint16_t* ys = static_cast<uint16_t*>(y);
        return C % 8 == 0 ? pool_fwd_launch<uint16_t, 8>(n, H, W, C, xs, ys, arg, s)
                          : pool_fwd_launch<uint16_t, 4>(n, H, W, C, xs, ys, arg, s);
    }
    return pool_fwd_launch<float, 4>(n, H, W, C, static_cast<const float*>(x), static_cast<float*>(y), arg, s);
}

hipError_t maxpool_bwd(int prec, int n, int H, int W, int C, const uint8_t* arg, const void* dy,
                       void* dx, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return cb_key("pool_bwd", prec, std::to_string(C) + "/" + cb_dims(H, W)); });
    if (prec == BF16) {
        const uint16_t* ds = static_cast<const uint16_t*>(dy);
        uint16_t* xs = static_cast<uint16_t*>(dx);
        return C % 8 == 0 ? pool_bwd_launch<uint16_t, 8>(n, H, W, C, arg, ds, xs, s)
                          : pool_bwd_launch<uint16_t, 4>(n, H, W, C, arg, ds, xs, s);
    }
    return pool_bwd_launch<float, 4>(n, H, W, C, arg, static_cast<const float*>(dy), static_cast<float*>(dx), s);
}

}  // namespace cb
