// 3x3 stride-2 SAME max-pool over NHWC activations, as the IMPALA-ResNet stages use.
// Padding follows XLA's SAME split: P = max((out-1)*2 + 3 - in, 0), pad_lo = P/2, and the
// padded cells never win (they behave as -inf). The forward pass also writes the argmax
// (0..8, row-major window order, first maximum wins) so the backward pass can route each
// window's gradient with a gather: every input cell sums the gradients of the (at most
// 2x2) windows whose argmax it is, in a fixed order -- no atomics.
//
// One thread handles VEC consecutive channels (8 in bf16 when the channel count allows, else
// 4) of one output (forward) or input (backward) cell; grid rows are frames, so in-frame
// indices stay 32-bit and divide exactly by a reciprocal multiply. These kernels are bound by
// vector-ALU issue as much as by HBM, so the index math is kept minimal.
#include "common.h"
#include "kernels.h"

namespace cb {

struct PoolGeom {
    int H, W, C, OH, OW, ph, pw, CG;   // CG = C / VEC channel groups
    float inv_CG, inv_W, inv_OW;
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

template <class T, int VEC>
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const uint8_t* __restrict__ arg,
                                                          const T* __restrict__ dy,
                                                          T* __restrict__ dx, PoolGeom g) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= g.H * g.W * g.CG) return;
    const int q = qdiv(t, g.inv_CG), c = (t - q * g.CG) * VEC;
    const int h = qdiv(q, g.inv_W), w = q - h * g.W;
    const int64_t n = blockIdx.y;
    const int64_t fo = n * g.OH * g.OW * g.C;
    const uint8_t* af = arg + fo + c;
    const T* df = dy + fo + c;
    float acc[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
    // windows oh with oh*2 - ph <= h <= oh*2 - ph + 2 (one or two per axis)
    const int hp = h + g.ph, wp = w + g.pw;
    const int oh_lo = hp >= 2 ? (hp - 1) >> 1 : 0, oh_hi = (hp >> 1) < g.OH - 1 ? hp >> 1 : g.OH - 1;
    const int ow_lo = wp >= 2 ? (wp - 1) >> 1 : 0, ow_hi = (wp >> 1) < g.OW - 1 ? wp >> 1 : g.OW - 1;
    for (int oh = oh_lo; oh <= oh_hi; ++oh) {
        for (int ow = ow_lo; ow <= ow_hi; ++ow) {
            const uint32_t k = uint32_t((hp - oh * 2) * 3 + (wp - ow * 2));
            const uint32_t o = uint32_t(oh * g.OW + ow) * g.C;
            uint32_t a4[VEC / 4];
            if constexpr (VEC == 8) { const uint2 u = *reinterpret_cast<const uint2*>(af + o); a4[0] = u.x; a4[1] = u.y; }
            else a4[0] = *reinterpret_cast<const uint32_t*>(af + o);
            float v[VEC];
            loadv<T, VEC>(df + o, v);
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (((a4[j >> 2] >> (8 * (j & 3))) & 0xffu) == k) acc[j] += v[j];
        }
    }
    storev<T, VEC>(dx + n * g.H * g.W * g.C + uint32_t(q) * g.C + c, acc);
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
    const int per = H * W * g.CG;
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
