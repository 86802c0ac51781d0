// 3x3 stride-2 SAME max-pool over NHWC activations, as the IMPALA-ResNet stages use.
// Padding follows XLA's SAME split: P = max((out-1)*2 + 3 - in, 0), pad_lo = P/2, and the
// padded cells never win (they behave as -inf). The forward pass also writes the argmax
// (0..8, row-major window order, first maximum wins) so the backward pass can route each
// window's gradient with a gather: every input cell sums the gradients of the (at most
// 2x2) windows whose argmax it is, in a fixed order -- no atomics.
//
// One thread handles 4 consecutive channels of one output (forward) or input (backward)
// cell, so each access is an 8-byte (bf16) or 16-byte (fp32) vector.
#include "common.h"
#include "kernels.h"

namespace cb {

struct PoolGeom {
    int H, W, C, OH, OW, ph, pw;
};

static inline PoolGeom pool_geom(int H, int W, int C) {
    PoolGeom g;
    g.H = H; g.W = W; g.C = C;
    g.OH = (H + 1) / 2; g.OW = (W + 1) / 2;
    const int PH = (g.OH - 1) * 2 + 3 - H, PW = (g.OW - 1) * 2 + 3 - W;
    g.ph = (PH > 0 ? PH : 0) / 2;
    g.pw = (PW > 0 ? PW : 0) / 2;
    return g;
}

template <class T>
__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                          uint8_t* __restrict__ arg, PoolGeom g,
                                                          int64_t total4) {
    const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (t >= total4) return;
    const int C4 = g.C / 4;
    const int c = int(t % C4) * 4;
    int64_t r = t / C4;
    const int ow = int(r % g.OW); r /= g.OW;
    const int oh = int(r % g.OH);
    const int64_t n = r / g.OH;
    float best[4];
    int bi[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) { best[j] = 0.f; bi[j] = -1; }
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
        const int h = oh * 2 + dy - g.ph;
        if (h < 0 || h >= g.H) continue;
#pragma unroll
        for (int dx = 0; dx < 3; ++dx) {
            const int w = ow * 2 + dx - g.pw;
            if (w < 0 || w >= g.W) continue;
            float v[4];
            load4(x + ((n * g.H + h) * g.W + w) * g.C + c, v);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (bi[j] < 0 || v[j] > best[j]) { best[j] = v[j]; bi[j] = dy * 3 + dx; }
        }
    }
    const int64_t o = ((n * g.OH + oh) * g.OW + ow) * g.C + c;
    store4(y + o, best[0], best[1], best[2], best[3]);
    *reinterpret_cast<uint32_t*>(arg + o) =
        uint32_t(bi[0]) | (uint32_t(bi[1]) << 8) | (uint32_t(bi[2]) << 16) | (uint32_t(bi[3]) << 24);
}

template <class T>
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const uint8_t* __restrict__ arg,
                                                          const T* __restrict__ dy,
                                                          T* __restrict__ dx, PoolGeom g,
                                                          int64_t total4) {
    const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (t >= total4) return;
    const int C4 = g.C / 4;
    const int c = int(t % C4) * 4;
    int64_t r = t / C4;
    const int w = int(r % g.W); r /= g.W;
    const int h = int(r % g.H);
    const int64_t n = r / g.H;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    // windows oh with oh*2 - ph <= h <= oh*2 - ph + 2
    const int hp = h + g.ph, wp = w + g.pw;
    const int oh_lo = hp >= 2 ? (hp - 1) / 2 : 0, oh_hi = hp / 2 < g.OH - 1 ? hp / 2 : g.OH - 1;
    const int ow_lo = wp >= 2 ? (wp - 1) / 2 : 0, ow_hi = wp / 2 < g.OW - 1 ? wp / 2 : g.OW - 1;
    for (int oh = oh_lo; oh <= oh_hi; ++oh) {
        for (int ow = ow_lo; ow <= ow_hi; ++ow) {
            const int k = (hp - oh * 2) * 3 + (wp - ow * 2);
            const int64_t o = ((n * g.OH + oh) * g.OW + ow) * g.C + c;
            const uint32_t a4 = *reinterpret_cast<const uint32_t*>(arg + o);
            float v[4];
            load4(dy + o, v);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (int((a4 >> (8 * j)) & 0xff) == k) acc[j] += v[j];
        }
    }
    store4(dx + ((n * g.H + h) * g.W + w) * g.C + c, acc[0], acc[1], acc[2], acc[3]);
}

hipError_t maxpool_fwd(int prec, int n, int H, int W, int C, const void* x, void* y, uint8_t* arg,
                       hipStream_t s) {
    const PoolGeom g = pool_geom(H, W, C);
    const int64_t total4 = int64_t(n) * g.OH * g.OW * (C / 4);
    if (total4 <= 0) return hipSuccess;
    const dim3 grid(unsigned((total4 + 255) / 256));
    ProfScope ps(s, [&] { return cb_key("pool_fwd", prec, std::to_string(C) + "/" + cb_dims(H, W)); });
    if (prec == BF16)
        hipLaunchKernelGGL(maxpool_fwd_kernel<uint16_t>, grid, dim3(256), 0, s,
                           static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y), arg, g, total4);
    else
        hipLaunchKernelGGL(maxpool_fwd_kernel<float>, grid, dim3(256), 0, s,
                           static_cast<const float*>(x), static_cast<float*>(y), arg, g, total4);
    return hipGetLastError();
}

hipError_t maxpool_bwd(int prec, int n, int H, int W, int C, const uint8_t* arg, const void* dy,
                       void* dx, hipStream_t s) {
    const PoolGeom g = pool_geom(H, W, C);
    const int64_t total4 = int64_t(n) * H * W * (C / 4);
    if (total4 <= 0) return hipSuccess;
    const dim3 grid(unsigned((total4 + 255) / 256));
    ProfScope ps(s, [&] { return cb_key("pool_bwd", prec, std::to_string(C) + "/" + cb_dims(H, W)); });
    if (prec == BF16)
        hipLaunchKernelGGL(maxpool_bwd_kernel<uint16_t>, grid, dim3(256), 0, s, arg,
                           static_cast<const uint16_t*>(dy), static_cast<uint16_t*>(dx), g, total4);
    else
        hipLaunchKernelGGL(maxpool_bwd_kernel<float>, grid, dim3(256), 0, s, arg,
                           static_cast<const float*>(dy), static_cast<float*>(dx), g, total4);
    return hipGetLastError();
}

}  // namespace cb
