// Global-norm gradient clipping and Adam over the flat float32 parameter buffer.
//
// Pass 1: each of up to 1024 blocks sums the squares of a fixed strided share of the
// gradient in float64 and writes one partial. Pass 2: every block first re-adds all
// partials in the same fixed order (so every block sees the identical norm), derives the
// clip scale, then updates params, m and v with 16-byte vector accesses. The update is
// HBM-bound: per parameter it reads p, g, m, v and writes p, m, v (28 bytes).
#include "common.h"
#include "kernels.h"

namespace cb {

constexpr int kAdamBlocks = 1024;

size_t adam_partial_floats(int64_t) { return 2 * kAdamBlocks; }

__global__ __launch_bounds__(256) void sumsq_kernel(int64_t n, const float* __restrict__ g,
                                                    double* __restrict__ part) {
    __shared__ double sh[256];
    double s = 0.0;
    const int64_t n4 = n / 4;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n4; i += int64_t(gridDim.x) * 256) {
        const float4 v = g4[i];
        s += double(v.x) * v.x + double(v.y) * v.y + double(v.z) * v.z + double(v.w) * v.w;
    }
    if (blockIdx.x == 0)
        for (int64_t i = n4 * 4 + threadIdx.x; i < n; i += 256) s += double(g[i]) * g[i];
    const double tot = block_sum<256>(s, sh);
    if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

// omb1 = 1 - b1 and omb2 = 1 - b2 arrive precomputed in double precision on the host:
// forming them from the float betas would carry the betas' representation error
// (1 - 0.999f differs from 0.001 by 1.3e-5 relative).
CB_DEV void adam_one(float& p, float g, float& m, float& v, float scale, float lr, float b1,
                     float b2, float omb1, float omb2, float bc1, float bc2, float eps) {
    g *= scale;
    m = b1 * m + omb1 * g;
    v = b2 * v + omb2 * g * g;
    const float mhat = m / bc1, vhat = v / bc2;
    p = p - lr * mhat / (sqrtf(vhat) + eps);
}

__global__ __launch_bounds__(256) void adam_kernel(int64_t n, float* __restrict__ p,
                                                   const float* __restrict__ g, float* __restrict__ m,
                                                   float* __restrict__ v, float lr, float b1, float b2,
                                                   float omb1, float omb2, float bc1, float bc2,
                                                   float eps, float max_norm,
                                                   const double* __restrict__ part, int nparts,
                                                   float* __restrict__ stats) {
    __shared__ double sh[256];
    double s = 0.0;
    for (int i = threadIdx.x; i < nparts; i += 256) s += part[i];
    const double tot = block_sum<256>(s, sh);
    const double norm = sqrt(tot);
    const float scale = (max_norm > 0.f && norm > double(max_norm)) ? float(double(max_norm) / norm) : 1.f;
    if (blockIdx.x == 0 && threadIdx.x == 0 && stats) {
        stats[0] = float(norm);
        stats[1] = isfinite(norm) ? 0.f : 1.f;
    }
    const int64_t n4 = n / 4;
    float4* p4 = reinterpret_cast<float4*>(p);
    float4* m4 = reinterpret_cast<float4*>(m);
    float4* v4 = reinterpret_cast<float4*>(v);
    const float4* g4 = reinterpret_cast<const float4*>(g);
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n4; i += int64_t(gridDim.x) * 256) {
        float4 pp = p4[i], mm = m4[i], vv = v4[i];
        const float4 gg = g4[i];
        adam_one(pp.x, gg.x, mm.x, vv.x, scale, lr, b1, b2, omb1, omb2, bc1, bc2, eps);
        adam_one(pp.y, gg.y, mm.y, vv.y, scale, lr, b1, b2, omb1, omb2, bc1, bc2, eps);
        adam_one(pp.z, gg.z, mm.z, vv.z, scale, lr, b1, b2, omb1, omb2, bc1, bc2, eps);
        adam_one(pp.w, gg.w, mm.w, vv.w, scale, lr, b1, b2, omb1, omb2, bc1, bc2, eps);
        p4[i] = pp; m4[i] = mm; v4[i] = vv;
    }
    if (blockIdx.x == 0)
        for (int64_t i = n4 * 4 + threadIdx.x; i < n; i += 256)
            adam_one(p[i], g[i], m[i], v[i], scale, lr, b1, b2, omb1, omb2, bc1, bc2, eps);
}

hipError_t adam(int64_t n, float* p, const float* g, float* m, float* v, float lr, float b1,
                float b2, float omb1, float omb2, float bc1, float bc2, float eps, float max_norm,
                float* stats, float* partial, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    double* part = reinterpret_cast<double*>(partial);
    int64_t blocks = (n / 4 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > kAdamBlocks) blocks = kAdamBlocks;
    {
        ProfScope ps(s, [&] { return "grad_sumsq/" + std::to_string(n); });
        hipLaunchKernelGGL(sumsq_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, n, g, part);
    }
    ProfScope ps(s, [&] { return "adam/" + std::to_string(n); });
    hipLaunchKernelGGL(adam_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, n, p, g, m, v, lr, b1, b2,
                       omb1, omb2, bc1, bc2, eps, max_norm, part, int(blocks), stats);
    return hipGetLastError();
}

}  // namespace cb
