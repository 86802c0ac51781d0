// Global-norm gradient clipping, then Adam or RMSprop, over the flat float32 parameter buffer.
//
// Pass 1: each of up to 1024 blocks sums the squares of a fixed strided share of the
// gradient in float64 and writes one partial. Pass 2: every block first re-adds all
// partials in the same fixed order (so every block sees the identical norm), derives the
// clip scale, then updates the parameters and the optimiser state with 16-byte vector
// accesses. The update is HBM-bound: per parameter Adam reads p, g, m, v and writes p, m, v
// (28 bytes); RMSprop reads p, g, nu and writes p, nu (20 bytes).
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace cb {

constexpr int kAdamBlocks = 1024;

size_t adam_partial_floats(int64_t) { return 2 * kAdamBlocks; }

// Norm partials of the allocation-free optimiser entry point: one file-scope buffer per GPU
// (each device holds its own copy until the process ends). Host code never passes the name
// `scratch` to a kernel: on the host it is only a stand-in for the symbol, so its device
// address is looked up per device with hipGetSymbolAddress and used instead.
constexpr size_t kNoAllocScratchBytes = size_t(2 * kAdamBlocks) * sizeof(float);
static __device__ __align__(256) double scratch[kNoAllocScratchBytes / sizeof(double)];

size_t noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

hipError_t noalloc_scratch(float** out) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!ptr) return hipErrorInvalidSymbol;
        addr[dev] = ptr;
    }
    *out = static_cast<float*>(addr[dev]);
    return hipSuccess;
}

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
CB_DEV void adam_one(float& p, float g, float& m, float& v, float scale, const OptArgs& a) {
    g *= scale;
    m = a.b1 * m + a.omb1 * g;
    v = a.b2 * v + a.omb2 * g * g;
    const float mhat = m / a.bc1, vhat = v / a.bc2;
    p = p - a.lr * mhat / (sqrtf(vhat) + a.eps);
}

// RMSprop with the decay in b2 and 1 - decay in omb2: nu <- decay nu + (1 - decay) g^2;
// p <- p - lr g / sqrt(nu + eps) (epsilon inside the root; nu starts at zero).
CB_DEV void rms_one(float& p, float g, float& nu, float scale, const OptArgs& a) {
    g *= scale;
    nu = a.b2 * nu + a.omb2 * g * g;
    p = p - a.lr * g / sqrtf(nu + a.eps);
}

template <int OPT>
CB_DEV void opt_one(float& p, float g, float& m, float& v, float scale, const OptArgs& a) {
    if constexpr (OPT == OPT_ADAM) adam_one(p, g, m, v, scale, a);
    else rms_one(p, g, v, scale, a);
}

template <int OPT>
CB_DEV void opt_four(float4& p, const float4& g, float4& m, float4& v, float scale, const OptArgs& a) {
    opt_one<OPT>(p.x, g.x, m.x, v.x, scale, a);
    opt_one<OPT>(p.y, g.y, m.y, v.y, scale, a);
    opt_one<OPT>(p.z, g.z, m.z, v.z, scale, a);
    opt_one<OPT>(p.w, g.w, m.w, v.w, scale, a);
}

// Clip scale from the norm partials (every block re-adds them in the same order); block 0's
// thread 0 records [norm, nonfinite]. pv: this thread's partials (indices t, t + 256, ...).
CB_DEV float clip_scale(const double (&pv)[4], int nparts, float max_norm, double* sh, float* stats) {
    double s = 0.0;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        if (int(threadIdx.x) + 256 * u < nparts) s += pv[u];
    const double norm = sqrt(block_sum<256>(s, sh));
    if (blockIdx.x == 0 && threadIdx.x == 0 && stats) {
        stats[0] = float(norm);
        stats[1] = isfinite(norm) ? 0.f : 1.f;
    }
    return (max_norm > 0.f && norm > double(max_norm)) ? float(double(max_norm) / norm) : 1.f;
}

// The bf16 mirror of updated parameters i .. i+k-1 (those inside the mirrored range).
CB_DEV void mirror_store(const OptArgs& a, int64_t i, const float* v, int k) {
    for (int e = 0; e < k; ++e) {
        const int64_t d = i + e - a.mir_off;
        if (d >= 0 && d < a.mir_len) a.mir[d] = f2bf(v[e]);
    }
}

// Each thread's first float4 of p, g, m, v is loaded before the norm is known (clamped
// index, so the loads are unconditional): their latency overlaps the re-addition of the
// norm partials, which are loaded before them (loads complete in order, so waiting for the
// partials does not wait for the parameters).
template <int OPT>
__global__ __launch_bounds__(256) void opt_kernel(OptArgs a, const double* __restrict__ part, int nparts,
                                                  float* __restrict__ stats) {
    __shared__ double sh[256];
    static_assert(kAdamBlocks <= 4 * 256, "four partials per thread");
    double pv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = int(threadIdx.x) + 256 * u;
        pv[u] = part[i < nparts ? i : 0];
    }
    const int64_t n4 = a.n / 4;
    if (n4 == 0) {   // fewer than four parameters: block 0 alone, element by element
        const float scale = clip_scale(pv, nparts, a.max_norm, sh, stats);
        if (blockIdx.x == 0)
            for (int64_t i = threadIdx.x; i < a.n; i += 256) {
                float mt = OPT == OPT_ADAM ? a.m[i] : 0.f;
                opt_one<OPT>(a.p[i], a.g[i], mt, a.v[i], scale, a);
                if constexpr (OPT == OPT_ADAM) a.m[i] = mt;
                if (a.mir) mirror_store(a, i, &a.p[i], 1);
            }
        return;
    }
    float4* p4 = reinterpret_cast<float4*>(a.p);
    float4* m4 = reinterpret_cast<float4*>(a.m);
    float4* v4 = reinterpret_cast<float4*>(a.v);
    const float4* g4 = reinterpret_cast<const float4*>(a.g);
    const int64_t i0 = int64_t(blockIdx.x) * 256 + threadIdx.x, stride = int64_t(gridDim.x) * 256;
    const int64_t ic = i0 < n4 ? i0 : n4 - 1;
    float4 pp = p4[ic], gg = g4[ic], vv = v4[ic];
    float4 mm = make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (OPT == OPT_ADAM) mm = m4[ic];
    const float scale = clip_scale(pv, nparts, a.max_norm, sh, stats);
    // the mirror takes 8-byte stores where its range and address are 4-element aligned
    const bool mvec = a.mir && (a.mir_off & 3) == 0 && (reinterpret_cast<uintptr_t>(a.mir) & 7) == 0;
    auto mirror4 = [&](int64_t i, const float4& q) {
        if (!a.mir) return;
        const int64_t d = 4 * i - a.mir_off;
        if (mvec) {
            if (d >= 0 && d + 4 <= a.mir_len)
                *reinterpret_cast<uint2*>(a.mir + d) = make_uint2(pack2bf(q.x, q.y), pack2bf(q.z, q.w));
            else if (d + 4 > 0 && d < a.mir_len) {
                const float t[4] = {q.x, q.y, q.z, q.w};
                mirror_store(a, 4 * i, t, 4);
            }
        } else if (d + 4 > 0 && d < a.mir_len) {
            const float t[4] = {q.x, q.y, q.z, q.w};
            mirror_store(a, 4 * i, t, 4);
        }
    };
    if (i0 < n4) {
        opt_four<OPT>(pp, gg, mm, vv, scale, a);
        p4[i0] = pp; v4[i0] = vv;
        if constexpr (OPT == OPT_ADAM) m4[i0] = mm;
        mirror4(i0, pp);
    }
    for (int64_t i = i0 + stride; i < n4; i += stride) {
        pp = p4[i]; gg = g4[i]; vv = v4[i];
        if constexpr (OPT == OPT_ADAM) mm = m4[i];
        opt_four<OPT>(pp, gg, mm, vv, scale, a);
        p4[i] = pp; v4[i] = vv;
        if constexpr (OPT == OPT_ADAM) m4[i] = mm;
        mirror4(i, pp);
    }
    if (blockIdx.x == 0)
        for (int64_t i = n4 * 4 + threadIdx.x; i < a.n; i += 256) {
            float mt = OPT == OPT_ADAM ? a.m[i] : 0.f;
            opt_one<OPT>(a.p[i], a.g[i], mt, a.v[i], scale, a);
            if constexpr (OPT == OPT_ADAM) a.m[i] = mt;
            if (a.mir) mirror_store(a, i, &a.p[i], 1);
        }
}

hipError_t clip_opt_step(int opt, const OptArgs& a, float* stats, float* partial, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    double* part = reinterpret_cast<double*>(partial);
    int64_t blocks = (a.n / 4 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > kAdamBlocks) blocks = kAdamBlocks;
    {
        ProfScope ps(s, [&] { return "grad_sumsq/" + std::to_string(a.n); });
        hipLaunchKernelGGL(sumsq_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, a.n, a.g, part);
    }
    ProfScope ps(s, [&] { return std::string(opt == OPT_ADAM ? "adam/" : "rmsprop/") + std::to_string(a.n); });
    if (opt == OPT_ADAM)
        hipLaunchKernelGGL(opt_kernel<OPT_ADAM>, dim3(unsigned(blocks)), dim3(256), 0, s, a, part, int(blocks), stats);
    else
        hipLaunchKernelGGL(opt_kernel<OPT_RMSPROP>, dim3(unsigned(blocks)), dim3(256), 0, s, a, part, int(blocks),
                           stats);
    return hipGetLastError();
}

}  // namespace cb
