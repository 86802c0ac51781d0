// Device-side helpers shared by the gfx950 kernels: bf16 storage, MFMA wrappers and
// the two precision traits (bf16 matrix-core operands or float32 validation mode).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define CB_DEV __device__ __forceinline__

#include <string>

// Profiling key of a launch: family/precision/shape (see include/cleanba_profile.h).
inline std::string cb_key(const char* family, int prec, const std::string& shape) {
    return std::string(family) + (prec == 0 ? "/bf16/" : "/fp32/") + shape;
}
inline std::string cb_dims(int a, int b) { return std::to_string(a) + "x" + std::to_string(b); }
// Key suffix naming what a conv-family launch moves besides x and y: uint8 frames or a relu
// on load (mode 2 / 1), and the mask / residual operands of its epilogue.
inline std::string cb_flags(int mode, bool mask, bool add) {
    std::string f;
    if (mode == 2) f += "/u8";
    if (mode == 1) f += "/relu";
    if (mask) f += "/mask";
    if (add) f += "/add";
    return f;
}

typedef __bf16 cb_bf16x8 __attribute__((ext_vector_type(8)));
typedef float cb_f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- bf16 storage
// Activations in bf16 mode are stored as raw 16-bit patterns (uint16_t).

CB_DEV float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// float -> bf16, round to nearest even (NaN stays NaN): gfx950 converts natively.
CB_DEV uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }

typedef __bf16 cb_bf16x2 __attribute__((ext_vector_type(2)));
typedef float cb_f32x2 __attribute__((ext_vector_type(2)));
// Two floats -> two bf16 (a in the low half) in one packed conversion.
CB_DEV uint32_t pack2bf(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(cb_f32x2{a, b}, cb_bf16x2));
}

// ---------------------------------------------------------------- precision traits
//
// A 16x16 MFMA tile computes D[i][n] += sum_k A[i][k] * B[k][n]. Lane l supplies A row
// (l % 16) and B column (l % 16) for its KPL consecutive k values starting at KPL*(l/16),
// and receives D rows 4*(l/16) .. +3 of column (l % 16). A and B use the same k
// assignment, so the sum covers each k exactly once.

struct PrecBF16 {
    using T = uint16_t;                  // storage element
    static constexpr int KPL = 8;        // k values per lane per MFMA
    static constexpr int KSTEP = 32;     // k per MFMA (v_mfma_f32_16x16x32_bf16)
    using Frag = uint4;                  // 8 bf16
    static CB_DEV float load(T v) { return bf2f(v); }
    static CB_DEV T store(float f) { return f2bf(f); }
    static CB_DEV cb_f32x4 mma(Frag a, Frag b, cb_f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(cb_bf16x8, a),
                                                       __builtin_bit_cast(cb_bf16x8, b), c, 0, 0, 0);
    }
    static CB_DEV Frag zero() { return make_uint4(0, 0, 0, 0); }
    static CB_DEV Frag lds_frag(const T* p) { return *reinterpret_cast<const uint4*>(p); }
};

struct PrecF32 {
    using T = float;
    static constexpr int KPL = 1;
    static constexpr int KSTEP = 4;      // v_mfma_f32_16x16x4_f32
    using Frag = float;
    static CB_DEV float load(T v) { return v; }
    static CB_DEV T store(float f) { return f; }
    static CB_DEV cb_f32x4 mma(Frag a, Frag b, cb_f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    static CB_DEV Frag zero() { return 0.f; }
    static CB_DEV Frag lds_frag(const T* p) { return *p; }
};

// Store / load 4 consecutive channels of one pixel.
CB_DEV void store4(uint16_t* p, float a, float b, float c, float d) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack2bf(a, b), pack2bf(c, d));
}
CB_DEV void store4(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
CB_DEV void load4(const uint16_t* p, float* o) {
    uint2 v = *reinterpret_cast<const uint2*>(p);
    o[0] = __uint_as_float(v.x << 16);
    o[1] = __uint_as_float(v.x & 0xffff0000u);
    o[2] = __uint_as_float(v.y << 16);
    o[3] = __uint_as_float(v.y & 0xffff0000u);
}
CB_DEV void load4(const float* p, float* o) {
    float4 v = *reinterpret_cast<const float4*>(p);
    o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
}

CB_DEV float relu_f(float x) { return x < 0.f ? 0.f : x; }   // keeps NaN

// ---------------------------------------------------------------- direct HBM -> LDS staging
// buffer_load ... lds writes each lane's 4 or 16 bytes to LDS at a wave-uniform base plus
// lane * size, without passing through registers.

typedef __attribute__((address_space(3))) void lds_t;

// Raw buffer resource over [base, base + bytes); loads at offsets >= bytes return zero.
CB_DEV __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), 0x00020000);
}
constexpr uint32_t kOOB = 0x80000000u;   // past every resource the launcher allows

// floor(q / d) for 0 <= q < 2^22, given inv = 1.0f / d: the relative error of the product
// (at most 2^-23) stays below the distance from (q + 0.5) / d to the nearest integer.
CB_DEV int qdiv(int q, float inv) { return int((float(q) + 0.5f) * inv); }

typedef short cb_s16x2 __attribute__((ext_vector_type(2)));
// relu on two bf16 patterns: every pattern with the sign bit set becomes +0.
CB_DEV uint32_t relu_bf16x2(uint32_t u) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(cb_s16x2, u),
                                                                  cb_s16x2{0, 0}));
}

// One DMA lane: 4 or 16 bytes at byte offset off of the resource -> LDS at lds + lane * size
// (lds is the same for the whole wave).
CB_DEV void dma4_to_lds(__amdgpu_buffer_rsrc_t r, unsigned char* lds, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_t*)(lds), 4, off, 0, 0, 0);
}
CB_DEV void dma16_to_lds(__amdgpu_buffer_rsrc_t r, unsigned char* lds, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_t*)(lds), 16, off, 0, 0, 0);
}

// Workgroup barrier that waits for this wave's LDS operations only: buffer -> LDS loads
// staging a later tile (and global stores) stay in flight across it.
CB_DEV void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Order-preserving 16-bit keys of two packed bf16 values: as unsigned integers the keys
// compare like the values (-0 sorts just below +0; NaNs sort beyond the infinities).
// A negative half is complemented, a positive one has its sign bit set; the sign masks come
// from one packed 16-bit arithmetic shift.
CB_DEV uint32_t sign_mask16x2(uint32_t u) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(cb_s16x2, u) >> cb_s16x2{15, 15});
}
CB_DEV uint32_t bf16x2_key(uint32_t u) { return u ^ (sign_mask16x2(u) | 0x80008000u); }
CB_DEV uint32_t bf16x2_unkey(uint32_t k) { return k ^ (~sign_mask16x2(k) | 0x80008000u); }

// Max-pool backward gathers. ka holds the argmax cells (0..8) of four channels, one per
// byte; d their bf16 gradients (channels 0, 1 in d.x, 2, 3 in d.y). arg_pick<T> keeps the
// gradients of the channels whose cell is T and makes the others +0. arg_sel gives byte
// selectors that name each channel's cell twice ([k0 k0 k1 k1], [k2 k2 k3 k3]): v_perm with
// such a selector looks up each cell in an 8-byte table (0xff at byte T) and widens the
// result to the channel's 16 bits. Cell 8 selects v_perm's sign-of-byte-1 entry, which is
// zero in every table but T = 1's; T = 1 therefore looks up cell ^ 1 in T = 0's table (cell
// 8 then selects the zero sign of byte 3), and T = 8, the only cell with bit 3 set, widens
// that bit with the sign-byte selectors.
CB_DEV uint32_t arg_sel01(uint32_t ka) { return __builtin_amdgcn_perm(0u, ka, 0x01010000u); }
CB_DEV uint32_t arg_sel23(uint32_t ka) { return __builtin_amdgcn_perm(0u, ka, 0x03030202u); }
template <int T>
CB_DEV uint2 arg_pick(uint2 d, uint32_t ka, uint32_t s01, uint32_t s23) {
    static_assert(T >= 0 && T <= 8, "a 3x3 window has cells 0..8");
    uint32_t m01, m23;
    if constexpr (T == 8) {
        const uint32_t a = ka << 4, b = ka << 12;   // bit 3 of cells 1, 3 at bits 15, 31 of a; 0, 2 of b
        m01 = __builtin_amdgcn_perm(b, a, 0x08080a0au);
        m23 = __builtin_amdgcn_perm(b, a, 0x09090b0bu);
    } else if constexpr (T == 1) {
        const uint32_t kb = ka ^ 0x01010101u;
        m01 = __builtin_amdgcn_perm(0u, 0xffu, arg_sel01(kb));
        m23 = __builtin_amdgcn_perm(0u, 0xffu, arg_sel23(kb));
    } else {
        constexpr uint32_t lo = T < 4 ? 0xffu << (8 * T) : 0u, hi = T < 4 ? 0u : 0xffu << (8 * (T - 4));
        m01 = __builtin_amdgcn_perm(hi, lo, s01);
        m23 = __builtin_amdgcn_perm(hi, lo, s23);
    }
    return make_uint2(d.x & m01, d.y & m23);
}
CB_DEV float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
CB_DEV float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

typedef short cb_s16x4 __attribute__((ext_vector_type(4)));
// LDS transpose read of 16-bit data (ds_read_b64_tr_b16). Every lane addresses an 8-byte
// chunk (4 elements); within each group of 16 lanes, lane i receives as its element j
// element (i % 4) of the chunk addressed by lane 4*j + i/4 of the group.
CB_DEV uint2 lds_read_tr16(const unsigned char* p) {
    typedef __attribute__((address_space(3))) cb_s16x4 lds_s16x4;
    return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p)));
}

CB_DEV uint2 u8x4_to_bf16(uint32_t u) {
    return make_uint2(pack2bf(float(u & 0xffu), float((u >> 8) & 0xffu)),
                      pack2bf(float((u >> 16) & 0xffu), float(u >> 24)));
}


// Block-wide reduction of a double over 256 threads (fixed order -> deterministic).
template <int NT>
CB_DEV double block_sum(double v, double* sh) {
    const int t = threadIdx.x;
    sh[t] = v;
    __syncthreads();
#pragma unroll
    for (int s = NT / 2; s > 0; s >>= 1) {
        if (t < s) sh[t] += sh[t + s];
        __syncthreads();
    }
    double r = sh[0];
    __syncthreads();
    return r;
}

// Entry-wise sum of `nparts` float32 partial vectors (stride `pstride` floats, a multiple of
// 4, 16-byte aligned) in a fixed order: a 1024-thread block covers 64 entries as 16 float4
// lanes x 64 slices; slice s adds the partials s, s + 64, s + 128, ... in turn (eight loads
// in flight), then a fixed pairwise tree over the slices. emit(e, v) gets entries e..e+3.
template <class F>
CB_DEV void sum_partials_x4(const float* __restrict__ partial, int nparts, int pstride, F&& emit) {
    __shared__ float4 sh[64][17];
    const int q = threadIdx.x & 15, sl = threadIdx.x >> 4;
    const int e = blockIdx.x * 64 + 4 * q;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (e < pstride) {
        const float4* p = reinterpret_cast<const float4*>(partial + e);
        const int64_t st = pstride / 4;
        int k = sl;
        for (; k + 7 * 64 < nparts; k += 8 * 64) {
            float4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = p[int64_t(k + 64 * u) * st];
#pragma unroll
            for (int u = 0; u < 8; ++u) { s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w; }
        }
        for (; k < nparts; k += 64) {
            const float4 v = p[int64_t(k) * st];
            s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
    }
    sh[sl][q] = s;
    __syncthreads();
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) {
        if (sl < w) {
            const float4 o = sh[sl + w][q];
            float4& m = sh[sl][q];
            m.x += o.x; m.y += o.y; m.z += o.z; m.w += o.w;
        }
        __syncthreads();
    }
    if (sl == 0 && e < pstride) emit(e, sh[0][q]);
}

// A pending weight-gradient reduce (PendingReduce, see kernels.h) done by the first work of a
// kernel with NT threads: blocks of 64 entries (16 float4 lanes x NT/16 slices, each slice
// adding the partials s, s + NT/16, ... in turn, then a fixed pairwise tree) spread over the
// grid, scattered to HWIO weights (times scale) and the bias. `lds` holds NT/16 x 17 float4.
// Ends with a barrier, so the caller may reuse the LDS.
template <int NT, class R>
CB_DEV void pending_reduce(const R& r, unsigned char* lds) {
    constexpr int SL = NT / 16;
    float4* sh = reinterpret_cast<float4*>(lds);
    const int q = threadIdx.x & 15, sl = threadIdx.x >> 4;
    const int NB = r.u8 ? 3 : 9 * r.cin / 16, NBB = NB + 1, cb16 = r.cin / 16 > 0 ? r.cin / 16 : 1;
    const int nrb = r.pstride / 64;
    const int64_t st = r.pstride / 4;
    for (int rb = blockIdx.x; rb < nrb; rb += gridDim.x) {
        const int e = rb * 64 + 4 * q;
        const float4* p = reinterpret_cast<const float4*>(r.partial + e);
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        int k = sl;
        for (; k + 7 * SL < r.nparts; k += 8 * SL) {
            float4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = p[int64_t(k + SL * u) * st];
#pragma unroll
            for (int u = 0; u < 8; ++u) { s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w; }
        }
        for (; k < r.nparts; k += SL) {
            const float4 v = p[int64_t(k) * st];
            s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
        sh[sl * 17 + q] = s;
        __syncthreads();
#pragma unroll
        for (int w = SL / 2; w >= 1; w >>= 1) {
            if (sl < w) {
                const float4 o = sh[(sl + w) * 17 + q];
                float4& m = sh[sl * 17 + q];
                m.x += o.x; m.y += o.y; m.z += o.z; m.w += o.w;
            }
            __syncthreads();
        }
        if (sl == 0) {
            const float4 v = sh[q];
            const float tv[4] = {v.x, v.y, v.z, v.w};
            const int tile = e >> 8, row = (e >> 4) & 15;
            const int mt = tile / NBB, nb = tile - mt * NBB, co = mt * 16 + row;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int col = (e & 15) + u;
                if (nb == NB) {
                    if (col == 0) r.db[co] = tv[u];
                } else {
                    const int tap = r.u8 ? nb * 4 + col / 4 : nb / cb16;
                    const int ci = r.u8 ? col % 4 : (nb % cb16) * 16 + col;
                    if (tap < 9) r.dw[(tap * r.cin + ci) * r.cout + co] = tv[u] * r.scale;
                }
            }
        }
        __syncthreads();
    }
}
