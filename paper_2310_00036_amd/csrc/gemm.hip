// Dense-layer and head GEMMs on gfx950 MFMA: D[m][n] = sum_k A(m,k) B(k,n), written to
// out[n*ld + m] (m contiguous, so a lane's 4 accumulator rows are 4 adjacent outputs).
//
// A and B are read from global memory in either orientation (k-contiguous or
// m/n-contiguous), converted to the compute type and staged k-contiguous in LDS; float32
// weights are rounded to bf16 on the way in when the compute type is bf16. A 64x64 output
// tile per workgroup, 4 waves of 32x32. Split-K writes float32 partials that a second
// kernel sums in a fixed order before applying the epilogue (bias, ReLU, mask, store).
#include "common.h"
#include "kernels.h"

#include <algorithm>

#include <type_traits>

namespace cb {

template <class P>
struct GemmTile {
    static constexpr int BM = 64, BN = 64;
    static constexpr int BK = P::KSTEP * (sizeof(typename P::T) == 2 ? 2 : 4);
    static constexpr int LDK = BK + (sizeof(typename P::T) == 2 ? 8 : 1);
};

template <class P>
CB_DEV float ld_elem(const void* base, int is_f32, int64_t idx) {
    if (is_f32) return static_cast<const float*>(base)[idx];
    return P::load(static_cast<const typename P::T*>(base)[idx]);
}

template <class P>
CB_DEV void gemm_epilogue(const GemmArgs& a, int m, int n, float v) {
    using T = typename P::T;
    if (m >= a.M || n >= a.N) return;
    const bool hi = m >= a.msplit;
    const float* bias = hi ? a.bias2 : a.bias1;
    v = v * a.alpha + (bias ? bias[hi ? m - a.msplit : m] : 0.f);
    if (a.relu) v = relu_f(v);
    if (a.mask && !(P::load(static_cast<const T*>(a.mask)[int64_t(n) * a.ldmask + m]) > 0.f)) v = 0.f;
    if (!hi) {
        const int64_t o = int64_t(n) * a.ld1 + m;
        if (a.out1_f32) static_cast<float*>(a.out1)[o] = v;
        else static_cast<T*>(a.out1)[o] = P::store(v);
    } else {
        const int64_t o = int64_t(n) * a.ld2 + (m - a.msplit);
        if (a.out2_f32) static_cast<float*>(a.out2)[o] = v;
        else static_cast<T*>(a.out2)[o] = P::store(v);
    }
}

// Four consecutive rows m .. m+3 of output column n at once (bf16 storage): one 8-byte
// mask load and one 8-byte store. Falls back to the per-element epilogue where the group
// straddles the row split or the edge, or the output is not 8-byte addressable that way.
CB_DEV bool gemm_epilogue4_ok(const GemmArgs& a) {
    const bool mask_ok = !a.mask || ((a.ldmask & 3) == 0 && (reinterpret_cast<uintptr_t>(a.mask) & 7) == 0);
    return !a.out1_f32 && (a.ld1 & 3) == 0 && (reinterpret_cast<uintptr_t>(a.out1) & 7) == 0 && mask_ok;
}
CB_DEV void gemm_epilogue4_bf16(const GemmArgs& a, bool vec_ok, int m, int n, cb_f32x4 v) {
    if (!vec_ok || n >= a.N || m + 4 > a.M || m + 4 > a.msplit) {
#pragma unroll
        for (int r = 0; r < 4; ++r) gemm_epilogue<PrecBF16>(a, m + r, n, v[r]);
        return;
    }
    float o[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        o[r] = v[r] * a.alpha + (a.bias1 ? a.bias1[m + r] : 0.f);
        if (a.relu) o[r] = relu_f(o[r]);
    }
    if (a.mask) {
        float mk[4];
        load4(static_cast<const uint16_t*>(a.mask) + int64_t(n) * a.ldmask + m, mk);
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = mk[r] > 0.f ? o[r] : 0.f;
    }
    store4(static_cast<uint16_t*>(a.out1) + int64_t(n) * a.ld1 + m, o[0], o[1], o[2], o[3]);
}

// Loads one BM(or BN) x BK tile of an operand into LDS as tile[row][k] (k contiguous).
// src(row, k) = base[row*ld + k] (kcontig) or base[k*ld + row]; 16-byte vector loads along
// the contiguous dimension when `vec` (aligned leading dimension and base), with a scalar
// fallback for ragged edges.
template <class P, int ROWS, int BK, int LDK>
CB_DEV void gemm_load_tile(typename P::T* tile, const void* base, int is_f32, int kcontig, int64_t ld,
                           int vec, int relu, int row0, int nrows, int k0, int kend, int tid) {
    using T = typename P::T;
    const int V = is_f32 ? 4 : (sizeof(T) == 2 ? 8 : 4);     // elements per 16 bytes
    if (kcontig) {
        const int nch = ROWS * (BK / V);
        for (int e = tid; e < nch; e += 256) {
            const int rr = e / (BK / V), kc = (e % (BK / V)) * V;
            const int row = row0 + rr, k = k0 + kc;
            float v[8];
            if (vec && row < nrows && k + V <= kend) {
                const int64_t off = int64_t(row) * ld + k;
                if (is_f32) {
                    const float4 f = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
                    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
                } else if (sizeof(T) == 2) {
                    const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + off);
                    const uint32_t* uu = reinterpret_cast<const uint32_t*>(&u);
                    for (int j = 0; j < 4; ++j) {
                        v[2 * j] = __uint_as_float(uu[j] << 16);
                        v[2 * j + 1] = __uint_as_float(uu[j] & 0xffff0000u);
                    }
                } else {
                    const float4 f = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
                    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
                }
            } else {
                for (int j = 0; j < V; ++j) {
                    v[j] = 0.f;
                    if (row < nrows && k + j < kend) {
                        const int64_t off = int64_t(row) * ld + k + j;
                        v[j] = is_f32 ? static_cast<const float*>(base)[off] : P::load(static_cast<const T*>(base)[off]);
                    }
                }
            }
            for (int j = 0; j < V; ++j) tile[rr * LDK + kc + j] = P::store(relu ? relu_f(v[j]) : v[j]);
        }
    } else {
        const int nch = BK * (ROWS / V);
        for (int e = tid; e < nch; e += 256) {
            const int kk = e / (ROWS / V), rc = (e % (ROWS / V)) * V;
            const int row = row0 + rc, k = k0 + kk;
            float v[8];
            if (vec && k < kend && row + V <= nrows) {
                const int64_t off = int64_t(k) * ld + row;
                if (is_f32 || sizeof(T) == 4) {
                    const float4 f = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
                    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
                } else {
                    const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + off);
                    const uint32_t* uu = reinterpret_cast<const uint32_t*>(&u);
                    for (int j = 0; j < 4; ++j) {
                        v[2 * j] = __uint_as_float(uu[j] << 16);
                        v[2 * j + 1] = __uint_as_float(uu[j] & 0xffff0000u);
                    }
                }
            } else {
                for (int j = 0; j < V; ++j) {
                    v[j] = 0.f;
                    if (k < kend && row + j < nrows) {
                        const int64_t off = int64_t(k) * ld + row + j;
                        v[j] = is_f32 ? static_cast<const float*>(base)[off] : P::load(static_cast<const T*>(base)[off]);
                    }
                }
            }
            for (int j = 0; j < V; ++j) tile[(rc + j) * LDK + kk] = P::store(relu ? relu_f(v[j]) : v[j]);
        }
    }
}

template <class P>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a, int kchunk, int avec, int bvec) {
    using T = typename P::T;
    using G = GemmTile<P>;
    using Frag = typename P::Frag;
    constexpr int BM = G::BM, BN = G::BN, BK = G::BK, LDK = G::LDK;
    __shared__ __align__(16) T As[BM * LDK];
    __shared__ __align__(16) T Bs[BN * LDK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
    const int k_begin = blockIdx.z * kchunk;
    const int k_end = min(a.K, k_begin + kchunk);

    cb_f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = cb_f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = k_begin; k0 < k_end; k0 += BK) {
        __syncthreads();
        gemm_load_tile<P, BM, BK, LDK>(As, a.a, a.a_f32, a.a_kcontig, a.lda, avec, 0, m0, a.M, k0, k_end, tid);
        gemm_load_tile<P, BN, BK, LDK>(Bs, a.b, a.b_f32, a.b_kcontig, a.ldb, bvec, a.b_relu, n0, a.N, k0, k_end, tid);
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < BK; ks += P::KSTEP) {
            Frag af[2], bf[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) af[i] = P::lds_frag(As + (wm * 32 + i * 16 + r16) * LDK + ks + g * P::KPL);
#pragma unroll
            for (int j = 0; j < 2; ++j) bf[j] = P::lds_frag(Bs + (wn * 32 + j * 16 + r16) * LDK + ks + g * P::KPL);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = P::mma(af[i], bf[j], acc[i][j]);
        }
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm * 32 + i * 16 + 4 * g + r;
                const int n = n0 + wn * 32 + j * 16 + r16;
                if (gridDim.z == 1) {
                    gemm_epilogue<P>(a, m, n, acc[i][j][r]);
                } else if (m < a.M && n < a.N) {
                    a.partial[(int64_t(blockIdx.z) * a.N + n) * a.M + m] = acc[i][j][r];
                }
            }
}

// ------------------------------------------------------------------ bf16 operands: DMA path
//
// When both operands are bf16 in memory (the dense layer, its weights cast once per pass), the
// tiles are staged straight from HBM into LDS with buffer->LDS loads in the layout they have
// in memory, double-buffered: the next k-block's loads are issued before this block's MFMAs.
// A k-contiguous tile is [128 rows][64 k] with 144-byte rows and is read as 16-byte
// fragments; a rows-contiguous tile is [64 k][128 rows] with 288-byte rows and is read with
// the LDS transpose read, which hands each lane 4 consecutive k of its row. The padding (one
// 16-byte slot per row, two for the k-major tile) keeps the 16-lane reads on distinct banks
// and is filled by out-of-range (zero) loads, as are the tails past M, N and K.
// 128x128 output tile per workgroup, 4 waves of 64x64 (4x4 MFMA 16x16x32 tiles).

namespace {
constexpr int kGB = 128, kGK = 64;
constexpr int kPK = 144, kPM = 288;            // row pitches (bytes) of the two tile layouts
constexpr int kGTile = kGB * kPK;              // bytes per operand tile (== kGK * kPM)
constexpr int kGStage = 2 * kGTile;            // A and B
static_assert(kGK * kPM == kGTile, "both layouts fill the same tile");
}  // namespace

// DMA of one operand tile: rows [r0, r0+128) of `nrows`, k [k0, k0+64) of `kend`. A lane's
// slots map to the same row and column of every k-block, so their offsets are formed once
// per workgroup (rows past `nrows` and padding slots: kOOB); a k-block adds k0 (k-contiguous)
// or k0 rows, and a slot past `kend` reads zero.
template <int KC>
struct GemmStage {
    static constexpr int SPR = KC ? kPK / 16 : kPM / 16;   // slots per LDS row
    static constexpr int DATA = KC ? 8 : 16;               // data slots per row
    static constexpr int NS = (KC ? kGB : kGK) * SPR;      // slots per tile (multiple of 64)
    static constexpr int NB = (NS / 64 + 3) / 4;           // DMA blocks per wave (at most)
    static_assert(NS % 64 == 0, "whole DMA blocks");
    uint32_t base[NB];   // byte offset at k0 = 0, or kOOB
    int kx[NB];          // the slot's k (k-contiguous: column, else row) within the block
    CB_DEV GemmStage(int ld, int r0, int nrows, int wave, int lane) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int b = wave + 4 * i;
            const int j = b * 64 + lane;
            const int row = j / SPR, c = j - row * SPR;
            bool ok = b < NS / 64 && c < DATA;
            if (KC) {
                ok = ok && r0 + row < nrows;
                base[i] = ok ? (uint32_t(r0 + row) * uint32_t(ld) + uint32_t(c * 8)) * 2u : kOOB;
                kx[i] = c * 8;
            } else {
                ok = ok && r0 + c * 8 < nrows;
                base[i] = ok ? (uint32_t(row) * uint32_t(ld) + uint32_t(r0 + c * 8)) * 2u : kOOB;
                kx[i] = row;
            }
        }
    }
    CB_DEV void issue(__amdgpu_buffer_rsrc_t rs, unsigned char* __restrict__ dst, int ld, int k0, int kend, int wave) const {
        const uint32_t kadd = KC ? uint32_t(k0) * 2u : uint32_t(k0) * uint32_t(ld) * 2u;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int b = wave + 4 * i;
            if (b < NS / 64) {
                const uint32_t off = (base[i] != kOOB && k0 + kx[i] < kend) ? base[i] + kadd : kOOB;
                dma16_to_lds(rs, dst + b * 1024, off);
            }
        }
    }
};

// Fragment of 8 consecutive k (k-step ks, lane group g) of tile row `row`.
template <int KC>
CB_DEV uint4 gemm_frag(const unsigned char* __restrict__ t, int row, int ks, int g, int lane) {
    if constexpr (KC) {
        return *reinterpret_cast<const uint4*>(t + row * kPK + ks * 64 + g * 16);
    } else {
        // transpose read: lane 4j+m of the 16-lane group addresses k = base + j, rows 4m..4m+3
        const int r16 = lane & 15, j = r16 >> 2, m = r16 & 3;
        const int rb = row - r16 + 4 * m;   // first row of this lane's 4-row chunk
        const uint2 lo = lds_read_tr16(t + (ks * 32 + g * 8 + j) * kPM + rb * 2);
        const uint2 hi = lds_read_tr16(t + (ks * 32 + g * 8 + 4 + j) * kPM + rb * 2);
        return make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
}

// One k-block: issue the next block's loads into `nxt`, then the MFMAs on `cur`. Both buffers
// are restrict parameters of the one call, so the compiler knows the loads in flight do not
// write what the MFMAs read and does not wait for them.
template <int AKC, int BKC, int BRELU>
CB_DEV void gemm_block(const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt, bool more,
                       __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb, const GemmStage<AKC>& sa,
                       const GemmStage<BKC>& sb, const GemmArgs& a, int k1, int k_end, int wave, int lane,
                       cb_f32x4 (&acc)[4][4]) {
    if (more) {
        sa.issue(ra, nxt, int(a.lda), k1, k_end, wave);
        sb.issue(rb, nxt + kGTile, int(a.ldb), k1, k_end, wave);
    }
    const int g = (lane >> 4) & 3, r16 = lane & 15;
    const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        uint4 af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = gemm_frag<AKC>(cur, wm * 64 + i * 16 + r16, ks, g, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            bf[j] = gemm_frag<BKC>(cur + kGTile, wn * 64 + j * 16 + r16, ks, g, lane);
            if constexpr (BRELU) {
                bf[j].x = relu_bf16x2(bf[j].x); bf[j].y = relu_bf16x2(bf[j].y);
                bf[j].z = relu_bf16x2(bf[j].z); bf[j].w = relu_bf16x2(bf[j].w);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = PrecBF16::mma(af[i], bf[j], acc[i][j]);
    }
}

template <int AKC, int BKC, int BRELU>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a, int kchunk) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int wm = wave >> 1, wn = wave & 1;
    // Workgroups go to the XCDs in turn (linear id mod 8), each XCD with its own L2. With split
    // k, a run of consecutive linear ids is given to one XCD, and within it the output tiles
    // advance along n first, so an XCD's workgroups share a few A tiles and the B tiles of one
    // k-split (dense forward 21.6 -> 19.0 us, weight gradient 24.7 -> 22.5 us at 2048 frames;
    // without split k this order measured no better).
    int tm = int(blockIdx.x), tn = int(blockIdx.y), tz = int(blockIdx.z);
    const int nwg = int(gridDim.x * gridDim.y * gridDim.z);
    if (gridDim.z > 1 && (nwg & 7) == 0) {
        const int bid = int(blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z));
        const int b2 = (bid & 7) * (nwg >> 3) + (bid >> 3);
        tn = b2 % int(gridDim.y);
        tm = (b2 / int(gridDim.y)) % int(gridDim.x);
        tz = b2 / int(gridDim.y * gridDim.x);
    }
    const int m0 = tm * kGB, n0 = tn * kGB;
    const int k_begin = tz * kchunk;
    const int k_end = min(a.K, k_begin + kchunk);
    const auto ra = buf_rsrc(a.a, uint32_t((AKC ? int64_t(a.M) : int64_t(a.K)) * a.lda * 2));
    const auto rb = buf_rsrc(a.b, uint32_t((BKC ? int64_t(a.N) : int64_t(a.K)) * a.ldb * 2));

    cb_f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = cb_f32x4{0.f, 0.f, 0.f, 0.f};

    const GemmStage<AKC> sa(int(a.lda), m0, a.M, wave, lane);
    const GemmStage<BKC> sb(int(a.ldb), n0, a.N, wave, lane);
    sa.issue(ra, smem, int(a.lda), k_begin, k_end, wave);
    sb.issue(rb, smem + kGTile, int(a.ldb), k_begin, k_end, wave);
    int it = 0;
    for (int k0 = k_begin; k0 < k_end; k0 += kGK, ++it) {
        __builtin_amdgcn_s_waitcnt(0);   // this block's loads (this wave's) are in LDS
        __syncthreads();                 // all waves' loads in; the other buffer is free
        unsigned char* cur = smem + (it & 1) * kGStage;
        unsigned char* nxt = smem + ((it + 1) & 1) * kGStage;
        gemm_block<AKC, BKC, BRELU>(cur, nxt, k0 + kGK < k_end, ra, rb, sa, sb, a, k0 + kGK, k_end, wave, lane, acc);
    }

    const bool vec_ok = gemm_epilogue4_ok(a);
    if (gridDim.z == 1 && vec_ok && m0 + kGB <= a.M && m0 + kGB <= a.msplit && n0 + kGB <= a.N) {
        // whole tile inside the output: every bias and mask load is issued before the first
        // use, so the epilogue waits for one load latency rather than sixteen
        uint2 mk[4][4];
        float bs[4][4];
        const uint16_t* mask = static_cast<const uint16_t*>(a.mask);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int mb = m0 + wm * 64 + i * 16 + 4 * g;
#pragma unroll
            for (int r = 0; r < 4; ++r) bs[i][r] = a.bias1 ? a.bias1[mb + r] : 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = n0 + wn * 64 + j * 16 + r16;
                mk[i][j] = mask ? *reinterpret_cast<const uint2*>(mask + int64_t(n) * a.ldmask + mb) : make_uint2(0u, 0u);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int mb = m0 + wm * 64 + i * 16 + 4 * g;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = n0 + wn * 64 + j * 16 + r16;
                float o[4];
                const uint32_t mw[4] = {mk[i][j].x << 16, mk[i][j].x & 0xffff0000u, mk[i][j].y << 16,
                                        mk[i][j].y & 0xffff0000u};
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    o[r] = acc[i][j][r] * a.alpha + bs[i][r];
                    if (a.relu) o[r] = relu_f(o[r]);
                    if (mask && !(__uint_as_float(mw[r]) > 0.f)) o[r] = 0.f;
                }
                store4(static_cast<uint16_t*>(a.out1) + int64_t(n) * a.ld1 + mb, o[0], o[1], o[2], o[3]);
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int mb = m0 + wm * 64 + i * 16 + 4 * g;
            const int n = n0 + wn * 64 + j * 16 + r16;
            if (gridDim.z == 1) {
                gemm_epilogue4_bf16(a, vec_ok, mb, n, acc[i][j]);
            } else if (n < a.N && mb < a.M) {
                float* pp = a.partial + (int64_t(tz) * a.N + n) * a.M + mb;
                if (mb + 4 <= a.M && (a.M & 3) == 0) {
                    *reinterpret_cast<float4*>(pp) = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) if (mb + r < a.M) pp[r] = acc[i][j][r];
                }
            }
        }
}

// Sums the split-K partials in split order; grid (ceil(M / 256), min(N, 65535)).
template <class P>
__global__ __launch_bounds__(256) void gemm_finish_kernel(GemmArgs a, int splits) {
    const int m = blockIdx.x * 256 + threadIdx.x;
    if (m >= a.M) return;
    const int64_t total = int64_t(a.M) * a.N;
    for (int n = blockIdx.y; n < a.N; n += gridDim.y) {
        const float* p = a.partial + int64_t(n) * a.M + m;
        float s = 0.f;
        int z = 0;
        for (; z + 8 <= splits; z += 8) {   // eight loads in flight, added in split order
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = p[(z + u) * total];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; z < splits; ++z) s += p[z * total];
        gemm_epilogue<P>(a, m, n, s);
    }
}

// Split-K so the grid covers the chip (about two workgroups per CU), never below 256 k per
// split and never above the caller's partial-buffer allowance `max_splits`.
static int auto_splits(int M, int N, int K, int max_splits, int bm, int bn) {
    const int tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    int s = (512 + tiles - 1) / tiles;
    if (s > max_splits) s = max_splits;
    while (s > 1 && K / s < 256) --s;
    return s < 1 ? 1 : s;
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

constexpr int kMaxSplits = 8;

size_t gemm_partial_floats(int M, int N, int K) {
    const int sp = auto_splits(M, N, K, kMaxSplits, 64, 64);
    // the bf16 DMA path: about two 128x128 workgroups per CU, at least 256 k per split
    const int tiles = ((M + 127) / 128) * ((N + 127) / 128);
    int sd = (512 + tiles - 1) / tiles;
    while (sd > 1 && K / sd < 256) --sd;
    const int spm = sp > sd ? sp : sd;
    return spm > 1 ? size_t(M) * N * spm : 0;
}

// ------------------------------------------------------------------ float32 -> bf16
__global__ void cast_bf16_kernel(const float* __restrict__ x, uint16_t* __restrict__ y, int64_t n) {
    const int64_t i = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 2;
    if (i + 1 < n) *reinterpret_cast<uint32_t*>(y + i) = pack2bf(x[i], x[i + 1]);
    else if (i < n) y[i] = f2bf(x[i]);
}

hipError_t cast_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "cast_bf16/" + std::to_string(n); });
    hipLaunchKernelGGL(cast_bf16_kernel, dim3(unsigned((n + 511) / 512)), dim3(256), 0, s, x, y, n);
    return hipGetLastError();
}

// Whether the DMA path takes this GEMM: bf16 operands with 16-byte aligned rows, multiples of
// 8 where a tile row is cut along the contiguous dimension, tiles worth filling, operands
// addressable with 32-bit offsets.
static bool gemm_dma_ok(const GemmArgs& a) {
    auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    if (a.a_f32 || a.b_f32 || a.M < 64 || a.N < 64 || a.K % 8) return false;
    if (!al(a.a) || !al(a.b) || a.lda % 8 || a.ldb % 8) return false;
    if (!a.a_kcontig && a.M % 8) return false;
    if (!a.b_kcontig && a.N % 8) return false;
    const int64_t abytes = (a.a_kcontig ? int64_t(a.M) : int64_t(a.K)) * a.lda * 2;
    const int64_t bbytes = (a.b_kcontig ? int64_t(a.N) : int64_t(a.K)) * a.ldb * 2;
    return abytes < (int64_t(1) << 31) && bbytes < (int64_t(1) << 31);
}

static hipError_t gemm_dma_launch(const GemmArgs& a, hipStream_t s) {
    const int tiles = ((a.M + kGB - 1) / kGB) * ((a.N + kGB - 1) / kGB);
    int splits = a.partial ? (512 + tiles - 1) / tiles : 1;   // about two workgroups per CU
    while (splits > 1 && a.K / splits < 256) --splits;
    while (splits > 1 && size_t(a.M) * a.N * splits > a.partial_floats) --splits;
    if (splits < 1) splits = 1;
    int kchunk = (a.K + splits - 1) / splits;
    kchunk = (kchunk + kGK - 1) / kGK * kGK;
    const int z = (a.K + kchunk - 1) / kchunk > 0 ? (a.K + kchunk - 1) / kchunk : 1;
    const dim3 grid((a.M + kGB - 1) / kGB, (a.N + kGB - 1) / kGB, z);
    const size_t lds = 2 * kGStage;
    const std::string shape = cb_dims(a.M, a.N) + "x" + std::to_string(a.K);
    {
        ProfScope ps(s, [&] { return cb_key("gemm", 0, shape); });
#define CB_GB(AK, BK, BR) \
        if (a.a_kcontig == AK && a.b_kcontig == BK && (a.b_relu != 0) == BR) \
            hipLaunchKernelGGL((gemm_bf16_kernel<AK, BK, BR>), grid, dim3(256), lds, s, a, kchunk);
        CB_GB(1, 1, 0) CB_GB(1, 0, 0) CB_GB(0, 1, 0) CB_GB(0, 0, 0)
        CB_GB(1, 1, 1) CB_GB(1, 0, 1) CB_GB(0, 1, 1) CB_GB(0, 0, 1)
#undef CB_GB
    }
    if (z > 1) {
        ProfScope ps(s, [&] { return cb_key("gemm_finish", 0, shape); });
        hipLaunchKernelGGL(gemm_finish_kernel<PrecBF16>, dim3(unsigned((a.M + 255) / 256), unsigned(std::min(a.N, 65535))),
                           dim3(256), 0, s, a, z);
    }
    return hipGetLastError();
}

template <class P>
static hipError_t gemm_launch(const GemmArgs& a, hipStream_t s) {
    using G = GemmTile<P>;
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    if (std::is_same_v<P, PrecBF16> && gemm_dma_ok(a)) return gemm_dma_launch(a, s);
    int splits = a.partial ? auto_splits(a.M, a.N, a.K, kMaxSplits, G::BM, G::BN) : 1;
    while (splits > 1 && size_t(a.M) * a.N * splits > a.partial_floats) --splits;
    int kchunk = (a.K + splits - 1) / splits;
    kchunk = (kchunk + G::BK - 1) / G::BK * G::BK;
    if (kchunk <= 0) kchunk = G::BK;
    const int z = (a.K + kchunk - 1) / kchunk > 0 ? (a.K + kchunk - 1) / kchunk : 1;
    const int va = (a.a_f32 || sizeof(typename P::T) == 4) ? 4 : 8;
    const int vb = (a.b_f32 || sizeof(typename P::T) == 4) ? 4 : 8;
    const int avec = aligned16(a.a) && a.lda % va == 0;
    const int bvec = aligned16(a.b) && a.ldb % vb == 0;
    dim3 grid((a.M + G::BM - 1) / G::BM, (a.N + G::BN - 1) / G::BN, z);
    const int pr = sizeof(typename P::T) == 2 ? 0 : 1;
    const std::string shape = cb_dims(a.M, a.N) + "x" + std::to_string(a.K);
    {
        ProfScope ps(s, [&] { return cb_key("gemm", pr, shape); });
        hipLaunchKernelGGL(gemm_kernel<P>, grid, dim3(256), 0, s, a, kchunk, avec, bvec);
    }
    if (z > 1) {
        ProfScope ps(s, [&] { return cb_key("gemm_finish", pr, shape); });
        hipLaunchKernelGGL(gemm_finish_kernel<P>, dim3(unsigned((a.M + 255) / 256), unsigned(std::min(a.N, 65535))), dim3(256),
                           0, s, a, z);
    }
    return hipGetLastError();
}

hipError_t gemm(int prec, const GemmArgs& a, hipStream_t s) {
    return prec == BF16 ? gemm_launch<PrecBF16>(a, s) : gemm_launch<PrecF32>(a, s);
}

}  // namespace cb
