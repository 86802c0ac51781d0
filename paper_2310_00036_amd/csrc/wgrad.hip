// Weight and bias gradient of a 3x3 stride-1 SAME convolution on gfx950 MFMA.
//
//   dW[ky][kx][ci][co] = sum over pixels (h, w) of xpad[h+ky][w+kx][ci] * dy[h][w][co]
//   db[co]             = sum over pixels of dy[h][w][co]
//
// The contraction runs over pixels, so both operands are staged in LDS channel-major
// (pixel index fastest). For a band of TH rows the pixel index is k' = r*PITCH + c' with
// PITCH = W+2 rounded up to 8. The input window is stored once as xT[ci][k'] (rows r of
// the zero-padded input, r = 0..TH+1). The output gradient is stored as three copies
// shifted by the kernel column kx: gS[kx][co][r*PITCH + c'] = dy[r][c' - kx][co]. Then
//   dW[ky][kx][ci][co] = sum_k' gS[kx][co][k'] * xT[ci][k' + ky*PITCH],
// and every MFMA fragment (8 consecutive k') is an aligned 16-byte LDS read for both
// operands. Output tiles are D[co][(ky, ci)] for each kx.
//
// Each workgroup accumulates over a fixed, interleaved set of (frame, band) chunks and
// writes one float32 partial. A second kernel sums the partials in a fixed order, so the
// result is deterministic (no atomics).
#include "common.h"
#include "kernels.h"

#include <algorithm>
#include <type_traits>

namespace cb {

template <class P, int CIN, int COUT>
struct WgGeom {
    static constexpr int NCOL = 3 * CIN;                 // (ky, ci) columns
    static constexpr int NTN = (NCOL + 15) / 16;         // column tiles
    static constexpr int MT = COUT / 16;
    static constexpr int TILES = 3 * MT * NTN;           // (kx, mt, nt)
    static constexpr int TPW = (TILES + 3) / 4;          // tiles per wave
    static constexpr int PSTRIDE = 3 * COUT * NTN * 16 + COUT;   // floats per partial
};

struct WgRun {
    int TH, nbands, nchunks, PITCH, KLEN, XP, GP;
    int nx, ng;   // load items per chunk: (TH+2)*W*NCI input items, TH*W*NCO gradient items
};

static inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

constexpr int kWgItems = 4;   // load items per thread per operand (register prefetch depth)

// One 16-byte (8 channels; 4 for uint8 frames) load item kept in registers between the
// global load and the LDS store, so the next chunk's loads overlap this chunk's MFMAs.
template <class P, int VEC>
struct WgItem {
    uint4 raw[sizeof(typename P::T) == 4 && VEC == 8 ? 2 : 1];
};

template <class P, int CIN, int COUT, int MODE>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a, WgRun g_) {
    using T = typename P::T;
    using Frag = typename P::Frag;
    using G = WgGeom<P, CIN, COUT>;
    constexpr int KPL = P::KPL, KSTEP = P::KSTEP;
    constexpr int VEC = MODE == IN_U8 ? 4 : 8;        // channels per input load item
    constexpr int NCI = CIN / VEC, NCO = COUT / 8;
    constexpr bool BF = sizeof(T) == 2;

    extern __shared__ __align__(16) unsigned char smem[];
    T* xT = reinterpret_cast<T*>(smem);               // [CIN][XP]
    T* gS = xT + CIN * g_.XP;                          // [3][COUT][GP]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TH = g_.TH, PITCH = g_.PITCH, KLEN = g_.KLEN;
    const int XP = g_.XP, GP = g_.GP;

    // Zero both tiles once: cells outside the image (halo columns, rows past the image,
    // k padding) are never written again, so they stay zero for every chunk.
    {
        const int words = (CIN * XP + 3 * COUT * GP) * int(sizeof(T)) / 4;
        uint32_t* z = reinterpret_cast<uint32_t*>(smem);
        for (int i = tid; i < words; i += 256) z[i] = 0u;
    }

    // Per-tile fragment bases (fixed for the whole kernel).
    int a_off[G::TPW], b_off[G::TPW];
    bool b_ok[G::TPW];
#pragma unroll
    for (int j = 0; j < G::TPW; ++j) {
        const int t = wave + 4 * j;
        const int tt = t < G::TILES ? t : 0;
        const int kx = tt / (G::MT * G::NTN), mt = (tt / G::NTN) % G::MT, nt = tt % G::NTN;
        a_off[j] = (kx * COUT + mt * 16 + r16) * GP + g * KPL;
        const int col = nt * 16 + r16;
        b_ok[j] = t < G::TILES && col < G::NCOL;
        const int cc = col < G::NCOL ? col : 0;
        b_off[j] = (cc % CIN) * XP + (cc / CIN) * PITCH + g * KPL;
    }
    cb_f32x4 acc[G::TPW];
#pragma unroll
    for (int j = 0; j < G::TPW; ++j) acc[j] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    float bsum[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) bsum[j] = 0.f;

    WgItem<P, VEC> xr[kWgItems];
    WgItem<P, 8> gr[kWgItems];
    const T* dy = static_cast<const T*>(a.dy);

    // Global -> registers for chunk ch (zeros outside the image).
    auto load = [&](int ch) {
        const int band = ch % g_.nbands, frame = ch / g_.nbands, h0 = band * TH;
#pragma unroll
        for (int i = 0; i < kWgItems; ++i) {
            const int idx = tid + 256 * i;
            xr[i].raw[0] = make_uint4(0, 0, 0, 0);
            if constexpr (sizeof(xr[i].raw) > 16) xr[i].raw[1] = make_uint4(0, 0, 0, 0);
            if (idx < g_.nx) {
                const int cg = idx % NCI, pos = idx / NCI;
                const int r = pos / W, w = pos % W, h = h0 + r - 1;
                if (h >= 0 && h < H) {
                    if constexpr (MODE == IN_U8) {
                        const int64_t row = a.row_idx ? a.row_idx[frame] : frame;
                        xr[i].raw[0].x = *reinterpret_cast<const uint32_t*>(
                            static_cast<const uint8_t*>(a.x) + ((row * H + h) * W + w) * 4);
                    } else {
                        const uint4* src = reinterpret_cast<const uint4*>(
                            static_cast<const T*>(a.x) + ((int64_t(frame) * H + h) * W + w) * CIN + cg * VEC);
                        xr[i].raw[0] = src[0];
                        if constexpr (sizeof(xr[i].raw) > 16) xr[i].raw[1] = src[1];
                    }
                }
            }
            gr[i].raw[0] = make_uint4(0, 0, 0, 0);
            if constexpr (sizeof(gr[i].raw) > 16) gr[i].raw[1] = make_uint4(0, 0, 0, 0);
            if (idx < g_.ng) {
                const int cg = idx % NCO, pos = idx / NCO;
                const int r = pos / W, w = pos % W;
                if (h0 + r < H) {
                    const uint4* src = reinterpret_cast<const uint4*>(
                        dy + ((int64_t(frame) * H + h0 + r) * W + w) * COUT + cg * 8);
                    gr[i].raw[0] = src[0];
                    if constexpr (sizeof(gr[i].raw) > 16) gr[i].raw[1] = src[1];
                }
            }
        }
    };

    auto unpack = [&](const uint4* raw, int n, float* v) {
        if constexpr (BF) {
            const uint32_t* u = reinterpret_cast<const uint32_t*>(raw);
            for (int j = 0; j < n / 2; ++j) {
                v[2 * j] = __uint_as_float(u[j] << 16);
                v[2 * j + 1] = __uint_as_float(u[j] & 0xffff0000u);
            }
        } else {
            const float* f = reinterpret_cast<const float*>(raw);
            for (int j = 0; j < n; ++j) v[j] = f[j];
        }
    };

    // Registers -> LDS: input channel-major, gradient in three column-shifted copies.
    auto store = [&]() {
#pragma unroll
        for (int i = 0; i < kWgItems; ++i) {
            const int idx = tid + 256 * i;
            if (idx < g_.nx) {
                const int cg = idx % NCI, pos = idx / NCI;
                const int r = pos / W, w = pos % W;
                float v[VEC];
                if constexpr (MODE == IN_U8) {
                    const uint32_t u = xr[i].raw[0].x;
#pragma unroll
                    for (int j = 0; j < 4; ++j) v[j] = float((u >> (8 * j)) & 0xff);
                } else {
                    unpack(xr[i].raw, VEC, v);
                    if (MODE == IN_RELU) {
#pragma unroll
                        for (int j = 0; j < VEC; ++j) v[j] = relu_f(v[j]);
                    }
                }
                T* dst = xT + (cg * VEC) * XP + r * PITCH + w + 1;
#pragma unroll
                for (int j = 0; j < VEC; ++j) dst[j * XP] = P::store(v[j]);
            }
            if (idx < g_.ng) {
                const int cg = idx % NCO, pos = idx / NCO;
                const int r = pos / W, w = pos % W;
                float v[8];
                unpack(gr[i].raw, 8, v);
#pragma unroll
                for (int j = 0; j < 8; ++j) bsum[j] += v[j];
                T* dst = gS + (cg * 8) * GP + r * PITCH + w;
#pragma unroll
                for (int kx = 0; kx < 3; ++kx)
#pragma unroll
                    for (int j = 0; j < 8; ++j) dst[(kx * COUT + j) * GP + kx] = P::store(v[j]);
            }
        }
    };

    int ch = blockIdx.x;
    if (ch < g_.nchunks) load(ch);
    for (; ch < g_.nchunks; ch += gridDim.x) {
        __syncthreads();   // zero fill / previous chunk's MFMA reads are done
        store();
        __syncthreads();
        if (ch + int(gridDim.x) < g_.nchunks) load(ch + gridDim.x);   // overlaps the MFMAs
        for (int k0 = 0; k0 < KLEN; k0 += KSTEP) {
#pragma unroll
            for (int j = 0; j < G::TPW; ++j) {
                if (wave + 4 * j < G::TILES) {
                    const Frag af = P::lds_frag(gS + a_off[j] + k0);
                    const Frag bf = b_ok[j] ? P::lds_frag(xT + b_off[j] + k0) : P::zero();
                    acc[j] = P::mma(af, bf, acc[j]);
                }
            }
        }
    }

    // ---- write this workgroup's partial: [kx][co][col] then the bias
    float* part = a.partial + int64_t(blockIdx.x) * G::PSTRIDE;
#pragma unroll
    for (int j = 0; j < G::TPW; ++j) {
        const int t = wave + 4 * j;
        if (t < G::TILES) {
            const int kx = t / (G::MT * G::NTN), mt = (t / G::NTN) % G::MT, nt = t % G::NTN;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int co = mt * 16 + 4 * g + i, col = nt * 16 + r16;
                part[(kx * COUT + co) * (G::NTN * 16) + col] = acc[j][i];
            }
        }
    }
    // bias: threads with the same channel group (tid % NCO) combine in a fixed order
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);      // [256][8]
#pragma unroll
    for (int j = 0; j < 8; ++j) red[tid * 8 + j] = bsum[j];
    __syncthreads();
    if (tid < COUT) {
        const int cg = tid / 8, j = tid % 8;
        float s = 0.f;
        for (int t = cg; t < 256; t += NCO) s += red[t * 8 + j];
        part[3 * COUT * G::NTN * 16 + tid] = s;
    }
}

// Fixed-order sum of `nparts` partials of `pstride` floats, 16 consecutive entries per
// 1024-thread block: slice s (of 64) adds partials s, s+64, ..., then a fixed pairwise tree
// over the slices. emit(entry, total) gets each entry's sum.
template <class F>
CB_DEV void sum_partials16(const float* __restrict__ partial, int nparts, int pstride, F&& emit) {
    __shared__ float sh[64][17];
    const int el = threadIdx.x & 15, sp = threadIdx.x >> 4;
    const int e = blockIdx.x * 16 + el;
    float s = 0.f;
    if (e < pstride)
        for (int p = sp; p < nparts; p += 64) s += partial[int64_t(p) * pstride + e];
    sh[sp][el] = s;
    __syncthreads();
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) {
        if (sp < w) sh[sp][el] += sh[sp + w][el];
        __syncthreads();
    }
    if (sp == 0 && e < pstride) emit(e, sh[0][el]);
}

// Sum the partials of all workgroups in a fixed order and scatter to HWIO / bias.
template <int CIN, int COUT>
__global__ __launch_bounds__(1024) void wgrad_reduce_kernel(const float* __restrict__ partial,
                                                            int nparts, float* dw, float* db,
                                                            float scale) {
    using G = WgGeom<PrecF32, CIN, COUT>;
    sum_partials16(partial, nparts, G::PSTRIDE, [&](int e, float tot) {
        constexpr int WSZ = 3 * COUT * G::NTN * 16;
        if (e < WSZ) {
            const int col = e % (G::NTN * 16), co = (e / (G::NTN * 16)) % COUT, kx = e / (COUT * G::NTN * 16);
            if (col < G::NCOL) {
                const int ky = col / CIN, ci = col % CIN;
                dw[((ky * 3 + kx) * CIN + ci) * COUT + co] = tot * scale;
            }
        } else {
            db[e - WSZ] = tot;
        }
    });
}

// ------------------------------------------------------------------ bf16: transpose reads
//
// The contraction runs over output pixels q, which an MFMA fragment wants consecutive in a
// lane, while NHWC tiles keep channels consecutive. Here both operands are staged in NHWC as
// they are, with direct buffer->LDS loads, and the fragments come from the LDS transpose
// read: in a group of 16 lanes, lane 4j+m addresses 4 channels (4m..4m+3 of a 16-channel
// block) of pixel q_j and lane i receives channel i of the four pixels q_0..q_3; two reads
// give a fragment's 8 pixels. A = dy^T (rows: output channels). B = the input window shifted
// by one tap (columns: 16 input channels of that tap; for uint8 frames, 4 taps x 4 channels).
// The bias gradient is one more column block whose B fragment is all ones, so it is summed
// in the same order as the weights. Waves split the column blocks, and when there are few
// blocks also the k-steps (summed across waves in a fixed order at the end). Each workgroup
// writes one float32 partial; a second kernel adds the partials in a fixed order.

template <int CIN, int COUT, int MODE>
struct WgTr {
    static constexpr bool U8 = MODE == IN_U8;
    // pixel pitches in bytes; 8 pixels x 32 bytes then cover distinct banks
    static constexpr int XPB = U8 ? 8 : CIN * 2 + (CIN >= 32 ? 32 : 0);
    static constexpr int DPB = COUT * 2 + (COUT >= 32 ? 32 : 0);
    static constexpr int MT = COUT / 16;
    static constexpr int NB = U8 ? 3 : 9 * CIN / 16;                  // weight column blocks
    static constexpr int NBB = NB + 1;                                 // + the bias block
    static constexpr int TILES = MT * NBB;
    // Row blocks per wave. One row block each while a wave's column blocks fit in 12
    // accumulator tiles; with 64 output channels and at least 32 input channels (19 or 37
    // column blocks) a wave keeps all four row blocks of a quarter of the column blocks, so
    // one B fragment read from LDS feeds four MFMAs (accumulators in AGPRs, one wave per SIMD).
    static constexpr int MTW = (MT == 4 && NBB > 12) ? 4 : 1;
    static constexpr int MTG = MT / MTW;                               // row-block groups
    // waves splitting k: as many as leave each wave at most 12 accumulator tiles (MTW = 1)
    static constexpr int kw_fits(int kw) {
        return MTW > 1 ? kw == 1 : ((4 / kw) % MT == 0 && (NBB + (4 / kw) / MT - 1) / ((4 / kw) / MT) <= 12);
    }
    static constexpr int KW = kw_fits(4) ? 4 : (kw_fits(2) ? 2 : 1);
    static constexpr int TG = 4 / KW;                                  // waves splitting tiles
    static constexpr int NPW = TG / MTG;                               // waves per row-block group
    static constexpr int TPW = (NBB + NPW - 1) / NPW;                  // column blocks per wave
    static constexpr int PSTRIDE = TILES * 256;                        // floats per partial
    static_assert(TG % MTG == 0, "row-block groups spread over whole wave groups");
};

struct WgTrRun {
    int TH, FR, nbands, ntiles;
    int raw_off, win_off, dy_off;   // LDS byte offsets; 16 zero bytes at offset 0
    float inv_W, inv_TW, inv_TH, inv_TR;
};

template <int CIN, int COUT, int MODE>
__global__ __launch_bounds__(256) void wgrad_tr_kernel(WgradArgs a, WgTrRun t) {
    using D = WgTr<CIN, COUT, MODE>;
    constexpr int XPB = D::XPB, DPB = D::DPB, NB = D::NB, NBB = D::NBB;
    constexpr int KW = D::KW, TG = D::TG, NPW = D::NPW, TPW = D::TPW, MTW = D::MTW, MTG = D::MTG;
    constexpr bool U8 = D::U8;
    constexpr int XSL = XPB / 16, DSL = DPB / 16;   // 16-byte DMA slots per pixel

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;
    unsigned char* raw = smem + t.raw_off;   // uint8 frames: [TR*TW] x 4 bytes
    unsigned char* win = smem + t.win_off;   // [FR][TR][TW] x XPB, bf16
    unsigned char* dyt = smem + t.dy_off;    // [FR*TH*W] x DPB, bf16

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const int kgrp = wave % KW, tgrp = wave / KW;
    const int mt0 = (tgrp % MTG) * MTW, nbw = tgrp / MTG;   // row blocks mt0 .. mt0+MTW-1
    const int H = a.H, W = a.W, TH = t.TH, FR = t.FR;
    const int TW = W + 2, TR = TH + 2;

    if (tid < 4) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;

    // Per-lane byte offset of each column block's chunk from the lane's tap-(0,0) window
    // pixel; -1 where the k values lie past the 9 taps (read as zero).
    int boff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = nbw + NPW * i;
        const int tap = U8 ? nb * 4 + m : nb / (CIN / 16 > 0 ? CIN / 16 : 1);
        const int ci = U8 ? 0 : (nb % (CIN / 16 > 0 ? CIN / 16 : 1)) * 16 + 4 * m;
        boff[i] = (nb < NB && tap < 9) ? ((tap / 3) * TW + tap % 3) * XPB + ci * 2 : -1;
    }
    cb_f32x4 acc[TPW][MTW];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int w = 0; w < MTW; ++w) acc[i][w] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

    int lg = blockIdx.x;   // neighbouring tiles (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int h0 = band * TH, f0 = fg * FR;
        const int nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int the = H - h0 < TH ? H - h0 : TH;
        const int npx = nf * the * W;   // FR > 1 only when a band is the whole frame
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage the input window and the output-gradient tile, HBM -> LDS
        if constexpr (U8) {
            const uint32_t fb = uint32_t(H) * W * 4;
            const int64_t row = a.row_idx ? a.row_idx[f0] : f0;
            const auto rx = buf_rsrc(static_cast<const uint8_t*>(a.x) + row * fb, fb);
            const int ns = TR * TW;
            for (int b = wave; b * 64 < ns; b += 4) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < ns) {
                    const int rr = qdiv(j, t.inv_TW), col = j - rr * TW, h = h0 + rr - 1;
                    if (col >= 1 && col <= W && h >= 0 && h < H) off = (uint32_t(h) * W + col - 1) * 4;
                }
                dma4_to_lds(rx, raw + b * 256, off);
            }
        } else {
            const uint32_t fb = uint32_t(H) * W * CIN * 2;
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + int64_t(f0) * H * W * CIN, uint32_t(nf) * fb);
            const int ns = FR * TR * TW * XSL;
            for (int b = wave; b * 64 < ns; b += 4) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < ns) {
                    const int p = j / XSL, c = j - p * XSL;
                    const int rowi = qdiv(p, t.inv_TW), col = p - rowi * TW;
                    const int f = qdiv(rowi, t.inv_TR), rr = rowi - f * TR, h = h0 + rr - 1;
                    if (c < CIN / 8 && col >= 1 && col <= W && h >= 0 && h < H)
                        off = ((uint32_t(f) * H + h) * W + col - 1) * (CIN * 2) + c * 16;
                }
                dma16_to_lds(rx, win + b * 1024, off);
            }
        }
        {
            const uint32_t gb = uint32_t(H) * W * COUT * 2;
            const auto rg = buf_rsrc(static_cast<const uint16_t*>(a.dy) + int64_t(f0) * H * W * COUT, uint32_t(nf) * gb);
            const int ns = npx * DSL;
            for (int b = wave; b * 64 < ns; b += 4) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < ns) {
                    const int q = j / DSL, c = j - q * DSL;
                    const int rowi = qdiv(q, t.inv_W), col = q - rowi * W;
                    const int f = qdiv(rowi, t.inv_TH), rr = rowi - f * TH;
                    if (c < COUT / 8) off = ((uint32_t(f) * H + h0 + rr) * W + col) * (COUT * 2) + c * 16;
                }
                dma16_to_lds(rg, dyt + b * 1024, off);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads have landed in LDS
        __syncthreads();                 // ... and everyone else's
        if constexpr (U8) {
            for (int p = tid; p < TR * TW; p += 256)
                *reinterpret_cast<uint2*>(win + p * 8) = u8x4_to_bf16(*reinterpret_cast<const uint32_t*>(raw + p * 4));
            __syncthreads();
        } else if constexpr (MODE == IN_RELU) {
            uint4* w4 = reinterpret_cast<uint4*>(win);
            for (int j = tid; j < FR * TR * TW * XSL; j += 256) {
                uint4 v = w4[j];
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                w4[j] = v;
            }
            __syncthreads();
        }

        // ---- k-steps of 32 pixels: lane (g, 4j+m) addresses pixels ks*32 + 16*half + 4g + j
        const int nks = (npx + 31) >> 5;
#pragma unroll 2
        for (int ks = kgrp; ks < nks; ks += KW) {
            uint2 av[2][MTW];
            int bp[2];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int q = ks * 32 + half * 16 + 4 * g + jj;
                const bool ok = q < npx;
                const int qc = ok ? q : 0;
                const int rowi = qdiv(qc, t.inv_W), col = qc - rowi * W;
                const int f = qdiv(rowi, t.inv_TH), r = rowi - f * TH;
                bp[half] = ((f * TR + r) * TW + col) * XPB;
#pragma unroll
                for (int w = 0; w < MTW; ++w)
                    av[half][w] = lds_read_tr16(ok ? dyt + q * DPB + ((mt0 + w) * 16 + 4 * m) * 2 : zero);
            }
            uint4 af[MTW];
#pragma unroll
            for (int w = 0; w < MTW; ++w) af[w] = make_uint4(av[0][w].x, av[0][w].y, av[1][w].x, av[1][w].y);
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
                const int nb = nbw + NPW * i;
                if (nb >= NBB) continue;
                uint4 bf = ones;
                if (nb < NB) {
                    const uint2 lo = lds_read_tr16(boff[i] >= 0 ? win + bp[0] + boff[i] : zero);
                    const uint2 hi = lds_read_tr16(boff[i] >= 0 ? win + bp[1] + boff[i] : zero);
                    bf = make_uint4(lo.x, lo.y, hi.x, hi.y);
                }
#pragma unroll
                for (int w = 0; w < MTW; ++w) acc[i][w] = PrecBF16::mma(af[w], bf, acc[i][w]);
            }
        }
    }

    // ---- this workgroup's partial: [mt*NBB + nb][row 16][col 16]
    if constexpr (KW > 1) {   // (MTW == 1 here)
        __syncthreads();   // tile LDS is free
        cb_f32x4* red = reinterpret_cast<cb_f32x4*>(smem);   // [KW][TG][TPW][64]
#pragma unroll
        for (int i = 0; i < TPW; ++i) red[((kgrp * TG + tgrp) * TPW + i) * 64 + lane] = acc[i][0];
        __syncthreads();
        if (kgrp == 0) {
#pragma unroll
            for (int i = 0; i < TPW; ++i)
                for (int k = 1; k < KW; ++k) acc[i][0] += red[((k * TG + tgrp) * TPW + i) * 64 + lane];
        }
    }
    if (kgrp == 0) {
        float* part = a.partial + int64_t(blockIdx.x) * D::PSTRIDE;
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const int nb = nbw + NPW * i;
            if (nb < NBB) {
#pragma unroll
                for (int w = 0; w < MTW; ++w)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        part[((mt0 + w) * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = acc[i][w][e];
            }
        }
    }
}

// Fixed-order sum of the partials, scattered to HWIO weights (times scale) and the bias.
template <int CIN, int COUT, int MODE>
__global__ __launch_bounds__(1024) void wgrad_tr_reduce_kernel(const float* __restrict__ partial,
                                                               int nparts, float* dw, float* db,
                                                               float scale) {
    using D = WgTr<CIN, COUT, MODE>;
    static_assert(D::PSTRIDE % 64 == 0, "whole 64-entry blocks");
    sum_partials_x4(partial, nparts, D::PSTRIDE, [&](int e0, float4 v) {
        const float tv[4] = {v.x, v.y, v.z, v.w};
        const int tile = e0 >> 8, row = (e0 >> 4) & 15;
        const int mt = tile / D::NBB, nb = tile % D::NBB, co = mt * 16 + row;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int col = (e0 & 15) + u;
            if (nb == D::NB) {
                if (col == 0) db[co] = tv[u];
            } else {
                const int tap = D::U8 ? nb * 4 + col / 4 : nb / (CIN / 16 > 0 ? CIN / 16 : 1);
                const int ci = D::U8 ? col % 4 : (nb % (CIN / 16 > 0 ? CIN / 16 : 1)) * 16 + col;
                if (tap < 9) dw[(tap * CIN + ci) * COUT + co] = tv[u] * scale;
            }
        }
    });
}

namespace {

constexpr int kWgradParts = 1024;        // upper bound on workgroups (and partials)
constexpr size_t kWgLds = 40 * 1024;      // aim for four workgroups per CU

template <class P, int CIN, int COUT>
size_t wg_lds(const WgRun& r) {
    return size_t(CIN * r.XP + 3 * COUT * r.GP) * sizeof(typename P::T);
}

template <class P, int CIN, int COUT, int MODE>
WgRun wg_plan(int n, int H, int W) {
    constexpr int VEC = MODE == IN_U8 ? 4 : 8;
    constexpr int NCI = CIN / VEC, NCO = COUT / 8;
    WgRun r;
    r.PITCH = round_up(W + 2, 8);
    for (int TH = H; TH >= 1; --TH) {
        r.TH = TH;
        r.KLEN = round_up(TH * r.PITCH, P::KSTEP);
        r.XP = round_up(r.KLEN + 2 * r.PITCH, 16) + 8;
        r.GP = round_up(r.KLEN, 16) + 8;
        r.nx = (TH + 2) * W * NCI;
        r.ng = TH * W * NCO;
        const bool fits = r.nx <= 256 * kWgItems && r.ng <= 256 * kWgItems;
        if (fits && (wg_lds<P, CIN, COUT>(r) <= kWgLds || TH == 1)) break;
    }
    r.nbands = (H + r.TH - 1) / r.TH;
    r.nchunks = n * r.nbands;
    return r;
}

// Workgroups (= partials): up to 1024 (four per CU), fewer when the partials would exceed
// ~40 MB (the fixed-order reduction reads them all once).
static int wg_parts_cap(int pstride) {
    int cap = int((40u << 20) / (sizeof(float) * size_t(pstride)));
    return cap < 256 ? 256 : (cap > kWgradParts ? kWgradParts : cap);
}

template <int CIN, int COUT>
int wg_parts(int nchunks) {
    const int cap = wg_parts_cap(WgGeom<PrecF32, CIN, COUT>::PSTRIDE);
    return nchunks < cap ? nchunks : cap;
}

template <class P, int CIN, int COUT, int MODE>
hipError_t wg_launch(const WgradArgs& a, hipStream_t s) {
    using G = WgGeom<P, CIN, COUT>;
    const WgRun r = wg_plan<P, CIN, COUT, MODE>(a.n, a.H, a.W);
    if (r.nx > 256 * kWgItems || r.ng > 256 * kWgItems) return hipErrorInvalidValue;
    const int parts = wg_parts<CIN, COUT>(r.nchunks);
    size_t lds = wg_lds<P, CIN, COUT>(r);
    if (lds < 256 * 8 * sizeof(float)) lds = 256 * 8 * sizeof(float);
    const int pr = sizeof(typename P::T) == 2 ? 0 : 1;
    const std::string shape = cb_dims(CIN, COUT) + "/" + cb_dims(a.H, a.W) + cb_flags(MODE, false, false);
    {
        ProfScope ps(s, [&] { return cb_key("wgrad", pr, shape); });
        hipLaunchKernelGGL((wgrad_kernel<P, CIN, COUT, MODE>), dim3(parts), dim3(256), lds, s, a, r);
    }
    {
        ProfScope ps(s, [&] { return cb_key("wgrad_reduce", pr, shape); });
        hipLaunchKernelGGL((wgrad_reduce_kernel<CIN, COUT>), dim3((G::PSTRIDE + 15) / 16), dim3(1024), 0,
                           s, a.partial, parts, a.dw, a.db, a.scale);
    }
    return hipGetLastError();
}

// ---- transpose-read kernel (bf16): band height that stages the fewest window rows within
// kWgTrLds of LDS; workgroups (= partials, summed afterwards) up to the resident count, with
// at most kWgTrPartBytes of partials.
constexpr int kWgTrLds = 40 * 1024;
constexpr size_t kWgTrPartBytes = 24u << 20;
constexpr int kWgTrPixMax = 2048;

static int wg_tr_parts_cap(size_t pstride) {
    const size_t cap = kWgTrPartBytes / (pstride * sizeof(float));
    return int(cap < 256 ? 256 : (cap > 1024 ? 1024 : cap));   // at least one workgroup per CU
}

// Channel pairs the transpose-read kernel takes (its accumulators fit in registers).
static bool wg_tr_ok(int cin, int cout) {
    return cin == 4 || (cin == 16 && (cout == 16 || cout == 32 || cout == 64)) ||
           (cin == 32 && (cout == 32 || cout == 64)) || (cin == 64 && cout == 64);
}
static size_t wg_tr_pstride(int cin, int cout) {
    const int nb = cin == 4 ? 3 : 9 * cin / 16;
    return size_t(cout / 16) * (nb + 1) * 256;
}

template <int CIN, int COUT, int MODE>
hipError_t wg_tr_launch(const WgradArgs& a, hipStream_t s) {
    using D = WgTr<CIN, COUT, MODE>;
    const int H = a.H, W = a.W;
    auto blk = [](int slots) { return (slots + 63) / 64; };
    auto regions = [&](int th, int fr, int& raw, int& win, int& dyb) {
        const int wp = fr * (th + 2) * (W + 2);
        raw = D::U8 ? blk(wp) * 256 : 0;
        win = D::U8 ? (wp * 8 + 15) / 16 * 16 : blk(wp * (D::XPB / 16)) * 1024;
        dyb = blk(fr * th * W * (D::DPB / 16)) * 1024;
    };
    auto lds = [&](int th, int fr) {
        int raw, win, dyb;
        regions(th, fr, raw, win, dyb);
        return size_t(16 + raw + win + dyb);
    };
    const size_t limit = std::min<size_t>(lds_limit(), 160 * 1024);
    // four row blocks per wave hold one workgroup per CU: it may use most of the CU's LDS
    const size_t budget = D::MTW > 1 ? std::min<size_t>(limit, 144 * 1024) : size_t(kWgTrLds);
    int thmax = std::min(H, std::max(1, kWgTrPixMax / W));
    while (thmax > 1 && lds(thmax, 1) > budget) --thmax;
    if (lds(thmax, 1) > limit) return hipErrorInvalidValue;
    int TH = 1, best = 1 << 30;
    for (int th = 1; th <= thmax; ++th) {
        const int rows = (H + th - 1) / th * (th + 2);
        if (rows <= best) { best = rows; TH = th; }
    }
    const int nbands = (H + TH - 1) / TH;
    int FR = 1;
    if (nbands == 1 && !D::U8)
        while (FR < a.n && lds(TH, FR + 1) <= budget && (FR + 1) * H * W <= kWgTrPixMax) ++FR;
    if (int64_t(FR) * H * W * std::max(CIN, COUT) * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    WgTrRun r{};
    r.TH = TH; r.FR = FR; r.nbands = nbands; r.ntiles = nbands * ((a.n + FR - 1) / FR);
    int raw, win, dyb;
    regions(TH, FR, raw, win, dyb);
    r.raw_off = 16; r.win_off = 16 + raw; r.dy_off = r.win_off + win;
    r.inv_W = 1.f / float(W); r.inv_TW = 1.f / float(W + 2);
    r.inv_TH = 1.f / float(TH); r.inv_TR = 1.f / float(TH + 2);
    size_t L = lds(TH, FR);
    if (D::KW > 1) L = std::max<size_t>(L, size_t(4) * D::TPW * 64 * 16);   // cross-wave sums
    const void* fn = reinterpret_cast<const void*>(&wgrad_tr_kernel<CIN, COUT, MODE>);
    int parts = std::min(resident_blocks(fn, 256, L), wg_tr_parts_cap(D::PSTRIDE));
    if (parts > r.ntiles) parts = r.ntiles;
    const std::string shape = cb_dims(CIN, COUT) + "/" + cb_dims(H, W) + cb_flags(MODE, false, false);
    {
        ProfScope ps(s, [&] { return cb_key("wgrad", 0, shape); });
        hipLaunchKernelGGL((wgrad_tr_kernel<CIN, COUT, MODE>), dim3(parts), dim3(256), L, s, a, r);
    }
    {
        ProfScope ps(s, [&] { return cb_key("wgrad_reduce", 0, shape); });
        hipLaunchKernelGGL((wgrad_tr_reduce_kernel<CIN, COUT, MODE>), dim3(D::PSTRIDE / 64), dim3(1024),
                           0, s, a.partial, parts, a.dw, a.db, a.scale);
    }
    return hipGetLastError();
}

template <class P>
hipError_t wg_dispatch(int cin, int cout, int mode, const WgradArgs& a, hipStream_t s) {
    if constexpr (std::is_same_v<P, PrecBF16>) {
#define CB_WGT(CI, CO, MD) \
        if (cin == CI && cout == CO && mode == MD) return wg_tr_launch<CI, CO, MD>(a, s);
        CB_WGT(4, 16, IN_U8) CB_WGT(4, 32, IN_U8) CB_WGT(4, 64, IN_U8)
        CB_WGT(16, 16, IN_PLAIN) CB_WGT(16, 32, IN_PLAIN) CB_WGT(16, 64, IN_PLAIN) CB_WGT(32, 32, IN_PLAIN)
        CB_WGT(32, 64, IN_PLAIN) CB_WGT(64, 64, IN_PLAIN)
        CB_WGT(16, 16, IN_RELU) CB_WGT(32, 32, IN_RELU) CB_WGT(64, 64, IN_RELU)
#undef CB_WGT
    }
#define CB_WG(CI, CO, MD) \
    if (cin == CI && cout == CO && mode == MD) return wg_launch<P, CI, CO, MD>(a, s);
    CB_WG(4, 16, IN_U8) CB_WG(4, 32, IN_U8) CB_WG(4, 64, IN_U8)
    CB_WG(16, 16, IN_PLAIN) CB_WG(16, 32, IN_PLAIN) CB_WG(16, 64, IN_PLAIN)
    CB_WG(32, 32, IN_PLAIN) CB_WG(32, 64, IN_PLAIN) CB_WG(64, 64, IN_PLAIN)
    CB_WG(16, 16, IN_RELU) CB_WG(32, 32, IN_RELU) CB_WG(64, 64, IN_RELU)
#undef CB_WG
    return hipErrorInvalidValue;
}

template <int CIN, int COUT>
size_t pstride() { return WgGeom<PrecF32, CIN, COUT>::PSTRIDE; }

}  // namespace

hipError_t wgrad_reduce_tr(int cin, int cout, const float* partial, int nparts, float* dw, float* db,
                           float scale, hipStream_t s) {
#define CB_RT(CI, CO, MD)                                                                              \
    if (cin == CI && cout == CO) {                                                                     \
        hipLaunchKernelGGL((wgrad_tr_reduce_kernel<CI, CO, MD>),                                       \
                           dim3(WgTr<CI, CO, MD>::PSTRIDE / 64), dim3(1024), 0, s, partial,            \
                           nparts, dw, db, scale);                                                     \
        return hipGetLastError();                                                                      \
    }
    CB_RT(16, 16, IN_PLAIN) CB_RT(16, 32, IN_PLAIN) CB_RT(32, 32, IN_PLAIN) CB_RT(32, 64, IN_PLAIN)
    CB_RT(64, 64, IN_PLAIN) CB_RT(4, 16, IN_U8) CB_RT(4, 32, IN_U8)
#undef CB_RT
    return hipErrorInvalidValue;
}

bool wgrad_supported(int cin, int cout, int mode) {
    auto ok = [](int c) { return c == 16 || c == 32 || c == 64; };
    if (mode == IN_U8) return cin == 4 && ok(cout);
    if (mode == IN_RELU) return cin == cout && ok(cin);
    return ok(cin) && ok(cout) && cin <= cout;
}

size_t wgrad_partial_floats(int prec, int cin, int cout, int H, int W) {
    (void)H; (void)W;
    if (prec == BF16 && wg_tr_ok(cin, cout)) {
        const size_t ps = wg_tr_pstride(cin, cout);
        return size_t(wg_tr_parts_cap(ps)) * ps;
    }
    const size_t ncol = size_t(3 * cin + 15) / 16 * 16;
    const size_t pst = 3 * size_t(cout) * ncol + cout;
    return size_t(wg_parts_cap(int(pst))) * pst;
}

hipError_t conv3x3_wgrad(int prec, int cin, int cout, int mode, const WgradArgs& a,
                         hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    return prec == BF16 ? wg_dispatch<PrecBF16>(cin, cout, mode, a, s)
                        : wg_dispatch<PrecF32>(cin, cout, mode, a, s);
}

__global__ __launch_bounds__(1024) void pending_reduce_kernel(PendingReduce r) {
    __shared__ __align__(16) unsigned char sh[64 * 17 * 16];
    pending_reduce<1024>(r, sh);
}

hipError_t flush_pending_reduce(const PendingReduce& r, hipStream_t s) {
    if (r.nparts <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "wgrad_reduce_pending/" + cb_dims(r.cin, r.cout); });
    hipLaunchKernelGGL(pending_reduce_kernel, dim3(unsigned(r.pstride / 64)), dim3(1024), 0, s, r);
    return hipGetLastError();
}

}  // namespace cb
