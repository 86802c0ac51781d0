// A whole IMPALA-ResNet residual block in one kernel (bf16 forward):
//
//   t = conv1(relu(x)) + b1,   y = x + conv2(relu(t)) + b2     (3x3 SAME convolutions, C -> C)
//
// Layer by layer the block moves five activation tensors through HBM (x for conv1; t, x and y
// for conv2; t written once); here it moves three (x read, t and y written). Each tile is a
// band of TH output rows of one frame:
//   - the input window, rows h0-2 .. h0+TH+1 of x, is staged HBM -> LDS (buffer loads, zero
//     padding from out-of-range offsets) and ReLU'd in place; the band's own rows of x are
//     staged a second time, unmodified, for the residual add;
//   - conv1 computes t on the band's rows plus one halo row above and below (the halo rows
//     are recomputed by the neighbouring bands); t is rounded to bf16, the band's own rows
//     are stored (the backward pass reads them) and relu(t) goes to an LDS window with zero
//     padding columns, exactly what conv2 would have read from HBM;
//   - conv2 reads that window and writes y with the bias and the residual add fused.
// The per-MFMA layout is that of the single convolution kernel: 16 output pixels per MFMA
// column tile, weights as [out][tap*C + in] in LDS, one 16-byte B fragment per lane and
// k-step from a window whose pixels are C/8 16-byte slots plus one zero slot.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace cb {

template <int C>
struct RbGeom {
    static constexpr int K = 9 * C;
    static constexpr int KSTEPS = (K + 31) / 32;
    static constexpr int KP = KSTEPS * 32;
    static constexpr int KPITCH = KP + 8;                  // bf16 elements per weight row
    static constexpr int MT = C / 16;
    static constexpr int SPP = C / 8 + 1;                  // 16-byte slots per window pixel
    static constexpr int PB = SPP * 16;
    static constexpr int OCH = C / 8;                      // 16-byte slots per add-tile pixel
    static constexpr int WB = (C * KPITCH * 2 + 15) / 16 * 16;   // one weight set (bytes)
    static constexpr bool HOIST = 2 * MT * KSTEPS <= 12;   // both convs' A fragments in VGPRs
    __host__ __device__ static int blocks(int slots) { return (slots + 63) / 64; }
    __host__ __device__ static int xwin_bytes(int TH, int W) { return blocks((TH + 4) * (W + 2) * SPP) * 1024; }
    __host__ __device__ static int twin_bytes(int TH, int W) { return ((TH + 2) * (W + 2) * PB + 15) / 16 * 16; }
    __host__ __device__ static int add_bytes(int TH, int W) { return blocks(TH * W * OCH) * 1024; }
};

struct RbTile {
    int TH, nbands, ntiles;
    int x_off, t_off, a_off, b_off;   // LDS byte offsets; the two weight sets sit at 0 and WB
    float inv_W, inv_TW;
};

// The MFMAs of NP 16-pixel column tiles: acc[p][mt] += W[mt rows] * window(taps at xb[p]);
// each A fragment read from LDS feeds all NP tiles.
template <int C, int NP>
CB_DEV void rb_mma(const unsigned char* const* xb, const int* boff, int twpb, const uint16_t* wl,
                   const uint4* wreg, int r16, int g, cb_f32x4 (*acc)[C / 16]) {
    using G = RbGeom<C>;
#pragma unroll
    for (int ks = 0; ks < G::KSTEPS; ++ks) {
        // 16 channels: per-lane table (a k-step spans two taps); 32: tap ks, lane's slot g
        const int bo = C < 32 ? boff[ks] : (ks / 3) * twpb + (ks % 3) * G::PB + g * 16;
        uint4 b[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) b[p] = *reinterpret_cast<const uint4*>(xb[p] + bo);
#pragma unroll
        for (int mt = 0; mt < G::MT; ++mt) {
            uint4 af;
            if constexpr (G::HOIST) af = wreg[ks * G::MT + mt];
            else af = PrecBF16::lds_frag(wl + (mt * 16 + r16) * G::KPITCH + ks * 32 + g * 8);
#pragma unroll
            for (int p = 0; p < NP; ++p) acc[p][mt] = PrecBF16::mma(af, b[p], acc[p][mt]);
        }
    }
}

template <int C, int NW>
__global__ __launch_bounds__(64 * NW, 4) void resblock_fwd_kernel(ResBlockArgs a, RbTile t) {
    using G = RbGeom<C>;
    constexpr int NT = 64 * NW, KSTEPS = G::KSTEPS, KPITCH = G::KPITCH, MT = G::MT;
    constexpr int SPP = G::SPP, PB = G::PB, OCH = G::OCH;
    constexpr int NP = 1;   // column tiles per pass (two would spill at 32 channels)

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* wl1 = reinterpret_cast<uint16_t*>(smem);
    uint16_t* wl2 = reinterpret_cast<uint16_t*>(smem + G::WB);
    unsigned char* xw = smem + t.x_off;   // relu(x) window [TH+4][W+2] pixels
    unsigned char* tw = smem + t.t_off;   // relu(t) window [TH+2][W+2] pixels
    unsigned char* xa = smem + t.a_off;   // x of the band's rows [TH*W][C], for the add

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TH = t.TH, TW = W + 2;

    // ---- both weight sets -> LDS once ([out][tap*C + in], zero k padding); relu(t) window
    // zeroed once (its padding columns and zero slots are never written afterwards)
    for (int e = tid; e < 9 * C * C; e += NT) {
        const int o = e % C, k = e / C;
        wl1[o * KPITCH + k] = f2bf(a.w1[e]);
        wl2[o * KPITCH + k] = f2bf(a.w2[e]);
    }
    if constexpr (G::KP > G::K) {
        constexpr int PADK = G::KP - G::K;
        for (int e = tid; e < C * PADK; e += NT) {
            wl1[(e / PADK) * KPITCH + G::K + e % PADK] = 0;
            wl2[(e / PADK) * KPITCH + G::K + e % PADK] = 0;
        }
    }
    for (int j = tid; j < G::twin_bytes(TH, W) / 16; j += NT) reinterpret_cast<uint4*>(tw)[j] = make_uint4(0, 0, 0, 0);
    float* bs = reinterpret_cast<float*>(smem + t.b_off);   // b1 then b2
    for (int e = tid; e < 2 * C; e += NT) bs[e] = e < C ? (a.b1 ? a.b1[e] : 0.f) : (a.b2 ? a.b2[e - C] : 0.f);
    __syncthreads();
    uint4 wr1[G::HOIST ? MT * KSTEPS : 1], wr2[G::HOIST ? MT * KSTEPS : 1];
    if constexpr (G::HOIST) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                wr1[ks * MT + mt] = PrecBF16::lds_frag(wl1 + (mt * 16 + r16) * KPITCH + ks * 32 + g * 8);
                wr2[ks * MT + mt] = PrecBF16::lds_frag(wl2 + (mt * 16 + r16) * KPITCH + ks * 32 + g * 8);
            }
    }
    // per-lane B-fragment offsets from the tap-(0,0) pixel (both windows share the pitch);
    // only 16 channels need the table
    int boff[C < 32 ? KSTEPS : 1];
    if constexpr (C < 32) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / C, c = (k0 % C) / 8;
            boff[ks] = tap < 9 ? ((tap / 3) * TW + tap % 3) * PB + c * 16 : (SPP - 1) * 16;
        }
    }
    const int twpb = TW * PB;

    int lg = blockIdx.x;   // neighbouring bands on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int h0 = band * TH, the = H - h0 < TH ? H - h0 : TH;
        const int64_t fo = int64_t(f) * H * W * C;   // frame offset (elements)
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage: x window rows h0-2 .. h0+TH+1 and the band's own rows of x
        {
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + fo, uint32_t(H) * W * C * 2);
            const int ns = (TH + 4) * TW * SPP;
            for (int b = wave; b * 64 < ns; b += NW) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < ns) {
                    const int p = j / SPP, c = j - p * SPP;
                    const int rr = qdiv(p, t.inv_TW), col = p - rr * TW, h = h0 - 2 + rr;
                    if (c < SPP - 1 && col >= 1 && col <= W && h >= 0 && h < H)
                        off = ((uint32_t(h) * W + col - 1) * C + c * 8) * 2;
                }
                dma16_to_lds(rx, xw + b * 1024, off);
            }
            const int na = the * W * OCH;
            for (int b = wave; b * 64 < na; b += NW) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < na) {
                    const int q = j / OCH, c = j - q * OCH;
                    off = ((uint32_t(h0) * W + q) * C + c * 8) * 2;
                }
                dma16_to_lds(rx, xa + b * 1024, off);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        {
            uint4* w4 = reinterpret_cast<uint4*>(xw);
            for (int j = tid; j < (TH + 4) * TW * SPP; j += NT) {
                uint4 v = w4[j];
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                w4[j] = v;
            }
        }
        // t rows tr of the window <-> image row h0 - 1 + tr; rows outside the image stay zero
        const int tr0 = h0 == 0 ? 1 : 0;
        const int tr1 = the + 2 < H - h0 + 1 ? the + 2 : H - h0 + 1;
        {
            uint4* t4 = reinterpret_cast<uint4*>(tw);
            const int row16 = TW * PB / 16;
            if (tr0 == 1)
                for (int j = tid; j < row16; j += NT) t4[j] = make_uint4(0, 0, 0, 0);
            for (int j = tid; j < (the + 2 - tr1) * row16; j += NT) t4[tr1 * row16 + j] = make_uint4(0, 0, 0, 0);
        }
        __syncthreads();

        // ---- conv1: t on rows [tr0, tr1)
        uint16_t* tbase = static_cast<uint16_t*>(a.t) + fo;
        const int npx1 = (tr1 - tr0) * W;
        for (int nt0 = wave; nt0 * 16 < npx1; nt0 += NW * NP) {
          int qv[NP], trv[NP], cv[NP];
          const unsigned char* xb[NP];
#pragma unroll
          for (int p = 0; p < NP; ++p) {
              qv[p] = (nt0 + p * NW) * 16 + r16;
              const int qc = qv[p] < npx1 ? qv[p] : npx1 - 1;
              const int rowi = qdiv(qc, t.inv_W);
              cv[p] = qc - rowi * W; trv[p] = tr0 + rowi;
              xb[p] = xw + (trv[p] * TW + cv[p]) * PB;
          }
          cb_f32x4 accs[NP][MT];
#pragma unroll
          for (int p = 0; p < NP; ++p)
#pragma unroll
              for (int mt = 0; mt < MT; ++mt) accs[p][mt] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
          rb_mma<C, NP>(xb, boff, twpb, wl1, wr1, r16, g, accs);
#pragma unroll
          for (int p = 0; p < NP; ++p) {
            const int q = qv[p], tr = trv[p], col = cv[p];
            const cb_f32x4* acc = accs[p];
            if (q < npx1) {
                const int h = h0 - 1 + tr;
                const bool own = h >= h0 && h < h0 + the;
                uint16_t* tp = tbase + (uint32_t(h) * W + col) * C + g * 4;
                unsigned char* twp = tw + (tr * TW + col + 1) * PB + g * 8;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const float4 b1 = *reinterpret_cast<const float4*>(bs + mt * 16 + g * 4);
                    const uint32_t u0 = pack2bf(acc[mt][0] + b1.x, acc[mt][1] + b1.y);
                    const uint32_t u1 = pack2bf(acc[mt][2] + b1.z, acc[mt][3] + b1.w);
                    if (own) *reinterpret_cast<uint2*>(tp + mt * 16) = make_uint2(u0, u1);
                    *reinterpret_cast<uint2*>(twp + mt * 32) = make_uint2(relu_bf16x2(u0), relu_bf16x2(u1));
                }
            }
          }
        }
        __syncthreads();

        // ---- conv2 + residual: y on the band's rows
        uint16_t* ybase = static_cast<uint16_t*>(a.y) + fo;
        const int npx2 = the * W;
        for (int nt0 = wave; nt0 * 16 < npx2; nt0 += NW * NP) {
          int qv[NP], rv[NP], cv[NP];
          const unsigned char* xb[NP];
#pragma unroll
          for (int p = 0; p < NP; ++p) {
              qv[p] = (nt0 + p * NW) * 16 + r16;
              const int qc = qv[p] < npx2 ? qv[p] : npx2 - 1;
              rv[p] = qdiv(qc, t.inv_W); cv[p] = qc - rv[p] * W;
              xb[p] = tw + (rv[p] * TW + cv[p]) * PB;
          }
          cb_f32x4 accs[NP][MT];
#pragma unroll
          for (int p = 0; p < NP; ++p)
#pragma unroll
              for (int mt = 0; mt < MT; ++mt) accs[p][mt] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
          rb_mma<C, NP>(xb, boff, twpb, wl2, wr2, r16, g, accs);
#pragma unroll
          for (int p = 0; p < NP; ++p) {
            const int q = qv[p], r = rv[p], col = cv[p];
            const cb_f32x4* acc = accs[p];
            if (q < npx2) {
                uint16_t* yp = ybase + (uint32_t(h0 + r) * W + col) * C + g * 4;
                const uint16_t* ap = reinterpret_cast<const uint16_t*>(xa) + q * C + g * 4;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const float4 b2 = *reinterpret_cast<const float4*>(bs + C + mt * 16 + g * 4);
                    float ad[4];
                    load4(ap + mt * 16, ad);
                    store4(yp + mt * 16, acc[mt][0] + b2.x + ad[0], acc[mt][1] + b2.y + ad[1],
                           acc[mt][2] + b2.z + ad[2], acc[mt][3] + b2.w + ad[3]);
                }
            }
          }
        }
    }
}

namespace {

constexpr int kRbWaves = 8;
constexpr size_t kRbLdsTarget = 80 * 1024;

template <int C>
hipError_t rb_fwd_launch(const ResBlockArgs& a, hipStream_t s) {
    using G = RbGeom<C>;
    const int H = a.H, W = a.W;
    auto lds = [&](int th) {
        return size_t(2 * G::WB) + G::xwin_bytes(th, W) + G::twin_bytes(th, W) + G::add_bytes(th, W) + 2 * C * 4;
    };
    int thmax = H;
    while (thmax > 1 && lds(thmax) > kRbLdsTarget) --thmax;
    if (lds(thmax) > std::min<size_t>(lds_limit(), 160 * 1024)) return hipErrorInvalidValue;
    if (int64_t(H) * W * C * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    int TH = 1, best = 1 << 30;   // fewest staged window rows per frame
    for (int th = 1; th <= thmax; ++th) {
        const int rows = (H + th - 1) / th * (th + 4);
        if (rows <= best) { best = rows; TH = th; }
    }
    RbTile t{};
    t.TH = TH; t.nbands = (H + TH - 1) / TH; t.ntiles = t.nbands * a.n;
    t.x_off = 2 * G::WB;
    t.t_off = t.x_off + G::xwin_bytes(TH, W);
    t.a_off = t.t_off + G::twin_bytes(TH, W);
    t.b_off = t.a_off + G::add_bytes(TH, W);
    t.inv_W = 1.f / float(W); t.inv_TW = 1.f / float(W + 2);
    const size_t L = lds(TH);
    const void* fn = reinterpret_cast<const void*>(&resblock_fwd_kernel<C, kRbWaves>);
    int gx = std::max(1, resident_blocks(fn, 64 * kRbWaves, L));
    if (gx > t.ntiles) gx = t.ntiles;
    ProfScope ps(s, [&] { return cb_key("resblock_fwd", 0, cb_dims(C, C) + "/" + cb_dims(H, W)); });
    hipLaunchKernelGGL((resblock_fwd_kernel<C, kRbWaves>), dim3(unsigned(gx)), dim3(64 * kRbWaves), L, s, a, t);
    return hipGetLastError();
}

}  // namespace

bool resblock_fwd_supported(int C) { return C == 16 || C == 32; }

hipError_t resblock_fwd(int C, const ResBlockArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    if (C == 16) return rb_fwd_launch<16>(a, s);
    if (C == 32) return rb_fwd_launch<32>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace cb
