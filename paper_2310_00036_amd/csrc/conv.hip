// 3x3 stride-1 SAME convolution as an implicit GEMM on gfx950 MFMA (NHWC activations).
//
// D[o][pixel] = sum_k Wt[o][k] * X[k][pixel], with k = tap*CIN + i over the 9 taps and the
// CIN input channels. One workgroup (4 wave64s) owns FR frames x TH rows x all W columns and
// up to COUT output channels. It stages the zero-padded input window (TH+2 rows) and the
// weights in LDS once, then each wave walks 16-pixel tiles: per MFMA a lane reads 8
// consecutive channels of one tap (16 bytes) as its B fragment and 8 consecutive k of one
// output channel as its A fragment. Output lanes hold 4 consecutive channels of one pixel,
// so the fused epilogue (scale, bias, mask, residual add) stores 8 (bf16) or 16 (fp32)
// contiguous bytes.
//
// The same kernel computes the input gradient (flip = 1): the adjoint of a 3x3 SAME conv is
// a 3x3 SAME conv of dy with the weights rotated by 180 degrees and in/out channels swapped.
#include "common.h"
#include "kernels.h"

#include <algorithm>
#include <type_traits>

namespace cb {

template <class P, int CIN>
struct ConvGeom {
    using T = typename P::T;
    static constexpr int K = 9 * CIN;
    static constexpr int KSTEPS = (K + P::KSTEP - 1) / P::KSTEP;
    static constexpr int KP = KSTEPS * P::KSTEP;
    // LDS pitches (elements), padded so 16-lane fragment reads spread over the banks.
    static constexpr int KPITCH = KP + (sizeof(T) == 2 ? 8 : 1);
    static constexpr int CP = sizeof(T) == 2 ? (CIN >= 8 ? CIN + 8 : CIN) : CIN + 1;
};

constexpr int kConvItems = 6;   // 16-byte input load items per thread (register prefetch)

template <class P, int CIN, int COUT, int MODE, int FLIP>
__global__ __launch_bounds__(256) void conv3x3_kernel(ConvArgs a, int TH, int FR, int nbands,
                                                      int ntiles, int cout_total) {
    using T = typename P::T;
    using G = ConvGeom<P, CIN>;
    using Frag = typename P::Frag;
    constexpr int KPL = P::KPL, KSTEP = P::KSTEP, KSTEPS = G::KSTEPS, KP = G::KP;
    constexpr int KPITCH = G::KPITCH, CP = G::CP, MT = COUT / 16;
    constexpr bool BF = sizeof(T) == 2;
    // input load items: one pixel of uint8 frames, else 16 bytes of channels
    constexpr int VEC = MODE == IN_U8 ? 4 : (BF ? 8 : 4);
    constexpr int NCH = CIN / VEC;
    // keep the weight fragments in registers when they are few
    constexpr bool HOIST = BF && MT * KSTEPS <= 10;
    static_assert(MODE != IN_U8 || CIN == 4, "uint8 frames carry 4 stacked channels");
    static_assert(COUT % 16 == 0, "output channels in 16-wide MFMA tiles");

    extern __shared__ __align__(16) unsigned char smem[];
    T* wl = reinterpret_cast<T*>(smem);
    constexpr int WL_ELEMS = ((COUT * KPITCH) + 7) / 8 * 8;
    T* xs = wl + WL_ELEMS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int og = blockIdx.y * COUT;                  // first output channel of this group
    const int H = a.H, W = a.W;
    const int TW = W + 2, TR = TH + 2;
    const int nitems = FR * TR * W * NCH;

    // ---- weights -> LDS once: wl[o][tap*CIN + i], zero in the k padding
    if (FLIP) {
        // forward HWIO [9][cout_total(=our out channels)][CIN(=forward out)]; rotate taps.
        for (int e = tid; e < 9 * COUT * CIN; e += 256) {
            const int i = e % CIN, o = (e / CIN) % COUT, tap = e / (CIN * COUT);
            const float wv = a.w[(int64_t(tap) * cout_total + og + o) * CIN + i];
            wl[o * KPITCH + (8 - tap) * CIN + i] = P::store(wv);
        }
    } else {
        for (int e = tid; e < 9 * CIN * COUT; e += 256) {
            const int o = e % COUT, k = e / COUT;
            wl[o * KPITCH + k] = P::store(a.w[int64_t(k) * cout_total + og + o]);
        }
    }
    if constexpr (KP > G::K) {
        constexpr int PADK = KP - G::K;
        for (int e = tid; e < COUT * PADK; e += 256)
            wl[(e / PADK) * KPITCH + G::K + e % PADK] = P::store(0.f);
    }
    // The two padding columns of the window (image columns -1 and W) are zero for every
    // tile: write them once.
    for (int e = tid; e < FR * TR * 2 * CP; e += 256) {
        const int c = e % CP, side = (e / CP) % 2, rowi = e / (2 * CP);
        xs[(rowi * TW + (side ? W + 1 : 0)) * CP + c] = P::store(0.f);
    }

    // ---- register prefetch of one tile's window (zeros outside the image / past n).
    // Windows larger than the prefetch capacity are loaded directly, kConvItems items per
    // thread at a time, without overlap.
    const bool prefetch = nitems <= 256 * kConvItems;
    uint4 pre[kConvItems];
    auto load = [&](int tile, int base) {
        const int band = tile % nbands, fg = tile / nbands;
        const int h0 = band * TH, f0 = fg * FR;
#pragma unroll
        for (int i = 0; i < kConvItems; ++i) {
            pre[i] = make_uint4(0, 0, 0, 0);
            const int idx = base + tid + 256 * i;
            if (idx < nitems) {
                const int ch = idx % NCH, pix = idx / NCH;
                const int w = pix % W, rr = (pix / W) % TR, f = pix / (W * TR);
                const int h = h0 + rr - 1, frame = f0 + f;
                if (h >= 0 && h < H && frame < a.n) {
                    if constexpr (MODE == IN_U8) {
                        const int64_t row = a.row_idx ? a.row_idx[frame] : frame;
                        pre[i].x = *reinterpret_cast<const uint32_t*>(static_cast<const uint8_t*>(a.x) +
                                                                      ((row * H + h) * W + w) * 4);
                    } else {
                        pre[i] = *reinterpret_cast<const uint4*>(static_cast<const T*>(a.x) +
                                                                 ((int64_t(frame) * H + h) * W + w) * CIN + ch * VEC);
                    }
                }
            }
        }
    };
    auto store = [&](int base) {
#pragma unroll
        for (int i = 0; i < kConvItems; ++i) {
            const int idx = base + tid + 256 * i;
            if (idx < nitems) {
                const int ch = idx % NCH, pix = idx / NCH;
                const int w = pix % W, rr = (pix / W) % TR, f = pix / (W * TR);
                T* dst = xs + ((f * TR + rr) * TW + w + 1) * CP + ch * VEC;
                uint4 v = pre[i];
                if constexpr (MODE == IN_U8) {
                    const uint32_t u = v.x;
                    if constexpr (BF) {
                        *reinterpret_cast<uint2*>(dst) = make_uint2(pack2bf(float(u & 0xff), float((u >> 8) & 0xff)),
                                                                    pack2bf(float((u >> 16) & 0xff), float(u >> 24)));
                    } else {
                        dst[0] = float(u & 0xff); dst[1] = float((u >> 8) & 0xff);
                        dst[2] = float((u >> 16) & 0xff); dst[3] = float(u >> 24);
                    }
                } else if constexpr (BF) {
                    if (MODE == IN_RELU) {
                        uint32_t* u = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            uint32_t lo = u[j] & 0xffffu, hi = u[j] >> 16;
                            if ((lo & 0x8000u) && (lo & 0x7fffu) <= 0x7f80u) lo = 0;   // negative, not NaN
                            if ((hi & 0x8000u) && (hi & 0x7fffu) <= 0x7f80u) hi = 0;
                            u[j] = lo | (hi << 16);
                        }
                    }
                    *reinterpret_cast<uint4*>(dst) = v;
                } else {
                    const float* fv = reinterpret_cast<const float*>(&v);
#pragma unroll
                    for (int j = 0; j < 4; ++j) dst[j] = MODE == IN_RELU ? relu_f(fv[j]) : fv[j];
                }
            }
        }
    };

    const int g = lane >> 4, r16 = lane & 15;
    const int npx = FR * TH * W;
    const int ntl = (npx + 15) / 16;

    // Per-lane LDS offset of its B fragment within the 3x3 window, per k-step.
    auto b_off = [&](int ks, int half) -> int {
        const int k0 = ks * KSTEP + g * KPL + half * 4;
        const int tap = k0 / CIN, i = k0 % CIN;
        if (tap >= 9) return -1;
        return ((tap / 3) * TW + (tap % 3)) * CP + i;
    };

    int tile = blockIdx.x;
    if (prefetch && tile < ntiles) load(tile, 0);
    __syncthreads();   // weights and padding columns visible
    Frag wreg[HOIST ? MT * KSTEPS : 1];
    if constexpr (HOIST) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                wreg[ks * MT + mt] = P::lds_frag(wl + (mt * 16 + r16) * KPITCH + ks * KSTEP + g * KPL);
    }

    for (; tile < ntiles; tile += gridDim.x) {
        const int band = tile % nbands, fg = tile / nbands;
        const int h0 = band * TH, f0 = fg * FR;
        __syncthreads();   // previous tile's MFMA reads are done
        if (prefetch) {
            store(0);
        } else {
            for (int base = 0; base < nitems; base += 256 * kConvItems) {
                load(tile, base);
                store(base);
            }
        }
        __syncthreads();
        if (prefetch && tile + int(gridDim.x) < ntiles) load(tile + gridDim.x, 0);   // overlaps the MFMAs

        for (int nt = wave; nt < ntl; nt += 4) {
            const int q = nt * 16 + r16;
            const int qc = q < npx ? q : npx - 1;
            const int c = qc % W, rr = (qc / W) % TH, f = qc / (W * TH);
            const T* xb = xs + ((f * TR + rr) * TW + c) * CP;
            cb_f32x4 acc[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[mt] = cb_f32x4{0.f, 0.f, 0.f, 0.f};

            if constexpr (BF) {
#pragma unroll
                for (int ks = 0; ks < KSTEPS; ++ks) {
                    Frag b;
                    if constexpr (CIN == 4) {
                        const int o0 = b_off(ks, 0), o1 = b_off(ks, 1);
                        const uint2 lo = o0 >= 0 ? *reinterpret_cast<const uint2*>(xb + o0) : make_uint2(0, 0);
                        const uint2 hi = o1 >= 0 ? *reinterpret_cast<const uint2*>(xb + o1) : make_uint2(0, 0);
                        b = make_uint4(lo.x, lo.y, hi.x, hi.y);
                    } else {
                        const int o0 = b_off(ks, 0);
                        b = o0 >= 0 ? P::lds_frag(xb + o0) : P::zero();
                    }
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        Frag af;
                        if constexpr (HOIST) af = wreg[ks * MT + mt];
                        else af = P::lds_frag(wl + (mt * 16 + r16) * KPITCH + ks * KSTEP + g * KPL);
                        acc[mt] = P::mma(af, b, acc[mt]);
                    }
                }
            } else {
                for (int ks = 0; ks < KSTEPS; ++ks) {
                    const int o0 = b_off(ks, 0);
                    const Frag b = o0 >= 0 ? P::lds_frag(xb + o0) : P::zero();
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const Frag af = P::lds_frag(wl + (mt * 16 + r16) * KPITCH + ks * KSTEP + g * KPL);
                        acc[mt] = P::mma(af, b, acc[mt]);
                    }
                }
            }

            // ---- fused epilogue
            const int hh = h0 + rr, frame = f0 + f;
            if (q < npx && hh < H && frame < a.n) {
                const int64_t pix = (int64_t(frame) * H + hh) * W + c;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const int co = og + mt * 16 + g * 4;
                    float v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) v[j] = acc[mt][j] * a.scale + (a.bias ? a.bias[co + j] : 0.f);
                    if (a.mask) {
                        float mk[4];
                        load4(static_cast<const T*>(a.mask) + pix * cout_total + co, mk);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] = mk[j] > 0.f ? v[j] : 0.f;
                    }
                    if (a.add) {
                        float ad[4];
                        load4(static_cast<const T*>(a.add) + pix * cout_total + co, ad);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] += ad[j];
                    }
                    store4(static_cast<T*>(a.y) + pix * cout_total + co, v[0], v[1], v[2], v[3]);
                }
            }
        }
    }
}

// ------------------------------------------------------------------ bf16 streaming kernel
//
// At these channel counts a bf16 conv does about 70 flops per byte it must move, so it is
// bound by HBM, not by the matrix cores; this kernel is organised around keeping enough
// bytes in flight. Each tile (FR frames x TH output rows x all W columns) is staged with
// direct buffer->LDS loads, which need no registers: the zero-padded input window and, when
// present, the epilogue's mask and residual operands for exactly the tile's output pixels.
// Padding (image borders, frames past n) comes from offsets past the end of the buffer
// resource, which read as zeros. The waves then run the implicit GEMM out of LDS and store
// straight from the MFMA accumulators. Several workgroups per CU interleave their staging
// and compute phases.
//
// LDS layout (bytes): weights [COUT][KPITCH] bf16 | window [FR][TH+2][W+2] pixels |
// mask [FR*TH*W][COUT] bf16 | residual [FR*TH*W][COUT] bf16. A bf16 window pixel holds CIN/8
// 16-byte slots plus one slot that stays zero: the odd slot pitch spreads the 16 lanes of a
// fragment read (consecutive pixels) over distinct banks, and the zero slot doubles as the
// source of empty fragments. A uint8 window pixel is its 4 frame bytes.


struct DmaTile {
    int TH, FR, nbands, ntiles, cout_total;
    int win_off, mask_off, add_off;   // LDS byte offsets of the regions
    float inv_W, inv_TW, inv_TH, inv_TR;
    // fused max-pool: PTH pooled rows per band, pooled size OH x OW, pads ph/pw, conv tile
    int PTH, OH, OW, ph, pw, ct_off, zero_off;   // zero_off: 16 zero bytes
    float inv_OW, inv_ppf;   // 1/OW, 1/(OH*OW)
    int buf_off;             // double-buffered tiles: LDS byte offset of the second buffer
};

template <int CIN, int COUT, int MODE>
struct DmaGeom {
    using G = ConvGeom<PrecBF16, CIN>;
    static constexpr bool U8 = MODE == IN_U8;
    static constexpr int SPP = U8 ? 1 : CIN / 8 + 1;   // 16-byte LDS slots per bf16 window pixel
    static constexpr int PB = U8 ? 8 : SPP * 16;       // bytes per (bf16) window pixel
    static constexpr int OCH = COUT / 8;               // 16-byte operand slots per pixel
    static constexpr int WLB = (COUT * G::KPITCH * 2 + 15) / 16 * 16;
    __host__ __device__ static int blocks(int slots) { return (slots + 63) / 64; }
    // bf16 window; uint8 frames also stage their raw bytes (4 per pixel) right after it
    __host__ __device__ static int bf_bytes(int TH, int FR, int W) {
        const int wp = FR * (TH + 2) * (W + 2);
        return U8 ? (wp * 8 + 15) / 16 * 16 : blocks(wp * SPP) * 1024;
    }
    __host__ __device__ static int win_bytes(int TH, int FR, int W) {
        return bf_bytes(TH, FR, W) + (U8 ? blocks(FR * (TH + 2) * (W + 2)) * 256 : 0);
    }
    __host__ __device__ static int op_bytes(int TH, int FR, int W) { return blocks(FR * TH * W * OCH) * 64 * 16; }
};

// Waves per SIMD the register allocation must allow: four (four 4-wave or two 8-wave
// workgroups per CU, as the LDS budgets are sized), except the 64-output-channel tiles that
// read their weights from LDS, whose accumulators need the registers of two.
template <int CIN, int COUT, int MODE>
constexpr int conv_min_waves() {
    return (COUT >= 64 && (COUT / 16) * ((9 * CIN + 31) / 32) > 10) ? 2 : 4;
}

template <int CIN, int COUT, int MODE, int FLIP, int POOL, int NW>
__global__ __launch_bounds__(64 * NW, (conv_min_waves<CIN, COUT, MODE>())) void conv3x3_bf16_kernel(ConvArgs a, DmaTile t) {
    using D = DmaGeom<CIN, COUT, MODE>;
    using G = ConvGeom<PrecBF16, CIN>;
    using P = PrecBF16;
    constexpr int KSTEPS = G::KSTEPS, KPITCH = G::KPITCH, MT = COUT / 16;
    constexpr int SPP = D::SPP, PB = D::PB, OCH = D::OCH;
    constexpr bool U8 = D::U8;
    constexpr bool HOIST = MT * KSTEPS <= 10;
    static_assert(!U8 || CIN == 4, "uint8 frames carry 4 stacked channels");
    static_assert(U8 || CIN % 16 == 0, "bf16 inputs in 16-channel multiples");

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* wl = reinterpret_cast<uint16_t*>(smem);
    unsigned char* win = smem + t.win_off;
    unsigned char* raw = win + D::bf_bytes(t.TH, t.FR, a.W);   // uint8 frames only
    unsigned char* opm = smem + t.mask_off;
    unsigned char* opa = smem + t.add_off;

    constexpr int NT = 64 * NW;   // threads per workgroup
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int og = blockIdx.y * COUT;
    const int H = a.H, W = a.W, TH = t.TH, FR = t.FR;
    const int TW = W + 2, TR = TH + 2;
    const bool has_mask = a.mask != nullptr, has_add = a.add != nullptr;

    // ---- weights -> LDS once: wl[o][tap*CIN + i], zero in the k padding
    if (FLIP) {
        for (int e = tid; e < 9 * COUT * CIN; e += NT) {
            const int i = e % CIN, o = (e / CIN) % COUT, tap = e / (CIN * COUT);
            wl[o * KPITCH + (8 - tap) * CIN + i] = P::store(a.w[(int64_t(tap) * t.cout_total + og + o) * CIN + i]);
        }
    } else {
        for (int e = tid; e < 9 * CIN * COUT; e += NT) {
            const int o = e % COUT, k = e / COUT;
            wl[o * KPITCH + k] = P::store(a.w[int64_t(k) * t.cout_total + og + o]);
        }
    }
    if constexpr (G::KP > G::K) {
        constexpr int PADK = G::KP - G::K;
        for (int e = tid; e < COUT * PADK; e += NT)
            wl[(e / PADK) * KPITCH + G::K + e % PADK] = 0;
    }
    if (POOL && tid < 4) reinterpret_cast<uint32_t*>(smem + t.zero_off)[tid] = 0u;
    float bias[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) bias[mt][j] = a.bias ? a.bias[og + mt * 16 + g * 4 + j] : 0.f;
    __syncthreads();
    uint4 wreg[HOIST ? MT * KSTEPS : 1];
    if constexpr (HOIST) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                wreg[ks * MT + mt] = P::lds_frag(wl + (mt * 16 + r16) * KPITCH + ks * 32 + g * 8);
    }

    // ---- per-lane B-fragment offsets from the lane's tap-(0,0) window pixel (bytes).
    // k = ks*32 + g*8 .. +7 covers taps k / CIN; past the 9 taps the fragment is zero.
    auto tap_off = [&](int tap) { return ((tap / 3) * TW + tap % 3) * PB; };
    // With 16 input channels a k-step spans two taps, chosen by the lane group: a per-lane
    // table. From 32 channels on the tap is the k-step's and only the channel slot is the
    // lane's, so the offset is computed in place (no registers held across the loop).
    constexpr bool BTAB = U8 || CIN < 32;
    int boff[BTAB ? KSTEPS : 1];
    if constexpr (BTAB) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            if constexpr (U8) {
                boff[ks] = 0;   // uint8 fragments are read per tap below
            } else {
                const int k0 = ks * 32 + g * 8, tap = k0 / CIN, c = (k0 % CIN) / 8;
                boff[ks] = tap < 9 ? tap_off(tap) + c * 16 : (SPP - 1) * 16;   // zero slot
            }
        }
    }
    const int twpb = TW * PB;
    auto b_offset = [&](int ks) -> int {
        if constexpr (BTAB) {
            return boff[ks];
        } else {
            constexpr int TPK = CIN / 32;   // k-steps per tap
            const int tap = ks / TPK, cs = (ks % TPK) * 4;
            return (tap / 3) * twpb + (tap % 3) * PB + (cs + g) * 16;
        }
    };
    // uint8: lane g holds taps 2g, 2g+1 in k-step 0 and tap 8 (g == 0) in k-step 1
    const int u0 = tap_off(U8 ? 2 * g : 0), u1 = tap_off(U8 ? 2 * g + 1 : 0), u2 = tap_off(8);

    int lg = blockIdx.x;   // neighbouring tiles (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int f0 = fg * FR;
        const int nf = a.n - f0 < FR ? a.n - f0 : FR;
        // conv rows [h0, h0 + the): a band of TH rows, or (fused pool) exactly the rows the
        // band's pooled rows [p0, p1) read
        int h0, the, p0 = 0, p1 = 0;
        if constexpr (POOL) {
            p0 = band * t.PTH;
            p1 = p0 + t.PTH < t.OH ? p0 + t.PTH : t.OH;
            h0 = 2 * p0 - t.ph > 0 ? 2 * p0 - t.ph : 0;
            const int h1 = 2 * (p1 - 1) - t.ph + 3;
            the = (h1 < H ? h1 : H) - h0;
        } else {
            h0 = band * TH;
            the = H - h0 < TH ? H - h0 : TH;
        }
        const int npx = nf * the * W;   // FR > 1 only when a band is the whole frame
        uint16_t* ybase = static_cast<uint16_t*>(a.y) + (int64_t(f0) * H + h0) * W * t.cout_total + og;
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage window (and operands) HBM -> LDS
        if constexpr (U8) {
            const uint32_t fb = uint32_t(H) * W * 4;
            const int64_t row = a.row_idx ? a.row_idx[f0] : f0;
            const auto rx = buf_rsrc(static_cast<const uint8_t*>(a.x) + row * fb, fb);
            const int ns = TR * TW;
            for (int b = wave; b * 64 < ns; b += NW) {
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
            const int ns = FR * TR * TW * SPP;
            for (int b = wave; b * 64 < ns; b += NW) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < ns) {
                    const int p = j / SPP, c = j - p * SPP;
                    const int rowi = qdiv(p, t.inv_TW), col = p - rowi * TW;
                    const int f = qdiv(rowi, t.inv_TR), rr = rowi - f * TR, h = h0 + rr - 1;
                    if (c < SPP - 1 && col >= 1 && col <= W && h >= 0 && h < H)
                        off = ((uint32_t(f) * H + h) * W + col - 1) * (CIN * 2) + c * 16;
                }
                dma16_to_lds(rx, win + b * 1024, off);
            }
        }
        if (has_mask || has_add) {
            const uint32_t ob = uint32_t(H) * W * t.cout_total * 2;
            const int64_t fo = int64_t(f0) * H * W * t.cout_total;
            const auto rm = buf_rsrc(has_mask ? static_cast<const uint16_t*>(a.mask) + fo : nullptr, has_mask ? uint32_t(nf) * ob : 0);
            const auto ra = buf_rsrc(has_add ? static_cast<const uint16_t*>(a.add) + fo : nullptr, has_add ? uint32_t(nf) * ob : 0);
            const int ns = npx * OCH;
            for (int b = wave; b * 64 < ns; b += NW) {
                const int j = b * 64 + lane;
                uint32_t off = kOOB;
                if (j < ns) {
                    const int q = j / OCH, c = j - q * OCH;
                    const int rowi = qdiv(q, t.inv_W), col = q - rowi * W;
                    const int f = qdiv(rowi, t.inv_TH), rr = rowi - f * TH;
                    off = ((uint32_t(f) * H + h0 + rr) * W + col) * (t.cout_total * 2) + (og + c * 8) * 2;
                }
                if (has_mask) dma16_to_lds(rm, opm + b * 1024, off);
                if (has_add) dma16_to_lds(ra, opa + b * 1024, off);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads have landed in LDS
        __syncthreads();                 // ... and everyone else's
        if constexpr (U8) {
            // frames -> bf16 once per pixel (4 channels, exact for 0..255)
            for (int p = tid; p < TR * TW; p += NT)
                *reinterpret_cast<uint2*>(win + p * 8) = u8x4_to_bf16(*reinterpret_cast<const uint32_t*>(raw + p * 4));
            __syncthreads();
        } else if constexpr (MODE == IN_RELU) {
            uint4* w4 = reinterpret_cast<uint4*>(win);
            const int ns = FR * TR * TW * SPP;
            for (int j = tid; j < ns; j += NT) {
                uint4 v = w4[j];
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                w4[j] = v;
            }
            __syncthreads();
        }

        // ---- implicit GEMM over the tile's output pixels, 16 per MFMA column tile. When the
        // weight fragments come from LDS, each wave of the 8-wave variant takes NP = 2 column
        // tiles per pass so every A-fragment read feeds two MFMAs (the 4-wave variant keeps
        // one: the extra registers would cost it a resident workgroup per CU).
        constexpr int NP = (HOIST || U8 || NW < 8) ? 1 : 2;
        auto epilogue = [&](int q, int f, int r, int col, const cb_f32x4* acc) {
            if (POOL && q < npx) {
                // the bf16 conv value as an order-preserving 16-bit key (pool compares keys)
                unsigned char* cp = smem + t.ct_off + (q * COUT + g * 4) * 2;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    float v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) v[j] = acc[mt][j] * a.scale + bias[mt][j];
                    *reinterpret_cast<uint2*>(cp + mt * 32) =
                        make_uint2(bf16x2_key(pack2bf(v[0], v[1])), bf16x2_key(pack2bf(v[2], v[3])));
                }
            } else if (q < npx) {
                // 32-bit offset from the tile's first output element (the launcher bounds FR frames)
                uint16_t* yp = ybase + ((uint32_t(f) * H + r) * W + col) * uint32_t(t.cout_total) + g * 4;
                const int oq = (q * COUT + g * 4) * 2;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    float v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) v[j] = acc[mt][j] * a.scale + bias[mt][j];
                    if (has_mask) {
                        float mk[4];
                        load4(reinterpret_cast<const uint16_t*>(opm + oq + mt * 32), mk);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] = mk[j] > 0.f ? v[j] : 0.f;
                    }
                    if (has_add) {
                        float ad[4];
                        load4(reinterpret_cast<const uint16_t*>(opa + oq + mt * 32), ad);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] += ad[j];
                    }
                    store4(yp + mt * 16, v[0], v[1], v[2], v[3]);
                }
            }
        };
        const int ntl = (npx + 15) >> 4;
        for (int nt0 = wave; nt0 < ntl; nt0 += NW * NP) {
            // with many weight fragments (more than 18: 64 input channels), those read
            // from LDS stay inside the loop: hoisted out of it they would all take registers
            if constexpr (!HOIST && MT * KSTEPS > 18) asm volatile("" ::: "memory");
            int qv[NP], fv[NP], rv[NP], cv[NP];
            const unsigned char* xb[NP];
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                qv[p] = (nt0 + p * NW) * 16 + r16;   // past npx: clamped, computed, not stored
                const int qc = qv[p] < npx ? qv[p] : npx - 1;
                const int rowi = qdiv(qc, t.inv_W);
                cv[p] = qc - rowi * W;
                fv[p] = 0; rv[p] = rowi;
                if (FR > 1) { fv[p] = qdiv(rowi, t.inv_TH); rv[p] = rowi - fv[p] * TH; }
                xb[p] = win + ((fv[p] * TR + rv[p]) * TW + cv[p]) * PB;
            }
            cb_f32x4 acc[NP][MT];
#pragma unroll
            for (int p = 0; p < NP; ++p)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) acc[p][mt] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks) {
                uint4 b[NP];
#pragma unroll
                for (int p = 0; p < NP; ++p) {
                    if constexpr (U8) {
                        if (ks == 0) {
                            const uint2 lo = *reinterpret_cast<const uint2*>(xb[p] + u0);
                            const uint2 hi = *reinterpret_cast<const uint2*>(xb[p] + u1);
                            b[p] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                        } else {
                            const uint2 lo = *reinterpret_cast<const uint2*>(xb[p] + u2);
                            b[p] = g == 0 ? make_uint4(lo.x, lo.y, 0, 0) : make_uint4(0, 0, 0, 0);
                        }
                    } else {
                        b[p] = *reinterpret_cast<const uint4*>(xb[p] + b_offset(ks));
                    }
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    uint4 af;
                    if constexpr (HOIST) af = wreg[ks * MT + mt];
                    else af = P::lds_frag(wl + (mt * 16 + r16) * KPITCH + ks * 32 + g * 8);
#pragma unroll
                    for (int p = 0; p < NP; ++p) acc[p][mt] = P::mma(af, b[p], acc[p][mt]);
                }
            }
#pragma unroll
            for (int p = 0; p < NP; ++p) epilogue(qv[p], fv[p], rv[p], cv[p], acc[p]);
        }

        if constexpr (POOL) {
            // ---- 3x3 stride-2 max-pool of the conv tile, 8 channels per item. Per channel the
            // candidate (key << 16) | (15 - k) of window cell k (row-major 0..8) is maximised as an
            // integer: the largest key wins and, among equal keys, the first cell. Padded cells
            // are skipped, so they never win.
            __syncthreads();
            constexpr int C8 = COUT / 8;
            const int prows = p1 - p0;
            const int ppf = prows * t.OW;
            const int items = nf * ppf * C8;
            const unsigned char* ct = smem + t.ct_off;
            const unsigned char* zero16 = smem + t.zero_off;
            uint16_t* pbase = static_cast<uint16_t*>(a.y) + (int64_t(f0) * t.OH + p0) * t.OW * t.cout_total + og;
            uint8_t* abase = a.arg + (int64_t(f0) * t.OH + p0) * t.OW * t.cout_total + og;
            for (int it = tid; it < items; it += NT) {
                const int c8 = it % C8, pp = it / C8;
                const int f = FR > 1 ? qdiv(pp, t.inv_ppf) : 0;
                const int rem = pp - f * ppf;
                const int ohl = qdiv(rem, t.inv_OW), ow = rem - ohl * t.OW, oh = p0 + ohl;
                uint32_t best[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) best[j] = 0u;
                // cell (dy, dx) of the window; padded cells read the zero keys (never win), so
                // all nine loads go out without branches
                const int hc = 2 * oh - t.ph, wc = 2 * ow - t.pw;
                const unsigned char* cb = ct + (((f * TH + hc - h0) * W + wc) * COUT + c8 * 8) * 2;
                const bool rv[3] = {hc >= 0, true, hc + 2 < H};
                const bool cv[3] = {wc >= 0, true, wc + 2 < W};
                uint4 cell[9];
#pragma unroll
                for (int dy = 0; dy < 3; ++dy)
#pragma unroll
                    for (int dx = 0; dx < 3; ++dx)
                        cell[dy * 3 + dx] = *reinterpret_cast<const uint4*>(
                            rv[dy] && cv[dx] ? cb + (dy * W + dx) * COUT * 2 : zero16);
#pragma unroll
                for (int dy = 0; dy < 3; ++dy) {
#pragma unroll
                    for (int dx = 0; dx < 3; ++dx) {
                        const uint4 k4 = cell[dy * 3 + dx];
                        const uint32_t tag = 15u - uint32_t(dy * 3 + dx);
                        const uint32_t kk[4] = {k4.x, k4.y, k4.z, k4.w};
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            best[2 * j] = max(best[2 * j], (kk[j] << 16) | tag);
                            best[2 * j + 1] = max(best[2 * j + 1], (kk[j] & 0xffff0000u) | tag);
                        }
                    }
                }
                uint32_t vals[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    vals[j] = bf16x2_unkey((best[2 * j] >> 16) | (best[2 * j + 1] & 0xffff0000u));
                uint32_t idx[2] = {0u, 0u};
#pragma unroll
                for (int j = 0; j < 8; ++j) idx[j >> 2] |= (15u - (best[j] & 15u)) << (8 * (j & 3));
                const uint32_t o = ((uint32_t(f) * t.OH + ohl) * t.OW + ow) * uint32_t(t.cout_total) + c8 * 8;
                *reinterpret_cast<uint4*>(pbase + o) = make_uint4(vals[0], vals[1], vals[2], vals[3]);
                *reinterpret_cast<uint2*>(abase + o) = make_uint2(idx[0], idx[1]);
            }
        }
    }
}

// ------------------------------------------------------------------ register-weight kernel
//
// 64 output channels from 32 or 64 bf16 input channels (the wide net's residual convolutions
// and their input gradients). Their weight tile (up to 72 KB) leaves room for one window per
// workgroup beside it, and read from LDS it costs an A-fragment read for every MFMA pair.
// Here the 8 waves of a workgroup split the output channels in two halves and each wave holds
// its half's A fragments in registers for the whole launch (2 x 18 x 4 = 144 registers at 64
// input channels), so every B-fragment read feeds two MFMAs and LDS holds only tiles. One
// workgroup per CU double-buffers them: the next tile's window and epilogue operands are
// staged by buffer -> LDS loads while this tile's MFMAs run. (Two workgroups per CU with one
// buffer each fall into step, staging together and computing together, so their phases add
// up instead of overlapping.) Tile shapes, window layout and epilogue are those of
// conv3x3_bf16_kernel.
constexpr int kRegwWaves = 8;
constexpr int kRegwMaxW = 10, kRegwMaxQ = 4;   // staging slots per lane: window, operands

// Epilogue operand tiles hold per output pixel q its 8 slots of 8 channels, slot c of pixel q
// at position c ^ ((q >> 1) & 7): the 8-byte reads of 16 consecutive pixels' same channels
// then fall on distinct bank quadruples (pixel q starts 32 q (mod 64) banks in, plus 4 x its
// position), where unswizzled every pixel pair 2 apart would share them.
CB_DEV int op_slot(int q, int c) { return c ^ ((q >> 1) & 7); }

// Window layout of these tiles. gfx950's LDS serves a 16-byte read of a wave in four passes of
// 16 lanes, each pass conflict-free when its reads land on distinct 16-byte bank groups (64
// four-byte banks). A B fragment is 16 consecutive output pixels (one 16-byte slot each) of
// two adjacent lane groups; a pixel pitch of P slots spreads such a pass over distinct groups
// when P = 2 (mod 4), so a pixel holds CIN/8 data slots plus two zero slots (10 or 6). A run
// of pixels that wraps to the next row jumps over the two padding columns; extra slots at the
// end of every row (row pitch = W*P (mod 16) slots) keep the wrapped run's groups as they would
// be without the jump.
template <int CIN>
struct RegwGeom {
    static constexpr int SPP = CIN / 8 + 2;   // 16-byte slots per window pixel
    static constexpr int PB = SPP * 16;
    static_assert(SPP % 4 == 2, "pixel pitch = 2 (mod 4) slots");
    __host__ __device__ static int row_slots(int W) {
        const int base = (W + 2) * SPP;
        return base + ((W * SPP - base) % 16 + 16) % 16;
    }
    __host__ __device__ static int win_bytes(int TH, int FR, int W) {
        return (FR * (TH + 2) * row_slots(W) + 63) / 64 * 1024;
    }
};

template <int CIN, int COUT, int MODE, int FLIP>
__global__ __launch_bounds__(64 * kRegwWaves, 2) void conv3x3_regw_kernel(ConvArgs a, DmaTile t) {
    using D = DmaGeom<CIN, COUT, MODE>;
    using G = ConvGeom<PrecBF16, CIN>;
    using P = PrecBF16;
    constexpr int NW = kRegwWaves, NT = 64 * NW;
    constexpr int KSTEPS = G::KSTEPS, KPITCH = G::KPITCH, MT = COUT / 16;
    using R = RegwGeom<CIN>;
    constexpr int SPP = R::SPP, PB = R::PB, OCH = D::OCH;
    constexpr int OS = 2, MTW = MT / OS, NWC = NW / OS;   // output halves, waves per half
    constexpr int TPK = CIN / 32;                         // k-steps per tap
    constexpr int KPD = 6;                                // B fragments read ahead of their MFMAs
    static_assert(MODE != IN_U8 && CIN % 32 == 0 && MT % OS == 0 && G::KP == G::K && OCH == 8,
                  "bf16 inputs in 32-channel multiples (k-steps never straddle a tap)");

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* wl = reinterpret_cast<uint16_t*>(smem);   // weight loading area, then the tiles
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int og = blockIdx.y * COUT;
    const int mt0 = (wave % OS) * MTW;   // the wave's first 16-channel output block
    const int H = a.H, W = a.W, TH = t.TH, FR = t.FR;
    const int TR = TH + 2;
    const int RS = R::row_slots(W), RB = RS * 16;        // window row pitch (slots, bytes)
    const float inv_RS = 1.f / float(RS);
    const bool has_mask = a.mask != nullptr, has_add = a.add != nullptr;

    // ---- weights -> LDS as wl[o][tap*CIN + i] (bf16) -> this wave's A fragments
    if (FLIP) {
        for (int e = tid; e < 9 * COUT * CIN; e += NT) {
            const int i = e % CIN, o = (e / CIN) % COUT, tap = e / (CIN * COUT);
            wl[o * KPITCH + (8 - tap) * CIN + i] = P::store(a.w[(int64_t(tap) * t.cout_total + og + o) * CIN + i]);
        }
    } else {
        for (int e = tid; e < 9 * CIN * COUT; e += NT) {
            const int o = e % COUT, k = e / COUT;
            wl[o * KPITCH + k] = P::store(a.w[int64_t(k) * t.cout_total + og + o]);
        }
    }
    float bias[MTW][4];
#pragma unroll
    for (int m = 0; m < MTW; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) bias[m][j] = a.bias ? a.bias[og + (mt0 + m) * 16 + g * 4 + j] : 0.f;
    __syncthreads();
    uint4 wreg[MTW * KSTEPS];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
        for (int m = 0; m < MTW; ++m)
            wreg[ks * MTW + m] = P::lds_frag(wl + ((mt0 + m) * 16 + r16) * KPITCH + ks * 32 + g * 8);
    __syncthreads();   // every wave holds its fragments: the tiles may overwrite the weights

    // ---- staging of a tile's zero-padded input window and epilogue operands into a buffer.
    // A lane's slots are the same in every tile, so their source offsets are formed once,
    // relative to the tile's first frame and row 0; a tile adds its first row h0. Window rows
    // above the frame come out negative and wrap past the end of the buffer resource (one
    // frame's bytes when bands split frames), as do rows below it, so they read zero; with
    // several frames per tile (whole frames, h0 = 0) the padding rows are marked here, and
    // frames past n lie beyond the resource. Padding columns and zero slots never load.
    uint32_t woff[kRegwMaxW], qoff[kRegwMaxQ];
#pragma unroll
    for (int k = 0; k < kRegwMaxW; ++k) {
        const int j = (wave + NW * k) * 64 + lane;
        const int rowi = qdiv(j, inv_RS), rem = j - rowi * RS;
        const int col = rem / SPP, c = rem - col * SPP;
        const int f = qdiv(rowi, t.inv_TR), rr = rowi - f * TR;
        const bool ok = j < FR * TR * RS && c < CIN / 8 && col >= 1 && col <= W && (FR == 1 || (rr >= 1 && rr <= H));
        woff[k] = ok ? uint32_t(((f * H + rr - 1) * W + col - 1) * (CIN * 2) + c * 16) : kOOB;
    }
#pragma unroll
    for (int k = 0; k < kRegwMaxQ; ++k) {
        const int j = (wave + NW * k) * 64 + lane;
        const int q = j / OCH, c = op_slot(q, j - q * OCH);
        const int rowi = qdiv(q, t.inv_W), col = q - rowi * W;
        const int f = qdiv(rowi, t.inv_TH), rr = rowi - f * TH;
        qoff[k] = uint32_t(((f * H + rr) * W + col) * (t.cout_total * 2) + (og + c * 8) * 2);
    }
    auto stage = [&](unsigned char* dst, int tile) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int f0 = fg * FR, nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int h0 = band * TH, the = H - h0 < TH ? H - h0 : TH;
        const uint32_t fb = uint32_t(H) * W * CIN * 2;
        const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + int64_t(f0) * H * W * CIN, uint32_t(nf) * fb);
        const uint32_t hx = uint32_t(h0) * W * CIN * 2;   // (kOOB + hx stays past every resource)
        const int ns = FR * TR * RS;
#pragma unroll
        for (int k = 0; k < kRegwMaxW; ++k)
            if ((wave + NW * k) * 64 < ns) dma16_to_lds(rx, dst + (wave + NW * k) * 1024, woff[k] + hx);
        if (has_mask || has_add) {
            const uint32_t ob = uint32_t(H) * W * t.cout_total * 2;
            const int64_t fo = int64_t(f0) * H * W * t.cout_total;
            const auto rm = buf_rsrc(has_mask ? static_cast<const uint16_t*>(a.mask) + fo : nullptr, has_mask ? uint32_t(nf) * ob : 0);
            const auto ra = buf_rsrc(has_add ? static_cast<const uint16_t*>(a.add) + fo : nullptr, has_add ? uint32_t(nf) * ob : 0);
            const uint32_t ho = uint32_t(h0) * W * t.cout_total * 2;
            const int ns2 = nf * the * W * OCH;
#pragma unroll
            for (int k = 0; k < kRegwMaxQ; ++k) {
                const int b = wave + NW * k;
                if (b * 64 < ns2) {
                    const uint32_t off = b * 64 + lane < ns2 ? qoff[k] + ho : kOOB;
                    if (has_mask) dma16_to_lds(rm, dst + t.mask_off + b * 1024, off);
                    if (has_add) dma16_to_lds(ra, dst + t.add_off + b * 1024, off);
                }
            }
        }
    };

    // ---- one tile out of `cur` while the next one lands in `nxt`. The buffers are restrict
    // parameters, so the compiler knows the loads in flight into nxt do not write what this
    // tile reads and does not wait for them before its LDS reads.
    auto run_tile = [&](unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt, int tile) {
        if (tile + int(gridDim.x) < t.ntiles) stage(nxt, tile + gridDim.x);
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int f0 = fg * FR, nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int h0 = band * TH, the = H - h0 < TH ? H - h0 : TH;
        const int npx = nf * the * W;
        uint16_t* ybase = static_cast<uint16_t*>(a.y) + (int64_t(f0) * H + h0) * W * t.cout_total + og;
        if constexpr (MODE == IN_RELU) {
            // (unrolled over the lane's slots, so their LDS reads are in flight together)
            uint4* w4 = reinterpret_cast<uint4*>(cur);
            const int ns = FR * TR * RS;
#pragma unroll
            for (int k = 0; k < kRegwMaxW; ++k) {
                const int j = tid + NT * k;
                if (j < ns) {
                    uint4 v = w4[j];
                    v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                    w4[j] = v;
                }
            }
            lds_barrier();
        }
        const unsigned char* opm = cur + t.mask_off;
        const unsigned char* opa = cur + t.add_off;
        const int ntl = (npx + 15) >> 4;
        for (int nt = wave / OS; nt < ntl; nt += NWC) {
            const int q = nt * 16 + r16;   // past npx: clamped, computed, not stored
            const int qc = q < npx ? q : npx - 1;
            const int rowi = qdiv(qc, t.inv_W), col = qc - rowi * W;
            int f = 0, r = rowi;
            if (FR > 1) { f = qdiv(rowi, t.inv_TH); r = rowi - f * TH; }
            const unsigned char* xb = cur + (f * TR + r) * RB + col * PB;
            // k-step ks: tap ks / TPK (window pixel offset), channels (ks % TPK) * 32 + 8g
            auto bfrag = [&](int ks) {
                const int tap = ks / TPK;
                return *reinterpret_cast<const uint4*>(xb + (tap / 3) * RB + (tap % 3) * PB + ((ks % TPK) * 4 + g) * 16);
            };
            cb_f32x4 acc[MTW];
#pragma unroll
            for (int m = 0; m < MTW; ++m) acc[m] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
            uint4 bq[KSTEPS];
#pragma unroll
            for (int ks = 0; ks < KPD && ks < KSTEPS; ++ks) bq[ks] = bfrag(ks);
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks) {
                if (ks + KPD < KSTEPS) bq[ks + KPD] = bfrag(ks + KPD);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int m = 0; m < MTW; ++m) acc[m] = P::mma(wreg[ks * MTW + m], bq[ks], acc[m]);
                __builtin_amdgcn_sched_barrier(0);
            }
            if (q < npx) {
                uint16_t* yp = ybase + ((uint32_t(f) * H + r) * W + col) * uint32_t(t.cout_total) + g * 4;
                const int oq = q * OCH * 16 + (g & 1) * 8;
#pragma unroll
                for (int m = 0; m < MTW; ++m) {
                    const int mt = mt0 + m;
                    const int os = oq + op_slot(q, 2 * mt + (g >> 1)) * 16;   // channels mt*16 + 4g .. +3
                    float v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) v[j] = acc[m][j] * a.scale + bias[m][j];
                    if (has_mask) {
                        float mk[4];
                        load4(reinterpret_cast<const uint16_t*>(opm + os), mk);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] = mk[j] > 0.f ? v[j] : 0.f;
                    }
                    if (has_add) {
                        float ad[4];
                        load4(reinterpret_cast<const uint16_t*>(opa + os), ad);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] += ad[j];
                    }
                    store4(yp + mt * 16, v[0], v[1], v[2], v[3]);
                }
            }
        }
    };

    int lg = blockIdx.x;   // neighbouring tiles (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    if (lg < t.ntiles) stage(smem, lg);
    int it = 0;
    for (int tile = lg; tile < t.ntiles; tile += gridDim.x, ++it) {
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of the tile have landed in LDS
        __syncthreads();                 // ... and everyone else's; the other buffer is free
        run_tile(smem + (it & 1) * t.buf_off, smem + ((it + 1) & 1) * t.buf_off, tile);
    }
}

// ------------------------------------------------------------------ launcher

namespace {

// Tiles aim at 64 KB of LDS (two or more workgroups per CU); layers whose weights alone
// need more may use up to the device's per-workgroup maximum.
constexpr size_t kLdsTarget = 40 * 1024;

template <class P, int CIN, int COUT>
size_t conv_lds_bytes(int TH, int FR, int W) {
    using G = ConvGeom<P, CIN>;
    const size_t wl = (size_t(COUT) * G::KPITCH + 7) / 8 * 8;
    return (wl + size_t(FR) * (TH + 2) * (W + 2) * G::CP) * sizeof(typename P::T);
}

template <class P, int CIN, int COUT, int MODE, int FLIP>
hipError_t launch(const ConvArgs& a, int cout_total, hipStream_t s) {
    // Tile: bands of about 640 output pixels (whole frames when small), as many input load
    // items as the register prefetch holds, within the LDS budget.
    constexpr int VEC = MODE == IN_U8 ? 4 : (sizeof(typename P::T) == 2 ? 8 : 4);
    constexpr int NCH = CIN / VEC;
    const int H = a.H, W = a.W;
    int TH, FR = 1;
    if (H * W >= 640) {
        const int target = (640 + W - 1) / W;
        const int nb = (H + target - 1) / target;
        TH = (H + nb - 1) / nb;
    } else {
        TH = H;
        FR = 640 / (H * W);
        if (FR < 1) FR = 1;
        if (FR > a.n) FR = a.n;
    }
    auto items = [&](int th, int fr) { return fr * (th + 2) * W * NCH; };
    const size_t budget = std::max(kLdsTarget, std::min<size_t>(lds_limit(), 160 * 1024));
    while ((items(TH, FR) > 256 * kConvItems && (FR > 1 || TH > 1)) ||
           conv_lds_bytes<P, CIN, COUT>(TH, FR, W) > (FR > 1 || TH > 4 ? kLdsTarget : budget)) {
        if (FR > 1) --FR;
        else if (TH > 1) {
            const int nb = (H + TH - 1) / TH + 1;
            const int next = (H + nb - 1) / nb;
            TH = next < TH ? next : TH - 1;
        } else return hipErrorInvalidValue;
    }
    const int nbands = (H + TH - 1) / TH;
    const int nfg = (a.n + FR - 1) / FR;
    const int ntiles = nbands * nfg;
    const size_t lds = conv_lds_bytes<P, CIN, COUT>(TH, FR, W);
    const int groups = cout_total / COUT;
    // persistent grid: as many workgroups as are resident at once, over the channel groups
    const void* fn = reinterpret_cast<const void*>(&conv3x3_kernel<P, CIN, COUT, MODE, FLIP>);
    int gx = std::max(1, resident_blocks(fn, 256, lds) / groups);
    if (gx > ntiles) gx = ntiles;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(groups));
    ProfScope ps(s, [&] {
        return cb_key(FLIP ? "conv_dgrad" : "conv_fwd", sizeof(typename P::T) == 2 ? 0 : 1,
                      cb_dims(CIN, cout_total) + "/" + cb_dims(H, W) + cb_flags(MODE, a.mask, a.add));
    });
    hipLaunchKernelGGL((conv3x3_kernel<P, CIN, COUT, MODE, FLIP>), grid, dim3(256), lds, s, a, TH,
                       FR, nbands, ntiles, cout_total);
    return hipGetLastError();
}

// Output channels per workgroup: all of them unless the weight tile would crowd LDS.
template <class P, int CIN, int COUT>
constexpr int conv_group() {
    int cg = COUT;
    while (cg > 16 && cg * ConvGeom<P, CIN>::KPITCH * int(sizeof(typename P::T)) > 24 * 1024) cg /= 2;
    return cg;
}

// bf16 tiles: a band height that keeps a workgroup within kDmaLdsTarget (four per CU) and
// stages the fewest window rows per frame; whole frames batch up to kDmaPixMax pixels.
constexpr int kDmaLdsTarget = 40 * 1024;
constexpr int kDmaPixMax = 2048;
// Layers whose full weight tile is large (here the input gradient of 32 -> 64, whose kernel
// maps 64 channels to 32; 64 output channels go to conv3x3_regw_kernel) keep all output
// channels in one 8-wave workgroup per CU, with most of the CU's LDS: every staged
// window is read once and each weight fragment feeds two column tiles, where 16-channel
// groups would stage each window once per group and feed one MFMA per fragment pair.
constexpr int kDmaWideLdsTarget = 150 * 1024;
template <int CIN, int COUT>
constexpr bool conv_wide_tile() { return COUT * ConvGeom<PrecBF16, CIN>::KPITCH * 2 > 24 * 1024; }

template <int CIN, int COUT, int MODE, int FLIP>
hipError_t launch_bf16(const ConvArgs& a, int cout_total, hipStream_t s) {
    constexpr bool WIDE = conv_wide_tile<CIN, COUT>();
    constexpr int NW = WIDE ? 8 : 4;
    const int target = WIDE ? kDmaWideLdsTarget : kDmaLdsTarget;
    using D = DmaGeom<CIN, COUT, MODE>;
    const int H = a.H, W = a.W;
    const int nops = (a.mask ? 1 : 0) + (a.add ? 1 : 0);
    auto lds = [&](int th, int fr) {
        return size_t(D::WLB) + size_t(D::win_bytes(th, fr, W)) + size_t(nops) * D::op_bytes(th, fr, W);
    };
    const size_t limit = std::min<size_t>(lds_limit(), 160 * 1024);
    int thmax = std::min(H, std::max(1, kDmaPixMax / W));
    while (thmax > 1 && lds(thmax, 1) > size_t(target)) --thmax;
    if (lds(thmax, 1) > limit) return hipErrorInvalidValue;
    int TH = 1, best = 1 << 30;
    for (int th = 1; th <= thmax; ++th) {
        const int rows = (H + th - 1) / th * (th + 2);
        if (rows <= best) { best = rows; TH = th; }
    }
    const int nbands = (H + TH - 1) / TH;
    int FR = 1;
    if (nbands == 1 && MODE != IN_U8)
        while (FR < a.n && lds(TH, FR + 1) <= size_t(target) && (FR + 1) * H * W <= kDmaPixMax) ++FR;
    // 32-bit buffer offsets cover FR frames of input and of each operand
    if (int64_t(FR) * H * W * std::max(MODE == IN_U8 ? 2 : CIN, cout_total) * 2 >= (int64_t(1) << 31))
        return hipErrorInvalidValue;
    const int ntiles = nbands * ((a.n + FR - 1) / FR);
    const size_t L = lds(TH, FR);
    DmaTile t{};
    t.TH = TH; t.FR = FR; t.nbands = nbands; t.ntiles = ntiles; t.cout_total = cout_total;
    t.win_off = D::WLB;
    t.mask_off = t.win_off + D::win_bytes(TH, FR, W);
    t.add_off = t.mask_off + (a.mask ? D::op_bytes(TH, FR, W) : 0);
    t.inv_W = 1.f / float(W); t.inv_TW = 1.f / float(W + 2);
    t.inv_TH = 1.f / float(TH); t.inv_TR = 1.f / float(TH + 2);
    const int groups = cout_total / COUT;
    const void* fn = reinterpret_cast<const void*>(&conv3x3_bf16_kernel<CIN, COUT, MODE, FLIP, 0, NW>);
    int gx = std::max(1, resident_blocks(fn, 64 * NW, L) / groups);
    if (gx > ntiles) gx = ntiles;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(groups));
    ProfScope ps(s, [&] {
        return cb_key(FLIP ? "conv_dgrad" : "conv_fwd", 0,
                      cb_dims(CIN, cout_total) + "/" + cb_dims(H, W) + cb_flags(MODE, a.mask, a.add));
    });
    hipLaunchKernelGGL((conv3x3_bf16_kernel<CIN, COUT, MODE, FLIP, 0, NW>), grid, dim3(64 * NW), L, s, a, t);
    return hipGetLastError();
}

// Register-weight tiles: two buffers per workgroup, each within half of the CU's LDS.
template <int CIN, int COUT, int MODE>
constexpr bool conv_regw() { return MODE != IN_U8 && COUT == 64 && CIN >= 32 && CIN % 32 == 0; }
constexpr int kRegwBufTarget = 80 * 1024;

template <int CIN, int COUT, int MODE, int FLIP>
hipError_t launch_regw(const ConvArgs& a, int cout_total, hipStream_t s) {
    using D = DmaGeom<CIN, COUT, MODE>;
    const int H = a.H, W = a.W;
    const int nops = (a.mask ? 1 : 0) + (a.add ? 1 : 0);
    using R = RegwGeom<CIN>;
    // (tiles whose staging slots exceed the per-lane offset registers count as too large)
    auto buf = [&](int th, int fr) {
        const bool fits = fr * (th + 2) * R::row_slots(W) <= kRegwMaxW * 64 * kRegwWaves &&
                          fr * th * W * D::OCH <= kRegwMaxQ * 64 * kRegwWaves;
        return fits ? size_t(R::win_bytes(th, fr, W)) + size_t(nops) * D::op_bytes(th, fr, W) : size_t(1) << 30;
    };
    int thmax = std::min(H, std::max(1, kDmaPixMax / W));
    while (thmax > 1 && buf(thmax, 1) > size_t(kRegwBufTarget)) --thmax;
    if (buf(thmax, 1) > size_t(kRegwBufTarget)) return hipErrorInvalidValue;
    int TH = 1, best = 1 << 30;   // fewest staged window rows per frame
    for (int th = 1; th <= thmax; ++th) {
        const int rows = (H + th - 1) / th * (th + 2);
        if (rows <= best) { best = rows; TH = th; }
    }
    const int nbands = (H + TH - 1) / TH;
    int FR = 1;
    if (nbands == 1)
        while (FR < a.n && buf(TH, FR + 1) <= size_t(kRegwBufTarget) && (FR + 1) * H * W <= kDmaPixMax) ++FR;
    // 32-bit buffer offsets cover FR frames of input and of each operand
    if (int64_t(FR) * H * W * std::max(CIN, cout_total) * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    DmaTile t{};
    t.TH = TH; t.FR = FR; t.nbands = nbands; t.ntiles = nbands * ((a.n + FR - 1) / FR); t.cout_total = cout_total;
    t.win_off = 0;
    t.mask_off = R::win_bytes(TH, FR, W);
    t.add_off = t.mask_off + (a.mask ? D::op_bytes(TH, FR, W) : 0);
    t.buf_off = int(buf(TH, FR));
    t.inv_W = 1.f / float(W); t.inv_TW = 1.f / float(W + 2);
    t.inv_TH = 1.f / float(TH); t.inv_TR = 1.f / float(TH + 2);
    const size_t L = std::max(size_t(D::WLB), 2 * buf(TH, FR));
    if (L > std::min<size_t>(lds_limit(), 160 * 1024)) return hipErrorInvalidValue;
    const int groups = cout_total / COUT;
    const void* fn = reinterpret_cast<const void*>(&conv3x3_regw_kernel<CIN, COUT, MODE, FLIP>);
    int gx = std::max(1, resident_blocks(fn, 64 * kRegwWaves, L) / groups);
    if (gx > t.ntiles) gx = t.ntiles;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(groups));
    ProfScope ps(s, [&] {
        return cb_key(FLIP ? "conv_dgrad" : "conv_fwd", 0,
                      cb_dims(CIN, cout_total) + "/" + cb_dims(H, W) + cb_flags(MODE, a.mask, a.add));
    });
    hipLaunchKernelGGL((conv3x3_regw_kernel<CIN, COUT, MODE, FLIP>), grid, dim3(64 * kRegwWaves), L, s, a, t);
    return hipGetLastError();
}

// Conv + fused max-pool (bf16): bands of PTH pooled rows; each computes the 2*PTH+1 conv
// rows they read into LDS. Whole frames batch as in launch_bf16. The conv tile has to sit
// in LDS beside the window, so these workgroups take 8 waves and twice the LDS of the plain
// conv's: twice the rows per tile for the same waves per CU, halving the per-tile latency
// that small tiles leave exposed.
constexpr int kPoolWaves = 8;
constexpr int kPoolLdsTarget = 80 * 1024;
constexpr int kPoolPixMax = 4096;
template <int CIN, int COUT, int MODE>
hipError_t launch_bf16_pool(const ConvArgs& a, int cout_total, hipStream_t s) {
    using D = DmaGeom<CIN, COUT, MODE>;
    const int H = a.H, W = a.W;
    const int OH = (H + 1) / 2, OW = (W + 1) / 2;
    const int PH = (OH - 1) * 2 + 3 - H, PW = (OW - 1) * 2 + 3 - W;
    auto cap = [&](int pth, int fr) { return fr > 1 || pth >= OH ? H : std::min(2 * pth + 1, H); };
    auto lds = [&](int pth, int fr) {
        const int th = cap(pth, fr);
        return size_t(D::WLB) + size_t(D::win_bytes(th, fr, W)) + size_t(fr) * th * W * COUT * 2 + 16;
    };
    const size_t limit = std::min<size_t>(lds_limit(), 160 * 1024);
    // the wide budget only where the weights alone would crowd two workgroups per CU
    const int target = D::WLB > 40 * 1024 ? kDmaWideLdsTarget : kPoolLdsTarget;
    int pmax = OH;
    while (pmax > 1 && (lds(pmax, 1) > size_t(target) || cap(pmax, 1) * W > kPoolPixMax)) --pmax;
    if (lds(pmax, 1) > limit) return hipErrorInvalidValue;
    const int nbands0 = (OH + pmax - 1) / pmax;
    const int PTH = (OH + nbands0 - 1) / nbands0;
    const int nbands = (OH + PTH - 1) / PTH;
    int FR = 1;
    if (nbands == 1 && MODE != IN_U8)
        while (FR < a.n && lds(PTH, FR + 1) <= size_t(target) && (FR + 1) * H * W <= kPoolPixMax) ++FR;
    const int TH = cap(PTH, FR);
    if (int64_t(FR) * H * W * std::max(MODE == IN_U8 ? 2 : CIN, cout_total) * 2 >= (int64_t(1) << 31))
        return hipErrorInvalidValue;
    DmaTile t{};
    t.TH = TH; t.FR = FR; t.nbands = nbands; t.ntiles = nbands * ((a.n + FR - 1) / FR);
    t.cout_total = cout_total;
    t.win_off = D::WLB;
    t.ct_off = t.win_off + D::win_bytes(TH, FR, W);
    t.mask_off = t.add_off = t.ct_off;
    t.zero_off = t.ct_off + FR * TH * W * COUT * 2;
    t.inv_W = 1.f / float(W); t.inv_TW = 1.f / float(W + 2);
    t.inv_TH = 1.f / float(TH); t.inv_TR = 1.f / float(TH + 2);
    t.PTH = PTH; t.OH = OH; t.OW = OW;
    t.ph = (PH > 0 ? PH : 0) / 2; t.pw = (PW > 0 ? PW : 0) / 2;
    t.inv_OW = 1.f / float(OW); t.inv_ppf = 1.f / float(OH * OW);
    const size_t L = lds(PTH, FR);
    const int groups = cout_total / COUT;
    const void* fn = reinterpret_cast<const void*>(&conv3x3_bf16_kernel<CIN, COUT, MODE, 0, 1, kPoolWaves>);
    int gx = std::max(1, resident_blocks(fn, 64 * kPoolWaves, L) / groups);
    if (gx > t.ntiles) gx = t.ntiles;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(groups));
    ProfScope ps(s, [&] {
        return cb_key("conv_pool", 0, cb_dims(CIN, cout_total) + "/" + cb_dims(H, W) + cb_flags(MODE, false, false));
    });
    hipLaunchKernelGGL((conv3x3_bf16_kernel<CIN, COUT, MODE, 0, 1, kPoolWaves>), grid, dim3(64 * kPoolWaves), L, s, a, t);
    return hipGetLastError();
}

template <class P, int CIN, int COUT, int MODE, int FLIP>
hipError_t launch_split(const ConvArgs& a, hipStream_t s) {
    if constexpr (std::is_same_v<P, PrecBF16> && conv_regw<CIN, COUT, MODE>())
        return launch_regw<CIN, COUT, MODE, FLIP>(a, COUT, s);
    else if constexpr (std::is_same_v<P, PrecBF16>)
        return launch_bf16<CIN, COUT, MODE, FLIP>(a, COUT, s);   // all output channels per workgroup
    else
        return launch<P, CIN, conv_group<P, CIN, COUT>(), MODE, FLIP>(a, COUT, s);
}

template <class P>
hipError_t dispatch(int cin, int cout, int mode, int flip, const ConvArgs& a, hipStream_t s) {
#define CB_CONV(CI, CO, MD, FL)                                                   \
    if (cin == CI && cout == CO && mode == MD && flip == FL)                      \
        return launch_split<P, CI, CO, MD, FL>(a, s);
    // forward: frames -> first stage
    CB_CONV(4, 16, IN_U8, 0) CB_CONV(4, 32, IN_U8, 0) CB_CONV(4, 64, IN_U8, 0)
    // forward: stage entry convs
    CB_CONV(16, 16, IN_PLAIN, 0) CB_CONV(16, 32, IN_PLAIN, 0) CB_CONV(16, 64, IN_PLAIN, 0)
    CB_CONV(32, 32, IN_PLAIN, 0) CB_CONV(32, 64, IN_PLAIN, 0) CB_CONV(64, 64, IN_PLAIN, 0)
    // forward: residual convs read relu(x)
    CB_CONV(16, 16, IN_RELU, 0) CB_CONV(32, 32, IN_RELU, 0) CB_CONV(64, 64, IN_RELU, 0)
    // input gradients (kernel cin = forward cout)
    CB_CONV(16, 16, IN_PLAIN, 1) CB_CONV(32, 16, IN_PLAIN, 1) CB_CONV(64, 16, IN_PLAIN, 1)
    CB_CONV(32, 32, IN_PLAIN, 1) CB_CONV(64, 32, IN_PLAIN, 1) CB_CONV(64, 64, IN_PLAIN, 1)
#undef CB_CONV
    return hipErrorInvalidValue;
}

}  // namespace

static bool ch_ok(int c) { return c == 16 || c == 32 || c == 64; }

// Channels are the forward conv's (cin -> cout) for both directions.
bool conv3x3_supported(int cin, int cout, int mode, int flip) {
    if (flip) return mode == IN_PLAIN && ch_ok(cin) && ch_ok(cout) && cin <= cout;
    if (mode == IN_U8) return cin == 4 && ch_ok(cout);
    if (mode == IN_RELU) return cin == cout && ch_ok(cin);
    return ch_ok(cin) && ch_ok(cout) && cin <= cout;
}

hipError_t conv3x3_pool(int cin, int cout, int mode, const ConvArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    if (conv_pool_fast_supported(cin, cout, mode)) return conv_pool_fast(cin, cout, mode, a, s);
    // all output channels per workgroup from 64 input channels; below that, 16/32-channel
    // groups (measured faster there: the conv tile shares LDS with the weights)
#define CB_CP(CI, CO, MD) \
    if (cin == CI && cout == CO && mode == MD) \
        return launch_bf16_pool<CI, (CI >= 64 ? CO : conv_group<PrecBF16, CI, CO>()), MD>(a, CO, s);
    CB_CP(4, 16, IN_U8) CB_CP(4, 32, IN_U8) CB_CP(4, 64, IN_U8)
    CB_CP(16, 16, IN_PLAIN) CB_CP(16, 32, IN_PLAIN) CB_CP(16, 64, IN_PLAIN)
    CB_CP(32, 32, IN_PLAIN) CB_CP(32, 64, IN_PLAIN) CB_CP(64, 64, IN_PLAIN)
#undef CB_CP
    return hipErrorInvalidValue;
}

hipError_t conv3x3(int prec, int cin, int cout, int mode, int flip, const ConvArgs& a,
                   hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    // flip: kernel in-channels = forward cout; kernel out-channels = forward cin
    const int kin = flip ? cout : cin, kout = flip ? cin : cout;
    return prec == BF16 ? dispatch<PrecBF16>(kin, kout, mode, flip, a, s)
                        : dispatch<PrecF32>(kin, kout, mode, flip, a, s);
}

}  // namespace cb
