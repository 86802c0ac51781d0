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

template <class P, int CIN, int COUT, int MODE, int FLIP>
__global__ __launch_bounds__(256) void conv3x3_kernel(ConvArgs a, int TH, int FR, int nbands,
                                                      int cout_total) {
    using T = typename P::T;
    using G = ConvGeom<P, CIN>;
    using Frag = typename P::Frag;
    constexpr int KPL = P::KPL, KSTEP = P::KSTEP, KSTEPS = G::KSTEPS, KP = G::KP;
    constexpr int KPITCH = G::KPITCH, CP = G::CP, MT = COUT / 16;
    static_assert(MODE != IN_U8 || CIN == 4, "uint8 frames carry 4 stacked channels");
    static_assert(COUT % 16 == 0, "output channels in 16-wide MFMA tiles");

    extern __shared__ __align__(16) unsigned char smem[];
    T* wl = reinterpret_cast<T*>(smem);
    constexpr int WL_ELEMS = ((COUT * KPITCH) + 7) / 8 * 8;
    T* xs = wl + WL_ELEMS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int band = blockIdx.x % nbands, fg = blockIdx.x / nbands;
    const int og = blockIdx.y * COUT;                  // first output channel of this group
    const int H = a.H, W = a.W;
    const int h0 = band * TH, f0 = fg * FR;
    const int TW = W + 2, TR = TH + 2;

    // ---- weights -> LDS: wl[o][tap*CIN + i], zero in the k padding
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

    // ---- zero-padded input window -> LDS: xs[f][r][c][i]
    const int npix = FR * TR * TW;
    if constexpr (MODE == IN_U8) {
        const uint8_t* obs = static_cast<const uint8_t*>(a.x);
        for (int p = tid; p < npix; p += 256) {
            const int col = p % TW, rr = (p / TW) % TR, f = p / (TW * TR);
            const int h = h0 + rr - 1, w = col - 1, frame = f0 + f;
            uint32_t v = 0;
            if (h >= 0 && h < H && w >= 0 && w < W && frame < a.n) {
                const int64_t row = a.row_idx ? a.row_idx[frame] : frame;
                v = *reinterpret_cast<const uint32_t*>(obs + ((row * H + h) * W + w) * 4);
            }
            T* dst = xs + p * CP;
            if constexpr (sizeof(T) == 2) {
                const uint32_t lo = pack2bf(float(v & 0xff), float((v >> 8) & 0xff));
                const uint32_t hi = pack2bf(float((v >> 16) & 0xff), float(v >> 24));
                *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
            } else {
                dst[0] = float(v & 0xff); dst[1] = float((v >> 8) & 0xff);
                dst[2] = float((v >> 16) & 0xff); dst[3] = float(v >> 24);
            }
        }
    } else {
        constexpr int VEC = sizeof(T) == 2 ? 8 : 4;   // channels per 16-byte chunk
        constexpr int NCH = CIN / VEC;
        const T* x = static_cast<const T*>(a.x);
        for (int e = tid; e < npix * NCH; e += 256) {
            const int ch = e % NCH, p = e / NCH;
            const int col = p % TW, rr = (p / TW) % TR, f = p / (TW * TR);
            const int h = h0 + rr - 1, w = col - 1, frame = f0 + f;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (h >= 0 && h < H && w >= 0 && w < W && frame < a.n)
                v = *reinterpret_cast<const uint4*>(x + ((int64_t(frame) * H + h) * W + w) * CIN + ch * VEC);
            T* dst = xs + p * CP + ch * VEC;
            if constexpr (sizeof(T) == 2) {
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
    __syncthreads();

    // ---- MFMA main loop over 16-pixel tiles
    const int g = lane >> 4, r16 = lane & 15;
    const int npx = FR * TH * W;
    const int ntiles = (npx + 15) / 16;

    // Per-lane LDS offset of its B fragment within the 3x3 window, per k-step.
    auto b_off = [&](int ks, int half) -> int {
        // k of this lane's first element (for CIN == 4 bf16: each half covers one tap)
        const int k0 = ks * KSTEP + g * KPL + half * 4;
        const int tap = k0 / CIN, i = k0 % CIN;
        if (tap >= 9) return -1;
        return ((tap / 3) * TW + (tap % 3)) * CP + i;
    };

    for (int nt = wave; nt < ntiles; nt += 4) {
        const int q = nt * 16 + r16;
        const int qc = q < npx ? q : npx - 1;
        const int c = qc % W, rr = (qc / W) % TH, f = qc / (W * TH);
        const T* xb = xs + ((f * TR + rr) * TW + c) * CP;
        cb_f32x4 acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = cb_f32x4{0.f, 0.f, 0.f, 0.f};

        if constexpr (sizeof(T) == 2) {
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
                    const Frag af = P::lds_frag(wl + (mt * 16 + r16) * KPITCH + ks * KSTEP + g * KPL);
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

// ------------------------------------------------------------------ launcher

namespace {

// Tiles aim at 64 KB of LDS (two or more workgroups per CU); layers whose weights alone
// need more may use up to the device's per-workgroup maximum.
constexpr size_t kLdsTarget = 64 * 1024;

template <class P, int CIN, int COUT>
size_t conv_lds_bytes(int TH, int FR, int W) {
    using G = ConvGeom<P, CIN>;
    const size_t wl = (size_t(COUT) * G::KPITCH + 7) / 8 * 8;
    return (wl + size_t(FR) * (TH + 2) * (W + 2) * G::CP) * sizeof(typename P::T);
}

template <class P, int CIN, int COUT, int MODE, int FLIP>
hipError_t launch(const ConvArgs& a, int cout_total, hipStream_t s) {
    // Tile: about 512 output pixels per workgroup, bands of equal height, within the LDS budget.
    const int H = a.H, W = a.W;
    int TH, FR = 1;
    if (H * W >= 512) {
        const int target = (512 + W - 1) / W;
        const int nb = (H + target - 1) / target;
        TH = (H + nb - 1) / nb;
    } else {
        TH = H;
        FR = 512 / (H * W);
        if (FR < 1) FR = 1;
        if (FR > a.n) FR = a.n;
    }
    const size_t budget = std::max(kLdsTarget, std::min<size_t>(lds_limit(), 160 * 1024));
    while (conv_lds_bytes<P, CIN, COUT>(TH, FR, W) > (FR > 1 || TH > 4 ? kLdsTarget : budget)) {
        if (FR > 1) --FR;
        else if (TH > 1) {
            const int nb = (H + TH - 1) / TH + 1;
            const int next = (H + nb - 1) / nb;
            TH = next < TH ? next : TH - 1;
        }
        else return hipErrorInvalidValue;
    }
    const int nbands = (H + TH - 1) / TH;
    const int nfg = (a.n + FR - 1) / FR;
    const size_t lds = conv_lds_bytes<P, CIN, COUT>(TH, FR, W);
    dim3 grid(unsigned(nbands * nfg), unsigned(cout_total / COUT));
    ProfScope ps(s, [&] {
        return cb_key(FLIP ? "conv_dgrad" : "conv_fwd", sizeof(typename P::T) == 2 ? 0 : 1,
                      cb_dims(CIN, cout_total) + "/" + cb_dims(H, W));
    });
    hipLaunchKernelGGL((conv3x3_kernel<P, CIN, COUT, MODE, FLIP>), grid, dim3(256), lds, s, a, TH,
                       FR, nbands, cout_total);
    return hipGetLastError();
}

// Output channels per workgroup: all of them unless the weight tile would crowd LDS.
template <class P, int CIN, int COUT>
constexpr int conv_group() {
    int cg = COUT;
    while (cg > 16 && cg * ConvGeom<P, CIN>::KPITCH * int(sizeof(typename P::T)) > 24 * 1024) cg /= 2;
    return cg;
}

template <class P, int CIN, int COUT, int MODE, int FLIP>
hipError_t launch_split(const ConvArgs& a, hipStream_t s) {
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

hipError_t conv3x3(int prec, int cin, int cout, int mode, int flip, const ConvArgs& a,
                   hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    // flip: kernel in-channels = forward cout; kernel out-channels = forward cin
    const int kin = flip ? cout : cin, kout = flip ? cin : cout;
    return prec == BF16 ? dispatch<PrecBF16>(kin, kout, mode, flip, a, s)
                        : dispatch<PrecF32>(kin, kout, mode, flip, a, s);
}

}  // namespace cb
