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
};

static inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

template <class P, int CIN, int COUT, int MODE>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a, WgRun g_) {
    using T = typename P::T;
    using Frag = typename P::Frag;
    using G = WgGeom<P, CIN, COUT>;
    constexpr int KPL = P::KPL, KSTEP = P::KSTEP;
    constexpr int VEC = MODE == IN_U8 ? 4 : 8;        // channels per global load
    constexpr int NCI = CIN / VEC, NCO = COUT / 8;

    extern __shared__ __align__(16) unsigned char smem[];
    T* xT = reinterpret_cast<T*>(smem);               // [CIN][XP]
    T* gS = xT + CIN * g_.XP;                          // [3][COUT][GP]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TH = g_.TH, PITCH = g_.PITCH, KLEN = g_.KLEN;
    const int XP = g_.XP, GP = g_.GP;

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

    const T* dy = static_cast<const T*>(a.dy);
    for (int ch = blockIdx.x; ch < g_.nchunks; ch += gridDim.x) {
        const int band = ch % g_.nbands, frame = ch / g_.nbands;
        const int h0 = band * TH;
        __syncthreads();   // previous chunk's MFMA reads are done

        // ---- input window, channel-major: xT[ci][r*PITCH + c'] = x[h0 + r - 1][c' - 1][ci]
        for (int e = tid; e < NCI * XP; e += 256) {
            const int cg = e % NCI, kk = e / NCI;
            const int r = kk / PITCH, cc = kk % PITCH;
            const int h = h0 + r - 1, w = cc - 1;
            const bool in = r < TH + 2 && h >= 0 && h < H && w >= 0 && w < W;
            float v[VEC];
            if constexpr (MODE == IN_U8) {
                uint32_t u = 0;
                if (in) {
                    const int64_t row = a.row_idx ? a.row_idx[frame] : frame;
                    u = *reinterpret_cast<const uint32_t*>(static_cast<const uint8_t*>(a.x) +
                                                           ((row * H + h) * W + w) * 4);
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) v[j] = float((u >> (8 * j)) & 0xff);
            } else {
                const T* src = static_cast<const T*>(a.x) + ((int64_t(frame) * H + h) * W + w) * CIN + cg * VEC;
                if constexpr (sizeof(T) == 2) {
                    uint4 u = in ? *reinterpret_cast<const uint4*>(src) : make_uint4(0, 0, 0, 0);
                    const uint32_t* uu = reinterpret_cast<const uint32_t*>(&u);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        v[2 * j] = __uint_as_float(uu[j] << 16);
                        v[2 * j + 1] = __uint_as_float(uu[j] & 0xffff0000u);
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < VEC; ++j) v[j] = in ? src[j] : 0.f;
                }
                if (MODE == IN_RELU) {
#pragma unroll
                    for (int j = 0; j < VEC; ++j) v[j] = relu_f(v[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < VEC; ++j) xT[(cg * VEC + j) * XP + kk] = P::store(v[j]);
        }

        // ---- output gradient, three column-shifted channel-major copies
        for (int e = tid; e < 3 * GP * NCO; e += 256) {
            const int cg = e % NCO, kk = (e / NCO) % GP, kx = e / (NCO * GP);
            const int r = kk / PITCH, w = kk % PITCH - kx;
            const bool in = kk < KLEN && r < TH && h0 + r < H && w >= 0 && w < W;
            float v[8];
            const T* src = dy + ((int64_t(frame) * H + h0 + r) * W + w) * COUT + cg * 8;
            if constexpr (sizeof(T) == 2) {
                uint4 u = in ? *reinterpret_cast<const uint4*>(src) : make_uint4(0, 0, 0, 0);
                const uint32_t* uu = reinterpret_cast<const uint32_t*>(&u);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    v[2 * j] = __uint_as_float(uu[j] << 16);
                    v[2 * j + 1] = __uint_as_float(uu[j] & 0xffff0000u);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) v[j] = in ? src[j] : 0.f;
            }
            if (kx == 0) {
#pragma unroll
                for (int j = 0; j < 8; ++j) bsum[j] += v[j];
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) gS[(kx * COUT + cg * 8 + j) * GP + kk] = P::store(v[j]);
        }
        __syncthreads();

        // ---- MFMA over the band's pixels
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

// Sum the partials of all workgroups in a fixed order and scatter to HWIO / bias.
template <int CIN, int COUT>
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ partial,
                                                           int nparts, float* dw, float* db,
                                                           float scale) {
    using G = WgGeom<PrecF32, CIN, COUT>;
    __shared__ float sh[4][64];
    const int e = blockIdx.x * 64 + (threadIdx.x & 63);
    const int sp = threadIdx.x >> 6;
    float s = 0.f;
    if (e < G::PSTRIDE) {
        for (int p = sp; p < nparts; p += 4) s += partial[int64_t(p) * G::PSTRIDE + e];
    }
    sh[sp][threadIdx.x & 63] = s;
    __syncthreads();
    if (sp == 0 && e < G::PSTRIDE) {
        const float tot = ((sh[0][threadIdx.x] + sh[1][threadIdx.x]) + sh[2][threadIdx.x]) + sh[3][threadIdx.x];
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
    }
}

namespace {

constexpr int kWgradParts = 256;
constexpr size_t kWgLds = 64 * 1024;

template <class P, int CIN, int COUT>
WgRun wg_plan(int n, int H, int W) {
    WgRun r;
    const int es = sizeof(typename P::T);
    r.PITCH = round_up(W + 2, 8);
    int TH = H;
    for (;;) {
        r.TH = TH;
        r.KLEN = round_up(TH * r.PITCH, P::KSTEP);
        r.XP = round_up(r.KLEN + 2 * r.PITCH, 16) + 8;
        r.GP = round_up(r.KLEN, 16) + 8;
        const size_t lds = size_t(CIN * r.XP + 3 * COUT * r.GP) * es;
        if ((lds <= kWgLds && TH * r.PITCH <= 512) || TH == 1) break;
        const int nb = (H + TH - 1) / TH + 1;
        const int next = (H + nb - 1) / nb;
        TH = next < TH ? next : TH - 1;
    }
    r.nbands = (H + r.TH - 1) / r.TH;
    r.nchunks = n * r.nbands;
    return r;
}

template <class P, int CIN, int COUT, int MODE>
hipError_t wg_launch(const WgradArgs& a, hipStream_t s) {
    using G = WgGeom<P, CIN, COUT>;
    const WgRun r = wg_plan<P, CIN, COUT>(a.n, a.H, a.W);
    const int parts = r.nchunks < kWgradParts ? r.nchunks : kWgradParts;
    size_t lds = size_t(CIN * r.XP + 3 * COUT * r.GP) * sizeof(typename P::T);
    if (lds < 256 * 8 * sizeof(float)) lds = 256 * 8 * sizeof(float);
    const int pr = sizeof(typename P::T) == 2 ? 0 : 1;
    const std::string shape = cb_dims(CIN, COUT) + "/" + cb_dims(a.H, a.W);
    {
        ProfScope ps(s, [&] { return cb_key("wgrad", pr, shape); });
        hipLaunchKernelGGL((wgrad_kernel<P, CIN, COUT, MODE>), dim3(parts), dim3(256), lds, s, a, r);
    }
    {
        ProfScope ps(s, [&] { return cb_key("wgrad_reduce", pr, shape); });
        hipLaunchKernelGGL((wgrad_reduce_kernel<CIN, COUT>), dim3((G::PSTRIDE + 63) / 64), dim3(256), 0,
                           s, a.partial, parts, a.dw, a.db, a.scale);
    }
    return hipGetLastError();
}

template <class P>
hipError_t wg_dispatch(int cin, int cout, int mode, const WgradArgs& a, hipStream_t s) {
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

bool wgrad_supported(int cin, int cout, int mode) {
    auto ok = [](int c) { return c == 16 || c == 32 || c == 64; };
    if (mode == IN_U8) return cin == 4 && ok(cout);
    if (mode == IN_RELU) return cin == cout && ok(cin);
    return ok(cin) && ok(cout) && cin <= cout;
}

size_t wgrad_partial_floats(int prec, int cin, int cout, int H, int W) {
    (void)prec; (void)H; (void)W;
    const size_t ncol = size_t(3 * cin + 15) / 16 * 16;
    return size_t(kWgradParts) * (3 * size_t(cout) * ncol + cout);
}

hipError_t conv3x3_wgrad(int prec, int cin, int cout, int mode, const WgradArgs& a,
                         hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    return prec == BF16 ? wg_dispatch<PrecBF16>(cin, cout, mode, a, s)
                        : wg_dispatch<PrecF32>(cin, cout, mode, a, s);
}

}  // namespace cb
