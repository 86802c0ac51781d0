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

// Sum the partials of all workgroups in a fixed order and scatter to HWIO / bias.
// Block: 64 consecutive partial entries x 16 interleaved slices of the partials.
template <int CIN, int COUT>
__global__ __launch_bounds__(1024) void wgrad_reduce_kernel(const float* __restrict__ partial,
                                                            int nparts, float* dw, float* db,
                                                            float scale) {
    using G = WgGeom<PrecF32, CIN, COUT>;
    __shared__ float sh[16][64];
    const int e = blockIdx.x * 64 + (threadIdx.x & 63);
    const int sp = threadIdx.x >> 6;
    float s = 0.f;
    if (e < G::PSTRIDE) {
        for (int p = sp; p < nparts; p += 16) s += partial[int64_t(p) * G::PSTRIDE + e];
    }
    sh[sp][threadIdx.x & 63] = s;
    __syncthreads();
    if (sp == 0 && e < G::PSTRIDE) {
        float tot = 0.f;
#pragma unroll
        for (int k = 0; k < 16; ++k) tot += sh[k][threadIdx.x];
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
    const std::string shape = cb_dims(CIN, COUT) + "/" + cb_dims(a.H, a.W);
    {
        ProfScope ps(s, [&] { return cb_key("wgrad", pr, shape); });
        hipLaunchKernelGGL((wgrad_kernel<P, CIN, COUT, MODE>), dim3(parts), dim3(256), lds, s, a, r);
    }
    {
        ProfScope ps(s, [&] { return cb_key("wgrad_reduce", pr, shape); });
        hipLaunchKernelGGL((wgrad_reduce_kernel<CIN, COUT>), dim3((G::PSTRIDE + 63) / 64), dim3(1024), 0,
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
    const size_t pst = 3 * size_t(cout) * ncol + cout;
    return size_t(wg_parts_cap(int(pst))) * pst;
}

hipError_t conv3x3_wgrad(int prec, int cin, int cout, int mode, const WgradArgs& a,
                         hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    return prec == BF16 ? wg_dispatch<PrecBF16>(cin, cout, mode, a, s)
                        : wg_dispatch<PrecF32>(cin, cout, mode, a, s);
}

}  // namespace cb
