// A stage's entry of Section 5's IMPALA-ResNet in one kernel (bf16): 3x3 SAME convolution,
// then 3x3 stride-2 SAME max-pool with XLA's padding split, keeping only the pooled map and
// its argmax (the full-resolution conv output never reaches HBM).
//
// A tile is a band of pooled rows of one frame; it needs conv rows hc0 .. hc1-1 and input
// rows hc0-1 .. hc1. Staged in LDS: the zero-padded input window (uint8 frames as bytes,
// then converted once to bf16, exact for 0..255; bf16 inputs as C/8 16-byte slots per pixel
// plus, from 32 channels on, two zero slots), with a zero guard pixel either side. The conv
// runs over the window's pixels padding columns included, 16 per MFMA column tile, so a
// fragment's address is the tile base plus a constant per k-step and the lane only tracks
// its column to skip the padding outputs. Each wave owns one 16-channel block of the outputs with its weight
// fragments in registers. Conv outputs (scale, bias, rounded to bf16) are kept as
// order-preserving 16-bit keys in an LDS tile whose padding columns stay zero (a zero key is
// below every finite value, so padding never wins). The pool compares (key << 16 | 15 - cell)
// as integers: the largest key wins and, among equal keys, the first cell in row-major
// window order.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace cb {

template <int CIN, int COUT, int MODE>
struct CpGeom {
    static constexpr bool U8 = MODE == IN_U8;
    // bf16 input: 16-byte slots per pixel. A 16-lane B-fragment read on consecutive window
    // pixels lands on distinct bank groups when the pitch is 2 (mod 4) slots: 16 channels fill
    // 2, from 32 on two zero slots are added (6, 10)
    static constexpr int SPP = U8 ? 1 : (CIN >= 32 ? CIN / 8 + 2 : CIN / 8);
    static constexpr int PB = U8 ? 8 : SPP * 16;           // window bytes per pixel
    static constexpr int K = 9 * CIN, KSTEPS = (K + 31) / 32;
    static constexpr int MT = COUT / 16;
    static constexpr int KPB = COUT * 2 + 16;              // key-tile bytes per pixel (odd slots)
    static constexpr int C8 = COUT / 8;
    static constexpr int MAXS = 6;                         // input staging slots per lane
    // 64 input channels: the weight fragments (72 registers) take the registers of two waves
    // per SIMD, so one workgroup per CU with most of the LDS; otherwise four waves per SIMD
    static constexpr int WPS = CIN >= 64 ? 2 : 4;
    static constexpr size_t LDS_TARGET = CIN >= 64 ? 150 * 1024 : 80 * 1024;
};

template <int CIN, int COUT, int MODE, int NW>
__global__ __launch_bounds__(64 * NW, (CpGeom<CIN, COUT, MODE>::WPS)) void conv_pool_kernel(ConvArgs a, CpTile t) {
    using G = CpGeom<CIN, COUT, MODE>;
    constexpr int NT = 64 * NW, KSTEPS = G::KSTEPS, MT = G::MT, PB = G::PB, KPB = G::KPB, C8 = G::C8;
    constexpr bool U8 = G::U8;
    static_assert(!U8 || CIN == 4, "uint8 frames carry 4 stacked channels");
    static_assert(NW % MT == 0, "waves split evenly over the output channel blocks");

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;                     // 64 zero bytes
    unsigned char* raw = smem + t.raw_off;          // uint8 frames: [TR][TW] x 4
    unsigned char* win = smem + t.win_off + PB;     // [TR][TW] x PB, a zero guard pixel either side
    unsigned char* keys = smem + t.key_off;         // [THmax][TW] x KPB

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TW = W + 2, TRM = t.THmax + 2;
    const int mt = wave % MT, co0 = mt * 16 + g * 4;

    // ---- weight fragments of this wave's output block: A[o][k] = w[k*COUT + o] (HWIO, k =
    // tap*CIN + i), zero past the 9 taps; biases of the lane's four output channels
    uint4 wr[KSTEPS];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int k = ks * 32 + g * 8 + j;
            v[j] = k < G::K ? a.w[k * COUT + mt * 16 + r16] : 0.f;
        }
        wr[ks] = make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]), pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
    }
    float bias[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) bias[j] = a.bias ? a.bias[co0 + j] : 0.f;
    // B-fragment offsets from the lane's tap-(0,0) pixel. uint8: k-step 0 holds taps 2g, 2g+1
    // (4 channels each), k-step 1 tap 8 (its other k have zero weights, so any finite value
    // serves); 16 channels: a k-step spans two taps (table; past the ninth, zeros);
    // 32: the k-step's tap, the lane's slot
    auto tapoff = [&](int tap) { return ((tap / 3) * TW + tap % 3) * PB; };
    int boff[U8 ? 3 : (CIN < 32 ? KSTEPS : 1)];
    if constexpr (U8) {
        boff[0] = tapoff(2 * g); boff[1] = tapoff(2 * g + 1); boff[2] = tapoff(8);
    } else if constexpr (CIN < 32) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / CIN, c = (k0 % CIN) / 8;
            boff[ks] = tap < 9 ? tapoff(tap) + c * 16 : 0;   // past the taps: zeroed below
        }
    }
    const int twpb = TW * PB;
    auto bfrag = [&](const unsigned char* xb, int ks) -> uint4 {
        if constexpr (U8) {
            if (ks == 0) {
                const uint2 lo = *reinterpret_cast<const uint2*>(xb + boff[0]);
                const uint2 hi = *reinterpret_cast<const uint2*>(xb + boff[1]);
                return make_uint4(lo.x, lo.y, hi.x, hi.y);
            }
            // tap 8 and the next pixel (a finite value against zero weights; the window ends
            // in a guard pixel)
            const uint2 t8 = *reinterpret_cast<const uint2*>(xb + boff[2]);
            const uint2 t9 = *reinterpret_cast<const uint2*>(xb + boff[2] + 8);
            return make_uint4(t8.x, t8.y, t9.x, t9.y);
        } else if constexpr (CIN < 32) {
            // 16 channels: lanes g >= 2 of the last k-step are past the 9 taps
            const uint4 v = *reinterpret_cast<const uint4*>(xb + boff[ks]);
            return ks == KSTEPS - 1 && g >= 2 ? make_uint4(0, 0, 0, 0) : v;
        } else {   // from 32 channels a tap spans CIN / 32 k-steps; the lane's slot within it
            constexpr int TPK = CIN / 32;
            const int tap = ks / TPK, cs = (ks % TPK) * 4;
            return *reinterpret_cast<const uint4*>(xb + (tap / 3) * twpb + (tap % 3) * PB + (cs + g) * 16);
        }
    };

    // ---- zero once: the zero area, the window guards, the key tile (padding columns stay 0)
    if (tid < 16) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;
    if (tid < PB / 4) {
        reinterpret_cast<uint32_t*>(win - PB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(win + t.win_guard)[tid] = 0u;
    }
    for (int j = tid; j < t.THmax * TW * KPB / 16; j += NT) reinterpret_cast<uint4*>(keys)[j] = make_uint4(0, 0, 0, 0);

    // ---- input staging offsets, tile-invariant per lane (slot k of this wave:
    // j = (wave + NW*k)*64 + lane), relative to window row 1 at image row 0; a tile adds hc0
    // rows. Rows off the frame fall outside the frame's buffer resource and read zero.
    const int ns = U8 ? TRM * TW : TRM * TW * G::SPP;
    uint32_t ox[G::MAXS];
#pragma unroll
    for (int k = 0; k < G::MAXS; ++k) {
        const int j = (wave + NW * k) * 64 + lane;
        if constexpr (U8) {
            const int rr = j / TW, col = j - rr * TW;
            ox[k] = (j < ns && col >= 1 && col <= W) ? uint32_t(((rr - 1) * W + col - 1) * 4) : kOOB;
        } else {
            const int p = j / G::SPP, c = j - p * G::SPP, rr = p / TW, col = p - rr * TW;
            ox[k] = (j < ns && c < CIN / 8 && col >= 1 && col <= W)
                        ? uint32_t((((rr - 1) * W + col - 1) * CIN + c * 8) * 2) : kOOB;
        }
    }
    __syncthreads();

    int lg = blockIdx.x;   // neighbouring bands on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    // input window of a tile, image rows hc0-1 .. hc0+THmax (uint8 frames: the raw bytes). The
    // next tile's window is issued as soon as the conv has read this one, so its latency
    // overlaps the max-pool.
    unsigned char* const sdst = U8 ? raw : win;
    auto stage = [&](unsigned char* dst, int tile) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int hc0 = max(2 * band * t.PTH - t.ph, 0);
        if constexpr (U8) {
            const int64_t row = a.row_idx ? a.row_idx[f] : f;
            const uint32_t fb = uint32_t(H) * W * 4;
            const auto rx = buf_rsrc(static_cast<const uint8_t*>(a.x) + row * fb, fb);
            const uint32_t hr = uint32_t(hc0 * W * 4);
#pragma unroll
            for (int k = 0; k < G::MAXS; ++k)
                if ((wave + NW * k) * 64 < ns) dma4_to_lds(rx, dst + (wave + NW * k) * 256, ox[k] + hr);
        } else {
            const uint32_t fb = uint32_t(H) * W * CIN * 2;
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + int64_t(f) * H * W * CIN, fb);
            const uint32_t hr = uint32_t(hc0 * W * CIN * 2);
#pragma unroll
            for (int k = 0; k < G::MAXS; ++k)
                if ((wave + NW * k) * 64 < ns) dma16_to_lds(rx, dst + (wave + NW * k) * 1024, ox[k] + hr);
        }
    };
    if (lg < t.ntiles) stage(sdst, lg);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int p0 = band * t.PTH, p1 = min(p0 + t.PTH, t.OH);
        const int hc0 = max(2 * p0 - t.ph, 0), hc1 = min(2 * (p1 - 1) - t.ph + 3, H);
        const int TH = hc1 - hc0;
        __builtin_amdgcn_s_waitcnt(0);   // this tile's window has landed
        __syncthreads();                 // ... everyone's, and the previous max-pool is done
        if constexpr (U8) {
            for (int p = tid; p < ns; p += NT)
                *reinterpret_cast<uint2*>(win + p * 8) = u8x4_to_bf16(*reinterpret_cast<const uint32_t*>(raw + p * 4));
            __syncthreads();
        }

        // ---- conv over window pixels p in [TW, (TH+1)*TW): output (image row hc0 + p/TW - 1,
        // column p%TW - 1), tap (0,0) at window pixel p - TW - 1; its key at key-tile pixel
        // p - TW. The padding columns get keys too (of wrapped windows); they are zeroed after.
        {
            constexpr int STEP = NW / MT;               // column tiles between a wave's passes
            const int S = 16 * STEP;                    // pixels per pass
            const int pend = (TH + 1) * TW;
            int p = TW + (wave / MT) * 16 + r16;
            const unsigned char* xb = win + (p - TW - 1) * PB;
            unsigned char* kp = keys + (p - TW) * KPB + co0 * 2;
            auto put = [&](const cb_f32x4& acc, unsigned char* k) {
                const uint32_t u0 = pack2bf(acc[0] * a.scale + bias[0], acc[1] * a.scale + bias[1]);
                const uint32_t u1 = pack2bf(acc[2] * a.scale + bias[2], acc[3] * a.scale + bias[3]);
                *reinterpret_cast<uint2*>(k) = make_uint2(bf16x2_key(u0), bf16x2_key(u1));
            };
            if constexpr (U8) {
                // two column tiles per pass, so that each one's fragment reads and MFMAs overlap
                // the other's (a missing second tile repeats the first and is not stored)
                for (int nt = wave / MT; nt * 16 < TH * TW; nt += 2 * STEP) {
                    const bool two = (nt + STEP) * 16 < TH * TW;
                    const unsigned char* xb2 = two ? xb + S * PB : xb;
                    cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f}, acc2 = acc;
#pragma unroll
                    for (int ks = 0; ks < KSTEPS; ++ks) {
                        acc = PrecBF16::mma(wr[ks], bfrag(xb, ks), acc);
                        acc2 = PrecBF16::mma(wr[ks], bfrag(xb2, ks), acc2);
                    }
                    if (p < pend) put(acc, kp);
                    if (two && p + S < pend) put(acc2, kp + S * KPB);
                    p += 2 * S; xb += 2 * S * PB; kp += 2 * S * KPB;
                }
            } else {
                for (int nt = wave / MT; nt * 16 < TH * TW; nt += STEP) {
                    cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KSTEPS; ++ks) acc = PrecBF16::mma(wr[ks], bfrag(xb, ks), acc);
                    if (p < pend) put(acc, kp);
                    p += S; xb += S * PB; kp += S * KPB;
                }
            }
        }
        __syncthreads();   // the conv has read the window (the next tile's may land there) and
                           // written the key tile
        // the key tile's padding columns back to zero keys (below every value)
        for (int j = tid; j < TH * 2 * C8; j += NT) {
            const int c8 = j % C8, e = j / C8, row = e >> 1;
            *reinterpret_cast<uint4*>(keys + (row * TW + (e & 1) * (TW - 1)) * KPB + c8 * 16) = make_uint4(0, 0, 0, 0);
        }
        __syncthreads();

        // ---- next tile's window, then the 3x3 stride-2 max-pool of the key tile, 8 channels per
        // item. The window and the key tile are restrict parameters of one call, so the compiler
        // knows that the loads in flight do not write what the max-pool reads.
        auto stage_pool = [&](unsigned char* __restrict__ dst, const unsigned char* __restrict__ kt,
                              const unsigned char* __restrict__ zr) {
            if (tile + int(gridDim.x) < t.ntiles) stage(dst, tile + gridDim.x);
            {
                const int prows = p1 - p0, items = prows * t.OW * C8;
                uint16_t* ybase = static_cast<uint16_t*>(a.y) + (int64_t(f) * t.OH + p0) * t.OW * COUT;
                uint8_t* abase = a.arg + (int64_t(f) * t.OH + p0) * t.OW * COUT;
                for (int it = tid; it < items; it += NT) {
                    const int c8 = it % C8, pp = it / C8;
                    const int ohl = qdiv(pp, t.inv_OW), ow = pp - ohl * t.OW;
                    const int hc = 2 * (p0 + ohl) - t.ph, wc = 2 * ow - t.pw;
                    // window cell (dy, dx): key-tile row hc + dy - hc0, column wc + dx + 1 (the
                    // padding columns hold zero keys); rows off the frame read the zero area
                    const unsigned char* kb = kt + ((hc - hc0) * TW + wc + 1) * KPB + c8 * 16;
                    const bool rv[3] = {hc >= 0, true, hc + 2 < H};
                    uint4 cell[9];
#pragma unroll
                    for (int dy = 0; dy < 3; ++dy)
#pragma unroll
                        for (int dx = 0; dx < 3; ++dx)
                            cell[dy * 3 + dx] = *reinterpret_cast<const uint4*>(rv[dy] ? kb + (dy * TW + dx) * KPB : zr);
                    uint32_t best[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) best[j] = 0u;
#pragma unroll
                    for (int cidx = 0; cidx < 9; ++cidx) {
                        const uint32_t tag = 15u - uint32_t(cidx);
                        const uint32_t kk[4] = {cell[cidx].x, cell[cidx].y, cell[cidx].z, cell[cidx].w};
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            best[2 * j] = max(best[2 * j], (kk[j] << 16) | tag);
                            best[2 * j + 1] = max(best[2 * j + 1], (kk[j] & 0xffff0000u) | tag);
                        }
                    }
                    uint32_t vals[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        vals[j] = bf16x2_unkey((best[2 * j] >> 16) | (best[2 * j + 1] & 0xffff0000u));
                    uint32_t idx[2] = {0u, 0u};
#pragma unroll
                    for (int j = 0; j < 8; ++j) idx[j >> 2] |= (15u - (best[j] & 15u)) << (8 * (j & 3));
                    const uint32_t o = (uint32_t(ohl) * t.OW + ow) * COUT + c8 * 8;
                    *reinterpret_cast<uint4*>(ybase + o) = make_uint4(vals[0], vals[1], vals[2], vals[3]);
                    *reinterpret_cast<uint2*>(abase + o) = make_uint2(idx[0], idx[1]);
                }
            }
        };
        stage_pool(sdst, keys, zero);
    }
}

namespace {

constexpr int kCpWaves = 8;
constexpr int kCpPixMax = 4096;

template <int CIN, int COUT, int MODE>
hipError_t cp_launch(const ConvArgs& a, hipStream_t s) {
    using G = CpGeom<CIN, COUT, MODE>;
    const int H = a.H, W = a.W, TW = W + 2;
    const int OH = (H + 1) / 2, OW = (W + 1) / 2;
    const int PH = (OH - 1) * 2 + 3 - H, PWd = (OW - 1) * 2 + 3 - W;
    const int ph = (PH > 0 ? PH : 0) / 2, pw = (PWd > 0 ? PWd : 0) / 2;
    auto thmax = [&](int pth) { return std::min(2 * pth + 1, H); };
    auto layout = [&](int pth, CpTile& t) {
        const int trm = thmax(pth) + 2;
        const int ns = G::U8 ? trm * TW : trm * TW * G::SPP;
        t.raw_off = 64;
        t.win_off = t.raw_off + (G::U8 ? (ns + 63) / 64 * 256 : 0);
        const int winb = G::U8 ? ns * 8 : (ns + 63) / 64 * 1024;
        t.win_guard = G::U8 ? trm * TW * 8 : winb;   // the rear guard, from the window start
        t.key_off = t.win_off + (G::PB + std::max(winb, t.win_guard) + G::PB + 15) / 16 * 16;
        return size_t(t.key_off) + size_t(thmax(pth)) * TW * G::KPB;
    };
    auto fits = [&](int pth) {
        const int trm = thmax(pth) + 2, per = kCpWaves * 64;
        const int ns = G::U8 ? trm * TW : trm * TW * G::SPP;
        return (ns + per - 1) / per <= G::MAXS && thmax(pth) * W <= kCpPixMax;
    };
    CpTile t{};
    int pmax = OH;
    while (pmax > 1 && (layout(pmax, t) > G::LDS_TARGET || !fits(pmax))) --pmax;
    if (layout(pmax, t) > std::min<size_t>(lds_limit(), 160 * 1024) || !fits(pmax)) return hipErrorInvalidValue;
    if (int64_t(H) * W * std::max(CIN, 2) * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    const int nb0 = (OH + pmax - 1) / pmax;
    const int PTH = (OH + nb0 - 1) / nb0;   // balanced bands
    const size_t L = layout(PTH, t);
    t.PTH = PTH; t.nbands = (OH + PTH - 1) / PTH; t.ntiles = t.nbands * a.n;
    t.OH = OH; t.OW = OW; t.ph = ph; t.pw = pw; t.THmax = thmax(PTH);
    t.inv_OW = 1.f / float(OW);
    const void* fn = reinterpret_cast<const void*>(&conv_pool_kernel<CIN, COUT, MODE, kCpWaves>);
    int gx = std::max(1, resident_blocks(fn, 64 * kCpWaves, L));
    if (gx > t.ntiles) gx = t.ntiles;
    ProfScope ps(s, [&] {
        return cb_key("conv_pool", 0, cb_dims(CIN, COUT) + "/" + cb_dims(H, W) + cb_flags(MODE, false, false));
    });
    hipLaunchKernelGGL((conv_pool_kernel<CIN, COUT, MODE, kCpWaves>), dim3(unsigned(gx)), dim3(64 * kCpWaves), L, s, a,
                       t);
    return hipGetLastError();
}

}  // namespace

bool conv_pool_fast_supported(int cin, int cout, int mode) {
    if (mode == IN_U8) return cin == 4 && (cout == 16 || cout == 32);
    return mode == IN_PLAIN && ((cin == 16 && (cout == 16 || cout == 32)) || (cin == 32 && (cout == 32 || cout == 64)) ||
                                (cin == 64 && cout == 64));
}

hipError_t conv_pool_fast(int cin, int cout, int mode, const ConvArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
#define CB_CPF(CI, CO, MD) \
    if (cin == CI && cout == CO && mode == MD) return cp_launch<CI, CO, MD>(a, s);
    CB_CPF(4, 16, IN_U8) CB_CPF(4, 32, IN_U8) CB_CPF(16, 16, IN_PLAIN) CB_CPF(16, 32, IN_PLAIN) CB_CPF(32, 32, IN_PLAIN)
    CB_CPF(32, 64, IN_PLAIN) CB_CPF(64, 64, IN_PLAIN)
#undef CB_CPF
    return hipErrorInvalidValue;
}

}  // namespace cb
