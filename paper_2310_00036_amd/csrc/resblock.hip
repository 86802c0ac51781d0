// A whole IMPALA-ResNet residual block in one kernel (bf16 forward):
//
//   t = conv1(relu(x)) + b1,   y = x + conv2(relu(t)) + b2     (3x3 SAME convolutions, C -> C)
//
// Layer by layer the block moves five activation tensors through HBM (x for conv1; t, x and y
// for conv2; t written once); here it moves three (x read, t and y written). Each tile is a
// band of TH output rows of one frame:
//   - the input window, rows h0-2 .. h0+TH+1 of x, is staged HBM -> LDS (buffer loads, zero
//     padding from out-of-range offsets) and ReLU'd in place;
//   - conv1 computes t on the band's rows plus one halo row above and below (the halo rows
//     are recomputed by the neighbouring bands); t is rounded to bf16, the band's own rows
//     are stored (the backward pass reads them) and relu(t) goes to an LDS window with zero
//     padding columns, exactly what conv2 would have read from HBM;
//   - conv2 reads that window and writes y with the bias and the residual add fused; the
//     residual x comes from global memory into registers, fetched with the tile's staging.
// Per MFMA: 16 output pixels per column tile, one 16-byte B fragment per lane and k-step
// from a window whose pixels are C/8 16-byte slots plus one zero slot (an odd slot count
// spreads a fragment read over the banks; the zero slot feeds k-steps past the 9 taps).
// Each wave owns one 16-channel block of the outputs and holds both convolutions' A
// fragments for it in registers, loaded once per workgroup, so LDS holds only the windows.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace cb {

template <int C>
struct RbGeom {
    static constexpr int K = 9 * C;
    static constexpr int KSTEPS = (K + 31) / 32;
    static constexpr int MT = C / 16;
    static constexpr int SPP = C / 8 + 1;                  // 16-byte slots per window pixel
    static constexpr int PB = SPP * 16;
    // Workgroup shape: 16 channels hold both weight sets in 8-wave workgroups at 4 waves per
    // SIMD (128 registers); 32 channels need about 170 registers, so 4-wave workgroups at 3
    // waves per SIMD (three workgroups per CU) instead of spilling.
    static constexpr int NW = C >= 32 ? 4 : 8;
    static constexpr int WPS = C >= 32 ? 3 : 4;            // waves per SIMD (register budget)
    static constexpr int WGS = WPS * 4 / NW;               // workgroups per CU
    static constexpr int MAXS = C >= 32 ? 8 : 5;           // x-window staging slots per lane
    // conv2 column tiles per wave and tile whose residual is fetched with the staging (with 32
    // channels the registers hold both weight sets, and the residual is read per column tile)
    static constexpr int MAXT = C >= 32 ? 0 : 5;
    __host__ __device__ static int blocks(int slots) { return (slots + 63) / 64; }
    __host__ __device__ static int xwin_bytes(int TH, int W) { return blocks((TH + 4) * (W + 2) * SPP) * 1024; }
    __host__ __device__ static int twin_bytes(int TH, int W) { return ((TH + 2) * (W + 2) * PB + 15) / 16 * 16; }
};

struct RbTile {
    int TH, nbands, ntiles;
    int x_off, t_off;   // LDS byte offsets of the two windows
    float inv_W, inv_TW;
};

template <int C, int NW>
__global__ __launch_bounds__(64 * NW, RbGeom<C>::WPS) void resblock_fwd_kernel(ResBlockArgs a, RbTile t) {
    using G = RbGeom<C>;
    constexpr int NT = 64 * NW, KSTEPS = G::KSTEPS, MT = G::MT, SPP = G::SPP, PB = G::PB;
    static_assert(NW % MT == 0, "waves split evenly over the output channel blocks");

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* xw = smem + t.x_off;   // relu(x) window [TH+4][W+2] pixels
    unsigned char* tw = smem + t.t_off;   // relu(t) window [TH+2][W+2] pixels

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TH = t.TH, TW = W + 2;
    const int mt = wave % MT;                     // this wave's output channel block
    const int co0 = mt * 16 + g * 4;              // the lane's first output channel

    // ---- A fragments of both convolutions for rows mt*16 .. +15: A[o][k] = w[tap][i][o]
    // with k = tap*C + i (zero past the 9 taps); biases of the lane's four output channels
    uint4 wr1[KSTEPS], wr2[KSTEPS];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
        const int o = mt * 16 + r16;
        float v1[8], v2[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int k = ks * 32 + g * 8 + j;
            v1[j] = k < G::K ? a.w1[k * C + o] : 0.f;
            v2[j] = k < G::K ? a.w2[k * C + o] : 0.f;
        }
        wr1[ks] = make_uint4(pack2bf(v1[0], v1[1]), pack2bf(v1[2], v1[3]), pack2bf(v1[4], v1[5]), pack2bf(v1[6], v1[7]));
        wr2[ks] = make_uint4(pack2bf(v2[0], v2[1]), pack2bf(v2[2], v2[3]), pack2bf(v2[4], v2[5]), pack2bf(v2[6], v2[7]));
        __builtin_amdgcn_sched_barrier(0);   // convert each k-step's weights before loading the next
    }
    float b1[4], b2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        b1[j] = a.b1 ? a.b1[co0 + j] : 0.f;
        b2[j] = a.b2 ? a.b2[co0 + j] : 0.f;
    }
    // per-lane B-fragment offsets from the tap-(0,0) pixel (both windows share the pitch);
    // only 16 channels need the table (a k-step spans two taps)
    int boff[C < 32 ? KSTEPS : 1];
    if constexpr (C < 32) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / C, c = (k0 % C) / 8;
            boff[ks] = tap < 9 ? ((tap / 3) * TW + tap % 3) * PB + c * 16 : (SPP - 1) * 16;
        }
    }
    const int twpb = TW * PB;
    auto mma = [&](const unsigned char* xb, const uint4* wr) {
        cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const int bo = C < 32 ? boff[ks] : (ks / 3) * twpb + (ks % 3) * PB + g * 16;
            acc = PrecBF16::mma(wr[ks], *reinterpret_cast<const uint4*>(xb + bo), acc);
            // with both weight sets held, keep at most three B fragments in flight
            if (C >= 32 && ks % 3 == 2) __builtin_amdgcn_sched_barrier(0);
        }
        return acc;
    };

    // ---- relu(t) window zeroed once (its padding columns and zero slots are never written)
    for (int j = tid; j < G::twin_bytes(TH, W) / 16; j += NT) reinterpret_cast<uint4*>(tw)[j] = make_uint4(0, 0, 0, 0);

    // ---- x-window staging offsets, tile-invariant per lane (slot k of this wave:
    // j = (wave + NW*k)*64 + lane), relative to image row 0; a tile adds h0 - 2 rows. Rows
    // off the frame fall outside the frame's buffer resource (negative, or past its end).
    const int nsx = (TH + 4) * TW * SPP;
    uint32_t ox[G::MAXS];
#pragma unroll
    for (int k = 0; k < G::MAXS; ++k) {
        const int j = (wave + NW * k) * 64 + lane, p = j / SPP, c = j - p * SPP;
        const int rr = p / TW, col = p - rr * TW;
        ox[k] = (j < nsx && c < SPP - 1 && col >= 1 && col <= W) ? uint32_t(((rr * W + col - 1) * C + c * 8) * 2)
                                                                   : kOOB;
    }
    __syncthreads();

    int lg = blockIdx.x;   // neighbouring bands on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    // x window of a tile, rows h0-2 .. h0+TH+1. The next tile's window is issued as soon as
    // conv1 has finished reading this one, so its latency overlaps conv2.
    auto stage_x = [&](int tile) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + int64_t(f) * H * W * C, uint32_t(H) * W * C * 2);
        const uint32_t hr = uint32_t((band * TH - 2) * W * C * 2);   // wraps for h0 < 2: rows off the frame
#pragma unroll
        for (int k = 0; k < G::MAXS; ++k)
            if ((wave + NW * k) * 64 < nsx) dma16_to_lds(rx, xw + (wave + NW * k) * 1024, ox[k] + hr);
    };
    if (lg < t.ntiles) stage_x(lg);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int h0 = band * TH, the = H - h0 < TH ? H - h0 : TH;
        const int64_t fo = int64_t(f) * H * W * C;   // frame offset (elements)
        // conv2's residual x for this wave's column tiles, fetched alongside the staging
        const uint16_t* xbase = static_cast<const uint16_t*>(a.x) + fo + int64_t(h0) * W * C;
        const int npx2 = the * W;
        uint2 xres[G::MAXT > 0 ? G::MAXT : 1];
#pragma unroll
        for (int k = 0; k < G::MAXT; ++k) {
            const int q = (wave / MT + k * (NW / MT)) * 16 + r16;
            xres[k] = q < npx2 ? *reinterpret_cast<const uint2*>(xbase + uint32_t(q * C + co0)) : make_uint2(0, 0);
        }
        __builtin_amdgcn_s_waitcnt(0);   // this tile's window (and the residual) have landed
        __syncthreads();
        {
            uint4* w4 = reinterpret_cast<uint4*>(xw);
            for (int j = tid; j < nsx; j += NT) {
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
        for (int nt = wave / MT; nt * 16 < npx1; nt += NW / MT) {
            const int q = nt * 16 + r16;
            const int qc = q < npx1 ? q : npx1 - 1;
            const int rowi = qdiv(qc, t.inv_W), col = qc - rowi * W, tr = tr0 + rowi;
            const cb_f32x4 acc = mma(xw + (tr * TW + col) * PB, wr1);
            if (q < npx1) {
                const int h = h0 - 1 + tr;
                const uint32_t u0 = pack2bf(acc[0] + b1[0], acc[1] + b1[1]);
                const uint32_t u1 = pack2bf(acc[2] + b1[2], acc[3] + b1[3]);
                if (h >= h0 && h < h0 + the)
                    *reinterpret_cast<uint2*>(tbase + (uint32_t(h) * W + col) * C + co0) = make_uint2(u0, u1);
                *reinterpret_cast<uint2*>(tw + (tr * TW + col + 1) * PB + co0 * 2) =
                    make_uint2(relu_bf16x2(u0), relu_bf16x2(u1));
            }
        }
        __syncthreads();   // conv1 has read the x window: the next tile's may land there
        if (tile + int(gridDim.x) < t.ntiles) stage_x(tile + gridDim.x);

        // ---- conv2 + residual: y on the band's rows
        uint16_t* ybase = static_cast<uint16_t*>(a.y) + fo + int64_t(h0) * W * C;
        auto conv2_tile = [&](int nt, const uint2* pre) {
            const int q = nt * 16 + r16;
            const int qc = q < npx2 ? q : npx2 - 1;
            const uint2 xr = pre ? *pre : *reinterpret_cast<const uint2*>(xbase + uint32_t(qc * C + co0));
            const int r = qdiv(qc, t.inv_W), col = qc - r * W;
            const cb_f32x4 acc = mma(tw + (r * TW + col) * PB, wr2);
            if (q < npx2)
                store4(ybase + uint32_t(q * C + co0), acc[0] + b2[0] + __uint_as_float(xr.x << 16),
                       acc[1] + b2[1] + __uint_as_float(xr.x & 0xffff0000u),
                       acc[2] + b2[2] + __uint_as_float(xr.y << 16),
                       acc[3] + b2[3] + __uint_as_float(xr.y & 0xffff0000u));
        };
        if constexpr (G::MAXT > 0) {
#pragma unroll
            for (int k = 0; k < G::MAXT; ++k)
                if ((wave / MT + k * (NW / MT)) * 16 < npx2) conv2_tile(wave / MT + k * (NW / MT), &xres[k]);
        } else {
            for (int nt = wave / MT; nt * 16 < npx2; nt += NW / MT) conv2_tile(nt, nullptr);
        }
    }
}

namespace {

constexpr size_t kRbLds = 160 * 1024;   // per CU, shared by the resident workgroups

template <int C>
hipError_t rb_fwd_launch(const ResBlockArgs& a, hipStream_t s) {
    using G = RbGeom<C>;
    constexpr int kRbWaves = G::NW;
    constexpr size_t kRbLdsTarget = kRbLds / G::WGS;
    const int H = a.H, W = a.W;
    auto lds = [&](int th) { return size_t(G::xwin_bytes(th, W)) + G::twin_bytes(th, W); };
    auto fits = [&](int th) {
        const int tiles = (th * W + 15) / 16, per = kRbWaves / G::MT;
        return ((th + 4) * (W + 2) * G::SPP + kRbWaves * 64 - 1) / (kRbWaves * 64) <= G::MAXS &&
               (G::MAXT == 0 || (tiles + per - 1) / per <= G::MAXT);
    };
    int thmax = H;
    while (thmax > 1 && (lds(thmax) > kRbLdsTarget || !fits(thmax))) --thmax;
    if (lds(thmax) > std::min<size_t>(lds_limit(), 160 * 1024) || !fits(thmax)) return hipErrorInvalidValue;
    if (int64_t(H) * W * C * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    int TH = 1, best = 1 << 30;   // fewest staged window rows per frame
    for (int th = 1; th <= thmax; ++th) {
        const int rows = (H + th - 1) / th * (th + 4);
        if (rows <= best) { best = rows; TH = th; }
    }
    RbTile t{};
    t.TH = TH; t.nbands = (H + TH - 1) / TH; t.ntiles = t.nbands * a.n;
    t.x_off = 0;
    t.t_off = G::xwin_bytes(TH, W);
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
