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
// LDS layout: each window is stored as C/16 planes of 16 channels, 32 bytes per pixel, pixels
// row-major with one zero padding column on each side. gfx950's LDS has 64 four-byte banks and
// serves a 16-byte read of a wave in four passes of 16 lanes (the lanes of each half-wave whose
// bits 2..4 have one parity); a pass is conflict-free when its 16 reads land on distinct 16-byte
// bank groups. A B fragment (lane (g, r): 8 k-values of pixel r) then spreads every pass over all
// 64 banks for any run of 16 consecutive window pixels, so a column tile is 16 consecutive window
// pixels, padding columns included (their outputs are dropped) and never a wrapped run of
// frame pixels, whose two-pixel jump at a row end would fold two reads onto one bank group.
// Per MFMA: 16 output pixels per column tile, one 16-byte B fragment per lane and k-step; with
// 16 channels the k-steps past the 9 taps read a zeroed 16-byte word.
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
    static constexpr int MT = C / 16;                      // 16-channel planes (and output blocks)
    static constexpr int PXB = 32;                         // bytes per pixel and plane
    // Workgroup shape: 16 channels hold both weight sets in 8-wave workgroups at 4 waves per
    // SIMD (128 registers); 32 channels need about 170 registers, so 4-wave workgroups at 3
    // waves per SIMD (three workgroups per CU) instead of spilling.
    static constexpr int NW = C >= 32 ? 4 : 8;
    static constexpr int WPS = C >= 32 ? 3 : 4;            // waves per SIMD (register budget)
    static constexpr int WGS = WPS * 4 / NW;               // workgroups per CU
    static constexpr int MAXS = C >= 32 ? 8 : 5;           // x-window staging slots per lane
    // conv2 column tiles per wave and tile whose residual is fetched at the tile's start; with 16
    // channels that covers all of them, with 32 (whose registers hold both weight sets) the
    // first two, and the rest are read per column tile
    static constexpr int MAXT = C >= 32 ? 2 : 5;
    static constexpr bool ALLPRE = C < 32;
    // x-window staging offsets kept in registers (with 32 channels, recomputed per tile)
    static constexpr bool OXREG = C < 32;
    __host__ __device__ static int blocks(int slots) { return (slots + 63) / 64; }
    // x window: MT planes of (TH+4) x (W+2) pixels, in whole 1 KB staging blocks
    __host__ __device__ static int xwin_bytes(int TH, int W) { return blocks(MT * (TH + 4) * (W + 2) * 2) * 1024; }
    // relu(t) window: MT planes of (TH+2) x (W+2) pixels, then a zeroed 32-byte word
    __host__ __device__ static int twin_bytes(int TH, int W) { return MT * (TH + 2) * (W + 2) * PXB + 32; }
};

struct RbTile {
    int TH, nbands, ntiles;
    int x_off, t_off;   // LDS byte offsets of the two windows
    int set_b;          // pipelined kernel: bytes from the first window pair to the second
    float inv_W, inv_TW;
};

template <int C, int NW>
__global__ __launch_bounds__(64 * NW, RbGeom<C>::WPS) void resblock_fwd_kernel(ResBlockArgs a, RbTile t) {
    using G = RbGeom<C>;
    constexpr int NT = 64 * NW, KSTEPS = G::KSTEPS, MT = G::MT, PXB = G::PXB;
    static_assert(NW % MT == 0, "waves split evenly over the output channel blocks");

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* xw = smem + t.x_off;   // relu(x) window, MT planes of [TH+4][W+2] pixels
    unsigned char* tw = smem + t.t_off;   // relu(t) window, MT planes of [TH+2][W+2] pixels

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TH = t.TH, TW = W + 2;
    const int xps = (TH + 4) * TW * PXB, tps = (TH + 2) * TW * PXB;   // plane strides (bytes)
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
    // Per-lane B-fragment offsets from the tap-(0,0) pixel. k-values 8g .. 8g+7 of a k-step are
    // channels (8g % C) .. +7 of one tap: plane (8g % C) / 16, half (g & 1) of the pixel's 32
    // bytes. With 16 channels a k-step spans two taps (table per k-step; lanes g >= 2 of the
    // last k-step are past the 9 taps and read the zero word); with 32, one tap per k-step.
    int boff[C < 32 ? KSTEPS : 1];
    if constexpr (C < 32) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const int tap = ks * 2 + (g >> 1);
            boff[ks] = ((tap / 3) * TW + tap % 3) * PXB + (g & 1) * 16;
        }
    }
    const bool zsel = C < 32 && g >= 2;
    const int lbx = C < 32 ? 0 : (g >> 1) * xps + (g & 1) * 16;   // lane's plane and half
    const int lbt = C < 32 ? 0 : (g >> 1) * tps + (g & 1) * 16;
    const int twb = TW * PXB;
    auto mma = [&](const unsigned char* xb, const unsigned char* zp, const uint4* wr) {
        cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const unsigned char* p;
            if constexpr (C < 32) p = ks == KSTEPS - 1 && zsel ? zp : xb + boff[ks];
            else p = xb + (ks / 3) * twb + (ks % 3) * PXB;
            acc = PrecBF16::mma(wr[ks], *reinterpret_cast<const uint4*>(p), acc);
            // with both weight sets held, keep at most three B fragments in flight
            if (C >= 32 && ks % 3 == 2) __builtin_amdgcn_sched_barrier(0);
        }
        return acc;
    };

    // ---- relu(t) window and zero word cleared once (padding columns are never written)
    for (int j = tid; j < G::twin_bytes(TH, W) / 16; j += NT) reinterpret_cast<uint4*>(tw)[j] = make_uint4(0, 0, 0, 0);

    // ---- x-window staging offsets, tile-invariant per lane (slot k of this wave:
    // j = (wave + NW*k)*64 + lane, 16 bytes: plane, pixel, half), relative to image row 0; a
    // tile adds h0 - 2 rows. Rows off the frame fall outside the frame's buffer resource
    // (negative, or past its end); padding columns read zero (kOOB).
    const int npx = (TH + 4) * TW, nsx = MT * npx * 2;
    auto x_off = [&](int k) {
        const int j = (wave + NW * k) * 64 + lane, pl = j / (npx * 2), rem = j - pl * npx * 2;
        const int p = rem >> 1, half = rem & 1;
        const int rr = p / TW, col = p - rr * TW;
        return (j < nsx && col >= 1 && col <= W) ? uint32_t(((rr * W + col - 1) * C + pl * 16 + half * 8) * 2) : kOOB;
    };
    uint32_t ox[G::OXREG ? G::MAXS : 1];
    if constexpr (G::OXREG) {
#pragma unroll
        for (int k = 0; k < G::MAXS; ++k) ox[k] = x_off(k);
    }
    __syncthreads();

    int lg = blockIdx.x;   // neighbouring bands on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    // x window of a tile, rows h0-2 .. h0+TH+1. The next tile's window is issued as soon as
    // conv1 has finished reading this one, so its latency overlaps conv2.
    auto stage_x = [&](unsigned char* dst, int tile) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + int64_t(f) * H * W * C, uint32_t(H) * W * C * 2);
        const uint32_t hr = uint32_t((band * TH - 2) * W * C * 2);   // wraps for h0 < 2: rows off the frame
#pragma unroll
        for (int k = 0; k < G::MAXS; ++k)
            if ((wave + NW * k) * 64 < nsx) dma16_to_lds(rx, dst + (wave + NW * k) * 1024, (G::OXREG ? ox[k] : x_off(k)) + hr);
    };
    if (lg < t.ntiles) stage_x(xw, lg);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int h0 = band * TH, the = H - h0 < TH ? H - h0 : TH;
        const int64_t fo = int64_t(f) * H * W * C;   // frame offset (elements)
        // conv2's outputs: window pixels 1 .. (the-1)*TW + W of the band's rows (row-major,
        // padding columns included and dropped); pixel pw is band row pw / TW, column pw % TW - 1
        const uint16_t* xbase = static_cast<const uint16_t*>(a.x) + fo + int64_t(h0) * W * C;
        const int npx2 = the * TW - 2;
        auto y_px = [&](int q, int& rb, int& cw) {   // clamped window pixel of conv2 output q
            const int pw = 1 + (q < npx2 ? q : npx2 - 1);
            rb = qdiv(pw, t.inv_TW);
            cw = pw - rb * TW;
            return pw;
        };
        auto res_off = [&](int rb, int cw) {   // residual x of that pixel (columns clamped)
            const int c = cw < 1 ? 1 : (cw > W ? W : cw);
            return uint32_t((rb * W + c - 1) * C + co0);
        };
        __builtin_amdgcn_s_waitcnt(0);   // this tile's window has landed
        __syncthreads();
        // conv2's residual for this wave's column tiles, in flight during the ReLU pass and conv1
        uint2 xres[G::MAXT];
#pragma unroll
        for (int k = 0; k < G::MAXT; ++k) {
            const int q = (wave / MT + k * (NW / MT)) * 16 + r16;
            int rb, cw;
            y_px(q, rb, cw);
            xres[k] = *reinterpret_cast<const uint2*>(xbase + res_off(rb, cw));
        }
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
            const int row16 = TW * PXB / 16;
            for (int pl = 0; pl < MT; ++pl) {
                uint4* t4 = reinterpret_cast<uint4*>(tw + pl * tps);
                if (tr0 == 1)
                    for (int j = tid; j < row16; j += NT) t4[j] = make_uint4(0, 0, 0, 0);
                for (int j = tid; j < (the + 2 - tr1) * row16; j += NT) t4[tr1 * row16 + j] = make_uint4(0, 0, 0, 0);
            }
        }
        __syncthreads();

        // ---- conv1: t on window rows [tr0, tr1), window pixels tr0*TW + 1 .. (tr1-1)*TW + W
        uint16_t* tbase = static_cast<uint16_t*>(a.t) + fo;
        const int npx1 = (tr1 - tr0) * TW - 2, pw1 = tr0 * TW + 1;
        for (int nt = wave / MT; nt * 16 < npx1; nt += NW / MT) {
            const int q = nt * 16 + r16;
            const int pw = pw1 + (q < npx1 ? q : npx1 - 1);
            const int tr = qdiv(pw, t.inv_TW), cw = pw - tr * TW;
            const cb_f32x4 acc = mma(xw + lbx + (pw - 1) * PXB, tw + MT * tps, wr1);   // tap (0,0): x-window pixel pw - 1
            if (q < npx1 && cw >= 1 && cw <= W) {
                const int h = h0 - 1 + tr;
                const uint32_t u0 = pack2bf(acc[0] + b1[0], acc[1] + b1[1]);
                const uint32_t u1 = pack2bf(acc[2] + b1[2], acc[3] + b1[3]);
                if (h >= h0 && h < h0 + the)
                    *reinterpret_cast<uint2*>(tbase + (uint32_t(h) * W + cw - 1) * C + co0) = make_uint2(u0, u1);
                *reinterpret_cast<uint2*>(tw + mt * tps + pw * PXB + g * 8) = make_uint2(relu_bf16x2(u0), relu_bf16x2(u1));
            }
        }
        __syncthreads();   // conv1 has read the x window: the next tile's may land there

        // ---- next tile's x window, then conv2 + residual (y on the band's rows). The two
        // windows are restrict parameters of one call, so the compiler knows that the loads in
        // flight into the x window do not write the relu(t) window that conv2 reads, and does
        // not wait for them before conv2's LDS reads.
        auto stage_conv2 = [&](unsigned char* __restrict__ xdst, const unsigned char* __restrict__ tsrc) {
            if (tile + int(gridDim.x) < t.ntiles) stage_x(xdst, tile + gridDim.x);
            uint16_t* ybase = static_cast<uint16_t*>(a.y) + fo + int64_t(h0) * W * C;
            auto conv2_tile = [&](int nt, const uint2* pre) {
                const int q = nt * 16 + r16;
                int rb, cw;
                const int pw = y_px(q, rb, cw);
                const uint2 xr = pre ? *pre : *reinterpret_cast<const uint2*>(xbase + res_off(rb, cw));
                const cb_f32x4 acc = mma(tsrc + lbt + (pw - 1) * PXB, tsrc + MT * tps, wr2);   // tap (0,0): t-window pixel pw - 1
                if (q < npx2 && cw >= 1 && cw <= W)
                    store4(ybase + uint32_t((rb * W + cw - 1) * C + co0), acc[0] + b2[0] + __uint_as_float(xr.x << 16),
                           acc[1] + b2[1] + __uint_as_float(xr.x & 0xffff0000u),
                           acc[2] + b2[2] + __uint_as_float(xr.y << 16),
                           acc[3] + b2[3] + __uint_as_float(xr.y & 0xffff0000u));
            };
#pragma unroll
            for (int k = 0; k < G::MAXT; ++k)
                if ((wave / MT + k * (NW / MT)) * 16 < npx2) conv2_tile(wave / MT + k * (NW / MT), &xres[k]);
            if constexpr (!G::ALLPRE)
                for (int nt = wave / MT + G::MAXT * (NW / MT); nt * 16 < npx2; nt += NW / MT) conv2_tile(nt, nullptr);
        };
        stage_conv2(xw, tw);
    }
}

// The 32-channel block in a 16-wave workgroup with two wave roles pipelined over tiles: while
// waves 0-7 form conv1 of a workgroup's next tile (its relu(x) window -> relu(t) window and the
// stored t), waves 8-15 form conv2 of its current tile (relu(t) window -> y). Each wave holds
// one convolution's A fragments for both 16-channel output blocks (72 registers), so every
// B-fragment read feeds two MFMAs, and the two convolutions of neighbouring tiles overlap
// instead of following each other between barriers. LDS holds two (x, t) window pairs: tile k
// uses pair k mod 2. Per step k (tile k's conv2, tile k+1's conv1) every wave meets two
// barriers: after the first, tile k+1's x window has landed and tile k's t window is complete;
// between them all waves ReLU tile k+1's x window in place and clear the t rows it has off the
// frame; after the second the conv1 waves issue tile k+2's x window into the pair tile k
// has left (its conv1 ran in the step before), then both roles run. Only the conv1 waves
// stage or wait for window loads, so the conv2 waves' residual loads and stores never queue
// behind them.
struct RbpGeom {
    static constexpr int C = 32, MT = 2, KS = 9, PXB = 32;
    static constexpr int NW = 16, NR = 8;   // waves per workgroup, per role
    static constexpr int MAXS = 6;          // x-window staging slots per conv1 lane
    __host__ __device__ static int xwin_bytes(int TH, int W) { return (MT * (TH + 4) * (W + 2) * 2 + 63) / 64 * 1024; }
    __host__ __device__ static int twin_bytes(int TH, int W) { return MT * (TH + 2) * (W + 2) * PXB; }
};

__global__ __launch_bounds__(64 * RbpGeom::NW, 1) void resblock_fwd_pipe_kernel(ResBlockArgs a, RbTile t) {
    using G = RbpGeom;
    constexpr int NT = 64 * G::NW, NR = G::NR, KS = G::KS, MT = G::MT, PXB = G::PXB, C = G::C;
    extern __shared__ __align__(16) unsigned char smem[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool role1 = wave < NR;   // conv1 (else conv2)
    const int rw = wave % NR;       // wave within its role
    const int g = lane >> 4, r16 = lane & 15;
    const int H = a.H, W = a.W, TH = t.TH, TW = W + 2;
    const int xps = (TH + 4) * TW * PXB, tps = (TH + 2) * TW * PXB;   // plane strides (bytes)
    const int twb = TW * PXB;
    const int npx = (TH + 4) * TW, nsx = MT * npx * 2;                 // x-window pixels, 16-byte slots

    // ---- both relu(t) windows cleared once (padding columns are never written)
    for (int s = 0; s < 2; ++s)
        for (int j = tid; j < G::twin_bytes(TH, W) / 16; j += NT)
            reinterpret_cast<uint4*>(smem + t.t_off + s * t.set_b)[j] = make_uint4(0, 0, 0, 0);

    // ---- this role's A fragments for both output blocks: A[o][k] = w[tap][i][o], k = tap*C + i
    // (one tap per k-step); the biases of the lane's four channels of each block
    const float* wsrc = role1 ? a.w1 : a.w2;
    const float* bsrc = role1 ? a.b1 : a.b2;
    uint4 wr[MT][KS];
#pragma unroll
    for (int b = 0; b < MT; ++b)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = wsrc[(ks * 32 + g * 8 + j) * C + b * 16 + r16];
            wr[b][ks] = make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]), pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
            __builtin_amdgcn_sched_barrier(0);   // convert each k-step's weights before loading the next
        }
    float bias[MT][4];
#pragma unroll
    for (int b = 0; b < MT; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) bias[b][j] = bsrc ? bsrc[b * 16 + g * 4 + j] : 0.f;
    // lane's B-fragment offset: k-values 8g .. 8g+7 of a k-step are channels 8g .. 8g+7 of its
    // tap, plane g / 2, half g % 2 of the pixel's 32 bytes
    const int lbx = (g >> 1) * xps + (g & 1) * 16, lbt = (g >> 1) * tps + (g & 1) * 16;
    auto mma2 = [&](const unsigned char* xb, cb_f32x4 (&acc)[MT]) {
#pragma unroll
        for (int b = 0; b < MT; ++b) acc[b] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const uint4 bf = *reinterpret_cast<const uint4*>(xb + (ks / 3) * twb + (ks % 3) * PXB);
#pragma unroll
            for (int b = 0; b < MT; ++b) acc[b] = PrecBF16::mma(wr[b][ks], bf, acc[b]);
            if (ks % 3 == 2) __builtin_amdgcn_sched_barrier(0);   // at most three B fragments in flight
        }
    };

    int lg = blockIdx.x;   // neighbouring bands on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    const int G0 = int(gridDim.x);
    const int cnt = lg < t.ntiles ? (t.ntiles - lg + G0 - 1) / G0 : 0;   // this workgroup's tiles
    auto band_of = [&](int k, int& h0, int& the, int64_t& fo) {
        const int tile = lg + k * G0, band = tile % t.nbands, f = tile / t.nbands;
        h0 = band * TH;
        the = H - h0 < TH ? H - h0 : TH;
        fo = int64_t(f) * H * W * C;
    };
    // tile k's x window ReLU'd in place; its t window's rows off the frame cleared
    auto prep = [&](int k) {
        if (k >= cnt) return;
        int h0, the;
        int64_t fo;
        band_of(k, h0, the, fo);
        uint4* w4 = reinterpret_cast<uint4*>(smem + t.x_off + (k & 1) * t.set_b);
        for (int j = tid; j < nsx; j += NT) {
            uint4 v = w4[j];
            v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
            w4[j] = v;
        }
        const int tr0 = h0 == 0 ? 1 : 0;
        const int tr1 = the + 2 < H - h0 + 1 ? the + 2 : H - h0 + 1;
        const int row16 = TW * PXB / 16;
        for (int pl = 0; pl < MT; ++pl) {
            uint4* t4 = reinterpret_cast<uint4*>(smem + t.t_off + (k & 1) * t.set_b + pl * tps);
            if (tr0 == 1)
                for (int j = tid; j < row16; j += NT) t4[j] = make_uint4(0, 0, 0, 0);
            for (int j = tid; j < (the + 2 - tr1) * row16; j += NT) t4[tr1 * row16 + j] = make_uint4(0, 0, 0, 0);
        }
    };

    if (role1) {
        // x-window staging offsets, tile-invariant per lane (slot k of this wave: j = (rw +
        // NR*k)*64 + lane: plane, pixel, half), relative to image row 0; a tile adds h0 - 2 rows.
        // Rows off the frame fall outside the frame's buffer resource; padding columns read zero.
        uint32_t ox[G::MAXS];
#pragma unroll
        for (int k = 0; k < G::MAXS; ++k) {
            const int j = (rw + NR * k) * 64 + lane, pl = j / (npx * 2), rem = j - pl * npx * 2;
            const int p = rem >> 1, half = rem & 1;
            const int rr = p / TW, col = p - rr * TW;
            ox[k] = (j < nsx && col >= 1 && col <= W) ? uint32_t(((rr * W + col - 1) * C + pl * 16 + half * 8) * 2) : kOOB;
        }
        auto stage = [&](unsigned char* dst, int k) {
            int h0, the;
            int64_t fo;
            band_of(k, h0, the, fo);
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + fo, uint32_t(H) * W * C * 2);
            const uint32_t hr = uint32_t((h0 - 2) * W * C * 2);   // wraps for h0 < 2: rows off the frame
#pragma unroll
            for (int s = 0; s < G::MAXS; ++s)
                if ((rw + NR * s) * 64 < nsx) dma16_to_lds(rx, dst + (rw + NR * s) * 1024, ox[s] + hr);
        };
        // conv1 of tile k (t on its band's rows plus a halo row either side), with tile k+1's x
        // window issued first; the windows are restrict parameters of one call, so the compiler
        // knows the loads in flight do not write what conv1 reads
        auto step = [&](unsigned char* __restrict__ xnext, const unsigned char* __restrict__ xw,
                        unsigned char* __restrict__ tw, int k) {
            if (k + 1 < cnt) stage(xnext, k + 1);
            if (k >= cnt) return;
            int h0, the;
            int64_t fo;
            band_of(k, h0, the, fo);
            const int tr0 = h0 == 0 ? 1 : 0;
            const int tr1 = the + 2 < H - h0 + 1 ? the + 2 : H - h0 + 1;
            uint16_t* tbase = static_cast<uint16_t*>(a.t) + fo;
            const int npx1 = (tr1 - tr0) * TW - 2, pw1 = tr0 * TW + 1;
            for (int nt = rw; nt * 16 < npx1; nt += NR) {
                const int q = nt * 16 + r16;
                const int pw = pw1 + (q < npx1 ? q : npx1 - 1);
                const int tr = qdiv(pw, t.inv_TW), cw = pw - tr * TW;
                cb_f32x4 acc[MT];
                mma2(xw + lbx + (pw - 1) * PXB, acc);   // tap (0,0): x-window pixel pw - 1
                if (q < npx1 && cw >= 1 && cw <= W) {
                    const int h = h0 - 1 + tr;
#pragma unroll
                    for (int b = 0; b < MT; ++b) {
                        const uint32_t u0 = pack2bf(acc[b][0] + bias[b][0], acc[b][1] + bias[b][1]);
                        const uint32_t u1 = pack2bf(acc[b][2] + bias[b][2], acc[b][3] + bias[b][3]);
                        if (h >= h0 && h < h0 + the)
                            *reinterpret_cast<uint2*>(tbase + (uint32_t(h) * W + cw - 1) * C + b * 16 + g * 4) = make_uint2(u0, u1);
                        *reinterpret_cast<uint2*>(tw + b * tps + pw * PXB + g * 8) = make_uint2(relu_bf16x2(u0), relu_bf16x2(u1));
                    }
                }
            }
        };
        if (cnt > 0) stage(smem + t.x_off, 0);
        for (int k = -1; k < cnt; ++k) {
            __builtin_amdgcn_s_waitcnt(0);   // tile k+1's x window (this wave's part) has landed
            lds_barrier();
            prep(k + 1);
            lds_barrier();
            const int s1 = (k + 1) & 1;
            step(smem + t.x_off + (s1 ^ 1) * t.set_b, smem + t.x_off + s1 * t.set_b, smem + t.t_off + s1 * t.set_b, k + 1);
        }
    } else {
        for (int k = -1; k < cnt; ++k) {
            lds_barrier();
            prep(k + 1);
            lds_barrier();
            if (k < 0) continue;
            // conv2 + bias + residual on tile k's band rows: window pixels 1 .. (the-1)*TW + W
            // (padding columns included and dropped); pixel pw is band row pw / TW, column pw % TW - 1
            int h0, the;
            int64_t fo;
            band_of(k, h0, the, fo);
            const unsigned char* tw = smem + t.t_off + (k & 1) * t.set_b;
            const uint16_t* xbase = static_cast<const uint16_t*>(a.x) + fo + int64_t(h0) * W * C;
            uint16_t* ybase = static_cast<uint16_t*>(a.y) + fo + int64_t(h0) * W * C;
            const int npx2 = the * TW - 2;
            auto px = [&](int nt, int& pw, int& rb, int& cw) {
                const int q = nt * 16 + r16;
                pw = 1 + (q < npx2 ? q : npx2 - 1);
                rb = qdiv(pw, t.inv_TW);
                cw = pw - rb * TW;
            };
            auto res = [&](int nt, uint2 (&xr)[MT]) {   // residual x of a column tile (columns clamped)
                int pw, rb, cw;
                px(nt, pw, rb, cw);
                const int c = cw < 1 ? 1 : (cw > W ? W : cw);
#pragma unroll
                for (int b = 0; b < MT; ++b)
                    xr[b] = *reinterpret_cast<const uint2*>(xbase + uint32_t((rb * W + c - 1) * C + b * 16 + g * 4));
            };
            uint2 xn[MT];
            if (rw * 16 < npx2) res(rw, xn);
            for (int nt = rw; nt * 16 < npx2; nt += NR) {
                uint2 xr[MT];
#pragma unroll
                for (int b = 0; b < MT; ++b) xr[b] = xn[b];
                if ((nt + NR) * 16 < npx2) res(nt + NR, xn);   // the next column tile's, in flight
                int pw, rb, cw;
                px(nt, pw, rb, cw);
                cb_f32x4 acc[MT];
                mma2(tw + lbt + (pw - 1) * PXB, acc);   // tap (0,0): t-window pixel pw - 1
                if (nt * 16 + r16 < npx2 && cw >= 1 && cw <= W) {
#pragma unroll
                    for (int b = 0; b < MT; ++b)
                        store4(ybase + uint32_t((rb * W + cw - 1) * C + b * 16 + g * 4),
                               acc[b][0] + bias[b][0] + __uint_as_float(xr[b].x << 16),
                               acc[b][1] + bias[b][1] + __uint_as_float(xr[b].x & 0xffff0000u),
                               acc[b][2] + bias[b][2] + __uint_as_float(xr[b].y << 16),
                               acc[b][3] + bias[b][3] + __uint_as_float(xr[b].y & 0xffff0000u));
                }
            }
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
        const int tiles = (th * (W + 2) - 2 + 15) / 16, per = kRbWaves / G::MT;
        return G::blocks(G::MT * (th + 4) * (W + 2) * 2) <= G::MAXS * kRbWaves &&
               (!G::ALLPRE || (tiles + per - 1) / per <= G::MAXT);
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

// The pipelined 32-channel kernel: two window pairs in the CU's LDS, one 16-wave workgroup per
// CU. It pays only where every workgroup runs many tiles: measured at 8192 frames of 42x42
// (128 tiles per workgroup) 950 against 995 us for the three-workgroup kernel, but at 2048
// frames (8 tiles per workgroup) 87 against 78 us at 21x21 and 54 against 29 us at 11x11,
// where the pipeline's first step and the two barriers per tile weigh more. Returns
// hipErrorNotSupported where no band height fits or a workgroup would get fewer than 32 tiles.
hipError_t rbp_launch(const ResBlockArgs& a, hipStream_t s) {
    using G = RbpGeom;
    const int H = a.H, W = a.W;
    auto pair = [&](int th) { return size_t(G::xwin_bytes(th, W)) + G::twin_bytes(th, W); };
    auto fits = [&](int th) {
        return 2 * pair(th) <= std::min<size_t>(lds_limit(), kRbLds) &&
               G::MT * (th + 4) * (W + 2) * 2 <= G::MAXS * G::NR * 64;
    };
    if (int64_t(H) * W * G::C * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    int TH = 0, best = 1 << 30;   // fewest staged window rows per frame
    for (int th = 1; th <= H; ++th) {
        if (!fits(th)) continue;
        const int rows = (H + th - 1) / th * (th + 4);
        if (rows <= best) { best = rows; TH = th; }
    }
    if (TH == 0) return hipErrorNotSupported;
    RbTile t{};
    t.TH = TH; t.nbands = (H + TH - 1) / TH; t.ntiles = t.nbands * a.n;
    t.x_off = 0;
    t.t_off = G::xwin_bytes(TH, W);
    t.set_b = int(pair(TH));
    t.inv_W = 1.f / float(W); t.inv_TW = 1.f / float(W + 2);
    const size_t L = 2 * pair(TH);
    const void* fn = reinterpret_cast<const void*>(&resblock_fwd_pipe_kernel);
    const int gx = resident_blocks(fn, 64 * G::NW, L);
    if (gx < 1 || t.ntiles < 32 * gx) return hipErrorNotSupported;
    ProfScope ps(s, [&] { return cb_key("resblock_fwd", 0, cb_dims(G::C, G::C) + "/" + cb_dims(H, W)); });
    hipLaunchKernelGGL(resblock_fwd_pipe_kernel, dim3(unsigned(gx)), dim3(64 * G::NW), L, s, a, t);
    return hipGetLastError();
}

}  // namespace

bool resblock_fwd_supported(int C) { return C == 16 || C == 32; }

hipError_t resblock_fwd(int C, const ResBlockArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    if (C == 16) return rb_fwd_launch<16>(a, s);
    if (C == 32) {
        const hipError_t e = rbp_launch(a, s);
        return e != hipErrorNotSupported ? e : rb_fwd_launch<32>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace cb
