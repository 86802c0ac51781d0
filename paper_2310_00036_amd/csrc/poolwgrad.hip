// Backward of the first stage entry (Section 5's IMPALA-ResNet: conv3x3 on the uint8 frames,
// then max-pool 3x3/2) in one kernel, bf16: the max-pool's input gradient is formed in LDS
// and feeds the conv's weight gradient directly, so the full-resolution gradient never goes
// through HBM.
//
//   dC[h][w][c]        = sum of dP[oh][ow][c] over the pool windows whose first maximum
//                        (arg) is cell (h, w)                         (max-pool backward)
//   dW[ky][kx][ci][co] = sum over pixels p of frames[p + d(tap)][ci] / 255 * dC[p][co]
//   db[co]             = sum over pixels p of dC[p][co]
//
// The frames need no input gradient. A tile is one frame's band of TB 2x2 pixel blocks
// (2*TB rows in the pool's padded coordinates): block (i, j) holds padded cells
// (2i + a, 2j + b), a, b in {0, 1}, and only windows (i-1 | i, j-1 | j) reach it, so the
// band needs pooled rows i0-1 .. i0+TB-1. Staged in LDS per tile:
//   - the frame window, image rows 2*i0 - ph - 1 .. 2*(i0+TB) - ph, all columns plus a zero
//     column either side, as uint8 then converted once to bf16 (exact for 0..255);
//   - those pooled-gradient and argmax rows, with a zero column either side (a zero window
//     adds +0, as the stand-alone max-pool backward adds for windows off the grid);
//   - dC for the band's rows, every window column (the padding columns stay zero), formed by
//     the same per-cell gather and summation order as the stand-alone max-pool backward,
//     rounded to bf16 as that kernel stores it.
// The weight gradient then contracts over dC's window pixels p (padding columns add zero):
// A = dC^T and B = the frame window at p - 1 + tap offset, both read with the LDS transpose
// read, every address advancing by a constant per k-step. B's 16 columns are 4 taps x 4
// channels (taps past the ninth give columns the reduction drops). The waves split the
// k-steps and add their accumulators in a fixed order at the end; one float32 partial per
// workgroup, summed in a fixed order by a second kernel.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace cb {

template <int CO>
struct PwGeom {
    static constexpr int MT = CO / 16;
    static constexpr int NB = 3, NBB = 4;                       // 3 column blocks + bias
    static constexpr int DPB = CO * 2 + (CO >= 32 ? 32 : 0);    // dC bytes per pixel
    static constexpr int CG = CO / 8;                           // 8-channel groups
    static constexpr int PSTRIDE = MT * NBB * 256;
    // staging slots per lane (8-wave workgroup) the planner stays within
    static constexpr int MAXR = 4, MAXP = 4, MAXG = 2;
};

template <int CO, int NW>
__global__ __launch_bounds__(64 * NW, 4) void pool_wgrad_u8_kernel(PoolWgArgs a, PwTile t) {
    using G = PwGeom<CO>;
    constexpr int NT = 64 * NW;
    constexpr int MT = G::MT, NBB = G::NBB, DPB = G::DPB, CG = G::CG;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;                     // 64 zero bytes
    unsigned char* raw = smem + t.raw_off;          // uint8 window [TR][TW] x 4
    unsigned char* win = smem + t.win_off + 16;     // bf16 window [TR][TW] x 8, guards either side
    unsigned char* dpl = smem + t.dp_off;           // pooled gradient [TB+1][OW+2] x CO bf16
    unsigned char* agl = smem + t.arg_off;          // argmax [TB+1][OW+2] x CO
    unsigned char* dcl = smem + t.dc_off;           // dC [2TB][TW] x DPB

    // an earlier launch's weight-gradient partials, summed first (LDS is free until staging)
    if (a.pend.nparts > 0) pending_reduce<NT>(a.pend, smem);
    if (a.pend2.nparts > 0) pending_reduce<NT>(a.pend2, smem);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const int H = a.H, W = a.W, TB = t.TB, OW = t.OW, OH = t.OH;
    const int TW = W + 2, TR = 2 * TB + 2, PW2 = OW + 2;

    // zero area, the window guards and the whole dC region (its padding columns are never
    // written by the gather)
    if (tid < 16) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;
    if (tid < 4) {
        reinterpret_cast<uint32_t*>(win - 16)[tid] = 0u;
        reinterpret_cast<uint32_t*>(win + t.win_guard)[tid] = 0u;
    }
    for (int j = tid; j < 2 * TB * TW * DPB / 16; j += NT) reinterpret_cast<uint4*>(dcl)[j] = make_uint4(0, 0, 0, 0);

    // ---- staging offsets, tile-invariant per lane (slot k of this wave: j = (wave+NW*k)*64 + lane),
    // relative to window row 0 at image row 0 / pooled row 0; a tile adds its first row. Rows
    // off the frame fall outside the buffer resource (negative, or past its end) and read zero.
    const int nsr = TR * TW, nsp = (TB + 1) * PW2 * CG, nsg = (TB + 1) * PW2 * (CO / 16);
    uint32_t orw[G::MAXR], opd[G::MAXP], oag[G::MAXG];
#pragma unroll
    for (int k = 0; k < G::MAXR; ++k) {
        const int j = (wave + NW * k) * 64 + lane, rr = j / TW, col = j - rr * TW;
        orw[k] = (j < nsr && col >= 1 && col <= W) ? uint32_t((rr * W + col - 1) * 4) : kOOB;
    }
#pragma unroll
    for (int k = 0; k < G::MAXP; ++k) {
        const int j = (wave + NW * k) * 64 + lane, px = j / CG, c = j - px * CG;
        const int rr = px / PW2, col = px - rr * PW2;
        opd[k] = (j < nsp && col >= 1 && col <= OW) ? uint32_t(((rr * OW + col - 1) * CO + c * 8) * 2) : kOOB;
    }
#pragma unroll
    for (int k = 0; k < G::MAXG; ++k) {
        const int j = (wave + NW * k) * 64 + lane, px = j / (CO / 16), c = j - px * (CO / 16);
        const int rr = px / PW2, col = px - rr * PW2;
        oag[k] = (j < nsg && col >= 1 && col <= OW) ? uint32_t((rr * OW + col - 1) * CO + c * 16) : kOOB;
    }

    // ---- weight-gradient fragments: B column block nb covers taps 4nb..4nb+3 (lane group m
    // takes tap 4nb+m; taps past the ninth read tap 8 and land in dropped columns)
    int boff[3];
#pragma unroll
    for (int nb = 0; nb < 3; ++nb) {
        const int tap = min(4 * nb + m, 8);
        boff[nb] = ((tap / 3) * TW + tap % 3 - 1) * 8;
    }
    cb_f32x4 acc[MT][NBB];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nb = 0; nb < NBB; ++nb) acc[mt][nb] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

    int lg = blockIdx.x;   // neighbouring bands on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    // a tile's inputs: frame rows hw0 .. of the window, pooled rows i0-1 .. of the gradient and the
    // argmax. The next tile's are issued once the max-pool backward has read this one's, so
    // their latency overlaps the weight gradient.
    auto stage = [&](unsigned char* rdst, unsigned char* pdst, unsigned char* gdst, int tile) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int i0 = band * TB;
        const int hw0 = 2 * i0 - t.ph - 1;
        const int64_t row = a.row_idx ? a.row_idx[f] : f;
        const uint32_t fb = uint32_t(H) * W * 4;
        const auto rf = buf_rsrc(a.obs + row * fb, fb);
        const uint32_t hr = uint32_t(hw0 * W * 4);   // wraps for hw0 = -1: reads zero
#pragma unroll
        for (int k = 0; k < G::MAXR; ++k)
            if ((wave + NW * k) * 64 < nsr) dma4_to_lds(rf, rdst + (wave + NW * k) * 256, orw[k] + hr);
        const uint32_t pb = uint32_t(OH) * OW * CO;   // pooled elements per frame
        const auto rp = buf_rsrc(static_cast<const uint16_t*>(a.dp) + int64_t(f) * pb, pb * 2);
        const auto rg = buf_rsrc(a.arg + int64_t(f) * pb, pb);
        const uint32_t pr = uint32_t((i0 - 1) * OW * CO);   // pooled row i0-1 (wraps at i0 = 0)
#pragma unroll
        for (int k = 0; k < G::MAXP; ++k)
            if ((wave + NW * k) * 64 < nsp) dma16_to_lds(rp, pdst + (wave + NW * k) * 1024, opd[k] + 2 * pr);
#pragma unroll
        for (int k = 0; k < G::MAXG; ++k)
            if ((wave + NW * k) * 64 < nsg) dma16_to_lds(rg, gdst + (wave + NW * k) * 1024, oag[k] + pr);
    };
    if (lg < t.ntiles) stage(raw, dpl, agl, lg);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int i0 = (tile % t.nbands) * TB;
        const int nbr = t.BH - i0 < TB ? t.BH - i0 : TB;   // block rows in this band
        __builtin_amdgcn_s_waitcnt(0);   // this tile's inputs have landed
        __syncthreads();                 // ... everyone's, and the previous weight gradient is done

        // ---- frames -> bf16 window (4 channels per pixel)
        for (int p = tid; p < nsr; p += NT)
            *reinterpret_cast<uint2*>(win + p * 8) = u8x4_to_bf16(*reinterpret_cast<const uint32_t*>(raw + p * 4));
        // ---- max-pool backward into dC: item (block row bi, block column j, 8 channels)
        {
            const int items = nbr * t.BW * CG;
            for (int it = tid; it < items; it += NT) {
                const int c8 = it % CG, blk = it / CG;
                const int bi = blk / t.BW, j = blk - bi * t.BW;
                // windows (bi-1+u, j-1+v) at LDS rows bi+u, columns j+v
                uint32_t ka[4][2], s01[4][2], s23[4][2];
                uint4 dv[4];
#pragma unroll
                for (int w4 = 0; w4 < 4; ++w4) {
                    const int px = (bi + (w4 >> 1)) * PW2 + j + (w4 & 1);
                    const uint2 k8 = *reinterpret_cast<const uint2*>(agl + px * CO + c8 * 8);
                    ka[w4][0] = k8.x; ka[w4][1] = k8.y;
#pragma unroll
                    for (int wd = 0; wd < 2; ++wd) { s01[w4][wd] = arg_sel01(ka[w4][wd]); s23[w4][wd] = arg_sel23(ka[w4][wd]); }
                    dv[w4] = *reinterpret_cast<const uint4*>(dpl + (px * CO + c8 * 8) * 2);
                }
                // window w4's gradients of channels 4wd .. 4wd+3 where its cell is T, else +0
#define CB_PICK(T, w4, wd) \
    arg_pick<T>((wd) ? make_uint2(dv[w4].z, dv[w4].w) : make_uint2(dv[w4].x, dv[w4].y), ka[w4][wd], s01[w4][wd], s23[w4][wd])
                // each cell adds its windows in (oh, ow) order; the lower-right cell has one
                // window, whose bf16 gradient it keeps as it is
                uint32_t c00[4], c01[4], c10[4], c11[4];
#pragma unroll
                for (int wd = 0; wd < 2; ++wd) {
                    const uint2 a0 = CB_PICK(8, 0, wd), a1 = CB_PICK(6, 1, wd), a2 = CB_PICK(2, 2, wd), a3 = CB_PICK(0, 3, wd);
                    const uint2 b1 = CB_PICK(7, 1, wd), b3 = CB_PICK(1, 3, wd);
                    const uint2 e2 = CB_PICK(5, 2, wd), e3 = CB_PICK(3, 3, wd);
                    const uint2 f3 = CB_PICK(4, 3, wd);
                    const uint32_t A0[2] = {a0.x, a0.y}, A1[2] = {a1.x, a1.y}, A2[2] = {a2.x, a2.y}, A3[2] = {a3.x, a3.y};
                    const uint32_t B1[2] = {b1.x, b1.y}, B3[2] = {b3.x, b3.y}, E2[2] = {e2.x, e2.y}, E3[2] = {e3.x, e3.y};
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        c00[2 * wd + h] = pack2bf(bf_lo(A0[h]) + bf_lo(A1[h]) + bf_lo(A2[h]) + bf_lo(A3[h]),
                                                  bf_hi(A0[h]) + bf_hi(A1[h]) + bf_hi(A2[h]) + bf_hi(A3[h]));
                        c01[2 * wd + h] = pack2bf(bf_lo(B1[h]) + bf_lo(B3[h]), bf_hi(B1[h]) + bf_hi(B3[h]));
                        c10[2 * wd + h] = pack2bf(bf_lo(E2[h]) + bf_lo(E3[h]), bf_hi(E2[h]) + bf_hi(E3[h]));
                    }
                    c11[2 * wd] = f3.x; c11[2 * wd + 1] = f3.y;
                }
#undef CB_PICK
                // cells (2bi + a, 2j + b) in padded coordinates -> dC row 2bi + a, window column
                // 2j + b - pw + 1; cells off the frame hold zero
                const int h = 2 * (i0 + bi) - t.ph, w = 2 * j - t.pw;
                const bool r0 = h >= 0 && h < a.H, r1 = h + 1 < a.H, q0 = w >= 0, q1 = w + 1 < W;
                unsigned char* cp = dcl + ((2 * bi) * TW + w + 1) * DPB + c8 * 16;
                auto put = [&](unsigned char* p, bool ok, const uint32_t* c) {
                    *reinterpret_cast<uint4*>(p) = ok ? make_uint4(c[0], c[1], c[2], c[3]) : make_uint4(0, 0, 0, 0);
                };
                put(cp, r0 && q0, c00);
                put(cp + DPB, r0 && q1, c01);
                put(cp + TW * DPB, r1 && q0, c10);
                put(cp + (TW + 1) * DPB, r1 && q1, c11);
            }
        }
        __syncthreads();   // the max-pool backward has read the inputs: the next tile's may land

        // ---- next tile's inputs, then the weight gradient over dC's window pixels (wave w takes
        // k-steps w, w+NW, ...). The staging buffers and the windows the weight gradient reads are
        // restrict parameters of one call, so the compiler does not wait for the loads in flight.
        auto stage_wgrad = [&](unsigned char* __restrict__ rdst, unsigned char* __restrict__ pdst,
                               unsigned char* __restrict__ gdst, const unsigned char* __restrict__ dc,
                               const unsigned char* __restrict__ wn, const unsigned char* __restrict__ zr) {
            if (tile + int(gridDim.x) < t.ntiles) stage(rdst, pdst, gdst, tile + gridDim.x);
            const int L = 2 * nbr * TW;
            const int nks = (L + 31) >> 5;
            const int o0 = 4 * g + jj;
            for (int ks = wave; ks < nks; ks += NW) {
                uint4 af[MT];
                int pb[2];
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int p = ks * 32 + half * 16 + o0;
                    const bool ok = p < L;
                    pb[half] = ok ? p : L - 1;
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const uint2 u = lds_read_tr16(ok ? dc + p * DPB + mt * 32 + 8 * m : zr);
                        if (half == 0) { af[mt].x = u.x; af[mt].y = u.y; } else { af[mt].z = u.x; af[mt].w = u.y; }
                    }
                }
#pragma unroll
                for (int nb = 0; nb < 3; ++nb) {
                    const uint2 lo = lds_read_tr16(wn + pb[0] * 8 + boff[nb]);
                    const uint2 hi = lds_read_tr16(wn + pb[1] * 8 + boff[nb]);
                    const uint4 bf = make_uint4(lo.x, lo.y, hi.x, hi.y);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) acc[mt][nb] = PrecBF16::mma(af[mt], bf, acc[mt][nb]);
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) acc[mt][3] = PrecBF16::mma(af[mt], ones, acc[mt][3]);
            }
        };
        stage_wgrad(raw, dpl, agl, dcl, win, zero);
    }

    // ---- add the waves' accumulators in wave order; wave 0 writes the partial
    __syncthreads();
    cb_f32x4* red = reinterpret_cast<cb_f32x4*>(smem + 64);   // [NW][MT*NBB][64]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nb = 0; nb < NBB; ++nb) red[(wave * MT * NBB + mt * NBB + nb) * 64 + lane] = acc[mt][nb];
    __syncthreads();
    if (wave == 0) {
        float* part = a.partial + int64_t(blockIdx.x) * G::PSTRIDE;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nb = 0; nb < NBB; ++nb) {
                cb_f32x4 s = red[(mt * NBB + nb) * 64 + lane];
                for (int w = 1; w < NW; ++w) s += red[(w * MT * NBB + mt * NBB + nb) * 64 + lane];
#pragma unroll
                for (int e = 0; e < 4; ++e) part[(mt * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = s[e];
            }
    }
}

namespace {

constexpr int kPwWaves = 8;
constexpr size_t kPwLdsTarget = 80 * 1024;
constexpr size_t kPwPartBytes = 16u << 20;

template <int CO>
int pw_parts_cap() {
    const size_t cap = kPwPartBytes / (size_t(PwGeom<CO>::PSTRIDE) * sizeof(float));
    return int(cap < 256 ? 256 : (cap > 1024 ? 1024 : cap));
}

template <int CO>
hipError_t pw_launch(const PoolWgArgs& a, hipStream_t s) {
    using G = PwGeom<CO>;
    const int H = a.H, W = a.W, TW = W + 2;
    const int OH = (H + 1) / 2, OW = (W + 1) / 2;
    const int PH = (OH - 1) * 2 + 3 - H, PWd = (OW - 1) * 2 + 3 - W;
    const int ph = (PH > 0 ? PH : 0) / 2, pw = (PWd > 0 ? PWd : 0) / 2;
    const int BH = (H + ph + 1) / 2, BW = (W + pw + 1) / 2;
    auto layout = [&](int tb, PwTile& t) {
        const int tr = 2 * tb + 2;
        t.raw_off = 64;
        t.win_off = t.raw_off + (tr * TW + 63) / 64 * 256;
        t.win_guard = tr * TW * 8;
        t.dp_off = t.win_off + (t.win_guard + 32 + 15) / 16 * 16;
        t.arg_off = t.dp_off + ((tb + 1) * (OW + 2) * G::CG + 63) / 64 * 1024;
        t.dc_off = t.arg_off + ((tb + 1) * (OW + 2) * (CO / 16) + 63) / 64 * 1024;
        const size_t end = size_t(t.dc_off) + size_t(2 * tb) * TW * G::DPB;
        const size_t red = 64 + size_t(kPwWaves) * G::MT * G::NBB * 64 * 16;   // final wave sums
        return std::max(end, red);
    };
    auto fits = [&](int tb) {
        const int per = kPwWaves * 64, tr = 2 * tb + 2;
        return (tr * TW + per - 1) / per <= G::MAXR && ((tb + 1) * (OW + 2) * G::CG + per - 1) / per <= G::MAXP &&
               ((tb + 1) * (OW + 2) * (CO / 16) + per - 1) / per <= G::MAXG;
    };
    const size_t limit = std::min<size_t>(lds_limit(), 160 * 1024);
    PwTile t{};
    int tbmax = BH;
    while (tbmax > 1 && (layout(tbmax, t) > kPwLdsTarget || !fits(tbmax))) --tbmax;
    if (layout(tbmax, t) > limit || !fits(tbmax)) return hipErrorInvalidValue;
    if (int64_t(H) * W * 4 >= (int64_t(1) << 31) || int64_t(OH) * OW * CO * 2 >= (int64_t(1) << 31))
        return hipErrorInvalidValue;
    const int nb0 = (BH + tbmax - 1) / tbmax;
    const int TB = (BH + nb0 - 1) / nb0;   // balanced bands
    const size_t L = std::max(layout(TB, t), size_t(kPwWaves * 4) * 17 * 16);   // (pending reduce)
    t.TB = TB; t.nbands = (BH + TB - 1) / TB; t.ntiles = t.nbands * a.n;
    t.OH = OH; t.OW = OW; t.ph = ph; t.pw = pw; t.BH = BH; t.BW = BW;
    const void* fn = reinterpret_cast<const void*>(&pool_wgrad_u8_kernel<CO, kPwWaves>);
    int parts = std::min(resident_blocks(fn, 64 * kPwWaves, L), pw_parts_cap<CO>());
    if (parts > t.ntiles) parts = t.ntiles;
    const std::string shape = cb_dims(4, CO) + "/" + cb_dims(H, W) + "/u8";
    {
        ProfScope ps(s, [&] { return cb_key("pool_wgrad", 0, shape); });
        hipLaunchKernelGGL((pool_wgrad_u8_kernel<CO, kPwWaves>), dim3(unsigned(parts)), dim3(64 * kPwWaves), L, s, a,
                           t);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    ProfScope ps(s, [&] { return cb_key("pool_wgrad_reduce", 0, shape); });
    return wgrad_reduce_tr(4, CO, a.partial, parts, a.dw, a.db, 1.f / 255.f, s);
}

}  // namespace

bool pool_wgrad_u8_supported(int cout) { return cout == 16 || cout == 32; }

size_t pool_wgrad_u8_partial_floats(int cout) {
    if (cout == 16) return size_t(pw_parts_cap<16>()) * PwGeom<16>::PSTRIDE;
    if (cout == 32) return size_t(pw_parts_cap<32>()) * PwGeom<32>::PSTRIDE;
    return 0;
}

hipError_t pool_wgrad_u8(int cout, const PoolWgArgs& a, hipStream_t s) {
    if (a.n <= 0) {
        const hipError_t e = flush_pending_reduce(a.pend, s);
        return e != hipSuccess ? e : flush_pending_reduce(a.pend2, s);
    }
    if (cout == 16) return pw_launch<16>(a, s);
    if (cout == 32) return pw_launch<32>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace cb
