// Backward pass of one 3x3 stride-1 SAME convolution in one kernel (bf16 storage, float32
// accumulation on gfx950 MFMA). For y = conv(X, w) + b with X = relu(x) or x:
//
//   dx[p][ci]          = sum over taps and co of w[tap][ci][co] * dy[p - d(tap)][co]
//                        (then * (x[p] > 0) when the conv read relu(x); then + add[p])
//   dW[ky][kx][ci][co] = sum over pixels p of X[p + d(tap)][ci] * dy[p][co]
//   db[co]             = sum over pixels p of dy[p][co]
//
// Computed separately, the input gradient and the weight gradient each read dy, and both
// read x (once as the mask, once as the weight-gradient operand). Here one tile (FR frames x
// TH rows x all W columns) stages the zero-padded windows of dy and of x in LDS once and both
// gradients are formed from them, so each tensor crosses HBM once: dy, x and the optional
// residual operand in, dx out. The weight gradient accumulates in registers over all tiles
// of a workgroup and is written as one float32 partial per workgroup; a second kernel adds
// the partials in a fixed order (deterministic, no atomics).
//
// Layouts in LDS:
//   - dy window [FR][TH+2][W+2] pixels of CO/8 16-byte slots plus zero slots (CbGeom::DSL):
//     the input gradient reads 8 consecutive channels of one tap per lane (16 bytes) as its
//     B fragment, and with 16 channels the zero slot feeds the k-steps past the 9 taps;
//   - x window [FR][TH+2][W+2] pixels of 2*CI bytes (+32 from 32 channels on); the weight
//     gradient reads its fragments, pixel-consecutive, with the LDS transpose read
//     (ds_read_b64_tr_b16), and the mask is read from it in the epilogue;
// The residual operand is read from global memory into registers before each 16-pixel
// column tile's MFMAs (a wave's read covers whole pixels, so it stays coalesced).
// The input-gradient weights (taps rotated by 180 degrees, in/out channels swapped) live in
// registers: each wave owns one 16-channel block of dx and holds its A fragments for all
// k-steps, loaded once per workgroup.
#include "common.h"
#include "kernels.h"

#include <algorithm>
#include <type_traits>

namespace cb {

template <int CI, int CO, bool SP = false>
struct CbGeom {
    // dy window: 16-byte slots per pixel, the data and one zero slot (16 channels: the k-steps
    // past the 9 taps read it), or two from 32 channels on, where a pitch of 2 (mod 4) slots
    // keeps the 16 pixels of a B-fragment read on distinct bank groups
    static constexpr int DSL = CO >= 32 ? CO / 8 + 2 : CO / 8 + 1;
    static constexpr int DYP = DSL * 16;                 // dy window: bytes per pixel
    static constexpr int XPB = CI * 2 + (CI >= 32 ? 32 : 0);   // x window: bytes per pixel
    static constexpr int XSL = XPB / 16;
    static constexpr int MTI = CI / 16, MTO = CO / 16;
    static constexpr int KSD = (9 * CO + 31) / 32;       // input-gradient k-steps
    static constexpr int NB = 9 * CI / 16;               // weight-gradient column blocks
    static constexpr int NBB = NB + 1;                   // ... and the bias block
    static constexpr int PSTRIDE = MTO * NBB * 256;      // floats per workgroup partial
    // 64 channels: the input-gradient weights (72 registers) and the weight-gradient
    // accumulators (up to 80) take the registers of two waves per SIMD, so one workgroup per CU
    // with all of the LDS (taller bands); otherwise two per CU
    static constexpr bool WIDE = CI >= 64 || CO >= 64;
    static constexpr int WPS = WIDE ? 2 : 4;
    static constexpr size_t LDS_TARGET = WIDE ? 160 * 1024 : 80 * 1024;
    // staging slots per lane (of an 8-wave workgroup) the tile planner stays within
    static constexpr int MAXD = WIDE ? 8 : (CO > CI ? 7 : 6), MAXX = WIDE || CO > CI ? (CI >= 32 ? 8 : 4) : 4;
    static constexpr int MAXT = WIDE ? 5 : (CI >= 32 ? 4 : 6);   // dx column tiles per wave and tile (with a residual)
    static constexpr int MAXP = CO >= 64 ? 4 : 3, MAXG = 2;      // pooled-gradient / argmax staging slots per lane
    // 64 channels: the waves specialise (of 8, the first half form input gradients, two dx
    // channel blocks per wave so that each B-fragment read feeds two MFMAs, the second half
    // the weight gradients), each half holding only its own registers, and run concurrently
    // on every tile. The stage entries from the pooled gradient at 16 -> 32 and 32 -> 32 (SP)
    // specialise too, one dx block per wave: their halves overlap (measured at 2048 frames:
    // 190 -> 181 us and 81 -> 76 us); otherwise every wave forms both, one dx block each (the
    // 32-channel relu/residual variants specialised were 3% slower; with two dx blocks per wave
    // they spill at four waves per SIMD)
    static constexpr bool SPEC = WIDE || (CI == 16 && CO == 32) || SP;
    static constexpr int NWD = SPEC ? 4 : 8;               // waves forming input gradients
    static constexpr int NWW = SPEC ? 4 : 8;               // ... and weight gradients
    static constexpr int DB = SPEC && WIDE && MTI >= 2 ? 2 : 1;   // dx channel blocks per input-gradient wave
    static constexpr int NCG = NWD / (MTI / DB);           // waves sharing a block group (column groups)
    __host__ __device__ static int blocks(int slots) { return (slots + 63) / 64; }
};

// the geometry of a launch: the 32 -> 32 stage entry from the pooled gradient specialises
template <int CI, int CO, int PDY>
using CbG = CbGeom<CI, CO, PDY && CI == 32 && CO == 32>;

template <int CI, int CO, int MODE, int ADD, int PDY, int NW>
__global__ __launch_bounds__(64 * NW, (CbGeom<CI, CO>::WPS)) void conv_bwd_kernel(ConvBwdArgs a, CbTile t) {
    using G = CbG<CI, CO, PDY>;
    constexpr int NT = 64 * NW;
    constexpr int DSL = G::DSL, DYP = G::DYP, XPB = G::XPB, XSL = G::XSL;
    constexpr int MTI = G::MTI, MTO = G::MTO, KSD = G::KSD, NB = G::NB, NBB = G::NBB;
    constexpr int TPW = (NBB + NW - 1) / NW;   // weight-gradient column blocks per wave
    constexpr int CB16 = CI / 16;
    static_assert(NW % MTI == 0, "waves split evenly over the dx channel blocks");
    static_assert(MODE == IN_PLAIN || MODE == IN_RELU, "bf16 activations");
    static_assert(!PDY || (!ADD && MODE == IN_PLAIN), "a pooled gradient feeds a stage-entry conv");

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;               // 64 zero bytes
    unsigned char* dyw = smem + t.dy_off;
    unsigned char* xw = smem + t.x_off + XPB;   // one zero guard pixel on either side

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar branches
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const int H = a.H, W = a.W, TH = t.TH, FR = t.FR;
    const int TW = W + 2, TR = TH + 2;

    // an earlier launch's weight-gradient partials, summed first (LDS is free until staging)
    if (a.pend.nparts > 0) pending_reduce<NT>(a.pend, smem);
    if (a.pend2.nparts > 0) pending_reduce<NT>(a.pend2, smem);
    if (tid < 16) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;
    if constexpr (PDY) {
        // the dy window is built in LDS: its padding columns and zero slots are never written
        for (int j = tid; j < (t.x_off - t.dy_off) / 16; j += NT) reinterpret_cast<uint4*>(dyw)[j] = make_uint4(0, 0, 0, 0);
    }
    // the x window's guard pixels (read only against zero dy padding, never staged)
    if (tid < XPB / 4) {
        reinterpret_cast<uint32_t*>(xw - XPB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(xw + t.x_guard)[tid] = 0u;
    }

    // ---- input gradient: this wave's dx channel block and its A fragments,
    // A[o][k] = w[8 - tap][o][co] with k = tap * CO + co (zero past the 9 taps)
    const int dmt = wave % MTI;
    const int ci0 = dmt * 16 + g * 4;   // the lane's first dx channel
    uint4 wf[KSD];
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks) {
        const int o = dmt * 16 + r16;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int k = ks * 32 + g * 8 + j, tap = k / CO, co = k % CO;
            v[j] = tap < 9 ? a.w[((8 - tap) * CI + o) * CO + co] : 0.f;
        }
        wf[ks] = make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]), pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
    }
    // its B fragments: byte offsets from the lane's tap-(0,0) dy-window pixel; with 16
    // channels a k-step spans two taps (a per-lane table), from 32 on the tap is the k-step's
    // and only the 16-byte slot is the lane's (formed in place)
    int dboff[CO < 32 ? KSD : 1];
    if constexpr (CO < 32) {
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / CO, slot = (k0 % CO) / 8;
            dboff[ks] = tap < 9 ? ((tap / 3) * TW + tap % 3) * DYP + slot * 16 : (DSL - 1) * 16;
        }
    }
    const int twdy = TW * DYP;
    auto dgrad_off = [&](int ks) -> int {
        if constexpr (CO < 32) return dboff[ks];
        else return (ks / (CO / 32) / 3) * twdy + (ks / (CO / 32) % 3) * DYP + ((ks % (CO / 32)) * 4 + g) * 16;
    };
    // ---- weight gradient: column blocks nb = wave + NW * i (16 input channels of one tap,
    // or the bias block), each for all CO/16 output-channel blocks
    int wboff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = wave + NW * i;
        const int tap = nb / CB16, cb = nb % CB16;
        wboff[i] = nb < NB ? ((tap / 3) * TW + tap % 3) * XPB + (cb * 16 + 4 * m) * 2 : 0;
    }
    cb_f32x4 wacc[TPW][MTO];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int mo = 0; mo < MTO; ++mo) wacc[i][mo] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

    // ---- staging offsets. Slot j of a window maps to the same frame / row / column of every
    // tile, so each lane's byte offsets are formed once, relative to image row 0 of the tile's
    // first frame; a tile adds h0 rows. Rows above the image come out negative and rows below
    // it past the tile's frames: both fall outside the buffer resource and read as zero.
    // Padding slots, padding columns and (multi-frame tiles) the halo rows between frames hold
    // kOOB. Slot k of this wave is j = (wave + NW * k) * 64 + lane.
    const int nsd = FR * TR * TW * DSL, nsx = FR * TR * TW * XSL;
    uint32_t od[G::MAXD], ox[G::MAXX];
    auto win_off = [&](int j, int slots, int nreal, int cbytes) -> uint32_t {
        const int p = j / slots, c = j - p * slots;
        const int rowi = p / TW, col = p - rowi * TW;
        const int f = rowi / TR, rr = rowi - f * TR;
        if (j >= FR * TR * TW * slots || c >= nreal || col < 1 || col > W) return kOOB;
        if (FR > 1 && (rr < 1 || rr > TH)) return kOOB;
        return uint32_t(((f * H + rr - 1) * W + col - 1) * cbytes + c * 16);
    };
#pragma unroll
    for (int k = 0; k < G::MAXD; ++k) od[k] = PDY ? kOOB : win_off((wave + NW * k) * 64 + lane, DSL, CO / 8, CO * 2);
    // pooled gradient / argmax rows (PDY): LDS row rr holds pooled row ib0 - 1 + rr with a zero
    // column either side; offsets relative to pooled row -1, a tile adds ib0 rows
    const int PW2 = t.OW + 2;
    const int nsp = t.PR * PW2 * (CO / 8), nsg = t.PR * PW2 * (CO / 16);
    uint32_t opd[PDY ? G::MAXP : 1], oag[PDY ? G::MAXG : 1];
    if constexpr (PDY) {
#pragma unroll
        for (int k = 0; k < G::MAXP; ++k) {
            const int j = (wave + NW * k) * 64 + lane, px = j / (CO / 8), c = j - px * (CO / 8);
            const int rr = px / PW2, col = px - rr * PW2;
            opd[k] = (j < nsp && col >= 1 && col <= t.OW) ? uint32_t((((rr - 1) * t.OW + col - 1) * CO + c * 8) * 2) : kOOB;
        }
#pragma unroll
        for (int k = 0; k < G::MAXG; ++k) {
            const int j = (wave + NW * k) * 64 + lane, px = j / (CO / 16), c = j - px * (CO / 16);
            const int rr = px / PW2, col = px - rr * PW2;
            oag[k] = (j < nsg && col >= 1 && col <= t.OW) ? uint32_t(((rr - 1) * t.OW + col - 1) * CO + c * 16) : kOOB;
        }
    }
#pragma unroll
    for (int k = 0; k < G::MAXX; ++k) ox[k] = win_off((wave + NW * k) * 64 + lane, XSL, CI / 8, CI * 2);

    int lg = blockIdx.x;   // neighbouring tiles (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int h0 = band * TH, f0 = fg * FR;
        const int nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int the = H - h0 < TH ? H - h0 : TH;
        const int npx = nf * the * W;   // FR > 1 only when a band is the whole frame
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage the dy and x windows (rows h0-1 .. h0+TH)
        {
            const int64_t fpx = int64_t(f0) * H * W;
            const auto rd = buf_rsrc(static_cast<const uint16_t*>(a.dy) + fpx * CO, uint32_t(nf) * H * W * CO * 2);
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + fpx * CI, uint32_t(nf) * H * W * CI * 2);
            const uint32_t hd = uint32_t(h0) * W * CO * 2, hx = uint32_t(h0) * W * CI * 2;
            if constexpr (PDY) {
                // pooled rows ib0-1 .. ib1 (this frame's pooled gradient and argmax)
                const int ib0 = (h0 - 1 + t.ph) >> 1;   // arithmetic shift: floor
                const uint32_t pb = uint32_t(t.OH) * t.OW * CO;
                const auto rp = buf_rsrc(static_cast<const uint16_t*>(a.dy) + int64_t(f0) * pb, pb * 2);
                const auto rg = buf_rsrc(a.arg + int64_t(f0) * pb, pb);
                const uint32_t pr = uint32_t(ib0 * t.OW * CO);   // wraps for ib0 < 0: rows off the grid
#pragma unroll
                for (int k = 0; k < G::MAXP; ++k)
                    if ((wave + NW * k) * 64 < nsp) dma16_to_lds(rp, smem + t.dp_off + (wave + NW * k) * 1024, opd[k] + 2 * pr);
#pragma unroll
                for (int k = 0; k < G::MAXG; ++k)
                    if ((wave + NW * k) * 64 < nsg) dma16_to_lds(rg, smem + t.ag_off + (wave + NW * k) * 1024, oag[k] + pr);
                // dy-window rows off the frame hold zero (no block covers every such row)
                for (int j = tid; j < TR * TW; j += NT) {
                    const int rr = j / TW, h = h0 - 1 + rr;
                    if (h < 0 || h >= H) {
                        uint4* p = reinterpret_cast<uint4*>(dyw + j * DYP);
#pragma unroll
                        for (int c = 0; c < CO / 8; ++c) p[c] = make_uint4(0, 0, 0, 0);
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < G::MAXD; ++k)
                    if ((wave + NW * k) * 64 < nsd) dma16_to_lds(rd, dyw + (wave + NW * k) * 1024, od[k] + hd);
            }
#pragma unroll
            for (int k = 0; k < G::MAXX; ++k)
                if ((wave + NW * k) * 64 < nsx) dma16_to_lds(rx, xw + (wave + NW * k) * 1024, ox[k] + hx);
        }
        // the residual operand of this wave's column tiles, fetched alongside the staging
        const int64_t tpx = (int64_t(f0) * H + h0) * W * CI;   // the tile's first dx element
        const int ntl = (npx + 15) >> 4;
        uint2 addr[ADD ? G::MAXT : 1];
        if constexpr (ADD) {
            const uint16_t* adg = static_cast<const uint16_t*>(a.add) + tpx;
#pragma unroll
            for (int k = 0; k < G::MAXT; ++k) {
                const int q = (wave / MTI + k * (NW / MTI)) * 16 + r16;
                addr[k] = q < npx ? *reinterpret_cast<const uint2*>(adg + uint32_t(q * CI + ci0)) : make_uint2(0, 0);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads have landed in LDS
        __syncthreads();                 // ... and everyone else's
        if constexpr (PDY) {
            // ---- max-pool backward into the dy window: 2x2 blocks of padded cells
            // (2i + a, 2j + b), windows (i-1 | i, j-1 | j) at LDS rows i - ib0, i - ib0 + 1 and
            // columns j, j + 1; the stand-alone pool backward's gather and summation order
            const int ib0 = (h0 - 1 + t.ph) >> 1;
            const int ib1 = min((h0 + the + t.ph) >> 1, t.BH - 1);
            const int ilo = max(ib0, 0);
            // an item is RPI block rows of one block column and 4 channels; with two, the
            // windows of the shared middle row are loaded once for both (with 32 input channels
            // the registers afford one)
            constexpr int RPI = CI < 32 ? 2 : 1;
            const int nbr = ib1 - ilo + 1;
            const int items = ((nbr + RPI - 1) / RPI) * t.BW * (CO / 4);
            const unsigned char* dpl = smem + t.dp_off;
            const unsigned char* agl = smem + t.ag_off;
            for (int it = tid; it < items; it += NT) {
                const int c4 = it % (CO / 4), blk = it / (CO / 4);
                const int bp2 = qdiv(blk, t.inv_BW), j = blk - bp2 * t.BW;
                const int i0 = ilo + RPI * bp2, lr0 = i0 - ib0;
                // window rows lr0, lr0+1 (the first block row), then lr0+2 replaces lr0 (the
                // second): the middle row is loaded once for both
                uint32_t ka[2][2], s01[2][2], s23[2][2];
                uint2 dg[2][2];   // 4 bf16 gradients
                auto load_row = [&](int slot, int lr) {
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        const int px = lr * PW2 + j + q;
                        ka[slot][q] = *reinterpret_cast<const uint32_t*>(agl + px * CO + c4 * 4);
                        dg[slot][q] = *reinterpret_cast<const uint2*>(dpl + (px * CO + c4 * 4) * 2);
                        s01[slot][q] = arg_sel01(ka[slot][q]);
                        s23[slot][q] = arg_sel23(ka[slot][q]);
                    }
                };
                load_row(0, lr0);
                load_row(1, lr0 + 1);
#pragma unroll
                for (int sb = 0; sb < RPI; ++sb) {
                    const int i = i0 + sb;
                    if (i > ib1) break;
                    if (sb == 1) load_row(0, lr0 + 2);   // rows: slot 1 = lr0+1 (top), slot 0 = lr0+2
                    const int top = sb == 0 ? 0 : 1, bot = sb == 0 ? 1 : 0;
                    // window w4's gradients where its cell is T, else +0; each cell adds its
                    // windows in (oh, ow) order, the lower-right cell has one and keeps its bf16
                    // gradient as it is
#define CB_PICK(T, w4)                                                                                 \
    arg_pick<T>(dg[((w4) >> 1) ? bot : top][(w4) & 1], ka[((w4) >> 1) ? bot : top][(w4) & 1], \
                s01[((w4) >> 1) ? bot : top][(w4) & 1], s23[((w4) >> 1) ? bot : top][(w4) & 1])
                    const uint2 a0 = CB_PICK(8, 0), a1 = CB_PICK(6, 1), a2 = CB_PICK(2, 2), a3 = CB_PICK(0, 3);
                    const uint2 b1 = CB_PICK(7, 1), b3 = CB_PICK(1, 3);
                    const uint2 e2 = CB_PICK(5, 2), e3 = CB_PICK(3, 3);
                    const uint2 c11 = CB_PICK(4, 3);
#undef CB_PICK
                    auto sum4 = [](uint32_t u0, uint32_t u1, uint32_t u2, uint32_t u3) {
                        return pack2bf(bf_lo(u0) + bf_lo(u1) + bf_lo(u2) + bf_lo(u3),
                                       bf_hi(u0) + bf_hi(u1) + bf_hi(u2) + bf_hi(u3));
                    };
                    auto sum2 = [](uint32_t u0, uint32_t u1) {
                        return pack2bf(bf_lo(u0) + bf_lo(u1), bf_hi(u0) + bf_hi(u1));
                    };
                    const uint2 c00 = make_uint2(sum4(a0.x, a1.x, a2.x, a3.x), sum4(a0.y, a1.y, a2.y, a3.y));
                    const uint2 c01 = make_uint2(sum2(b1.x, b3.x), sum2(b1.y, b3.y));
                    const uint2 c10 = make_uint2(sum2(e2.x, e3.x), sum2(e2.y, e3.y));
                    // cells -> dy-window row h - h0 + 1, column w + 1; off the frame: zero
                    const int h = 2 * i - t.ph, w = 2 * j - t.pw;
                    auto put = [&](int hh, int ww, uint2 c) {
                        const int rr = hh - h0 + 1;
                        if (rr < 0 || rr >= the + 2) return;
                        const bool in = hh >= 0 && hh < H && ww >= 0 && ww < W;
                        *reinterpret_cast<uint2*>(dyw + (rr * TW + ww + 1) * DYP + c4 * 8) = in ? c : make_uint2(0, 0);
                    };
                    put(h, w, c00);
                    put(h, w + 1, c01);
                    put(h + 1, w, c10);
                    put(h + 1, w + 1, c11);
                }
            }
            __syncthreads();
        }
        if constexpr (MODE == IN_RELU) {
            // the conv read relu(x); relu(x) > 0 exactly where x > 0, so the mask reads it too
            uint4* w4 = reinterpret_cast<uint4*>(xw);
            for (int j = tid; j < FR * TR * TW * XSL; j += NT) {
                uint4 v = w4[j];
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                w4[j] = v;
            }
            __syncthreads();
        }

        // ---- weight gradient over the band's window rows, padding columns included (dy is
        // zero there, so they add nothing): pixel p = TW + ks*32 + o of the dy window pairs with
        // x-window pixel p - TW - 1 + tap, and every address advances by a constant per k-step.
        // Lane (g, 4jj+m) takes pixels o = 16*half + 4g + jj (dy / x channels 4m.. of a block).
        // Between frames of a multi-frame tile the two halo rows are outside the image: zero dy.
        // With 16 output channels, specialised per wave, so that each column block's kind
        // (loaded or bias) is known at compile time and the k-step loop carries no branches.
        {
            const int L = ((nf - 1) * TR + the) * TW;   // contracted window pixels
            auto run = [&](auto wv) {
                const int WV = wv;   // a compile-time constant when specialised
                const int nfull = L >> 5;
                const int o0 = 4 * g + jj;
                const unsigned char* ap = dyw + (TW + o0) * DYP + 8 * m;
                const unsigned char* bp = xw + (o0 - 1) * XPB;
                auto kstep = [&](const unsigned char* a0, const unsigned char* a1, const unsigned char* b0,
                                 const unsigned char* b1) {
                    uint4 af[MTO];
#pragma unroll
                    for (int mo = 0; mo < MTO; ++mo) {
                        const uint2 lo = lds_read_tr16(a0 + mo * 32);   // a0, a1: zero for pixels past L
                        const uint2 hi = lds_read_tr16(a1 + mo * 32);
                        af[mo] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                    }
#pragma unroll
                    for (int i = 0; i < TPW; ++i) {
                        const int nb = WV + NW * i;
                        if constexpr (MTO == 1) {
                            if (nb < NB) {
                                const uint2 lo = lds_read_tr16(b0 + wboff[i]);
                                const uint2 hi = lds_read_tr16(b1 + wboff[i]);
                                wacc[i][0] = PrecBF16::mma(af[0], make_uint4(lo.x, lo.y, hi.x, hi.y), wacc[i][0]);
                            } else if (nb == NB) {   // the bias block: a column of ones
                                wacc[i][0] = PrecBF16::mma(af[0], ones, wacc[i][0]);
                            }
                        } else {
                            if (nb >= NBB) continue;
                            uint4 bf = ones;   // the bias block: a column of ones
                            if (nb < NB) {
                                const uint2 lo = lds_read_tr16(b0 + wboff[i]);
                                const uint2 hi = lds_read_tr16(b1 + wboff[i]);
                                bf = make_uint4(lo.x, lo.y, hi.x, hi.y);
                            }
#pragma unroll
                            for (int mo = 0; mo < MTO; ++mo) wacc[i][mo] = PrecBF16::mma(af[mo], bf, wacc[i][mo]);
                        }
                    }
                };
                int ks = 0;
                if constexpr (MTO == 1) {   // two k-steps per trip: half the pointer updates
                    for (; ks + 2 <= nfull; ks += 2) {
                        kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                        kstep(ap + 32 * DYP, ap + 48 * DYP, bp + 32 * XPB, bp + 48 * XPB);
                        ap += 64 * DYP;
                        bp += 64 * XPB;
                    }
                }
                for (; ks < nfull; ++ks) {
                    kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                    ap += 32 * DYP;
                    bp += 32 * XPB;
                }
                if (L & 31) {   // the last, partial k-step: pixels past L read zero dy
                    const int o = nfull * 32 + o0;
                    const bool ok0 = o < L, ok1 = o + 16 < L;
                    kstep(ok0 ? ap : zero, ok1 ? ap + 16 * DYP : zero, ok0 ? bp : xw - XPB,
                          ok1 ? bp + 16 * XPB : xw - XPB);
                }
            };
            if constexpr (MTO == 1) {
                static_assert(NW == 8, "one specialisation per wave");
                switch (wave) {
                    case 0: run(std::integral_constant<int, 0>{}); break;
                    case 1: run(std::integral_constant<int, 1>{}); break;
                    case 2: run(std::integral_constant<int, 2>{}); break;
                    case 3: run(std::integral_constant<int, 3>{}); break;
                    case 4: run(std::integral_constant<int, 4>{}); break;
                    case 5: run(std::integral_constant<int, 5>{}); break;
                    case 6: run(std::integral_constant<int, 6>{}); break;
                    default: run(std::integral_constant<int, 7>{}); break;
                }
            } else {
                run(wave);   // 32 output channels: the registers afford no specialised copies
            }
        }

        // ---- input gradient: 16-pixel column tiles of this wave's dx channel block. Band pixel
        // q sits at window row q / W (+ 2 per earlier frame of a multi-frame tile), and dx and
        // the residual operand are addressed by q itself from the tile's first pixel.
        {
            uint16_t* dxt = static_cast<uint16_t*>(a.dx) + tpx;
            auto column_tile = [&](int nt, uint2 addv) {
                const int q = nt * 16 + r16;
                const int qc = q < npx ? q : npx - 1;   // past npx: computed, not stored
                const int row = qdiv(qc, t.inv_W), col = qc - row * W;
                const int wrow = FR > 1 ? row + 2 * qdiv(row, t.inv_TH) : row;
                const int wpx = wrow * TW + col;
                const unsigned char* xb = dyw + wpx * DYP;
                cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks)
                    acc = PrecBF16::mma(wf[ks], *reinterpret_cast<const uint4*>(xb + dgrad_off(ks)), acc);
                if (q < npx) {
                    float v[4] = {acc[0], acc[1], acc[2], acc[3]};
                    if constexpr (MODE == IN_RELU) {
                        float mk[4];
                        load4(reinterpret_cast<const uint16_t*>(xw + (wpx + TW + 1) * XPB + ci0 * 2), mk);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] = mk[j] > 0.f ? v[j] : 0.f;
                    }
                    if constexpr (ADD) {
                        v[0] += __uint_as_float(addv.x << 16);
                        v[1] += __uint_as_float(addv.x & 0xffff0000u);
                        v[2] += __uint_as_float(addv.y << 16);
                        v[3] += __uint_as_float(addv.y & 0xffff0000u);
                    }
                    store4(dxt + uint32_t(q * CI + ci0), v[0], v[1], v[2], v[3]);
                }
            };
            if constexpr (ADD) {
#pragma unroll
                for (int k = 0; k < G::MAXT; ++k)
                    if (wave / MTI + k * (NW / MTI) < ntl) column_tile(wave / MTI + k * (NW / MTI), addr[k]);
            } else {
                for (int nt = wave / MTI; nt < ntl; nt += NW / MTI) column_tile(nt, make_uint2(0, 0));
            }
        }
    }

    // ---- this workgroup's weight-gradient partial: [mo*NBB + nb][row co 16][col ci 16]
    float* part = a.partial + int64_t(blockIdx.x) * G::PSTRIDE;
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = wave + NW * i;
        if (nb < NBB) {
#pragma unroll
            for (int mo = 0; mo < MTO; ++mo)
#pragma unroll
                for (int e = 0; e < 4; ++e) part[(mo * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = wacc[i][mo][e];
        }
    }
}

// The same backward with specialised waves, for 64 channels (one workgroup per CU) and the
// 16 -> 32 stage entry (two per CU). There every wave forming both gradients reads each
// input-gradient B fragment for one dx channel block (1 KB of LDS per MFMA, more than the LDS
// delivers at the matrix cores' rate) and holds the weight-gradient accumulators beside the
// input-gradient weights. Here the first half of the waves forms the input gradient, two dx
// channel blocks per wave where there are two or more (at 64 channels 144 registers of
// weights, each B fragment feeding two MFMAs), and the second half the weight gradients, each
// for a quarter of the column blocks against all output channels; the halves run
// concurrently on every tile, in two loops, so each keeps only its own registers live.
// Staging, the max-pool backward and the relu pass are shared, with the same barriers.
template <int CI, int CO, int MODE, int ADD, int PDY, int NW>
__global__ __launch_bounds__(64 * NW, (CbGeom<CI, CO>::WPS)) void conv_bwd_spec_kernel(ConvBwdArgs a, CbTile t) {
    using G = CbG<CI, CO, PDY>;
    constexpr int NT = 64 * NW;
    constexpr int DSL = G::DSL, DYP = G::DYP, XPB = G::XPB, XSL = G::XSL;
    constexpr int MTI = G::MTI, MTO = G::MTO, KSD = G::KSD, NB = G::NB, NBB = G::NBB;
    constexpr int NWW = G::NWW, DB = G::DB, NCG = G::NCG, NBG = MTI / DB;
    constexpr int TPW = (NBB + NWW - 1) / NWW;   // weight-gradient column blocks per wave
    constexpr int CB16 = CI / 16;
    static_assert(G::SPEC && NW == 8 && G::NWD % NBG == 0 && MTI % DB == 0, "waves split evenly over the dx channel blocks");
    static_assert(MODE == IN_PLAIN || MODE == IN_RELU, "bf16 activations");
    static_assert(!PDY || (!ADD && MODE == IN_PLAIN), "a pooled gradient feeds a stage-entry conv");

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;               // 64 zero bytes
    unsigned char* dyw = smem + t.dy_off;
    unsigned char* xw = smem + t.x_off + XPB;   // one zero guard pixel on either side

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar branches
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const int H = a.H, W = a.W, TH = t.TH, FR = t.FR;
    const int TW = W + 2, TR = TH + 2;

    // an earlier launch's weight-gradient partials, summed first (LDS is free until staging)
    if (a.pend.nparts > 0) pending_reduce<NT>(a.pend, smem);
    if (a.pend2.nparts > 0) pending_reduce<NT>(a.pend2, smem);
    if (tid < 16) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;
    if constexpr (PDY) {
        // the dy window is built in LDS: its padding columns and zero slots are never written
        for (int j = tid; j < (t.x_off - t.dy_off) / 16; j += NT) reinterpret_cast<uint4*>(dyw)[j] = make_uint4(0, 0, 0, 0);
    }
    // the x window's guard pixels (read only against zero dy padding, never staged)
    if (tid < XPB / 4) {
        reinterpret_cast<uint32_t*>(xw - XPB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(xw + t.x_guard)[tid] = 0u;
    }

    // ---- input gradient: this wave's dx channel block and its A fragments,
    // A[o][k] = w[8 - tap][o][co] with k = tap * CO + co (zero past the 9 taps)
    // (specialised: waves 0 .. NWD-1 form the input gradient, NWD .. NW-1 the weight gradient)
    const bool is_dg = wave < G::NWD;
    const int wd = wave;                          // input-gradient wave index
    const int ww = wave - G::NWD;   // weight-gradient wave index
    const int dmt = (wd % NBG) * DB;              // the wave's first dx channel block
    const int ci0 = dmt * 16 + g * 4;             // the lane's first dx channel
    auto load_wf = [&](uint4 (&wf)[DB][KSD]) {
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
            for (int ks = 0; ks < KSD; ++ks) {
                const int o = (dmt + b) * 16 + r16;
                float v[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int k = ks * 32 + g * 8 + j, tap = k / CO, co = k % CO;
                    v[j] = tap < 9 ? a.w[((8 - tap) * CI + o) * CO + co] : 0.f;
                }
                wf[b][ks] = make_uint4(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]), pack2bf(v[4], v[5]), pack2bf(v[6], v[7]));
            }
    };
    // its B fragments: byte offsets from the lane's tap-(0,0) dy-window pixel; with 16
    // channels a k-step spans two taps (a per-lane table), from 32 on the tap is the k-step's
    // and only the 16-byte slot is the lane's (formed in place)
    int dboff[CO < 32 ? KSD : 1];
    if constexpr (CO < 32) {
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / CO, slot = (k0 % CO) / 8;
            dboff[ks] = tap < 9 ? ((tap / 3) * TW + tap % 3) * DYP + slot * 16 : (DSL - 1) * 16;
        }
    }
    const int twdy = TW * DYP;
    auto dgrad_off = [&](int ks) -> int {
        if constexpr (CO < 32) return dboff[ks];
        else return (ks / (CO / 32) / 3) * twdy + (ks / (CO / 32) % 3) * DYP + ((ks % (CO / 32)) * 4 + g) * 16;
    };
    // ---- weight gradient: column blocks nb = wave + NW * i (16 input channels of one tap,
    // or the bias block), each for all CO/16 output-channel blocks
    int wboff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = ww + NWW * i;
        const int tap = nb / CB16, cb = nb % CB16;
        wboff[i] = nb < NB ? ((tap / 3) * TW + tap % 3) * XPB + (cb * 16 + 4 * m) * 2 : 0;
    }
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

    // ---- staging offsets. Slot j of a window maps to the same frame / row / column of every
    // tile, so each lane's byte offsets are formed once, relative to image row 0 of the tile's
    // first frame; a tile adds h0 rows. Rows above the image come out negative and rows below
    // it past the tile's frames: both fall outside the buffer resource and read as zero.
    // Padding slots, padding columns and (multi-frame tiles) the halo rows between frames hold
    // kOOB. Slot k of this wave is j = (wave + NW * k) * 64 + lane.
    const int nsd = FR * TR * TW * DSL, nsx = FR * TR * TW * XSL;
    uint32_t od[G::MAXD], ox[G::MAXX];
    auto win_off = [&](int j, int slots, int nreal, int cbytes) -> uint32_t {
        const int p = j / slots, c = j - p * slots;
        const int rowi = p / TW, col = p - rowi * TW;
        const int f = rowi / TR, rr = rowi - f * TR;
        if (j >= FR * TR * TW * slots || c >= nreal || col < 1 || col > W) return kOOB;
        if (FR > 1 && (rr < 1 || rr > TH)) return kOOB;
        return uint32_t(((f * H + rr - 1) * W + col - 1) * cbytes + c * 16);
    };
#pragma unroll
    for (int k = 0; k < G::MAXD; ++k) od[k] = PDY ? kOOB : win_off((wave + NW * k) * 64 + lane, DSL, CO / 8, CO * 2);
    // pooled gradient / argmax rows (PDY): LDS row rr holds pooled row ib0 - 1 + rr with a zero
    // column either side; offsets relative to pooled row -1, a tile adds ib0 rows
    const int PW2 = t.OW + 2;
    const int nsp = t.PR * PW2 * (CO / 8), nsg = t.PR * PW2 * (CO / 16);
    uint32_t opd[PDY ? G::MAXP : 1], oag[PDY ? G::MAXG : 1];
    if constexpr (PDY) {
#pragma unroll
        for (int k = 0; k < G::MAXP; ++k) {
            const int j = (wave + NW * k) * 64 + lane, px = j / (CO / 8), c = j - px * (CO / 8);
            const int rr = px / PW2, col = px - rr * PW2;
            opd[k] = (j < nsp && col >= 1 && col <= t.OW) ? uint32_t((((rr - 1) * t.OW + col - 1) * CO + c * 8) * 2) : kOOB;
        }
#pragma unroll
        for (int k = 0; k < G::MAXG; ++k) {
            const int j = (wave + NW * k) * 64 + lane, px = j / (CO / 16), c = j - px * (CO / 16);
            const int rr = px / PW2, col = px - rr * PW2;
            oag[k] = (j < nsg && col >= 1 && col <= t.OW) ? uint32_t(((rr - 1) * t.OW + col - 1) * CO + c * 16) : kOOB;
        }
    }
#pragma unroll
    for (int k = 0; k < G::MAXX; ++k) ox[k] = win_off((wave + NW * k) * 64 + lane, XSL, CI / 8, CI * 2);

    int lg = blockIdx.x;   // neighbouring tiles (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    // ---- a tile's staging, its waits and barriers, the max-pool backward and the relu pass:
    // every wave runs them (in either role), so all waves meet the same barriers. `mid` runs
    // between the staging loads' issue and the wait for them.
    auto prologue = [&](int tile, auto&& mid) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int h0 = band * TH, f0 = fg * FR;
        const int nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int the = H - h0 < TH ? H - h0 : TH;
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage the dy and x windows (rows h0-1 .. h0+TH)
        {
            const int64_t fpx = int64_t(f0) * H * W;
            const auto rd = buf_rsrc(static_cast<const uint16_t*>(a.dy) + fpx * CO, uint32_t(nf) * H * W * CO * 2);
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + fpx * CI, uint32_t(nf) * H * W * CI * 2);
            const uint32_t hd = uint32_t(h0) * W * CO * 2, hx = uint32_t(h0) * W * CI * 2;
            if constexpr (PDY) {
                // pooled rows ib0-1 .. ib1 (this frame's pooled gradient and argmax)
                const int ib0 = (h0 - 1 + t.ph) >> 1;   // arithmetic shift: floor
                const uint32_t pb = uint32_t(t.OH) * t.OW * CO;
                const auto rp = buf_rsrc(static_cast<const uint16_t*>(a.dy) + int64_t(f0) * pb, pb * 2);
                const auto rg = buf_rsrc(a.arg + int64_t(f0) * pb, pb);
                const uint32_t pr = uint32_t(ib0 * t.OW * CO);   // wraps for ib0 < 0: rows off the grid
#pragma unroll
                for (int k = 0; k < G::MAXP; ++k)
                    if ((wave + NW * k) * 64 < nsp) dma16_to_lds(rp, smem + t.dp_off + (wave + NW * k) * 1024, opd[k] + 2 * pr);
#pragma unroll
                for (int k = 0; k < G::MAXG; ++k)
                    if ((wave + NW * k) * 64 < nsg) dma16_to_lds(rg, smem + t.ag_off + (wave + NW * k) * 1024, oag[k] + pr);
                // dy-window rows off the frame hold zero (no block covers every such row)
                for (int j = tid; j < TR * TW; j += NT) {
                    const int rr = j / TW, h = h0 - 1 + rr;
                    if (h < 0 || h >= H) {
                        uint4* p = reinterpret_cast<uint4*>(dyw + j * DYP);
#pragma unroll
                        for (int c = 0; c < CO / 8; ++c) p[c] = make_uint4(0, 0, 0, 0);
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < G::MAXD; ++k)
                    if ((wave + NW * k) * 64 < nsd) dma16_to_lds(rd, dyw + (wave + NW * k) * 1024, od[k] + hd);
            }
#pragma unroll
            for (int k = 0; k < G::MAXX; ++k)
                if ((wave + NW * k) * 64 < nsx) dma16_to_lds(rx, xw + (wave + NW * k) * 1024, ox[k] + hx);
        }
        mid();
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads have landed in LDS
        __syncthreads();                 // ... and everyone else's
        if constexpr (PDY) {
            // ---- max-pool backward into the dy window: 2x2 blocks of padded cells
            // (2i + a, 2j + b), windows (i-1 | i, j-1 | j) at LDS rows i - ib0, i - ib0 + 1 and
            // columns j, j + 1; the stand-alone pool backward's gather and summation order
            const int ib0 = (h0 - 1 + t.ph) >> 1;
            const int ib1 = min((h0 + the + t.ph) >> 1, t.BH - 1);
            const int ilo = max(ib0, 0);
            // an item is RPI block rows of one block column and 4 channels; with two, the
            // windows of the shared middle row are loaded once for both (with 32 input channels
            // the registers afford one)
            constexpr int RPI = CI < 32 ? 2 : 1;
            const int nbr = ib1 - ilo + 1;
            const int items = ((nbr + RPI - 1) / RPI) * t.BW * (CO / 4);
            const unsigned char* dpl = smem + t.dp_off;
            const unsigned char* agl = smem + t.ag_off;
            for (int it = tid; it < items; it += NT) {
                const int c4 = it % (CO / 4), blk = it / (CO / 4);
                const int bp2 = qdiv(blk, t.inv_BW), j = blk - bp2 * t.BW;
                const int i0 = ilo + RPI * bp2, lr0 = i0 - ib0;
                // window rows lr0, lr0+1 (the first block row), then lr0+2 replaces lr0 (the
                // second): the middle row is loaded once for both
                uint32_t ka[2][2], s01[2][2], s23[2][2];
                uint2 dg[2][2];   // 4 bf16 gradients
                auto load_row = [&](int slot, int lr) {
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        const int px = lr * PW2 + j + q;
                        ka[slot][q] = *reinterpret_cast<const uint32_t*>(agl + px * CO + c4 * 4);
                        dg[slot][q] = *reinterpret_cast<const uint2*>(dpl + (px * CO + c4 * 4) * 2);
                        s01[slot][q] = arg_sel01(ka[slot][q]);
                        s23[slot][q] = arg_sel23(ka[slot][q]);
                    }
                };
                load_row(0, lr0);
                load_row(1, lr0 + 1);
#pragma unroll
                for (int sb = 0; sb < RPI; ++sb) {
                    const int i = i0 + sb;
                    if (i > ib1) break;
                    if (sb == 1) load_row(0, lr0 + 2);   // rows: slot 1 = lr0+1 (top), slot 0 = lr0+2
                    const int top = sb == 0 ? 0 : 1, bot = sb == 0 ? 1 : 0;
                    // window w4's gradients where its cell is T, else +0; each cell adds its
                    // windows in (oh, ow) order, the lower-right cell has one and keeps its bf16
                    // gradient as it is
#define CB_PICK(T, w4)                                                                                 \
    arg_pick<T>(dg[((w4) >> 1) ? bot : top][(w4) & 1], ka[((w4) >> 1) ? bot : top][(w4) & 1], \
                s01[((w4) >> 1) ? bot : top][(w4) & 1], s23[((w4) >> 1) ? bot : top][(w4) & 1])
                    const uint2 a0 = CB_PICK(8, 0), a1 = CB_PICK(6, 1), a2 = CB_PICK(2, 2), a3 = CB_PICK(0, 3);
                    const uint2 b1 = CB_PICK(7, 1), b3 = CB_PICK(1, 3);
                    const uint2 e2 = CB_PICK(5, 2), e3 = CB_PICK(3, 3);
                    const uint2 c11 = CB_PICK(4, 3);
#undef CB_PICK
                    auto sum4 = [](uint32_t u0, uint32_t u1, uint32_t u2, uint32_t u3) {
                        return pack2bf(bf_lo(u0) + bf_lo(u1) + bf_lo(u2) + bf_lo(u3),
                                       bf_hi(u0) + bf_hi(u1) + bf_hi(u2) + bf_hi(u3));
                    };
                    auto sum2 = [](uint32_t u0, uint32_t u1) {
                        return pack2bf(bf_lo(u0) + bf_lo(u1), bf_hi(u0) + bf_hi(u1));
                    };
                    const uint2 c00 = make_uint2(sum4(a0.x, a1.x, a2.x, a3.x), sum4(a0.y, a1.y, a2.y, a3.y));
                    const uint2 c01 = make_uint2(sum2(b1.x, b3.x), sum2(b1.y, b3.y));
                    const uint2 c10 = make_uint2(sum2(e2.x, e3.x), sum2(e2.y, e3.y));
                    // cells -> dy-window row h - h0 + 1, column w + 1; off the frame: zero
                    const int h = 2 * i - t.ph, w = 2 * j - t.pw;
                    auto put = [&](int hh, int ww, uint2 c) {
                        const int rr = hh - h0 + 1;
                        if (rr < 0 || rr >= the + 2) return;
                        const bool in = hh >= 0 && hh < H && ww >= 0 && ww < W;
                        *reinterpret_cast<uint2*>(dyw + (rr * TW + ww + 1) * DYP + c4 * 8) = in ? c : make_uint2(0, 0);
                    };
                    put(h, w, c00);
                    put(h, w + 1, c01);
                    put(h + 1, w, c10);
                    put(h + 1, w + 1, c11);
                }
            }
            __syncthreads();
        }
        if constexpr (MODE == IN_RELU) {
            // the conv read relu(x); relu(x) > 0 exactly where x > 0, so the mask reads it too
            uint4* w4 = reinterpret_cast<uint4*>(xw);
            for (int j = tid; j < FR * TR * TW * XSL; j += NT) {
                uint4 v = w4[j];
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                w4[j] = v;
            }
            __syncthreads();
        }

    };
    (void)FR;

    // ---- weight gradients of one tile, into this wave's accumulators
    auto wgrad_tile = [&](int tile, cb_f32x4 (&wacc)[TPW][MTO]) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int f0 = fg * FR, h0 = band * TH;
        const int nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int the = H - h0 < TH ? H - h0 : TH;
        (void)h0;
        // ---- weight gradient over the band's window rows, padding columns included (dy is
        // zero there, so they add nothing): pixel p = TW + ks*32 + o of the dy window pairs with
        // x-window pixel p - TW - 1 + tap, and every address advances by a constant per k-step.
        // Lane (g, 4jj+m) takes pixels o = 16*half + 4g + jj (dy / x channels 4m.. of a block).
        // Between frames of a multi-frame tile the two halo rows are outside the image: zero dy.
        // With 16 output channels, specialised per wave, so that each column block's kind
        // (loaded or bias) is known at compile time and the k-step loop carries no branches.
        {
            const int L = ((nf - 1) * TR + the) * TW;   // contracted window pixels
            auto run = [&](auto wv) {
                const int WV = wv;   // a compile-time constant when specialised
                const int nfull = L >> 5;
                const int o0 = 4 * g + jj;
                const unsigned char* ap = dyw + (TW + o0) * DYP + 8 * m;
                const unsigned char* bp = xw + (o0 - 1) * XPB;
                auto kstep = [&](const unsigned char* a0, const unsigned char* a1, const unsigned char* b0,
                                 const unsigned char* b1) {
                    uint4 af[MTO];
#pragma unroll
                    for (int mo = 0; mo < MTO; ++mo) {
                        const uint2 lo = lds_read_tr16(a0 + mo * 32);   // a0, a1: zero for pixels past L
                        const uint2 hi = lds_read_tr16(a1 + mo * 32);
                        af[mo] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                    }
#pragma unroll
                    for (int i = 0; i < TPW; ++i) {
                        const int nb = WV + NWW * i;
                        if constexpr (MTO == 1) {
                            if (nb < NB) {
                                const uint2 lo = lds_read_tr16(b0 + wboff[i]);
                                const uint2 hi = lds_read_tr16(b1 + wboff[i]);
                                wacc[i][0] = PrecBF16::mma(af[0], make_uint4(lo.x, lo.y, hi.x, hi.y), wacc[i][0]);
                            } else if (nb == NB) {   // the bias block: a column of ones
                                wacc[i][0] = PrecBF16::mma(af[0], ones, wacc[i][0]);
                            }
                        } else {
                            if (nb >= NBB) continue;
                            uint4 bf = ones;   // the bias block: a column of ones
                            if (nb < NB) {
                                const uint2 lo = lds_read_tr16(b0 + wboff[i]);
                                const uint2 hi = lds_read_tr16(b1 + wboff[i]);
                                bf = make_uint4(lo.x, lo.y, hi.x, hi.y);
                            }
#pragma unroll
                            for (int mo = 0; mo < MTO; ++mo) wacc[i][mo] = PrecBF16::mma(af[mo], bf, wacc[i][mo]);
                        }
                    }
                };
                int ks = 0;
                if constexpr (MTO == 1) {   // two k-steps per trip: half the pointer updates
                    for (; ks + 2 <= nfull; ks += 2) {
                        kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                        kstep(ap + 32 * DYP, ap + 48 * DYP, bp + 32 * XPB, bp + 48 * XPB);
                        ap += 64 * DYP;
                        bp += 64 * XPB;
                    }
                }
                for (; ks < nfull; ++ks) {
                    kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                    ap += 32 * DYP;
                    bp += 32 * XPB;
                }
                if (L & 31) {   // the last, partial k-step: pixels past L read zero dy
                    const int o = nfull * 32 + o0;
                    const bool ok0 = o < L, ok1 = o + 16 < L;
                    kstep(ok0 ? ap : zero, ok1 ? ap + 16 * DYP : zero, ok0 ? bp : xw - XPB,
                          ok1 ? bp + 16 * XPB : xw - XPB);
                }
            };
            if constexpr (MTO == 1) {
                static_assert(NWW == 8, "one specialisation per wave");
                switch (ww) {
                    case 0: run(std::integral_constant<int, 0>{}); break;
                    case 1: run(std::integral_constant<int, 1>{}); break;
                    case 2: run(std::integral_constant<int, 2>{}); break;
                    case 3: run(std::integral_constant<int, 3>{}); break;
                    case 4: run(std::integral_constant<int, 4>{}); break;
                    case 5: run(std::integral_constant<int, 5>{}); break;
                    case 6: run(std::integral_constant<int, 6>{}); break;
                    default: run(std::integral_constant<int, 7>{}); break;
                }
            } else {
                run(ww);   // 32 output channels: the registers afford no specialised copies
            }
        }

    };

    // ---- input gradient: 16-pixel column tiles of the wave's DB dx channel blocks (each B
    // fragment feeds DB MFMAs). Band pixel q sits at window row q / W (+ 2 per earlier frame of a
    // multi-frame tile), and dx and the residual operand are addressed by q itself from the
    // tile's first pixel. The residual of the wave's first MAXT column tiles is fetched with
    // the staging (prefetch).
    auto tile_span = [&](int tile, int& npx, int64_t& tpx) {
        const int band = tile % t.nbands, fg = tile / t.nbands;
        const int h0 = band * TH, f0 = fg * FR;
        const int nf = a.n - f0 < FR ? a.n - f0 : FR;
        const int the = H - h0 < TH ? H - h0 : TH;
        npx = nf * the * W;   // FR > 1 only when a band is the whole frame
        tpx = (int64_t(f0) * H + h0) * W * CI;   // the tile's first dx element
    };
    auto prefetch = [&](int tile, uint2 (&addr)[ADD ? G::MAXT : 1][DB]) {
        if constexpr (ADD) {
            int npx;
            int64_t tpx;
            tile_span(tile, npx, tpx);
            const uint16_t* adg = static_cast<const uint16_t*>(a.add) + tpx;
#pragma unroll
            for (int k = 0; k < G::MAXT; ++k) {
                const int q = (wd / NBG + k * NCG) * 16 + r16;
#pragma unroll
                for (int b = 0; b < DB; ++b)
                    addr[k][b] = q < npx ? *reinterpret_cast<const uint2*>(adg + uint32_t(q * CI + ci0 + b * 16)) : make_uint2(0, 0);
            }
        }
    };
    auto dgrad_tile = [&](int tile, const uint4 (&wf)[DB][KSD], const uint2 (&addr)[ADD ? G::MAXT : 1][DB]) {
        int npx;
        int64_t tpx;
        tile_span(tile, npx, tpx);
        const int ntl = (npx + 15) >> 4;
        uint16_t* dxt = static_cast<uint16_t*>(a.dx) + tpx;
        auto column_tile = [&](int nt, const uint2* addv) {
            const int q = nt * 16 + r16;
            const int qc = q < npx ? q : npx - 1;   // past npx: computed, not stored
            const int row = qdiv(qc, t.inv_W), col = qc - row * W;
            const int wrow = FR > 1 ? row + 2 * qdiv(row, t.inv_TH) : row;
            const int wpx = wrow * TW + col;
            const unsigned char* xb = dyw + wpx * DYP;
            cb_f32x4 acc[DB];
#pragma unroll
            for (int b = 0; b < DB; ++b) acc[b] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KSD; ++ks) {
                const uint4 bf = *reinterpret_cast<const uint4*>(xb + dgrad_off(ks));
#pragma unroll
                for (int b = 0; b < DB; ++b) acc[b] = PrecBF16::mma(wf[b][ks], bf, acc[b]);
            }
            if (q < npx) {
#pragma unroll
                for (int b = 0; b < DB; ++b) {
                    float v[4] = {acc[b][0], acc[b][1], acc[b][2], acc[b][3]};
                    if constexpr (MODE == IN_RELU) {
                        float mk[4];
                        load4(reinterpret_cast<const uint16_t*>(xw + (wpx + TW + 1) * XPB + (ci0 + b * 16) * 2), mk);
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] = mk[j] > 0.f ? v[j] : 0.f;
                    }
                    if constexpr (ADD) {
                        v[0] += __uint_as_float(addv[b].x << 16);
                        v[1] += __uint_as_float(addv[b].x & 0xffff0000u);
                        v[2] += __uint_as_float(addv[b].y << 16);
                        v[3] += __uint_as_float(addv[b].y & 0xffff0000u);
                    }
                    store4(dxt + uint32_t(q * CI + ci0 + b * 16), v[0], v[1], v[2], v[3]);
                }
            }
        };
        if constexpr (ADD) {
#pragma unroll
            for (int k = 0; k < G::MAXT; ++k)
                if (wd / NBG + k * NCG < ntl) column_tile(wd / NBG + k * NCG, addr[k]);
        } else {
            for (int nt = wd / NBG; nt < ntl; nt += NCG) column_tile(nt, nullptr);
        }
    };

    // ---- this workgroup's weight-gradient partial: [mo*NBB + nb][row co 16][col ci 16]
    auto write_partial = [&](const cb_f32x4 (&wacc)[TPW][MTO]) {
        float* part = a.partial + int64_t(blockIdx.x) * G::PSTRIDE;
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const int nb = ww + NWW * i;
            if (nb < NBB) {
#pragma unroll
                for (int mo = 0; mo < MTO; ++mo)
#pragma unroll
                    for (int e = 0; e < 4; ++e) part[(mo * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = wacc[i][mo][e];
            }
        }
    };
    auto zero_acc = [&](cb_f32x4 (&wacc)[TPW][MTO]) {
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int mo = 0; mo < MTO; ++mo) wacc[i][mo] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    };

    // two loops over the same tiles, one per role, so that each role's registers (the
    // input-gradient weights, the weight-gradient accumulators) are live only in its own
    if (is_dg) {
        uint4 wf[DB][KSD];
        load_wf(wf);
        for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
            uint2 addr[ADD ? G::MAXT : 1][DB];
            prologue(tile, [&] { prefetch(tile, addr); });
            dgrad_tile(tile, wf, addr);
        }
    } else {
        cb_f32x4 wacc[TPW][MTO];
        zero_acc(wacc);
        for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
            prologue(tile, [] {});
            wgrad_tile(tile, wacc);
        }
        write_partial(wacc);
    }
}

namespace {

constexpr int kCbWaves = 8;
constexpr int kCbPixMax = 2048;
constexpr size_t kCbPartBytes = 24u << 20;

template <int CI, int CO>
int cb_parts_cap() {
    const size_t cap = kCbPartBytes / (size_t(CbGeom<CI, CO>::PSTRIDE) * sizeof(float));
    return int(cap < 256 ? 256 : (cap > 1024 ? 1024 : cap));
}

template <int CI, int CO, int MODE, int ADD, int PDY>
hipError_t cb_launch(const ConvBwdArgs& a, hipStream_t s, PendingReduce* deferred) {
    using G = CbG<CI, CO, PDY>;
    const int H = a.H, W = a.W;
    // max-pool geometry of a pooled input gradient (PDY): XLA SAME padding split
    const int OH = (H + 1) / 2, OW = (W + 1) / 2;
    const int PH = (OH - 1) * 2 + 3 - H, PWd = (OW - 1) * 2 + 3 - W;
    const int ph = (PH > 0 ? PH : 0) / 2, pw = (PWd > 0 ? PWd : 0) / 2;
    auto prows = [](int th) { return (th + 1) / 2 + 3; };   // pooled rows a band reads
    auto regions = [&](int th, int fr, int& dyb, int& xb, int& pb, int& gb) {
        const int wp = fr * (th + 2) * (W + 2);
        dyb = G::blocks(wp * G::DSL) * 1024;
        xb = G::blocks(wp * G::XSL) * 1024 + 2 * G::XPB;   // + a guard pixel on either side
        pb = PDY ? G::blocks(prows(th) * (OW + 2) * (CO / 8)) * 1024 : 0;
        gb = PDY ? G::blocks(prows(th) * (OW + 2) * (CO / 16)) * 1024 : 0;
    };
    auto lds = [&](int th, int fr) {
        int dyb, xb, pb, gb;
        regions(th, fr, dyb, xb, pb, gb);
        return size_t(64 + dyb + xb + pb + gb);
    };
    // staging slots per lane within the kernel's register tables
    auto fits = [&](int th, int fr) {
        const int per = kCbWaves * 64, wp = fr * (th + 2) * (W + 2);
        const int tiles = (fr * th * W + 15) / 16;   // dx column tiles, shared by NCG waves per block group
        return (PDY || (wp * G::DSL + per - 1) / per <= G::MAXD) && (wp * G::XSL + per - 1) / per <= G::MAXX &&
               (!ADD || (tiles + G::NCG - 1) / G::NCG <= G::MAXT) &&
               (!PDY || (fr == 1 && (prows(th) * (OW + 2) * (CO / 8) + per - 1) / per <= G::MAXP &&
                         (prows(th) * (OW + 2) * (CO / 16) + per - 1) / per <= G::MAXG));
    };
    const size_t limit = std::min<size_t>(lds_limit(), 160 * 1024);
    int thmax = std::min(H, std::max(1, kCbPixMax / W));
    while (thmax > 1 && (lds(thmax, 1) > G::LDS_TARGET || !fits(thmax, 1))) --thmax;
    if (lds(thmax, 1) > limit || !fits(thmax, 1)) return hipErrorInvalidValue;
    int TH = 1, best = 1 << 30;   // band height staging the fewest window rows per frame
    for (int th = 1; th <= thmax; ++th) {
        const int rows = (H + th - 1) / th * (th + 2);
        if (rows <= best) { best = rows; TH = th; }
    }
    const int nbands = (H + TH - 1) / TH;
    int FR = 1;
    if (nbands == 1 && !PDY)
        while (FR < a.n && lds(TH, FR + 1) <= G::LDS_TARGET && fits(TH, FR + 1) && (FR + 1) * H * W <= kCbPixMax) ++FR;
    // 32-bit buffer offsets cover FR frames of each operand
    if (int64_t(FR) * H * W * std::max(CI, CO) * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    CbTile t{};
    t.TH = TH; t.FR = FR; t.nbands = nbands; t.ntiles = nbands * ((a.n + FR - 1) / FR);
    int dyb, xb, pb, gb;
    regions(TH, FR, dyb, xb, pb, gb);
    t.dy_off = 64; t.x_off = t.dy_off + dyb;
    t.x_guard = xb - 2 * G::XPB;   // byte offset of the rear guard from the window start
    t.dp_off = t.x_off + xb; t.ag_off = t.dp_off + pb;
    t.PR = PDY ? prows(TH) : 0;
    t.OH = OH; t.OW = OW; t.ph = ph; t.pw = pw; t.BH = (H + ph + 1) / 2; t.BW = (W + pw + 1) / 2;
    t.inv_W = 1.f / float(W); t.inv_TW = 1.f / float(W + 2);
    t.inv_TH = 1.f / float(TH); t.inv_TR = 1.f / float(TH + 2); t.inv_BW = 1.f / float(t.BW);
    const size_t L = std::max(lds(TH, FR), size_t(kCbWaves * 4) * 17 * 16);   // (pending reduce)
    if (PDY && int64_t(OH) * OW * CO * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    const void* fn;
    if constexpr (G::SPEC) fn = reinterpret_cast<const void*>(&conv_bwd_spec_kernel<CI, CO, MODE, ADD, PDY, kCbWaves>);
    else fn = reinterpret_cast<const void*>(&conv_bwd_kernel<CI, CO, MODE, ADD, PDY, kCbWaves>);
    int parts = std::min(resident_blocks(fn, 64 * kCbWaves, L), cb_parts_cap<CI, CO>());
    if (parts > t.ntiles) parts = t.ntiles;
    const std::string shape = cb_dims(CI, CO) + "/" + cb_dims(H, W) + cb_flags(MODE, false, ADD) + (PDY ? "/pool" : "");
    {
        ProfScope ps(s, [&] { return cb_key("conv_bwd", 0, shape); });
        if constexpr (G::SPEC)
            hipLaunchKernelGGL((conv_bwd_spec_kernel<CI, CO, MODE, ADD, PDY, kCbWaves>), dim3(unsigned(parts)),
                               dim3(64 * kCbWaves), L, s, a, t);
        else
            hipLaunchKernelGGL((conv_bwd_kernel<CI, CO, MODE, ADD, PDY, kCbWaves>), dim3(unsigned(parts)),
                               dim3(64 * kCbWaves), L, s, a, t);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (deferred) {
        *deferred = PendingReduce{a.partial, a.dw, a.db, parts, G::PSTRIDE, CI, CO, 0, 1.f};
        return hipSuccess;
    }
    ProfScope ps(s, [&] { return cb_key("conv_bwd_reduce", 0, shape); });
    return wgrad_reduce_tr(CI, CO, a.partial, parts, a.dw, a.db, 1.f, s);
}

}  // namespace

bool conv3x3_bwd_supported(int cin, int cout, int mode, int add, int pooled) {
    if (mode == IN_RELU) return !pooled && cin == cout && (cin == 16 || cin == 32 || cin == 64);
    if (mode == IN_PLAIN)
        return !add && ((cin == 16 && (cout == 16 || cout == 32)) || (cin == 32 && (cout == 32 || cout == 64)) ||
                        (cin == 64 && cout == 64));
    return false;
}

size_t conv3x3_bwd_partial_floats(int cin, int cout) {
    size_t best = 0;
#define CB_PF(CI, CO) \
    if (cin == CI && cout == CO) best = size_t(cb_parts_cap<CI, CO>()) * CbGeom<CI, CO>::PSTRIDE;
    CB_PF(16, 16) CB_PF(16, 32) CB_PF(32, 32) CB_PF(32, 64) CB_PF(64, 64)
#undef CB_PF
    return best;
}

hipError_t conv3x3_bwd(int cin, int cout, int mode, const ConvBwdArgs& a, hipStream_t s, PendingReduce* deferred) {
    if (deferred) deferred->nparts = 0;
    if (a.n <= 0) {
        const hipError_t e = flush_pending_reduce(a.pend, s);
        return e != hipSuccess ? e : flush_pending_reduce(a.pend2, s);
    }
    const int add = a.add != nullptr, pdy = a.arg != nullptr;
#define CB_B(CI, CO, MD, AD, PD) \
    if (cin == CI && cout == CO && mode == MD && add == AD && pdy == PD) return cb_launch<CI, CO, MD, AD, PD>(a, s, deferred);
    CB_B(16, 16, IN_RELU, 0, 0) CB_B(16, 16, IN_RELU, 1, 0) CB_B(32, 32, IN_RELU, 0, 0) CB_B(32, 32, IN_RELU, 1, 0)
    CB_B(64, 64, IN_RELU, 0, 0) CB_B(64, 64, IN_RELU, 1, 0)
    CB_B(16, 16, IN_PLAIN, 0, 0) CB_B(16, 32, IN_PLAIN, 0, 0) CB_B(32, 32, IN_PLAIN, 0, 0)
    CB_B(32, 64, IN_PLAIN, 0, 0) CB_B(64, 64, IN_PLAIN, 0, 0)
    CB_B(16, 16, IN_PLAIN, 0, 1) CB_B(16, 32, IN_PLAIN, 0, 1) CB_B(32, 32, IN_PLAIN, 0, 1)
    CB_B(32, 64, IN_PLAIN, 0, 1) CB_B(64, 64, IN_PLAIN, 0, 1)
#undef CB_B
    return hipErrorInvalidValue;
}

}  // namespace cb
