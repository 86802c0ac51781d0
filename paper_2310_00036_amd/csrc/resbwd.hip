// Backward pass of a whole IMPALA-ResNet residual block (Section 5's network) in one kernel,
// bf16 storage and float32 accumulation on gfx950 MFMA. With the block's forward
//
//   t = conv_a(relu(x)) + b_a,   y = x + conv_b(relu(t)) + b_b     (3x3 SAME convolutions, C -> C)
//
// and the gradient dy at its output:
//
//   dt  = conv_b^T(dy) * [t > 0]           dWb = sum_p relu(t)[p + d(tap)] dy[p],  dbb = sum_p dy[p]
//   dx  = conv_a^T(dt) * [x > 0] + dy      dWa = sum_p relu(x)[p + d(tap)] dt[p],  dba = sum_p dt[p]
//
// As two fused conv backward launches this moves seven activation tensors through HBM (dy and
// t in, dt out; dt, x and dy in, dx out). Here a tile, a band of TH rows of one frame, stages
// dy on rows h0-2 .. h0+TH+1 and t and x on rows h0-1 .. h0+TH, forms dt on rows h0-1 .. h0+TH
// (the band and one halo row either side, which the neighbouring bands form too) in an LDS
// window, rounded to bf16 as the two-launch path stores it, and moves four tensors: dy, t and
// x in, dx out. The skip term of dx comes from the staged dy window.
//
// Each half follows the single conv backward kernel: the input-gradient weights (taps rotated
// by 180 degrees, channels swapped) live in registers, each wave owning one 16-channel block;
// the weight gradients run over the band's own rows with the linear window walk (padding
// columns included, where dy and dt are zero) and accumulate in registers over all tiles of a
// workgroup; each workgroup writes one float32 partial per conv, summed in a fixed order by a
// later launch (deterministic, no atomics).
#include "common.h"
#include "kernels.h"

#include <algorithm>
#include <type_traits>

namespace cb {

template <int C>
struct RbbGeom {
    // dy / dt windows: 16-byte slots per pixel. A 16-lane B-fragment read on consecutive
    // pixels lands on distinct bank groups when the pitch is 2 (mod 4) slots: 16 channels fill
    // 2; 32 channels take two extra slots (never read) for 6
    static constexpr int DSL = C >= 32 ? C / 8 + 2 : C / 8;
    static constexpr int DYP = DSL * 16;
    static constexpr int XPB = C * 2 + (C >= 32 ? 32 : 0);    // t / x windows: bytes per pixel
    static constexpr int XSL = XPB / 16;
    static constexpr int MT = C / 16;
    static constexpr int KSD = (9 * C + 31) / 32;          // input-gradient k-steps
    static constexpr int NB = 9 * C / 16, NBB = NB + 1;    // weight-gradient column blocks (+ bias)
    static constexpr int PSTRIDE = MT * NBB * 256;         // floats per workgroup partial, one conv
    static constexpr int MAXD = C >= 32 ? 6 : 4, MAXX = C >= 32 ? 6 : 4;   // staging slots per lane (8 waves)
    // 16 channels: two workgroups per CU (4 waves per SIMD, 128 registers); 32 channels hold
    // both convs' input-gradient weights (72 registers) and wider accumulators: one
    // workgroup per CU with 256 registers and all of the LDS
    static constexpr int WPS = C >= 32 ? 2 : 4;
    static constexpr size_t LDS_TARGET = C >= 32 ? 160 * 1024 : 80 * 1024;
    __host__ __device__ static int blocks(int slots) { return (slots + 63) / 64; }
};

template <int C, int NW>
__global__ __launch_bounds__(64 * NW, RbbGeom<C>::WPS) void resblock_bwd_kernel(ResBwdArgs a, RbbTile t) {
    using G = RbbGeom<C>;
    constexpr int NT = 64 * NW;
    constexpr int DSL = G::DSL, DYP = G::DYP, XPB = G::XPB, XSL = G::XSL;
    constexpr int MT = G::MT, KSD = G::KSD, NB = G::NB, NBB = G::NBB;
    // weight gradients: waves 0 .. NW/2-1 form conv_b's, the others conv_a's, each wave TPW
    // column blocks, so each dy / dt fragment is read by half the waves
    constexpr int NWG = NW / 2;
    constexpr int TPW = (NBB + NWG - 1) / NWG;   // weight-gradient column blocks per wave
    constexpr int CB16 = C / 16;
    static_assert(NW % MT == 0, "waves split evenly over the channel blocks");

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;                   // 64 zero bytes
    unsigned char* dyw = smem + t.dy_off;         // dy [TH+4][W+2], row 0 = image row h0-2
    unsigned char* tw = smem + t.t_off + XPB;     // relu(t) [TH+2][W+2], row 0 = h0-1, guard pixels
    unsigned char* xw = smem + t.x_off + XPB;     // relu(x) [TH+2][W+2], likewise
    unsigned char* dtw = smem + t.dt_off;         // dt [TH+2][W+2], row 0 = h0-1

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const int H = a.H, W = a.W, TH = t.TH;
    const int TW = W + 2;

    // earlier launches' weight-gradient partials, summed first (LDS is free until staging)
    if (a.pend.nparts > 0) pending_reduce<NT>(a.pend, smem);
    if (a.pend2.nparts > 0) pending_reduce<NT>(a.pend2, smem);
    if (tid < 16) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;
    // the dt window: its padding columns and zero slots are never written
    for (int j = tid; j < t.dt_bytes / 16; j += NT) reinterpret_cast<uint4*>(dtw)[j] = make_uint4(0, 0, 0, 0);
    // the t and x windows' guard pixels (read only against zero dy / dt, never staged)
    if (tid < XPB / 4) {
        reinterpret_cast<uint32_t*>(tw - XPB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(tw + t.tx_guard)[tid] = 0u;
        reinterpret_cast<uint32_t*>(xw - XPB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(xw + t.tx_guard)[tid] = 0u;
    }

    // ---- input-gradient A fragments of both convs for this wave's channel block:
    // A[o][k] = w[8 - tap][o][co] with k = tap * C + co (zero past the 9 taps)
    const int dmt = wave % MT;
    const int ci0 = dmt * 16 + g * 4;   // the lane's first output channel
    uint4 wfa[KSD], wfb[KSD];
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks) {
        const int o = dmt * 16 + r16;
        float va[8], vb[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int k = ks * 32 + g * 8 + j, tap = k / C, co = k % C;
            va[j] = tap < 9 ? a.wa[((8 - tap) * C + o) * C + co] : 0.f;
            vb[j] = tap < 9 ? a.wb[((8 - tap) * C + o) * C + co] : 0.f;
        }
        wfa[ks] = make_uint4(pack2bf(va[0], va[1]), pack2bf(va[2], va[3]), pack2bf(va[4], va[5]), pack2bf(va[6], va[7]));
        wfb[ks] = make_uint4(pack2bf(vb[0], vb[1]), pack2bf(vb[2], vb[3]), pack2bf(vb[4], vb[5]), pack2bf(vb[6], vb[7]));
    }
    // B-fragment byte offsets from the lane's tap-(0,0) pixel of a dy-like window; with 16
    // channels a k-step spans two taps (a per-lane table), from 32 on only the slot is the lane's.
    // Past the ninth tap the weights are zero, so those lanes re-read tap 8 (a value that
    // already enters the sum through tap 8 itself)
    int dboff[C < 32 ? KSD : 1];
    if constexpr (C < 32) {
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / C, slot = (k0 % C) / 8;
            const int tp = tap < 9 ? tap : 8;
            dboff[ks] = ((tp / 3) * TW + tp % 3) * DYP + slot * 16;
        }
    }
    const int twdy = TW * DYP;
    auto dgrad_off = [&](int ks) -> int {
        if constexpr (C < 32) return dboff[ks];
        else return (ks / (C / 32) / 3) * twdy + (ks / (C / 32) % 3) * DYP + ((ks % (C / 32)) * 4 + g) * 16;
    };
    // weight-gradient column blocks nb = wg + NWG * i (16 input channels of one tap, or the
    // bias block), each for all C/16 output-channel blocks, of conv_b (grp 0) or conv_a (grp 1)
    const int wg = wave % NWG, grp = wave / NWG;
    int wboff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = wg + NWG * i;
        const int tap = nb / CB16, cb = nb % CB16;
        wboff[i] = nb < NB ? ((tap / 3) * TW + tap % 3) * XPB + (cb * 16 + 4 * m) * 2 : 0;
    }
    cb_f32x4 wacc[TPW][MT];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int mo = 0; mo < MT; ++mo) wacc[i][mo] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

    // ---- staging offsets, tile-invariant per lane (slot k of this wave: j = (wave + NW*k)*64
    // + lane), relative to the window's first row at image row 0; a tile adds that row's
    // image row. Rows off the frame fall outside the frame's buffer resource and read zero,
    // as do padding slots and columns (kOOB).
    const int nsd = (TH + 4) * TW * DSL, nsx = (TH + 2) * TW * XSL;
    auto win_off = [&](int j, int slots, int rows) -> uint32_t {
        const int p = j / slots, c = j - p * slots;
        const int rr = p / TW, col = p - rr * TW;
        if (j >= rows * TW * slots || c >= C / 8 || col < 1 || col > W) return kOOB;
        return uint32_t(((rr * W + col - 1) * C + c * 8) * 2);
    };
    uint32_t od[G::MAXD], ox[G::MAXX];
#pragma unroll
    for (int k = 0; k < G::MAXD; ++k) od[k] = win_off((wave + NW * k) * 64 + lane, DSL, TH + 4);
#pragma unroll
    for (int k = 0; k < G::MAXX; ++k) ox[k] = win_off((wave + NW * k) * 64 + lane, XSL, TH + 2);

    // ---- one weight gradient over the band's own rows: dy-like window dwin (own row 0 at
    // window row drow0) against the relu'd window bwin (row 0 = image row h0-1): pixel idx of
    // the own rows pairs with bwin pixel idx - 1 + tap offset. Lane (g, 4jj+m) takes pixels
    // o = 16*half + 4g + jj (channels 4m.. of a 16-channel block).
    auto wgrad = [&](const unsigned char* dwin, int drow0, const unsigned char* bwin, const unsigned char* bguard,
                     int L) {
        // specialised per wave, so that each column block's kind (loaded or bias) is known at
        // compile time and the k-step loop carries no branches
        auto run = [&](auto wv) {
            constexpr int WG = decltype(wv)::value;
            const int nfull = L >> 5;
            const int o0 = 4 * g + jj;
            const unsigned char* ap = dwin + (drow0 * TW + o0) * DYP + 8 * m;
            const unsigned char* bp = bwin + (o0 - 1) * XPB;
            auto kstep = [&](const unsigned char* a0, const unsigned char* a1, const unsigned char* b0,
                             const unsigned char* b1) {
                uint4 af[MT];
#pragma unroll
                for (int mo = 0; mo < MT; ++mo) {
                    const uint2 lo = lds_read_tr16(a0 + mo * 32);   // a0, a1: zero past L
                    const uint2 hi = lds_read_tr16(a1 + mo * 32);
                    af[mo] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                }
#pragma unroll
                for (int i = 0; i < TPW; ++i) {
                    const int nb = WG + NWG * i;
                    if (nb < NB) {
                        const uint2 lo = lds_read_tr16(b0 + wboff[i]);
                        const uint2 hi = lds_read_tr16(b1 + wboff[i]);
                        const uint4 bf = make_uint4(lo.x, lo.y, hi.x, hi.y);
#pragma unroll
                        for (int mo = 0; mo < MT; ++mo) wacc[i][mo] = PrecBF16::mma(af[mo], bf, wacc[i][mo]);
                    } else if (nb == NB) {   // the bias block: a column of ones
#pragma unroll
                        for (int mo = 0; mo < MT; ++mo) wacc[i][mo] = PrecBF16::mma(af[mo], ones, wacc[i][mo]);
                    }
                }
            };
            int ks = 0;
            for (; ks + 2 <= nfull; ks += 2) {   // two k-steps per trip: half the pointer updates
                kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                kstep(ap + 32 * DYP, ap + 48 * DYP, bp + 32 * XPB, bp + 48 * XPB);
                ap += 64 * DYP;
                bp += 64 * XPB;
            }
            if (ks < nfull) {
                kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                ap += 32 * DYP;
                bp += 32 * XPB;
            }
            if (L & 31) {   // the last, partial k-step
                const int o = nfull * 32 + o0;
                const bool ok0 = o < L, ok1 = o + 16 < L;
                kstep(ok0 ? ap : zero, ok1 ? ap + 16 * DYP : zero, ok0 ? bp : bguard, ok1 ? bp + 16 * XPB : bguard);
            }
        };
        static_assert(NWG == 4, "one specialisation per wave of a group");
        switch (wg) {
            case 0: run(std::integral_constant<int, 0>{}); break;
            case 1: run(std::integral_constant<int, 1>{}); break;
            case 2: run(std::integral_constant<int, 2>{}); break;
            default: run(std::integral_constant<int, 3>{}); break;
        }
    };

    int lg = blockIdx.x;   // neighbouring bands (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int h0 = band * TH;
        const int the = H - h0 < TH ? H - h0 : TH;
        const int64_t fo = int64_t(f) * H * W * C;   // the frame's first element
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage dy (rows h0-2 ..), t and x (rows h0-1 ..)
        {
            const uint32_t fb = uint32_t(H) * W * C * 2;
            const auto rd = buf_rsrc(static_cast<const uint16_t*>(a.dy) + fo, fb);
            const auto rt = buf_rsrc(static_cast<const uint16_t*>(a.t) + fo, fb);
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + fo, fb);
            const uint32_t hd = uint32_t((h0 - 2) * W * C * 2);   // wraps above the frame: reads zero
            const uint32_t hx = uint32_t((h0 - 1) * W * C * 2);
#pragma unroll
            for (int k = 0; k < G::MAXD; ++k)
                if ((wave + NW * k) * 64 < nsd) dma16_to_lds(rd, dyw + (wave + NW * k) * 1024, od[k] + hd);
#pragma unroll
            for (int k = 0; k < G::MAXX; ++k)
                if ((wave + NW * k) * 64 < nsx) {
                    dma16_to_lds(rt, tw + (wave + NW * k) * 1024, ox[k] + hx);
                    dma16_to_lds(rx, xw + (wave + NW * k) * 1024, ox[k] + hx);
                }
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        {
            // both convs read relu'd inputs; relu(v) > 0 exactly where v > 0, so the masks
            // read the same windows
            uint4* t4 = reinterpret_cast<uint4*>(tw);
            uint4* x4 = reinterpret_cast<uint4*>(xw);
            for (int j = tid; j < nsx; j += NT) {
                uint4 u = t4[j], v = x4[j];
                u.x = relu_bf16x2(u.x); u.y = relu_bf16x2(u.y); u.z = relu_bf16x2(u.z); u.w = relu_bf16x2(u.w);
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                t4[j] = u;
                x4[j] = v;
            }
        }
        __syncthreads();

        // ---- conv_b's input gradient dt on window rows r = 0 .. the+1 (image rows h0-1+r;
        // zero off the frame), 16-pixel column tiles, into the dt window
        {
            const int npx = (the + 2) * W;
            for (int nt = wave / MT; nt * 16 < npx; nt += NW / MT) {
                const int q = nt * 16 + r16;
                const int qc = q < npx ? q : npx - 1;   // past npx: computed, not stored
                const int row = qdiv(qc, t.inv_W), col = qc - row * W;
                const unsigned char* xb = dyw + (row * TW + col) * DYP;
                cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks)
                    acc = PrecBF16::mma(wfb[ks], *reinterpret_cast<const uint4*>(xb + dgrad_off(ks)), acc);
                if (q < npx) {
                    const int h = h0 - 1 + row;
                    uint2 o = make_uint2(0u, 0u);
                    if (h >= 0 && h < H) {
                        float mk[4];
                        load4(reinterpret_cast<const uint16_t*>(tw + (row * TW + col + 1) * XPB + ci0 * 2), mk);
                        o = make_uint2(pack2bf(mk[0] > 0.f ? acc[0] : 0.f, mk[1] > 0.f ? acc[1] : 0.f),
                                       pack2bf(mk[2] > 0.f ? acc[2] : 0.f, mk[3] > 0.f ? acc[3] : 0.f));
                    }
                    *reinterpret_cast<uint2*>(dtw + (row * TW + col + 1) * DYP + ci0 * 2) = o;
                }
            }
        }
        __syncthreads();   // the dt window is complete

        // ---- dx = conv_a^T(dt) * [x > 0] + dy on the band's rows
        {
            const int npx = the * W;
            uint16_t* dxt = static_cast<uint16_t*>(a.dx) + fo + int64_t(h0) * W * C;
            for (int nt = wave / MT; nt * 16 < npx; nt += NW / MT) {
                const int q = nt * 16 + r16;
                const int qc = q < npx ? q : npx - 1;
                const int row = qdiv(qc, t.inv_W), col = qc - row * W;
                const unsigned char* xb = dtw + (row * TW + col) * DYP;
                cb_f32x4 acc = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSD; ++ks)
                    acc = PrecBF16::mma(wfa[ks], *reinterpret_cast<const uint4*>(xb + dgrad_off(ks)), acc);
                if (q < npx) {
                    float mk[4], sk[4];
                    load4(reinterpret_cast<const uint16_t*>(xw + ((row + 1) * TW + col + 1) * XPB + ci0 * 2), mk);
                    load4(reinterpret_cast<const uint16_t*>(dyw + ((row + 2) * TW + col + 1) * DYP + ci0 * 2), sk);
                    float v[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) v[j] = (mk[j] > 0.f ? acc[j] : 0.f) + sk[j];
                    store4(dxt + uint32_t(q * C + ci0), v[0], v[1], v[2], v[3]);
                }
            }
        }
        // ---- the weight gradients: conv_b's, dy (own rows from dy-window row 2) against
        // relu(t), by the first half of the waves; conv_a's, dt (own rows from dt-window row
        // 1) against relu(x), by the second
        if (grp == 0) wgrad(dyw, 2, tw, tw - XPB, the * TW);
        else wgrad(dtw, 1, xw, xw - XPB, the * TW);
    }

    // ---- this workgroup's partials: conv_b's set, then conv_a's, each [mo*NBB + nb][co 16][ci 16]
    float* part = a.partial + (grp == 0 ? 0 : t.pset) + int64_t(blockIdx.x) * G::PSTRIDE;
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = wg + NWG * i;
        if (nb < NBB) {
#pragma unroll
            for (int mo = 0; mo < MT; ++mo)
#pragma unroll
                for (int e = 0; e < 4; ++e) part[(mo * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = wacc[i][mo][e];
        }
    }
}

// The 32-channel block backward with specialised waves. Every wave forming dt and dx for one
// 16-channel block reads each B fragment for that block alone and holds both convs'
// weight-gradient accumulators beside the input-gradient weights. Here waves 0-3 form dt and
// dx for both channel blocks (each B fragment feeding two MFMAs; 144 registers of weights)
// and waves 4-7 both weight gradients (conv_b's while dt is formed, conv_a's once it is
// complete), each for a quarter of the column blocks.
template <int C, int NW>
__global__ __launch_bounds__(64 * NW, RbbGeom<C>::WPS) void resblock_bwd_spec_kernel(ResBwdArgs a, RbbTile t) {
    using G = RbbGeom<C>;
    constexpr int NT = 64 * NW;
    constexpr int DSL = G::DSL, DYP = G::DYP, XPB = G::XPB, XSL = G::XSL;
    constexpr int MT = G::MT, KSD = G::KSD, NB = G::NB, NBB = G::NBB;
    // weight gradients: waves 0 .. NW/2-1 form conv_b's, the others conv_a's, each wave TPW
    // column blocks, so each dy / dt fragment is read by half the waves
    constexpr int NWG = NW / 2;
    constexpr int TPW = (NBB + NWG - 1) / NWG;   // weight-gradient column blocks per wave
    constexpr int CB16 = C / 16;
    static_assert(C == 32 && NW == 8 && NWG == 4, "32 channels: four input-gradient and four weight-gradient waves");
    constexpr int DB = MT;   // dx / dt channel blocks per input-gradient wave (all of them)

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* zero = smem;                   // 64 zero bytes
    unsigned char* dyw = smem + t.dy_off;         // dy [TH+4][W+2], row 0 = image row h0-2
    unsigned char* tw = smem + t.t_off + XPB;     // relu(t) [TH+2][W+2], row 0 = h0-1, guard pixels
    unsigned char* xw = smem + t.x_off + XPB;     // relu(x) [TH+2][W+2], likewise
    unsigned char* dtw = smem + t.dt_off;         // dt [TH+2][W+2], row 0 = h0-1

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const int H = a.H, W = a.W, TH = t.TH;
    const int TW = W + 2;

    // earlier launches' weight-gradient partials, summed first (LDS is free until staging)
    if (a.pend.nparts > 0) pending_reduce<NT>(a.pend, smem);
    if (a.pend2.nparts > 0) pending_reduce<NT>(a.pend2, smem);
    if (tid < 16) reinterpret_cast<uint32_t*>(zero)[tid] = 0u;
    // the dt window: its padding columns and zero slots are never written
    for (int j = tid; j < t.dt_bytes / 16; j += NT) reinterpret_cast<uint4*>(dtw)[j] = make_uint4(0, 0, 0, 0);
    // the t and x windows' guard pixels (read only against zero dy / dt, never staged)
    if (tid < XPB / 4) {
        reinterpret_cast<uint32_t*>(tw - XPB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(tw + t.tx_guard)[tid] = 0u;
        reinterpret_cast<uint32_t*>(xw - XPB)[tid] = 0u;
        reinterpret_cast<uint32_t*>(xw + t.tx_guard)[tid] = 0u;
    }

    // ---- input-gradient A fragments of both convs for this wave's channel block:
    // A[o][k] = w[8 - tap][o][co] with k = tap * C + co (zero past the 9 taps)
    const int ci0 = g * 4;   // the lane's first channel of each block (block b adds 16 b)
    auto load_w = [&](uint4 (&wfa)[DB][KSD], uint4 (&wfb)[DB][KSD]) {
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
            for (int ks = 0; ks < KSD; ++ks) {
                const int o = b * 16 + r16;
                float va[8], vb[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int k = ks * 32 + g * 8 + j, tap = k / C, co = k % C;
                    va[j] = tap < 9 ? a.wa[((8 - tap) * C + o) * C + co] : 0.f;
                    vb[j] = tap < 9 ? a.wb[((8 - tap) * C + o) * C + co] : 0.f;
                }
                wfa[b][ks] = make_uint4(pack2bf(va[0], va[1]), pack2bf(va[2], va[3]), pack2bf(va[4], va[5]), pack2bf(va[6], va[7]));
                wfb[b][ks] = make_uint4(pack2bf(vb[0], vb[1]), pack2bf(vb[2], vb[3]), pack2bf(vb[4], vb[5]), pack2bf(vb[6], vb[7]));
            }
    };
    // B-fragment byte offsets from the lane's tap-(0,0) pixel of a dy-like window; with 16
    // channels a k-step spans two taps (a per-lane table), from 32 on only the slot is the lane's.
    // Past the ninth tap the weights are zero, so those lanes re-read tap 8 (a value that
    // already enters the sum through tap 8 itself)
    int dboff[C < 32 ? KSD : 1];
    if constexpr (C < 32) {
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
            const int k0 = ks * 32 + g * 8, tap = k0 / C, slot = (k0 % C) / 8;
            const int tp = tap < 9 ? tap : 8;
            dboff[ks] = ((tp / 3) * TW + tp % 3) * DYP + slot * 16;
        }
    }
    const int twdy = TW * DYP;
    auto dgrad_off = [&](int ks) -> int {
        if constexpr (C < 32) return dboff[ks];
        else return (ks / (C / 32) / 3) * twdy + (ks / (C / 32) % 3) * DYP + ((ks % (C / 32)) * 4 + g) * 16;
    };
    // weight-gradient column blocks nb = wg + NWG * i (16 input channels of one tap, or the
    // bias block), each for all C/16 output-channel blocks, of both convs (waves 4..7)
    const int wg = wave % NWG;
    int wboff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int nb = wg + NWG * i;
        const int tap = nb / CB16, cb = nb % CB16;
        wboff[i] = nb < NB ? ((tap / 3) * TW + tap % 3) * XPB + (cb * 16 + 4 * m) * 2 : 0;
    }
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

    // ---- staging offsets, tile-invariant per lane (slot k of this wave: j = (wave + NW*k)*64
    // + lane), relative to the window's first row at image row 0; a tile adds that row's
    // image row. Rows off the frame fall outside the frame's buffer resource and read zero,
    // as do padding slots and columns (kOOB).
    const int nsd = (TH + 4) * TW * DSL, nsx = (TH + 2) * TW * XSL;
    auto win_off = [&](int j, int slots, int rows) -> uint32_t {
        const int p = j / slots, c = j - p * slots;
        const int rr = p / TW, col = p - rr * TW;
        if (j >= rows * TW * slots || c >= C / 8 || col < 1 || col > W) return kOOB;
        return uint32_t(((rr * W + col - 1) * C + c * 8) * 2);
    };
    uint32_t od[G::MAXD], ox[G::MAXX];
#pragma unroll
    for (int k = 0; k < G::MAXD; ++k) od[k] = win_off((wave + NW * k) * 64 + lane, DSL, TH + 4);
#pragma unroll
    for (int k = 0; k < G::MAXX; ++k) ox[k] = win_off((wave + NW * k) * 64 + lane, XSL, TH + 2);

    // ---- one weight gradient over the band's own rows: dy-like window dwin (own row 0 at
    // window row drow0) against the relu'd window bwin (row 0 = image row h0-1): pixel idx of
    // the own rows pairs with bwin pixel idx - 1 + tap offset. Lane (g, 4jj+m) takes pixels
    // o = 16*half + 4g + jj (channels 4m.. of a 16-channel block).
    auto wgrad = [&](const unsigned char* dwin, int drow0, const unsigned char* bwin, const unsigned char* bguard,
                     int L, cb_f32x4 (&wacc)[TPW][MT]) {
        // specialised per wave, so that each column block's kind (loaded or bias) is known at
        // compile time and the k-step loop carries no branches
        auto run = [&](auto wv) {
            constexpr int WG = decltype(wv)::value;
            const int nfull = L >> 5;
            const int o0 = 4 * g + jj;
            const unsigned char* ap = dwin + (drow0 * TW + o0) * DYP + 8 * m;
            const unsigned char* bp = bwin + (o0 - 1) * XPB;
            auto kstep = [&](const unsigned char* a0, const unsigned char* a1, const unsigned char* b0,
                             const unsigned char* b1) {
                uint4 af[MT];
#pragma unroll
                for (int mo = 0; mo < MT; ++mo) {
                    const uint2 lo = lds_read_tr16(a0 + mo * 32);   // a0, a1: zero past L
                    const uint2 hi = lds_read_tr16(a1 + mo * 32);
                    af[mo] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                }
#pragma unroll
                for (int i = 0; i < TPW; ++i) {
                    const int nb = WG + NWG * i;
                    if (nb < NB) {
                        const uint2 lo = lds_read_tr16(b0 + wboff[i]);
                        const uint2 hi = lds_read_tr16(b1 + wboff[i]);
                        const uint4 bf = make_uint4(lo.x, lo.y, hi.x, hi.y);
#pragma unroll
                        for (int mo = 0; mo < MT; ++mo) wacc[i][mo] = PrecBF16::mma(af[mo], bf, wacc[i][mo]);
                    } else if (nb == NB) {   // the bias block: a column of ones
#pragma unroll
                        for (int mo = 0; mo < MT; ++mo) wacc[i][mo] = PrecBF16::mma(af[mo], ones, wacc[i][mo]);
                    }
                }
            };
            int ks = 0;
            for (; ks + 2 <= nfull; ks += 2) {   // two k-steps per trip: half the pointer updates
                kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                kstep(ap + 32 * DYP, ap + 48 * DYP, bp + 32 * XPB, bp + 48 * XPB);
                ap += 64 * DYP;
                bp += 64 * XPB;
            }
            if (ks < nfull) {
                kstep(ap, ap + 16 * DYP, bp, bp + 16 * XPB);
                ap += 32 * DYP;
                bp += 32 * XPB;
            }
            if (L & 31) {   // the last, partial k-step
                const int o = nfull * 32 + o0;
                const bool ok0 = o < L, ok1 = o + 16 < L;
                kstep(ok0 ? ap : zero, ok1 ? ap + 16 * DYP : zero, ok0 ? bp : bguard, ok1 ? bp + 16 * XPB : bguard);
            }
        };
        static_assert(NWG == 4, "one specialisation per wave of a group");
        switch (wg) {
            case 0: run(std::integral_constant<int, 0>{}); break;
            case 1: run(std::integral_constant<int, 1>{}); break;
            case 2: run(std::integral_constant<int, 2>{}); break;
            default: run(std::integral_constant<int, 3>{}); break;
        }
    };

    int lg = blockIdx.x;   // neighbouring bands (which share halo rows) on one XCD
    if ((gridDim.x & 7) == 0) lg = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);

    auto prologue = [&](int tile) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        const int h0 = band * TH;
        const int64_t fo = int64_t(f) * H * W * C;   // the frame's first element
        __syncthreads();   // the previous tile's LDS reads are done

        // ---- stage dy (rows h0-2 ..), t and x (rows h0-1 ..)
        {
            const uint32_t fb = uint32_t(H) * W * C * 2;
            const auto rd = buf_rsrc(static_cast<const uint16_t*>(a.dy) + fo, fb);
            const auto rt = buf_rsrc(static_cast<const uint16_t*>(a.t) + fo, fb);
            const auto rx = buf_rsrc(static_cast<const uint16_t*>(a.x) + fo, fb);
            const uint32_t hd = uint32_t((h0 - 2) * W * C * 2);   // wraps above the frame: reads zero
            const uint32_t hx = uint32_t((h0 - 1) * W * C * 2);
#pragma unroll
            for (int k = 0; k < G::MAXD; ++k)
                if ((wave + NW * k) * 64 < nsd) dma16_to_lds(rd, dyw + (wave + NW * k) * 1024, od[k] + hd);
#pragma unroll
            for (int k = 0; k < G::MAXX; ++k)
                if ((wave + NW * k) * 64 < nsx) {
                    dma16_to_lds(rt, tw + (wave + NW * k) * 1024, ox[k] + hx);
                    dma16_to_lds(rx, xw + (wave + NW * k) * 1024, ox[k] + hx);
                }
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        {
            // both convs read relu'd inputs; relu(v) > 0 exactly where v > 0, so the masks
            // read the same windows
            uint4* t4 = reinterpret_cast<uint4*>(tw);
            uint4* x4 = reinterpret_cast<uint4*>(xw);
            for (int j = tid; j < nsx; j += NT) {
                uint4 u = t4[j], v = x4[j];
                u.x = relu_bf16x2(u.x); u.y = relu_bf16x2(u.y); u.z = relu_bf16x2(u.z); u.w = relu_bf16x2(u.w);
                v.x = relu_bf16x2(v.x); v.y = relu_bf16x2(v.y); v.z = relu_bf16x2(v.z); v.w = relu_bf16x2(v.w);
                t4[j] = u;
                x4[j] = v;
            }
        }
        __syncthreads();

    };

    auto band_of = [&](int tile, int& h0, int& the, int64_t& fo) {
        const int band = tile % t.nbands, f = tile / t.nbands;
        h0 = band * TH;
        the = H - h0 < TH ? H - h0 : TH;
        fo = int64_t(f) * H * W * C;
    };

    // Two loops over the same tiles, one per role, so that each role keeps only its own
    // registers live; every wave runs the prologue's barriers and the one between the halves
    // of a tile (after dt / after conv_b's weight gradient, which need no dt).
    if (wave < NWG) {
        uint4 wfa[DB][KSD], wfb[DB][KSD];
        load_w(wfa, wfb);
        for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
            prologue(tile);
            int h0, the;
            int64_t fo;
            band_of(tile, h0, the, fo);
            // ---- conv_b's input gradient dt on window rows r = 0 .. the+1 (image rows h0-1+r;
            // zero off the frame), 16-pixel column tiles, into the dt window
            {
                const int npx = (the + 2) * W;
                for (int nt = wave; nt * 16 < npx; nt += NWG) {
                    const int q = nt * 16 + r16;
                    const int qc = q < npx ? q : npx - 1;   // past npx: computed, not stored
                    const int row = qdiv(qc, t.inv_W), col = qc - row * W;
                    const unsigned char* xb = dyw + (row * TW + col) * DYP;
                    cb_f32x4 acc[DB];
    #pragma unroll
                    for (int b = 0; b < DB; ++b) acc[b] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                    for (int ks = 0; ks < KSD; ++ks) {
                        const uint4 bf = *reinterpret_cast<const uint4*>(xb + dgrad_off(ks));
    #pragma unroll
                        for (int b = 0; b < DB; ++b) acc[b] = PrecBF16::mma(wfb[b][ks], bf, acc[b]);
                    }
                    if (q < npx) {
                        const int h = h0 - 1 + row;
    #pragma unroll
                        for (int b = 0; b < DB; ++b) {
                            uint2 o = make_uint2(0u, 0u);
                            if (h >= 0 && h < H) {
                                float mk[4];
                                load4(reinterpret_cast<const uint16_t*>(tw + (row * TW + col + 1) * XPB + (ci0 + 16 * b) * 2), mk);
                                o = make_uint2(pack2bf(mk[0] > 0.f ? acc[b][0] : 0.f, mk[1] > 0.f ? acc[b][1] : 0.f),
                                               pack2bf(mk[2] > 0.f ? acc[b][2] : 0.f, mk[3] > 0.f ? acc[b][3] : 0.f));
                            }
                            *reinterpret_cast<uint2*>(dtw + (row * TW + col + 1) * DYP + (ci0 + 16 * b) * 2) = o;
                        }
                    }
                }
            }
            __syncthreads();   // the dt window is complete
            // ---- dx = conv_a^T(dt) * [x > 0] + dy on the band's rows
            {
                const int npx = the * W;
                uint16_t* dxt = static_cast<uint16_t*>(a.dx) + fo + int64_t(h0) * W * C;
                for (int nt = wave; nt * 16 < npx; nt += NWG) {
                    const int q = nt * 16 + r16;
                    const int qc = q < npx ? q : npx - 1;
                    const int row = qdiv(qc, t.inv_W), col = qc - row * W;
                    const unsigned char* xb = dtw + (row * TW + col) * DYP;
                    cb_f32x4 acc[DB];
    #pragma unroll
                    for (int b = 0; b < DB; ++b) acc[b] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
                    for (int ks = 0; ks < KSD; ++ks) {
                        const uint4 bf = *reinterpret_cast<const uint4*>(xb + dgrad_off(ks));
    #pragma unroll
                        for (int b = 0; b < DB; ++b) acc[b] = PrecBF16::mma(wfa[b][ks], bf, acc[b]);
                    }
                    if (q < npx) {
    #pragma unroll
                        for (int b = 0; b < DB; ++b) {
                            const int cb = ci0 + 16 * b;
                            float mk[4], sk[4];
                            load4(reinterpret_cast<const uint16_t*>(xw + ((row + 1) * TW + col + 1) * XPB + cb * 2), mk);
                            load4(reinterpret_cast<const uint16_t*>(dyw + ((row + 2) * TW + col + 1) * DYP + cb * 2), sk);
                            float v[4];
    #pragma unroll
                            for (int j = 0; j < 4; ++j) v[j] = (mk[j] > 0.f ? acc[b][j] : 0.f) + sk[j];
                            store4(dxt + uint32_t(q * C + cb), v[0], v[1], v[2], v[3]);
                        }
                    }
                }
            }
        }
    } else {
        cb_f32x4 wb_acc[TPW][MT], wa_acc[TPW][MT];
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int mo = 0; mo < MT; ++mo) wb_acc[i][mo] = wa_acc[i][mo] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
        for (int tile = lg; tile < t.ntiles; tile += gridDim.x) {
            prologue(tile);
            int h0, the;
            int64_t fo;
            band_of(tile, h0, the, fo);
            (void)h0;
            (void)fo;
            // conv_b's: dy (own rows from dy-window row 2) against relu(t); then, once dt is
            // complete, conv_a's: dt (own rows from dt-window row 1) against relu(x)
            wgrad(dyw, 2, tw, tw - XPB, the * TW, wb_acc);
            __syncthreads();   // the dt window is complete
            wgrad(dtw, 1, xw, xw - XPB, the * TW, wa_acc);
        }
        // ---- this workgroup's partials: conv_b's set, then conv_a's, each [mo*NBB + nb][co 16][ci 16]
        float* pb = a.partial + int64_t(blockIdx.x) * G::PSTRIDE;
        float* pa = pb + t.pset;
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const int nb = wg + NWG * i;
            if (nb < NBB) {
#pragma unroll
                for (int mo = 0; mo < MT; ++mo)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        pb[(mo * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = wb_acc[i][mo][e];
                        pa[(mo * NBB + nb) * 256 + (4 * g + e) * 16 + r16] = wa_acc[i][mo][e];
                    }
            }
        }
    }
}

namespace {

constexpr int kRbbWaves = 8;
constexpr size_t kRbbPartBytes = 24u << 20;   // both partial sets

template <int C>
int rbb_parts_cap() {
    const size_t cap = kRbbPartBytes / (2 * size_t(RbbGeom<C>::PSTRIDE) * sizeof(float));
    return int(cap < 256 ? 256 : (cap > 1024 ? 1024 : cap));
}

template <int C>
hipError_t rbb_launch(const ResBwdArgs& a, hipStream_t s, PendingReduce out[2]) {
    using G = RbbGeom<C>;
    const int H = a.H, W = a.W, TW = W + 2;
    auto regions = [&](int th, int& dyb, int& txb, int& dtb) {
        dyb = G::blocks((th + 4) * TW * G::DSL) * 1024;
        txb = G::blocks((th + 2) * TW * G::XSL) * 1024 + 2 * G::XPB;   // + a guard pixel either side
        dtb = ((th + 2) * TW * G::DYP + 15) / 16 * 16;
    };
    auto lds = [&](int th) {
        int dyb, txb, dtb;
        regions(th, dyb, txb, dtb);
        return size_t(64 + dyb + 2 * txb + dtb);
    };
    auto fits = [&](int th) {
        const int per = kRbbWaves * 64;
        return ((th + 4) * TW * G::DSL + per - 1) / per <= G::MAXD && ((th + 2) * TW * G::XSL + per - 1) / per <= G::MAXX;
    };
    const size_t limit = std::min<size_t>(lds_limit(), 160 * 1024);
    int thmax = H;
    while (thmax > 1 && (lds(thmax) > G::LDS_TARGET || !fits(thmax))) --thmax;
    if (lds(thmax) > limit || !fits(thmax)) return hipErrorInvalidValue;
    if (int64_t(H) * W * C * 2 >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    const int nb0 = (H + thmax - 1) / thmax;
    const int TH = (H + nb0 - 1) / nb0;   // balanced bands
    RbbTile t{};
    t.TH = TH; t.nbands = (H + TH - 1) / TH; t.ntiles = t.nbands * a.n;
    int dyb, txb, dtb;
    regions(TH, dyb, txb, dtb);
    t.dy_off = 64; t.t_off = t.dy_off + dyb; t.x_off = t.t_off + txb; t.dt_off = t.x_off + txb;
    t.tx_guard = txb - 2 * G::XPB;
    t.dt_bytes = dtb;
    t.inv_W = 1.f / float(W);
    const size_t L = std::max(lds(TH), size_t(kRbbWaves * 4) * 17 * 16);   // (pending reduce)
    const void* fn;
    if constexpr (C == 32) fn = reinterpret_cast<const void*>(&resblock_bwd_spec_kernel<C, kRbbWaves>);
    else fn = reinterpret_cast<const void*>(&resblock_bwd_kernel<C, kRbbWaves>);
    int parts = std::min(resident_blocks(fn, 64 * kRbbWaves, L), rbb_parts_cap<C>());
    if (parts > t.ntiles) parts = t.ntiles;
    t.pset = parts * G::PSTRIDE;
    const std::string shape = cb_dims(C, C) + "/" + cb_dims(H, W);
    {
        ProfScope ps(s, [&] { return cb_key("resblock_bwd", 0, shape); });
        if constexpr (C == 32)
            hipLaunchKernelGGL((resblock_bwd_spec_kernel<C, kRbbWaves>), dim3(unsigned(parts)), dim3(64 * kRbbWaves), L, s, a, t);
        else
            hipLaunchKernelGGL((resblock_bwd_kernel<C, kRbbWaves>), dim3(unsigned(parts)), dim3(64 * kRbbWaves), L, s, a, t);
    }
    out[0] = PendingReduce{a.partial, a.dwb, a.dbb, parts, G::PSTRIDE, C, C, 0, 1.f};
    out[1] = PendingReduce{a.partial + t.pset, a.dwa, a.dba, parts, G::PSTRIDE, C, C, 0, 1.f};
    return hipGetLastError();
}

}  // namespace

bool resblock_bwd_supported(int C) { return C == 16 || C == 32; }

// With 32 channels the block backward (its specialised-wave form) beats the two conv backward
// launches at every shape the networks use (2048 frames: 11x11 55 against 75 us, 21x21 136
// against 148 us; 8192 frames at 42x42: 1.66 against 1.97 ms).
bool resblock_bwd_preferred(int C, int H, int W) { return (C == 16 || C == 32) && H > 0 && W > 0; }

size_t resblock_bwd_partial_floats(int C) {
    if (C == 16) return 2 * size_t(rbb_parts_cap<16>()) * RbbGeom<16>::PSTRIDE;
    if (C == 32) return 2 * size_t(rbb_parts_cap<32>()) * RbbGeom<32>::PSTRIDE;
    return 0;
}

hipError_t resblock_bwd(int C, const ResBwdArgs& a, hipStream_t s, PendingReduce out[2]) {
    out[0].nparts = 0;
    out[1].nparts = 0;
    if (a.n <= 0) {
        const hipError_t e = flush_pending_reduce(a.pend, s);
        return e != hipSuccess ? e : flush_pending_reduce(a.pend2, s);
    }
    if (C == 16) return rbb_launch<16>(a, s, out);
    if (C == 32) return rbb_launch<32>(a, s, out);
    return hipErrorInvalidValue;
}

}  // namespace cb
