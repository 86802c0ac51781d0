// Policy-logit and value heads of the network (Section 5: the dense layer's output feeds a
// linear policy head over the actions and a linear value head), forward and backward.
//
// Both heads together are one [J] -> [A + 1] linear map (column A is the value head). It is
// a few MFLOP per minibatch, so these kernels use float32 FMAs with the weights staged in
// LDS and make every pass over the hidden activations h count:
//   forward:  logits and value for 16 rows per workgroup;
//   backward: one pass over h and the head gradients dz produces the masked hidden
//             gradient dh = (dz W^T) * (h > 0) in the storage type, and per-workgroup
//             partial sums of the head weight gradient h^T dz, of the head bias gradient
//             (column sums of dz) and of the dense-layer bias gradient (column sums of dh
//             as stored); a second kernel adds the partials in a fixed order.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace cb {

namespace {

constexpr int kHR = 16;    // rows per row group
constexpr int kHJ = 256;   // hidden units per chunk: one per thread
constexpr size_t kHeadsPartialCap = size_t(8) << 20;   // floats of partials at most
constexpr int kHmWaves = 4;                              // MFMA forward: waves per workgroup
constexpr int kHmOut = 32;                               // MFMA kernels: head outputs (A + 1) at most

template <class T>
CB_DEV float ld_st(const T* p, int64_t i) {
    if constexpr (sizeof(T) == 2) return bf2f(p[i]);
    else return p[i];
}

// ws[jj][aa] (pitch MA | 1, odd: conflict-free column reads) = W(j0 + jj, aa) for the chunk:
// the logit weights' row for aa < A, the value weight for aa == A, zero for aa > A and for
// units past the chunk's nj, so the inner loops run over all MA columns and 256 units
// without conditions. Thread t stages unit t's row; its loads are unconditional (clamped
// indices) and all issued before the first store. AC > 0 fixes the action count at compile
// time (MA = AC + 1: no padding columns, no uniform branches around the loads); 0 reads it
// from the arguments.
template <int AC, int MA>
CB_DEV void stage_head_w(float* ws, const HeadsArgs& a, int j0, int nj) {
    constexpr int PW = MA | 1;
    const int A = AC > 0 ? AC : a.A;
    const int t = threadIdx.x;
    const int jc = j0 + min(t, nj - 1);
    const float* wr = a.wl + int64_t(jc) * A;
    const float wv = a.wv[jc];
    float v[MA];
#pragma unroll
    for (int c = 0; c < MA; ++c) {
        const float x = wr[min(c, A - 1)];
        v[c] = c < A ? x : (c == A ? wv : 0.f);
    }
    const bool ok = t < nj;
#pragma unroll
    for (int c = 0; c < MA; ++c) ws[t * PW + c] = ok ? v[c] : 0.f;
}

// logits[i][a] = bl[a] + sum_j h[i][j] wl[j][a]; value[i] = bv + sum_j h[i][j] wv[j].
// Thread (r, q) of the 16 x 16 layout takes row r and the units 16q .. 16q+15 of every
// chunk (two 16-byte loads of h for bf16), accumulating all MA columns over them in order;
// the 16 slices' sums are then added in slice order through LDS.
template <class T, int AC, int MA>
__global__ __launch_bounds__(256) void heads_fwd_kernel(HeadsArgs a, float* __restrict__ logits,
                                                        float* __restrict__ value) {
    extern __shared__ float sm[];
    constexpr int PW = MA | 1;
    const int A = AC > 0 ? AC : a.A;
    float* ws = sm;   // [kHJ][PW]; reused as the slice sums [16 q][16 r][MA] at the end
    const int tid = threadIdx.x, r = tid & 15, q = tid >> 4;
    const int64_t row0 = int64_t(blockIdx.x) * kHR;
    const int64_t rowc = std::min<int64_t>(row0 + r, a.n - 1);
    const bool row_ok = row0 + r < a.n;
    const T* h = static_cast<const T*>(a.h);
    float acc[MA];
#pragma unroll
    for (int c = 0; c < MA; ++c) acc[c] = 0.f;
    for (int j0 = 0; j0 < a.J; j0 += kHJ) {
        const int nj = min(kHJ, a.J - j0);
        float hv[16];
        if (sizeof(T) == 2 && (a.J & 7) == 0 && j0 + 16 * q + 16 <= a.J) {
            const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.h) + rowc * a.J + j0 + 16 * q);
            const uint4 u0 = p[0], u1 = p[1];
            const uint32_t w[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                hv[2 * k] = __uint_as_float(w[k] << 16);
                hv[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
            }
        } else {
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                const int jj = min(16 * q + k, nj - 1);
                hv[k] = 16 * q + k < nj ? ld_st(h, rowc * a.J + j0 + jj) : 0.f;
            }
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) hv[k] = row_ok ? hv[k] : 0.f;
        __syncthreads();
        stage_head_w<AC, MA>(ws, a, j0, nj);
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const float* wr = ws + (16 * q + k) * PW;
#pragma unroll
            for (int c = 0; c < MA; ++c) acc[c] += hv[k] * wr[c];
            if (k % 2 == 1) __builtin_amdgcn_sched_barrier(0);   // bounds the LDS reads in flight
        }
    }
    __syncthreads();
    float* red = sm;
#pragma unroll
    for (int c = 0; c < MA; ++c) red[(q * 16 + r) * MA + c] = acc[c];
    __syncthreads();
    const int A1 = A + 1;
    for (int o = tid; o < 16 * A1; o += kHJ) {
        const int rr = o / A1, aa = o - rr * A1;
        float t = 0.f;
#pragma unroll
        for (int qq = 0; qq < 16; ++qq) t += red[(qq * 16 + rr) * MA + aa];
        const int64_t row = row0 + rr;
        if (row < a.n) {
            if (aa < A) logits[row * A + aa] = t + a.bl[aa];
            else value[row] = t + a.bv[0];
        }
    }
}

// Partial layout per workgroup (stride pstride):
//   [aa * J + j]          sum over its rows of h[i][j] dz[i][aa]    (aa <= A)
//   [(A + 1) * J + j]     sum over its rows of dh[i][j] (as stored)
//   [(A + 2) * J + aa]    sum over its rows of dz[i][aa]            (aa <= A)
// Workgroup b takes the row groups b, b + gridDim.x, ... in increasing order; thread t owns
// hidden unit j0 + t of each chunk.
template <class T, int AC, int MA>
__global__ __launch_bounds__(256) void heads_bwd_kernel(HeadsArgs a, const float* __restrict__ dl,
                                                        const float* __restrict__ dv, T* __restrict__ dh,
                                                        float* __restrict__ partial, int pstride) {
    extern __shared__ float sm[];
    constexpr int PW = MA | 1;
    const int A = AC > 0 ? AC : a.A;
    const int A1 = A + 1;
    float* ws = sm;               // [kHJ][PW]
    float* dzs = sm + kHJ * PW;   // [MA][16]: the row group's dz, action-major, zero past A
    const int tid = threadIdx.x;
    const int64_t ngroups = (a.n + kHR - 1) / kHR;
    float* part = partial + int64_t(blockIdx.x) * pstride;
    const T* h = static_cast<const T*>(a.h);
    float hb = 0.f;
    for (int j0 = 0; j0 < a.J; j0 += kHJ) {
        const int nj = min(kHJ, a.J - j0);
        const int j = j0 + min(tid, nj - 1);
        const bool own = tid < nj;
        __syncthreads();
        stage_head_w<AC, MA>(ws, a, j0, nj);
        float pw[MA];
#pragma unroll
        for (int aa = 0; aa < MA; ++aa) pw[aa] = 0.f;
        float pb = 0.f;
        for (int64_t grp = blockIdx.x; grp < ngroups; grp += gridDim.x) {
            const int64_t r0 = grp * kHR;
            const int nr = int(std::min<int64_t>(kHR, a.n - r0));
            float hv[kHR];
#pragma unroll
            for (int rr = 0; rr < kHR; ++rr) hv[rr] = ld_st(h, std::min<int64_t>(r0 + rr, a.n - 1) * a.J + j);
            __syncthreads();
            {
                // the group's dz, action-major: thread (rr, g) stages actions g, g + 16, ...
                // of row rr; zero past A and for rows past n
                constexpr int U = (MA + 15) / 16;
                const int rr = tid & 15, g = tid >> 4;
                const int64_t rowc = r0 + min(rr, nr - 1);
                const float dvr = dv[rowc];
                float v[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int aa = g + 16 * u;
                    const float x = dl[rowc * A + min(aa, A - 1)];
                    v[u] = rr < nr ? (aa < A ? x : (aa == A ? dvr : 0.f)) : 0.f;
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (g + 16 * u < MA) dzs[(g + 16 * u) * kHR + rr] = v[u];
            }
            __syncthreads();
            if (j0 == 0 && tid < A1) {
#pragma unroll
                for (int rr = 0; rr < kHR; ++rr) hb += dzs[tid * kHR + rr];
            }
#pragma unroll
            for (int rr = 0; rr < kHR; ++rr) hv[rr] = rr < nr ? hv[rr] : 0.f;
            float acc[kHR];
#pragma unroll
            for (int rr = 0; rr < kHR; ++rr) acc[rr] = 0.f;
            const float* wr = ws + min(tid, nj - 1) * PW;
#pragma unroll
            for (int aa = 0; aa < MA; ++aa) {
                const float w = wr[aa];
                const float4* d4 = reinterpret_cast<const float4*>(dzs + aa * kHR);
                float s = pw[aa];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 d = d4[q];
                    acc[4 * q] += d.x * w; s += hv[4 * q] * d.x;
                    acc[4 * q + 1] += d.y * w; s += hv[4 * q + 1] * d.y;
                    acc[4 * q + 2] += d.z * w; s += hv[4 * q + 2] * d.z;
                    acc[4 * q + 3] += d.w * w; s += hv[4 * q + 3] * d.w;
                }
                pw[aa] = s;
                if (aa % 4 == 3) __builtin_amdgcn_sched_barrier(0);   // bounds the LDS reads in flight
            }
            if (own) {
#pragma unroll
                for (int rr = 0; rr < kHR; ++rr) {
                    if (rr < nr) {
                        const int64_t row = r0 + rr;
                        const float v = hv[rr] > 0.f ? acc[rr] : 0.f;
                        if constexpr (sizeof(T) == 2) {
                            const uint16_t b = f2bf(v);
                            dh[row * a.J + j] = b;
                            pb += bf2f(b);
                        } else {
                            dh[row * a.J + j] = v;
                            pb += v;
                        }
                    }
                }
            }
        }
        if (own) {
#pragma unroll
            for (int aa = 0; aa < MA; ++aa)
                if (aa < A1) part[int64_t(aa) * a.J + j] = pw[aa];
            part[int64_t(A1) * a.J + j] = pb;
        }
    }
    if (tid < A1) part[int64_t(A1 + 1) * a.J + tid] = hb;
}

// ---- bf16 backward on the matrix cores, for A + 1 <= 32 outputs and J = 64 * NJB hidden units.
// Per group of 32 rows (the workgroup's groups in turn), with dz = [dlogits | dvalue] rounded to
// bf16 (zero past A and for rows past n) and the head weights Wh (bf16) in LDS:
//   dh[i][j] = (sum_o Wh[j][o] dz[i][o]) * (h[i][j] > 0)      MFMA D[j][i], k = o (one k-step);
//   gW[j][o] += sum_i h[i][j] dz[i][o]                         MFMA D[j][o], k = the 32 rows;
//   dense bias += sum_i dh[i][j] as stored; head bias += sum_i dz[i][o].
// Wave w takes the 16-unit blocks jb = w + 4 u (u < NJB). The h and dz tiles are row-major in
// LDS; the weight-gradient fragments, which run along rows, are read with the transpose read.
// Each workgroup writes the partial layout heads_reduce_kernel sums (the float32 kernel's).
constexpr int kHbRows = 32;
constexpr int kHzP = 40;   // dz tile and weight rows: 32 outputs + 8 (80 bytes, an odd count of 16-byte slots)

// Stages a group of 32 rows for the MFMA head backward: h rows (clamped past n: their dz is
// zero) into the h tile, dz = [dlogits | dvalue] rounded to bf16 (zero past A and for rows past
// n) into the dz tile, thread (rr, c) taking outputs 4c .. 4c+3 of row rr.
template <int NJB>
CB_DEV void hb_stage(const HeadsArgs& a, const float* __restrict__ dl, const float* __restrict__ dv,
                     const uint16_t* __restrict__ h, int64_t r0, int tid, uint16_t* hs, uint16_t* zs) {
    constexpr int J = 64 * NJB, PH = J + 8;
    const int A = a.A;
#pragma unroll
    for (int u = 0; u < NJB; ++u) {
        const int e = tid + 256 * u, rr = e / (J / 8), c = e - rr * (J / 8);
        const int64_t row = std::min<int64_t>(r0 + rr, a.n - 1);
        *reinterpret_cast<uint4*>(hs + rr * PH + c * 8) = *reinterpret_cast<const uint4*>(h + row * J + c * 8);
    }
    const int rr = tid >> 3, c = tid & 7;
    const int64_t rowc = std::min<int64_t>(r0 + rr, a.n - 1);
    const bool live = r0 + rr < a.n;
    const float dvr = dv[rowc];
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int o = 4 * c + e;
        const float x = dl[rowc * A + (o < A ? o : A - 1)];
        v[e] = live ? (o < A ? x : (o == A ? dvr : 0.f)) : 0.f;
    }
    *reinterpret_cast<uint2*>(zs + rr * kHzP + 4 * c) = make_uint2(pack2bf(v[0], v[1]), pack2bf(v[2], v[3]));
}

template <int NJB>
__global__ __launch_bounds__(256) void heads_bwd_mfma_kernel(HeadsArgs a, const float* __restrict__ dl,
                                                             const float* __restrict__ dv, uint16_t* __restrict__ dh,
                                                             float* __restrict__ partial, int pstride) {
    constexpr int J = 64 * NJB, PH = J + 8;   // h tile pitch (elements)
    extern __shared__ __align__(16) uint16_t hsm[];
    uint16_t* wsh = hsm;                       // [J][kHzP]   Wh[j][o]
    uint16_t* hs = wsh + J * kHzP;             // [32][PH]    h rows of the group
    uint16_t* zs = hs + kHbRows * PH;          // [32][kHzP]  dz rows of the group
    const int A = a.A, A1 = A + 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15, jj = r16 >> 2, m = r16 & 3;
    const uint16_t* h = static_cast<const uint16_t*>(a.h);

    // the first group's tiles are staged before the weights, so the two load latencies overlap
    const int64_t ngroups = (a.n + kHbRows - 1) / kHbRows;
    if (blockIdx.x < ngroups) hb_stage<NJB>(a, dl, dv, h, int64_t(blockIdx.x) * kHbRows, tid, hs, zs);

    for (int j = tid; j < J; j += 256) {   // unit j's weights: clamped, unconditional loads
        const float* wr = a.wl + int64_t(j) * A;
        const float wv = a.wv[j];
        float v[kHmOut];
#pragma unroll
        for (int o = 0; o < kHmOut; ++o) {
            const float x = wr[o < A ? o : A - 1];
            v[o] = o < A ? x : (o == A ? wv : 0.f);
        }
#pragma unroll
        for (int c = 0; c < kHmOut / 8; ++c)
            *reinterpret_cast<uint4*>(wsh + j * kHzP + c * 8) =
                make_uint4(pack2bf(v[8 * c], v[8 * c + 1]), pack2bf(v[8 * c + 2], v[8 * c + 3]),
                           pack2bf(v[8 * c + 4], v[8 * c + 5]), pack2bf(v[8 * c + 6], v[8 * c + 7]));
    }

    cb_f32x4 gw[NJB][2];
    float pb[NJB][4];
#pragma unroll
    for (int u = 0; u < NJB; ++u) {
        gw[u][0] = gw[u][1] = cb_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) pb[u][e] = 0.f;
    }
    float hb = 0.f;   // thread o < A1: head bias partial
    __syncthreads();
    for (int64_t grp = blockIdx.x; grp < ngroups; grp += gridDim.x) {
        const int64_t r0 = grp * kHbRows;
        if (grp != int64_t(blockIdx.x)) {
            __syncthreads();   // the previous group's tiles are read
            hb_stage<NJB>(a, dl, dv, h, r0, tid, hs, zs);
            __syncthreads();
        }
        if (tid < A1) {
#pragma unroll 8
            for (int rr = 0; rr < kHbRows; ++rr) hb += bf2f(zs[rr * kHzP + tid]);
        }
        // dz fragments (k = outputs) of the two 16-row tiles; transposed (k = rows) of the two
        // 16-output blocks
        uint4 zf[2], zt[2];
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
            zf[t2] = *reinterpret_cast<const uint4*>(zs + (t2 * 16 + r16) * kHzP + g * 8);
            const uint2 lo = lds_read_tr16(reinterpret_cast<const unsigned char*>(zs + (g * 8 + jj) * kHzP + t2 * 16 + 4 * m));
            const uint2 hi = lds_read_tr16(reinterpret_cast<const unsigned char*>(zs + (g * 8 + 4 + jj) * kHzP + t2 * 16 + 4 * m));
            zt[t2] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
#pragma unroll
        for (int u = 0; u < NJB; ++u) {
            const int jb = wave + 4 * u;
            // dh on the two row tiles
            const uint4 wf = *reinterpret_cast<const uint4*>(wsh + (jb * 16 + r16) * kHzP + g * 8);
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                const cb_f32x4 d = PrecBF16::mma(wf, zf[t2], cb_f32x4{0.f, 0.f, 0.f, 0.f});
                const int rr = t2 * 16 + r16, j0 = jb * 16 + 4 * g;
                const uint2 hm = *reinterpret_cast<const uint2*>(hs + rr * PH + j0);
                const uint32_t u0 = pack2bf(bf_lo(hm.x) > 0.f ? d[0] : 0.f, bf_hi(hm.x) > 0.f ? d[1] : 0.f);
                const uint32_t u1 = pack2bf(bf_lo(hm.y) > 0.f ? d[2] : 0.f, bf_hi(hm.y) > 0.f ? d[3] : 0.f);
                if (r0 + rr < a.n) *reinterpret_cast<uint2*>(dh + (r0 + rr) * J + j0) = make_uint2(u0, u1);
                pb[u][0] += bf_lo(u0); pb[u][1] += bf_hi(u0); pb[u][2] += bf_lo(u1); pb[u][3] += bf_hi(u1);
            }
            // head weight gradient: h^T fragments (k = rows) against dz
            const uint2 lo = lds_read_tr16(reinterpret_cast<const unsigned char*>(hs + (g * 8 + jj) * PH + jb * 16 + 4 * m));
            const uint2 hi = lds_read_tr16(reinterpret_cast<const unsigned char*>(hs + (g * 8 + 4 + jj) * PH + jb * 16 + 4 * m));
            const uint4 hf = make_uint4(lo.x, lo.y, hi.x, hi.y);
#pragma unroll
            for (int ob = 0; ob < 2; ++ob) gw[u][ob] = PrecBF16::mma(hf, zt[ob], gw[u][ob]);
        }
    }
    // ---- partials: [A1][J] weight gradient, [J] dense bias, [A1] head bias
    float* part = partial + int64_t(blockIdx.x) * pstride;
#pragma unroll
    for (int u = 0; u < NJB; ++u) {
        const int j0 = (wave + 4 * u) * 16 + 4 * g;
#pragma unroll
        for (int ob = 0; ob < 2; ++ob) {
            const int o = ob * 16 + r16;
            if (o < A1)
                *reinterpret_cast<float4*>(part + int64_t(o) * J + j0) =
                    make_float4(gw[u][ob][0], gw[u][ob][1], gw[u][ob][2], gw[u][ob][3]);
        }
        // the dense bias: this lane's four units summed over its 16 row lanes, in a fixed order
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float v = pb[u][e];
#pragma unroll
            for (int sh = 1; sh < 16; sh <<= 1) v += __shfl_xor(v, sh, 64);
            pb[u][e] = v;
        }
        if (r16 == 0)
            *reinterpret_cast<float4*>(part + int64_t(A1) * J + j0) = make_float4(pb[u][0], pb[u][1], pb[u][2], pb[u][3]);
    }
    if (tid < A1) part[int64_t(A1 + 1) * J + tid] = hb;
}

struct HeadsOut {
    float* dwl; float* dwv; float* dbl; float* dbv; float* db_dense;
    int J, A;
};

__global__ __launch_bounds__(1024) void heads_reduce_kernel(const float* __restrict__ partial, int nparts,
                                                            int pstride, HeadsOut o) {
    const int A1 = o.A + 1;
    const int64_t nw = int64_t(A1) * o.J, nd = nw + o.J, nt = nd + A1;
    sum_partials_x4(partial, nparts, pstride, [&](int e0, float4 v) {
        const float t[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t e = e0 + u;
            if (e < nw) {
                const int aa = int(e / o.J), j = int(e - int64_t(aa) * o.J);
                if (aa < o.A) o.dwl[int64_t(j) * o.A + aa] = t[u];
                else o.dwv[j] = t[u];
            } else if (e < nd) {
                o.db_dense[e - nw] = t[u];
            } else if (e < nt) {
                const int aa = int(e - nd);
                if (aa < o.A) o.dbl[aa] = t[u];
                else o.dbv[0] = t[u];
            }
        }
    });
}

int heads_pstride(int J, int A) {
    const int64_t ps = int64_t(A + 2) * J + (A + 1);
    return int((ps + 63) / 64 * 64);
}

int heads_bwd_blocks(int64_t n, int J, int A) {
    const int64_t groups = (n + kHR - 1) / kHR;
    const int64_t cap = std::max<int64_t>(1, int64_t(kHeadsPartialCap / size_t(heads_pstride(J, A))));
    return int(std::max<int64_t>(1, std::min<int64_t>({groups, cap, 4096})));
}

std::string heads_shape(const HeadsArgs& a) {
    return std::to_string(a.n) + "x" + std::to_string(a.J) + "x" + std::to_string(a.A);
}

// ---- bf16 forward on the matrix cores: [logits | value] = h Wh + [bl | bv] as an MFMA product
// D[o][i] = sum_j Wh[j][o] h[i][j] with the A + 1 <= 32 outputs in two 16-row blocks (rows past
// A zero) and k = hidden units, 32 per k-step. The workgroup stages Wh rounded to bf16 in LDS
// as [o][j] rows (pitch J + 8 elements: an odd count of 16-byte slots, so the 16 rows of a
// fragment read land on distinct bank groups); each wave takes 16 rows i of h, whose
// B fragments (8 consecutive hidden units of one row) are plain 16-byte loads from h.

__global__ __launch_bounds__(64 * kHmWaves) void heads_fwd_mfma_kernel(HeadsArgs a, float* __restrict__ logits,
                                                                      float* __restrict__ value) {
    extern __shared__ __align__(16) uint16_t wsh[];   // [kHmOut][J + 8]
    const int J = a.J, A = a.A, P = J + 8, nk = J / 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int64_t i0 = (int64_t(blockIdx.x) * kHmWaves + wave) * 16;
    const bool live = i0 < a.n;
    const int64_t ir = live ? std::min<int64_t>(i0 + r16, a.n - 1) : 0;   // rows past n: computed, not stored
    const uint16_t* hrow = static_cast<const uint16_t*>(a.h) + ir * J + g * 8;
    // B fragments of up to eight k-steps in flight at once; the first eight are issued before
    // the weights are staged, so their latencies overlap
    constexpr int KC = 8;
    uint4 bfr[KC];
#pragma unroll
    for (int u = 0; u < KC; ++u)
        if (u < nk) bfr[u] = *reinterpret_cast<const uint4*>(hrow + u * 32);
    for (int j = tid; j < J; j += 64 * kHmWaves) {   // unit j's row: clamped, unconditional loads in flight at once
        const float* wr = a.wl + int64_t(j) * A;
        const float wv = a.wv[j];
        float v[kHmOut];
#pragma unroll
        for (int o = 0; o < kHmOut; ++o) {
            const float x = wr[o < A ? o : A - 1];
            v[o] = o < A ? x : (o == A ? wv : 0.f);
        }
#pragma unroll
        for (int o = 0; o < kHmOut; ++o) wsh[o * P + j] = f2bf(v[o]);
    }
    __syncthreads();
    if (!live) return;
    cb_f32x4 acc[2] = {cb_f32x4{0.f, 0.f, 0.f, 0.f}, cb_f32x4{0.f, 0.f, 0.f, 0.f}};
    for (int c0 = 0; c0 < nk; c0 += KC) {
        if (c0 > 0) {
#pragma unroll
            for (int u = 0; u < KC; ++u)
                if (c0 + u < nk) bfr[u] = *reinterpret_cast<const uint4*>(hrow + (c0 + u) * 32);
        }
#pragma unroll
        for (int u = 0; u < KC; ++u)
            if (c0 + u < nk) {
#pragma unroll
                for (int ob = 0; ob < 2; ++ob) {
                    const uint4 af = *reinterpret_cast<const uint4*>(wsh + (ob * 16 + r16) * P + (c0 + u) * 32 + g * 8);
                    acc[ob] = PrecBF16::mma(af, bfr[u], acc[ob]);
                }
            }
    }
    if (i0 + r16 >= a.n) return;
    const int64_t i = i0 + r16;
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int o = ob * 16 + 4 * g + e;
            if (o < A) logits[i * A + o] = acc[ob][e] + (a.bl ? a.bl[o] : 0.f);
            else if (o == A) value[i] = acc[ob][e] + (a.bv ? a.bv[0] : 0.f);
        }
}

}  // namespace

size_t heads_bwd_partial_floats(int64_t n, int J, int A) {
    return size_t(heads_bwd_blocks(n, J, A)) * size_t(heads_pstride(J, A));
}

namespace {
// Column count of the staged weights: A + 1 when the action count has a compile-time
// variant (18: the Atari action set; 6), else padded to 20 or 68.
int heads_ma(int A) { return A == 18 || A == 6 ? A + 1 : (A + 1 <= 20 ? 20 : 68); }
}  // namespace

hipError_t heads_fwd(int prec, const HeadsArgs& a, float* logits, float* value, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    if (a.A < 1 || a.A > 64 || a.J < 1) return hipErrorInvalidValue;
    ProfScope ps(s, [&] { return cb_key("heads_fwd", prec, heads_shape(a)); });
    if (prec == BF16 && a.A + 1 <= kHmOut && a.J % 32 == 0 && a.J <= 2048 &&
        (reinterpret_cast<uintptr_t>(a.h) & 15) == 0) {
        const int64_t waves = (a.n + 15) / 16;
        const size_t lds = size_t(kHmOut) * (a.J + 8) * sizeof(uint16_t);
        hipLaunchKernelGGL(heads_fwd_mfma_kernel, dim3(unsigned((waves + kHmWaves - 1) / kHmWaves)),
                           dim3(64 * kHmWaves), lds, s, a, logits, value);
        return hipGetLastError();
    }
    const int MA = heads_ma(a.A);
    const size_t lds = std::max(size_t(kHJ) * (MA | 1), size_t(kHJ) * MA) * sizeof(float);
    const dim3 grid(unsigned((a.n + kHR - 1) / kHR));
#define CB_HF(T, AC, MA) hipLaunchKernelGGL((heads_fwd_kernel<T, AC, MA>), grid, dim3(kHJ), lds, s, a, logits, value)
#define CB_HF_ALL(T)                                 \
    if (a.A == 18) CB_HF(T, 18, 19);                 \
    else if (a.A == 6) CB_HF(T, 6, 7);               \
    else if (a.A + 1 <= 20) CB_HF(T, 0, 20);         \
    else CB_HF(T, 0, 68);
    if (prec == BF16) {
        CB_HF_ALL(uint16_t)
    } else {
        CB_HF_ALL(float)
    }
#undef CB_HF_ALL
#undef CB_HF
    return hipGetLastError();
}

hipError_t heads_bwd(int prec, const HeadsArgs& a, const float* dlogits, const float* dvalue, void* dh,
                     float* dwl, float* dbl, float* dwv, float* dbv, float* db_dense, float* partial,
                     size_t partial_floats, hipStream_t s) {
    if (a.A < 1 || a.A > 64 || a.J < 1) return hipErrorInvalidValue;
    const int pstride = heads_pstride(a.J, a.A);
    const int nblk = heads_bwd_blocks(a.n > 0 ? a.n : 1, a.J, a.A);
    if (size_t(nblk) * size_t(pstride) > partial_floats) return hipErrorInvalidValue;
    const int MA = heads_ma(a.A);
    const size_t lds = (size_t(kHJ) * (MA | 1) + size_t(MA) * kHR) * sizeof(float);
    const bool mfma = prec == BF16 && a.A + 1 <= kHmOut && (a.J == 256 || a.J == 512) &&
                      (reinterpret_cast<uintptr_t>(a.h) & 15) == 0 && (reinterpret_cast<uintptr_t>(dh) & 7) == 0;
    if (mfma) {
        const int64_t groups = (std::max<int64_t>(a.n, 1) + kHbRows - 1) / kHbRows;
        const int nb = int(std::min<int64_t>({groups, int64_t(nblk), 256}));
        const size_t lm = (size_t(a.J) * kHzP + size_t(kHbRows) * (a.J + 8) + size_t(kHbRows) * kHzP) * sizeof(uint16_t);
        {
            ProfScope ps(s, [&] { return cb_key("heads_bwd", prec, heads_shape(a)); });
            if (a.J == 256)
                hipLaunchKernelGGL(heads_bwd_mfma_kernel<4>, dim3(unsigned(nb)), dim3(256), lm, s, a, dlogits, dvalue,
                                   static_cast<uint16_t*>(dh), partial, pstride);
            else
                hipLaunchKernelGGL(heads_bwd_mfma_kernel<8>, dim3(unsigned(nb)), dim3(256), lm, s, a, dlogits, dvalue,
                                   static_cast<uint16_t*>(dh), partial, pstride);
        }
        HeadsOut o{dwl, dwv, dbl, dbv, db_dense, a.J, a.A};
        ProfScope ps(s, [&] { return cb_key("heads_reduce", prec, heads_shape(a)); });
        hipLaunchKernelGGL(heads_reduce_kernel, dim3(unsigned((pstride + 63) / 64)), dim3(1024), 0, s, partial, nb,
                           pstride, o);
        return hipGetLastError();
    }
    {
        ProfScope ps(s, [&] { return cb_key("heads_bwd", prec, heads_shape(a)); });
#define CB_HB(T, AC, MA) \
        hipLaunchKernelGGL((heads_bwd_kernel<T, AC, MA>), dim3(unsigned(nblk)), dim3(kHJ), lds, s, a, dlogits, dvalue, \
                           static_cast<T*>(dh), partial, pstride)
#define CB_HB_ALL(T)                                 \
        if (a.A == 18) CB_HB(T, 18, 19);             \
        else if (a.A == 6) CB_HB(T, 6, 7);           \
        else if (a.A + 1 <= 20) CB_HB(T, 0, 20);     \
        else CB_HB(T, 0, 68);
        if (prec == BF16) {
            CB_HB_ALL(uint16_t)
        } else {
            CB_HB_ALL(float)
        }
#undef CB_HB_ALL
#undef CB_HB
    }
    HeadsOut o{dwl, dwv, dbl, dbv, db_dense, a.J, a.A};
    {
        ProfScope ps(s, [&] { return cb_key("heads_reduce", prec, heads_shape(a)); });
        hipLaunchKernelGGL(heads_reduce_kernel, dim3(unsigned((pstride + 63) / 64)), dim3(1024), 0, s, partial, nblk,
                           pstride, o);
    }
    return hipGetLastError();
}

}  // namespace cb
