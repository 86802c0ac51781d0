// Fused policy / value / entropy losses and their logit and value gradients, one thread per
// minibatch row (A <= 64 logits per row), plus the actor's Gumbel-max sampler.
//
// Minibatches up to kFusedRows rows run as one single-workgroup launch (advantage
// statistics, row gradients and loss statistics); callers with a workspace (the learner
// step) spread the row work of such minibatches over many workgroups with results bit-
// identical to the single launch. Larger minibatches reduce over workgroups: per-workgroup
// partial sums in a fixed order, then one workgroup adds them in a fixed order. Every sum is
// float64 and every reduction order is fixed, so results are bit-reproducible.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace cb {

constexpr int kStatThreads = 1024;

// Log-softmax of one row, kept as (zmax, lse): log pi_j = (z_j - zmax) - lse, recomputed from
// the logits where needed (no per-row array, so nothing spills to scratch). Also the entropy.
struct RowLsm {
    float zmax, lse, H;
    CB_DEV float l(float zj) const { return (zj - zmax) - lse; }
};

CB_DEV RowLsm row_log_softmax(const float* z, int A) {
    RowLsm r;
    r.zmax = z[0];
    for (int j = 1; j < A; ++j) r.zmax = fmaxf(r.zmax, z[j]);
    float se = 0.f;
    for (int j = 0; j < A; ++j) se += expf(z[j] - r.zmax);
    r.lse = logf(se);
    r.H = 0.f;
    for (int j = 0; j < A; ++j) {
        const float l = r.l(z[j]);
        r.H -= expf(l) * l;
    }
    return r;
}

struct PpoRow {
    RowLsm s;
    float H, ratio, A_hat, pg, kappa;
    int a;
};

// One row's terms from its logits and the row's scalars (action, behaviour log-prob, raw
// advantage).
CB_DEV PpoRow ppo_row_v(const float* zr, int A, int a, float old_logp, float adv, int norm_adv, float clip,
                        float mean, float std) {
    PpoRow r;
    r.s = row_log_softmax(zr, A);
    r.H = r.s.H;
    r.a = a;
    r.A_hat = adv;
    if (norm_adv) r.A_hat = (r.A_hat - mean) / (std + 1e-8f);
    // an action outside [0, A) poisons the row with NaN instead of reading past the row
    const float la = (r.a >= 0 && r.a < A) ? r.s.l(zr[r.a]) : __builtin_nanf("");
    r.ratio = expf(la - old_logp);
    const float pg1 = -r.A_hat * r.ratio;
    const float pg2 = -r.A_hat * fminf(fmaxf(r.ratio, 1.f - clip), 1.f + clip);
    r.pg = fmaxf(pg1, pg2);
    r.kappa = pg2 > pg1 ? 0.f : 1.f;   // clipped branch strictly larger: no ratio gradient
    return r;
}

// ---- single-workgroup variants for minibatches up to kFusedRows rows: the advantage
// statistics, the per-row gradients and the loss statistics in one launch (each row's terms
// are computed once). Sums are float64: each wave adds its lanes in a fixed butterfly order,
// then every thread adds the wave totals in wave order, so every thread holds the same
// deterministic totals.
constexpr int kFusedThreads = 512;
constexpr int64_t kFusedRows = 16384;

template <int K>
CB_DEV void fused_block_sum(double (&v)[K], double* sh) {
    constexpr int NWV = kFusedThreads / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) v[k] += __shfl_xor(v[k], off);
    if (lane == 0)
#pragma unroll
        for (int k = 0; k < K; ++k) sh[wave * K + k] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        double t = 0.0;
        for (int w = 0; w < NWV; ++w) t += sh[w * K + k];
        v[k] = t;
    }
    __syncthreads();
}

// Rows are processed in chunks: the chunk's logits are read into LDS with coalesced loads,
// each thread works on one row there (writing its logit gradients in place), and the chunk's
// gradients leave with coalesced stores. With the action count fixed at compile time, the
// next chunk's logits and row scalars are loaded into registers while the current chunk is
// being worked on (and the first chunk's during the advantage statistics), so each chunk
// costs its arithmetic rather than a chain of load latencies.
CB_DEV constexpr int fused_chunk_rows(int A) { return (kFusedThreads * 64 / A) < kFusedThreads ? (kFusedThreads * 64 / A) : kFusedThreads; }

// Thread t's share of a chunk's nr * A contiguous logits: elements t, t + 512, ...
template <int LPT>
struct ChunkRegs {
    float v[LPT];
    CB_DEV void load(const float* __restrict__ z, int64_t c0, int nr, int A) {
        const int n = nr * A;
        const float* p = z + c0 * A;
#pragma unroll
        for (int u = 0; u < LPT; ++u) {   // unconditional loads (clamped) keep all in flight
            const int e = u * kFusedThreads + int(threadIdx.x);
            v[u] = p[e < n ? e : n - 1];
        }
    }
    CB_DEV void store(float* zs, int nr, int A) const {
        const int n = nr * A;
#pragma unroll
        for (int u = 0; u < LPT; ++u) {
            const int e = u * kFusedThreads + int(threadIdx.x);
            if (e < n) zs[e] = v[u];
        }
    }
};

template <int AC>
constexpr int fused_lpt() { return AC > 0 ? (fused_chunk_rows(AC) * AC + kFusedThreads - 1) / kFusedThreads : 1; }

struct PpoScal {
    int a;
    float olp, adv, ret, val;
};

// Row i's source row (rows past m read row m - 1: unconditional loads stay in flight; such
// rows are never used). Issued before a chunk's logits so that waiting for it does not wait
// for them (loads complete in order).
template <bool ROWS>
CB_DEV int64_t ppo_src(int64_t i, int64_t m, const int32_t* __restrict__ rows) {
    const int64_t ic = i < m ? i : m - 1;
    if constexpr (ROWS) return rows[ic];
    else return ic;
}

CB_DEV PpoScal ppo_scal(int64_t i, int64_t m, int64_t src, const int32_t* __restrict__ act,
                        const float* __restrict__ old_logp, const float* __restrict__ adv,
                        const float* __restrict__ ret, const float* __restrict__ val) {
    const int64_t ic = i < m ? i : m - 1;
    return PpoScal{act[src], old_logp[src], adv[src], ret[src], val[ic]};
}

// This thread's float64 sums of the minibatch advantages and their squares (rows tid,
// tid + 512, ...), four rows' loads in flight. The block sum and the mean / population std
// follow in adv_mean_std.
template <bool ROWS>
CB_DEV void adv_sums(int64_t m, const float* __restrict__ adv, const int32_t* __restrict__ rows, double (&ms)[2]) {
    ms[0] = 0.0;
    ms[1] = 0.0;
    for (int64_t i0 = threadIdx.x; i0 < m; i0 += 4 * kFusedThreads) {
        int64_t src[4];
        float av[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            src[u] = ppo_src<ROWS>(i0 + u * kFusedThreads, m, rows);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) av[u] = adv[src[u]];
        __builtin_amdgcn_sched_barrier(0);   // all four gathers in flight before the first use
#pragma unroll
        for (int u = 0; u < 4; ++u) {   // rows past m add zero
            const double a = i0 + u * kFusedThreads < m ? double(av[u]) : 0.0;
            ms[0] += a;
            ms[1] += a * a;
        }
    }
}

CB_DEV void adv_mean_std(int64_t m, double (&ms)[2], double* sh, float& mean, float& std) {
    fused_block_sum<2>(ms, sh);
    const double dmean = ms[0] / double(m), dvar = ms[1] / double(m) - dmean * dmean;
    mean = float(dmean);
    std = float(sqrt(dvar > 0.0 ? dvar : 0.0));
}

// AC > 0 fixes the action count at compile time (the row loops unroll); 0 reads it from A_.
// ROWS: the rows are gathered through `rows` (else rows is NULL and row i is row i).
template <int AC, bool ROWS>
__global__ __launch_bounds__(kFusedThreads) void ppo_fused_kernel(
    int64_t m, int A_, const float* __restrict__ z, const float* __restrict__ val,
    const int32_t* __restrict__ act, const float* __restrict__ old_logp,
    const float* __restrict__ adv, const float* __restrict__ ret, const int32_t* __restrict__ rows,
    int norm_adv, float clip, float vf, float ent, float* __restrict__ dz, float* __restrict__ dv,
    float* __restrict__ stats) {
    extern __shared__ float zs[];   // [chunk rows][A]
    __shared__ double sh[(kFusedThreads / 64) * 5];
    const int A = AC > 0 ? AC : A_;
    const int tid = threadIdx.x;
    const int CR = fused_chunk_rows(A);
    // the advantage sums' loads first (loads complete in order), then the first chunk's
    // prefetch, which the block sum overlaps
    double ms[2];
    adv_sums<ROWS>(m, adv, rows, ms);
    ChunkRegs<fused_lpt<AC>()> cz;
    PpoScal nx{};
    if constexpr (AC > 0) {
        const int64_t src = ppo_src<ROWS>(tid, m, rows);
        cz.load(z, 0, int(m < CR ? m : CR), A);
        nx = ppo_scal(tid, m, src, act, old_logp, adv, ret, val);
    }
    float mean, std;
    adv_mean_std(m, ms, sh, mean, std);
    // rows: gradients and loss terms
    const float inv_m = 1.f / float(m);
    double st[5] = {0, 0, 0, 0, 0};
    for (int64_t c0 = 0; c0 < m; c0 += CR) {
        const int nr = m - c0 < CR ? int(m - c0) : CR;
        __syncthreads();   // the previous chunk's gradients have left LDS
        PpoScal cur;
        if constexpr (AC > 0) {
            cz.store(zs, nr, A);
            cur = nx;
            if (c0 + CR < m) {
                const int64_t c1 = c0 + CR;
                const int64_t src = ppo_src<ROWS>(c1 + tid, m, rows);
                cz.load(z, c1, int(m - c1 < CR ? m - c1 : CR), A);
                nx = ppo_scal(c1 + tid, m, src, act, old_logp, adv, ret, val);
            }
        } else {
            for (int e = tid; e < nr * A; e += kFusedThreads) zs[e] = z[c0 * A + e];
            cur = ppo_scal(c0 + tid, m, ppo_src<ROWS>(c0 + tid, m, rows), act, old_logp, adv, ret, val);
        }
        __syncthreads();
        if (tid < nr) {
            const int64_t i = c0 + tid;
            float* zr = zs + tid * A;
            const PpoRow r = ppo_row_v(zr, A, cur.a, cur.olp, cur.adv, norm_adv, clip, mean, std);
            const float coef = -r.kappa * r.A_hat * r.ratio;
            for (int j = 0; j < A; ++j) {
                const float l = r.s.l(zr[j]);
                const float p = expf(l);
                zr[j] = (coef * ((j == r.a ? 1.f : 0.f) - p) + ent * p * (l + r.H)) * inv_m;
            }
            const float vi = cur.val, ri = cur.ret;
            dv[i] = vf * (vi - ri) * inv_m;
            const double dvl = double(vi) - double(ri);
            st[0] += r.pg;
            st[1] += dvl * dvl;
            st[2] += r.H;
            st[3] += double(r.ratio - 1.f) - double(logf(r.ratio));
            st[4] += fabsf(r.ratio - 1.f) > clip ? 1.0 : 0.0;
        }
        __syncthreads();
        for (int e = tid; e < nr * A; e += kFusedThreads) dz[c0 * A + e] = zs[e];
    }
    fused_block_sum<5>(st, sh);
    if (tid == 0) {
        const double inv = 1.0 / double(m);
        const double pg = st[0] * inv, vl = 0.5 * st[1] * inv, H = st[2] * inv;
        stats[0] = float(pg + vf * vl - ent * H);
        stats[1] = float(pg); stats[2] = float(vl); stats[3] = float(H);
        stats[4] = float(st[3] * inv); stats[5] = float(st[4] * inv);
        stats[6] = mean; stats[7] = std;
    }
}

struct ImpScal {
    int a;
    float adv, val, vs;
};

CB_DEV ImpScal imp_scal(int64_t i, int64_t m, const int32_t* __restrict__ act, const float* __restrict__ pgadv,
                        const float* __restrict__ val, const float* __restrict__ vs) {
    const int64_t ic = i < m ? i : m - 1;
    return ImpScal{act[ic], pgadv[ic], val[ic], vs[ic]};
}

template <int AC>
__global__ __launch_bounds__(kFusedThreads) void impala_fused_kernel(
    int64_t m, int A_, const float* __restrict__ z, const float* __restrict__ val,
    const int32_t* __restrict__ act, const float* __restrict__ vs, const float* __restrict__ pgadv,
    float pgc, float vf, float ent, float* __restrict__ dz, float* __restrict__ dv,
    float* __restrict__ stats) {
    extern __shared__ float zs[];   // [chunk rows][A]
    __shared__ double sh[(kFusedThreads / 64) * 5];
    const int A = AC > 0 ? AC : A_;
    const int tid = threadIdx.x;
    const float inv_m = 1.f / float(m);
    const int CR = fused_chunk_rows(A);
    ChunkRegs<fused_lpt<AC>()> cz;
    ImpScal nx{};
    if constexpr (AC > 0) {
        cz.load(z, 0, int(m < CR ? m : CR), A);
        nx = imp_scal(tid, m, act, pgadv, val, vs);
    }
    double st[5] = {0, 0, 0, 0, 0};
    for (int64_t c0 = 0; c0 < m; c0 += CR) {
        const int nr = m - c0 < CR ? int(m - c0) : CR;
        __syncthreads();
        ImpScal cur;
        if constexpr (AC > 0) {
            cz.store(zs, nr, A);
            cur = nx;
            if (c0 + CR < m) {
                const int64_t c1 = c0 + CR;
                cz.load(z, c1, int(m - c1 < CR ? m - c1 : CR), A);
                nx = imp_scal(c1 + tid, m, act, pgadv, val, vs);
            }
        } else {
            for (int e = tid; e < nr * A; e += kFusedThreads) zs[e] = z[c0 * A + e];
            cur = imp_scal(c0 + tid, m, act, pgadv, val, vs);
        }
        __syncthreads();
        if (tid < nr) {
            const int64_t i = c0 + tid;
            float* zr = zs + tid * A;
            const RowLsm rs = row_log_softmax(zr, A);
            const float H = rs.H;
            const int a = cur.a;
            const float adv = cur.adv;
            const bool a_ok = a >= 0 && a < A;
            const double la = a_ok ? double(rs.l(zr[a])) : double(__builtin_nanf(""));
            for (int j = 0; j < A; ++j) {
                const float l = rs.l(zr[j]);
                const float p = expf(l);
                zr[j] = a_ok ? (-pgc * adv * ((j == a ? 1.f : 0.f) - p) + ent * p * (l + H)) * inv_m
                             : __builtin_nanf("");
            }
            const float vi = cur.val, vsi = cur.vs;
            dv[i] = vf * (vi - vsi) * inv_m;
            const double dvl = double(vi) - double(vsi);
            st[0] += -double(adv) * la;
            st[1] += dvl * dvl;
            st[2] += H;
            st[3] += adv;
            st[4] += vsi;
        }
        __syncthreads();
        for (int e = tid; e < nr * A; e += kFusedThreads) dz[c0 * A + e] = zs[e];
    }
    fused_block_sum<5>(st, sh);
    if (tid == 0) {
        const double inv = 1.0 / double(m);
        const double pg = st[0] * inv, vl = 0.5 * st[1] * inv, H = st[2] * inv;
        stats[0] = float(pgc * pg + vf * vl - ent * H);
        stats[1] = float(pg); stats[2] = float(vl); stats[3] = float(H);
        stats[4] = float(st[3] * inv); stats[5] = float(st[4] * inv);
        stats[6] = 0.f; stats[7] = 0.f;
    }
}

// ---- wide variants for callers with a workspace (the learner step). The same arithmetic as
// the single-workgroup kernels, spread over many workgroups: (1) one workgroup forms the
// advantage statistics exactly as the fused kernel does; (2) one thread per row forms the
// row's gradients and its five loss terms (stored per row, float64); (3) one workgroup adds
// the row terms in the fused kernel's order (thread t: rows t, t + 512, ...; then the same
// block sum). Every output is bit-identical to the single-workgroup kernel's.
constexpr int kWideRows = 256;   // rows (one per thread) per workgroup of (2)

size_t loss_ws_bytes(int64_t m) { return 256 + size_t(m > 0 ? m : 1) * 5 * sizeof(double); }

// Workgroup u: the statistics of the minibatch at rows + (u / per) * stride2 + (u % per) *
// stride (one launch can serve every minibatch of a learning phase; each workgroup's
// arithmetic is the single minibatch's).
template <bool ROWS>
__global__ __launch_bounds__(kFusedThreads) void adv_stats_ws_kernel(int64_t m, const float* __restrict__ adv,
                                                                   const int32_t* __restrict__ rows, int64_t stride,
                                                                   int per, int64_t stride2,
                                                                   float* __restrict__ ms_out) {
    __shared__ double sh[(kFusedThreads / 64) * 5];
    double ms[2];
    const int u = int(blockIdx.x);
    adv_sums<ROWS>(m, adv, ROWS ? rows + int64_t(u / per) * stride2 + int64_t(u % per) * stride : rows, ms);
    float mean, std;
    adv_mean_std(m, ms, sh, mean, std);
    if (threadIdx.x == 0) { ms_out[2 * blockIdx.x] = mean; ms_out[2 * blockIdx.x + 1] = std; }
}

bool ppo_adv_stats_batched(int64_t m) { return m > kWideRows && m <= kFusedRows; }

hipError_t ppo_adv_stats(int64_t m, int nmb, const float* adv, const int32_t* rows, int64_t stride, int per,
                         int64_t stride2, float* ms, hipStream_t s) {
    if (m <= 0 || nmb <= 0 || per <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "ppo_adv_stats/" + std::to_string(m) + "x" + std::to_string(nmb); });
    if (rows)
        hipLaunchKernelGGL(adv_stats_ws_kernel<true>, dim3(unsigned(nmb)), dim3(kFusedThreads), 0, s, m, adv, rows,
                           stride, per, stride2, ms);
    else
        hipLaunchKernelGGL(adv_stats_ws_kernel<false>, dim3(unsigned(nmb)), dim3(kFusedThreads), 0, s, m, adv, rows,
                           stride, per, stride2, ms);
    return hipGetLastError();
}

// The workgroup's rows' logits into LDS with coalesced loads (unconditional, clamped; all in
// flight before the first store).
template <int AC>
CB_DEV void stage_rows(float* zs, const float* __restrict__ z, int64_t r0, int nr, int A) {
    if constexpr (AC > 0) {
        const int n = nr * AC;
        const float* p = z + r0 * AC;
        float v[AC];
#pragma unroll
        for (int u = 0; u < AC; ++u) {
            const int e = u * kWideRows + int(threadIdx.x);
            v[u] = p[e < n ? e : n - 1];
        }
#pragma unroll
        for (int u = 0; u < AC; ++u) {
            const int e = u * kWideRows + int(threadIdx.x);
            if (e < n) zs[e] = v[u];
        }
    } else {
        for (int e = threadIdx.x; e < nr * A; e += kWideRows) zs[e] = z[r0 * A + e];
    }
}

template <int AC, bool ROWS>
__global__ __launch_bounds__(kWideRows) void ppo_rows_ws_kernel(
    int64_t m, int A_, const float* __restrict__ z, const float* __restrict__ val,
    const int32_t* __restrict__ act, const float* __restrict__ old_logp,
    const float* __restrict__ adv, const float* __restrict__ ret, const int32_t* __restrict__ rows,
    int norm_adv, float clip, float vf, float ent, float* __restrict__ dz, float* __restrict__ dv,
    const float* __restrict__ ms, double* __restrict__ terms) {
    extern __shared__ float zs[];   // [kWideRows][A]
    const int A = AC > 0 ? AC : A_;
    const int tid = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * kWideRows;
    const int nr = m - r0 < kWideRows ? int(m - r0) : kWideRows;
    const int64_t src = ppo_src<ROWS>(r0 + tid, m, rows);
    stage_rows<AC>(zs, z, r0, nr, A);
    const PpoScal cur = ppo_scal(r0 + tid, m, src, act, old_logp, adv, ret, val);
    const float mean = ms[0], std = ms[1];
    const float inv_m = 1.f / float(m);
    __syncthreads();
    if (tid < nr) {
        const int64_t i = r0 + tid;
        float* zr = zs + tid * A;
        const PpoRow r = ppo_row_v(zr, A, cur.a, cur.olp, cur.adv, norm_adv, clip, mean, std);
        const float coef = -r.kappa * r.A_hat * r.ratio;
        for (int j = 0; j < A; ++j) {
            const float l = r.s.l(zr[j]);
            const float p = expf(l);
            zr[j] = (coef * ((j == r.a ? 1.f : 0.f) - p) + ent * p * (l + r.H)) * inv_m;
        }
        const float vi = cur.val, ri = cur.ret;
        dv[i] = vf * (vi - ri) * inv_m;
        const double dvl = double(vi) - double(ri);
        double* tr = terms + i * 5;
        tr[0] = r.pg;
        tr[1] = dvl * dvl;
        tr[2] = r.H;
        tr[3] = double(r.ratio - 1.f) - double(logf(r.ratio));
        tr[4] = fabsf(r.ratio - 1.f) > clip ? 1.0 : 0.0;
    }
    __syncthreads();
    for (int e = tid; e < nr * A; e += kWideRows) dz[r0 * A + e] = zs[e];
}

template <int AC>
__global__ __launch_bounds__(kWideRows) void impala_rows_ws_kernel(
    int64_t m, int A_, const float* __restrict__ z, const float* __restrict__ val,
    const int32_t* __restrict__ act, const float* __restrict__ vs, const float* __restrict__ pgadv,
    float pgc, float vf, float ent, float* __restrict__ dz, float* __restrict__ dv, double* __restrict__ terms) {
    extern __shared__ float zs[];   // [kWideRows][A]
    const int A = AC > 0 ? AC : A_;
    const int tid = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * kWideRows;
    const int nr = m - r0 < kWideRows ? int(m - r0) : kWideRows;
    stage_rows<AC>(zs, z, r0, nr, A);
    const ImpScal cur = imp_scal(r0 + tid, m, act, pgadv, val, vs);
    const float inv_m = 1.f / float(m);
    __syncthreads();
    if (tid < nr) {
        const int64_t i = r0 + tid;
        float* zr = zs + tid * A;
        const RowLsm rs = row_log_softmax(zr, A);
        const float H = rs.H;
        const int a = cur.a;
        const float advv = cur.adv;
        const bool a_ok = a >= 0 && a < A;
        const double la = a_ok ? double(rs.l(zr[a])) : double(__builtin_nanf(""));
        for (int j = 0; j < A; ++j) {
            const float l = rs.l(zr[j]);
            const float p = expf(l);
            zr[j] = a_ok ? (-pgc * advv * ((j == a ? 1.f : 0.f) - p) + ent * p * (l + H)) * inv_m
                         : __builtin_nanf("");
        }
        const float vi = cur.val, vsi = cur.vs;
        dv[i] = vf * (vi - vsi) * inv_m;
        const double dvl = double(vi) - double(vsi);
        double* tr = terms + i * 5;
        tr[0] = -double(advv) * la;
        tr[1] = dvl * dvl;
        tr[2] = H;
        tr[3] = advv;
        tr[4] = vsi;
    }
    __syncthreads();
    for (int e = tid; e < nr * A; e += kWideRows) dz[r0 * A + e] = zs[e];
}

// (3): the row terms summed in the fused kernel's order, then its statistics.
template <bool PPO>
__global__ __launch_bounds__(kFusedThreads) void loss_final_ws_kernel(int64_t m, float pgc, float vf, float ent,
                                                                    const double* __restrict__ terms,
                                                                    const float* __restrict__ ms,
                                                                    float* __restrict__ stats) {
    __shared__ double sh[(kFusedThreads / 64) * 5];
    double st[5] = {0, 0, 0, 0, 0};
    for (int64_t i = threadIdx.x; i < m; i += kFusedThreads) {
#pragma unroll
        for (int k = 0; k < 5; ++k) st[k] += terms[i * 5 + k];
    }
    fused_block_sum<5>(st, sh);
    if (threadIdx.x == 0) {
        const double inv = 1.0 / double(m);
        const double pg = st[0] * inv, vl = 0.5 * st[1] * inv, H = st[2] * inv;
        stats[0] = float(PPO ? pg + vf * vl - ent * H : pgc * pg + vf * vl - ent * H);
        stats[1] = float(pg); stats[2] = float(vl); stats[3] = float(H);
        stats[4] = float(st[3] * inv); stats[5] = float(st[4] * inv);
        stats[6] = PPO ? ms[0] : 0.f;
        stats[7] = PPO ? ms[1] : 0.f;
    }
}

// ---- minibatches beyond kFusedRows rows: every reduction over workgroups. Each workgroup
// (kWideRows rows, one per thread) reduces its rows' advantage sums or loss terms in a fixed
// order into one partial; a single workgroup then adds the partials in a fixed order. The
// partials live in the caller's workspace when there is one; without it they live in dvalue
// before the gradients are written there (its m floats hold the 5 doubles per 256 rows).
// With a workspace the row kernel forms the gradients and the loss partials in one pass over
// the logits; without it a first pass forms the partials and a second one the gradients.
template <bool ROWS>
__global__ __launch_bounds__(kWideRows) void adv_part_kernel(int64_t m, const float* __restrict__ adv,
                                                           const int32_t* __restrict__ rows,
                                                           double* __restrict__ part) {
    __shared__ double sh[kWideRows];
    const int64_t i = int64_t(blockIdx.x) * kWideRows + threadIdx.x;
    const double a = i < m ? double(adv[ppo_src<ROWS>(i, m, rows)]) : 0.0;
    const double s = block_sum<kWideRows>(a, sh);
    const double s2 = block_sum<kWideRows>(a * a, sh);
    if (threadIdx.x == 0) {
        part[2 * blockIdx.x] = s;
        part[2 * blockIdx.x + 1] = s2;
    }
}

// One workgroup adds nb partials of K doubles (thread t: partials t, t + kStatThreads, ...;
// then a fixed tree) and writes the statistics. KIND 0: advantage mean and population std
// into stats[6], stats[7]; 1: PPO loss statistics into stats[0..5]; 2: IMPALA's into
// stats[0..7].
template <int K, int KIND>
__global__ __launch_bounds__(kStatThreads) void part_final_kernel(int64_t m, int nb, float pgc, float vf,
                                                                  float ent, const double* __restrict__ part,
                                                                  float* __restrict__ stats) {
    __shared__ double sh[kStatThreads];
    double st[K];
#pragma unroll
    for (int k = 0; k < K; ++k) st[k] = 0.0;
    for (int b = threadIdx.x; b < nb; b += kStatThreads)
#pragma unroll
        for (int k = 0; k < K; ++k) st[k] += part[int64_t(b) * K + k];
    double tot[K];
#pragma unroll
    for (int k = 0; k < K; ++k) tot[k] = block_sum<kStatThreads>(st[k], sh);
    if (threadIdx.x != 0) return;
    const double inv = 1.0 / double(m);
    if constexpr (KIND == 0) {
        const double mean = tot[0] * inv, var = tot[1] * inv - mean * mean;
        stats[6] = float(mean);
        stats[7] = float(sqrt(var > 0.0 ? var : 0.0));
    } else {
        const double pg = tot[0] * inv, vl = 0.5 * tot[1] * inv, H = tot[2] * inv;
        stats[0] = float(KIND == 1 ? pg + vf * vl - ent * H : pgc * pg + vf * vl - ent * H);
        stats[1] = float(pg); stats[2] = float(vl); stats[3] = float(H);
        stats[4] = float(tot[3] * inv); stats[5] = float(tot[4] * inv);
        if constexpr (KIND == 2) { stats[6] = 0.f; stats[7] = 0.f; }
    }
}

// This workgroup's five loss terms, reduced in a fixed order into part[5 * blockIdx.x ..].
CB_DEV void block_terms(const double (&t)[5], double* sh, double* __restrict__ part) {
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const double s = block_sum<kWideRows>(t[k], sh);
        if (threadIdx.x == 0) part[5 * int64_t(blockIdx.x) + k] = s;
    }
}

// PPO rows of a large minibatch: GRAD writes dlogits / dvalue, PART the loss partials; the
// advantage statistics come from stats[6], stats[7].
template <int AC, bool ROWS, bool GRAD, bool PART>
__global__ __launch_bounds__(kWideRows) void ppo_big_rows_kernel(
    int64_t m, int A_, const float* __restrict__ z, const float* __restrict__ val,
    const int32_t* __restrict__ act, const float* __restrict__ old_logp,
    const float* __restrict__ adv, const float* __restrict__ ret, const int32_t* __restrict__ rows,
    int norm_adv, float clip, float vf, float ent, float* __restrict__ dz, float* __restrict__ dv,
    const float* __restrict__ stats, double* __restrict__ part) {
    extern __shared__ float zs[];   // [kWideRows][A]
    __shared__ double sh[kWideRows];
    const int A = AC > 0 ? AC : A_;
    const int tid = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * kWideRows;
    const int nr = m - r0 < kWideRows ? int(m - r0) : kWideRows;
    const int64_t src = ppo_src<ROWS>(r0 + tid, m, rows);
    stage_rows<AC>(zs, z, r0, nr, A);
    const PpoScal cur = ppo_scal(r0 + tid, m, src, act, old_logp, adv, ret, val);
    const float mean = stats[6], std = stats[7];
    const float inv_m = 1.f / float(m);
    __syncthreads();
    double t[5] = {0, 0, 0, 0, 0};
    if (tid < nr) {
        const int64_t i = r0 + tid;
        float* zr = zs + tid * A;
        const PpoRow r = ppo_row_v(zr, A, cur.a, cur.olp, cur.adv, norm_adv, clip, mean, std);
        if constexpr (GRAD) {
            const float coef = -r.kappa * r.A_hat * r.ratio;
            for (int j = 0; j < A; ++j) {
                const float l = r.s.l(zr[j]);
                const float p = expf(l);
                zr[j] = (coef * ((j == r.a ? 1.f : 0.f) - p) + ent * p * (l + r.H)) * inv_m;
            }
            dv[i] = vf * (cur.val - cur.ret) * inv_m;
        }
        const double dvl = double(cur.val) - double(cur.ret);
        t[0] = r.pg;
        t[1] = dvl * dvl;
        t[2] = r.H;
        t[3] = double(r.ratio - 1.f) - double(logf(r.ratio));
        t[4] = fabsf(r.ratio - 1.f) > clip ? 1.0 : 0.0;
    }
    if constexpr (PART) block_terms(t, sh, part);
    if constexpr (GRAD) {
        __syncthreads();
        for (int e = tid; e < nr * A; e += kWideRows) dz[r0 * A + e] = zs[e];
    }
}

template <int AC, bool GRAD, bool PART>
__global__ __launch_bounds__(kWideRows) void impala_big_rows_kernel(
    int64_t m, int A_, const float* __restrict__ z, const float* __restrict__ val,
    const int32_t* __restrict__ act, const float* __restrict__ vs, const float* __restrict__ pgadv,
    float pgc, float vf, float ent, float* __restrict__ dz, float* __restrict__ dv, double* __restrict__ part) {
    extern __shared__ float zs[];   // [kWideRows][A]
    __shared__ double sh[kWideRows];
    const int A = AC > 0 ? AC : A_;
    const int tid = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * kWideRows;
    const int nr = m - r0 < kWideRows ? int(m - r0) : kWideRows;
    stage_rows<AC>(zs, z, r0, nr, A);
    const ImpScal cur = imp_scal(r0 + tid, m, act, pgadv, val, vs);
    const float inv_m = 1.f / float(m);
    __syncthreads();
    double t[5] = {0, 0, 0, 0, 0};
    if (tid < nr) {
        const int64_t i = r0 + tid;
        float* zr = zs + tid * A;
        const RowLsm rs = row_log_softmax(zr, A);
        const int a = cur.a;
        const bool a_ok = a >= 0 && a < A;
        const double la = a_ok ? double(rs.l(zr[a])) : double(__builtin_nanf(""));
        if constexpr (GRAD) {
            for (int j = 0; j < A; ++j) {
                const float l = rs.l(zr[j]);
                const float p = expf(l);
                zr[j] = a_ok ? (-pgc * cur.adv * ((j == a ? 1.f : 0.f) - p) + ent * p * (l + rs.H)) * inv_m
                             : __builtin_nanf("");
            }
            dv[i] = vf * (cur.val - cur.vs) * inv_m;
        }
        const double dvl = double(cur.val) - double(cur.vs);
        t[0] = -double(cur.adv) * la;
        t[1] = dvl * dvl;
        t[2] = rs.H;
        t[3] = cur.adv;
        t[4] = cur.vs;
    }
    if constexpr (PART) block_terms(t, sh, part);
    if constexpr (GRAD) {
        __syncthreads();
        for (int e = tid; e < nr * A; e += kWideRows) dz[r0 * A + e] = zs[e];
    }
}

// The partial buffer: the workspace's, else dvalue's memory (8-byte aligned within it).
static double* big_part(void* ws, float* dv) {
    if (ws) return reinterpret_cast<double*>(static_cast<char*>(ws) + 256);
    const uintptr_t p = reinterpret_cast<uintptr_t>(dv);
    return reinterpret_cast<double*>(p & 7 ? p + 4 : p);
}

static hipError_t ppo_loss_big(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                               const float* old_logp, const float* adv, const float* ret, const int32_t* rows,
                               int norm_adv, float clip, float vf, float ent, float* dz, float* dv, float* stats,
                               void* ws, hipStream_t s) {
    const int nb = int((m + kWideRows - 1) / kWideRows);
    const size_t lds = size_t(kWideRows) * A * sizeof(float);
    double* part = big_part(ws, dv);
    if (rows) hipLaunchKernelGGL(adv_part_kernel<true>, dim3(nb), dim3(kWideRows), 0, s, m, adv, rows, part);
    else hipLaunchKernelGGL(adv_part_kernel<false>, dim3(nb), dim3(kWideRows), 0, s, m, adv, rows, part);
    hipLaunchKernelGGL((part_final_kernel<2, 0>), dim3(1), dim3(kStatThreads), 0, s, m, nb, 0.f, vf, ent, part, stats);
#define CB_PB(AC, RW, GR, PT) \
    hipLaunchKernelGGL((ppo_big_rows_kernel<AC, RW, GR, PT>), dim3(nb), dim3(kWideRows), lds, s, m, A, z, v, act, \
                       old_logp, adv, ret, rows, norm_adv, clip, vf, ent, dz, dv, stats, part)
#define CB_PBA(RW, GR, PT) \
    if (A == 18) CB_PB(18, RW, GR, PT); else if (A == 6) CB_PB(6, RW, GR, PT); else CB_PB(0, RW, GR, PT)
#define CB_PBR(GR, PT) \
    if (rows) { CB_PBA(true, GR, PT); } else { CB_PBA(false, GR, PT); }
    if (ws) {
        CB_PBR(true, true);
        hipLaunchKernelGGL((part_final_kernel<5, 1>), dim3(1), dim3(kStatThreads), 0, s, m, nb, 0.f, vf, ent, part,
                           stats);
    } else {
        CB_PBR(false, true);
        hipLaunchKernelGGL((part_final_kernel<5, 1>), dim3(1), dim3(kStatThreads), 0, s, m, nb, 0.f, vf, ent, part,
                           stats);
        CB_PBR(true, false);
    }
#undef CB_PBR
#undef CB_PBA
#undef CB_PB
    return hipGetLastError();
}

static hipError_t impala_loss_big(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                                  const float* vs, const float* pg, float pgc, float vf, float ent, float* dz,
                                  float* dv, float* stats, void* ws, hipStream_t s) {
    const int nb = int((m + kWideRows - 1) / kWideRows);
    const size_t lds = size_t(kWideRows) * A * sizeof(float);
    double* part = big_part(ws, dv);
#define CB_IB(AC, GR, PT) \
    hipLaunchKernelGGL((impala_big_rows_kernel<AC, GR, PT>), dim3(nb), dim3(kWideRows), lds, s, m, A, z, v, act, vs, \
                       pg, pgc, vf, ent, dz, dv, part)
#define CB_IBA(GR, PT) \
    if (A == 18) CB_IB(18, GR, PT); else if (A == 6) CB_IB(6, GR, PT); else CB_IB(0, GR, PT)
    if (ws) {
        CB_IBA(true, true);
        hipLaunchKernelGGL((part_final_kernel<5, 2>), dim3(1), dim3(kStatThreads), 0, s, m, nb, pgc, vf, ent, part,
                           stats);
    } else {
        CB_IBA(false, true);
        hipLaunchKernelGGL((part_final_kernel<5, 2>), dim3(1), dim3(kStatThreads), 0, s, m, nb, pgc, vf, ent, part,
                           stats);
        CB_IBA(true, false);
    }
#undef CB_IBA
#undef CB_IB
    return hipGetLastError();
}

static size_t fused_lds(int A) {
    const int cr = std::min(kFusedThreads * 64 / A, kFusedThreads);
    return size_t(cr) * A * sizeof(float);
}

hipError_t ppo_loss(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                    const float* old_logp, const float* adv, const float* ret, const int32_t* rows,
                    int norm_adv, float clip, float vf, float ent, float* dz, float* dv, float* stats,
                    hipStream_t s) {
    if (m <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "ppo_loss/" + cb_dims(int(m), A); });
    if (m <= kFusedRows) {
        auto k = rows ? (A == 18 ? ppo_fused_kernel<18, true> : (A == 6 ? ppo_fused_kernel<6, true> : ppo_fused_kernel<0, true>))
                      : (A == 18 ? ppo_fused_kernel<18, false>
                                 : (A == 6 ? ppo_fused_kernel<6, false> : ppo_fused_kernel<0, false>));
        hipLaunchKernelGGL(k, dim3(1), dim3(kFusedThreads), fused_lds(A), s, m, A, z, v, act, old_logp, adv, ret, rows,
                           norm_adv, clip, vf, ent, dz, dv, stats);
        return hipGetLastError();
    }
    return ppo_loss_big(m, A, z, v, act, old_logp, adv, ret, rows, norm_adv, clip, vf, ent, dz, dv, stats, nullptr,
                        s);
}

hipError_t impala_loss(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                       const float* vs, const float* pg, float pgc, float vf, float ent, float* dz,
                       float* dv, float* stats, hipStream_t s) {
    if (m <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "impala_loss/" + cb_dims(int(m), A); });
    if (m <= kFusedRows) {
        auto k = A == 18 ? impala_fused_kernel<18> : (A == 6 ? impala_fused_kernel<6> : impala_fused_kernel<0>);
        hipLaunchKernelGGL(k, dim3(1), dim3(kFusedThreads), fused_lds(A), s, m, A, z, v, act, vs, pg, pgc, vf, ent, dz,
                           dv, stats);
        return hipGetLastError();
    }
    return impala_loss_big(m, A, z, v, act, vs, pg, pgc, vf, ent, dz, dv, stats, nullptr, s);
}

hipError_t ppo_loss_ws(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                       const float* old_logp, const float* adv, const float* ret, const int32_t* rows,
                       int norm_adv, float clip, float vf, float ent, float* dz, float* dv, float* stats,
                       void* ws, hipStream_t s, const float* ms_pre) {
    if (m <= 0) return hipSuccess;
    if (m <= kWideRows)   // one workgroup's worth
        return ppo_loss(m, A, z, v, act, old_logp, adv, ret, rows, norm_adv, clip, vf, ent, dz, dv, stats, s);
    if (m > kFusedRows) {
        ProfScope ps(s, [&] { return "ppo_loss/" + cb_dims(int(m), A); });
        return ppo_loss_big(m, A, z, v, act, old_logp, adv, ret, rows, norm_adv, clip, vf, ent, dz, dv, stats, ws, s);
    }
    const float* ms = ms_pre ? ms_pre : static_cast<const float*>(ws);
    double* terms = reinterpret_cast<double*>(static_cast<char*>(ws) + 256);
    const int nb = int((m + kWideRows - 1) / kWideRows);
    const size_t lds = size_t(kWideRows) * A * sizeof(float);
    ProfScope ps(s, [&] { return "ppo_loss/" + cb_dims(int(m), A); });
    if (!ms_pre) {
        float* mo = static_cast<float*>(ws);
        if (rows)
            hipLaunchKernelGGL(adv_stats_ws_kernel<true>, dim3(1), dim3(kFusedThreads), 0, s, m, adv, rows, 0, 1, 0, mo);
        else
            hipLaunchKernelGGL(adv_stats_ws_kernel<false>, dim3(1), dim3(kFusedThreads), 0, s, m, adv, rows, 0, 1, 0, mo);
    }
#define CB_PR(AC, RW) \
    hipLaunchKernelGGL((ppo_rows_ws_kernel<AC, RW>), dim3(unsigned(nb)), dim3(kWideRows), lds, s, m, A, z, v, act, \
                       old_logp, adv, ret, rows, norm_adv, clip, vf, ent, dz, dv, ms, terms)
    if (rows) {
        if (A == 18) CB_PR(18, true); else if (A == 6) CB_PR(6, true); else CB_PR(0, true);
    } else {
        if (A == 18) CB_PR(18, false); else if (A == 6) CB_PR(6, false); else CB_PR(0, false);
    }
#undef CB_PR
    hipLaunchKernelGGL(loss_final_ws_kernel<true>, dim3(1), dim3(kFusedThreads), 0, s, m, 0.f, vf, ent, terms, ms,
                       stats);
    return hipGetLastError();
}

hipError_t impala_loss_ws(int64_t m, int A, const float* z, const float* v, const int32_t* act,
                          const float* vs, const float* pg, float pgc, float vf, float ent, float* dz,
                          float* dv, float* stats, void* ws, hipStream_t s) {
    if (m <= 0) return hipSuccess;
    if (m <= kWideRows)
        return impala_loss(m, A, z, v, act, vs, pg, pgc, vf, ent, dz, dv, stats, s);
    if (m > kFusedRows) {
        ProfScope ps(s, [&] { return "impala_loss/" + cb_dims(int(m), A); });
        return impala_loss_big(m, A, z, v, act, vs, pg, pgc, vf, ent, dz, dv, stats, ws, s);
    }
    float* ms = static_cast<float*>(ws);
    double* terms = reinterpret_cast<double*>(static_cast<char*>(ws) + 256);
    const int nb = int((m + kWideRows - 1) / kWideRows);
    const size_t lds = size_t(kWideRows) * A * sizeof(float);
    ProfScope ps(s, [&] { return "impala_loss/" + cb_dims(int(m), A); });
#define CB_IR(AC) \
    hipLaunchKernelGGL((impala_rows_ws_kernel<AC>), dim3(unsigned(nb)), dim3(kWideRows), lds, s, m, A, z, v, act, vs, \
                       pg, pgc, vf, ent, dz, dv, terms)
    if (A == 18) CB_IR(18); else if (A == 6) CB_IR(6); else CB_IR(0);
#undef CB_IR
    hipLaunchKernelGGL(loss_final_ws_kernel<false>, dim3(1), dim3(kFusedThreads), 0, s, m, pgc, vf, ent, terms, ms,
                       stats);
    return hipGetLastError();
}

// ---- log pi(a) per row (IMPALA target log-probs for V-trace)
__global__ void action_logp_kernel(int64_t m, int A, const float* __restrict__ z,
                                   const int32_t* __restrict__ act, float* __restrict__ logp) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i >= m) return;
    const float* zr = z + i * A;
    const RowLsm rs = row_log_softmax(zr, A);
    const int a = act[i];
    logp[i] = (a >= 0 && a < A) ? rs.l(zr[a]) : __builtin_nanf("");
}

hipError_t action_logp(int64_t m, int A, const float* z, const int32_t* act, float* logp,
                       hipStream_t s) {
    if (m <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "action_logp/" + cb_dims(int(m), A); });
    hipLaunchKernelGGL(action_logp_kernel, dim3(unsigned((m + 255) / 256)), dim3(256), 0, s, m, A, z,
                       act, logp);
    return hipGetLastError();
}

// ---- Gumbel-max sampling: a = argmax_j (z_j + g_j), ties to the lowest index
__global__ void gumbel_max_kernel(int64_t m, int A, const float* __restrict__ z,
                                  const float* __restrict__ g, int32_t* __restrict__ act,
                                  float* __restrict__ logp) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i >= m) return;
    const float* zr = z + i * A;
    const float* gr = g + i * A;
    int best = 0;
    float bv = zr[0] + gr[0];
    for (int j = 1; j < A; ++j) {
        const float v = zr[j] + gr[j];
        if (v > bv) { bv = v; best = j; }
    }
    const RowLsm rs = row_log_softmax(zr, A);
    act[i] = best;
    logp[i] = rs.l(zr[best]);
}

hipError_t gumbel_max(int64_t m, int A, const float* z, const float* g, int32_t* act, float* logp,
                      hipStream_t s) {
    if (m <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "gumbel_max/" + cb_dims(int(m), A); });
    hipLaunchKernelGGL(gumbel_max_kernel, dim3(unsigned((m + 255) / 256)), dim3(256), 0, s, m, A, z, g,
                       act, logp);
    return hipGetLastError();
}

}  // namespace cb
