// Reverse-time target scans over time-major [T, E] rollouts: GAE (PPO) and V-trace (IMPALA).
//
// Each recurrence is independent per env and sequential in t, so one lane owns one env.
// A block covers 64 envs; it walks the rollout backwards in chunks of TC steps. All 256
// threads stage a chunk of every input in LDS with coalesced row reads (64 consecutive
// envs = 256 contiguous bytes per row), one wave runs the recurrence out of LDS, and all
// threads write the chunk's outputs back coalesced. The recurrence state (carry, next
// value, next done flag) stays in registers across chunks.
#include "common.h"
#include "kernels.h"

namespace cb {

constexpr int kSE = 64;   // envs per block
constexpr int kTC = 32;   // time steps per chunk

__global__ __launch_bounds__(256) void gae_kernel(int T, int E, const float* __restrict__ r,
                                                  const float* __restrict__ v,
                                                  const uint8_t* __restrict__ d,
                                                  const float* __restrict__ nv,
                                                  const uint8_t* __restrict__ nd, float gamma,
                                                  float lam, float* __restrict__ adv,
                                                  float* __restrict__ ret) {
    __shared__ float sr[kTC][kSE], sv[kTC][kSE];
    __shared__ uint8_t sd[kTC][kSE];
    const int tid = threadIdx.x;
    const int e0 = blockIdx.x * kSE;
    const int le = tid & (kSE - 1);
    const int e = e0 + le;
    float carry = 0.f, v_next = 0.f, d_next = 0.f;
    if (tid < kSE && e < E) { v_next = nv[e]; d_next = float(nd[e]); }
    for (int t1 = T; t1 > 0; t1 -= kTC) {
        const int t0 = t1 - kTC > 0 ? t1 - kTC : 0;
        __syncthreads();
        for (int i = tid; i < (t1 - t0) * kSE; i += 256) {
            const int tt = i / kSE, ee = e0 + i % kSE;
            if (ee < E) {
                const int64_t o = int64_t(t0 + tt) * E + ee;
                sr[tt][i % kSE] = r[o]; sv[tt][i % kSE] = v[o]; sd[tt][i % kSE] = d[o];
            }
        }
        __syncthreads();
        if (tid < kSE && e < E) {
            for (int tt = t1 - t0 - 1; tt >= 0; --tt) {
                const float nonterm = 1.f - d_next;
                const float V = sv[tt][le];
                const float delta = sr[tt][le] + gamma * nonterm * v_next - V;
                carry = delta + gamma * lam * nonterm * carry;
                sr[tt][le] = carry;            // advantage
                sv[tt][le] = carry + V;        // return
                v_next = V;
                d_next = float(sd[tt][le]);
            }
        }
        __syncthreads();
        for (int i = tid; i < (t1 - t0) * kSE; i += 256) {
            const int tt = i / kSE, ee = e0 + i % kSE;
            if (ee < E) {
                const int64_t o = int64_t(t0 + tt) * E + ee;
                adv[o] = sr[tt][i % kSE]; ret[o] = sv[tt][i % kSE];
            }
        }
    }
}

__global__ __launch_bounds__(256) void vtrace_kernel(int T, int E, const float* __restrict__ mu,
                                                     const float* __restrict__ pi,
                                                     const float* __restrict__ r,
                                                     const float* __restrict__ v,
                                                     const uint8_t* __restrict__ d,
                                                     const float* __restrict__ bv,
                                                     const uint8_t* __restrict__ nd, float gamma,
                                                     float lam, float rho_bar, float c_bar,
                                                     float pg_rho_bar, float* __restrict__ vs,
                                                     float* __restrict__ pg) {
    __shared__ float sr[kTC][kSE], sv[kTC][kSE], slr[kTC][kSE];
    __shared__ uint8_t sd[kTC][kSE];
    const int tid = threadIdx.x;
    const int e0 = blockIdx.x * kSE;
    const int le = tid & (kSE - 1);
    const int e = e0 + le;
    float acc = 0.f, v_next = 0.f, vs_next = 0.f, d_next = 0.f;
    if (tid < kSE && e < E) { v_next = bv[e]; vs_next = bv[e]; d_next = float(nd[e]); }
    for (int t1 = T; t1 > 0; t1 -= kTC) {
        const int t0 = t1 - kTC > 0 ? t1 - kTC : 0;
        __syncthreads();
        for (int i = tid; i < (t1 - t0) * kSE; i += 256) {
            const int tt = i / kSE, ee = e0 + i % kSE;
            if (ee < E) {
                const int64_t o = int64_t(t0 + tt) * E + ee;
                sr[tt][i % kSE] = r[o]; sv[tt][i % kSE] = v[o]; sd[tt][i % kSE] = d[o];
                slr[tt][i % kSE] = pi[o] - mu[o];
            }
        }
        __syncthreads();
        if (tid < kSE && e < E) {
            for (int tt = t1 - t0 - 1; tt >= 0; --tt) {
                const float disc = gamma * (1.f - d_next);
                const float is = expf(slr[tt][le]);
                const float rho = fminf(rho_bar, is), c = lam * fminf(c_bar, is);
                const float V = sv[tt][le], R = sr[tt][le];
                const float delta = rho * (R + disc * v_next - V);
                acc = delta + disc * c * acc;
                const float vs_t = acc + V;
                const float q = R + disc * (lam * vs_next + (1.f - lam) * v_next);
                sr[tt][le] = vs_t;
                slr[tt][le] = fminf(pg_rho_bar, is) * (q - V);
                vs_next = vs_t;
                v_next = V;
                d_next = float(sd[tt][le]);
            }
        }
        __syncthreads();
        for (int i = tid; i < (t1 - t0) * kSE; i += 256) {
            const int tt = i / kSE, ee = e0 + i % kSE;
            if (ee < E) {
                const int64_t o = int64_t(t0 + tt) * E + ee;
                vs[o] = sr[tt][i % kSE]; pg[o] = slr[tt][i % kSE];
            }
        }
    }
}

hipError_t gae(int T, int E, const float* r, const float* v, const uint8_t* d, const float* nv,
               const uint8_t* nd, float gamma, float lam, float* adv, float* ret, hipStream_t s) {
    if (T <= 0 || E <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "gae/" + cb_dims(T, E); });
    hipLaunchKernelGGL(gae_kernel, dim3((E + kSE - 1) / kSE), dim3(256), 0, s, T, E, r, v, d, nv, nd,
                       gamma, lam, adv, ret);
    return hipGetLastError();
}

hipError_t vtrace(int T, int E, const float* mu, const float* pi, const float* r, const float* v,
                  const uint8_t* d, const float* bv, const uint8_t* nd, float gamma, float lam,
                  float rho_bar, float c_bar, float pg_rho_bar, float* vs, float* pg,
                  hipStream_t s) {
    if (T <= 0 || E <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "vtrace/" + cb_dims(T, E); });
    hipLaunchKernelGGL(vtrace_kernel, dim3((E + kSE - 1) / kSE), dim3(256), 0, s, T, E, mu, pi, r, v,
                       d, bv, nd, gamma, lam, rho_bar, c_bar, pg_rho_bar, vs, pg);
    return hipGetLastError();
}

// ---- IMPALA minibatch k: the env block [e0, e0 + Eb) over all T steps. rows[i] for
// i = t*Eb + e' is the rollout row t*E + e0 + e' (t = T: the bootstrap frames, rows T*E..);
// the block's actions, behaviour log-probs, rewards and dones are gathered to [T, Eb], and
// its next_done to [Eb].
__global__ __launch_bounds__(256) void env_block_gather_kernel(int T, int E, int e0, int Eb,
                                                               const int32_t* __restrict__ act,
                                                               const float* __restrict__ mu,
                                                               const float* __restrict__ r,
                                                               const uint8_t* __restrict__ d,
                                                               const uint8_t* __restrict__ nd,
                                                               EnvBlock b) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i >= int64_t(T + 1) * Eb) return;
    const int t = int(i / Eb), e = e0 + int(i - int64_t(t) * Eb);
    const int64_t src = int64_t(t) * E + e;
    b.rows[i] = int32_t(src);
    if (t < T) {
        b.act[i] = act[src];
        b.mu[i] = mu[src];
        b.r[i] = r[src];
        b.d[i] = d[src];
    } else {
        b.nd[i - int64_t(T) * Eb] = nd[e];
    }
}

hipError_t env_block_gather(int T, int E, int e0, int Eb, const int32_t* act, const float* mu, const float* r,
                            const uint8_t* d, const uint8_t* nd, const EnvBlock& b, hipStream_t s) {
    const int64_t n = int64_t(T + 1) * Eb;
    if (n <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "env_block_gather/" + cb_dims(T, Eb); });
    hipLaunchKernelGGL(env_block_gather_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, T, E, e0, Eb, act,
                       mu, r, d, nd, b);
    return hipGetLastError();
}

}  // namespace cb
