// C-ABI of the learner-update library: argument validation on the host (before any HIP
// call), workspace planning, and the learning-phase orchestration of Algorithm 1.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/cleanba_layers.h"
#include "../../include/cleanba_learner.h"
#include "../../include/cleanba_profile.h"
#include "kernels.h"
#include "plan.h"

using namespace cb;

namespace {

thread_local std::string g_err;

impala_status_t fail(impala_status_t code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

impala_status_t ok() {
    g_err.clear();
    return IMPALA_OK;
}

impala_status_t hip_status(hipError_t e, const char* where) {
    if (e == hipSuccess) return ok();
    return fail(IMPALA_EHIP, "%s: %s", where, hipGetErrorString(e));
}

#define CHECK_PTR(p) \
    if (!(p)) return fail(IMPALA_EINVAL, "%s: argument '%s' is NULL", __func__, #p)

bool valid_prec(int p) { return p == IMPALA_PREC_BF16 || p == IMPALA_PREC_FP32; }

// Learner workspace layout (bytes from the start of ws).
struct LearnerLayout {
    NetPlan plan;
    size_t cnn, adv, ret, tlogp, logits, value, dlogits, dvalue, grads, apart;
    size_t rows, gact, gmu, grew, gdone, gnd;   // IMPALA minibatch gathers (more than one)
    size_t lossws;                               // the loss kernels' statistics and row terms
    size_t advms;                                // PPO: every update's advantage mean / std
    size_t total;
    int64_t fwd_rows, mb;
};

size_t a256(size_t x) { return (x + 255) / 256 * 256; }

std::string check_cfg(const learner_cfg_t* c) {
    if (!c) return "cfg is NULL";
    if (c->algo != LEARNER_PPO && c->algo != LEARNER_IMPALA) return "cfg.algo must be PPO or IMPALA";
    if (!valid_prec(c->prec)) return "cfg.prec must be BF16 or FP32";
    if (c->T < 1 || c->E < 1) return "cfg.T and cfg.E must be >= 1";
    if (int64_t(c->T) * c->E > (int64_t(1) << 26)) return "cfg.T * cfg.E too large";
    if (c->algo == LEARNER_PPO) {
        if (c->update_epochs < 1 || c->num_minibatches < 1 || c->minibatch_size < 1)
            return "PPO needs update_epochs, num_minibatches, minibatch_size >= 1";
        if (int64_t(c->num_minibatches) * c->minibatch_size > int64_t(c->T) * c->E)
            return "num_minibatches * minibatch_size exceeds T * E";
    } else {
        if (c->num_minibatches < 1 || c->E % c->num_minibatches)
            return "IMPALA needs num_minibatches >= 1 dividing E (minibatches are env blocks)";
    }
    if (c->optimizer != LEARNER_OPT_ADAM && c->optimizer != LEARNER_OPT_RMSPROP)
        return "cfg.optimizer must be ADAM or RMSPROP";
    if (!(c->lr >= 0.f)) return "cfg.lr must be >= 0";
    if (c->optimizer == LEARNER_OPT_ADAM &&
        (!(c->adam_eps >= 0.f) || !(c->beta1 >= 0.f && c->beta1 < 1.f) || !(c->beta2 >= 0.f && c->beta2 < 1.f)))
        return "cfg Adam hyperparameters out of range";
    if (c->optimizer == LEARNER_OPT_RMSPROP && (!(c->rms_eps >= 0.f) || !(c->rms_decay >= 0.f && c->rms_decay < 1.f)))
        return "cfg RMSprop hyperparameters out of range";
    return "";
}

LearnerLayout learner_layout(const impala_net_t& net, const learner_cfg_t& c) {
    LearnerLayout L;
    const int64_t TE = int64_t(c.T) * c.E;
    const int A = net.num_actions;
    const int nmb = c.algo == LEARNER_PPO ? 1 : c.num_minibatches;
    const int64_t Eb = c.E / nmb;   // IMPALA: envs per minibatch
    L.mb = c.algo == LEARNER_PPO ? c.minibatch_size : int64_t(c.T) * Eb;
    L.fwd_rows = c.algo == LEARNER_PPO ? c.minibatch_size : int64_t(c.T) * Eb + Eb;
    L.plan = make_plan(net, c.prec, L.fwd_rows, 1);
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t o = off; off += a256(bytes); return o; };
    L.cnn = take(L.plan.total);
    L.adv = take(TE * sizeof(float));
    L.ret = take(TE * sizeof(float));
    L.tlogp = take(TE * sizeof(float));
    L.logits = take(size_t(L.fwd_rows) * A * sizeof(float));
    L.value = take(size_t(L.fwd_rows) * sizeof(float));
    L.dlogits = take(size_t(L.mb) * A * sizeof(float));
    L.dvalue = take(size_t(L.mb) * sizeof(float));
    L.grads = take(size_t(L.plan.po.total) * sizeof(float));
    L.apart = take(adam_partial_floats(L.plan.po.total) * sizeof(float));
    const bool gather = c.algo == LEARNER_IMPALA && nmb > 1;
    L.rows = take(gather ? size_t(L.fwd_rows) * sizeof(int32_t) : 0);
    L.gact = take(gather ? size_t(L.mb) * sizeof(int32_t) : 0);
    L.gmu = take(gather ? size_t(L.mb) * sizeof(float) : 0);
    L.grew = take(gather ? size_t(L.mb) * sizeof(float) : 0);
    L.gdone = take(gather ? size_t(L.mb) : 0);
    L.gnd = take(gather ? size_t(Eb) : 0);
    L.lossws = take(loss_ws_bytes(L.mb));
    L.advms = take(c.algo == LEARNER_PPO ? size_t(2) * c.update_epochs * c.num_minibatches * sizeof(float) : 0);
    L.total = off;
    return L;
}

}  // namespace

namespace cb {

__global__ void fill_zero_kernel(float* p, int64_t n) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

size_t lds_limit() {
    static thread_local int dev_cached = -1;
    static thread_local size_t bytes = 64 * 1024;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 64 * 1024;
    if (dev != dev_cached) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && v > 0)
            bytes = size_t(v);
        dev_cached = dev;
    }
    return bytes;
}

int resident_blocks(const void* fn, int threads, size_t lds) {
    struct Entry { int dev; const void* fn; int threads; size_t lds; int blocks; };
    static std::mutex mu;
    static std::vector<Entry> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    std::lock_guard<std::mutex> lock(mu);
    for (const Entry& e : cache)
        if (e.dev == dev && e.fn == fn && e.threads == threads && e.lds == lds) return e.blocks;
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds) != hipSuccess || per_cu < 1)
        per_cu = 1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 1;
    (void)hipGetLastError();   // a failed query must not be reported by the next launch
    cache.push_back(Entry{dev, fn, threads, lds, per_cu * cus});
    return per_cu * cus;
}

hipError_t fill_zero(float* p, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    ProfScope ps(s, [&] { return "fill_zero/" + std::to_string(n); });
    hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace cb

extern "C" {

const char* impala_last_error(void) { return g_err.c_str(); }

int64_t impala_param_count(const impala_net_t* net) {
    const std::string e = check_net(net);
    if (!e.empty()) { fail(IMPALA_EINVAL, "impala_param_count: %s", e.c_str()); return -1; }
    ok();
    return param_offsets(*net).total;
}

int impala_param_layout(const impala_net_t* net, impala_tensor_desc_t* out, int cap) {
    const std::string e = check_net(net);
    if (!e.empty()) return fail(IMPALA_EINVAL, "impala_param_layout: %s", e.c_str());
    if (!out && cap > 0) return fail(IMPALA_EINVAL, "impala_param_layout: out is NULL");
    const ParamOffsets po = param_offsets(*net);
    int k = 0;
    auto put = [&](const char* name, int64_t off, int nd, int s0, int s1, int s2, int s3) {
        if (k < cap) {
            impala_tensor_desc_t& d = out[k];
            std::memset(&d, 0, sizeof(d));
            std::snprintf(d.name, sizeof(d.name), "%s", name);
            d.offset = off; d.ndim = nd;
            d.shape[0] = s0; d.shape[1] = s1; d.shape[2] = s2; d.shape[3] = s3;
        }
        ++k;
    };
    int cin = net->in_c;
    char nm[32];
    for (int s = 0; s < 3; ++s) {
        const int c = net->ch[s];
        std::snprintf(nm, sizeof(nm), "s%d.conv.w", s); put(nm, po.conv_w[s][0], 4, 3, 3, cin, c);
        std::snprintf(nm, sizeof(nm), "s%d.conv.b", s); put(nm, po.conv_b[s][0], 1, c, 0, 0, 0);
        for (int r = 0; r < 2; ++r)
            for (int q = 0; q < 2; ++q) {
                std::snprintf(nm, sizeof(nm), "s%d.res%d.conv%d.w", s, r, q);
                put(nm, po.conv_w[s][1 + 2 * r + q], 4, 3, 3, c, c);
                std::snprintf(nm, sizeof(nm), "s%d.res%d.conv%d.b", s, r, q);
                put(nm, po.conv_b[s][1 + 2 * r + q], 1, c, 0, 0, 0);
            }
        cin = c;
    }
    const int flat = int((po.dense_b - po.dense_w) / net->hidden);
    put("dense.w", po.dense_w, 2, flat, net->hidden, 0, 0);
    put("dense.b", po.dense_b, 1, net->hidden, 0, 0, 0);
    put("logits.w", po.logits_w, 2, net->hidden, net->num_actions, 0, 0);
    put("logits.b", po.logits_b, 1, net->num_actions, 0, 0, 0);
    put("value.w", po.value_w, 2, net->hidden, 1, 0, 0);
    put("value.b", po.value_b, 1, 1, 0, 0, 0);
    ok();
    return k;
}

int impala_activation_layout(const impala_net_t* net, impala_prec_t prec, int64_t n_frames,
                             impala_activation_desc_t* out, int cap) {
    const std::string e = check_net(net);
    if (!e.empty()) return fail(IMPALA_EINVAL, "impala_activation_layout: %s", e.c_str());
    if (!valid_prec(prec)) return fail(IMPALA_EINVAL, "impala_activation_layout: bad prec %d", int(prec));
    if (n_frames < 1 || n_frames > (int64_t(1) << 24))
        return fail(IMPALA_EINVAL, "impala_activation_layout: n_frames out of range");
    if (!out && cap > 0) return fail(IMPALA_EINVAL, "impala_activation_layout: out is NULL");
    const NetPlan p = make_plan(*net, prec, n_frames, 1);
    const int act = prec == IMPALA_PREC_BF16 ? IMPALA_DT_BF16 : IMPALA_DT_F32;
    int k = 0;
    auto put = [&](const char* name, size_t off, int dtype, int es, int64_t s1, int64_t s2, int64_t s3) {
        if (k < cap) {
            impala_activation_desc_t& d = out[k];
            std::memset(&d, 0, sizeof(d));
            std::snprintf(d.name, sizeof(d.name), "%s", name);
            d.offset = int64_t(off);
            d.dtype = dtype;
            d.ndim = s3 > 0 ? 4 : 2;
            d.shape[0] = n_frames; d.shape[1] = s1; d.shape[2] = s3 > 0 ? s2 : 0; d.shape[3] = s3;
            d.bytes = n_frames * s1 * (s3 > 0 ? s2 * s3 : 1) * es;
        }
        ++k;
    };
    char nm[32];
    for (int s = 0; s < 3; ++s) {
        const int C = p.C[s + 1], OH = p.H[s + 1], OW = p.W[s + 1];
        if (prec == IMPALA_PREC_FP32) {
            std::snprintf(nm, sizeof(nm), "s%d.conv", s);
            put(nm, p.c[s], act, p.es, p.H[s], p.W[s], C);
        }
        std::snprintf(nm, sizeof(nm), "s%d.arg", s);
        put(nm, p.idx[s], IMPALA_DT_U8, 1, OH, OW, C);
        for (int r = 0; r < 3; ++r) {
            std::snprintf(nm, sizeof(nm), "s%d.x%d", s, r);
            put(nm, p.x[s][r], act, p.es, OH, OW, C);
        }
        for (int r = 0; r < 2; ++r) {
            std::snprintf(nm, sizeof(nm), "s%d.t%d", s, r);
            put(nm, p.t[s][r], act, p.es, OH, OW, C);
        }
    }
    put("h", p.h, act, p.es, p.hidden, 0, 0);
    ok();
    return k;
}

size_t impala_workspace_bytes(const impala_net_t* net, int64_t n_frames, impala_prec_t prec,
                              int training) {
    const std::string e = check_net(net);
    if (!e.empty()) { fail(IMPALA_EINVAL, "impala_workspace_bytes: %s", e.c_str()); return 0; }
    if (!valid_prec(prec) || n_frames < 0) { fail(IMPALA_EINVAL, "impala_workspace_bytes: bad prec or n"); return 0; }
    ok();
    return make_plan(*net, prec, n_frames > 0 ? n_frames : 1, training ? 1 : 0).total;
}

impala_status_t impala_cnn_fwd(const impala_net_t* net, impala_prec_t prec, const float* params,
                               const uint8_t* obs, const int32_t* row_idx, int64_t n, void* ws,
                               size_t ws_bytes, int training, float* logits, float* value,
                               hipStream_t stream) {
    const std::string e = check_net(net);
    if (!e.empty()) return fail(IMPALA_EINVAL, "impala_cnn_fwd: %s", e.c_str());
    if (!valid_prec(prec)) return fail(IMPALA_EINVAL, "impala_cnn_fwd: bad prec %d", int(prec));
    if (n < 0 || n > (int64_t(1) << 24)) return fail(IMPALA_EINVAL, "impala_cnn_fwd: n out of range");
    if (n == 0) return ok();
    CHECK_PTR(params); CHECK_PTR(obs); CHECK_PTR(ws); CHECK_PTR(logits); CHECK_PTR(value);
    const NetPlan p = make_plan(*net, prec, n, training ? 1 : 0);
    if (ws_bytes < p.total)
        return fail(IMPALA_EWORKSPACE, "impala_cnn_fwd: workspace %zu < %zu bytes", ws_bytes, p.total);
    return hip_status(run_forward(p, params, obs, row_idx, n, static_cast<char*>(ws), logits, value, stream),
                      "impala_cnn_fwd");
}

impala_status_t impala_cnn_bwd(const impala_net_t* net, impala_prec_t prec, const float* params,
                               const uint8_t* obs, const int32_t* row_idx, int64_t n, void* ws,
                               size_t ws_bytes, const float* dlogits, const float* dvalue,
                               float* grads, hipStream_t stream) {
    const std::string e = check_net(net);
    if (!e.empty()) return fail(IMPALA_EINVAL, "impala_cnn_bwd: %s", e.c_str());
    if (!valid_prec(prec)) return fail(IMPALA_EINVAL, "impala_cnn_bwd: bad prec %d", int(prec));
    if (n < 0 || n > (int64_t(1) << 24)) return fail(IMPALA_EINVAL, "impala_cnn_bwd: n out of range");
    CHECK_PTR(params); CHECK_PTR(grads);
    const NetPlan p = make_plan(*net, prec, n > 0 ? n : 1, 1);
    if (n == 0) return hip_status(fill_zero(grads, p.po.total, stream), "impala_cnn_bwd");
    CHECK_PTR(obs); CHECK_PTR(ws); CHECK_PTR(dlogits); CHECK_PTR(dvalue);
    if (ws_bytes < p.total)
        return fail(IMPALA_EWORKSPACE, "impala_cnn_bwd: workspace %zu < %zu bytes", ws_bytes, p.total);
    return hip_status(run_backward(p, params, obs, row_idx, n, static_cast<char*>(ws), dlogits, dvalue,
                                   grads, stream),
                      "impala_cnn_bwd");
}

impala_status_t gae_advantages(int32_t T, int32_t E, const float* rewards, const float* values,
                               const uint8_t* dones, const float* next_value,
                               const uint8_t* next_done, float gamma, float lambda, float* adv,
                               float* ret, hipStream_t stream) {
    if (T < 0 || E < 0) return fail(IMPALA_EINVAL, "gae_advantages: T and E must be >= 0");
    if (T == 0 || E == 0) return ok();
    CHECK_PTR(rewards); CHECK_PTR(values); CHECK_PTR(dones); CHECK_PTR(next_value);
    CHECK_PTR(next_done); CHECK_PTR(adv); CHECK_PTR(ret);
    return hip_status(gae(T, E, rewards, values, dones, next_value, next_done, gamma, lambda, adv, ret, stream),
                      "gae_advantages");
}

impala_status_t vtrace_targets(int32_t T, int32_t E, const float* behav_logp,
                               const float* target_logp, const float* rewards, const float* values,
                               const uint8_t* dones, const float* bootstrap_value,
                               const uint8_t* next_done, float gamma, float lambda, float rho_bar,
                               float c_bar, float pg_rho_bar, float* vs, float* pg_adv,
                               hipStream_t stream) {
    if (T < 0 || E < 0) return fail(IMPALA_EINVAL, "vtrace_targets: T and E must be >= 0");
    if (T == 0 || E == 0) return ok();
    CHECK_PTR(behav_logp); CHECK_PTR(target_logp); CHECK_PTR(rewards); CHECK_PTR(values);
    CHECK_PTR(dones); CHECK_PTR(bootstrap_value); CHECK_PTR(next_done); CHECK_PTR(vs); CHECK_PTR(pg_adv);
    return hip_status(vtrace(T, E, behav_logp, target_logp, rewards, values, dones, bootstrap_value,
                             next_done, gamma, lambda, rho_bar, c_bar, pg_rho_bar, vs, pg_adv, stream),
                      "vtrace_targets");
}

size_t loss_workspace_bytes(int64_t m) { return loss_ws_bytes(m > 0 ? m : 1); }

impala_status_t ppo_loss_grad(int64_t m, int32_t A, const float* logits, const float* value,
                              const int32_t* actions, const float* old_logp, const float* adv,
                              const float* ret, int32_t norm_adv, float clip_eps, float vf_coef,
                              float ent_coef, float* dlogits, float* dvalue, float* stats, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
    if (m < 1 || m > (int64_t(1) << 26)) return fail(IMPALA_EINVAL, "ppo_loss_grad: m out of range");
    if (A < 1 || A > 64) return fail(IMPALA_EINVAL, "ppo_loss_grad: A must be in [1, 64]");
    CHECK_PTR(logits); CHECK_PTR(value); CHECK_PTR(actions); CHECK_PTR(old_logp); CHECK_PTR(adv);
    CHECK_PTR(ret); CHECK_PTR(dlogits); CHECK_PTR(dvalue); CHECK_PTR(stats);
    if (ws && ws_bytes < loss_ws_bytes(m))
        return fail(IMPALA_EWORKSPACE, "ppo_loss_grad: workspace %zu < %zu bytes", ws_bytes, loss_ws_bytes(m));
    const hipError_t e = ws ? ppo_loss_ws(m, A, logits, value, actions, old_logp, adv, ret, nullptr, norm_adv,
                                          clip_eps, vf_coef, ent_coef, dlogits, dvalue, stats, ws, stream)
                            : ppo_loss(m, A, logits, value, actions, old_logp, adv, ret, nullptr, norm_adv,
                                       clip_eps, vf_coef, ent_coef, dlogits, dvalue, stats, stream);
    return hip_status(e, "ppo_loss_grad");
}

impala_status_t impala_loss_grad(int64_t m, int32_t A, const float* logits, const float* value,
                                 const int32_t* actions, const float* vs, const float* pg_adv,
                                 float pg_coef, float vf_coef, float ent_coef, float* dlogits,
                                 float* dvalue, float* stats, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (m < 1 || m > (int64_t(1) << 26)) return fail(IMPALA_EINVAL, "impala_loss_grad: m out of range");
    if (A < 1 || A > 64) return fail(IMPALA_EINVAL, "impala_loss_grad: A must be in [1, 64]");
    CHECK_PTR(logits); CHECK_PTR(value); CHECK_PTR(actions); CHECK_PTR(vs); CHECK_PTR(pg_adv);
    CHECK_PTR(dlogits); CHECK_PTR(dvalue); CHECK_PTR(stats);
    if (ws && ws_bytes < loss_ws_bytes(m))
        return fail(IMPALA_EWORKSPACE, "impala_loss_grad: workspace %zu < %zu bytes", ws_bytes, loss_ws_bytes(m));
    const hipError_t e = ws ? impala_loss_ws(m, A, logits, value, actions, vs, pg_adv, pg_coef, vf_coef, ent_coef,
                                             dlogits, dvalue, stats, ws, stream)
                            : impala_loss(m, A, logits, value, actions, vs, pg_adv, pg_coef, vf_coef, ent_coef,
                                          dlogits, dvalue, stats, stream);
    return hip_status(e, "impala_loss_grad");
}

namespace {
// Adam's constants from the caller's float betas: 1 - beta and the bias corrections
// 1 - beta^t formed in double (in float, 1 - beta would lose the low bits of beta: for
// 0.999f about 1e-5 relative).
OptArgs adam_args(int64_t n, float* p, const float* g, float* m, float* v, int32_t step, float lr, float b1,
                  float b2, float eps, float max_norm) {
    OptArgs a{};
    a.n = n; a.p = p; a.g = g; a.m = m; a.v = v;
    a.lr = lr; a.b1 = b1; a.b2 = b2; a.eps = eps; a.max_norm = max_norm;
    a.omb1 = float(1.0 - double(b1));
    a.omb2 = float(1.0 - double(b2));
    a.bc1 = float(1.0 - std::pow(double(b1), double(step)));
    a.bc2 = float(1.0 - std::pow(double(b2), double(step)));
    return a;
}

// RMSprop's: decay in b2, 1 - decay (formed in double) in omb2.
OptArgs rmsprop_args(int64_t n, float* p, const float* g, float* nu, float lr, float decay, float eps,
                     float max_norm) {
    OptArgs a{};
    a.n = n; a.p = p; a.g = g; a.m = nullptr; a.v = nu;
    a.lr = lr; a.b2 = decay; a.omb2 = float(1.0 - double(decay)); a.eps = eps; a.max_norm = max_norm;
    return a;
}
}  // namespace

size_t adam_workspace_bytes(int64_t n_params) {
    return adam_partial_floats(n_params > 0 ? n_params : 1) * sizeof(float);
}

impala_status_t adam_step(int64_t n_params, float* params, const float* grads, float* m, float* v,
                          int32_t step, float lr, float beta1, float beta2, float eps,
                          float max_grad_norm, float* stats, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    if (n_params < 0) return fail(IMPALA_EINVAL, "adam_step: n_params < 0");
    if (step < 1) return fail(IMPALA_EINVAL, "adam_step: step is 1-based");
    if (!(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f))
        return fail(IMPALA_EINVAL, "adam_step: betas must be in [0, 1)");
    if (n_params == 0) return ok();
    CHECK_PTR(params); CHECK_PTR(grads); CHECK_PTR(m); CHECK_PTR(v); CHECK_PTR(ws);
    const size_t need = adam_workspace_bytes(n_params);
    if (ws_bytes < need) return fail(IMPALA_EWORKSPACE, "adam_step: workspace %zu < %zu bytes", ws_bytes, need);
    const OptArgs a = adam_args(n_params, params, grads, m, v, step, lr, beta1, beta2, eps, max_grad_norm);
    return hip_status(clip_opt_step(OPT_ADAM, a, stats, static_cast<float*>(ws), stream), "adam_step");
}

impala_status_t adam_step_noalloc(int64_t n_params, float* params, const float* grads, float* m, float* v,
                                  int32_t step, float lr, float beta1, float beta2, float eps,
                                  float max_grad_norm, float* stats, hipStream_t stream) {
    if (n_params < 0) return fail(IMPALA_EINVAL, "adam_step_noalloc: n_params < 0");
    if (step < 1) return fail(IMPALA_EINVAL, "adam_step_noalloc: step is 1-based");
    if (!(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f))
        return fail(IMPALA_EINVAL, "adam_step_noalloc: betas must be in [0, 1)");
    if (n_params == 0) return ok();
    CHECK_PTR(params); CHECK_PTR(grads); CHECK_PTR(m); CHECK_PTR(v);
    const size_t need = adam_workspace_bytes(n_params);
    if (need > noalloc_scratch_bytes())
        return fail(IMPALA_EINVAL, "adam_step_noalloc: needs %zu bytes of scratch, the built-in buffer holds %zu",
                    need, noalloc_scratch_bytes());
    float* part = nullptr;
    const hipError_t e = noalloc_scratch(&part);
    if (e != hipSuccess) return hip_status(e, "adam_step_noalloc: scratch address");
    const OptArgs a = adam_args(n_params, params, grads, m, v, step, lr, beta1, beta2, eps, max_grad_norm);
    return hip_status(clip_opt_step(OPT_ADAM, a, stats, part, stream), "adam_step_noalloc");
}

size_t rmsprop_workspace_bytes(int64_t n_params) { return adam_workspace_bytes(n_params); }

impala_status_t rmsprop_step(int64_t n_params, float* params, const float* grads, float* nu, float lr,
                             float decay, float eps, float max_grad_norm, float* stats, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
    if (n_params < 0) return fail(IMPALA_EINVAL, "rmsprop_step: n_params < 0");
    if (!(decay >= 0.f && decay < 1.f)) return fail(IMPALA_EINVAL, "rmsprop_step: decay must be in [0, 1)");
    if (!(eps >= 0.f)) return fail(IMPALA_EINVAL, "rmsprop_step: eps must be >= 0");
    if (n_params == 0) return ok();
    CHECK_PTR(params); CHECK_PTR(grads); CHECK_PTR(nu); CHECK_PTR(ws);
    const size_t need = rmsprop_workspace_bytes(n_params);
    if (ws_bytes < need) return fail(IMPALA_EWORKSPACE, "rmsprop_step: workspace %zu < %zu bytes", ws_bytes, need);
    const OptArgs a = rmsprop_args(n_params, params, grads, nu, lr, decay, eps, max_grad_norm);
    return hip_status(clip_opt_step(OPT_RMSPROP, a, stats, static_cast<float*>(ws), stream), "rmsprop_step");
}

size_t learner_workspace_bytes(const impala_net_t* net, const learner_cfg_t* cfg) {
    std::string e = check_net(net);
    if (e.empty()) e = check_cfg(cfg);
    if (!e.empty()) { fail(IMPALA_EINVAL, "learner_workspace_bytes: %s", e.c_str()); return 0; }
    ok();
    return learner_layout(*net, *cfg).total;
}

impala_status_t learner_step(const impala_net_t* net, const learner_cfg_t* cfg,
                             const rollout_t* ro, float* params, float* m, float* v,
                             int32_t* step, const int32_t* perm, void* ws, size_t ws_bytes,
                             float* stats, hipStream_t stream) {
    std::string e = check_net(net);
    if (e.empty()) e = check_cfg(cfg);
    if (!e.empty()) return fail(IMPALA_EINVAL, "learner_step: %s", e.c_str());
    CHECK_PTR(ro); CHECK_PTR(params); CHECK_PTR(v); CHECK_PTR(step); CHECK_PTR(ws);
    CHECK_PTR(stats);
    if (cfg->optimizer == LEARNER_OPT_ADAM) CHECK_PTR(m);
    CHECK_PTR(ro->obs); CHECK_PTR(ro->actions); CHECK_PTR(ro->behav_logp); CHECK_PTR(ro->rewards);
    CHECK_PTR(ro->dones); CHECK_PTR(ro->next_done);
    if (*step < 0) return fail(IMPALA_EINVAL, "learner_step: *step must be >= 0");
    const learner_cfg_t& c = *cfg;
    if (c.algo == LEARNER_PPO) {
        CHECK_PTR(ro->values); CHECK_PTR(ro->next_value); CHECK_PTR(perm);
    }
    const LearnerLayout L = learner_layout(*net, c);
    if (ws_bytes < L.total)
        return fail(IMPALA_EWORKSPACE, "learner_step: workspace %zu < %zu bytes", ws_bytes, L.total);
    char* w = static_cast<char*>(ws);
    const NetPlan& P = L.plan;
    const int A = net->num_actions;
    const int64_t TE = int64_t(c.T) * c.E;
    float* grads = reinterpret_cast<float*>(w + L.grads);
    float* apart = reinterpret_cast<float*>(w + L.apart);
    float* logits = reinterpret_cast<float*>(w + L.logits);
    float* value = reinterpret_cast<float*>(w + L.value);
    float* dlogits = reinterpret_cast<float*>(w + L.dlogits);
    float* dvalue = reinterpret_cast<float*>(w + L.dvalue);
    char* cnn = w + L.cnn;
    hipError_t he;
#define LS_TRY(x, what) \
    if ((he = (x)) != hipSuccess) return hip_status(he, what)
    // clip, then the configured optimiser (Adam: m, v; RMSprop: v holds nu), at step *step
    // bf16: the optimiser also writes the bf16 copy of the updated dense weights that the next
    // forward's dense GEMMs read (the rounding the forward's own cast applies), so only the
    // first forward of the call casts them
    bool dense_ready = false;
    auto opt_step = [&](float* st) {
        OptArgs oa = c.optimizer == LEARNER_OPT_ADAM
                         ? adam_args(P.po.total, params, grads, m, v, *step, c.lr, c.beta1, c.beta2, c.adam_eps,
                                     c.max_grad_norm)
                         : rmsprop_args(P.po.total, params, grads, v, c.lr, c.rms_decay, c.rms_eps, c.max_grad_norm);
        if (P.prec == BF16) {
            oa.mir = reinterpret_cast<uint16_t*>(cnn + P.wdb);
            oa.mir_off = P.po.dense_w;
            oa.mir_len = int64_t(P.flat) * P.hidden;
        }
        const hipError_t e = clip_opt_step(c.optimizer == LEARNER_OPT_ADAM ? OPT_ADAM : OPT_RMSPROP, oa, st, apart,
                                           stream);
        dense_ready = e == hipSuccess && P.prec == BF16;
        return e;
    };

    if (c.algo == LEARNER_PPO) {
        float* adv = reinterpret_cast<float*>(w + L.adv);
        float* ret = reinterpret_cast<float*>(w + L.ret);
        LS_TRY(gae(c.T, c.E, ro->rewards, ro->values, ro->dones, ro->next_value, ro->next_done, c.gamma,
                   c.lambda, adv, ret, stream), "learner_step: gae");
        // the advantages are fixed for the whole phase: every update's minibatch statistics in
        // one launch (update u = j * num_minibatches + k reads rows perm + j * T * E + k * minibatch_size)
        float* advms = reinterpret_cast<float*>(w + L.advms);
        const bool pre = ppo_adv_stats_batched(c.minibatch_size);
        if (pre)
            LS_TRY(ppo_adv_stats(c.minibatch_size, c.update_epochs * c.num_minibatches, adv, perm, c.minibatch_size,
                                 c.num_minibatches, TE, advms, stream),
                   "learner_step: advantage statistics");
        int u = 0;
        for (int j = 0; j < c.update_epochs; ++j) {
            for (int k = 0; k < c.num_minibatches; ++k, ++u) {
                const int32_t* rows = perm + int64_t(j) * TE + int64_t(k) * c.minibatch_size;
                const int64_t mb = c.minibatch_size;
                LS_TRY(run_forward(P, params, ro->obs, rows, mb, cnn, logits, value, stream, dense_ready),
                       "learner_step: forward");
                LS_TRY(ppo_loss_ws(mb, A, logits, value, ro->actions, ro->behav_logp, adv, ret, rows,
                                   c.norm_adv, c.clip_eps, c.vf_coef, c.ent_coef, dlogits, dvalue,
                                   stats + 8 * u, w + L.lossws, stream, pre ? advms + 2 * u : nullptr),
                       "learner_step: ppo loss");
                LS_TRY(run_backward(P, params, ro->obs, rows, mb, cnn, dlogits, dvalue, grads, stream),
                       "learner_step: backward");
                *step += 1;
                LS_TRY(opt_step(stats + 8 * u + 6), "learner_step: optimiser");
            }
        }
    } else {
        // minibatch k: the env block [k*Eb, (k+1)*Eb) over all T steps plus its bootstrap frames
        float* tlogp = reinterpret_cast<float*>(w + L.tlogp);
        float* vs = reinterpret_cast<float*>(w + L.adv);
        float* pg = reinterpret_cast<float*>(w + L.ret);
        const int nmb = c.num_minibatches, Eb = c.E / nmb;
        const int64_t n = int64_t(c.T) * Eb, n1 = n + Eb;
        for (int k = 0; k < nmb; ++k) {
            const int32_t* rows = nullptr;
            const int32_t* act = ro->actions;
            const float* mu = ro->behav_logp;
            const float* rw = ro->rewards;
            const uint8_t* dn = ro->dones;
            const uint8_t* nd = ro->next_done;
            if (nmb > 1) {
                EnvBlock b{reinterpret_cast<int32_t*>(w + L.rows), reinterpret_cast<int32_t*>(w + L.gact),
                           reinterpret_cast<float*>(w + L.gmu), reinterpret_cast<float*>(w + L.grew),
                           reinterpret_cast<uint8_t*>(w + L.gdone), reinterpret_cast<uint8_t*>(w + L.gnd)};
                LS_TRY(env_block_gather(c.T, c.E, k * Eb, Eb, ro->actions, ro->behav_logp, ro->rewards, ro->dones,
                                        ro->next_done, b, stream), "learner_step: minibatch gather");
                rows = b.rows; act = b.act; mu = b.mu; rw = b.r; dn = b.d; nd = b.nd;
            }
            LS_TRY(run_forward(P, params, ro->obs, rows, n1, cnn, logits, value, stream, dense_ready),
                   "learner_step: forward");
            LS_TRY(action_logp(n, A, logits, act, tlogp, stream), "learner_step: logp");
            LS_TRY(vtrace(c.T, Eb, mu, tlogp, rw, value, dn, value + n, nd, c.gamma, c.lambda, c.rho_bar, c.c_bar,
                          c.pg_rho_bar, vs, pg, stream),
                   "learner_step: vtrace");
            LS_TRY(impala_loss_ws(n, A, logits, value, act, vs, pg, c.pg_coef, c.vf_coef, c.ent_coef, dlogits,
                                  dvalue, stats + 8 * k, w + L.lossws, stream),
                   "learner_step: impala loss");
            LS_TRY(run_backward(P, params, ro->obs, rows, n, cnn, dlogits, dvalue, grads, stream),
                   "learner_step: backward");
            *step += 1;
            LS_TRY(opt_step(stats + 8 * k + 6), "learner_step: optimiser");
        }
    }
#undef LS_TRY
    return ok();
}

impala_status_t impala_actor_step(const impala_net_t* net, impala_prec_t prec, const float* params,
                                  const uint8_t* obs, int64_t n, const float* gumbel, void* ws,
                                  size_t ws_bytes, int32_t* actions, float* logp, float* value,
                                  float* logits, hipStream_t stream) {
    const std::string e = check_net(net);
    if (!e.empty()) return fail(IMPALA_EINVAL, "impala_actor_step: %s", e.c_str());
    if (!valid_prec(prec)) return fail(IMPALA_EINVAL, "impala_actor_step: bad prec");
    if (n < 0 || n > (int64_t(1) << 24)) return fail(IMPALA_EINVAL, "impala_actor_step: n out of range");
    if (n == 0) return ok();
    CHECK_PTR(params); CHECK_PTR(obs); CHECK_PTR(gumbel); CHECK_PTR(ws); CHECK_PTR(actions);
    CHECK_PTR(logp); CHECK_PTR(value);
    const NetPlan p = make_plan(*net, prec, n, 0);
    const size_t extra = logits ? 0 : a256(size_t(n) * net->num_actions * sizeof(float));
    if (ws_bytes < p.total + extra)
        return fail(IMPALA_EWORKSPACE, "impala_actor_step: workspace %zu < %zu bytes (add n*A*4 when logits is NULL)",
                    ws_bytes, p.total + extra);
    float* z = logits ? logits : reinterpret_cast<float*>(static_cast<char*>(ws) + p.total);
    hipError_t he = run_forward(p, params, obs, nullptr, n, static_cast<char*>(ws), z, value, stream);
    if (he != hipSuccess) return hip_status(he, "impala_actor_step: forward");
    return hip_status(gumbel_max(n, net->num_actions, z, gumbel, actions, logp, stream),
                      "impala_actor_step: sample");
}

// ------------------------------------------------------------------ layer-level entry points

static impala_status_t check_layer(const char* fn, int prec, int64_t n, int H, int W, int cin, int cout) {
    if (!valid_prec(prec)) return fail(IMPALA_EINVAL, "%s: bad prec", fn);
    if (n < 0 || n > (int64_t(1) << 24) || H < 1 || W < 1 || H > 256 || W > 256)
        return fail(IMPALA_EINVAL, "%s: shape out of range", fn);
    (void)cin; (void)cout;
    return IMPALA_OK;
}

impala_status_t impala_conv3x3_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t cin,
                                   int32_t cout, const void* x, int32_t x_mode,
                                   const int32_t* row_idx, const float* w, const float* bias,
                                   const void* add, void* y, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, cin, cout);
    if (st) return st;
    if (x_mode < 0 || x_mode > 2 || !conv3x3_supported(cin, cout, x_mode, 0))
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_fwd: unsupported cin=%d cout=%d x_mode=%d", cin, cout, x_mode);
    if (n == 0) return ok();
    CHECK_PTR(x); CHECK_PTR(w); CHECK_PTR(y);
    ConvArgs a{};
    a.x = x; a.row_idx = x_mode == IN_U8 ? row_idx : nullptr; a.w = w; a.bias = bias; a.add = add;
    a.y = y; a.n = int(n); a.H = H; a.W = W; a.scale = x_mode == IN_U8 ? 1.f / 255.f : 1.f;
    return hip_status(conv3x3(prec, cin, cout, x_mode, 0, a, stream), "impala_conv3x3_fwd");
}

impala_status_t impala_conv3x3_pool_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t cin,
                                        int32_t cout, const void* x, int32_t x_mode,
                                        const int32_t* row_idx, const float* w, const float* bias,
                                        void* y, uint8_t* arg, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, cin, cout);
    if (st) return st;
    if (prec != IMPALA_PREC_BF16)
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_pool_fwd: bf16 only (float32: conv, then max-pool)");
    if ((x_mode != IN_U8 && x_mode != IN_PLAIN) || !conv3x3_supported(cin, cout, x_mode, 0))
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_pool_fwd: unsupported cin=%d cout=%d x_mode=%d", cin, cout, x_mode);
    if (n == 0) return ok();
    CHECK_PTR(x); CHECK_PTR(w); CHECK_PTR(y); CHECK_PTR(arg);
    ConvArgs a{};
    a.x = x; a.row_idx = x_mode == IN_U8 ? row_idx : nullptr; a.w = w; a.bias = bias;
    a.y = y; a.arg = arg; a.n = int(n); a.H = H; a.W = W; a.scale = x_mode == IN_U8 ? 1.f / 255.f : 1.f;
    return hip_status(conv3x3_pool(cin, cout, x_mode, a, stream), "impala_conv3x3_pool_fwd");
}

impala_status_t impala_resblock_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                   const void* x, const float* w1, const float* b1, const float* w2,
                                   const float* b2, void* t, void* y, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, C, C);
    if (st) return st;
    if (prec != IMPALA_PREC_BF16 || !resblock_fwd_supported(C))
        return fail(IMPALA_EUNSUPPORTED, "impala_resblock_fwd: bf16 with C = 16 or 32 only (got prec=%d C=%d)", int(prec), C);
    if (n == 0) return ok();
    CHECK_PTR(x); CHECK_PTR(w1); CHECK_PTR(w2); CHECK_PTR(t); CHECK_PTR(y);
    ResBlockArgs a{};
    a.x = x; a.w1 = w1; a.b1 = b1; a.w2 = w2; a.b2 = b2; a.t = t; a.y = y;
    a.n = int(n); a.H = H; a.W = W;
    return hip_status(resblock_fwd(C, a, stream), "impala_resblock_fwd");
}

impala_status_t impala_conv3x3_dgrad(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t cin,
                                     int32_t cout, const void* dy, const float* w, const void* mask,
                                     const void* add, void* dx, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, cin, cout);
    if (st) return st;
    if (!conv3x3_supported(cin, cout, IN_PLAIN, 1))
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_dgrad: unsupported cin=%d cout=%d", cin, cout);
    if (n == 0) return ok();
    CHECK_PTR(dy); CHECK_PTR(w); CHECK_PTR(dx);
    ConvArgs a{};
    a.x = dy; a.w = w; a.mask = mask; a.add = add; a.y = dx;
    a.n = int(n); a.H = H; a.W = W; a.scale = 1.f;
    return hip_status(conv3x3(prec, cin, cout, IN_PLAIN, 1, a, stream), "impala_conv3x3_dgrad");
}

size_t impala_conv3x3_wgrad_workspace_bytes(impala_prec_t prec, int32_t H, int32_t W, int32_t cin,
                                            int32_t cout) {
    if (!valid_prec(prec) || H < 1 || W < 1) return 0;
    return wgrad_partial_floats(prec, cin, cout, H, W) * sizeof(float);
}

impala_status_t impala_conv3x3_wgrad(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t cin,
                                     int32_t cout, const void* x, int32_t x_mode,
                                     const int32_t* row_idx, const void* dy, float* dw, float* db,
                                     void* ws, size_t ws_bytes, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, cin, cout);
    if (st) return st;
    if (x_mode < 0 || x_mode > 2 || !wgrad_supported(cin, cout, x_mode))
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_wgrad: unsupported cin=%d cout=%d x_mode=%d", cin, cout, x_mode);
    CHECK_PTR(dw); CHECK_PTR(db);
    if (n == 0) {
        hipError_t he = fill_zero(dw, int64_t(9) * cin * cout, stream);
        if (he == hipSuccess) he = fill_zero(db, cout, stream);
        return hip_status(he, "impala_conv3x3_wgrad");
    }
    CHECK_PTR(x); CHECK_PTR(dy); CHECK_PTR(ws);
    const size_t need = wgrad_partial_floats(prec, cin, cout, H, W) * sizeof(float);
    if (ws_bytes < need) return fail(IMPALA_EWORKSPACE, "impala_conv3x3_wgrad: workspace %zu < %zu", ws_bytes, need);
    WgradArgs a{};
    a.x = x; a.row_idx = x_mode == IN_U8 ? row_idx : nullptr; a.dy = dy; a.dw = dw; a.db = db;
    a.partial = static_cast<float*>(ws); a.n = int(n); a.H = H; a.W = W;
    a.scale = x_mode == IN_U8 ? 1.f / 255.f : 1.f;
    return hip_status(conv3x3_wgrad(prec, cin, cout, x_mode, a, stream), "impala_conv3x3_wgrad");
}

size_t impala_conv3x3_bwd_workspace_bytes(impala_prec_t prec, int32_t cin, int32_t cout) {
    if (prec != IMPALA_PREC_BF16) return 0;
    return conv3x3_bwd_partial_floats(cin, cout) * sizeof(float);
}

impala_status_t impala_conv3x3_bwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t cin,
                                   int32_t cout, const void* dy, const uint8_t* pool_arg, const void* x,
                                   int32_t x_mode, const float* w, const void* add, void* dx, float* dw,
                                   float* db, void* ws, size_t ws_bytes, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, cin, cout);
    if (st) return st;
    if (prec != IMPALA_PREC_BF16 || !conv3x3_bwd_supported(cin, cout, x_mode, add != nullptr, pool_arg != nullptr))
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_bwd: unsupported prec=%d cin=%d cout=%d x_mode=%d add=%d pooled=%d",
                    int(prec), cin, cout, x_mode, int(add != nullptr), int(pool_arg != nullptr));
    CHECK_PTR(dw); CHECK_PTR(db);
    if (n == 0) {
        hipError_t he = fill_zero(dw, int64_t(9) * cin * cout, stream);
        if (he == hipSuccess) he = fill_zero(db, cout, stream);
        return hip_status(he, "impala_conv3x3_bwd");
    }
    CHECK_PTR(dy); CHECK_PTR(x); CHECK_PTR(w); CHECK_PTR(dx); CHECK_PTR(ws);
    const size_t need = conv3x3_bwd_partial_floats(cin, cout) * sizeof(float);
    if (ws_bytes < need) return fail(IMPALA_EWORKSPACE, "impala_conv3x3_bwd: workspace %zu < %zu", ws_bytes, need);
    ConvBwdArgs a{};
    a.dy = dy; a.arg = pool_arg; a.x = x; a.w = w; a.add = add; a.dx = dx; a.dw = dw; a.db = db;
    a.partial = static_cast<float*>(ws); a.n = int(n); a.H = H; a.W = W;
    return hip_status(conv3x3_bwd(cin, cout, x_mode, a, stream), "impala_conv3x3_bwd");
}

size_t impala_resblock_bwd_workspace_bytes(impala_prec_t prec, int32_t C) {
    if (prec != IMPALA_PREC_BF16) return 0;
    return resblock_bwd_partial_floats(C) * sizeof(float);
}

impala_status_t impala_resblock_bwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                    const void* dy, const void* t, const void* x, const float* wa,
                                    const float* wb, void* dx, float* dwa, float* dba, float* dwb,
                                    float* dbb, void* ws, size_t ws_bytes, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, C, C);
    if (st) return st;
    if (prec != IMPALA_PREC_BF16 || !resblock_bwd_supported(C))
        return fail(IMPALA_EUNSUPPORTED, "impala_resblock_bwd: bf16 with C = 16 or 32 only (got prec=%d C=%d)", int(prec), C);
    CHECK_PTR(dwa); CHECK_PTR(dba); CHECK_PTR(dwb); CHECK_PTR(dbb);
    if (n == 0) {
        hipError_t he = fill_zero(dwa, int64_t(9) * C * C, stream);
        if (he == hipSuccess) he = fill_zero(dba, C, stream);
        if (he == hipSuccess) he = fill_zero(dwb, int64_t(9) * C * C, stream);
        if (he == hipSuccess) he = fill_zero(dbb, C, stream);
        return hip_status(he, "impala_resblock_bwd");
    }
    CHECK_PTR(dy); CHECK_PTR(t); CHECK_PTR(x); CHECK_PTR(wa); CHECK_PTR(wb); CHECK_PTR(dx); CHECK_PTR(ws);
    const size_t need = resblock_bwd_partial_floats(C) * sizeof(float);
    if (ws_bytes < need) return fail(IMPALA_EWORKSPACE, "impala_resblock_bwd: workspace %zu < %zu", ws_bytes, need);
    ResBwdArgs a{};
    a.dy = dy; a.t = t; a.x = x; a.wa = wa; a.wb = wb; a.dx = dx;
    a.dwa = dwa; a.dba = dba; a.dwb = dwb; a.dbb = dbb;
    a.partial = static_cast<float*>(ws); a.n = int(n); a.H = H; a.W = W;
    PendingReduce out[2];
    hipError_t he = resblock_bwd(C, a, stream, out);
    if (he == hipSuccess) he = flush_pending_reduce(out[0], stream);
    if (he == hipSuccess) he = flush_pending_reduce(out[1], stream);
    return hip_status(he, "impala_resblock_bwd");
}

size_t impala_conv3x3_pool_wgrad_u8_workspace_bytes(impala_prec_t prec, int32_t cout) {
    if (prec != IMPALA_PREC_BF16) return 0;
    return pool_wgrad_u8_partial_floats(cout) * sizeof(float);
}

impala_status_t impala_conv3x3_pool_wgrad_u8(impala_prec_t prec, int64_t n, int32_t H, int32_t W,
                                             int32_t cout, const uint8_t* obs, const int32_t* row_idx,
                                             const void* dpool, const uint8_t* arg, float* dw, float* db,
                                             void* ws, size_t ws_bytes, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, 4, cout);
    if (st) return st;
    if (prec != IMPALA_PREC_BF16 || !pool_wgrad_u8_supported(cout))
        return fail(IMPALA_EUNSUPPORTED, "impala_conv3x3_pool_wgrad_u8: bf16 with cout = 16 or 32 only (got prec=%d cout=%d)",
                    int(prec), cout);
    CHECK_PTR(dw); CHECK_PTR(db);
    if (n == 0) {
        hipError_t he = fill_zero(dw, int64_t(36) * cout, stream);
        if (he == hipSuccess) he = fill_zero(db, cout, stream);
        return hip_status(he, "impala_conv3x3_pool_wgrad_u8");
    }
    CHECK_PTR(obs); CHECK_PTR(dpool); CHECK_PTR(arg); CHECK_PTR(ws);
    const size_t need = pool_wgrad_u8_partial_floats(cout) * sizeof(float);
    if (ws_bytes < need)
        return fail(IMPALA_EWORKSPACE, "impala_conv3x3_pool_wgrad_u8: workspace %zu < %zu", ws_bytes, need);
    PoolWgArgs a{};
    a.obs = obs; a.row_idx = row_idx; a.dp = dpool; a.arg = arg; a.dw = dw; a.db = db;
    a.partial = static_cast<float*>(ws); a.n = int(n); a.H = H; a.W = W;
    return hip_status(pool_wgrad_u8(cout, a, stream), "impala_conv3x3_pool_wgrad_u8");
}

impala_status_t impala_maxpool_fwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                   const void* x, void* y, uint8_t* arg, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, C, C);
    if (st) return st;
    if (C < 4 || C % 4 || C > 256) return fail(IMPALA_EUNSUPPORTED, "impala_maxpool_fwd: C must be a multiple of 4 up to 256");
    if (n == 0) return ok();
    CHECK_PTR(x); CHECK_PTR(y); CHECK_PTR(arg);
    return hip_status(maxpool_fwd(prec, int(n), H, W, C, x, y, arg, stream), "impala_maxpool_fwd");
}

impala_status_t impala_maxpool_bwd(impala_prec_t prec, int64_t n, int32_t H, int32_t W, int32_t C,
                                   const uint8_t* arg, const void* dy, void* dx, hipStream_t stream) {
    impala_status_t st = check_layer(__func__, prec, n, H, W, C, C);
    if (st) return st;
    if (C < 4 || C % 4 || C > 256) return fail(IMPALA_EUNSUPPORTED, "impala_maxpool_bwd: C must be a multiple of 4 up to 256");
    if (n == 0) return ok();
    CHECK_PTR(arg); CHECK_PTR(dy); CHECK_PTR(dx);
    return hip_status(maxpool_bwd(prec, int(n), H, W, C, arg, dy, dx, stream), "impala_maxpool_bwd");
}

impala_status_t impala_action_logp(int64_t n, int32_t A, const float* logits, const int32_t* actions,
                                   float* logp, hipStream_t stream) {
    if (n < 0 || n > (int64_t(1) << 26) || A < 1 || A > 64)
        return fail(IMPALA_EINVAL, "impala_action_logp: bad n or A");
    if (n == 0) return ok();
    CHECK_PTR(logits); CHECK_PTR(actions); CHECK_PTR(logp);
    return hip_status(action_logp(n, A, logits, actions, logp, stream), "impala_action_logp");
}

impala_status_t impala_gumbel_sample(int64_t n, int32_t A, const float* logits, const float* gumbel,
                                     int32_t* actions, float* logp, hipStream_t stream) {
    if (n < 0 || A < 1 || A > 64) return fail(IMPALA_EINVAL, "impala_gumbel_sample: bad n or A");
    if (n == 0) return ok();
    CHECK_PTR(logits); CHECK_PTR(gumbel); CHECK_PTR(actions); CHECK_PTR(logp);
    return hip_status(gumbel_max(n, A, logits, gumbel, actions, logp, stream), "impala_gumbel_sample");
}

impala_status_t impala_probe_mfma_bf16(int32_t blocks, int32_t iters, float* sink, int64_t* flop,
                                       hipStream_t stream) {
    if (blocks < 1 || blocks > 65536 || iters < 1 || iters > (1 << 20))
        return fail(IMPALA_EINVAL, "impala_probe_mfma_bf16: bad blocks or iters");
    CHECK_PTR(sink); CHECK_PTR(flop);
    *flop = mfma_probe_flop(blocks, iters);
    return hip_status(mfma_probe(blocks, iters, sink, stream), "impala_probe_mfma_bf16");
}

}  // extern "C"
