"""ctypes binding of libcleanba_learner.so: the C-ABI of include/cleanba_learner.h and
include/cleanba_layers.h under the same names.

This layer only marshals arguments (torch tensors -> device pointers, the current HIP
stream, C structs) and turns non-zero statuses into exceptions; every step of the learner
runs in the library's HIP kernels. Importing it fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcleanba_learner.so")

PREC_BF16, PREC_FP32 = 0, 1
LEARNER_PPO, LEARNER_IMPALA = 0, 1
LEARNER_OPT_ADAM, LEARNER_OPT_RMSPROP = 0, 1
X_PLAIN, X_RELU, X_U8 = 0, 1, 2
STATUS = {0: "OK", -1: "EINVAL", -2: "EWORKSPACE", -3: "EUNSUPPORTED", -4: "EHIP"}


class ImpalaNet(C.Structure):
    _fields_ = [("in_h", C.c_int32), ("in_w", C.c_int32), ("in_c", C.c_int32),
                ("ch", C.c_int32 * 3), ("hidden", C.c_int32), ("num_actions", C.c_int32)]


class TensorDesc(C.Structure):
    _fields_ = [("name", C.c_char * 32), ("offset", C.c_int64), ("ndim", C.c_int32),
                ("shape", C.c_int32 * 4)]


class ActivationDesc(C.Structure):
    _fields_ = [("name", C.c_char * 32), ("offset", C.c_int64), ("bytes", C.c_int64), ("dtype", C.c_int32),
                ("ndim", C.c_int32), ("shape", C.c_int64 * 4)]


DT_U8, DT_BF16, DT_F32 = 0, 1, 2


class LearnerCfg(C.Structure):
    _fields_ = [("algo", C.c_int32), ("prec", C.c_int32), ("T", C.c_int32), ("E", C.c_int32),
                ("update_epochs", C.c_int32), ("num_minibatches", C.c_int32),
                ("minibatch_size", C.c_int32), ("norm_adv", C.c_int32),
                ("gamma", C.c_float), ("lambda_", C.c_float), ("clip_eps", C.c_float),
                ("vf_coef", C.c_float), ("ent_coef", C.c_float), ("pg_coef", C.c_float),
                ("rho_bar", C.c_float), ("c_bar", C.c_float), ("pg_rho_bar", C.c_float),
                ("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float),
                ("adam_eps", C.c_float), ("max_grad_norm", C.c_float),
                ("optimizer", C.c_int32), ("rms_decay", C.c_float), ("rms_eps", C.c_float)]


class Rollout(C.Structure):
    _fields_ = [("obs", C.c_void_p), ("actions", C.c_void_p), ("behav_logp", C.c_void_p),
                ("rewards", C.c_void_p), ("dones", C.c_void_p), ("values", C.c_void_p),
                ("next_value", C.c_void_p), ("next_done", C.c_void_p)]


_P, _I32, _I64, _F, _SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_size_t
_NETP = C.POINTER(ImpalaNet)

_SIGS = {
    "impala_param_count": (_I64, [_NETP]),
    "impala_param_layout": (C.c_int, [_NETP, C.POINTER(TensorDesc), C.c_int]),
    "impala_workspace_bytes": (_SZ, [_NETP, _I64, C.c_int, C.c_int]),
    "impala_activation_layout": (C.c_int, [_NETP, C.c_int, _I64, C.POINTER(ActivationDesc), C.c_int]),
    "impala_last_error": (C.c_char_p, []),
    "impala_cnn_fwd": (C.c_int, [_NETP, C.c_int, _P, _P, _P, _I64, _P, _SZ, C.c_int, _P, _P, _P]),
    "impala_cnn_bwd": (C.c_int, [_NETP, C.c_int, _P, _P, _P, _I64, _P, _SZ, _P, _P, _P, _P]),
    "gae_advantages": (C.c_int, [_I32, _I32, _P, _P, _P, _P, _P, _F, _F, _P, _P, _P]),
    "vtrace_targets": (C.c_int, [_I32, _I32, _P, _P, _P, _P, _P, _P, _P, _F, _F, _F, _F, _F, _P, _P, _P]),
    "loss_workspace_bytes": (_SZ, [_I64]),
    "ppo_loss_grad": (C.c_int, [_I64, _I32, _P, _P, _P, _P, _P, _P, _I32, _F, _F, _F, _P, _P, _P, _P, _SZ, _P]),
    "impala_loss_grad": (C.c_int, [_I64, _I32, _P, _P, _P, _P, _P, _F, _F, _F, _P, _P, _P, _P, _SZ, _P]),
    "adam_workspace_bytes": (_SZ, [_I64]),
    "adam_step": (C.c_int, [_I64, _P, _P, _P, _P, _I32, _F, _F, _F, _F, _F, _P, _P, _SZ, _P]),
    "adam_step_noalloc": (C.c_int, [_I64, _P, _P, _P, _P, _I32, _F, _F, _F, _F, _F, _P, _P]),
    "rmsprop_workspace_bytes": (_SZ, [_I64]),
    "rmsprop_step": (C.c_int, [_I64, _P, _P, _P, _F, _F, _F, _F, _P, _P, _SZ, _P]),
    "learner_workspace_bytes": (_SZ, [_NETP, C.POINTER(LearnerCfg)]),
    "learner_step": (C.c_int, [_NETP, C.POINTER(LearnerCfg), C.POINTER(Rollout), _P, _P, _P,
                               C.POINTER(_I32), _P, _P, _SZ, _P, _P]),
    "impala_actor_step": (C.c_int, [_NETP, C.c_int, _P, _P, _I64, _P, _P, _SZ, _P, _P, _P, _P, _P]),
    "impala_conv3x3_fwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _I32, _P, _I32, _P, _P, _P, _P, _P, _P]),
    "impala_conv3x3_pool_fwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _I32, _P, _I32, _P, _P, _P, _P, _P,
                                          _P]),
    "impala_resblock_fwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P]),
    "impala_conv3x3_dgrad": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P]),
    "impala_conv3x3_wgrad_workspace_bytes": (_SZ, [C.c_int, _I32, _I32, _I32, _I32]),
    "impala_conv3x3_wgrad": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _I32, _P, _I32, _P, _P, _P, _P,
                                       _P, _SZ, _P]),
    "impala_conv3x3_bwd_workspace_bytes": (_SZ, [C.c_int, _I32, _I32]),
    "impala_conv3x3_bwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _I32, _P, _P, _P, _P,
                                     _P, _P, _SZ, _P]),
    "impala_resblock_bwd_workspace_bytes": (_SZ, [C.c_int, _I32]),
    "impala_resblock_bwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                      _P, _SZ, _P]),
    "impala_conv3x3_pool_wgrad_u8_workspace_bytes": (_SZ, [C.c_int, _I32]),
    "impala_conv3x3_pool_wgrad_u8": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                               _P]),
    "impala_maxpool_fwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _P, _P, _P, _P]),
    "impala_maxpool_bwd": (C.c_int, [C.c_int, _I64, _I32, _I32, _I32, _P, _P, _P, _P]),
    "impala_gumbel_sample": (C.c_int, [_I64, _I32, _P, _P, _P, _P, _P]),
    "impala_action_logp": (C.c_int, [_I64, _I32, _P, _P, _P, _P]),
    "impala_profile_begin": (C.c_int, [C.c_char_p, _I32]),
    "impala_profile_end": (C.c_int, []),
    "impala_profile_key": (C.c_int, [_I32, C.c_char_p, _SZ, C.POINTER(C.c_double), C.POINTER(_I32)]),
    "impala_profile_dropped": (_I32, []),
    "impala_probe_mfma_bf16": (C.c_int, [_I32, _I32, _P, C.POINTER(_I64), _P]),
}


def _load() -> C.CDLL:
    # PyTorch's HIP runtime must be the one in the process before the library loads: its
    # soname matches the library's dependency, so the loader reuses it and device memory,
    # streams and kernels all live in a single runtime.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2310_00036_amd.build.build() "
                          "(the learner has no fallback path)")
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


class LibraryError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = (lib.impala_last_error() or b"").decode()
        super().__init__(f"{fn} -> {STATUS.get(status, status)}: {msg}")
        self.status = status


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise LibraryError(fn, status)


def net_struct(shape) -> ImpalaNet:
    """ImpalaNet from anything with in_h, in_w, in_c, ch, hidden, num_actions."""
    n = ImpalaNet()
    n.in_h, n.in_w, n.in_c = shape.in_h, shape.in_w, shape.in_c
    for i in range(3):
        n.ch[i] = shape.ch[i]
    n.hidden, n.num_actions = shape.hidden, shape.num_actions
    return n


def ptr(t) -> int | None:
    """Device pointer of a contiguous torch tensor (None passes NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def stream_handle(stream=None) -> int | None:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


# ------------------------------------------------------------------ thin wrappers


def impala_param_count(net) -> int:
    n = lib.impala_param_count(C.byref(net_struct(net)))
    if n < 0:
        raise LibraryError("impala_param_count", -1)
    return int(n)


def impala_param_layout(net) -> list:
    descs = (TensorDesc * 64)()
    k = lib.impala_param_layout(C.byref(net_struct(net)), descs, 64)
    if k < 0:
        raise LibraryError("impala_param_layout", k)
    return [(d.name.decode(), tuple(d.shape[i] for i in range(d.ndim)), int(d.offset))
            for d in descs[:k]]


def impala_workspace_bytes(net, n_frames: int, prec: int, training: int) -> int:
    return int(lib.impala_workspace_bytes(C.byref(net_struct(net)), n_frames, prec, training))


def impala_activation_layout(net, prec: int, n_frames: int) -> list:
    """[(name, byte offset, bytes, dtype, shape)] of the activations a training-mode forward on
    n_frames frames leaves in its workspace (dtype: DT_U8, DT_BF16 or DT_F32)."""
    descs = (ActivationDesc * 64)()
    k = lib.impala_activation_layout(C.byref(net_struct(net)), prec, n_frames, descs, 64)
    if k < 0:
        raise LibraryError("impala_activation_layout", k)
    return [(d.name.decode(), int(d.offset), int(d.bytes), int(d.dtype), tuple(d.shape[i] for i in range(d.ndim)))
            for d in descs[:k]]


def impala_cnn_fwd(net, prec, params, obs, row_idx, n, ws, training, logits, value, stream=None):
    _check("impala_cnn_fwd", lib.impala_cnn_fwd(
        C.byref(net_struct(net)), prec, ptr(params), ptr(obs), ptr(row_idx), n, ptr(ws),
        ws.numel() * ws.element_size(), training, ptr(logits), ptr(value), stream_handle(stream)))


def impala_cnn_bwd(net, prec, params, obs, row_idx, n, ws, dlogits, dvalue, grads, stream=None):
    _check("impala_cnn_bwd", lib.impala_cnn_bwd(
        C.byref(net_struct(net)), prec, ptr(params), ptr(obs), ptr(row_idx), n, ptr(ws),
        ws.numel() * ws.element_size(), ptr(dlogits), ptr(dvalue), ptr(grads), stream_handle(stream)))


def gae_advantages(T, E, rewards, values, dones, next_value, next_done, gamma, lam, adv, ret,
                   stream=None):
    _check("gae_advantages", lib.gae_advantages(
        T, E, ptr(rewards), ptr(values), ptr(dones), ptr(next_value), ptr(next_done), gamma, lam,
        ptr(adv), ptr(ret), stream_handle(stream)))


def vtrace_targets(T, E, behav_logp, target_logp, rewards, values, dones, bootstrap_value,
                   next_done, gamma, lam, rho_bar, c_bar, pg_rho_bar, vs, pg_adv, stream=None):
    _check("vtrace_targets", lib.vtrace_targets(
        T, E, ptr(behav_logp), ptr(target_logp), ptr(rewards), ptr(values), ptr(dones),
        ptr(bootstrap_value), ptr(next_done), gamma, lam, rho_bar, c_bar, pg_rho_bar, ptr(vs),
        ptr(pg_adv), stream_handle(stream)))


def loss_workspace_bytes(m: int) -> int:
    return int(lib.loss_workspace_bytes(m))


def _ws_args(ws):
    return (ptr(ws), ws.numel() * ws.element_size()) if ws is not None else (None, 0)


def ppo_loss_grad(m, A, logits, value, actions, old_logp, adv, ret, norm_adv, clip_eps, vf_coef,
                  ent_coef, dlogits, dvalue, stats, ws=None, stream=None):
    _check("ppo_loss_grad", lib.ppo_loss_grad(
        m, A, ptr(logits), ptr(value), ptr(actions), ptr(old_logp), ptr(adv), ptr(ret), norm_adv,
        clip_eps, vf_coef, ent_coef, ptr(dlogits), ptr(dvalue), ptr(stats), *_ws_args(ws),
        stream_handle(stream)))


def impala_loss_grad(m, A, logits, value, actions, vs, pg_adv, pg_coef, vf_coef, ent_coef,
                     dlogits, dvalue, stats, ws=None, stream=None):
    _check("impala_loss_grad", lib.impala_loss_grad(
        m, A, ptr(logits), ptr(value), ptr(actions), ptr(vs), ptr(pg_adv), pg_coef, vf_coef,
        ent_coef, ptr(dlogits), ptr(dvalue), ptr(stats), *_ws_args(ws), stream_handle(stream)))


def adam_workspace_bytes(n_params: int) -> int:
    return int(lib.adam_workspace_bytes(n_params))


def adam_step(n_params, params, grads, m, v, step, lr, beta1, beta2, eps, max_grad_norm, stats,
              ws, stream=None):
    _check("adam_step", lib.adam_step(
        n_params, ptr(params), ptr(grads), ptr(m), ptr(v), step, lr, beta1, beta2, eps,
        max_grad_norm, ptr(stats), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))


def adam_step_noalloc(n_params, params, grads, m, v, step, lr, beta1, beta2, eps, max_grad_norm, stats,
                      stream=None):
    _check("adam_step_noalloc", lib.adam_step_noalloc(
        n_params, ptr(params), ptr(grads), ptr(m), ptr(v), step, lr, beta1, beta2, eps, max_grad_norm,
        ptr(stats), stream_handle(stream)))


def rmsprop_workspace_bytes(n_params: int) -> int:
    return int(lib.rmsprop_workspace_bytes(n_params))


def rmsprop_step(n_params, params, grads, nu, lr, decay, eps, max_grad_norm, stats, ws, stream=None):
    _check("rmsprop_step", lib.rmsprop_step(
        n_params, ptr(params), ptr(grads), ptr(nu), lr, decay, eps, max_grad_norm, ptr(stats), ptr(ws),
        ws.numel() * ws.element_size(), stream_handle(stream)))


def learner_cfg(wl, prec: int) -> LearnerCfg:
    """LearnerCfg from a workload description (synth.Workload or anything alike)."""
    c = LearnerCfg()
    c.algo = LEARNER_PPO if wl.algo == "ppo" else LEARNER_IMPALA
    c.prec = prec
    c.T, c.E = wl.T, wl.E
    c.update_epochs, c.num_minibatches, c.minibatch_size = wl.epochs, wl.num_minibatches, wl.mb
    c.norm_adv = int(wl.norm_adv)
    c.gamma, c.lambda_, c.clip_eps = wl.gamma, wl.lam, wl.clip_eps
    c.vf_coef, c.ent_coef, c.pg_coef = wl.vf_coef, wl.ent_coef, wl.pg_coef
    c.rho_bar, c.c_bar, c.pg_rho_bar = wl.rho_bar, wl.c_bar, wl.pg_rho_bar
    c.lr, c.beta1, c.beta2, c.adam_eps = wl.lr, wl.beta1, wl.beta2, wl.adam_eps
    c.max_grad_norm = wl.max_grad_norm
    c.optimizer = LEARNER_OPT_RMSPROP if getattr(wl, "optimizer", "adam") == "rmsprop" else LEARNER_OPT_ADAM
    c.rms_decay, c.rms_eps = getattr(wl, "rms_decay", 0.99), getattr(wl, "rms_eps", 0.01)
    return c


def learner_workspace_bytes(net, cfg: LearnerCfg) -> int:
    return int(lib.learner_workspace_bytes(C.byref(net_struct(net)), C.byref(cfg)))


def rollout_struct(obs, actions, behav_logp, rewards, dones, values, next_value, next_done) -> Rollout:
    r = Rollout()
    r.obs, r.actions, r.behav_logp = ptr(obs), ptr(actions), ptr(behav_logp)
    r.rewards, r.dones, r.values = ptr(rewards), ptr(dones), ptr(values)
    r.next_value, r.next_done = ptr(next_value), ptr(next_done)
    return r


def learner_step(net, cfg: LearnerCfg, rollout: Rollout, params, m, v, step: int, perm, ws, stats,
                 stream=None) -> int:
    """Runs one learning phase; returns the updated 1-based update count."""
    st = C.c_int32(step)
    _check("learner_step", lib.learner_step(
        C.byref(net_struct(net)), C.byref(cfg), C.byref(rollout), ptr(params), ptr(m), ptr(v),
        C.byref(st), ptr(perm), ptr(ws), ws.numel() * ws.element_size(), ptr(stats),
        stream_handle(stream)))
    return st.value


def impala_actor_step(net, prec, params, obs, n, gumbel, ws, actions, logp, value, logits=None,
                      stream=None):
    _check("impala_actor_step", lib.impala_actor_step(
        C.byref(net_struct(net)), prec, ptr(params), ptr(obs), n, ptr(gumbel), ptr(ws),
        ws.numel() * ws.element_size(), ptr(actions), ptr(logp), ptr(value), ptr(logits),
        stream_handle(stream)))


def impala_conv3x3_fwd(prec, n, H, W, cin, cout, x, x_mode, row_idx, w, bias, add, y, stream=None):
    _check("impala_conv3x3_fwd", lib.impala_conv3x3_fwd(
        prec, n, H, W, cin, cout, ptr(x), x_mode, ptr(row_idx), ptr(w), ptr(bias), ptr(add), ptr(y),
        stream_handle(stream)))


def impala_conv3x3_pool_fwd(prec, n, H, W, cin, cout, x, x_mode, row_idx, w, bias, y, arg, stream=None):
    _check("impala_conv3x3_pool_fwd", lib.impala_conv3x3_pool_fwd(
        prec, n, H, W, cin, cout, ptr(x), x_mode, ptr(row_idx), ptr(w), ptr(bias), ptr(y), ptr(arg),
        stream_handle(stream)))


def impala_resblock_fwd(prec, n, H, W, C_, x, w1, b1, w2, b2, t, y, stream=None):
    _check("impala_resblock_fwd", lib.impala_resblock_fwd(
        prec, n, H, W, C_, ptr(x), ptr(w1), ptr(b1), ptr(w2), ptr(b2), ptr(t), ptr(y), stream_handle(stream)))


def impala_conv3x3_dgrad(prec, n, H, W, cin, cout, dy, w, mask, add, dx, stream=None):
    _check("impala_conv3x3_dgrad", lib.impala_conv3x3_dgrad(
        prec, n, H, W, cin, cout, ptr(dy), ptr(w), ptr(mask), ptr(add), ptr(dx), stream_handle(stream)))


def impala_conv3x3_wgrad_workspace_bytes(prec, H, W, cin, cout) -> int:
    return int(lib.impala_conv3x3_wgrad_workspace_bytes(prec, H, W, cin, cout))


def impala_conv3x3_wgrad(prec, n, H, W, cin, cout, x, x_mode, row_idx, dy, dw, db, ws, stream=None):
    _check("impala_conv3x3_wgrad", lib.impala_conv3x3_wgrad(
        prec, n, H, W, cin, cout, ptr(x), x_mode, ptr(row_idx), ptr(dy), ptr(dw), ptr(db), ptr(ws),
        ws.numel() * ws.element_size(), stream_handle(stream)))


def impala_conv3x3_bwd_workspace_bytes(prec, cin, cout) -> int:
    return int(lib.impala_conv3x3_bwd_workspace_bytes(prec, cin, cout))


def impala_conv3x3_bwd(prec, n, H, W, cin, cout, dy, x, x_mode, w, add, dx, dw, db, ws, stream=None,
                       pool_arg=None):
    _check("impala_conv3x3_bwd", lib.impala_conv3x3_bwd(
        prec, n, H, W, cin, cout, ptr(dy), ptr(pool_arg), ptr(x), x_mode, ptr(w), ptr(add), ptr(dx), ptr(dw),
        ptr(db), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))


def impala_resblock_bwd_workspace_bytes(prec, C_) -> int:
    return int(lib.impala_resblock_bwd_workspace_bytes(prec, C_))


def impala_resblock_bwd(prec, n, H, W, C_, dy, t, x, wa, wb, dx, dwa, dba, dwb, dbb, ws, stream=None):
    _check("impala_resblock_bwd", lib.impala_resblock_bwd(
        prec, n, H, W, C_, ptr(dy), ptr(t), ptr(x), ptr(wa), ptr(wb), ptr(dx), ptr(dwa), ptr(dba), ptr(dwb),
        ptr(dbb), ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))


def impala_conv3x3_pool_wgrad_u8_workspace_bytes(prec, cout) -> int:
    return int(lib.impala_conv3x3_pool_wgrad_u8_workspace_bytes(prec, cout))


def impala_conv3x3_pool_wgrad_u8(prec, n, H, W, cout, obs, row_idx, dpool, arg, dw, db, ws, stream=None):
    _check("impala_conv3x3_pool_wgrad_u8", lib.impala_conv3x3_pool_wgrad_u8(
        prec, n, H, W, cout, ptr(obs), ptr(row_idx), ptr(dpool), ptr(arg), ptr(dw), ptr(db), ptr(ws),
        ws.numel() * ws.element_size(), stream_handle(stream)))


def impala_maxpool_fwd(prec, n, H, W, C_, x, y, arg, stream=None):
    _check("impala_maxpool_fwd", lib.impala_maxpool_fwd(prec, n, H, W, C_, ptr(x), ptr(y), ptr(arg),
                                                        stream_handle(stream)))


def impala_maxpool_bwd(prec, n, H, W, C_, arg, dy, dx, stream=None):
    _check("impala_maxpool_bwd", lib.impala_maxpool_bwd(prec, n, H, W, C_, ptr(arg), ptr(dy), ptr(dx),
                                                        stream_handle(stream)))


def impala_gumbel_sample(n, A, logits, gumbel, actions, logp, stream=None):
    _check("impala_gumbel_sample", lib.impala_gumbel_sample(n, A, ptr(logits), ptr(gumbel), ptr(actions),
                                                            ptr(logp), stream_handle(stream)))


def impala_action_logp(n, A, logits, actions, logp, stream=None):
    _check("impala_action_logp", lib.impala_action_logp(n, A, ptr(logits), ptr(actions), ptr(logp),
                                                        stream_handle(stream)))


def impala_probe_mfma_bf16(blocks, iters, sink, stream=None) -> int:
    """Launch the register-only MFMA loop (cleanba_profile.h); returns its matrix-core flop."""
    flop = C.c_int64()
    _check("impala_probe_mfma_bf16", lib.impala_probe_mfma_bf16(blocks, iters, ptr(sink), C.byref(flop),
                                                                stream_handle(stream)))
    return flop.value


def impala_profile_begin(only_key: str | None = None, max_launches: int = 1 << 16) -> None:
    _check("impala_profile_begin", lib.impala_profile_begin(
        only_key.encode() if only_key else None, max_launches))


def impala_profile_end() -> list:
    """Close the profile; returns [(key, total_ms, launches)] sorted by total time."""
    k = lib.impala_profile_end()
    if k < 0:
        raise LibraryError("impala_profile_end", k)
    out = []
    buf = C.create_string_buffer(128)
    ms, cnt = C.c_double(), C.c_int32()
    for i in range(k):
        _check("impala_profile_key", lib.impala_profile_key(i, buf, 128, C.byref(ms), C.byref(cnt)))
        out.append((buf.value.decode(), ms.value, cnt.value))
    return sorted(out, key=lambda r: -r[1])
