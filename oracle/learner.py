"""One learner update of Cleanba's PPO (Algorithm 1, learning phase) and IMPALA, plus the
actor's sampling step, composed from the oracle's parts.

The rollout is time-major [T, E] and is flattened row-major (row t*E + e), as Algorithm 1
prepares and flattens the batch B. Minibatch k of epoch j takes rows
perm[j, k*m:(k+1)*m]; the permutation is an input.
"""
from __future__ import annotations

import numpy as np

from . import losses, net as netmod, optim, targets


def _opt_update(params, g, m, v, step, cfg, dtype):
    """Clip the gradient's global norm, then the configured optimiser: Adam (m, v) or
    RMSprop (v holds its second-moment estimate; m passes through)."""
    g, gnorm = optim.clip_by_global_norm(g, cfg.max_grad_norm, dtype)
    if getattr(cfg, "optimizer", "adam") == "rmsprop":
        p, v = optim.rmsprop(params, g, v, cfg.lr, cfg.rms_decay, cfg.rms_eps, dtype)
        return p, m, v, gnorm
    p, m, v = optim.adam(params, g, m, v, step, cfg.lr, cfg.beta1, cfg.beta2, cfg.adam_eps, dtype)
    return p, m, v, gnorm


def ppo_learner_step(net, cfg, ro, params, m, v, step, perm, prec="fp64"):
    """GAE once over the rollout, then update_epochs x num_minibatches updates, each:
    normalise advantages -> losses -> back-propagate -> clip grad norm -> optimiser step.

    ro: dict with obs [T*E, H, W, C] u8, actions [T*E], logp [T*E] (behaviour), rewards,
    values, dones [T, E], next_value [E], next_done [E].
    Returns (params, m, v, step, stats [n_updates, 8]) with stats rows
    [total, policy, value, entropy, approx_kl, clipfrac, grad_norm, nonfinite].
    """
    dtype = np.float64 if prec == "fp64" else np.float32
    adv, ret = targets.gae(ro["rewards"], ro["values"], ro["dones"], ro["next_value"],
                           ro["next_done"], cfg.gamma, cfg.lam, dtype)
    adv, ret = adv.ravel(), ret.ravel()
    mb = cfg.mb
    out = []
    p, m_, v_ = (np.asarray(a, dtype) for a in (params, m, v))
    for j in range(cfg.epochs):
        for k in range(cfg.num_minibatches):
            rows = perm[j, k * mb:(k + 1) * mb]
            z, val, cache = netmod.forward(net, p, ro["obs"][rows], prec)
            _, dz, dv, st = losses.ppo_loss_grad(z, val, ro["actions"][rows], ro["logp"][rows],
                                                 adv[rows], ret[rows], cfg.clip_eps, cfg.vf_coef,
                                                 cfg.ent_coef, bool(cfg.norm_adv), dtype=dtype)
            g = netmod.backward(net, cache, dz, dv)
            step += 1
            p, m_, v_, gn = _opt_update(p, g, m_, v_, step, cfg, dtype)
            out.append(list(st[:6]) + [gn, float(not np.isfinite(gn))])
    return p, m_, v_, step, np.array(out)


def impala_learner_step(net, cfg, ro, params, m, v, step, prec="fp64"):
    """num_minibatches updates, minibatch k being the env block [k*E/N, (k+1)*E/N) over all T
    steps (V-trace runs along time, so a minibatch keeps whole trajectories). Each update:
    forward over the block's T*Eb rollout frames plus its Eb bootstrap frames, V-trace from the
    current policy's log-probs and values (constants), IMPALA loss, backward over the rollout
    rows (the bootstrap rows get zero gradient), clip, optimiser step.

    ro: obs [(T+1)*E, H, W, C] u8 (row t*E + e; rows T*E.. are the bootstrap frames), actions
    [T*E], logp [T*E] (behaviour mu), rewards, dones [T, E], next_done [E].
    """
    dtype = np.float64 if prec == "fp64" else np.float32
    T, E = ro["rewards"].shape
    nmb = getattr(cfg, "num_minibatches", 1) or 1
    if E % nmb:
        raise ValueError("IMPALA minibatches split the envs evenly")
    Eb = E // nmb
    p, m_, v_ = (np.asarray(a, dtype) for a in (params, m, v))
    out = []
    for k in range(nmb):
        envs = np.arange(k * Eb, (k + 1) * Eb)
        rows = (np.arange(T + 1)[:, None] * E + envs[None, :]).ravel()   # (t, e) order, t = T: bootstrap
        n = T * Eb
        z, val, cache = netmod.forward(net, p, ro["obs"][rows], prec)
        act = ro["actions"][rows[:n]]
        tlogp = losses.log_softmax(z[:n])[np.arange(n), act]
        vs, pg_adv = targets.vtrace(ro["logp"][rows[:n]].reshape(T, Eb), tlogp.reshape(T, Eb),
                                    ro["rewards"][:, envs], val[:n].reshape(T, Eb), ro["dones"][:, envs],
                                    val[n:], ro["next_done"][envs], cfg.gamma, cfg.lam, cfg.rho_bar,
                                    cfg.c_bar, cfg.pg_rho_bar, dtype)
        _, dz, dv, st = losses.impala_loss_grad(z[:n], val[:n], act, vs.ravel(), pg_adv.ravel(),
                                                cfg.pg_coef, cfg.vf_coef, cfg.ent_coef, dtype)
        dz_all = np.zeros_like(z)
        dz_all[:n] = dz
        dv_all = np.zeros_like(val)
        dv_all[:n] = dv
        g = netmod.backward(net, cache, dz_all, dv_all)
        step += 1
        p, m_, v_, gn = _opt_update(p, g, m_, v_, step, cfg, dtype)
        out.append(list(st[:6]) + [gn, float(not np.isfinite(gn))])
    return p, m_, v_, step, np.array(out)


def actor_step(net, params, obs, gumbel, prec="fp64"):
    """Algorithm 1's 'a_t ~ pi(.|s_t), v_t = v(s_t)': forward then Gumbel-max sampling.
    Returns (actions, log pi(a), value, logits)."""
    z, val, _ = netmod.forward(net, params, obs, prec)
    a, logp = losses.gumbel_max(z, gumbel)
    return a, logp, val, z


def behaviour_rollout(wl, params, raw, prec="fp64"):
    """Turn the raw random draws of one rollout into learner inputs using the initial policy.

    PPO: actions ~ pi_0 by Gumbel-max, values and next_value from pi_0's value head, and the
    stored behaviour log-prob is log pi_0(a) plus N(0, s) noise (so ratios start near 1).
    IMPALA: behaviour logits mu = pi_0's logits plus per-logit N(0, s) noise, actions ~ mu,
    behaviour log-prob log mu(a) (so the rollout is off-policy).
    """
    net = wl.net
    T, E = wl.T, wl.E
    n = T * E
    obs = raw["obs"].reshape((T + 1) * E, net.in_h, net.in_w, net.in_c)
    z, val, _ = netmod.forward(net, params, obs, prec)
    ro = dict(rewards=raw["rewards"], dones=raw["dones"], next_done=raw["next_done"])
    if wl.algo == "ppo":
        a, logp = losses.gumbel_max(z[:n], raw["gumbel"][:n])
        ro.update(obs=obs[:n], actions=a, logp=(logp + raw["bnoise"]).astype(np.float32),
                  values=val[:n].reshape(T, E).astype(np.float32),
                  next_value=val[n:].astype(np.float32))
    else:
        mu = z[:n] + raw["bnoise"]
        a, logp = losses.gumbel_max(mu, raw["gumbel"][:n])
        ro.update(obs=obs, actions=a, logp=logp.astype(np.float32))
    return ro
