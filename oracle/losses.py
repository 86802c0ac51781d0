"""PPO and IMPALA losses over a minibatch, with their analytic gradients w.r.t. the logits
and the value output.

All losses are means over the m rows of the minibatch. The stats vector has 8 entries:
[total, policy, value, entropy, approx_kl, clipfrac, adv_mean, adv_std] for PPO and
[total, policy, value, entropy, mean pg_adv, mean vs, 0, 0] for IMPALA.
"""
from __future__ import annotations

import numpy as np


def log_softmax(z):
    zmax = z.max(axis=1, keepdims=True)
    s = z - zmax
    return s - np.log(np.exp(s).sum(axis=1, keepdims=True))


def ppo_loss_grad(logits, value, actions, old_logp, adv, ret, clip_eps, vf_coef, ent_coef,
                  norm_adv=True, adv_stats=None, dtype=np.float64):
    """Joint PPO loss L = -L^pi + c1 L^V - c2 L^S of Algorithm 1 (learning phase), with
    L^pi the clipped surrogate J^CLIP and S the entropy bonus of the full objective
    (Appendix A).

    A_hat = (A - mean A) / (std A + 1e-8) over the minibatch (population std), a constant;
    r = exp(log pi(a) - old_logp); per row pg = max(-A_hat r, -A_hat clip(r, 1-eps, 1+eps));
    H = -sum p log p; L = mean(pg) + c1 * 0.5 mean((V - R)^2) - c2 mean(H).

    dL/dz_ij = (1/m) [-kappa_i A_hat_i r_i (1[j=a_i] - p_ij) + c2 p_ij (log p_ij + H_i)]
    with kappa_i = 0 where the clipped branch is strictly larger (its derivative in r is 0
    there) and 1 otherwise; dL/dV_i = (c1/m) (V_i - R_i).

    ``adv_stats`` = (mean, std) overrides the minibatch statistics (used to express the
    data-parallel equivalence of Appendix A's Option 1 and Option 2).
    """
    z = np.asarray(logits, dtype)
    V = np.asarray(value, dtype)
    a_idx = np.asarray(actions, np.int64)
    A_raw = np.asarray(adv, dtype)
    R = np.asarray(ret, dtype)
    m, nA = z.shape
    mean, std = (A_raw.mean(), A_raw.std()) if adv_stats is None else adv_stats
    A_hat = (A_raw - mean) / (std + 1e-8) if norm_adv else A_raw
    logp_all = log_softmax(z)
    p = np.exp(logp_all)
    rows = np.arange(m)
    logp = logp_all[rows, a_idx]
    ratio = np.exp(logp - np.asarray(old_logp, dtype))
    pg_unclipped = -A_hat * ratio
    pg_clipped = -A_hat * np.clip(ratio, 1 - clip_eps, 1 + clip_eps)
    pg = np.maximum(pg_unclipped, pg_clipped)
    H = -(p * logp_all).sum(1)
    v_loss = 0.5 * ((V - R) ** 2).mean()
    loss = pg.mean() + vf_coef * v_loss - ent_coef * H.mean()

    kappa = np.where(pg_clipped > pg_unclipped, 0.0, 1.0)
    onehot = np.zeros_like(z)
    onehot[rows, a_idx] = 1
    dz = (-(kappa * A_hat * ratio)[:, None] * (onehot - p)
          + ent_coef * p * (logp_all + H[:, None])) / m
    dV = vf_coef * (V - R) / m
    approx_kl = ((ratio - 1) - np.log(ratio)).mean()
    clipfrac = (np.abs(ratio - 1) > clip_eps).mean()
    stats = np.array([loss, pg.mean(), v_loss, H.mean(), approx_kl, clipfrac, mean, std], dtype)
    return loss, dz, dV, stats


def impala_loss_grad(logits, value, actions, vs, pg_adv, pg_coef, vf_coef, ent_coef,
                     dtype=np.float64):
    """IMPALA loss (Appendix B's IMPALA table: policy gradient, value coefficient c1,
    entropy coefficient c2): L = c_pg mean(-pg_adv log pi(a)) + c1 * 0.5 mean((V - v_s)^2)
    - c2 mean(H). pg_adv and v_s are constants (stop-gradient).

    dL/dz_ij = (1/m) [-c_pg pg_adv_i (1[j=a_i] - p_ij) + c2 p_ij (log p_ij + H_i)];
    dL/dV_i = (c1/m) (V_i - v_s,i).
    """
    z = np.asarray(logits, dtype)
    V = np.asarray(value, dtype)
    a_idx = np.asarray(actions, np.int64)
    adv = np.asarray(pg_adv, dtype)
    tgt = np.asarray(vs, dtype)
    m, nA = z.shape
    logp_all = log_softmax(z)
    p = np.exp(logp_all)
    rows = np.arange(m)
    logp = logp_all[rows, a_idx]
    H = -(p * logp_all).sum(1)
    pg = -adv * logp
    v_loss = 0.5 * ((V - tgt) ** 2).mean()
    loss = pg_coef * pg.mean() + vf_coef * v_loss - ent_coef * H.mean()
    onehot = np.zeros_like(z)
    onehot[rows, a_idx] = 1
    dz = (-(pg_coef * adv)[:, None] * (onehot - p) + ent_coef * p * (logp_all + H[:, None])) / m
    dV = vf_coef * (V - tgt) / m
    stats = np.array([loss, pg.mean(), v_loss, H.mean(), adv.mean(), tgt.mean(), 0, 0], dtype)
    return loss, dz, dV, stats


def gumbel_max(logits, gumbel):
    """Categorical sample a = argmax_j(z_j + g_j) with g ~ Gumbel(0,1) supplied by the caller
    (the actor's 'a_t ~ pi(.|s_t)' of Algorithm 1); ties go to the lowest index.
    Returns (actions int32, log pi(a))."""
    z = np.asarray(logits)
    a = np.argmax(z + np.asarray(gumbel, z.dtype), axis=1).astype(np.int32)
    return a, log_softmax(z)[np.arange(z.shape[0]), a]
