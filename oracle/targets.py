"""Learning targets: GAE for PPO and V-trace for IMPALA, as reverse-time recurrences.

Data are time-major [T, E]. Done flags follow Algorithm 1's rollout phase: the flag stored
with step t is the one cached *before* stepping, so d_t = 1 means s_t begins a new episode.
Transition t therefore continues into t+1 only when d_{t+1} = 0, with d_T := next_done and
V_T := the bootstrap value of s_next.
"""
from __future__ import annotations

import numpy as np


def gae(rewards, values, dones, next_value, next_done, gamma, lam, dtype=np.float64):
    """Generalised advantage estimation (the estimator J^CLIP's advantage refers to, Appendix A;
    computed in Algorithm 1's learning phase).

    delta_t = r_t + gamma (1 - d_{t+1}) V_{t+1} - V_t
    A_t     = delta_t + gamma lam (1 - d_{t+1}) A_{t+1},  A_T = 0
    R_t     = A_t + V_t
    """
    r = np.asarray(rewards, dtype)
    v = np.asarray(values, dtype)
    T, E = r.shape
    nonterm = 1 - np.concatenate([np.asarray(dones, dtype)[1:], np.asarray(next_done, dtype)[None]], 0)
    v_next = np.concatenate([v[1:], np.asarray(next_value, dtype)[None]], 0)
    adv = np.zeros((T, E), dtype)
    carry = np.zeros(E, dtype)
    for t in range(T - 1, -1, -1):
        delta = r[t] + gamma * nonterm[t] * v_next[t] - v[t]
        carry = delta + gamma * lam * nonterm[t] * carry
        adv[t] = carry
    return adv, adv + v


def vtrace(behav_logp, target_logp, rewards, values, dones, bootstrap_value, next_done,
           gamma, lam=1.0, rho_bar=1.0, c_bar=1.0, pg_rho_bar=1.0, dtype=np.float64):
    """V-trace value targets and policy-gradient advantages (Appendix B defers to rlax's
    ``vtrace_td_error_and_advantage``; definition of Espeholt et al. 2018, Sec. 4.1).

    is_t     = exp(log pi(a_t|s_t) - log mu(a_t|s_t))
    gamma_t  = gamma (1 - d_{t+1})
    rho_t    = min(rho_bar, is_t);  c_t = lam * min(c_bar, is_t)
    delta_t  = rho_t (r_t + gamma_t V_{t+1} - V_t)
    v_t      = V_t + delta_t + gamma_t c_t (v_{t+1} - V_{t+1}),  v_T = V_T
    q_t      = r_t + gamma_t (lam v_{t+1} + (1 - lam) V_{t+1})
    pg_adv_t = min(pg_rho_bar, is_t) (q_t - V_t)
    """
    mu = np.asarray(behav_logp, dtype)
    pi = np.asarray(target_logp, dtype)
    r = np.asarray(rewards, dtype)
    v = np.asarray(values, dtype)
    T, E = r.shape
    disc = gamma * (1 - np.concatenate([np.asarray(dones, dtype)[1:],
                                        np.asarray(next_done, dtype)[None]], 0))
    v_next = np.concatenate([v[1:], np.asarray(bootstrap_value, dtype)[None]], 0)
    ratio = np.exp(pi - mu)
    rho = np.minimum(rho_bar, ratio)
    c = lam * np.minimum(c_bar, ratio)
    delta = rho * (r + disc * v_next - v)
    vs_minus_v = np.zeros((T, E), dtype)
    carry = np.zeros(E, dtype)
    for t in range(T - 1, -1, -1):
        carry = delta[t] + disc[t] * c[t] * carry
        vs_minus_v[t] = carry
    vs = vs_minus_v + v
    vs_next = np.concatenate([vs[1:], np.asarray(bootstrap_value, dtype)[None]], 0)
    q = r + disc * (lam * vs_next + (1 - lam) * v_next)
    pg_adv = np.minimum(pg_rho_bar, ratio) * (q - v)
    return vs, pg_adv
