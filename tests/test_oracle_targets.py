"""Pins of GAE and V-trace against closed forms and explicit (non-recursive) sums."""
import json
import os

import numpy as np
import pytest

from oracle import targets

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rollout(T, E, seed, done_p=0.2):
    rng = np.random.default_rng(seed)
    return dict(r=rng.choice([-1.0, 0.0, 1.0], size=(T, E), p=[.2, .6, .2]),
                v=rng.standard_normal((T, E)), d=(rng.random((T, E)) < done_p).astype(np.uint8),
                nv=rng.standard_normal(E), nd=(rng.random(E) < done_p).astype(np.uint8))


def _discounted_return(ro, gamma):
    """Explicit sum: R_t = sum_k gamma^k r_{t+k} up to the episode end, plus gamma^n V_T if
    the rollout ends first (d_{t+1} = 1 means the transition at t ended the episode)."""
    T, E = ro["r"].shape
    d_next = np.concatenate([ro["d"][1:], ro["nd"][None]], 0)
    R = np.zeros((T, E))
    for e in range(E):
        for t in range(T):
            total, disc, k = 0.0, 1.0, t
            while True:
                total += disc * ro["r"][k, e]
                if d_next[k, e]:
                    break
                disc *= gamma
                k += 1
                if k == T:
                    total += disc * ro["nv"][e]
                    break
            R[t, e] = total
    return R


def test_gae_lambda1_is_discounted_return_minus_value():
    ro = _rollout(9, 5, 0)
    adv, ret = targets.gae(ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.97, 1.0)
    R = _discounted_return(ro, 0.97)
    np.testing.assert_allclose(ret, R, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(adv, R - ro["v"], rtol=1e-12, atol=1e-12)


def test_gae_lambda0_is_td_error():
    ro = _rollout(7, 3, 1)
    adv, _ = targets.gae(ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.9, 0.0)
    d_next = np.concatenate([ro["d"][1:], ro["nd"][None]], 0)
    v_next = np.concatenate([ro["v"][1:], ro["nv"][None]], 0)
    np.testing.assert_allclose(adv, ro["r"] + 0.9 * (1 - d_next) * v_next - ro["v"], atol=1e-14)


def test_gae_all_done_is_reward_minus_value():
    ro = _rollout(6, 4, 2)
    ro["d"][:] = 1
    ro["nd"][:] = 1
    adv, _ = targets.gae(ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.99, 0.95)
    np.testing.assert_allclose(adv, ro["r"] - ro["v"], atol=1e-14)


def test_gae_explicit_lambda_sum():
    """A_t = sum_k (gamma lam)^k delta_{t+k} within the episode (the definition of GAE)."""
    ro = _rollout(8, 3, 3)
    g, lam = 0.99, 0.8
    adv, _ = targets.gae(ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], g, lam)
    d_next = np.concatenate([ro["d"][1:], ro["nd"][None]], 0)
    v_next = np.concatenate([ro["v"][1:], ro["nv"][None]], 0)
    delta = ro["r"] + g * (1 - d_next) * v_next - ro["v"]
    T, E = delta.shape
    for e in range(E):
        for t in range(T):
            s, w = 0.0, 1.0
            for k in range(t, T):
                s += w * delta[k, e]
                if d_next[k, e]:
                    break
                w *= g * lam
            assert np.isclose(adv[t, e], s, rtol=1e-12, atol=1e-12)


def _vtrace_explicit(mu, pi, r, v, d, bv, nd, gamma, lam, rho_bar, c_bar, pg_rho_bar):
    """Espeholt et al. (2018) eq. (1) as an explicit sum over future steps:
    v_s = V_s + sum_{t>=s} (prod_{i=s}^{t-1} gamma_i c_i) rho_t (r_t + gamma_t V_{t+1} - V_t)."""
    T, E = r.shape
    d_next = np.concatenate([d[1:], nd[None]], 0)
    gam = gamma * (1 - d_next)
    vn = np.concatenate([v[1:], bv[None]], 0)
    is_ = np.exp(pi - mu)
    rho = np.minimum(rho_bar, is_)
    c = lam * np.minimum(c_bar, is_)
    vs = np.zeros((T, E))
    for e in range(E):
        for s in range(T):
            acc, w = v[s, e], 1.0
            for t in range(s, T):
                acc += w * rho[t, e] * (r[t, e] + gam[t, e] * vn[t, e] - v[t, e])
                w *= gam[t, e] * c[t, e]
            vs[s, e] = acc
    vsn = np.concatenate([vs[1:], bv[None]], 0)
    pg = np.minimum(pg_rho_bar, is_) * (r + gam * (lam * vsn + (1 - lam) * vn) - v)
    return vs, pg


@pytest.mark.parametrize("lam,rho_bar,c_bar", [(1.0, 1.0, 1.0), (0.9, 1.0, 1.0), (1.0, 0.7, 1.3)])
def test_vtrace_matches_explicit_sum(lam, rho_bar, c_bar):
    ro = _rollout(10, 4, 4)
    rng = np.random.default_rng(5)
    mu = rng.standard_normal((10, 4)) * 0.5 - 1.5
    pi = mu + rng.standard_normal((10, 4)) * 0.4
    vs, pg = targets.vtrace(mu, pi, ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.95, lam,
                            rho_bar, c_bar, 0.8)
    vs2, pg2 = _vtrace_explicit(mu, pi, ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.95, lam,
                                rho_bar, c_bar, 0.8)
    np.testing.assert_allclose(vs, vs2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(pg, pg2, rtol=1e-12, atol=1e-12)


def test_vtrace_on_policy_equals_gae_lambda1():
    """With mu = pi and rho_bar = c_bar = 1, V-trace's target is the n-step bootstrapped
    return and its advantage is GAE(lambda=1)'s."""
    ro = _rollout(12, 6, 6)
    lp = np.random.default_rng(6).standard_normal((12, 6))
    vs, pg = targets.vtrace(lp, lp, ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.99)
    adv, ret = targets.gae(ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.99, 1.0)
    np.testing.assert_allclose(vs, ret, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(pg, adv, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(vs, _discounted_return(ro, 0.99), rtol=1e-12, atol=1e-12)


def test_vtrace_no_trace_is_one_step_clipped_td():
    ro = _rollout(5, 3, 7)
    rng = np.random.default_rng(7)
    mu, pi = rng.standard_normal((5, 3)), rng.standard_normal((5, 3))
    vs, _ = targets.vtrace(mu, pi, ro["r"], ro["v"], ro["d"], ro["nv"], ro["nd"], 0.9, c_bar=0.0)
    d_next = np.concatenate([ro["d"][1:], ro["nd"][None]], 0)
    vn = np.concatenate([ro["v"][1:], ro["nv"][None]], 0)
    rho = np.minimum(1.0, np.exp(pi - mu))
    np.testing.assert_allclose(vs, ro["v"] + rho * (ro["r"] + 0.9 * (1 - d_next) * vn - ro["v"]),
                               atol=1e-14)


def test_vtrace_hand_worked_example():
    """T=2, E=1 cases worked by hand (tests/golden/vtrace_t2.json)."""
    with open(os.path.join(GOLDEN, "vtrace_t2.json")) as f:
        cases = json.load(f)["cases"]
    for g in cases:
        i = g["inputs"]
        vs, pg = targets.vtrace(np.array(i["mu"]), np.array(i["pi"]), np.array(i["r"]),
                                np.array(i["v"]), np.array(i["d"], np.uint8), np.array(i["bv"]),
                                np.array(i["nd"], np.uint8), i["gamma"], i["lam"], i["rho_bar"],
                                i["c_bar"], i["pg_rho_bar"])
        np.testing.assert_allclose(vs.ravel(), g["expect"]["vs"], rtol=1e-12)
        np.testing.assert_allclose(pg.ravel(), g["expect"]["pg_adv"], rtol=1e-12)
