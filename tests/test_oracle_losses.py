"""Pins of the PPO / IMPALA losses, Adam, clipping and the batch nomenclature."""
import json
import os

import numpy as np
import pytest

from oracle import cfg as ocfg, losses, optim

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _batch(m, A, seed):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((m, A)) * 2
    a = rng.integers(0, A, m)
    lp = losses.log_softmax(z)[np.arange(m), a]
    return dict(z=z, v=rng.standard_normal(m), a=a, old=lp + 0.15 * rng.standard_normal(m),
                adv=rng.standard_normal(m) * 3 + 0.4, ret=rng.standard_normal(m),
                vs=rng.standard_normal(m), pg=rng.standard_normal(m))


def _fd(f, x, h=1e-6):
    g = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        g[idx] = (f(xp) - f(xm)) / (2 * h)
    return g


def test_ppo_grad_matches_finite_differences():
    b = _batch(16, 5, 0)
    st = (b["adv"].mean(), b["adv"].std())

    def L(z, v):
        return losses.ppo_loss_grad(z, v, b["a"], b["old"], b["adv"], b["ret"], 0.1, 0.5, 0.01,
                                    True, adv_stats=st)[0]
    _, dz, dv, stats = losses.ppo_loss_grad(b["z"], b["v"], b["a"], b["old"], b["adv"], b["ret"],
                                            0.1, 0.5, 0.01, True)
    assert 0 < stats[5] < 1, "the batch should exercise both clipped and unclipped rows"
    np.testing.assert_allclose(dz, _fd(lambda z: L(z, b["v"]), b["z"]), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(dv, _fd(lambda v: L(b["z"], v), b["v"]), rtol=1e-6, atol=1e-9)


def test_impala_grad_matches_finite_differences():
    b = _batch(12, 4, 1)

    def L(z, v):
        return losses.impala_loss_grad(z, v, b["a"], b["vs"], b["pg"], 1.0, 0.5, 0.01)[0]
    _, dz, dv, _ = losses.impala_loss_grad(b["z"], b["v"], b["a"], b["vs"], b["pg"], 1.0, 0.5, 0.01)
    np.testing.assert_allclose(dz, _fd(lambda z: L(z, b["v"]), b["z"]), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(dv, _fd(lambda v: L(b["z"], v), b["v"]), rtol=1e-6, atol=1e-9)


def test_logit_grads_sum_to_zero_per_row():
    b = _batch(20, 7, 2)
    _, dz, _, _ = losses.ppo_loss_grad(b["z"], b["v"], b["a"], b["old"], b["adv"], b["ret"],
                                       0.2, 0.5, 0.05, True)
    np.testing.assert_allclose(dz.sum(1), 0, atol=1e-15)
    _, dz, _, _ = losses.impala_loss_grad(b["z"], b["v"], b["a"], b["vs"], b["pg"], 1.0, 0.5, 0.05)
    np.testing.assert_allclose(dz.sum(1), 0, atol=1e-15)


def test_uniform_logits_entropy_is_log_A():
    m, A = 5, 18
    z = np.full((m, A), 0.37)
    _, _, _, st = losses.impala_loss_grad(z, np.zeros(m), np.zeros(m, int), np.zeros(m),
                                          np.zeros(m), 1.0, 0.5, 0.01)
    assert np.isclose(st[3], np.log(A), rtol=1e-14)


def test_on_policy_ratio_is_normalised_reinforce():
    """old_logp = current log-prob gives r = 1: the clip is inactive and the policy term is
    -mean(A_hat); its logit gradient is -(1/m) A_hat (onehot - p)."""
    b = _batch(10, 4, 3)
    m, A = b["z"].shape
    lp = losses.log_softmax(b["z"])
    old = lp[np.arange(m), b["a"]]
    L, dz, _, st = losses.ppo_loss_grad(b["z"], b["v"], b["a"], old, b["adv"], b["ret"], 0.1, 0.0,
                                        0.0, True)
    ahat = (b["adv"] - b["adv"].mean()) / (b["adv"].std() + 1e-8)
    assert np.isclose(st[1], -ahat.mean(), atol=1e-15)
    onehot = np.eye(A)[b["a"]]
    np.testing.assert_allclose(dz, -(ahat[:, None] * (onehot - np.exp(lp))) / m, atol=1e-15)
    assert st[5] == 0 and abs(st[4]) < 1e-15


def test_ppo_hand_worked_example():
    """Two rows, two actions, worked by hand (tests/golden/ppo_m2.json)."""
    with open(os.path.join(GOLDEN, "ppo_m2.json")) as f:
        g = json.load(f)
    i = g["inputs"]
    L, dz, dv, st = losses.ppo_loss_grad(np.array(i["z"]), np.array(i["v"]), np.array(i["a"]),
                                         np.array(i["old_logp"]), np.array(i["adv"]),
                                         np.array(i["ret"]), i["clip"], i["vf"], i["ent"],
                                         bool(i["norm_adv"]))
    e = g["expect"]
    assert np.isclose(L, e["loss"], rtol=1e-12)
    np.testing.assert_allclose(dz, e["dlogits"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dv, e["dvalue"], rtol=1e-12)


def test_adam_first_step_closed_form():
    rng = np.random.default_rng(4)
    p, g = rng.standard_normal(50), rng.standard_normal(50)
    p1, m1, v1 = optim.adam(p, g, np.zeros(50), np.zeros(50), 1, 2.5e-4, eps=1e-5)
    np.testing.assert_allclose(p1 - p, -2.5e-4 * g / (np.abs(g) + 1e-5), rtol=1e-12)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-14)
    np.testing.assert_allclose(v1, 0.001 * g * g, rtol=1e-14)


def test_adam_second_step_by_hand():
    # g1 = 1, g2 = -1, lr = 1, eps = 0: m2 = 0.9*0.1 - 0.1 = -0.01, v2 = 0.999*0.001 + 0.001
    p, m, v = optim.adam(np.array([0.0]), np.array([1.0]), np.zeros(1), np.zeros(1), 1, 1.0, eps=0.0)
    p, m, v = optim.adam(p, np.array([-1.0]), m, v, 2, 1.0, eps=0.0)
    mhat = -0.01 / (1 - 0.81)
    vhat = (0.999 * 0.001 + 0.001) / (1 - 0.999 ** 2)
    assert np.isclose(p[0], -1.0 - mhat / np.sqrt(vhat), rtol=1e-14)


def test_rmsprop_first_step_by_hand():
    # Appendix B's IMPALA values (decay 0.99, eps 0.01), g = 3, lr = 1, nu0 = 0:
    # nu = 0.01 * 9 = 0.09; step = 3 / sqrt(0.09 + 0.01) = 3 / sqrt(0.1) = 9.486832980505138
    # (epsilon outside the root would give 3 / 0.31 = 9.677...)
    p, nu = optim.rmsprop(np.array([0.0]), np.array([3.0]), np.zeros(1), 1.0, 0.99, 0.01)
    assert np.isclose(nu[0], 0.09, rtol=1e-14)
    assert np.isclose(p[0], -9.486832980505138, rtol=1e-14)


def test_rmsprop_constant_gradient_closed_form():
    # with a constant gradient from nu0 = 0 the recurrence sums a geometric series:
    # nu_t = (1 - decay^t) g^2, so the t-th step is g / sqrt((1 - decay^t) g^2 + eps)
    rng = np.random.default_rng(8)
    g = rng.standard_normal(40) * 3
    p0 = rng.standard_normal(40)
    p, nu = p0.copy(), np.zeros(40)
    lr, decay, eps = 6e-4, 0.99, 0.01
    for _ in range(25):
        p, nu = optim.rmsprop(p, g, nu, lr, decay, eps)
    np.testing.assert_allclose(nu, (1 - decay ** 25) * g * g, rtol=1e-12)
    want = p0 - lr * sum(g / np.sqrt((1 - decay ** t) * g * g + eps) for t in range(1, 26))
    np.testing.assert_allclose(p, want, rtol=1e-12, atol=1e-15)


def test_rmsprop_without_decay_or_eps_steps_by_the_sign():
    # decay 0, eps 0: nu = g^2 and the step is lr * g / |g| = lr * sign(g)
    g = np.array([-2.5, 0.125, 7.0, -1e-3])
    p, _ = optim.rmsprop(np.zeros(4), g, np.full(4, 5.0), 0.1, 0.0, 0.0)
    np.testing.assert_allclose(p, -0.1 * np.sign(g), rtol=1e-15)


@pytest.mark.parametrize("scale,max_norm", [(0.1, 0.5), (10.0, 0.5), (3.0, 40.0), (100.0, 40.0), (5.0, 0.0)])
def test_clip_norm_is_min_of_norm_and_threshold(scale, max_norm):
    g = np.random.default_rng(5).standard_normal(1000) * scale
    n = np.linalg.norm(g)
    gc, n0 = optim.clip_by_global_norm(g, max_norm)
    assert np.isclose(n0, n)
    want = min(n, max_norm) if max_norm > 0 else n
    assert np.isclose(np.linalg.norm(gc), want, rtol=1e-12)
    assert np.allclose(gc / np.linalg.norm(gc), g / n)


def test_batch_nomenclature_matches_paper_examples():
    with open(os.path.join(GOLDEN, "cfg_examples.json")) as f:
        g = json.load(f)
    for case in g["cases"]:
        got = ocfg.derive(**case["inputs"])
        for k, v in case["expect"].items():
            assert got[k] == v, (case["source"], k, got[k], v)


def test_gumbel_max_ties_go_to_lowest_index():
    z = np.array([[0.0, 1.0, 1.0, 0.5], [2.0, 2.0, 2.0, 2.0]])
    a, lp = losses.gumbel_max(z, np.zeros_like(z))
    assert list(a) == [1, 0]
    assert np.isclose(lp[1], -np.log(4))
