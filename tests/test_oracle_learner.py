"""Learner-level pins of the oracle: data-parallel equivalence, determinism, resume, bf16 floor."""
import hashlib

import numpy as np
import pytest

from oracle import learner, losses, net as onet, optim
from synth import WORKLOADS, NetShape, draw_params, draw_rollout


def test_option1_equals_option2_gradient_average(tiny_net):
    """Appendix A: two copies each averaging over half the minibatch, with their gradients
    averaged, give the single-copy gradient of the whole minibatch (advantage statistics
    taken over the whole minibatch)."""
    net = tiny_net
    rng = np.random.default_rng(0)
    flat = draw_params(net, 3).astype(np.float64)
    m = 8
    obs = rng.integers(0, 256, size=(m, net.in_h, net.in_w, net.in_c), dtype=np.uint8)
    a = rng.integers(0, net.num_actions, m)
    adv, ret = rng.standard_normal(m), rng.standard_normal(m)
    z, v, cache = onet.forward(net, flat, obs)
    old = losses.log_softmax(z)[np.arange(m), a] + 0.2 * rng.standard_normal(m)
    st = (adv.mean(), adv.std())

    def grad(rows):
        zz, vv, cc = onet.forward(net, flat, obs[rows])
        _, dz, dv, _ = losses.ppo_loss_grad(zz, vv, a[rows], old[rows], adv[rows], ret[rows],
                                            0.1, 0.5, 0.01, True, adv_stats=st)
        return onet.backward(net, cc, dz, dv)
    full = grad(np.arange(m))
    shards = 0.5 * (grad(np.arange(0, m // 2)) + grad(np.arange(m // 2, m)))
    np.testing.assert_allclose(shards, full, rtol=1e-10, atol=1e-14)


def test_synthetic_inputs_are_deterministic():
    wl = WORKLOADS[0]
    h = [hashlib.sha256(b"".join(np.ascontiguousarray(v).tobytes() for v in draw_rollout(wl).values())).hexdigest()
         for _ in range(2)]
    assert h[0] == h[1]
    p1, p2 = draw_params(wl.net, wl.seed), draw_params(wl.net, wl.seed)
    assert p1.tobytes() == p2.tobytes()
    ro = draw_rollout(wl)
    assert ro["obs"].shape == (9, 4, 84, 84, 4) and ro["obs"].dtype == np.uint8
    assert set(np.unique(ro["rewards"])) <= {-1.0, 0.0, 1.0}
    assert sorted(ro["perm"][0]) == list(range(32))


def _tiny_workload(net):
    from synth import Workload
    return Workload("tiny", "ppo", T=4, E=3, net=net, epochs=2, num_minibatches=2, seed=9)


def test_ppo_learner_resume_is_exact(tiny_net):
    """State is (params, m, v, step): two learning phases in a row equal one phase, a save and
    reload of that state, then the second phase."""
    wl = _tiny_workload(tiny_net)
    p0 = draw_params(wl.net, 1).astype(np.float64)
    raw = draw_rollout(wl)
    ro = learner.behaviour_rollout(wl, p0, raw)
    z = np.zeros_like(p0)
    a = learner.ppo_learner_step(wl.net, wl, ro, p0, z, z, 0, raw["perm"])
    b = learner.ppo_learner_step(wl.net, wl, ro, *a[:4], raw["perm"])
    saved = [np.array(x, copy=True) for x in a[:3]]
    c = learner.ppo_learner_step(wl.net, wl, ro, *saved, a[3], raw["perm"])
    assert b[3] == c[3] == 8
    for x, y in zip(b[:3], c[:3]):
        np.testing.assert_array_equal(x, y)
    assert np.all(np.isfinite(b[4]))


def test_impala_learner_runs_and_moves_params(tiny_net):
    from synth import Workload
    wl = Workload("tiny_impala", "impala", T=5, E=2, net=tiny_net, lam=1.0, lr=6e-4,
                  max_grad_norm=40.0, behav_logp_noise=0.0, behav_logit_noise=0.3, seed=4)
    p0 = draw_params(wl.net, 2).astype(np.float64)
    raw = draw_rollout(wl)
    ro = learner.behaviour_rollout(wl, p0, raw)
    z = np.zeros_like(p0)
    p1, m1, v1, step, stats = learner.impala_learner_step(wl.net, wl, ro, p0, z, z, 0)
    assert step == 1 and stats.shape == (1, 8) and np.all(np.isfinite(stats))
    # First Adam step moves every parameter with a non-zero gradient by about lr.
    moved = np.abs(p1 - p0)
    assert moved.max() <= 6e-4 * 1.0001


def test_impala_minibatches_are_env_blocks_in_order(tiny_net):
    """N IMPALA minibatches are N updates on the env blocks of the rollout, one after the
    other: equal to single-minibatch learner steps on each block's own sub-rollout (its
    trajectories and bootstrap frames), chained through params and optimiser state."""
    from synth import Workload
    wl = Workload("tiny_impala_mb", "impala", T=4, E=4, net=tiny_net, num_minibatches=2, lam=1.0,
                  lr=6e-4, max_grad_norm=40.0, optimizer="rmsprop", behav_logp_noise=0.0,
                  behav_logit_noise=0.3, seed=9)
    p0 = draw_params(wl.net, 5).astype(np.float64)
    raw = draw_rollout(wl)
    ro = learner.behaviour_rollout(wl, p0, raw)
    z = np.zeros_like(p0)
    got = learner.impala_learner_step(wl.net, wl, ro, p0, z, z, 0)
    T, E, Eb = wl.T, wl.E, 2
    state = (p0, z, z, 0)
    rows_all = []
    for k in range(2):
        envs = np.arange(k * Eb, (k + 1) * Eb)
        rows = (np.arange(T + 1)[:, None] * E + envs[None, :]).ravel()
        sub = dict(obs=ro["obs"][rows], actions=ro["actions"][rows[:T * Eb]], logp=ro["logp"][rows[:T * Eb]],
                   rewards=ro["rewards"][:, envs], dones=ro["dones"][:, envs], next_done=ro["next_done"][envs])
        out = learner.impala_learner_step(wl.net, wl.replace(E=Eb, num_minibatches=1), sub, *state)
        state = out[:4]
        rows_all.append(out[4])
    assert got[3] == state[3] == 2
    for x, y in zip(got[:3], state[:3]):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(got[4], np.concatenate(rows_all))


def test_bf16_emulation_floor_on_tiny_ppo_batch():
    """Measure the intrinsic bf16 error floor (bf16-emulating oracle vs float64 oracle) on 8
    Atari-shaped frames with the full-size network. Parity unpinned against the paper.

    Finding: the forward logits stay within 1e-2, and the head/dense gradients within 2e-2,
    but trunk conv gradients sit at 4-17% because a bf16-sized perturbation of the forward
    flips max-pool argmax and ReLU decisions, and the wgrad sums cancel heavily. The bound
    below guards that finding; the per-kernel bf16 tests carry the tight parity.
    """
    net = NetShape(num_actions=6)
    p = draw_params(net, 0)
    rng = np.random.default_rng(1)
    n = 8
    obs = rng.integers(0, 256, size=(n, 84, 84, 4), dtype=np.uint8)
    a = rng.integers(0, 6, n)
    z64, v64, c64 = onet.forward(net, p, obs, "fp64")
    zb, vb, cb = onet.forward(net, p, obs, "bf16")
    assert np.linalg.norm(zb - z64) / np.linalg.norm(z64) < 1e-2
    old = losses.log_softmax(z64)[np.arange(n), a] + 0.05 * rng.standard_normal(n)
    adv, ret = rng.standard_normal(n), rng.standard_normal(n)
    _, dz, dv, _ = losses.ppo_loss_grad(z64, v64, a, old, adv, ret, 0.1, 0.5, 0.01)
    g64 = onet.backward(net, c64, dz, dv)
    gb = onet.backward(net, cb, dz, dv)
    errs = {}
    for name, shape, off in onet.param_layout(net):
        sl = slice(off, off + int(np.prod(shape)))
        errs[name] = np.linalg.norm(gb[sl] - g64[sl]) / np.linalg.norm(g64[sl])
    for name in ("logits.w", "logits.b", "value.w", "value.b"):
        assert errs[name] < 2e-2, (name, errs[name])
    assert max(errs.values()) < 0.3, errs
