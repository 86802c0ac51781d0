"""Cleanba's actor-learner composition (Section 4.2, Table 1): which policy version collects
each rollout and which rollout each update consumes, independent of thread timing. These CPU
tests drive the pipeline with a small host-side stand-in agent (a linear policy stepped by a
deterministic rule) so that only the queues and the two loops are under test."""
import hashlib

import numpy as np
import pytest

P = pytest.importorskip("paper_2310_00036_amd")
from paper_2310_00036_amd import pipeline as PL  # noqa: E402
from synth import NetShape, Workload  # noqa: E402


class HostAgent:
    """Linear policy over the mean of each frame channel; learn() moves the parameters by a
    deterministic function of the rollout, so every later rollout depends on every earlier
    update."""

    def __init__(self, A):
        self.A = A
        self.p = np.linspace(-1, 1, 4 * A + 4).astype(np.float64)

    def snapshot(self):
        return self.p.copy()

    def act(self, params, obs, gumbel):
        f = obs.reshape(obs.shape[0], -1, obs.shape[-1]).mean(1) / 255.0
        z = f @ params[:4 * self.A].reshape(4, self.A)
        a = np.argmax(z + gumbel, axis=1).astype(np.int32)
        lz = z - np.log(np.exp(z - z.max(1, keepdims=True)).sum(1, keepdims=True)) - z.max(1, keepdims=True)
        v = f @ params[4 * self.A:]
        return a, lz[np.arange(len(a)), a].astype(np.float32), v.astype(np.float32)

    def learn(self, ro):
        h = int(hashlib.sha256(ro.obs.tobytes() + ro.actions.tobytes()).hexdigest()[:8], 16)
        self.p = self.p + 1e-3 * np.sin(np.arange(self.p.size) + h % 1000) + 1e-2 * ro.rewards.mean()
        return np.array([[ro.rewards.sum(), float(ro.index)]])


def _wl(algo="ppo"):
    net = NetShape(in_h=6, in_w=5, ch=(16, 16, 16), hidden=8, num_actions=3)
    return Workload("pipe", algo, T=5, E=3, net=net, seed=2)


def _same(a, b):
    (pa, ra), (pb, rb) = a, b
    assert ra.rollouts == rb.rollouts
    assert ra.updates == rb.updates
    np.testing.assert_array_equal(pa, pb)
    for x, y in zip(ra.stats, rb.stats):
        np.testing.assert_array_equal(x, y)


def test_composition_follows_table_1():
    """Rollouts 1 and 2 come from pi_1, rollout k >= 3 from pi_{k-1}; update k consumes rollout
    k and produces pi_{k+1} (from iteration 3 on the learner trains on the second latest
    policy's data)."""
    wl = _wl()
    _, rec = PL.run_pipeline(HostAgent(3), wl, 6, seed=1)
    assert [(k, v) for k, v, _ in rec.rollouts] == [(1, 1), (2, 1), (3, 2), (4, 3), (5, 4), (6, 5)]
    assert rec.updates == [(k, k, k + 1) for k in range(1, 7)]


@pytest.mark.parametrize("algo", ["ppo", "impala"])
def test_composition_does_not_depend_on_timing(algo):
    """Slow actor, slow learner, or randomly jittered: the same rollouts (bit for bit), the same
    updates and the same final parameters as the one-thread replay of the composition."""
    wl = _wl(algo)
    ref = PL.run_sequential(HostAgent(3), wl, 5, seed=4)
    jit = np.random.default_rng(0).random(16) * 0.02
    for ad, ld in ((lambda k: 0.03, None), (None, lambda k: 0.03), (lambda k: jit[k], lambda k: jit[k + 5])):
        _same(PL.run_pipeline(HostAgent(3), wl, 5, seed=4, actor_delay=ad, learner_delay=ld), ref)


def test_rollouts_depend_on_the_policy_and_the_seed():
    """The stand-in environments respond to the actions: a different policy version, or a
    different seed, changes the data (so the composition test above is not vacuous)."""
    wl = _wl()
    a = PL.run_sequential(HostAgent(3), wl, 4, seed=4)[1].rollouts
    b = PL.run_sequential(HostAgent(3), wl, 4, seed=5)[1].rollouts
    assert all(x[2] != y[2] for x, y in zip(a, b))
    agent = HostAgent(3)
    agent.p = agent.p[::-1].copy()
    c = PL.run_sequential(agent, wl, 4, seed=4)[1].rollouts
    assert a[0][2] != c[0][2]


def test_environment_stacks_frames_and_marks_episode_starts():
    net = NetShape(in_h=4, in_w=3, ch=(16, 16, 16), hidden=8, num_actions=3)
    env = PL.SyntheticAtari(2, net, seed=3, done_prob=0.3)
    assert env.done.tolist() == [1, 1]
    prev = env.obs.copy()
    for _ in range(20):
        obs, r, d = env.step(np.array([0, 1]))
        for e in range(2):
            if d[e]:
                assert (obs[e] == obs[e, :, :, :1]).all()      # a fresh episode: one frame stacked
            else:
                np.testing.assert_array_equal(obs[e, :, :, :-1], prev[e, :, :, 1:])
        assert set(np.unique(r)) <= {-1.0, 0.0, 1.0}
        prev = obs


def test_a_failing_learner_stops_the_actor():
    class Broken(HostAgent):
        def learn(self, ro):
            raise RuntimeError("learner failed")
    with pytest.raises(RuntimeError, match="learner failed"):
        PL.run_pipeline(Broken(3), _wl(), 6, seed=1, timeout=30)
