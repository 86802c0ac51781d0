"""Cleanba's actor-learner pipeline on the GPU (Section 4.2, Table 1): impala_actor_step on the
actor's stream and learner_step on the learner's, overlapping. The run equals, bit for bit,
the one-thread replay of the same composition, with or without delays that change which
thread waits."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

P = pytest.importorskip("paper_2310_00036_amd")
from paper_2310_00036_amd import pipeline as PL  # noqa: E402
from synth import NetShape, Workload, draw_params  # noqa: E402

WLS = {
    "ppo": Workload("pipe_ppo", "ppo", T=8, E=4, net=NetShape(num_actions=6), epochs=2, num_minibatches=2, seed=3),
    "impala": Workload("pipe_impala", "impala", T=5, E=4, net=NetShape(num_actions=6), num_minibatches=2, lam=1.0,
                       lr=6e-4, max_grad_norm=40.0, optimizer="rmsprop", seed=4),
}


def _agent(wl):
    return PL.LibraryAgent(wl, P.PREC_BF16, draw_params(wl.net, wl.seed))


@pytest.mark.parametrize("algo", ["ppo", "impala"])
def test_pipeline_equals_sequential_replay(algo):
    torch = pytest.importorskip("torch")
    wl = WLS[algo]
    iters = 5
    p_ref, ref = PL.run_sequential(_agent(wl), wl, iters, seed=9)
    assert [(k, v) for k, v, _ in ref.rollouts] == [(1, 1), (2, 1), (3, 2), (4, 3), (5, 4)]
    for ad, ld in ((None, None), (None, lambda k: 0.05), (lambda k: 0.05, None)):
        p, rec = PL.run_pipeline(_agent(wl), wl, iters, seed=9, actor_delay=ad, learner_delay=ld)
        assert rec.rollouts == ref.rollouts
        assert rec.updates == ref.updates
        assert torch.equal(p, p_ref)
        for x, y in zip(rec.stats, ref.stats):
            np.testing.assert_array_equal(x, y)
        assert np.isfinite(np.concatenate(rec.stats)).all()
    assert not torch.equal(p_ref, torch.as_tensor(draw_params(wl.net, wl.seed)).to(p_ref.device))
