"""The allocation-free Adam entry point (adam_step_noalloc) against adam_step: the same kernels,
so the same parameters, moments and statistics bit for bit, on two calls in a row, the second
on a smaller buffer (its norm partials are fewer; none of the first call's may leak in)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

from tests import gpu_util as G  # noqa: E402

P = pytest.importorskip("paper_2310_00036_amd")


def _inputs(n, seed, scale):
    rng = np.random.default_rng(seed)
    return dict(p=rng.standard_normal(n).astype(np.float32),
                g=(rng.standard_normal(n) * scale / np.sqrt(n) * 30).astype(np.float32),
                m=(rng.standard_normal(n) * 1e-3).astype(np.float32),
                v=(rng.random(n) * 1e-5).astype(np.float32))


def _run(fn, b, step, max_norm):
    torch = G.torch()
    n = b["p"].size
    dp, dg, dm, dv = (G.dev_f32(b[k]) for k in ("p", "g", "m", "v"))
    st = torch.full((2,), -1.0, dtype=torch.float32, device="cuda:0")
    if fn == "ws":
        ws = G.ws_bytes(P.adam_workspace_bytes(n))
        P.adam_step(n, dp, dg, dm, dv, step, 2.5e-4, 0.9, 0.999, 1e-5, max_norm, st, ws)
    else:
        P.adam_step_noalloc(n, dp, dg, dm, dv, step, 2.5e-4, 0.9, 0.999, 1e-5, max_norm, st)
    G.sync()
    return [t.cpu().numpy() for t in (dp, dm, dv, st)]


def test_noalloc_adam_equals_adam_step_twice():
    calls = [(4_364_211, 11, 10.0, 3, 0.5),    # the wide net's parameters, clip active
             (1_001, 12, 1.0, 1, 40.0)]        # then a much smaller buffer, clip inactive
    for n, seed, scale, step, max_norm in calls:
        b = _inputs(n, seed, scale)
        want = _run("ws", b, step, max_norm)
        got = _run("noalloc", b, step, max_norm)
        for g, w, what in zip(got, want, ("params", "m", "v", "stats")):
            assert np.array_equal(g.view(np.uint32), w.view(np.uint32)), (n, what)
        assert got[3][1] == 0 and got[3][0] > 0
