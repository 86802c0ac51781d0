"""Decision-forced parity of the network's backward pass, at the workload shapes, and of
whole updates chained from the oracle's state.

Max-pool argmaxes and ReLU masks are discontinuous decisions. Two correct evaluations that
round differently take some of them differently: in bf16 about 1% of the max-pool routings
differ between any two evaluations of the 84x84 network, and a gradient routed to another
cell moves a trunk weight gradient by several percent (4-17% per tensor on 8 frames). No
free-running bf16 backward pass can therefore be compared with another to the 2e-2 bound.

These tests evaluate the GPU backward pass at the oracle's decisions instead. The oracle runs
the forward pass (bf16-emulating for the bf16 path, float64 for the float32 mode); its saved
activations and max-pool argmaxes are written into the workspace of a GPU training forward
at the places impala_activation_layout() names; impala_cnn_bwd then differentiates the network
at exactly the oracle's activations and decisions. Its gradient is compared tensor by tensor
with the oracle's backward pass over the same activations: relative L2 within 2e-2 per tensor
for bf16 and 1e-4 for float32, plus a small share of the whole gradient's norm for tensors
whose own gradient is below the arithmetic's resolution. Data flow one way only: oracle
values go into the GPU workspace; nothing the GPU computes enters the oracle. The GPU's own
forward outputs are checked against the oracle's in the same tests.

Sizes: the tiny PPO batch (32 frames, 6 actions), the 2048-frame PPO minibatch and the
IMPALA batch of 64 envs x 20 steps plus 64 bootstrap frames with every row carrying gradient;
the wide net's 8192-frame minibatch and the float32 mode at full sizes with the upstream
gradient on sampled rows (the backward is then that of those rows alone, and every other
frame contributes exact zeros).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

from oracle import learner as olearner, losses as olosses, net as onet, optim as ooptim  # noqa: E402
from oracle import targets as otargets  # noqa: E402
from synth import NetShape, WORKLOADS, draw_params, draw_rollout  # noqa: E402
from tests import gpu_util as G  # noqa: E402

P = pytest.importorskip("paper_2310_00036_amd")

PNAME = {G.BF16: "bf16", G.FP32: "fp32"}
TOL = {G.BF16: 2e-2, G.FP32: 1e-4}          # relative L2 per parameter tensor
SLACK = {G.BF16: 2.0 ** -12, G.FP32: 2.0 ** -20}   # share of the whole gradient's norm
OUT_TOL = {G.BF16: 2e-2, G.FP32: 1e-4}      # forward logits / values
MODE = {G.BF16: "bf16", G.FP32: "fp64"}     # oracle mode each GPU precision is compared with
CHUNK = 128


def f32(x):
    """A hyperparameter as the library receives it (float32), for the oracle's side."""
    return float(np.float32(x))


# ----------------------------------------------------------------------------- oracle side


def _oracle_forward(net, params, frames, mode):
    """Oracle forward in frame chunks (independent frames), one chunk after another (numpy's
    BLAS is not called from several threads: concurrent calls have returned wrong rows);
    returns logits, values and the per-chunk caches with their frame slices."""
    n = frames.shape[0]
    chunks = [slice(i, min(i + CHUNK, n)) for i in range(0, n, CHUNK)]
    outs = [onet.forward(net, params, frames[sl], mode) for sl in chunks]
    z = np.concatenate([o[0] for o in outs])
    v = np.concatenate([o[1] for o in outs])
    return z, v, list(zip(chunks, [o[2] for o in outs]))


def _oracle_backward(net, fc, dz, dv):
    """Sum over the chunks of the oracle's backward pass (float64 sum of the chunk gradients)."""
    gs = [onet.backward(net, c, dz[sl], dv[sl]) for sl, c in fc]
    return np.sum([g.astype(np.float64) for g in gs], axis=0)


def _saved(cache, name):
    """The oracle cache's array for one workspace region (None: not read by the backward)."""
    if name == "h":
        return cache["h"]
    st, key = name.split(".")
    s = int(st[1:])
    if key == "conv":
        return None
    if key == "arg":
        return cache[f"s{s}"][1]
    if key == "x2":
        return cache[f"s{s + 1}"][0] if s < 2 else cache["last"]
    blk = cache[f"s{s}.res{int(key[1])}"]
    return blk[0] if key[0] == "x" else blk[1]


# ----------------------------------------------------------------------------- GPU side


def _inject(ws, net, prec, n, fc, positions):
    """Write the oracle's activations and argmaxes of the frames at `positions` (in the order
    of the oracle's frames) into a training forward's workspace."""
    torch = G.torch()
    tdt = {P.DT_U8: torch.uint8, P.DT_BF16: torch.bfloat16, P.DT_F32: torch.float32}
    pos = torch.from_numpy(np.asarray(positions, np.int64)).to("cuda:0")
    written = 0
    for name, off, nbytes, dt, shape in P.impala_activation_layout(net, prec, n):
        parts = [_saved(c, name) for _, c in fc]
        if parts[0] is None:
            continue
        arr = np.concatenate(parts)
        if dt == P.DT_U8:
            assert arr.min() >= 0 and arr.max() <= 8
            host = torch.from_numpy(np.ascontiguousarray(arr.astype(np.uint8)))
        else:
            a32 = np.ascontiguousarray(arr.astype(np.float32))
            if dt == P.DT_BF16:   # the bf16-emulating oracle stores bf16-representable values
                assert np.array_equal(onet.bf16_round(a32), a32), name
            host = torch.from_numpy(a32).to(tdt[dt])
        region = ws[off:off + nbytes].view(tdt[dt]).view(shape)
        region[pos] = host.to("cuda:0")
        written += 1
    assert written == 19


def _gpu_forced(net, prec, params, obs, rows, n, fc, positions, dz, dv):
    """GPU training forward on n frames (obs[rows[i]]), the oracle's activations written over
    the frames at `positions`, then the backward pass with upstream gradient dz, dv on those
    frames (zero elsewhere). Returns (logits, values, grads) as float64 arrays."""
    torch = G.torch()
    A = net.num_actions
    ws = G.ws_bytes(P.impala_workspace_bytes(net, n, prec, 1))
    p = G.dev_f32(params)
    o = G.dev_u8(obs)
    r = G.dev_i32(rows) if rows is not None else None
    logits = torch.empty((n, A), dtype=torch.float32, device="cuda:0")
    value = torch.empty(n, dtype=torch.float32, device="cuda:0")
    P.impala_cnn_fwd(net, prec, p, o, r, n, ws, 1, logits, value)
    _inject(ws, net, prec, n, fc, positions)
    dzf = np.zeros((n, A), np.float32)
    dvf = np.zeros(n, np.float32)
    dzf[positions] = dz
    dvf[positions] = dv
    grads = torch.empty(onet.param_count(net), dtype=torch.float32, device="cuda:0")
    P.impala_cnn_bwd(net, prec, p, o, r, n, ws, G.dev_f32(dzf), G.dev_f32(dvf), grads)
    G.sync()
    return G.host(logits), G.host(value), G.host(grads)


def _check(got, want, net, prec, label):
    """Per tensor: ||got - want|| <= TOL ||want_t|| + SLACK ||want||; prints the errors."""
    gnorm = np.linalg.norm(want)
    errs, bad = {}, {}
    for name, shape, off in onet.param_layout(net):
        sl = slice(off, off + int(np.prod(shape)))
        d, gt = np.linalg.norm(got[sl] - want[sl]), np.linalg.norm(want[sl])
        errs[name] = d / gt if gt > 0 else d
        if d > TOL[prec] * gt + SLACK[prec] * gnorm:
            bad[name] = (float(errs[name]), float(gt / gnorm))
    worst = max(errs, key=errs.get)
    print(f"\n[{label} {PNAME[prec]} forced] worst tensor {errs[worst]:.2e} ({worst}); global "
          f"{G.rel_l2(got, want):.2e}; trunk convs worst "
          f"{max(v for k, v in errs.items() if k.startswith('s')):.2e}", flush=True)
    assert not bad, bad


def _check_outputs(z, v, z_w, v_w, prec):
    """The GPU's own forward outputs against the oracle's: 1e-4 (float32) or 2e-2 (bf16, against
    the bf16 emulation) relative L2 per array, and elementwise scaled to the array's magnitude."""
    for got, want, what in ((z, z_w, "logits"), (v, v_w, "value")):
        print(f"\n[{PNAME[prec]} forward {what}] relative L2 {G.rel_l2(got, want):.2e}; worst |diff| "
              f"{np.abs(np.asarray(got, np.float64) - want).max():.3e} against max |want| "
              f"{np.abs(want).max():.3e}", flush=True)
        G.assert_close(got, want, OUT_TOL[prec], what)


# ----------------------------------------------------------------------------- inputs


def _ppo_minibatch_upstream(wl, z, v, rows, actions, logp, adv, ret):
    """The PPO loss gradient at the oracle's logits and values for the minibatch rows."""
    _, dz, dv, _ = olosses.ppo_loss_grad(z, v, actions[rows], logp[rows], adv[rows], ret[rows], wl.clip_eps,
                                         wl.vf_coef, wl.ent_coef, bool(wl.norm_adv))
    return dz.astype(np.float32), dv.astype(np.float32)


def _synthetic_behaviour(wl, seed):
    """Behaviour data drawn without the network (actions uniform, log-probs near log 1/A,
    values small), for the large shapes whose behaviour forward would dominate the test."""
    rng = np.random.default_rng(seed)
    T, E, A = wl.T, wl.E, wl.net.num_actions
    return dict(actions=rng.integers(0, A, T * E).astype(np.int32),
                logp=(np.log(1.0 / A) + 0.05 * rng.standard_normal(T * E)).astype(np.float32),
                values=(0.1 * rng.standard_normal((T, E))).astype(np.float32),
                next_value=(0.1 * rng.standard_normal(E)).astype(np.float32))


# ----------------------------------------------------------------------------- tests


@pytest.mark.parametrize("prec", [G.BF16, G.FP32], ids=lambda p: PNAME[p])
def test_forced_backward_tiny_ppo_batch(prec):
    """The tiny PPO workload's whole batch (4 envs x 8 steps, 6 actions, behaviour data from
    the initial policy), every row carrying its PPO loss gradient."""
    wl = WORKLOADS[0]
    net = wl.net
    params = draw_params(net, wl.seed)
    raw = draw_rollout(wl)
    ro = olearner.behaviour_rollout(wl, params, raw)
    adv, ret = otargets.gae(ro["rewards"], ro["values"], ro["dones"], ro["next_value"], ro["next_done"],
                            wl.gamma, wl.lam)
    n = wl.batch
    rows = raw["perm"][0, :n]
    z_w, v_w, fc = _oracle_forward(net, params, ro["obs"][rows], MODE[prec])
    dz, dv = _ppo_minibatch_upstream(wl, z_w, v_w, rows, ro["actions"], ro["logp"], adv.ravel(), ret.ravel())
    g_w = _oracle_backward(net, fc, dz, dv)
    z, v, g = _gpu_forced(net, prec, params, ro["obs"], rows, n, fc, np.arange(n), dz, dv)
    _check_outputs(z, v, z_w, v_w, prec)
    _check(g, g_w, net, prec, "ppo 4x8")


def test_forced_backward_ppo_minibatch_2048():
    """The Cleanba-like PPO workload's first minibatch: 2048 rows perm[0, :2048] of the
    64 x 128 rollout gathered in the first conv's load, every row carrying its PPO loss
    gradient (advantages from GAE over the rollout), bf16, in the launch configuration of
    learner_step."""
    wl = WORKLOADS[1]
    net = wl.net
    params = draw_params(net, wl.seed)
    raw = draw_rollout(wl)
    T, E = wl.T, wl.E
    obs = raw["obs"][:T].reshape(T * E, 84, 84, 4)
    b = _synthetic_behaviour(wl, 1)
    adv, ret = otargets.gae(raw["rewards"], b["values"], raw["dones"], b["next_value"], raw["next_done"],
                            wl.gamma, wl.lam)
    rows = raw["perm"][0, :wl.mb]
    z_w, v_w, fc = _oracle_forward(net, params, obs[rows], "bf16")
    dz, dv = _ppo_minibatch_upstream(wl, z_w, v_w, rows, b["actions"], b["logp"], adv.ravel(), ret.ravel())
    g_w = _oracle_backward(net, fc, dz, dv)
    z, v, g = _gpu_forced(net, G.BF16, params, obs, rows, wl.mb, fc, np.arange(wl.mb), dz, dv)
    _check_outputs(z, v, z_w, v_w, G.BF16)
    _check(g, g_w, net, G.BF16, "ppo mb2048")


def _impala_upstream(wl, z, v, actions, behav_logp, rewards, dones, next_done):
    """V-trace from the oracle's logits and values (the bootstrap frames last), then the IMPALA
    loss gradient on the rollout rows; the bootstrap rows get zero."""
    T, E = rewards.shape
    n = T * E
    tlogp = olosses.log_softmax(z[:n])[np.arange(n), actions]
    vs, pg = otargets.vtrace(behav_logp.reshape(T, E), tlogp.reshape(T, E), rewards, v[:n].reshape(T, E),
                             dones, v[n:], next_done, wl.gamma, wl.lam, wl.rho_bar, wl.c_bar, wl.pg_rho_bar)
    _, dz, dv, _ = olosses.impala_loss_grad(z[:n], v[:n], actions, vs.ravel(), pg.ravel(), wl.pg_coef,
                                            wl.vf_coef, wl.ent_coef)
    dzf = np.zeros_like(z)
    dvf = np.zeros_like(v)
    dzf[:n], dvf[:n] = dz, dv
    return dzf.astype(np.float32), dvf.astype(np.float32)


def test_forced_backward_impala_64x20():
    """The IMPALA / V-trace workload: 64 envs x 20 steps plus the 64 bootstrap frames in one
    forward (1344 frames), V-trace from that forward, the IMPALA loss gradient on the 1280
    rollout rows and none on the bootstrap rows; bf16. Behaviour log-probs are drawn without
    the network (log 1/A plus N(0, 0.3) noise, so the rollout is off-policy)."""
    wl = WORKLOADS[2]
    net = wl.net
    T, E, A = wl.T, wl.E, net.num_actions
    n1 = (T + 1) * E
    params = draw_params(net, wl.seed)
    raw = draw_rollout(wl)
    obs = raw["obs"].reshape(n1, 84, 84, 4)
    rng = np.random.default_rng(2)
    actions = rng.integers(0, A, T * E).astype(np.int32)
    behav = (np.log(1.0 / A) + 0.3 * rng.standard_normal(T * E)).astype(np.float32)
    z_w, v_w, fc = _oracle_forward(net, params, obs, "bf16")
    dz, dv = _impala_upstream(wl, z_w, v_w, actions, behav, raw["rewards"], raw["dones"], raw["next_done"])
    g_w = _oracle_backward(net, fc, dz, dv)
    z, v, g = _gpu_forced(net, G.BF16, params, obs, None, n1, fc, np.arange(n1), dz, dv)
    _check_outputs(z, v, z_w, v_w, G.BF16)
    _check(g, g_w, net, G.BF16, "impala 64x20+64")


SAMPLED = {
    # (workload id, precision, frames with upstream gradient)
    "ppo_mb2048_fp32": (1, G.FP32, 24),
    "impala_64x20_fp32": (2, G.FP32, 24),
    "wide_mb8192_bf16": (4, G.BF16, 16),
    "wide_mb8192_fp32": (4, G.FP32, 12),
}


@pytest.mark.parametrize("case", sorted(SAMPLED))
def test_forced_backward_sampled_rows_at_full_size(case):
    """Full launch sizes (2048, 1344 or the wide net's 8192 frames), the upstream gradient on
    frames spread over the launch (first, last and seeded picks), the oracle's activations
    written over those frames."""
    wid, prec, k = SAMPLED[case]
    wl = WORKLOADS[wid]
    net = wl.net
    params = draw_params(net, wl.seed)
    raw = draw_rollout(wl)
    T, E = wl.T, wl.E
    if wl.algo == "ppo":
        obs = raw["obs"][:T].reshape(T * E, 84, 84, 4)
        rows = raw["perm"][0, :wl.mb]
        n = wl.mb
    else:
        obs = raw["obs"].reshape((T + 1) * E, 84, 84, 4)
        rows = None
        n = (T + 1) * E
    rng = np.random.default_rng(wid * 100 + k)
    pick = np.unique(np.concatenate([[0, n - 1], rng.choice(n, k - 2, replace=False)]))
    frames = obs[rows[pick]] if rows is not None else obs[pick]
    z_w, v_w, fc = _oracle_forward(net, params, frames, MODE[prec])
    dz = (0.1 * rng.standard_normal((len(pick), net.num_actions))).astype(np.float32)
    dv = rng.standard_normal(len(pick)).astype(np.float32)
    g_w = _oracle_backward(net, fc, dz, dv)
    z, v, g = _gpu_forced(net, prec, params, obs, rows, n, fc, pick, dz, dv)
    _check_outputs(z[pick], v[pick], z_w, v_w, prec)
    _check(g, g_w, net, prec, case)


# ----------------------------------------------------------------------------- whole updates


def _gpu_update_forced(net, prec, theta, m, v, step, obs, rows, n, fc, positions, z_w, v_w, dz_w, dv_w, g_w,
                       loss, opt):
    """One update through the C-ABI from the oracle's state, each step fed the oracle's inputs:
    forward, the oracle's activations written in, the loss kernels on the oracle's logits and
    values (loss(logits, values) runs ppo_loss_grad or the target log-prob + V-trace +
    impala_loss_grad chain on device tensors and returns dlogits, dvalue for the n frames), the
    backward pass from the oracle's dlogits, dvalue (dz_w, dv_w), and the optimiser on the
    oracle's gradient g_w. Returns (dlogits, dvalue, grads, new params, m, v) as float64
    arrays."""
    torch = G.torch()
    A = net.num_actions
    ws = G.ws_bytes(P.impala_workspace_bytes(net, n, prec, 1))
    p = G.dev_f32(theta)
    o = G.dev_u8(obs)
    r = G.dev_i32(rows) if rows is not None else None
    logits = torch.empty((n, A), dtype=torch.float32, device="cuda:0")
    value = torch.empty(n, dtype=torch.float32, device="cuda:0")
    P.impala_cnn_fwd(net, prec, p, o, r, n, ws, 1, logits, value)
    _inject(ws, net, prec, n, fc, positions)
    G.sync()
    _check_outputs(G.host(logits)[positions], G.host(value)[positions], z_w, v_w, prec)
    dz, dv = loss(G.dev_f32(z_w), G.dev_f32(v_w))
    grads = torch.empty_like(p)
    P.impala_cnn_bwd(net, prec, p, o, r, n, ws, G.dev_f32(dz_w), G.dev_f32(dv_w), grads)
    dm, dvv = G.dev_f32(m), G.dev_f32(v)
    opt(p, G.dev_f32(g_w), dm, dvv, step)
    G.sync()
    return G.host(dz), G.host(dv), G.host(grads), G.host(p), G.host(dm), G.host(dvv)


def _check_dlogits(got, want, coef, logp, ent_coef, label):
    """Loss gradients against the oracle's from the same logits. With He-normal parameters the
    logits reach ~50 and the softmax saturates: a row's gradient is then made of 1 - p(a) and
    of probabilities far below float32's resolution of the O(1) values they are formed from.
    Each element is held to float32 resolution of its row's operands: |got - want| <=
    1e-5 |want| + 2^-20 (coef_i + ent_coef (1 + max_j |log p_ij|)) / m, with coef_i the row's
    policy-gradient weight (|A_hat r| for PPO, pg_coef |pg_adv| for IMPALA). The loss kernels
    are pinned to 1e-5 on well-conditioned logits by the kernel tests."""
    m = want.shape[0]
    scale = (coef + ent_coef * (1 + np.abs(logp).max(axis=1))) / m
    bad = np.abs(got - want) > 1e-5 * np.abs(want) + 2.0 ** -20 * scale[:, None]
    assert not bad.any(), f"{label} dlogits: {int(bad.sum())} elements beyond float32 resolution"


def _r32(x):
    """Values as the library receives them: rounded to float32 (kept in float64)."""
    return np.asarray(x, np.float32).astype(np.float64)


def _check_dvalue(got, want, values, targets, vf_coef, label):
    """Value-loss gradients vf_coef (V - target) / m: each element to 1e-5 relative plus
    float32's resolution of its operands, 2^-20 vf_coef (|V| + |target|) / m (late in training
    V-trace targets can sit within float32 rounding of the values)."""
    m = want.shape[0]
    bad = np.abs(got - want) > 1e-5 * np.abs(want) + 2.0 ** -20 * vf_coef * (np.abs(values) + np.abs(targets)) / m
    assert not bad.any(), f"{label} dvalue: {int(bad.sum())} elements beyond float32 resolution"


def _check_opt(got, want, theta, label, extra=0.0, floors=(0.0, 0.0)):
    """The optimiser fed the oracle's gradient, against the oracle's optimiser applied in float64
    to the same float32 inputs (parameters, state, gradient, hyperparameters): the new float32
    parameters within 2 ulps plus 1e-5 of the step plus `extra` (the step's sensitivity to the
    float32 rounding of a cancelling moment update; and below float32's normal range, where the
    arithmetic itself is denormal, within 2^-126), and the step to 1e-3 where it spans at
    least 1024 ulps (below that the result's own rounding dominates); the optimiser state to
    1e-5 relative L2, and elementwise to 1e-5 plus `floors` (float32's resolution of each state
    update's terms) plus 2^-126 (denormal results, e.g. the square of a gradient near 1e-20)."""
    p, pw = got[0], want[0]
    ulp = np.spacing(np.abs(pw).astype(np.float32)).astype(np.float64)
    bad = np.abs(p - pw) > 2 * ulp + 1e-5 * np.abs(pw - theta) + extra + 2.0 ** -126
    i = int(np.argmax(bad)) if bad.any() else 0
    assert not bad.any(), (f"{label}: {int(bad.sum())} parameters off the oracle's, e.g. [{i}]: got {p[i]!r} "
                           f"want {pw[i]!r} from {theta[i]!r} (ulp {ulp[i]:.3e})")
    big = np.abs(pw - theta) >= 1024 * ulp
    if big.sum() >= 16:
        G.assert_close(p[big] - theta[big], (pw - theta)[big], 1e-3, label + " parameter step")
    for g, w, fl, what in zip(got[1:], want[1:], floors, ("first moment", "second moment")):
        if w is not None:
            assert G.rel_l2(g, w) <= 1e-5, f"{label} {what}: relative L2 {G.rel_l2(g, w):.2e}"
            bad = np.abs(g - w) > 1e-5 * np.abs(w) + fl + 2.0 ** -126
            assert not bad.any(), f"{label} {what}: {int(bad.sum())} elements beyond float32 resolution"


@pytest.mark.parametrize("prec", [G.BF16, G.FP32], ids=lambda p: PNAME[p])
def test_forced_ppo_updates_chain_from_oracle_state(prec):
    """Six PPO updates (6 envs x 4 steps, 2 epochs x 3 minibatches of 8, 84x84 frames, 5
    actions), each run on the GPU through the C-ABI from the oracle's state after the previous
    update, with the oracle's activations: per update, the loss gradient (1e-5), the parameter
    gradient (per tensor, as above), and Adam fed the oracle's gradient (parameter step and
    moments to 1e-5)."""
    from synth import Workload
    wl = Workload("ppo_small", "ppo", T=4, E=6, net=NetShape(num_actions=5), epochs=2, num_minibatches=3, seed=21)
    net, A, mb = wl.net, wl.net.num_actions, wl.mb
    mode = MODE[prec]
    params = draw_params(net, wl.seed)
    raw = draw_rollout(wl)
    ro = olearner.behaviour_rollout(wl, params, raw)
    adv, ret = otargets.gae(ro["rewards"], ro["values"], ro["dones"], ro["next_value"], ro["next_done"],
                            wl.gamma, wl.lam)
    adv, ret = adv.ravel(), ret.ravel()
    dt = np.float64 if mode == "fp64" else np.float32
    theta, m_, v_ = params.astype(dt), np.zeros(params.size, dt), np.zeros(params.size, dt)
    aws = G.ws_bytes(P.adam_workspace_bytes(params.size))
    for u in range(wl.n_updates):
        j, k = divmod(u, wl.num_minibatches)
        rows = raw["perm"][j, k * mb:(k + 1) * mb]
        z_w, v_w, fc = _oracle_forward(net, theta, ro["obs"][rows], mode)
        _, dz_w, dv_w, _ = olosses.ppo_loss_grad(z_w, v_w, ro["actions"][rows], ro["logp"][rows], adv[rows],
                                                 ret[rows], wl.clip_eps, wl.vf_coef, wl.ent_coef, True, dtype=dt)
        g_w = _oracle_backward(net, fc, dz_w, dv_w)
        gc, _ = ooptim.clip_by_global_norm(g_w, f32(wl.max_grad_norm), dt)
        t_next, m_next, v_next = ooptim.adam(theta, gc, m_, v_, u + 1, f32(wl.lr), f32(wl.beta1), f32(wl.beta2),
                                             f32(wl.adam_eps), dt)
        dr = G.dev_i32(rows)

        def loss(zd, vd):
            dz, dv = G.torch().empty_like(zd), G.torch().empty_like(vd)
            st = G.torch().zeros(8, dtype=G.torch().float32, device="cuda:0")
            rl = dr.long()
            P.ppo_loss_grad(mb, A, zd, vd, G.dev_i32(ro["actions"])[rl].contiguous(),
                            G.dev_f32(ro["logp"])[rl].contiguous(), G.dev_f32(adv)[rl].contiguous(),
                            G.dev_f32(ret)[rl].contiguous(), 1, wl.clip_eps, wl.vf_coef, wl.ent_coef, dz, dv, st)
            return dz, dv

        def opt(p, g, m, v, step):
            P.adam_step(p.numel(), p, g, m, v, step, wl.lr, wl.beta1, wl.beta2, wl.adam_eps, wl.max_grad_norm,
                        None, aws)

        got = _gpu_update_forced(net, prec, theta, m_, v_, u + 1, ro["obs"], rows, mb, fc, np.arange(mb),
                                 z_w, v_w, dz_w, dv_w, g_w, loss, opt)
        ah = (adv[rows] - adv[rows].mean()) / (adv[rows].std() + 1e-8)
        lsm = olosses.log_softmax(z_w)
        ratio = np.exp(lsm[np.arange(mb), ro["actions"][rows]] - ro["logp"][rows])
        _check_dlogits(got[0], dz_w, np.abs(ah) * ratio, lsm, wl.ent_coef, f"update {u}")
        _check_dvalue(got[1], dv_w, v_w, ret[rows], wl.vf_coef, f"update {u}")
        _check(got[2], g_w, net, prec, f"ppo update {u}")
        g32, _ = ooptim.clip_by_global_norm(_r32(g_w), f32(wl.max_grad_norm))
        want_opt = ooptim.adam(_r32(theta), g32, _r32(m_), _r32(v_), u + 1, f32(wl.lr), f32(wl.beta1),
                               f32(wl.beta2), f32(wl.adam_eps))
        # m = b1 m + (1 - b1) g rounds in float32: where the two terms cancel, the step inherits
        # 2^-22 (b1 |m| + (1 - b1) |g|) through lr / ((1 - b1^t)(sqrt(v_hat) + eps))
        b1, b2, t = f32(wl.beta1), f32(wl.beta2), u + 1
        extra = f32(wl.lr) * 2.0 ** -22 * (b1 * np.abs(_r32(m_)) + (1 - b1) * np.abs(g32)) / (
            (1 - b1 ** t) * (np.sqrt(want_opt[2] / (1 - b2 ** t)) + f32(wl.adam_eps)))
        floors = (2.0 ** -22 * (b1 * np.abs(_r32(m_)) + (1 - b1) * np.abs(g32)),
                  2.0 ** -22 * (b2 * _r32(v_) + (1 - b2) * g32 * g32))
        _check_opt(got[3:], want_opt, _r32(theta), f"ppo update {u}", extra, floors)
        theta, m_, v_ = t_next, m_next, v_next


@pytest.mark.parametrize("prec", [G.BF16, G.FP32], ids=lambda p: PNAME[p])
def test_forced_impala_env_block_updates_chain_from_oracle_state(prec):
    """Appendix B's IMPALA setting at a small size (8 envs x 5 steps, 4 env-block minibatches,
    RMSprop decay 0.99 eps 0.01, the paper's lr 6e-4, omega 40): each of the four updates on
    the GPU from the oracle's state after the previous one, through the C-ABI (forward over the
    block's rollout and bootstrap frames, target log-probs, V-trace, IMPALA loss, backward,
    RMSprop), with the oracle's activations."""
    wl = WORKLOADS[6].replace(T=5, E=8, seed=24)
    net, A = wl.net, wl.net.num_actions
    T, E, nmb = wl.T, wl.E, wl.num_minibatches
    Eb = E // nmb
    n = T * Eb
    mode = MODE[prec]
    dt = np.float64 if mode == "fp64" else np.float32
    params = draw_params(net, wl.seed)
    raw = draw_rollout(wl)
    ro = olearner.behaviour_rollout(wl, params, raw)
    theta, nu = params.astype(dt), np.zeros(params.size, dt)
    rws = G.ws_bytes(P.rmsprop_workspace_bytes(params.size))
    torch = G.torch()
    for k in range(nmb):
        envs = np.arange(k * Eb, (k + 1) * Eb)
        rows = (np.arange(T + 1)[:, None] * E + envs[None, :]).ravel()
        act = ro["actions"][rows[:n]]
        mu = ro["logp"][rows[:n]]
        rew, dn, nd = ro["rewards"][:, envs], ro["dones"][:, envs], ro["next_done"][envs]
        z_w, v_w, fc = _oracle_forward(net, theta, ro["obs"][rows], mode)
        tl = olosses.log_softmax(z_w[:n])[np.arange(n), act]
        vs, pg = otargets.vtrace(mu.reshape(T, Eb), tl.reshape(T, Eb), rew, v_w[:n].reshape(T, Eb), dn, v_w[n:],
                                 nd, wl.gamma, wl.lam, wl.rho_bar, wl.c_bar, wl.pg_rho_bar, dt)
        _, dz_w, dv_w, _ = olosses.impala_loss_grad(z_w[:n], v_w[:n], act, vs.ravel(), pg.ravel(), wl.pg_coef,
                                                    wl.vf_coef, wl.ent_coef, dt)
        dz_all, dv_all = np.zeros_like(z_w), np.zeros_like(v_w)
        dz_all[:n], dv_all[:n] = dz_w, dv_w
        g_w = _oracle_backward(net, fc, dz_all, dv_all)
        gc, _ = ooptim.clip_by_global_norm(g_w, f32(wl.max_grad_norm), dt)
        t_next, nu_next = ooptim.rmsprop(theta, gc, nu, f32(wl.lr), f32(wl.rms_decay), f32(wl.rms_eps), dt)

        def loss(zd, vd):
            tlogp = torch.empty(n, dtype=torch.float32, device="cuda:0")
            P.impala_action_logp(n, A, zd, G.dev_i32(act), tlogp)
            vsd, pgd = torch.empty(n, dtype=torch.float32, device="cuda:0"), torch.empty(n, dtype=torch.float32,
                                                                                        device="cuda:0")
            P.vtrace_targets(T, Eb, G.dev_f32(mu), tlogp, G.dev_f32(rew), vd[:n].contiguous(), G.dev_u8(dn),
                             vd[n:].contiguous(), G.dev_u8(nd), wl.gamma, wl.lam, wl.rho_bar, wl.c_bar,
                             wl.pg_rho_bar, vsd, pgd)
            dz, dv = torch.zeros_like(zd), torch.zeros_like(vd)
            st = torch.zeros(8, dtype=torch.float32, device="cuda:0")
            P.impala_loss_grad(n, A, zd, vd, G.dev_i32(act), vsd, pgd, wl.pg_coef, wl.vf_coef, wl.ent_coef,
                               dz, dv, st)
            return dz, dv

        def opt(p, g, m, v, step):
            P.rmsprop_step(p.numel(), p, g, v, wl.lr, wl.rms_decay, wl.rms_eps, wl.max_grad_norm, None, rws)

        got = _gpu_update_forced(net, prec, theta, np.zeros_like(theta), nu, k + 1, ro["obs"], rows, n + Eb, fc,
                                 np.arange(n + Eb), z_w, v_w, dz_all, dv_all, g_w, loss, opt)
        _check_dlogits(got[0][:n], dz_w, wl.pg_coef * np.abs(pg.ravel()), olosses.log_softmax(z_w[:n]),
                       wl.ent_coef, f"update {k}")
        assert not got[0][n:].any()
        assert not got[1][n:].any()
        _check_dvalue(got[1][:n], dv_w, v_w[:n], vs.ravel(), wl.vf_coef, f"update {k}")
        _check(got[2], g_w, net, prec, f"impala update {k}")
        g32, _ = ooptim.clip_by_global_norm(_r32(g_w), f32(wl.max_grad_norm))
        p_o, nu_o = ooptim.rmsprop(_r32(theta), g32, _r32(nu), f32(wl.lr), f32(wl.rms_decay), f32(wl.rms_eps))
        d = f32(wl.rms_decay)
        _check_opt((got[3], None, got[5]), (p_o, None, nu_o), _r32(theta), f"impala update {k}",
                   floors=(0.0, 2.0 ** -22 * (d * _r32(nu) + (1 - d) * g32 * g32)))
        theta, nu = t_next, nu_next
