"""CPU tests of the C-ABI boundary: the library loads, exports every declared symbol, agrees
with the oracle's parameter layout, and rejects bad arguments before any HIP call."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
P = pytest.importorskip("paper_2310_00036_amd")

from oracle import net as onet  # noqa: E402
from synth import NetShape, WORKLOADS  # noqa: E402


def _declared_functions():
    names = set()
    for h in ("cleanba_learner.h", "cleanba_layers.h", "cleanba_profile.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(",
                             src, flags=re.M):
            names.add(m.group(1))
    return names


def test_exports_every_declared_symbol():
    names = _declared_functions()
    for want in ("impala_cnn_fwd", "impala_cnn_bwd", "gae_advantages", "vtrace_targets",
                 "ppo_loss_grad", "impala_loss_grad", "adam_step", "learner_step"):
        assert want in names
    lib = C.CDLL(P._lib.LIB_PATH)
    missing = [n for n in sorted(names) if not hasattr(lib, n)]
    assert not missing, missing
    assert names <= set(P._lib._SIGS), sorted(names - set(P._lib._SIGS))


@pytest.mark.parametrize("net", [NetShape(), NetShape(num_actions=6), NetShape(ch=(32, 64, 64), hidden=512),
                                 NetShape(in_h=12, in_w=10, ch=(16, 16, 32), hidden=8, num_actions=3)])
def test_param_layout_matches_oracle(net):
    got = P.impala_param_layout(net)
    want = [(n, tuple(s), o) for n, s, o in onet.param_layout(net)]
    assert got == want
    assert P.impala_param_count(net) == onet.param_count(net)


def test_invalid_nets_are_rejected():
    for bad in (NetShape(in_c=3), NetShape(ch=(16, 24, 32)), NetShape(ch=(32, 16, 16)),
                NetShape(num_actions=65), NetShape(hidden=0), NetShape(in_h=0)):
        with pytest.raises(P.LibraryError) as e:
            P.impala_param_count(bad)
        assert e.value.status == -1


def _net():
    return C.byref(P.net_struct(NetShape()))


def test_null_pointers_and_small_workspace_fail_before_hip():
    lib = P.lib
    # forward with NULL params
    st = lib.impala_cnn_fwd(_net(), 0, None, 1, None, 4, 1, 1 << 40, 1, 1, 1, None)
    assert st == -1 and b"params" in lib.impala_last_error()
    # workspace too small
    need = lib.impala_workspace_bytes(_net(), 4, 0, 1)
    st = lib.impala_cnn_fwd(_net(), 0, 1, 1, None, 4, 1, need - 1, 1, 1, 1, None)
    assert st == -2
    st = lib.impala_cnn_bwd(_net(), 1, 1, 1, None, 4, 1, 16, 1, 1, 1, None)
    assert st == -2
    # bad precision
    assert lib.impala_cnn_fwd(_net(), 7, 1, 1, None, 4, 1, 1 << 40, 1, 1, 1, None) == -1
    # scans and losses
    assert lib.gae_advantages(-1, 4, 1, 1, 1, 1, 1, 0.99, 0.95, 1, 1, None) == -1
    assert lib.gae_advantages(8, 4, None, 1, 1, 1, 1, 0.99, 0.95, 1, 1, None) == -1
    assert lib.vtrace_targets(8, 4, 1, 1, 1, 1, 1, 1, None, .99, 1, 1, 1, 1, 1, 1, None) == -1
    assert lib.ppo_loss_grad(16, 0, 1, 1, 1, 1, 1, 1, 1, .1, .5, .01, 1, 1, 1, None, 0, None) == -1
    assert lib.ppo_loss_grad(16, 65, 1, 1, 1, 1, 1, 1, 1, .1, .5, .01, 1, 1, 1, None, 0, None) == -1
    assert lib.impala_loss_grad(0, 6, 1, 1, 1, 1, 1, 1., .5, .01, 1, 1, 1, None, 0, None) == -1
    need = lib.loss_workspace_bytes(4096)
    assert need >= 4096 * 40
    assert lib.ppo_loss_grad(4096, 18, 1, 1, 1, 1, 1, 1, 1, .1, .5, .01, 1, 1, 1, 1, need - 1, None) == -2
    assert lib.impala_loss_grad(4096, 18, 1, 1, 1, 1, 1, 1., .5, .01, 1, 1, 1, 1, need - 1, None) == -2
    # adam
    assert lib.adam_step(10, 1, 1, 1, 1, 0, 1e-3, .9, .999, 1e-5, .5, None, 1, 1 << 20, None) == -1
    assert lib.adam_step(10, 1, 1, 1, 1, 1, 1e-3, 1.0, .999, 1e-5, .5, None, 1, 1 << 20, None) == -1
    assert lib.adam_step(10, 1, 1, 1, 1, 1, 1e-3, .9, .999, 1e-5, .5, None, 1, 8, None) == -2
    # rmsprop
    assert lib.rmsprop_step(10, 1, 1, 1, 6e-4, 1.0, .01, 40., None, 1, 1 << 20, None) == -1
    assert lib.rmsprop_step(10, 1, 1, 1, 6e-4, .99, -1., 40., None, 1, 1 << 20, None) == -1
    assert lib.rmsprop_step(10, 1, 1, None, 6e-4, .99, .01, 40., None, 1, 1 << 20, None) == -1
    assert lib.rmsprop_step(10, 1, 1, 1, 6e-4, .99, .01, 40., None, 1, 8, None) == -2
    assert lib.rmsprop_step(0, None, None, None, 6e-4, .99, .01, 40., None, None, 0, None) == 0
    # layers
    assert lib.impala_conv3x3_fwd(0, 4, 84, 84, 4, 24, 1, 2, None, 1, None, None, 1, None) == -3
    assert lib.impala_conv3x3_dgrad(0, 4, 42, 42, 32, 16, 1, 1, None, None, 1, None) == -3
    assert lib.impala_maxpool_fwd(0, 4, 42, 42, 6, 1, 1, 1, None) == -3
    # the fused residual-block backward: 16 or 32 channels in bf16 only, a workspace, no NULLs
    rb_ws = lib.impala_resblock_bwd_workspace_bytes(P.PREC_BF16, 16)
    assert rb_ws > 0 and lib.impala_resblock_bwd_workspace_bytes(P.PREC_FP32, 16) == 0
    assert lib.impala_resblock_bwd_workspace_bytes(P.PREC_BF16, 32) > 0
    rb = (1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1)
    assert lib.impala_resblock_bwd(P.PREC_BF16, 4, 42, 42, 64, *rb, 1 << 40, None) == -3
    assert lib.impala_resblock_bwd(P.PREC_FP32, 4, 42, 42, 16, *rb, 1 << 40, None) == -3
    assert lib.impala_resblock_bwd(P.PREC_BF16, 4, 42, 42, 16, *rb, rb_ws - 1, None) == -2
    assert lib.impala_resblock_bwd(P.PREC_BF16, 4, 42, 42, 16, None, *rb[1:], rb_ws, None) == -1
    # zero-size work is a no-op success
    assert lib.gae_advantages(0, 4, None, None, None, None, None, .99, .95, None, None, None) == 0
    assert lib.impala_cnn_fwd(_net(), 0, None, None, None, 0, None, 0, 1, None, None, None) == 0


def test_learner_cfg_validation():
    wl = WORKLOADS[1]
    cfg = P.learner_cfg(wl, P.PREC_BF16)
    assert P.learner_workspace_bytes(wl.net, cfg) > 0
    bad = P.learner_cfg(wl.replace(minibatch_size=5000), P.PREC_BF16)   # 4 * 5000 > 8192
    assert P.lib.learner_workspace_bytes(C.byref(P.net_struct(wl.net)), C.byref(bad)) == 0
    assert b"exceeds" in P.lib.impala_last_error()
    ro = P.Rollout()
    st = C.c_int32(0)
    r = P.lib.learner_step(C.byref(P.net_struct(wl.net)), C.byref(cfg), C.byref(ro), 1, 1, 1,
                           C.byref(st), 1, 1, 1 << 40, 1, None)
    assert r == -1 and b"obs" in P.lib.impala_last_error()
    bad = P.learner_cfg(wl.replace(optimizer="rmsprop", rms_decay=1.0), P.PREC_BF16)
    assert P.lib.learner_workspace_bytes(C.byref(P.net_struct(wl.net)), C.byref(bad)) == 0
    assert b"RMSprop" in P.lib.impala_last_error()
    bad.optimizer = 7
    assert P.lib.learner_workspace_bytes(C.byref(P.net_struct(wl.net)), C.byref(bad)) == 0


def test_workspace_grows_with_frames_and_precision():
    """Linear in the frame count (activations) on top of a fixed part (partial-sum buffers);
    float32 storage needs more than bf16; inference less than training."""
    net = NetShape()
    a = P.impala_workspace_bytes(net, 256, P.PREC_BF16, 1)
    b = P.impala_workspace_bytes(net, 512, P.PREC_BF16, 1)
    e = P.impala_workspace_bytes(net, 1024, P.PREC_BF16, 1)
    c = P.impala_workspace_bytes(net, 256, P.PREC_FP32, 1)
    d = P.impala_workspace_bytes(net, 256, P.PREC_BF16, 0)
    assert b > a and abs((e - b) - 2 * (b - a)) <= 0.02 * (e - b)
    assert c > 1.5 * a and d < a


@pytest.mark.parametrize("prec", [0, 1], ids=["bf16", "fp32"])
@pytest.mark.parametrize("net", [NetShape(), NetShape(ch=(32, 64, 64), hidden=512),
                                 NetShape(in_h=12, in_w=10, ch=(16, 16, 32), hidden=8, num_actions=3)])
def test_activation_layout_is_disjoint_and_inside_the_workspace(net, prec):
    """The saved-activation regions of a training forward: the names and shapes of the network's
    stages, disjoint, inside impala_workspace_bytes(net, n, prec, 1), element sizes per dtype."""
    n = 37
    lay = P.impala_activation_layout(net, prec, n)
    total = P.impala_workspace_bytes(net, n, prec, 1)
    es = {P.DT_U8: 1, P.DT_BF16: 2, P.DT_F32: 4}
    act = P.DT_BF16 if prec == 0 else P.DT_F32
    names = [d[0] for d in lay]
    want = []
    h, w = net.in_h, net.in_w
    shapes = {}
    for s, c in enumerate(net.ch):
        oh, ow = -(-h // 2), -(-w // 2)
        if prec == 1:
            want.append(f"s{s}.conv")
            shapes[f"s{s}.conv"] = ((n, h, w, c), act)
        for k in ("arg", "x0", "x1", "x2", "t0", "t1"):
            want.append(f"s{s}.{k}")
            shapes[f"s{s}.{k}"] = ((n, oh, ow, c), P.DT_U8 if k == "arg" else act)
        h, w = oh, ow
    want.append("h")
    shapes["h"] = ((n, net.hidden), act)
    assert names == want and len(lay) == (22 if prec == 1 else 19)
    spans = []
    for name, off, nbytes, dt, shape in lay:
        assert (shape, dt) == shapes[name], name
        assert nbytes == int(np.prod(shape)) * es[dt]
        assert off % 256 == 0 and off + nbytes <= total
        spans.append((off, off + nbytes))
    spans.sort()
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
    with pytest.raises(P.LibraryError):
        P.impala_activation_layout(net, prec, 0)


def test_noalloc_adam_validates_before_hip():
    """adam_step_noalloc rejects bad arguments on the host and returns OK for an empty buffer
    before touching the GPU."""
    lib = P.lib
    assert lib.adam_step_noalloc(-1, 1, 1, 1, 1, 1, 1e-3, 0.9, 0.999, 1e-5, 0.5, None, None) == -1
    assert lib.adam_step_noalloc(10, 1, 1, 1, 1, 0, 1e-3, 0.9, 0.999, 1e-5, 0.5, None, None) == -1
    assert b"1-based" in lib.impala_last_error()
    assert lib.adam_step_noalloc(10, 1, 1, 1, 1, 1, 1e-3, 1.0, 0.999, 1e-5, 0.5, None, None) == -1
    assert lib.adam_step_noalloc(10, None, 1, 1, 1, 1, 1e-3, 0.9, 0.999, 1e-5, 0.5, None, None) == -1
    assert lib.adam_step_noalloc(0, None, None, None, None, 1, 1e-3, 0.9, 0.999, 1e-5, 0.5, None, None) == 0


def test_mfma_probe_validates_before_hip():
    """impala_probe_mfma_bf16 rejects bad sizes and NULL pointers on the host (no launch)."""
    lib = P.lib
    flop = C.c_int64()
    fake = C.c_void_p(16)   # never dereferenced: every call below fails validation first
    assert lib.impala_probe_mfma_bf16(0, 1, fake, C.byref(flop), None) == -1
    assert lib.impala_probe_mfma_bf16(1, 0, fake, C.byref(flop), None) == -1
    assert lib.impala_probe_mfma_bf16(65537, 1, fake, C.byref(flop), None) == -1
    assert lib.impala_probe_mfma_bf16(1, (1 << 20) + 1, fake, C.byref(flop), None) == -1
    assert lib.impala_probe_mfma_bf16(1, 1, None, C.byref(flop), None) == -1
    assert lib.impala_probe_mfma_bf16(1, 1, fake, None, None) == -1
    assert b"NULL" in lib.impala_last_error()
