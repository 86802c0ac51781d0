"""GPU parity of every kernel against the oracle on identical inputs (via the C-ABI).

bf16 mode: inputs are bf16-representable, so the only difference from the exact result is
float32 accumulation order and the final rounding of stored outputs (checked to 1 bf16 ulp
for stored activations, 1e-5 relative for float32 outputs). fp32 mode: 1e-5 relative.
Shapes span several tiles and ragged tails (widths and heights that are not multiples of
the tile, frame counts that are not multiples of the frames per workgroup).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

from oracle import losses as olosses, net as onet, optim as ooptim, targets as otargets  # noqa: E402
from tests import gpu_util as G  # noqa: E402

P = pytest.importorskip("paper_2310_00036_amd")

PRECS = [G.BF16, G.FP32]
PNAME = {G.BF16: "bf16", G.FP32: "fp32"}


def _relu(x):
    return np.maximum(x, 0)


# (n, H, W, cin, cout, mode): the network's conv shapes (base and wide) plus ragged ones
CONV_CASES = [
    (3, 84, 84, 4, 16, P.X_U8), (2, 84, 84, 4, 32, P.X_U8), (2, 13, 9, 4, 64, P.X_U8),
    (3, 42, 42, 16, 16, P.X_RELU), (3, 42, 42, 16, 32, P.X_PLAIN), (2, 21, 21, 32, 32, P.X_PLAIN),
    (5, 21, 21, 32, 32, P.X_RELU), (7, 11, 11, 32, 32, P.X_RELU), (3, 42, 42, 32, 64, P.X_PLAIN),
    (3, 21, 21, 64, 64, P.X_RELU), (5, 11, 11, 64, 64, P.X_PLAIN), (2, 17, 23, 16, 64, P.X_PLAIN),
    (4, 9, 13, 32, 64, P.X_PLAIN), (6, 7, 5, 64, 64, P.X_RELU),
]


def _conv_inputs(n, H, W, cin, cout, mode, prec, seed):
    rng = np.random.default_rng(seed)
    if mode == P.X_U8:
        x = rng.integers(0, 256, size=(n + 2, H, W, cin), dtype=np.uint8)
        rows = rng.permutation(n + 2)[:n].astype(np.int32)
        xin = x[rows].astype(np.float64) / 255.0
    else:
        x = G.q(rng.standard_normal((n, H, W, cin)), prec)
        rows = None
        xin = _relu(x) if mode == P.X_RELU else x
    w = rng.standard_normal((3, 3, cin, cout)).astype(np.float32) * np.sqrt(2.0 / (9 * cin))
    b = (0.1 * rng.standard_normal(cout)).astype(np.float32)
    return x, rows, xin, w, b


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "n%d_%dx%d_%d-%d_m%d" % c)
def test_conv_forward(case, prec):
    n, H, W, cin, cout, mode = case
    x, rows, xin, w, b = _conv_inputs(n, H, W, cin, cout, mode, prec, 11)
    wq = G.q(w, prec)
    add = G.q(np.random.default_rng(5).standard_normal((n, H, W, cout)), prec) if mode == P.X_RELU else None
    want = onet.conv3x3(xin, wq, b.astype(np.float64)) + (add if add is not None else 0)
    absum = onet.conv3x3(np.abs(xin), np.abs(wq), np.abs(b).astype(np.float64)) + \
        (np.abs(add) if add is not None else 0)
    dx = G.dev_u8(x) if mode == P.X_U8 else G.dev_act(x, prec)
    y = G.empty_act((n, H, W, cout), prec)
    P.impala_conv3x3_fwd(prec, n, H, W, cin, cout, dx, mode, G.dev_i32(rows) if rows is not None else None,
                         G.dev_f32(w), G.dev_f32(b), G.dev_act(add, prec) if add is not None else None, y)
    G.sync()
    got = G.host(y)
    if prec == G.BF16:
        G.assert_bf16_ulp(got, want, absum, "conv fwd")
    else:
        G.assert_sum_close(got, want, absum, 1e-5, "conv fwd")


POOL_CASES = [(3, 84, 84, 4, 16, P.X_U8), (2, 84, 84, 4, 32, P.X_U8), (2, 13, 9, 4, 64, P.X_U8),
              (3, 42, 42, 16, 32, P.X_PLAIN), (2, 42, 42, 16, 16, P.X_PLAIN), (4, 21, 21, 32, 32, P.X_PLAIN),
              (5, 11, 11, 32, 64, P.X_PLAIN), (2, 17, 23, 16, 64, P.X_PLAIN), (3, 21, 21, 64, 64, P.X_PLAIN),
              (3, 17, 23, 16, 32, P.X_PLAIN), (2, 13, 9, 4, 16, P.X_U8), (4, 9, 7, 32, 32, P.X_PLAIN),
              (5, 11, 11, 32, 32, P.X_PLAIN), (1, 6, 5, 16, 16, P.X_PLAIN), (2, 23, 19, 4, 32, P.X_U8),
              (2, 42, 42, 32, 64, P.X_PLAIN), (3, 9, 11, 64, 64, P.X_PLAIN), (2, 11, 11, 64, 64, P.X_PLAIN)]


def _pool_windows(x, fill):
    """[9, n, OH, OW, C]: the 3x3 stride-2 SAME windows of x, padded cells = fill."""
    n, h, w, c = x.shape
    oh, ph0, ph1 = onet.same_pool_pads(h)
    ow, pw0, pw1 = onet.same_pool_pads(w)
    xp = np.full((n, h + ph0 + ph1, w + pw0 + pw1, c), fill, np.float64)
    xp[:, ph0:ph0 + h, pw0:pw0 + w] = x
    return np.stack(onet._pool_views(xp, oh, ow))


@pytest.mark.parametrize("case", POOL_CASES, ids=lambda c: "n%d_%dx%d_%d-%d_m%d" % c)
def test_conv_pool_forward(case):
    """Fused conv + max-pool (bf16): the conv output is never stored, so the check works on
    the exact conv: the pooled value is within 1 bf16 ulp of the exact conv at the chosen
    cell, that cell is a maximum up to rounding, and wherever the window's maximum is clear
    by more than 4 ulps the argmax is the oracle's."""
    _conv_pool_check(case)


@pytest.mark.parametrize("case", [(1024, 84, 84, 4, 16, P.X_U8), (1024, 42, 42, 16, 32, P.X_PLAIN),
                                  (1024, 42, 42, 32, 64, P.X_PLAIN), (1024, 21, 21, 64, 64, P.X_PLAIN)],
                         ids=lambda c: "n%d_%dx%d_%d-%d_m%d" % c)
def test_conv_pool_forward_many_tiles_per_workgroup(case):
    """The same checks at a frame count where every workgroup runs several tiles (each tile's
    window is staged during the previous tile's max-pool), on frames spread over the launch."""
    _conv_pool_check(case, sample=[0, 1, 517, case[0] - 1])


def _conv_pool_check(case, sample=None):
    n, H, W, cin, cout, mode = case
    x, rows, xin, w, b = _conv_inputs(n, H, W, cin, cout, mode, G.BF16, 13)
    fs = slice(None) if sample is None else np.asarray(sample)   # frames checked
    xin = xin[fs]
    wq = G.q(w, G.BF16)
    conv = onet.conv3x3(xin, wq, b.astype(np.float64))
    absum = onet.conv3x3(np.abs(xin), np.abs(wq), np.abs(b).astype(np.float64))
    win, wabs = _pool_windows(conv, -np.inf), _pool_windows(absum, 0.0)
    OH, OW = win.shape[2:4]
    torch = G.torch()
    y = G.empty_act((n, OH, OW, cout), G.BF16)
    arg = torch.empty((n, OH, OW, cout), dtype=torch.uint8, device="cuda:0")
    dx = G.dev_u8(x) if mode == P.X_U8 else G.dev_act(x, G.BF16)
    P.impala_conv3x3_pool_fwd(G.BF16, n, H, W, cin, cout, dx, mode, G.dev_i32(rows) if rows is not None else None,
                              G.dev_f32(w), G.dev_f32(b), y, arg)
    G.sync()
    got_arg = arg.cpu().numpy().astype(np.int64)[fs]
    assert got_arg.max() <= 8
    sel = np.take_along_axis(win, got_arg[None], 0)[0]
    assert np.isfinite(sel).all(), "argmax points at a padded cell"
    G.assert_bf16_ulp(G.host(y)[fs], sel, np.take_along_axis(wabs, got_arg[None], 0)[0], "pooled value")
    best = win.max(0)
    amax = wabs.max(0)
    spacing = np.maximum(np.abs(best), 1e-30) * 2.0 ** -7
    assert (sel >= best - 2 * spacing - 2.0 ** -19 * amax).all(), "argmax is not a maximum"
    top2 = np.sort(win, 0)[-2:]
    clear = top2[1] - top2[0] > 4 * spacing + 2.0 ** -18 * amax
    assert clear.mean() > 0.5
    np.testing.assert_array_equal(got_arg[clear], win.argmax(0)[clear])


@pytest.mark.parametrize("prec", [G.FP32])
def test_conv_pool_rejects_fp32(prec):
    with pytest.raises(P.LibraryError):
        P.impala_conv3x3_pool_fwd(prec, 1, 8, 8, 16, 16, G.dev_act(np.zeros((1, 8, 8, 16)), prec), P.X_PLAIN, None,
                                  G.dev_f32(np.zeros((3, 3, 16, 16))), None, G.empty_act((1, 4, 4, 16), prec),
                                  G.torch().empty((1, 4, 4, 16), dtype=G.torch().uint8, device="cuda:0"))


RES_CASES = [(3, 42, 42, 16), (4, 21, 21, 32), (5, 11, 11, 32), (2, 17, 23, 16), (3, 9, 7, 32), (2, 84, 84, 16)]


@pytest.mark.parametrize("case", RES_CASES, ids=lambda c: "n%d_%dx%d_c%d" % c)
def test_resblock_forward(case):
    """Fused residual block (bf16): t against the exact conv1 of relu(x), y against the exact
    conv2 of relu(t) using the t the kernel returned (so t's rounding does not propagate)."""
    _resblock_fwd_check(case)


@pytest.mark.parametrize("case", [(1024, 42, 42, 16), (2048, 21, 21, 32), (2053, 42, 42, 32)],
                         ids=lambda c: "n%d_%dx%d_c%d" % c)
def test_resblock_forward_many_tiles_per_workgroup(case):
    """The same checks at a frame count where every workgroup runs several tiles (each tile's
    window is staged during the previous tile's conv2), on frames spread over the launch. At
    2053 frames of 42x42 with 32 channels every workgroup runs 32 or 33 tiles, which selects the
    kernel whose two wave roles run conv1 and conv2 of neighbouring tiles at once."""
    _resblock_fwd_check(case, sample=[0, 1, 517, case[0] - 1])


def _resblock_fwd_check(case, sample=None):
    n, H, W, C = case
    fs = slice(None) if sample is None else np.asarray(sample)   # frames checked
    rng = np.random.default_rng(17)
    x = G.q(rng.standard_normal((n, H, W, C)), G.BF16)
    w1, w2 = (rng.standard_normal((2, 3, 3, C, C)) * np.sqrt(2.0 / (9 * C))).astype(np.float32)
    b1, b2 = (0.1 * rng.standard_normal((2, C))).astype(np.float32)
    w1q, w2q = G.q(w1, G.BF16), G.q(w2, G.BF16)
    t = G.empty_act((n, H, W, C), G.BF16)
    y = G.empty_act((n, H, W, C), G.BF16)
    P.impala_resblock_fwd(G.BF16, n, H, W, C, G.dev_act(x, G.BF16), G.dev_f32(w1), G.dev_f32(b1), G.dev_f32(w2),
                          G.dev_f32(b2), t, y)
    G.sync()
    x = x[fs]
    rx = _relu(x)
    t_want = onet.conv3x3(rx, w1q, b1.astype(np.float64))
    t_abs = onet.conv3x3(np.abs(rx), np.abs(w1q), np.abs(b1).astype(np.float64))
    got_t = G.host(t)[fs]
    G.assert_bf16_ulp(got_t, t_want, t_abs, "resblock t")
    rt = _relu(got_t)
    y_want = onet.conv3x3(rt, w2q, b2.astype(np.float64)) + x
    y_abs = onet.conv3x3(np.abs(rt), np.abs(w2q), np.abs(b2).astype(np.float64)) + np.abs(x)
    G.assert_bf16_ulp(G.host(y)[fs], y_want, y_abs, "resblock y")


def test_resblock_rejects_unsupported():
    x = G.dev_act(np.zeros((1, 8, 8, 64)), G.BF16)
    w = G.dev_f32(np.zeros((3, 3, 64, 64)))
    with pytest.raises(P.LibraryError):
        P.impala_resblock_fwd(G.BF16, 1, 8, 8, 64, x, w, None, w, None, G.empty_act((1, 8, 8, 64), G.BF16),
                              G.empty_act((1, 8, 8, 64), G.BF16))
    x16 = G.dev_act(np.zeros((1, 8, 8, 16)), G.FP32)
    w16 = G.dev_f32(np.zeros((3, 3, 16, 16)))
    with pytest.raises(P.LibraryError):
        P.impala_resblock_fwd(G.FP32, 1, 8, 8, 16, x16, w16, None, w16, None, G.empty_act((1, 8, 8, 16), G.FP32),
                              G.empty_act((1, 8, 8, 16), G.FP32))


@pytest.mark.parametrize("case", [(1024, 21, 21, 64, 64, 1), (1024, 21, 21, 64, 64, 0), (1027, 11, 11, 64, 64, 1),
                                  (1026, 11, 11, 64, 64, 0), (300, 42, 42, 32, 64, 0)],
                         ids=lambda c: "n%d_%dx%d_%d-%d_add%d" % c)
def test_conv_forward_many_tiles_per_workgroup(case):
    """bf16 forward conv at frame counts where every workgroup of the persistent grid runs many
    tiles (the wide net's 64-channel residual convs, relu(x) in, with and without the residual
    add; several frames per tile at 11x11 with a ragged last tile), checked on frames spread
    over the launch."""
    n, H, W, cin, cout, with_add = case
    mode = P.X_RELU if cin == cout else P.X_PLAIN
    fs = np.asarray([0, 1, n // 2 + 5, n - 2, n - 1])
    x, rows, xin, w, b = _conv_inputs(n, H, W, cin, cout, mode, G.BF16, 17)
    wq = G.q(w, G.BF16)
    add = G.q(np.random.default_rng(6).standard_normal((n, H, W, cout)), G.BF16) if with_add else None
    want = onet.conv3x3(xin[fs], wq, b.astype(np.float64)) + (add[fs] if with_add else 0)
    absum = onet.conv3x3(np.abs(xin[fs]), np.abs(wq), np.abs(b).astype(np.float64)) + \
        (np.abs(add[fs]) if with_add else 0)
    y = G.empty_act((n, H, W, cout), G.BF16)
    P.impala_conv3x3_fwd(G.BF16, n, H, W, cin, cout, G.dev_act(x, G.BF16), mode, None, G.dev_f32(w),
                         G.dev_f32(b), G.dev_act(add, G.BF16) if with_add else None, y)
    G.sync()
    G.assert_bf16_ulp(G.host(y)[fs], want, absum, "conv fwd (many tiles)")


DGRAD_CASES = [(3, 42, 42, 16, 16), (3, 42, 42, 16, 32), (4, 21, 21, 32, 32), (7, 11, 11, 32, 32),
               (2, 42, 42, 32, 64), (3, 21, 21, 64, 64), (2, 17, 23, 16, 64)]


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("case", DGRAD_CASES, ids=lambda c: "n%d_%dx%d_%d-%d" % c)
@pytest.mark.parametrize("epi", ["plain", "mask_add"])
def test_conv_input_gradient(case, prec, epi):
    n, H, W, cin, cout = case
    rng = np.random.default_rng(21)
    dy = G.q(rng.standard_normal((n, H, W, cout)), prec)
    w = (rng.standard_normal((3, 3, cin, cout)) * np.sqrt(2.0 / (9 * cin))).astype(np.float32)
    mask = G.q(rng.standard_normal((n, H, W, cin)), prec) if epi == "mask_add" else None
    add = G.q(rng.standard_normal((n, H, W, cin)), prec) if epi == "mask_add" else None
    want = onet.conv3x3_dgrad(dy, G.q(w, prec))
    absum = onet.conv3x3_dgrad(np.abs(dy), np.abs(G.q(w, prec)))
    if mask is not None:
        want = want * (mask > 0) + add
        absum = absum * (mask > 0) + np.abs(add)
    out = G.empty_act((n, H, W, cin), prec)
    P.impala_conv3x3_dgrad(prec, n, H, W, cin, cout, G.dev_act(dy, prec), G.dev_f32(w),
                           G.dev_act(mask, prec) if mask is not None else None,
                           G.dev_act(add, prec) if add is not None else None, out)
    G.sync()
    if prec == G.BF16:
        G.assert_bf16_ulp(G.host(out), want, absum, "dgrad")
    else:
        G.assert_sum_close(G.host(out), want, absum, 1e-5, "dgrad")


# (n, H, W, cin, cout, x_mode, add): the network's backward convs (residual convs read relu(x),
# the second of a block adds the block's output gradient; stage entries read x as stored)
# plus ragged shapes, many frames per tile and several bands per frame
CONV_BWD_CASES = [
    (3, 42, 42, 16, 16, P.X_RELU, 1), (2, 42, 42, 16, 16, P.X_RELU, 0), (4, 21, 21, 32, 32, P.X_RELU, 1),
    (3, 21, 21, 32, 32, P.X_RELU, 0), (5, 11, 11, 32, 32, P.X_RELU, 1), (37, 11, 11, 32, 32, P.X_RELU, 0),
    (3, 42, 42, 16, 32, P.X_PLAIN, 0), (2, 21, 21, 32, 32, P.X_PLAIN, 0), (2, 17, 23, 16, 16, P.X_RELU, 1),
    (3, 9, 7, 32, 32, P.X_RELU, 1), (1, 84, 84, 16, 16, P.X_RELU, 1), (6, 5, 3, 16, 32, P.X_PLAIN, 0),
    # the wide net's 64-channel layers: bands of 21x21 frames, multi-frame 11x11 tiles, ragged
    (3, 21, 21, 64, 64, P.X_RELU, 1), (2, 21, 21, 64, 64, P.X_RELU, 0), (7, 11, 11, 64, 64, P.X_RELU, 1),
    (5, 11, 11, 64, 64, P.X_RELU, 0), (2, 13, 9, 64, 64, P.X_RELU, 1), (2, 21, 21, 64, 64, P.X_PLAIN, 0),
    (2, 42, 42, 32, 64, P.X_PLAIN, 0), (3, 7, 5, 32, 64, P.X_PLAIN, 0),
    # frame counts at which each workgroup runs several tiles (weight gradients accumulating)
    (300, 21, 21, 64, 64, P.X_RELU, 1), (400, 11, 11, 64, 64, P.X_RELU, 0), (300, 21, 21, 32, 32, P.X_RELU, 1),
]


@pytest.mark.parametrize("case", CONV_BWD_CASES, ids=lambda c: "n%d_%dx%d_%d-%d_m%d_a%d" % c)
def test_conv_backward_fused(case):
    """One-pass conv backward (bf16): dx against the exact adjoint (masked by x > 0 for relu
    inputs, plus the residual operand) to 1 bf16 ulp, dw and db against the exact sums."""
    n, H, W, cin, cout, mode, has_add = case
    rng = np.random.default_rng(41)
    x = G.q(rng.standard_normal((n, H, W, cin)), G.BF16)
    dy = G.q(rng.standard_normal((n, H, W, cout)), G.BF16)
    add = G.q(rng.standard_normal((n, H, W, cin)), G.BF16) if has_add else None
    w = (rng.standard_normal((3, 3, cin, cout)) * np.sqrt(2.0 / (9 * cin))).astype(np.float32)
    wq = G.q(w, G.BF16)
    xin = _relu(x) if mode == P.X_RELU else x
    want = onet.conv3x3_dgrad(dy, wq)
    absum = onet.conv3x3_dgrad(np.abs(dy), np.abs(wq))
    if mode == P.X_RELU:
        want, absum = want * (x > 0), absum * (x > 0)
    if add is not None:
        want, absum = want + add, absum + np.abs(add)
    want_w, want_b = onet.conv3x3_wgrad(xin, dy)
    abs_w, abs_b = onet.conv3x3_wgrad(np.abs(xin), np.abs(dy))
    dx = G.empty_act((n, H, W, cin), G.BF16)
    dw = G.dev_f32(np.full((3, 3, cin, cout), np.nan))
    db = G.dev_f32(np.full(cout, np.nan))
    ws = G.ws_bytes(P.impala_conv3x3_bwd_workspace_bytes(G.BF16, cin, cout))
    P.impala_conv3x3_bwd(G.BF16, n, H, W, cin, cout, G.dev_act(dy, G.BF16), G.dev_act(x, G.BF16), mode,
                         G.dev_f32(w), G.dev_act(add, G.BF16) if add is not None else None, dx, dw, db, ws)
    G.sync()
    G.assert_bf16_ulp(G.host(dx), want, absum, "conv_bwd dx")
    G.assert_sum_close(G.host(dw), want_w, abs_w, 1e-5, "conv_bwd dw")
    G.assert_sum_close(G.host(db), want_b, abs_b, 1e-5, "conv_bwd db")


# (n, H, W, C): the residual blocks' backward, base and ragged bands, tiny frames, and frame
# counts at which every workgroup of the persistent grid runs several tiles (its weight
# gradients accumulating over them)
RES_BWD_CASES = [(3, 42, 42, 16), (2, 17, 23, 16), (4, 9, 7, 16), (1, 84, 84, 16), (5, 3, 4, 16), (2, 43, 11, 16),
                 (4, 21, 21, 32), (5, 11, 11, 32), (3, 9, 7, 32), (2, 23, 17, 32), (1, 42, 42, 32),
                 (150, 42, 42, 16), (600, 11, 11, 32), (300, 21, 21, 32), (96, 42, 42, 32)]


def _resblock_bwd(n, H, W, C, dy, t, x, wa, wb):
    dx = G.empty_act((n, H, W, C), G.BF16)
    out = [G.dev_f32(np.full(shape, np.nan)) for shape in ((3, 3, C, C), (C,), (3, 3, C, C), (C,))]
    ws = G.ws_bytes(P.impala_resblock_bwd_workspace_bytes(G.BF16, C))
    P.impala_resblock_bwd(G.BF16, n, H, W, C, dy, t, x, wa, wb, dx, *out, ws)
    G.sync()
    return G.host(dx), [G.host(o) for o in out]


@pytest.mark.parametrize("case", RES_BWD_CASES, ids=lambda c: "n%d_%dx%d_c%d" % c)
def test_resblock_backward_fused(case):
    """Whole residual-block backward in one pass (bf16) against the exact sums. dy and conv_b's
    weights are small integers, so dt = conv_b^T(dy) * [t > 0] is an integer below 256: exact in
    float32 and in bf16 on both sides, and dx, the weight and bias gradients are checked to the
    usual bounds (dx to 1 bf16 ulp of the exact value, the sums to float32 accumulation)."""
    n, H, W, C = case
    rng = np.random.default_rng(53)
    x = G.q(rng.standard_normal((n, H, W, C)), G.BF16)
    t = G.q(rng.standard_normal((n, H, W, C)), G.BF16)
    dy = rng.choice([-1.0, 0.0, 0.0, 1.0], size=(n, H, W, C))
    wb = rng.choice([-1.0, 0.0, 0.0, 1.0], size=(3, 3, C, C)).astype(np.float32)
    wa = (rng.standard_normal((3, 3, C, C)) * np.sqrt(2.0 / (9 * C))).astype(np.float32)
    waq = G.q(wa, G.BF16)
    dt = onet.conv3x3_dgrad(dy, wb.astype(np.float64)) * (t > 0)
    assert np.array_equal(G.q(dt, G.BF16), dt) and np.abs(dt).max() < 256
    want_dx = onet.conv3x3_dgrad(dt, waq) * (x > 0) + dy
    abs_dx = onet.conv3x3_dgrad(np.abs(dt), np.abs(waq)) * (x > 0) + np.abs(dy)
    rt, rx = _relu(t), _relu(x)
    want_wb, want_bb = onet.conv3x3_wgrad(rt, dy)
    abs_wb, abs_bb = onet.conv3x3_wgrad(np.abs(rt), np.abs(dy))
    want_wa, want_ba = onet.conv3x3_wgrad(rx, dt)
    abs_wa, abs_ba = onet.conv3x3_wgrad(np.abs(rx), np.abs(dt))
    got_dx, (dwa, dba, dwb, dbb) = _resblock_bwd(n, H, W, C, G.dev_act(dy, G.BF16), G.dev_act(t, G.BF16),
                                                 G.dev_act(x, G.BF16), G.dev_f32(wa), G.dev_f32(wb))
    G.assert_bf16_ulp(got_dx, want_dx, abs_dx, "resblock_bwd dx")
    G.assert_sum_close(dwb, want_wb, abs_wb, 1e-5, "resblock_bwd dwb")
    G.assert_sum_close(dbb, want_bb, abs_bb, 1e-5, "resblock_bwd dbb")
    G.assert_sum_close(dwa, want_wa, abs_wa, 1e-5, "resblock_bwd dwa")
    G.assert_sum_close(dba, want_ba, abs_ba, 1e-5, "resblock_bwd dba")


@pytest.mark.parametrize("case", [(3, 42, 42, 16), (2, 17, 23, 16), (5, 3, 4, 16), (2, 21, 21, 32), (3, 11, 11, 32)],
                         ids=lambda c: "n%d_%dx%d_c%d" % c)
def test_resblock_backward_matches_two_conv_backwards(case):
    """On real-valued data the fused block backward equals the two single-conv backward passes
    it replaces: dt is rounded from the same float32 sums, so dx is bit-identical; the weight
    gradients are the same float32 sums in another order."""
    n, H, W, C = case
    rng = np.random.default_rng(59)
    x, t, dy = (G.q(rng.standard_normal((n, H, W, C)), G.BF16) for _ in range(3))
    wa, wb = (rng.standard_normal((2, 3, 3, C, C)) * np.sqrt(2.0 / (9 * C))).astype(np.float32)
    dyd, td, xd, wad, wbd = (G.dev_act(dy, G.BF16), G.dev_act(t, G.BF16), G.dev_act(x, G.BF16), G.dev_f32(wa),
                             G.dev_f32(wb))
    got_dx, (dwa, dba, dwb, dbb) = _resblock_bwd(n, H, W, C, dyd, td, xd, wad, wbd)
    ws = G.ws_bytes(P.impala_conv3x3_bwd_workspace_bytes(G.BF16, C, C))
    dt = G.empty_act((n, H, W, C), G.BF16)
    dx2 = G.empty_act((n, H, W, C), G.BF16)
    ref = [G.dev_f32(np.zeros(shape)) for shape in ((3, 3, C, C), (C,), (3, 3, C, C), (C,))]
    P.impala_conv3x3_bwd(G.BF16, n, H, W, C, C, dyd, td, P.X_RELU, wbd, None, dt, ref[2], ref[3], ws)
    P.impala_conv3x3_bwd(G.BF16, n, H, W, C, C, dt, xd, P.X_RELU, wad, dyd, dx2, ref[0], ref[1], ws)
    G.sync()
    np.testing.assert_array_equal(got_dx, G.host(dx2))
    dt_h = G.host(dt)
    abs_wa, abs_ba = onet.conv3x3_wgrad(np.abs(_relu(x)), np.abs(dt_h))
    abs_wb, abs_bb = onet.conv3x3_wgrad(np.abs(_relu(t)), np.abs(dy))
    for got, want, ab, what in ((dwa, ref[0], abs_wa, "dwa"), (dba, ref[1], abs_ba, "dba"),
                                (dwb, ref[2], abs_wb, "dwb"), (dbb, ref[3], abs_bb, "dbb")):
        G.assert_sum_close(got, G.host(want), 2.0 * ab, 1e-5, "resblock_bwd vs two launches " + what)


def test_resblock_backward_rejects_unsupported():
    z = G.dev_act(np.zeros((1, 8, 8, 64)), G.BF16)
    w = G.dev_f32(np.zeros((3, 3, 64, 64)))
    g = [G.dev_f32(np.zeros(shape)) for shape in ((3, 3, 64, 64), (64,), (3, 3, 64, 64), (64,))]
    with pytest.raises(P.LibraryError):   # 64 channels: not in the fused set
        P.impala_resblock_bwd(G.BF16, 1, 8, 8, 64, z, z, z, w, w, z, *g, G.ws_bytes(1 << 22))
    b16 = G.dev_act(np.zeros((1, 8, 8, 16)), G.BF16)
    w16 = G.dev_f32(np.zeros((3, 3, 16, 16)))
    g16 = [G.dev_f32(np.zeros(shape)) for shape in ((3, 3, 16, 16), (16,), (3, 3, 16, 16), (16,))]
    with pytest.raises(P.LibraryError):   # too small a workspace
        P.impala_resblock_bwd(G.BF16, 1, 8, 8, 16, b16, b16, b16, w16, w16, b16, *g16, G.ws_bytes(16))


# (n, H, W, cin, cout): stage entries fed by a max-pool (base and ragged, odd and even padding)
CONV_BWD_POOL_CASES = [(3, 42, 42, 16, 32), (2, 21, 21, 32, 32), (4, 42, 42, 16, 16), (2, 17, 23, 16, 32),
                       (5, 9, 7, 32, 32), (1, 84, 84, 16, 16), (3, 11, 11, 32, 32), (6, 4, 5, 16, 16),
                       (2, 42, 42, 32, 64), (3, 21, 21, 64, 64), (4, 9, 11, 32, 64), (5, 11, 11, 64, 64),
                       (80, 42, 42, 32, 64), (300, 21, 21, 64, 64), (200, 42, 42, 16, 32)]


@pytest.mark.parametrize("case", CONV_BWD_POOL_CASES, ids=lambda c: "n%d_%dx%d_%d-%d" % c)
def test_conv_backward_fused_pooled(case):
    """Stage-entry backward in one pass (bf16): the conv-output gradient is the max-pool
    backward of the pooled gradient (first-max rule, many ties), rounded to bf16 as the
    stand-alone pool backward stores it; dx to 1 bf16 ulp, dw and db against the exact sums."""
    n, H, W, cin, cout = case
    rng = np.random.default_rng(47)
    conv_out = rng.integers(-4, 5, size=(n, H, W, cout)).astype(np.float64) * 0.25
    _, arg = onet.maxpool(conv_out)
    OH, OW = arg.shape[1:3]
    dp = G.q(rng.standard_normal((n, OH, OW, cout)), G.BF16)
    dc = G.q(onet.maxpool_backward(arg, dp, (n, H, W, cout)), G.BF16)
    x = G.q(rng.standard_normal((n, H, W, cin)), G.BF16)
    w = (rng.standard_normal((3, 3, cin, cout)) * np.sqrt(2.0 / (9 * cin))).astype(np.float32)
    wq = G.q(w, G.BF16)
    want = onet.conv3x3_dgrad(dc, wq)
    absum = onet.conv3x3_dgrad(np.abs(dc), np.abs(wq))
    want_w, want_b = onet.conv3x3_wgrad(x, dc)
    abs_w, abs_b = onet.conv3x3_wgrad(np.abs(x), np.abs(dc))
    dx = G.empty_act((n, H, W, cin), G.BF16)
    dw = G.dev_f32(np.full((3, 3, cin, cout), np.nan))
    db = G.dev_f32(np.full(cout, np.nan))
    ws = G.ws_bytes(P.impala_conv3x3_bwd_workspace_bytes(G.BF16, cin, cout))
    P.impala_conv3x3_bwd(G.BF16, n, H, W, cin, cout, G.dev_act(dp, G.BF16), G.dev_act(x, G.BF16), P.X_PLAIN,
                         G.dev_f32(w), None, dx, dw, db, ws, pool_arg=G.dev_u8(arg))
    G.sync()
    G.assert_bf16_ulp(G.host(dx), want, absum, "conv_bwd pooled dx")
    G.assert_sum_close(G.host(dw), want_w, abs_w, 1e-5, "conv_bwd pooled dw")
    G.assert_sum_close(G.host(db), want_b, abs_b, 1e-5, "conv_bwd pooled db")


def test_conv_backward_fused_rejects_unsupported():
    ws = G.ws_bytes(1 << 20)
    z = G.dev_act(np.zeros((1, 8, 8, 64)), G.BF16)
    w = G.dev_f32(np.zeros((3, 3, 64, 64)))
    dw, db = G.dev_f32(np.zeros((3, 3, 64, 64))), G.dev_f32(np.zeros(64))
    z16 = G.dev_act(np.zeros((1, 8, 8, 16)), G.BF16)
    with pytest.raises(P.LibraryError):   # 16 -> 64 channels: not in the fused set
        P.impala_conv3x3_bwd(G.BF16, 1, 8, 8, 16, 64, z, z16, P.X_PLAIN, w, None, z16, dw, db, ws)
    z16 = G.dev_act(np.zeros((1, 8, 8, 16)), G.FP32)
    w16 = G.dev_f32(np.zeros((3, 3, 16, 16)))
    with pytest.raises(P.LibraryError):   # float32 storage
        P.impala_conv3x3_bwd(G.FP32, 1, 8, 8, 16, 16, z16, z16, P.X_RELU, w16, None, z16, dw, db, ws)
    b16 = G.dev_act(np.zeros((1, 8, 8, 16)), G.BF16)
    with pytest.raises(P.LibraryError):   # too small a workspace
        P.impala_conv3x3_bwd(G.BF16, 1, 8, 8, 16, 16, b16, b16, P.X_RELU, w16, None, b16, dw, db, G.ws_bytes(16))
    with pytest.raises(P.LibraryError):   # a pooled gradient feeds a plain (stage-entry) conv only
        P.impala_conv3x3_bwd(G.BF16, 1, 8, 8, 16, 16, b16, b16, P.X_RELU, w16, None, b16, dw, db, ws,
                             pool_arg=G.dev_u8(np.zeros((1, 4, 4, 16))))


# (n, H, W, cout): the first stage entry (base and wide) plus ragged and odd-padding shapes
POOL_WGRAD_CASES = [(3, 84, 84, 16), (2, 84, 84, 32), (4, 13, 9, 16), (3, 11, 11, 32), (2, 42, 42, 16),
                    (5, 7, 5, 16), (2, 23, 17, 32)]


@pytest.mark.parametrize("case", POOL_WGRAD_CASES, ids=lambda c: "n%d_%dx%d_c%d" % c)
def test_pool_wgrad_u8_fused(case):
    """First stage entry backward in one pass (bf16): the max-pool gradient dC (first-max rule,
    many ties), rounded to bf16 as the stand-alone pool backward stores it, contracted with the
    gathered frames / 255; dw and db against the exact sums."""
    n, H, W, C = case
    rng = np.random.default_rng(43)
    frames = rng.integers(0, 256, size=(n + 2, H, W, 4), dtype=np.uint8)
    rows = rng.permutation(n + 2)[:n].astype(np.int32)
    conv_out = rng.integers(-4, 5, size=(n, H, W, C)).astype(np.float64) * 0.25
    _, arg = onet.maxpool(conv_out)
    OH, OW = arg.shape[1:3]
    dp = G.q(rng.standard_normal((n, OH, OW, C)), G.BF16)
    dc = G.q(onet.maxpool_backward(arg, dp, (n, H, W, C)), G.BF16)
    xin = frames[rows].astype(np.float64) / 255.0
    want_w, want_b = onet.conv3x3_wgrad(xin, dc)
    abs_w, abs_b = onet.conv3x3_wgrad(xin, np.abs(dc))
    dw = G.dev_f32(np.full((3, 3, 4, C), np.nan))
    db = G.dev_f32(np.full(C, np.nan))
    ws = G.ws_bytes(P.impala_conv3x3_pool_wgrad_u8_workspace_bytes(G.BF16, C))
    P.impala_conv3x3_pool_wgrad_u8(G.BF16, n, H, W, C, G.dev_u8(frames), G.dev_i32(rows), G.dev_act(dp, G.BF16),
                                   G.dev_u8(arg), dw, db, ws)
    G.sync()
    G.assert_sum_close(G.host(dw), want_w, abs_w, 1e-5, "pool_wgrad dw")
    G.assert_sum_close(G.host(db), want_b, abs_b, 1e-5, "pool_wgrad db")



def test_pool_wgrad_u8_many_tiles_per_workgroup():
    """The first stage entry backward at a frame count where every workgroup runs several
    tiles (each tile's inputs are staged during the previous tile's weight gradient): the
    pooled gradient is non-zero on three frames spread over the launch only, so dw and db are
    those frames' exact sums."""
    n, H, W, C = 1024, 84, 84, 16
    pick = np.array([0, 517, n - 1])
    rng = np.random.default_rng(47)
    frames = rng.integers(0, 256, size=(n + 2, H, W, 4), dtype=np.uint8)
    rows = rng.permutation(n + 2)[:n].astype(np.int32)
    _, arg_p = onet.maxpool(rng.integers(-4, 5, size=(len(pick), H, W, C)).astype(np.float64) * 0.25)
    OH, OW = arg_p.shape[1:3]
    dp_p = G.q(rng.standard_normal((len(pick), OH, OW, C)), G.BF16)
    arg = np.zeros((n, OH, OW, C), np.uint8)
    arg[pick] = arg_p
    dp = np.zeros((n, OH, OW, C), np.float32)
    dp[pick] = dp_p
    dc = G.q(onet.maxpool_backward(arg_p, dp_p, (len(pick), H, W, C)), G.BF16)
    xin = frames[rows[pick]].astype(np.float64) / 255.0
    want_w, want_b = onet.conv3x3_wgrad(xin, dc)
    abs_w, abs_b = onet.conv3x3_wgrad(xin, np.abs(dc))
    dw = G.dev_f32(np.full((3, 3, 4, C), np.nan))
    db = G.dev_f32(np.full(C, np.nan))
    ws = G.ws_bytes(P.impala_conv3x3_pool_wgrad_u8_workspace_bytes(G.BF16, C))
    P.impala_conv3x3_pool_wgrad_u8(G.BF16, n, H, W, C, G.dev_u8(frames), G.dev_i32(rows), G.dev_act(dp, G.BF16),
                                   G.dev_u8(arg), dw, db, ws)
    G.sync()
    G.assert_sum_close(G.host(dw), want_w, abs_w, 1e-5, "pool_wgrad dw")
    G.assert_sum_close(G.host(db), want_b, abs_b, 1e-5, "pool_wgrad db")

def test_pool_wgrad_u8_rejects_unsupported():
    z8 = G.dev_u8(np.zeros((1, 8, 8, 4)))
    dp = G.dev_act(np.zeros((1, 4, 4, 64)), G.BF16)
    ag = G.dev_u8(np.zeros((1, 4, 4, 64)))
    dw, db = G.dev_f32(np.zeros((3, 3, 4, 64))), G.dev_f32(np.zeros(64))
    with pytest.raises(P.LibraryError):   # 64 output channels
        P.impala_conv3x3_pool_wgrad_u8(G.BF16, 1, 8, 8, 64, z8, None, dp, ag, dw, db, G.ws_bytes(1 << 22))
    with pytest.raises(P.LibraryError):   # float32 storage
        P.impala_conv3x3_pool_wgrad_u8(G.FP32, 1, 8, 8, 16, z8, None, dp, ag, dw, db, G.ws_bytes(1 << 22))
    with pytest.raises(P.LibraryError):   # workspace too small
        P.impala_conv3x3_pool_wgrad_u8(G.BF16, 1, 8, 8, 16, z8, None, dp, ag, dw, db, G.ws_bytes(16))


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "n%d_%dx%d_%d-%d_m%d" % c)
def test_conv_weight_gradient(case, prec):
    n, H, W, cin, cout, mode = case
    x, rows, xin, _, _ = _conv_inputs(n, H, W, cin, cout, mode, prec, 31)
    dy = G.q(np.random.default_rng(32).standard_normal((n, H, W, cout)), prec)
    want_w, want_b = onet.conv3x3_wgrad(xin, dy)
    abs_w, abs_b = onet.conv3x3_wgrad(np.abs(xin), np.abs(dy))
    dw = G.dev_f32(np.zeros((3, 3, cin, cout)))
    db = G.dev_f32(np.zeros(cout))
    ws = G.ws_bytes(P.impala_conv3x3_wgrad_workspace_bytes(prec, H, W, cin, cout))
    dx = G.dev_u8(x) if mode == P.X_U8 else G.dev_act(x, prec)
    P.impala_conv3x3_wgrad(prec, n, H, W, cin, cout, dx, mode,
                           G.dev_i32(rows) if rows is not None else None, G.dev_act(dy, prec), dw, db, ws)
    G.sync()
    G.assert_sum_close(G.host(dw), want_w, abs_w, 1e-5, "wgrad w")
    G.assert_sum_close(G.host(db), want_b, abs_b, 1e-5, "wgrad b")


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("shape", [(3, 84, 84, 16), (2, 42, 42, 32), (5, 21, 21, 32), (2, 11, 11, 64),
                                   (3, 7, 9, 16)], ids=lambda s: "n%d_%dx%dx%d" % s)
def test_maxpool_forward_backward(shape, prec):
    n, H, W, C = shape
    rng = np.random.default_rng(41)
    # small integers: many exact ties, so the first-max rule is exercised
    x = rng.integers(-4, 5, size=shape).astype(np.float64) * 0.25
    y_want, arg_want = onet.maxpool(x)
    OH, OW = y_want.shape[1:3]
    y = G.empty_act((n, OH, OW, C), prec)
    torch = G.torch()
    arg = torch.empty((n, OH, OW, C), dtype=torch.uint8, device="cuda:0")
    P.impala_maxpool_fwd(prec, n, H, W, C, G.dev_act(x, prec), y, arg)
    dy = G.q(rng.standard_normal(y_want.shape), prec)
    dx = G.empty_act(shape, prec)
    P.impala_maxpool_bwd(prec, n, H, W, C, arg, G.dev_act(dy, prec), dx)
    G.sync()
    np.testing.assert_array_equal(G.host(y), y_want)
    np.testing.assert_array_equal(arg.cpu().numpy(), arg_want)
    want_dx = onet.maxpool_backward(arg_want, dy, shape)
    abs_dx = onet.maxpool_backward(arg_want, np.abs(dy), shape)
    if prec == G.BF16:
        G.assert_bf16_ulp(G.host(dx), want_dx, abs_dx, "pool bwd")
    else:
        G.assert_sum_close(G.host(dx), want_dx, abs_dx, 1e-6, "pool bwd")


@pytest.mark.parametrize("T,E", [(128, 64), (20, 64), (37, 100), (1, 3), (8, 4), (128, 128), (65, 257)])
def test_gae_matches_oracle(T, E):
    rng = np.random.default_rng(T * 1000 + E)
    r = rng.choice([-1.0, 0.0, 1.0], size=(T, E), p=[.05, .9, .05]).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < 0.05).astype(np.uint8)
    nv = rng.standard_normal(E).astype(np.float32)
    nd = (rng.random(E) < 0.05).astype(np.uint8)
    adv_w, ret_w = otargets.gae(r, v, d, nv, nd, 0.99, 0.95)
    adv, ret = G.dev_f32(np.zeros((T, E))), G.dev_f32(np.zeros((T, E)))
    P.gae_advantages(T, E, G.dev_f32(r), G.dev_f32(v), G.dev_u8(d), G.dev_f32(nv), G.dev_u8(nd),
                     0.99, 0.95, adv, ret)
    G.sync()
    G.assert_close(G.host(adv), adv_w, 1e-5, "adv")
    G.assert_close(G.host(ret), ret_w, 1e-5, "ret")


@pytest.mark.parametrize("T,E,lam,rho,cbar", [(20, 64, 1.0, 1.0, 1.0), (128, 70, 0.95, 1.0, 1.0),
                                              (33, 5, 1.0, 0.8, 1.2), (1, 1, 1.0, 1.0, 1.0)])
def test_vtrace_matches_oracle(T, E, lam, rho, cbar):
    rng = np.random.default_rng(7 * T + E)
    r = rng.choice([-1.0, 0.0, 1.0], size=(T, E), p=[.05, .9, .05]).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < 0.05).astype(np.uint8)
    bv = rng.standard_normal(E).astype(np.float32)
    nd = (rng.random(E) < 0.05).astype(np.uint8)
    mu = (rng.standard_normal((T, E)) * 0.5 - 2).astype(np.float32)
    pi = (mu + 0.3 * rng.standard_normal((T, E))).astype(np.float32)
    vs_w, pg_w = otargets.vtrace(mu, pi, r, v, d, bv, nd, 0.99, lam, rho, cbar, 1.0)
    vs, pg = G.dev_f32(np.zeros((T, E))), G.dev_f32(np.zeros((T, E)))
    P.vtrace_targets(T, E, G.dev_f32(mu), G.dev_f32(pi), G.dev_f32(r), G.dev_f32(v), G.dev_u8(d),
                     G.dev_f32(bv), G.dev_u8(nd), 0.99, lam, rho, cbar, 1.0, vs, pg)
    G.sync()
    G.assert_close(G.host(vs), vs_w, 1e-5, "vs")
    G.assert_close(G.host(pg), pg_w, 1e-5, "pg_adv")


def _loss_batch(m, A, seed):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((m, A)) * 3).astype(np.float32)
    a = rng.integers(0, A, m).astype(np.int32)
    lp = olosses.log_softmax(z.astype(np.float64))[np.arange(m), a]
    return dict(z=z, v=rng.standard_normal(m).astype(np.float32), a=a,
                old=(lp + 0.1 * rng.standard_normal(m)).astype(np.float32),
                adv=(rng.standard_normal(m) * 2 + 0.3).astype(np.float32),
                ret=rng.standard_normal(m).astype(np.float32),
                vs=rng.standard_normal(m).astype(np.float32),
                pg=rng.standard_normal(m).astype(np.float32))


@pytest.mark.parametrize("m,A,norm", [(2048, 18, 1), (32, 6, 1), (8192, 18, 1), (1000, 7, 0), (1, 18, 0),
                                      (16385, 18, 1), (70001, 7, 1), (262144, 18, 1), (40000, 6, 0)])
def test_ppo_loss_matches_oracle(m, A, norm):
    """Against the oracle without a workspace; with one, the same outputs bit for bit."""
    b = _loss_batch(m, A, m + A)
    L, dz_w, dv_w, st_w = olosses.ppo_loss_grad(b["z"], b["v"], b["a"], b["old"], b["adv"], b["ret"],
                                                0.1, 0.5, 0.01, bool(norm))
    outs = []
    for ws in (None, G.ws_bytes(P.loss_workspace_bytes(m))):
        dz, dv, st = G.dev_f32(np.zeros((m, A))), G.dev_f32(np.zeros(m)), G.dev_f32(np.zeros(8))
        P.ppo_loss_grad(m, A, G.dev_f32(b["z"]), G.dev_f32(b["v"]), G.dev_i32(b["a"]), G.dev_f32(b["old"]),
                        G.dev_f32(b["adv"]), G.dev_f32(b["ret"]), norm, 0.1, 0.5, 0.01, dz, dv, st, ws)
        G.sync()
        outs.append((dz, dv, st))
    dz, dv, st = outs[0]
    G.assert_close(G.host(dz), dz_w, 1e-5, "dlogits")
    G.assert_close(G.host(dv), dv_w, 1e-5, "dvalue")
    got = G.host(st)
    idx = [0, 1, 2, 3, 4, 6, 7] if m > 1 else [0, 1, 2, 3, 4, 6]
    G.assert_close(got[idx], st_w[idx], 1e-5, "stats")
    assert abs(got[5] - st_w[5]) <= 1.0 / m   # clip fraction: a count over rows
    torch = G.torch()
    assert all(torch.equal(x, y) for x, y in zip(outs[0], outs[1]))


@pytest.mark.parametrize("m,A", [(1280, 18), (37, 6), (4096, 64), (16385, 18), (50001, 6), (262144, 18),
                                 (20000, 64)])
def test_impala_loss_matches_oracle(m, A):
    """Against the oracle without a workspace; with one, the same outputs bit for bit."""
    b = _loss_batch(m, A, 3 * m + A)
    L, dz_w, dv_w, st_w = olosses.impala_loss_grad(b["z"], b["v"], b["a"], b["vs"], b["pg"], 1.0, 0.5, 0.01)
    outs = []
    for ws in (None, G.ws_bytes(P.loss_workspace_bytes(m))):
        dz, dv, st = G.dev_f32(np.zeros((m, A))), G.dev_f32(np.zeros(m)), G.dev_f32(np.zeros(8))
        P.impala_loss_grad(m, A, G.dev_f32(b["z"]), G.dev_f32(b["v"]), G.dev_i32(b["a"]), G.dev_f32(b["vs"]),
                           G.dev_f32(b["pg"]), 1.0, 0.5, 0.01, dz, dv, st, ws)
        G.sync()
        outs.append((dz, dv, st))
    dz, dv, st = outs[0]
    G.assert_close(G.host(dz), dz_w, 1e-5, "dlogits")
    G.assert_close(G.host(dv), dv_w, 1e-5, "dvalue")
    G.assert_close(G.host(st)[:6], st_w[:6], 1e-5, "stats")
    torch = G.torch()
    assert all(torch.equal(x, y) for x, y in zip(outs[0], outs[1]))


@pytest.mark.parametrize("n,scale,max_norm,step", [(1_094_115, 1e-3, 0.5, 1), (1_094_115, 10.0, 0.5, 7),
                                                    (4_364_211, 1.0, 40.0, 3), (1001, 1.0, 0.0, 2),
                                                    (3, 1.0, 0.5, 1)])
def test_adam_matches_oracle(n, scale, max_norm, step):
    rng = np.random.default_rng(n + step)
    p = rng.standard_normal(n).astype(np.float32)
    g = (rng.standard_normal(n) * scale / np.sqrt(n) * 30).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = (rng.random(n) * 1e-5).astype(np.float32)
    # the library receives float32 hyperparameters; the oracle gets the same values
    f = lambda x: float(np.float32(x))  # noqa: E731
    gc, norm = ooptim.clip_by_global_norm(g, f(max_norm))
    pw, mw, vw = ooptim.adam(p, gc, m, v, step, f(2.5e-4), f(0.9), f(0.999), f(1e-5))
    dp, dg, dm, dv = G.dev_f32(p), G.dev_f32(g), G.dev_f32(m), G.dev_f32(v)
    st = G.dev_f32(np.zeros(2))
    ws = G.ws_bytes(P.adam_workspace_bytes(n))
    P.adam_step(n, dp, dg, dm, dv, step, 2.5e-4, 0.9, 0.999, 1e-5, max_norm, st, ws)
    G.sync()
    G.assert_close(G.host(dm), mw, 1e-5, "m")
    G.assert_close(G.host(dv), vw, 1e-5, "v")
    # the new float32 parameter can only be as exact as its own rounding: within 2 ulps
    # of the oracle's value, plus 1e-5 of the update
    got_p = G.host(dp)
    ulp = np.spacing(np.abs(pw).astype(np.float32)).astype(np.float64)
    assert (np.abs(got_p - pw) <= 2 * ulp + 1e-5 * np.abs(pw - p)).all()
    G.assert_close(got_p - p, pw - p, 1e-3, "param update")
    s = G.host(st)
    assert abs(s[0] - norm) <= 1e-5 * norm and s[1] == 0


@pytest.mark.parametrize("n,scale,max_norm", [(1_094_115, 1e-3, 40.0), (1_094_115, 100.0, 40.0),
                                             (4_364_211, 1.0, 0.5), (1001, 1.0, 0.0), (3, 1.0, 40.0)])
def test_rmsprop_matches_oracle(n, scale, max_norm):
    """Appendix B's IMPALA optimiser (decay 0.99, eps 0.01) after the global-norm clip."""
    rng = np.random.default_rng(n + 17)
    p = rng.standard_normal(n).astype(np.float32)
    g = (rng.standard_normal(n) * scale / np.sqrt(n) * 30).astype(np.float32)
    nu = (rng.random(n) * 1e-3).astype(np.float32)
    f = lambda x: float(np.float32(x))  # noqa: E731
    gc, norm = ooptim.clip_by_global_norm(g, f(max_norm))
    pw, nuw = ooptim.rmsprop(p, gc, nu, f(6e-4), f(0.99), f(0.01))
    dp, dg, dnu = G.dev_f32(p), G.dev_f32(g), G.dev_f32(nu)
    st = G.dev_f32(np.zeros(2))
    ws = G.ws_bytes(P.rmsprop_workspace_bytes(n))
    P.rmsprop_step(n, dp, dg, dnu, 6e-4, 0.99, 0.01, max_norm, st, ws)
    G.sync()
    G.assert_close(G.host(dnu), nuw, 1e-5, "nu")
    got_p = G.host(dp)
    ulp = np.spacing(np.abs(pw).astype(np.float32)).astype(np.float64)
    assert (np.abs(got_p - pw) <= 2 * ulp + 1e-5 * np.abs(pw - p)).all()
    # the step is proportional to g while g^2 << eps: for small gradients it is a few ulps of
    # the parameter, so the step itself is compared where it spans at least 1024 ulps (the
    # result's own rounding then stays below 5e-4 of the step)
    big = np.abs(pw - p) >= 1024 * ulp
    if big.sum() >= 16:
        G.assert_close(got_p[big] - p[big], (pw - p)[big], 1e-3, "param update")
    s = G.host(st)
    assert abs(s[0] - norm) <= 1e-5 * norm and s[1] == 0


@pytest.mark.parametrize("n,A", [(128, 18), (1000, 6), (7, 64)])
def test_gumbel_sample_bit_exact(n, A):
    rng = np.random.default_rng(n)
    z = (rng.standard_normal((n, A)) * 2).astype(np.float32)
    z[::5, 1] = z[::5, 0]                           # exact ties in the logits
    g = rng.gumbel(size=(n, A)).astype(np.float32)
    g[::7] = 0.0                                     # ties in z + g, resolved to the lowest index
    a_w, lp_w = olosses.gumbel_max(z, g)
    act, lp = G.dev_i32(np.zeros(n)), G.dev_f32(np.zeros(n))
    P.impala_gumbel_sample(n, A, G.dev_f32(z), G.dev_f32(g), act, lp)
    G.sync()
    np.testing.assert_array_equal(act.cpu().numpy(), a_w)
    G.assert_close(G.host(lp), olosses.log_softmax(z.astype(np.float64))[np.arange(n), a_w], 1e-5, "logp")


def test_mfma_probe_runs_its_matrix_products():
    """The matrix-core probe does the MFMAs it counts: every thread's checksum equals the sum,
    written out, of its lane's accumulator rows (16x16x32 products of the per-lane bf16
    operands it builds, exact in float32), and two launches agree bit for bit."""
    import torch
    blocks, iters = 8, 16
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    flop = P.impala_probe_mfma_bf16(blocks, iters, sink)
    assert flop == blocks * 4 * iters * 8 * (16 * 16 * 32 * 2)
    G.sync()
    first = sink.cpu().numpy().copy()
    P.impala_probe_mfma_bf16(blocks, iters, sink)
    G.sync()
    np.testing.assert_array_equal(first, sink.cpu().numpy())
    # A[i][8g+m] = x[i+16g] (m even) or 1, B[8g+m][n] = y[n+16g] (m even) or 0.5, lane l
    # supplying row / column l % 16 for k = 8(l // 16) .. +7 and receiving rows 4(l // 16) .. +3
    x = 1.0 + np.arange(64) / 128.0
    y = 1.0 - np.arange(64) / 256.0
    D = np.zeros((16, 16))
    for g in range(4):
        D += 4.0 * np.outer(x[16 * g:16 * g + 16], y[16 * g:16 * g + 16]) + 2.0
    lane = np.arange(256) % 64
    want = np.array([8 * iters * D[4 * (l // 16):4 * (l // 16) + 4, l % 16].sum() for l in lane])
    # the MFMA sums are exact (15 fractional bits, below 2^9); the 32-term float32 checksum rounds
    np.testing.assert_allclose(first.reshape(blocks, 256), np.broadcast_to(want, (blocks, 256)), rtol=1e-5)
