"""Pins of the oracle's network against brute force and finite differences (CPU only)."""
import numpy as np
import pytest

from oracle import losses, net as onet
from synth import NetShape, draw_params, param_count as synth_count, param_shapes


def brute_conv(x, w, b):
    n, h, wd, ci = x.shape
    co = w.shape[3]
    y = np.zeros((n, h, wd, co))
    for a in range(n):
        for i in range(h):
            for j in range(wd):
                for o in range(co):
                    s = b[o]
                    for ky in range(3):
                        for kx in range(3):
                            ii, jj = i + ky - 1, j + kx - 1
                            if 0 <= ii < h and 0 <= jj < wd:
                                for c in range(ci):
                                    s += x[a, ii, jj, c] * w[ky, kx, c, o]
                    y[a, i, j, o] = s
    return y


def test_conv_matches_brute_force():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 5, 4, 3))
    w = rng.standard_normal((3, 3, 3, 2))
    b = rng.standard_normal(2)
    np.testing.assert_allclose(onet.conv3x3(x, w, b), brute_conv(x, w, b), rtol=1e-12, atol=1e-12)


def test_conv_adjoints_by_inner_product():
    # <conv(x) - b, dy> = <x, dgrad(dy)> = <w, wgrad(x, dy)>: bilinearity fixes both adjoints.
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 6, 5, 3))
    w = rng.standard_normal((3, 3, 3, 4))
    dy = rng.standard_normal((2, 6, 5, 4))
    lhs = np.sum((onet.conv3x3(x, w, np.zeros(4))) * dy)
    assert np.isclose(lhs, np.sum(x * onet.conv3x3_dgrad(dy, w)), rtol=1e-12)
    dw, db = onet.conv3x3_wgrad(x, dy)
    assert np.isclose(lhs, np.sum(w * dw), rtol=1e-12)
    np.testing.assert_allclose(db, dy.sum((0, 1, 2)), rtol=1e-12)


@pytest.mark.parametrize("size,expect", [(84, (42, 0, 1)), (42, (21, 0, 1)), (21, (11, 1, 1)),
                                         (12, (6, 0, 1)), (6, (3, 0, 1)), (3, (2, 1, 1))])
def test_same_pool_geometry(size, expect):
    assert onet.same_pool_pads(size) == expect


def brute_pool(x):
    n, h, w, c = x.shape
    oh, plo, _ = onet.same_pool_pads(h)
    ow, qlo, _ = onet.same_pool_pads(w)
    y = np.zeros((n, oh, ow, c))
    arg = np.zeros((n, oh, ow, c), int)
    for a in range(n):
        for i in range(oh):
            for j in range(ow):
                for k in range(c):
                    best, bi = -np.inf, -1
                    for t, (dy, dx) in enumerate([(u, v) for u in range(3) for v in range(3)]):
                        ii, jj = 2 * i + dy - plo, 2 * j + dx - qlo
                        if 0 <= ii < h and 0 <= jj < w and x[a, ii, jj, k] > best:
                            best, bi = x[a, ii, jj, k], t
                    y[a, i, j, k], arg[a, i, j, k] = best, bi
    return y, arg


@pytest.mark.parametrize("h,w", [(12, 12), (7, 9), (21, 21), (3, 3)])
def test_maxpool_matches_brute_force(h, w):
    rng = np.random.default_rng(h * 31 + w)
    x = rng.integers(-3, 4, size=(2, h, w, 2)).astype(np.float64)   # many ties
    y, arg = onet.maxpool(x)
    yb, ab = brute_pool(x)
    np.testing.assert_array_equal(y, yb)
    np.testing.assert_array_equal(arg, ab)


def test_maxpool_backward_is_adjoint_of_selection():
    # With the argmax fixed, pooling is linear selection; its adjoint routes dy back.
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 9, 8, 3))
    y, arg = onet.maxpool(x)
    dy = rng.standard_normal(y.shape)
    dx = onet.maxpool_backward(arg, dy, x.shape)
    eps = 1e-7
    d = rng.standard_normal(x.shape)
    y2, arg2 = onet.maxpool(x + eps * d)
    assert np.array_equal(arg, arg2)
    assert np.isclose(np.sum((y2 - y) / eps * dy), np.sum(d * dx), rtol=1e-6)


def test_param_layout_counts():
    base = NetShape()
    assert onet.param_count(base) == 1_094_115
    assert onet.param_count(NetShape(num_actions=6)) == 1_091_031
    assert onet.param_count(NetShape(ch=(32, 64, 64), hidden=512)) == 4_364_211
    assert len(onet.param_layout(base)) == 36
    for n in (base, NetShape(ch=(32, 64, 64), hidden=512)):
        assert [(a, tuple(s)) for a, s, _ in onet.param_layout(n)] == \
               [(a, tuple(s)) for a, s, _ in param_shapes(n)]
        assert onet.param_count(n) == synth_count(n)


def test_bf16_round_known_values():
    vals = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -7, -2.5, 3.0e38, 1 + 2 ** -9], np.float32)
    want = np.array([1.0, 1.0, 1 + 2 ** -6, 1 + 2 ** -7, -2.5, 2.9975e38, 1.0], np.float32)
    got = onet.bf16_round(vals)
    np.testing.assert_array_equal(got[[0, 1, 2, 3, 4, 6]], want[[0, 1, 2, 3, 4, 6]])
    assert abs(got[5] - 3.0e38) / 3.0e38 < 2 ** -8


def _loss_of_params(net, flat, obs, aux, algo):
    z, v, cache = onet.forward(net, flat, obs)
    if algo == "ppo":
        L, dz, dv, _ = losses.ppo_loss_grad(z, v, aux["a"], aux["old"], aux["adv"], aux["ret"],
                                            0.1, 0.5, 0.01, True, adv_stats=aux["stats"])
    else:
        L, dz, dv, _ = losses.impala_loss_grad(z, v, aux["a"], aux["vs"], aux["pg"], 1.0, 0.5, 0.01)
    return L, dz, dv, cache


@pytest.mark.parametrize("algo", ["ppo", "impala"])
def test_network_gradient_finite_differences(tiny_net, algo):
    """Central differences in float64 on every one of the 36 parameter tensors."""
    net = tiny_net
    rng = np.random.default_rng(7 if algo == "ppo" else 8)
    flat = draw_params(net, 11).astype(np.float64)
    flat += 0.05 * rng.standard_normal(flat.shape)          # non-zero biases too
    obs = rng.integers(0, 256, size=(4, net.in_h, net.in_w, net.in_c), dtype=np.uint8)
    z0, _, _ = onet.forward(net, flat, obs)
    a = rng.integers(0, net.num_actions, 4)
    adv = rng.standard_normal(4)
    aux = dict(a=a, old=losses.log_softmax(z0)[np.arange(4), a] + 0.3 * rng.standard_normal(4),
               adv=adv, ret=rng.standard_normal(4), stats=(adv.mean(), adv.std()),
               vs=rng.standard_normal(4), pg=rng.standard_normal(4))
    _, dz, dv, cache = _loss_of_params(net, flat, obs, aux, algo)
    grad = onet.backward(net, cache, dz, dv)
    h = 1e-6
    for name, shape, off in onet.param_layout(net):
        size = int(np.prod(shape))
        idx = rng.choice(size, size=min(size, 5), replace=False) + off
        for i in idx:
            fp, fm = flat.copy(), flat.copy()
            fp[i] += h
            fm[i] -= h
            lp = _loss_of_params(net, fp, obs, aux, algo)[0]
            lm = _loss_of_params(net, fm, obs, aux, algo)[0]
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad[i]) <= 1e-6 * max(1.0, abs(grad[i])) + 1e-8, (name, i, fd, grad[i])


def test_forward_scaling_of_obs(tiny_net):
    """Frames enter as obs/255: a net whose first conv weights are scaled by 255 and fed
    obs/255-equivalent bytes gives the same logits as the unscaled definition."""
    net = tiny_net
    rng = np.random.default_rng(3)
    flat = draw_params(net, 2).astype(np.float64)
    obs = rng.integers(0, 256, size=(2, net.in_h, net.in_w, net.in_c), dtype=np.uint8)
    z, v, _ = onet.forward(net, flat, obs)
    P = onet.unflatten(flat, net)
    x = obs / 255.0
    c = onet.conv3x3(x, P["s0.conv.w"], P["s0.conv.b"])
    c255 = onet.conv3x3(obs.astype(np.float64), P["s0.conv.w"], 255 * P["s0.conv.b"]) / 255
    np.testing.assert_allclose(c, c255, rtol=1e-12, atol=1e-12)
    assert z.shape == (2, net.num_actions) and v.shape == (2,)
