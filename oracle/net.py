"""IMPALA-ResNet forward and backward, written out as plain definitions.

The paper trains every agent with "IMPALA's ResNet" (Section 5, Experiments) and does not
print it; this follows the network of Espeholt et al. (2018, Fig. 3, large architecture) as
Cleanba instantiates it: for each stage width c, a 3x3 stride-1 SAME conv, a 3x3 stride-2 SAME
max-pool, then two pre-activation residual blocks ``x + conv(relu(conv(relu(x))))``; then
ReLU, flatten in (H, W, C) order, a dense ReLU layer, and linear policy-logit and value heads.
Frames are NHWC uint8 scaled by 1/255.

Conventions (recorded as readings in the design notes):
* conv weights HWIO [3,3,Cin,Cout]; dense weights [in, out]; biases added after the sum;
* SAME conv pads one zero on every side;
* SAME max-pool uses XLA's split of the padding (lo = P // 2, hi = P - lo) with -inf fill;
* the max-pool gradient goes to the first maximal element of each window in row-major
  (dy, dx) order; overlapping windows add up;
* relu'(0) = 0.
"""
from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------- layout


def out_hw(h: int, w: int) -> tuple:
    """Spatial size after one stride-2 SAME pool: ceil(h/2) x ceil(w/2)."""
    return -(-h // 2), -(-w // 2)


def param_layout(net) -> list:
    """[(name, shape, offset)] of the 36 tensors in the flat parameter buffer.

    Order: per stage the entry conv (w, b), then block0 conv0, block0 conv1, block1 conv0,
    block1 conv1 (w, b each); then dense, logits, value (w, b each).
    """
    shapes = []
    cin = net.in_c
    h, w = net.in_h, net.in_w
    for s, c in enumerate(net.ch):
        shapes += [(f"s{s}.conv.w", (3, 3, cin, c)), (f"s{s}.conv.b", (c,))]
        for r in range(2):
            for k in range(2):
                shapes += [(f"s{s}.res{r}.conv{k}.w", (3, 3, c, c)), (f"s{s}.res{r}.conv{k}.b", (c,))]
        cin = c
        h, w = out_hw(h, w)
    flat = h * w * net.ch[2]
    shapes += [("dense.w", (flat, net.hidden)), ("dense.b", (net.hidden,)),
               ("logits.w", (net.hidden, net.num_actions)), ("logits.b", (net.num_actions,)),
               ("value.w", (net.hidden, 1)), ("value.b", (1,))]
    out, off = [], 0
    for name, shape in shapes:
        out.append((name, shape, off))
        off += int(np.prod(shape))
    return out


def param_count(net) -> int:
    name, shape, off = param_layout(net)[-1]
    return off + int(np.prod(shape))


def unflatten(flat: np.ndarray, net) -> dict:
    return {name: flat[off:off + int(np.prod(shape))].reshape(shape)
            for name, shape, off in param_layout(net)}


def flatten(tensors: dict, net) -> np.ndarray:
    return np.concatenate([np.asarray(tensors[name]).ravel() for name, _, _ in param_layout(net)])


# ----------------------------------------------------------------------------- precision


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    rounded = ((bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    out = rounded.view(np.float32).copy()
    nan = np.isnan(x)
    out[nan] = x[nan]
    return out


def _mode(prec: str):
    if prec == "fp64":
        return np.float64, (lambda a: a)
    if prec == "fp32":
        return np.float32, (lambda a: a)
    if prec == "bf16":
        return np.float32, bf16_round
    raise ValueError(prec)


def relu(x):
    return np.maximum(x, 0)


# ----------------------------------------------------------------------------- conv / pool


def _pad1(x):
    n, h, w, c = x.shape
    xp = np.zeros((n, h + 2, w + 2, c), x.dtype)
    xp[:, 1:-1, 1:-1] = x
    return xp


def conv3x3(x, w, b):
    """y[n,i,j,:] = b + sum over taps (ky,kx) of xpad[n,i+ky,j+kx,:] @ w[ky,kx]."""
    n, h, wd, ci = x.shape
    co = w.shape[3]
    xp = _pad1(x)
    y = np.empty((n, h, wd, co), x.dtype)
    y[...] = b
    for ky in range(3):
        for kx in range(3):
            tap = np.ascontiguousarray(xp[:, ky:ky + h, kx:kx + wd, :]).reshape(-1, ci)
            y += (tap @ w[ky, kx]).reshape(n, h, wd, co)
    return y


def conv3x3_wgrad(x, dy):
    """dL/dw[ky,kx] = sum over pixels of xpad-tap^T dy; dL/db = sum over pixels of dy."""
    n, h, wd, ci = x.shape
    co = dy.shape[3]
    xp = _pad1(x)
    dy2 = dy.reshape(-1, co)
    dw = np.empty((3, 3, ci, co), x.dtype)
    for ky in range(3):
        for kx in range(3):
            dw[ky, kx] = np.ascontiguousarray(xp[:, ky:ky + h, kx:kx + wd, :]).reshape(-1, ci).T @ dy2
    return dw, dy2.sum(0)


def conv3x3_dgrad(dy, w):
    """Adjoint of conv3x3 w.r.t. its input: scatter dy @ w[ky,kx]^T back onto every tap."""
    n, h, wd, co = dy.shape
    ci = w.shape[2]
    dxp = np.zeros((n, h + 2, wd + 2, ci), dy.dtype)
    dy2 = dy.reshape(-1, co)
    for ky in range(3):
        for kx in range(3):
            dxp[:, ky:ky + h, kx:kx + wd, :] += (dy2 @ w[ky, kx].T).reshape(n, h, wd, ci)
    return dxp[:, 1:-1, 1:-1, :]


def same_pool_pads(size: int) -> tuple:
    """(out, pad_lo, pad_hi) of a 3-wide stride-2 SAME window over ``size`` (XLA split)."""
    out = -(-size // 2)
    p = max((out - 1) * 2 + 3 - size, 0)
    return out, p // 2, p - p // 2


_WIN = [(dy, dx) for dy in range(3) for dx in range(3)]


def _pool_views(xp, oh, ow):
    return [xp[:, dy:dy + 2 * oh - 1:2, dx:dx + 2 * ow - 1:2, :] for dy, dx in _WIN]


def maxpool(x):
    """3x3 stride-2 SAME max-pool; returns (y, arg) with arg the first argmax in 0..8."""
    n, h, w, c = x.shape
    oh, ph0, ph1 = same_pool_pads(h)
    ow, pw0, pw1 = same_pool_pads(w)
    xp = np.full((n, h + ph0 + ph1, w + pw0 + pw1, c), -np.inf, x.dtype)
    xp[:, ph0:ph0 + h, pw0:pw0 + w] = x
    stack = np.stack(_pool_views(xp, oh, ow))
    arg = stack.argmax(0)
    y = np.take_along_axis(stack, arg[None], 0)[0]
    return y, arg


def maxpool_backward(arg, dy, in_shape):
    """Route each window's gradient to its argmax; overlapping windows add."""
    n, h, w, c = in_shape
    oh, ph0, ph1 = same_pool_pads(h)
    ow, pw0, pw1 = same_pool_pads(w)
    dxp = np.zeros((n, h + ph0 + ph1, w + pw0 + pw1, c), dy.dtype)
    for k, view in enumerate(_pool_views(dxp, oh, ow)):
        view += np.where(arg == k, dy, 0)
    return dxp[:, ph0:ph0 + h, pw0:pw0 + w]


# ----------------------------------------------------------------------------- network


def forward(net, params, obs, prec: str = "fp64"):
    """Policy logits [n, A] and value [n] of uint8 frames obs [n, H, W, C].

    Returns (logits, value, cache); the cache holds what the backward pass reads.
    """
    dt, q = _mode(prec)
    P = unflatten(np.asarray(params, dtype=dt), net)
    W = {k: (q(v) if k.endswith(".w") else v) for k, v in P.items()}
    x = obs.astype(dt) / dt(255.0)
    cache = {"n": obs.shape[0]}
    for s in range(3):
        c = q(conv3x3(x, W[f"s{s}.conv.w"], W[f"s{s}.conv.b"]))
        p, arg = maxpool(c)
        cache[f"s{s}"] = (x, arg, c.shape)
        x = p
        for r in range(2):
            pre = f"s{s}.res{r}"
            t = q(conv3x3(relu(x), W[pre + ".conv0.w"], W[pre + ".conv0.b"]))
            y = q(x + conv3x3(relu(t), W[pre + ".conv1.w"], W[pre + ".conv1.b"]))
            cache[pre] = (x, t)
            x = y
    n = x.shape[0]
    f = relu(x).reshape(n, -1)
    h = q(relu(f @ W["dense.w"] + W["dense.b"]))
    logits = h @ W["logits.w"] + W["logits.b"]
    value = (h @ W["value.w"] + W["value.b"])[:, 0]
    cache.update(last=x, f=f, h=h, W=W, prec=prec)
    return logits, value, cache


def backward(net, cache, dlogits, dvalue):
    """Flat gradient of sum(dlogits * logits) + sum(dvalue * value) w.r.t. every parameter."""
    dt, q = _mode(cache["prec"])
    W, h, f, A = cache["W"], cache["h"], cache["f"], net.num_actions
    g = {}
    dz = q(np.concatenate([np.asarray(dlogits, dt), np.asarray(dvalue, dt)[:, None]], axis=1))
    g["logits.w"] = h.T @ dz[:, :A]
    g["logits.b"] = dz[:, :A].sum(0)
    g["value.w"] = h.T @ dz[:, A:]
    g["value.b"] = dz[:, A:].sum(0)
    dh = q((dz[:, :A] @ W["logits.w"].T + dz[:, A:] @ W["value.w"].T) * (h > 0))
    g["dense.w"] = f.T @ dh
    g["dense.b"] = dh.sum(0)
    dx = q((dh @ W["dense.w"].T) * (f > 0)).reshape(cache["last"].shape)
    for s in reversed(range(3)):
        for r in reversed(range(2)):
            pre = f"s{s}.res{r}"
            x, t = cache[pre]
            gy = dx
            g[pre + ".conv1.w"], g[pre + ".conv1.b"] = conv3x3_wgrad(relu(t), gy)
            dt_ = q(conv3x3_dgrad(gy, W[pre + ".conv1.w"]) * (t > 0))
            g[pre + ".conv0.w"], g[pre + ".conv0.b"] = conv3x3_wgrad(relu(x), dt_)
            dx = q(gy + conv3x3_dgrad(dt_, W[pre + ".conv0.w"]) * (x > 0))
        x_in, arg, c_shape = cache[f"s{s}"]
        dc = q(maxpool_backward(arg, dx, c_shape))
        g[f"s{s}.conv.w"], g[f"s{s}.conv.b"] = conv3x3_wgrad(x_in, dc)
        if s > 0:
            dx = q(conv3x3_dgrad(dc, W[f"s{s}.conv.w"]))
    return flatten(g, net).astype(dt)
