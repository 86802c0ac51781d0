"""Certify that a forward pass has no decision near its switching point.

Max-pool argmaxes and ReLU masks are discontinuous decisions: when two window entries are
within float32 rounding of each other (or a ReLU input is within rounding of zero), two
correct float32 evaluations that merely sum in different orders may route gradient to
different cells, and a single such flip moves a conv-weight gradient by ~1e-3 relative.
Exact-parity tests in float32 therefore run on inputs whose smallest decision margin,
measured by the float64 oracle relative to each tensor's largest magnitude, is well above
float32 rounding.
"""
from __future__ import annotations

import numpy as np

from oracle import losses, net as onet


def _pool_gaps(c):
    n, h, w, ch = c.shape
    oh, ph0, ph1 = onet.same_pool_pads(h)
    ow, pw0, pw1 = onet.same_pool_pads(w)
    xp = np.full((n, h + ph0 + ph1, w + pw0 + pw1, ch), -np.inf)
    xp[:, ph0:ph0 + h, pw0:pw0 + w] = c
    stack = np.sort(np.stack(onet._pool_views(xp, oh, ow)), axis=0)
    gap = stack[-1] - stack[-2]
    gap[~np.isfinite(gap)] = np.inf          # a window with one real cell cannot flip
    return gap.min() / np.abs(c).max()


def _relu_margin(x):
    return np.abs(x).min() / np.abs(x).max()


def decision_margin(net, params, obs):
    """Smallest relative margin over every max-pool window (top-2 gap) and every ReLU input."""
    P = onet.unflatten(np.asarray(params, np.float64), net)
    x = obs.astype(np.float64) / 255.0
    margins = []
    for s in range(3):
        c = onet.conv3x3(x, P[f"s{s}.conv.w"], P[f"s{s}.conv.b"])
        margins.append(_pool_gaps(c))
        x, _ = onet.maxpool(c)
        for r in range(2):
            pre = f"s{s}.res{r}"
            margins.append(_relu_margin(x))
            t = onet.conv3x3(np.maximum(x, 0), P[pre + ".conv0.w"], P[pre + ".conv0.b"])
            margins.append(_relu_margin(t))
            x = x + onet.conv3x3(np.maximum(t, 0), P[pre + ".conv1.w"], P[pre + ".conv1.b"])
    margins.append(_relu_margin(x))
    f = np.maximum(x, 0).reshape(x.shape[0], -1)
    margins.append(_relu_margin(f @ P["dense.w"] + P["dense.b"]))
    return float(min(margins))


def ppo_clip_margin(logits, actions, old_logp, clip_eps):
    """Smallest |r - (1 +- eps)| over rows (the clip decision), for ratios from float64 logits."""
    lp = losses.log_softmax(np.asarray(logits, np.float64))[np.arange(len(actions)), actions]
    r = np.exp(lp - old_logp)
    return float(min(np.abs(r - (1 + clip_eps)).min(), np.abs(r - (1 - clip_eps)).min()))


def certified_frames(net, params, n, threshold=2e-6, max_seeds=200, first_seed=0):
    """First seed whose uint8 frames [n, H, W, C] have decision margin > threshold."""
    for seed in range(first_seed, first_seed + max_seeds):
        obs = np.random.default_rng(seed).integers(0, 256, size=(n, net.in_h, net.in_w, net.in_c),
                                                   dtype=np.uint8)
        m = decision_margin(net, params, obs)
        if m > threshold:
            return seed, obs, m
    raise RuntimeError("no certified input found")
