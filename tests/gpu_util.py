"""Helpers shared by the GPU parity tests: device buffers in the library's storage types and
the comparison rules. Inputs come from seeded numpy draws; expected values from the oracle."""
from __future__ import annotations

import numpy as np

from oracle.net import bf16_round

BF16, FP32 = 0, 1


def torch():
    import torch as t
    return t


def dev_f32(x):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda:0")


def dev_i32(x):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(np.asarray(x, np.int32))).to("cuda:0")


def dev_u8(x):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(np.asarray(x, np.uint8))).to("cuda:0")


def q(x, prec):
    """Values as the storage type holds them (bf16-rounded or float32), as float64."""
    x = np.asarray(x, np.float32)
    return (bf16_round(x) if prec == BF16 else x).astype(np.float64)


def dev_act(x, prec):
    """Activation tensor in the storage type (x must already be representable for bf16)."""
    t = torch()
    f = t.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32)))
    return (f.to(t.bfloat16) if prec == BF16 else f).to("cuda:0")


def empty_act(shape, prec):
    t = torch()
    return t.empty(shape, dtype=t.bfloat16 if prec == BF16 else t.float32, device="cuda:0")


def host(tensor):
    return tensor.detach().float().cpu().numpy().astype(np.float64)


def ws_bytes(nbytes):
    t = torch()
    return t.empty(max(int(nbytes), 1), dtype=t.uint8, device="cuda:0")


def sync():
    torch().cuda.synchronize()


def rel_l2(got, want):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    den = np.linalg.norm(want)
    return float(np.linalg.norm(got - want) / den) if den > 0 else float(np.linalg.norm(got))


def assert_close(got, want, rtol, what="", atol_frac=1.0):
    """Per array: relative L2 error ||got - want|| / ||want|| <= rtol, and elementwise
    |got - want| <= rtol * (|want| + atol_frac * max|want|): the elementwise guard is scaled
    to the array's magnitude because float32 errors on values produced by cancellation are
    relative to the operands, not to the (small) result."""
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    r = rel_l2(got, want)
    assert r <= rtol, f"{what}: relative L2 error {r:.3e} > {rtol:.1e}"
    scale = np.abs(want).max() if want.size else 0.0
    bad = np.abs(got - want) > rtol * (np.abs(want) + atol_frac * scale) + 1e-30
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements outside tolerance; worst at "
                           f"{np.unravel_index(np.argmax(np.abs(got - want)), got.shape)}")


def assert_sum_close(got, want, absum, rtol=1e-5, what=""):
    """Float32-accumulated sums: |got - want| <= rtol |want| + 2^-20 * sum|terms| elementwise
    (absum = the same sum over absolute values), and relative L2 <= rtol."""
    got, want, absum = (np.asarray(a, np.float64) for a in (got, want, absum))
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    bad = np.abs(got - want) > rtol * np.abs(want) + 2.0 ** -20 * absum
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements outside tolerance; "
                           f"worst |diff| {np.abs(got - want).max():.3e}")
    r = rel_l2(got, want)
    assert r <= rtol, f"{what}: relative L2 error {r:.3e} > {rtol:.1e}"


def assert_bf16_ulp(got, want_exact, absum, what="", ulps=1):
    """bf16-stored result within `ulps` bf16 units of the exact result rounded to bf16, plus
    the float32 accumulation error bound 2^-20 * sum|terms| (matters only near zero)."""
    want = q(want_exact, BF16)
    got = np.asarray(got, np.float64)
    spacing = np.maximum(np.abs(want), 1e-30) * 2.0 ** -7
    bad = np.abs(got - want) > ulps * spacing + 2.0 ** -20 * np.asarray(absum, np.float64)
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements beyond {ulps} bf16 ulp; "
                           f"worst |diff| {np.abs(got - want).max():.3e}")
