#!/usr/bin/env python3
"""Learner-update benchmark on one MI355X: learner frames/s of Cleanba's PPO learning phase.

One step is one learner_step over a synthetic Atari-shaped rollout resident in HBM: GAE,
then update_epochs x num_minibatches updates of (IMPALA-ResNet forward, PPO loss, backward,
global-norm clip, Adam). The default workload is PPO at a Cleanba-like shape: 64 envs x 128
steps = 8192 frames, 4 minibatches of 2048, 2 epochs (8 updates, 16384 frame-passes per
step), network (16,32,32)/256 with 18 actions, bf16 matrix-core operands with float32
accumulation. `value` counts frame-passes through forward+backward+loss+Adam per second.

Prints one JSON line. Also reports, for the kernel that takes the most time, its average
launch duration measured with HIP events on its own stream inside the timed region and the
fraction of the MI355X peak it reaches, and the oracle's CPU throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"bf16": (2500.0, "TFLOP/s"), "fp32": (157.3, "TFLOP/s"), "hbm": (8000.0, "GB/s")}
WORKLOAD_NAMES = {1: "ppo_64x128_mb2048x4_e2", 2: "impala_vtrace_64x20", 3: "actor_infer_b128",
                  4: "ppo_wide_128x128_mb8192",
                  5: "ppo_paper_128x128_mb4096x4_e4", 6: "impala_paper_128x20_mb4"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=1, choices=[w for w in sorted(WORKLOAD_NAMES) if w != 3])
    ap.add_argument("--prec", default="bf16", choices=["bf16", "fp32"])
    ap.add_argument("--cpu-sample-frames", type=int, default=1024,
                    help="frames in the oracle's timed CPU update (0 skips the CPU baseline)")
    ap.add_argument("--layer", default=None,
                    help="replay one profiling key's launch (e.g. conv_dgrad/bf16/32x32/21x21/mask/add) "
                         "--steps times through the C-ABI on the minibatch size, for counter runs")
    ap.add_argument("--kernels", type=int, default=24, help="launch keys listed in kernels_top")
    ap.add_argument("--no-extras", dest="extras", action="store_false",
                    help="skip the other workloads, the actor latency and the HBM sweep")
    ap.add_argument("--only", choices=["sweep", "actor"], default=None,
                    help="run only the HBM sweep or only the actor latency (profiling runs)")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="time a plain device copy of this many MiB --steps times (counter calibration)")
    return ap.parse_args()


def run_layer(P, key, n, steps):
    """Launch the layer a profiling key names, `steps` times, on synthetic bf16/uint8 data of
    the minibatch's shape; prints the average launch time."""
    import torch
    parts = key.split("/")
    fam, prec = parts[0], (P.PREC_BF16 if parts[1] != "fp32" else P.PREC_FP32)
    dt = torch.bfloat16 if prec == P.PREC_BF16 else torch.float32
    g = torch.Generator(device="cuda").manual_seed(7)
    act = lambda h, w, c: (torch.randn(n, h, w, c, device="cuda", generator=g) * 0.5).to(dt)  # noqa: E731
    if fam == "ppo_loss":   # key: ppo_loss/<rows>x<actions>
        m, A = map(int, parts[1].split("x"))
        z = torch.randn(m, A, device="cuda", generator=g)
        v, ret, adv = (torch.randn(m, device="cuda", generator=g) for _ in range(3))
        a = torch.randint(0, A, (m,), dtype=torch.int32, device="cuda", generator=g)
        olp = torch.log_softmax(z, 1).gather(1, a.long()[:, None])[:, 0] + 0.1 * torch.randn(m, device="cuda", generator=g)
        dz, dv = torch.empty_like(z), torch.empty_like(v)
        st = torch.empty(8, device="cuda")
        fn = lambda: P.ppo_loss_grad(m, A, z, v, a, olp, adv, ret, 1, 0.1, 0.5, 0.01, dz, dv, st)  # noqa: E731
    elif fam in ("pool_fwd", "pool_bwd"):
        c = int(parts[2])
        h, w = map(int, parts[3].split("x"))
        oh, ow = (h + 1) // 2, (w + 1) // 2
        x, y = act(h, w, c), act(oh, ow, c)
        arg = torch.randint(0, 9, (n, oh, ow, c), dtype=torch.uint8, device="cuda", generator=g)
        fn = ((lambda: P.impala_maxpool_fwd(prec, n, h, w, c, x, y, arg)) if fam == "pool_fwd"
              else (lambda: P.impala_maxpool_bwd(prec, n, h, w, c, arg, y, x)))
    else:
        ci, co = map(int, parts[2].split("x"))
        h, w = map(int, parts[3].split("x"))
        flags = set(parts[4:])
        mode = P.X_U8 if "u8" in flags else (P.X_RELU if "relu" in flags else P.X_PLAIN)
        x = (torch.randint(0, 256, (n, h, w, 4), dtype=torch.uint8, device="cuda", generator=g)
             if mode == P.X_U8 else act(h, w, ci))
        if fam == "pool_wgrad":
            oh, ow = (h + 1) // 2, (w + 1) // 2
            dp = act(oh, ow, co)
            arg = torch.randint(0, 9, (n, oh, ow, co), dtype=torch.uint8, device="cuda", generator=g)
            dw = torch.empty(3, 3, 4, co, device="cuda")
            db = torch.empty(co, device="cuda")
            ws = torch.empty(P.impala_conv3x3_pool_wgrad_u8_workspace_bytes(prec, co), dtype=torch.uint8,
                             device="cuda")
            fn = lambda: P.impala_conv3x3_pool_wgrad_u8(prec, n, h, w, co, x, None, dp, arg, dw, db, ws)  # noqa: E731
        elif fam == "resblock_fwd":
            w1, w2 = (torch.randn(3, 3, ci, ci, device="cuda", generator=g) * 0.1 for _ in range(2))
            b1, b2 = torch.zeros(ci, device="cuda"), torch.zeros(ci, device="cuda")
            x, tt, y = act(h, w, ci), act(h, w, ci), act(h, w, ci)
            fn = lambda: P.impala_resblock_fwd(prec, n, h, w, ci, x, w1, b1, w2, b2, tt, y)  # noqa: E731
        elif fam == "resblock_bwd":
            wa, wb = (torch.randn(3, 3, ci, ci, device="cuda", generator=g) * 0.1 for _ in range(2))
            dy, tt, x, dx = act(h, w, ci), act(h, w, ci), act(h, w, ci), act(h, w, ci)
            gw = [torch.empty(shape, device="cuda") for shape in ((3, 3, ci, ci), (ci,), (3, 3, ci, ci), (ci,))]
            ws = torch.empty(P.impala_resblock_bwd_workspace_bytes(prec, ci), dtype=torch.uint8, device="cuda")
            fn = lambda: P.impala_resblock_bwd(prec, n, h, w, ci, dy, tt, x, wa, wb, dx, *gw, ws)  # noqa: E731
        elif fam == "conv_bwd":     # key channels: forward cin x cout
            pooled = "pool" in flags
            oh, ow = (h + 1) // 2, (w + 1) // 2
            dy = act(oh, ow, co) if pooled else act(h, w, co)
            parg = torch.randint(0, 9, (n, oh, ow, co), dtype=torch.uint8, device="cuda", generator=g) if pooled else None
            wt = torch.randn(3, 3, ci, co, device="cuda", generator=g) * 0.1
            add = act(h, w, ci) if "add" in flags else None
            dx = act(h, w, ci)
            dw = torch.empty(3, 3, ci, co, device="cuda")
            db = torch.empty(co, device="cuda")
            ws = torch.empty(P.impala_conv3x3_bwd_workspace_bytes(prec, ci, co), dtype=torch.uint8, device="cuda")
            fn = lambda: P.impala_conv3x3_bwd(prec, n, h, w, ci, co, dy, x, mode, wt, add, dx, dw, db, ws,  # noqa: E731
                                              pool_arg=parg)
        elif fam == "conv_dgrad":   # key channels: dy (forward cout) x dx (forward cin)
            wt = torch.randn(3, 3, co, ci, device="cuda", generator=g) * 0.1
            mask = act(h, w, co) if "mask" in flags else None
            add = act(h, w, co) if "add" in flags else None
            out = act(h, w, co)
            fn = lambda: P.impala_conv3x3_dgrad(prec, n, h, w, co, ci, x, wt, mask, add, out)  # noqa: E731
        else:
            wt = torch.randn(3, 3, ci, co, device="cuda", generator=g) * 0.1
            b = torch.zeros(co, device="cuda")
            if fam == "conv_fwd":
                add = act(h, w, co) if "add" in flags else None
                out = act(h, w, co)
                fn = lambda: P.impala_conv3x3_fwd(prec, n, h, w, ci, co, x, mode, None, wt, b, add, out)  # noqa: E731
            elif fam == "conv_pool":
                oh, ow = (h + 1) // 2, (w + 1) // 2
                out = act(oh, ow, co)
                arg = torch.empty((n, oh, ow, co), dtype=torch.uint8, device="cuda")
                fn = lambda: P.impala_conv3x3_pool_fwd(prec, n, h, w, ci, co, x, mode, None, wt, b, out, arg)  # noqa: E731
            elif fam == "wgrad":
                dy = act(h, w, co)
                dw = torch.empty(3, 3, ci, co, device="cuda")
                db = torch.empty(co, device="cuda")
                ws = torch.empty(P.impala_conv3x3_wgrad_workspace_bytes(prec, h, w, ci, co), dtype=torch.uint8,
                                 device="cuda")
                fn = lambda: P.impala_conv3x3_wgrad(prec, n, h, w, ci, co, x, mode, None, dy, dw, db, ws)  # noqa: E731
            else:
                raise SystemExit(f"--layer: no replay for {key}")
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / steps * 1e3
    print(json.dumps({"layer": key, "n": n, "launches": steps + 1, "avg_launch_us": round(us, 2)}), flush=True)


def run_copy(mb, steps):
    import torch
    a = torch.empty(mb << 18, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        b.copy_(a)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    print(json.dumps({"copy_mib": mb, "launches": steps + 1, "bytes_read": a.numel() * 4,
                      "bytes_written": a.numel() * 4, "avg_s": dt}), flush=True)


def build_inputs(P, wl, prec):
    """Synthetic rollout on the GPU. Actions, behaviour log-probs and values come from the
    actor's pass over the frames with the initial parameters (Algorithm 1's rollout phase),
    run by the library's own actor entry point."""
    import torch
    from synth import draw_params, draw_rollout
    net = wl.net
    T, E, A = wl.T, wl.E, net.num_actions
    raw = draw_rollout(wl)
    params = torch.from_numpy(draw_params(net, wl.seed)).cuda()
    obs = torch.from_numpy(raw["obs"].reshape((T + 1) * E, net.in_h, net.in_w, net.in_c)).cuda()
    n_all = (T + 1) * E
    chunk = 2048
    ws = torch.empty(P.impala_workspace_bytes(net, chunk, prec, 0) + chunk * A * 4, dtype=torch.uint8,
                     device="cuda")
    gumbel = torch.from_numpy(raw["gumbel"]).cuda()
    actions = torch.empty(n_all, dtype=torch.int32, device="cuda")
    logp = torch.empty(n_all, dtype=torch.float32, device="cuda")
    value = torch.empty(n_all, dtype=torch.float32, device="cuda")
    logits = torch.empty((n_all, A), dtype=torch.float32, device="cuda")
    for s in range(0, n_all, chunk):
        e = min(n_all, s + chunk)
        P.impala_actor_step(net, prec, params, obs[s:e], e - s, gumbel[s:e].contiguous(), ws,
                            actions[s:e], logp[s:e], value[s:e], logits[s:e])
    bnoise = torch.from_numpy(raw["bnoise"]).cuda()
    TE = T * E
    if wl.algo == "ppo":
        behav_logp = (logp[:TE] + bnoise).contiguous()
        ro = dict(obs=obs[:TE].contiguous(), actions=actions[:TE].contiguous(), logp=behav_logp,
                  values=value[:TE].contiguous(), next_value=value[TE:].contiguous())
    else:
        mu = (logits[:TE] + bnoise).contiguous()
        P.impala_gumbel_sample(TE, A, mu, gumbel[:TE].contiguous(), actions[:TE], logp[:TE])
        ro = dict(obs=obs, actions=actions[:TE].contiguous(), logp=logp[:TE].contiguous(),
                  values=None, next_value=None)
    ro["rewards"] = torch.from_numpy(raw["rewards"]).cuda()
    ro["dones"] = torch.from_numpy(raw["dones"]).cuda()
    ro["next_done"] = torch.from_numpy(raw["next_done"]).cuda()
    perm = torch.from_numpy(raw["perm"]).cuda() if wl.algo == "ppo" else None
    torch.cuda.synchronize()
    return params, ro, perm


def kernel_work(key, n):
    """Algorithmic work of one launch of a profiling key on n frames (rows, parameters):
    {"bytes": HBM bytes the method must move once, "flop": matrix-core flop or None}.

    Bytes: the convolution family moves its input (1 byte per channel for uint8 frames), its
    output and any mask / residual operand; a fused conv + pool stores the pooled output and
    its uint8 argmax; a weight gradient reads x and dy; the fused backward kernels read x and dy
    (or the pooled dy and argmax) and the residual and write dx; pools move input, output and
    argmax; GAE 17 B per element + 5 B per env; V-trace 25 B + 4 B; the PPO loss (8A + 24) B
    per row, the IMPALA loss (8A + 20) B; Adam 28 B per parameter, RMSprop 20 B, the norm pass
    4 B. Flop: 2 per multiply-add of the convolutions and dense GEMMs (a residual block's
    forward is two 3x3 convs, its backward four: two input and two weight gradients)."""
    parts = key.split("/")
    fam = parts[0]
    es = 2 if len(parts) > 1 and parts[1] == "bf16" else 4
    if fam == "resblock_fwd":   # one pass: x in, t and y out
        c = int(parts[2].split("x")[0])
        h, w = map(int, parts[3].split("x"))
        px = n * h * w
        return {"bytes": float(px * c * es * 3), "flop": 2.0 * 2.0 * px * 9 * c * c}
    if fam == "resblock_bwd":   # one pass: dy, t and x in, dx out (dt stays on chip)
        c = int(parts[2].split("x")[0])
        h, w = map(int, parts[3].split("x"))
        px = n * h * w
        return {"bytes": float(px * c * es * 4), "flop": 4.0 * 2.0 * px * 9 * c * c}
    if fam == "pool_wgrad":   # one pass: frames, pooled gradient and argmax in
        co = int(parts[2].split("x")[1])
        h, w = map(int, parts[3].split("x"))
        oh, ow = (h + 1) // 2, (w + 1) // 2
        return {"bytes": float(n * (h * w * 4 + oh * ow * co * (es + 1))), "flop": 2.0 * n * h * w * 36 * co}
    if fam == "conv_bwd":   # one pass: x, dy (or the pooled dy and argmax) and the residual in, dx out
        ci, co = map(int, parts[2].split("x"))
        h, w = map(int, parts[3].split("x"))
        px = n * h * w
        dyb = (n * ((h + 1) // 2) * ((w + 1) // 2) * co * (es + 1)) if "pool" in parts[4:] else px * co * es
        b = px * es * (ci + ci + (ci if "add" in parts[4:] else 0)) + dyb
        return {"bytes": float(b), "flop": 2.0 * 2.0 * px * 9 * ci * co}
    if fam in ("conv_fwd", "conv_dgrad", "wgrad", "conv_pool"):
        ci, co = map(int, parts[2].split("x"))
        h, w = map(int, parts[3].split("x"))
        flags = set(parts[4:])
        xb = 1 if "u8" in flags else es
        px = n * h * w
        if fam == "wgrad":
            b = px * (ci * xb + co * es)
        elif fam == "conv_pool":
            oh, ow = (h + 1) // 2, (w + 1) // 2
            b = px * ci * xb + n * oh * ow * co * (es + 1)
        else:
            b = px * (ci * xb + co * es * (1 + ("mask" in flags) + ("add" in flags)))
        return {"bytes": float(b), "flop": 2.0 * px * 9 * ci * co}
    if fam in ("pool_fwd", "pool_bwd"):
        c = int(parts[2])
        h, w = map(int, parts[3].split("x"))
        oh, ow = (h + 1) // 2, (w + 1) // 2
        return {"bytes": float(n * (h * w * c * es + oh * ow * c * (es + 1))), "flop": None}
    if fam == "gemm":
        m, nn, k = map(int, parts[2].split("x"))
        return {"bytes": float(es * (m * k + k * nn) + 4 * m * nn), "flop": 2.0 * m * nn * k}
    if fam in ("ppo_loss", "impala_loss"):   # key: <family>/<rows>x<actions>
        m, A = map(int, parts[1].split("x"))
        return {"bytes": float((8 * A + (24 if fam == "ppo_loss" else 20)) * m), "flop": None}
    if fam in ("gae", "vtrace"):              # key: <family>/<T>x<E>
        T, E = map(int, parts[1].split("x"))
        return {"bytes": float((17 * T + 5) * E if fam == "gae" else (25 * T + 4) * E), "flop": None}
    if fam in ("adam", "rmsprop", "grad_sumsq"):
        return {"bytes": {"adam": 28.0, "rmsprop": 20.0, "grad_sumsq": 4.0}[fam] * int(parts[1]), "flop": None}
    return {"bytes": None, "flop": None}


def roofline(work, avg_s, prec):
    """The launch's place on the roofline. Contractions (work with flop) are bound by the
    matrix-core peak of their dtype: frac is the MFMA fraction; the HBM fraction of the same
    launch and the attainable ceiling min(1, intensity * HBM peak / MFMA peak) sit beside it.
    Everything else is bound by HBM bandwidth."""
    hbm_peak = PEAK["hbm"][0]
    out = {}
    if work["flop"]:
        peak, unit = PEAK[prec]
        tf = work["flop"] / avg_s / 1e12
        out.update(bound="mfma", achieved=round(tf, 2), peak=peak, unit=unit, frac=round(tf / peak, 4))
        if work["bytes"]:
            gbs = work["bytes"] / avg_s / 1e9
            inten = work["flop"] / work["bytes"]
            out.update(hbm_achieved=round(gbs, 1), hbm_frac=round(gbs / hbm_peak, 4),
                       intensity_flop_per_byte=round(inten, 1),
                       attainable_frac=round(min(1.0, inten * hbm_peak * 1e9 / (peak * 1e12)), 4))
    elif work["bytes"]:
        gbs = work["bytes"] / avg_s / 1e9
        out.update(bound="hbm", achieved=round(gbs, 1), peak=hbm_peak, unit="GB/s", frac=round(gbs / hbm_peak, 4))
    return out


def source_digest(key):
    fam = key.split("/")[0]
    src = {"conv_fwd": "conv.hip", "conv_dgrad": "conv.hip", "conv_pool": "conv.hip", "wgrad": "wgrad.hip",
           "gemm": "gemm.hip", "adam": "adam.hip", "pool_fwd": "pool.hip", "pool_bwd": "pool.hip",
           "resblock_fwd": "resblock.hip", "resblock_bwd": "resbwd.hip", "conv_bwd": "convbwd.hip",
           "pool_wgrad": "poolwgrad.hip"}.get(fam)
    if not src:
        return None
    path = os.path.join(ROOT, "paper_2310_00036_amd", "csrc", src)
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def traffic_for(key, n):
    """HBM bytes per launch from the committed counter summary, if it was taken on this
    kernel key, at this frame count and on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    try:
        c = json.load(open(path))
    except (OSError, ValueError):
        return None
    e = c.get(key)
    if not e or e.get("source_sha") != source_digest(key) or e.get("n") != n:
        return None
    return e.get("hbm_bytes_per_launch")


def cpu_baseline(wl, frames):
    """The oracle (float32 mode, as it stands) timed on the host cores: one PPO update
    (forward, loss, backward, clip, Adam) on a minibatch of `frames` frames."""
    from threadpoolctl import threadpool_info
    from oracle import losses, net as onet, optim
    from synth import draw_params
    net = wl.net
    rng = np.random.default_rng(0)
    params = draw_params(net, wl.seed)
    obs = rng.integers(0, 256, size=(frames, net.in_h, net.in_w, net.in_c), dtype=np.uint8)
    a = rng.integers(0, net.num_actions, frames)
    t0 = time.perf_counter()
    z, v, cache = onet.forward(net, params, obs, "fp32")
    _, dz, dv, _ = losses.ppo_loss_grad(z, v, a, np.zeros(frames), rng.standard_normal(frames),
                                        rng.standard_normal(frames), wl.clip_eps, wl.vf_coef,
                                        wl.ent_coef, dtype=np.float32)
    g = onet.backward(net, cache, dz, dv)
    g, _ = optim.clip_by_global_norm(g, wl.max_grad_norm, np.float32)
    z0 = np.zeros_like(params)
    optim.adam(params, g, z0, z0, 1, wl.lr, dtype=np.float32)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": round(frames / dt, 2), "unit": "frames/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one PPO update (forward, loss, backward, clip, Adam) on a {frames}-frame "
                      f"minibatch, float32 numpy oracle, {dt:.1f} s"}


def time_learner(P, wl, prec_name, steps, warmup):
    """learner_step on workload wl: `warmup` untimed steps, one profiling pass (every launch
    timed, to find the dominant kernel), then `steps` timed steps with the dominant kernel's
    launches bracketed by HIP events on the stream they run on."""
    import torch
    prec = P.PREC_BF16 if prec_name == "bf16" else P.PREC_FP32
    net = wl.net
    params, ro, perm = build_inputs(P, wl, prec)
    cfg = P.learner_cfg(wl, prec)
    ws = torch.empty(P.learner_workspace_bytes(net, cfg), dtype=torch.uint8, device="cuda")
    rs = P.rollout_struct(ro["obs"], ro["actions"], ro["logp"], ro["rewards"], ro["dones"],
                          ro["values"], ro["next_value"], ro["next_done"])
    m = torch.zeros_like(params)
    v = torch.zeros_like(params)
    stats = torch.zeros((wl.n_updates, 8), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    step = 0
    mb = wl.mb if wl.algo == "ppo" else wl.T * wl.E // wl.num_minibatches   # rollout rows per update
    fwd_n = mb if wl.algo == "ppo" else mb + wl.E // wl.num_minibatches   # frames per forward

    def run(k):
        nonlocal step
        for _ in range(k):
            step = P.learner_step(net, cfg, rs, params, m, v, step, perm, ws, stats, stream)

    run(warmup)
    torch.cuda.synchronize()
    P.impala_profile_begin(None, 1 << 16)
    run(1)
    table = P.impala_profile_end()
    profiled_total = sum(r[1] for r in table)
    fwd_fams = ("conv_pool", "resblock_fwd", "conv_fwd", "pool_fwd")
    frames_of = lambda key: fwd_n if key.split("/")[0] in fwd_fams else mb  # noqa: E731
    dominant = next((r for r in table if any(kernel_work(r[0], frames_of(r[0])).values())), table[0])

    P.impala_profile_begin(dominant[0], max(1, dominant[2]) * steps + 16)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    run(steps)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    _, kms, kcnt = P.impala_profile_end()[0]
    gpu_ms = ev0.elapsed_time(ev1)
    stat_rows = stats.cpu().numpy()
    assert np.isfinite(stat_rows).all() and (stat_rows[:, 7] == 0).all(), "non-finite learner statistics"
    del params, ro, perm, ws, m, v, stats
    torch.cuda.empty_cache()
    frames_per_step = wl.n_updates * mb
    avg_s = kms / kcnt / 1e3
    dn = frames_of(dominant[0])
    rl = roofline(kernel_work(dominant[0], dn), avg_s, prec_name)
    rl.update(kernel=dominant[0], avg_launch_us=round(avg_s * 1e6, 2), launches_timed=kcnt,
              share_of_step=round(dominant[1] / profiled_total, 3) if profiled_total else None)
    top = []
    for k, t, c in table:
        e = {"key": k, "ms_per_step": round(t, 3), "launches": c}
        r = roofline(kernel_work(k, frames_of(k)), t / c / 1e3, prec_name)
        if r:
            e.update(bound=r["bound"], frac=r["frac"])
            if "hbm_frac" in r:
                e["hbm_frac"] = r["hbm_frac"]
        top.append(e)
    return dict(value=frames_per_step * steps / (gpu_ms / 1e3), ms_per_step=gpu_ms / steps, wall=wall,
                mb=mb, fwd_n=fwd_n, frames_per_step=frames_per_step, roofline=rl, dominant_n=dn,
                kernels=top, rollout_fps=wl.T * wl.E * steps / (gpu_ms / 1e3))


def actor_latency(P, wl, prec_name, calls):
    """impala_actor_step on a batch of wl.T frames with Gumbel noise, `calls` times: each call's
    device time (HIP events around it on its stream) and host round trip (call + synchronize)."""
    import torch
    from synth import draw_actor_batch, draw_params
    prec = P.PREC_BF16 if prec_name == "bf16" else P.PREC_FP32
    net, n = wl.net, wl.T
    b = draw_actor_batch(wl)
    params = torch.from_numpy(draw_params(net, wl.seed)).cuda()
    obs = torch.from_numpy(b["obs"]).cuda()
    gumbel = torch.from_numpy(b["gumbel"]).cuda()
    # without a logits output the call keeps the logits in its workspace: n * A floats more
    ws = torch.empty(P.impala_workspace_bytes(net, n, prec, 0) + (n * net.num_actions * 4 + 255) // 256 * 256,
                     dtype=torch.uint8, device="cuda")
    act = torch.empty(n, dtype=torch.int32, device="cuda")
    logp, value = (torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(2))
    stream = torch.cuda.current_stream()
    call = lambda: P.impala_actor_step(net, prec, params, obs, n, gumbel, ws, act, logp, value, None, stream)  # noqa: E731
    for _ in range(20):
        call()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(calls)]
    host = np.empty(calls)
    for i in range(calls):
        t0 = time.perf_counter()
        evs[i][0].record(stream)
        call()
        evs[i][1].record(stream)
        torch.cuda.synchronize()
        host[i] = time.perf_counter() - t0
    dev = np.array([a.elapsed_time(z) * 1e3 for a, z in evs])
    host *= 1e6
    return {"workload": WORKLOAD_NAMES[3], "frames_per_call": n, "calls": calls,
            "device_us": {"p50": round(float(np.percentile(dev, 50)), 1), "p99": round(float(np.percentile(dev, 99)), 1)},
            "host_round_trip_us": {"p50": round(float(np.percentile(host, 50)), 1),
                                   "p99": round(float(np.percentile(host, 99)), 1)},
            "note": "device: HIP events around each call on its stream; host: call plus synchronize"}


def hbm_sweep(P, reps=20):
    """The HBM-bound kernels at the configurations' sizes and at scaled sizes (labelled), each
    call timed with HIP events on its stream over `reps` calls after a warm-up call; GB/s of the
    algorithmic bytes (kernel_work) against the 8 TB/s peak."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(11)
    dev = dict(device="cuda")
    out = []

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        z.record()
        torch.cuda.synchronize()
        return a.elapsed_time(z) / reps / 1e3

    def add(kernel, label, shape, nbytes, sec):
        gbs = nbytes / sec / 1e9
        out.append({"kernel": kernel, "size": label, "shape": shape, "bytes": int(nbytes),
                    "us": round(sec * 1e6, 2), "achieved": round(gbs, 1), "unit": "GB/s",
                    "frac": round(gbs / PEAK["hbm"][0], 4)})

    for T, E, label in ((128, 64, "config"), (128, 128, "config"), (128, 1 << 20, "scaled")):
        r = torch.randint(-1, 2, (T, E), generator=g, **dev).float()
        vals = torch.randn(T, E, generator=g, **dev)
        d = (torch.rand(T, E, generator=g, **dev) < 0.02).to(torch.uint8)
        nv = torch.randn(E, generator=g, **dev)
        nd = (torch.rand(E, generator=g, **dev) < 0.02).to(torch.uint8)
        adv, ret = torch.empty_like(vals), torch.empty_like(vals)
        sec = timed(lambda: P.gae_advantages(T, E, r, vals, d, nv, nd, 0.99, 0.95, adv, ret))
        add("gae", label, f"{T}x{E}", kernel_work(f"gae/{T}x{E}", 0)["bytes"], sec)
        del r, vals, d, adv, ret
    for T, E, label in ((20, 64, "config"), (20, 1 << 20, "scaled")):
        mu = torch.randn(T, E, generator=g, **dev) * 0.5 - 2
        pi = mu + 0.3 * torch.randn(T, E, generator=g, **dev)
        r = torch.randint(-1, 2, (T, E), generator=g, **dev).float()
        vals = torch.randn(T, E, generator=g, **dev)
        d = (torch.rand(T, E, generator=g, **dev) < 0.02).to(torch.uint8)
        bv = torch.randn(E, generator=g, **dev)
        nd = (torch.rand(E, generator=g, **dev) < 0.02).to(torch.uint8)
        vs, pg = torch.empty_like(vals), torch.empty_like(vals)
        sec = timed(lambda: P.vtrace_targets(T, E, mu, pi, r, vals, d, bv, nd, 0.99, 1.0, 1.0, 1.0, 1.0, vs, pg))
        add("vtrace", label, f"{T}x{E}", kernel_work(f"vtrace/{T}x{E}", 0)["bytes"], sec)
        del mu, pi, r, vals, d, vs, pg
    A = 18
    for fam, m, label in (("ppo_loss", 2048, "config"), ("ppo_loss", 8192, "config"), ("ppo_loss", 1 << 20, "scaled"),
                          ("impala_loss", 1280, "config"), ("impala_loss", 1 << 20, "scaled")):
        z = torch.randn(m, A, generator=g, **dev) * 3
        v, ret, adv = (torch.randn(m, generator=g, **dev) for _ in range(3))
        a = torch.randint(0, A, (m,), generator=g, dtype=torch.int32, **dev)
        old = torch.log_softmax(z, 1).gather(1, a.long()[:, None])[:, 0] + 0.1 * torch.randn(m, generator=g, **dev)
        dz, dv = torch.empty_like(z), torch.empty_like(v)
        st = torch.empty(8, **dev)
        lws = torch.empty(P.loss_workspace_bytes(m), dtype=torch.uint8, **dev)
        if fam == "ppo_loss":
            sec = timed(lambda: P.ppo_loss_grad(m, A, z, v, a, old, adv, ret, 1, 0.1, 0.5, 0.01, dz, dv, st, lws))
        else:
            sec = timed(lambda: P.impala_loss_grad(m, A, z, v, a, ret, adv, 1.0, 0.5, 0.01, dz, dv, st, lws))
        add(fam, label, f"{m}x{A}", kernel_work(f"{fam}/{m}x{A}", 0)["bytes"], sec)
        del z, v, ret, adv, a, old, dz, dv, lws
    for n, label in ((1_094_115, "config"), (4_364_211, "config"), (1 << 26, "scaled")):
        p = torch.randn(n, generator=g, **dev)
        gr = torch.randn(n, generator=g, **dev) * 1e-3
        m1, v1 = torch.zeros(n, **dev), torch.zeros(n, **dev)
        ws = torch.empty(P.adam_workspace_bytes(n), dtype=torch.uint8, **dev)
        st = torch.empty(2, **dev)
        sec = timed(lambda: P.adam_step(n, p, gr, m1, v1, 1, 2.5e-4, 0.9, 0.999, 1e-5, 0.5, st, ws))
        add("grad_sumsq+adam", label, str(n), kernel_work(f"adam/{n}", 0)["bytes"] +
            kernel_work(f"grad_sumsq/{n}", 0)["bytes"], sec)
        del p, gr, m1, v1
    torch.cuda.empty_cache()
    return out


def mfma_loop_peak(P, reps=5):
    """The achievable bf16 matrix-core rate of this device: impala_probe_mfma_bf16 (register-only
    loops of independent MFMAs, four 4-wave workgroups per CU), timed with HIP events."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks, iters = 4 * cus, 4096
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    flop = P.impala_probe_mfma_bf16(blocks, iters, sink)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        P.impala_probe_mfma_bf16(blocks, iters, sink)
    e1.record()
    torch.cuda.synchronize()
    tf = flop / (e0.elapsed_time(e1) / 1e3 / reps) / 1e12
    return {"achieved": round(tf, 1), "unit": "TFLOP/s", "published": PEAK["bf16"][0],
            "frac_of_published": round(tf / PEAK["bf16"][0], 4), "blocks": blocks, "iters": iters}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the learner's "
              f"data-parallel sharding across GPUs is not part of this build.", file=sys.stderr)
        sys.exit(2)
    import torch  # noqa: F401
    import paper_2310_00036_amd as P
    from synth import WORKLOADS

    wl = WORKLOADS[args.workload]
    if args.copy_mb:
        return run_copy(args.copy_mb, args.steps)
    if args.layer:
        return run_layer(P, args.layer, wl.mb, args.steps)
    if args.only == "sweep":
        return print(json.dumps({"hbm_sweep": hbm_sweep(P)}), flush=True)
    if args.only == "actor":
        return print(json.dumps({"actor_latency": actor_latency(P, WORKLOADS[3], args.prec, 1000)}), flush=True)
    net = wl.net
    head = time_learner(P, wl, args.prec, args.steps, args.warmup)
    rl = head["roofline"]
    rl["traffic"] = traffic_for(rl["kernel"], head["dominant_n"])
    loop_peak = mfma_loop_peak(P)
    if rl.get("bound") == "mfma" and args.prec == "bf16":
        rl["frac_of_loop_peak"] = round(rl["achieved"] / loop_peak["achieved"], 4)
    line = {
        "metric": "learner frames/sec (fwd+bwd+loss+Adam), IMPALA-CNN; % MFMA peak",
        "value": round(head["value"], 1),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.prec,
        "data": "synthetic (seeded uniform uint8 84x84x4 frames, rewards in {-1,0,1}, Bernoulli(0.02) "
                "dones; behaviour data from the library's actor pass at the He-normal initial params)",
        "config": {"workload": WORKLOAD_NAMES[args.workload], "algo": wl.algo, "envs": wl.E,
                   "steps_per_env": wl.T, "minibatch": head["mb"], "updates_per_step": wl.n_updates,
                   "frame_passes_per_step": head["frames_per_step"],
                   "net": f"{net.ch}/{net.hidden}/A{net.num_actions}", "optimizer": wl.optimizer,
                   "rollout_frames_per_s": round(head["rollout_fps"], 1), "wall_s": round(head["wall"], 3)},
        "roofline": rl,
        "mfma_loop_peak": loop_peak,
        "kernels_top": head["kernels"][:args.kernels],
    }
    if args.extras:
        others = {}
        for wid, steps in ((2, max(args.steps, 20)), (4, max(3, args.steps // 4))):
            if wid == args.workload:
                continue
            r = time_learner(P, WORKLOADS[wid], args.prec, steps, 2)
            others[WORKLOAD_NAMES[wid]] = {
                "value": round(r["value"], 1), "unit": "frames/s", "ms_per_step": round(r["ms_per_step"], 3),
                "steps": steps, "updates_per_step": WORKLOADS[wid].n_updates, "minibatch": r["mb"],
                "roofline": r["roofline"], "kernels_top": r["kernels"][:8]}
        line["workloads"] = others
        line["actor_latency"] = actor_latency(P, WORKLOADS[3], args.prec, 1000)
        line["hbm_sweep"] = hbm_sweep(P)
    if args.cpu_sample_frames > 0:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_frames)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
