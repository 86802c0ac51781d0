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
WORKLOAD_NAMES = {1: "ppo_64x128_mb2048x4_e2", 2: "impala_vtrace_64x20", 4: "ppo_wide_128x128_mb8192",
                  5: "ppo_paper_128x128_mb4096x4_e4", 6: "impala_paper_128x20_mb4"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=1, choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--prec", default="bf16", choices=["bf16", "fp32"])
    ap.add_argument("--cpu-sample-frames", type=int, default=1024,
                    help="frames in the oracle's timed CPU update (0 skips the CPU baseline)")
    ap.add_argument("--layer", default=None,
                    help="replay one profiling key's launch (e.g. conv_dgrad/bf16/32x32/21x21/mask/add) "
                         "--steps times through the C-ABI on the minibatch size, for counter runs")
    ap.add_argument("--kernels", type=int, default=24, help="launch keys listed in kernels_top")
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


def kernel_work(key, n, prec):
    """(bound, algorithmic amount per launch, unit, flop) for a profiling key.

    The convolution family is bound by HBM at these channel counts (9 * Cin * Cout * 2 flop
    per pixel against (Cin + Cout) * 2 bytes: 72-144 flop/byte, below the bf16 ridge of
    2500 / 8 = 312), so its amount is the bytes it must move once: the input (1 byte per
    channel for uint8 frames), the output and any mask / residual operand; a fused conv +
    pool stores the pooled output and its uint8 argmax; a weight gradient reads x and dy.
    Pools move their input, output and argmax; adam 28 bytes per parameter. gemm is counted
    in flop against the matrix-core peak. `flop` is the MFMA work (None if none)."""
    parts = key.split("/")
    fam = parts[0]
    es = 2 if len(parts) > 1 and parts[1] == "bf16" else 4
    if fam == "resblock_fwd":   # one pass: x in, t and y out
        c = int(parts[2].split("x")[0])
        h, w = map(int, parts[3].split("x"))
        px = n * h * w
        return "hbm", float(px * c * es * 3), "B", 2.0 * 2.0 * px * 9 * c * c
    if fam == "resblock_bwd":   # one pass: dy, t and x in, dx out (dt stays on chip)
        c = int(parts[2].split("x")[0])
        h, w = map(int, parts[3].split("x"))
        px = n * h * w
        return "hbm", float(px * c * es * 4), "B", 4.0 * 2.0 * px * 9 * c * c
    if fam == "pool_wgrad":   # one pass: frames, pooled gradient and argmax in
        co = int(parts[2].split("x")[1])
        h, w = map(int, parts[3].split("x"))
        oh, ow = (h + 1) // 2, (w + 1) // 2
        return "hbm", float(n * (h * w * 4 + oh * ow * co * (es + 1))), "B", 2.0 * n * h * w * 36 * co
    if fam == "conv_bwd":   # one pass: x, dy (or the pooled dy and argmax) and the residual in, dx out
        ci, co = map(int, parts[2].split("x"))
        h, w = map(int, parts[3].split("x"))
        px = n * h * w
        dyb = (n * ((h + 1) // 2) * ((w + 1) // 2) * co * (es + 1)) if "pool" in parts[4:] else px * co * es
        b = px * es * (ci + ci + (ci if "add" in parts[4:] else 0)) + dyb
        return "hbm", float(b), "B", 2.0 * 2.0 * px * 9 * ci * co
    if fam in ("conv_fwd", "conv_dgrad", "wgrad", "conv_pool"):
        ci, co = map(int, parts[2].split("x"))
        h, w = map(int, parts[3].split("x"))
        flags = set(parts[4:])
        xb = 1 if "u8" in flags else es
        px = n * h * w
        flop = 2.0 * px * 9 * ci * co
        if fam == "wgrad":
            b = px * (ci * xb + co * es)
        elif fam == "conv_pool":
            oh, ow = (h + 1) // 2, (w + 1) // 2
            b = px * ci * xb + n * oh * ow * co * (es + 1)
        else:
            b = px * (ci * xb + co * es * (1 + ("mask" in flags) + ("add" in flags)))
        return "hbm", float(b), "B", flop
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
        return "hbm", float(n * (h * w * c * es + oh * ow * c * (es + 1))), "B", None
    if fam == "gemm":
        m, nn, k = map(int, parts[2].split("x"))
        return "mfma", 2.0 * m * nn * k, "FLOP", 2.0 * m * nn * k
    if fam == "adam":
        return "hbm", 28.0 * int(parts[2]), "B", None
    return None, None, None, None


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


def traffic_for(key, launches_per_step):
    """HBM bytes per launch from the committed counter summary, if it was taken on this
    kernel key and on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    try:
        c = json.load(open(path))
    except (OSError, ValueError):
        return None
    e = c.get(key)
    if not e or e.get("source_sha") != source_digest(key):
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


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the learner's "
              f"data-parallel sharding across GPUs is not part of this build.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2310_00036_amd as P
    from synth import WORKLOADS

    wl = WORKLOADS[args.workload]
    if args.copy_mb:
        return run_copy(args.copy_mb, args.steps)
    if args.layer:
        return run_layer(P, args.layer, wl.mb, args.steps)
    prec = P.PREC_BF16 if args.prec == "bf16" else P.PREC_FP32
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
    frames_per_step = wl.n_updates * mb

    def run(k):
        nonlocal step
        for _ in range(k):
            step = P.learner_step(net, cfg, rs, params, m, v, step, perm, ws, stats, stream)

    run(args.warmup)
    torch.cuda.synchronize()

    # Profiling pass (one step, every launch timed) to find the dominant kernel.
    P.impala_profile_begin(None, 1 << 16)
    run(1)
    table = P.impala_profile_end()
    dominant = next((r for r in table if kernel_work(r[0], mb, args.prec)[0]), table[0])
    profiled_total = sum(r[1] for r in table)

    # Timed region: K steps; the dominant kernel's launches are bracketed by HIP events
    # recorded on the stream they run on.
    P.impala_profile_begin(dominant[0], max(1, dominant[2]) * args.steps + 16)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    run(args.steps)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    _, kms, kcnt = P.impala_profile_end()[0]
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = gpu_ms / args.steps
    value = frames_per_step * args.steps / (gpu_ms / 1e3)

    bound, work, unit, flop = kernel_work(dominant[0], mb, args.prec)
    avg_s = kms / kcnt / 1e3
    if bound == "mfma":
        achieved = work / avg_s / 1e12
        peak, punit = PEAK[args.prec]
    else:
        achieved = work / avg_s / 1e9
        peak, punit = PEAK["hbm"]
    mfma_tflops = flop / avg_s / 1e12 if flop else None
    traffic = traffic_for(dominant[0], dominant[2])
    line = {
        "metric": "learner frames/sec (fwd+bwd+loss+Adam), IMPALA-CNN; % MFMA peak",
        "value": round(value, 1),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.prec,
        "data": "synthetic (seeded uniform uint8 84x84x4 frames, rewards in {-1,0,1}, Bernoulli(0.02) "
                "dones; behaviour data from the library's actor pass at the He-normal initial params)",
        "config": {"workload": WORKLOAD_NAMES[args.workload], "algo": wl.algo, "envs": wl.E,
                   "steps_per_env": wl.T, "minibatch": mb, "updates_per_step": wl.n_updates,
                   "frame_passes_per_step": frames_per_step, "net": f"{net.ch}/{net.hidden}/A{net.num_actions}",
                   "optimizer": wl.optimizer,
                   "rollout_frames_per_s": round(wl.T * wl.E * args.steps / (gpu_ms / 1e3), 1),
                   "wall_s": round(wall, 3)},
        "roofline": {"bound": bound, "kernel": dominant[0], "achieved": round(achieved, 2), "peak": peak,
                     "unit": punit, "frac": round(achieved / peak, 4),
                     "avg_launch_us": round(avg_s * 1e6, 2), "launches_timed": kcnt,
                     "share_of_step": round(dominant[1] / profiled_total, 3) if profiled_total else None,
                     "traffic": traffic, "algorithmic_bytes": work if unit == "B" else None,
                     "mfma_tflops": round(mfma_tflops, 2) if mfma_tflops else None,
                     "mfma_frac": round(mfma_tflops / PEAK[args.prec][0], 4) if mfma_tflops else None},
        "kernels_top": [{"key": k, "ms_per_step": round(t, 3), "launches": c} for k, t, c in table[:args.kernels]],
    }
    if args.cpu_sample_frames > 0:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_frames)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
