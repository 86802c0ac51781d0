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
WORKLOAD_NAMES = {1: "ppo_64x128_mb2048x4_e2", 2: "impala_vtrace_64x20", 4: "ppo_wide_128x128_mb8192"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=1, choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--prec", default="bf16", choices=["bf16", "fp32"])
    ap.add_argument("--cpu-sample-frames", type=int, default=1024,
                    help="frames in the oracle's timed CPU update (0 skips the CPU baseline)")
    return ap.parse_args()


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
    """(bound, algorithmic amount per launch, unit) for a profiling key.
    conv_fwd / conv_dgrad / wgrad: 2 * n * H * W * 9 * Cin * Cout FLOP (a 3x3 conv's MACs);
    gemm: 2 * M * N * K FLOP; adam: 28 bytes per parameter."""
    fam, _, shape = key.split("/", 2) if key.count("/") >= 2 else (key.split("/")[0], "", key.split("/", 1)[1])
    if fam in ("conv_fwd", "conv_dgrad", "wgrad"):
        ch, hw = shape.split("/")
        cin, cout = map(int, ch.split("x"))
        h, w = map(int, hw.split("x"))
        return "mfma", 2.0 * n * h * w * 9 * cin * cout, "FLOP"
    if fam == "gemm":
        m, nn, k = map(int, shape.split("x"))
        return "mfma", 2.0 * m * nn * k, "FLOP"
    if fam == "adam":
        return "hbm", 28.0 * int(shape), "B"
    return None, None, None


def source_digest(key):
    fam = key.split("/")[0]
    src = {"conv_fwd": "conv.hip", "conv_dgrad": "conv.hip", "wgrad": "wgrad.hip", "gemm": "gemm.hip",
           "adam": "adam.hip"}.get(fam)
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
    mb = wl.mb if wl.algo == "ppo" else wl.T * wl.E
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

    bound, work, unit = kernel_work(dominant[0], mb, args.prec)
    avg_s = kms / kcnt / 1e3
    if bound == "mfma":
        achieved = work / avg_s / 1e12
        peak, punit = PEAK[args.prec]
    else:
        achieved = work / avg_s / 1e9
        peak, punit = PEAK["hbm"]
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
                   "rollout_frames_per_s": round(wl.T * wl.E * args.steps / (gpu_ms / 1e3), 1),
                   "wall_s": round(wall, 3)},
        "roofline": {"bound": bound, "kernel": dominant[0], "achieved": round(achieved, 2), "peak": peak,
                     "unit": punit, "frac": round(achieved / peak, 4),
                     "avg_launch_us": round(avg_s * 1e6, 2), "launches_timed": kcnt,
                     "share_of_step": round(dominant[1] / profiled_total, 3) if profiled_total else None,
                     "traffic": traffic},
        "kernels_top": [{"key": k, "ms_per_step": round(t, 3), "launches": c} for k, t, c in table[:8]],
    }
    if args.cpu_sample_frames > 0:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_frames)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
