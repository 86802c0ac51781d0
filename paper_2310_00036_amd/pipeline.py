"""Cleanba's actor-learner pipeline on one GPU (Section 4.2, Deterministic Rollout Data
Composition; Table 1 and the Cleanba-architecture pseudocode of Figure 3).

The actor and the learner run in two threads, each on its own HIP stream, and meet through
two queues that hold at most one item: `data_q` (rollouts, actor -> learner) and `param_q`
(parameter snapshots, learner -> actor). The actor takes fresh parameters before every
rollout except the second, so the learner always trains on data from the second latest
policy: rollouts 1 and 2 come from pi_1, rollout k >= 3 from pi_{k-1}, and update k turns
pi_k into pi_{k+1} with rollout k. A blocking get on an empty queue and a blocking put on a
full one fix that composition whatever the relative speed of the two threads, so a run is
reproducible bit for bit (the learner's kernels are deterministic) while rollout k+1 is
collected during update k.

Everything the agent computes runs in the library's kernels (impala_actor_step for the
actor's inference and sampling, learner_step for the update). The environments are a seeded
synthetic stand-in for EnvPool's Atari (84x84 greyscale, 4 stacked frames, rewards in
{-1, 0, 1}, Bernoulli episode ends), stepped on the host as EnvPool steps on the CPU; a frame
depends on the env, the step and the action taken, so a different policy produces different
data.

`run_pipeline` drives any agent object with `snapshot`, `act`, `learn` methods (LibraryAgent
is the one on the GPU); `run_sequential` replays the same composition in one thread, the
reference a pipelined run must equal.
"""
from __future__ import annotations

import hashlib
import queue
import threading
import time
from dataclasses import dataclass, field

import numpy as np

from . import _lib as L


# ----------------------------------------------------------------------------- environments


class SyntheticAtari:
    """`num_envs` seeded environments with Atari's observation shape. The frame an env shows
    after action a at its step t is drawn from a generator keyed by (seed, env, t, a); the
    observation stacks the last `in_c` frames (the oldest first); rewards follow
    `reward_probs` over {-1, 0, 1}; an episode ends with probability `done_prob` per step and
    the env then starts a new one (its stack refilled with a fresh frame)."""

    def __init__(self, num_envs, net, seed=0, reward_probs=(0.05, 0.9, 0.05), done_prob=0.02):
        self.E, self.h, self.w, self.c = num_envs, net.in_h, net.in_w, net.in_c
        self.seed = seed
        self.reward_probs = np.asarray(reward_probs, np.float64)
        self.done_prob = done_prob
        self.t = 0
        self.obs = np.empty((num_envs, self.h, self.w, self.c), np.uint8)
        for e in range(num_envs):
            self.obs[e] = self._rng(e, -1, 0).integers(0, 256, (self.h, self.w, self.c), dtype=np.uint8)
        self.done = np.ones(num_envs, np.uint8)   # every env starts an episode

    def _rng(self, e, t, a):
        return np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, e, t + 1, int(a)])))

    def step(self, actions):
        """Advance every env by one step; returns (obs [E, H, W, C] u8, reward [E] f32,
        done [E] u8), done = 1 meaning the returned observation starts a new episode."""
        actions = np.asarray(actions)
        rew = np.empty(self.E, np.float32)
        done = np.empty(self.E, np.uint8)
        for e in range(self.E):
            g = self._rng(e, self.t, actions[e])
            frame = g.integers(0, 256, (self.h, self.w), dtype=np.uint8)
            rew[e] = g.choice(np.array([-1.0, 0.0, 1.0], np.float32), p=self.reward_probs)
            done[e] = g.random() < self.done_prob
            if done[e]:
                self.obs[e] = frame[:, :, None]
            else:
                self.obs[e, :, :, :-1] = self.obs[e, :, :, 1:]
                self.obs[e, :, :, -1] = frame
        self.t += 1
        self.done = done
        return self.obs.copy(), rew, done.copy()


# ----------------------------------------------------------------------------- rollouts


@dataclass
class Rollout:
    """One rollout, host arrays (the agent moves them to the device): Algorithm 1's D plus the
    bootstrap state. obs: PPO [T*E, H, W, C]; IMPALA [(T+1)*E, H, W, C] with s_next last."""
    index: int
    policy_version: int
    obs: np.ndarray
    actions: np.ndarray
    logp: np.ndarray
    rewards: np.ndarray
    dones: np.ndarray
    values: np.ndarray | None
    next_value: np.ndarray | None
    next_done: np.ndarray

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.obs, self.actions, self.logp, self.rewards, self.dones, self.values, self.next_value,
                  self.next_done):
            if a is not None:
                h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()[:16]


def gumbel_noise(seed, rollout, t, shape):
    """The actor's standard Gumbel draws for step t of rollout k (seeded per step, so they do
    not depend on thread timing)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7919, rollout, t])))
    return g.gumbel(size=shape).astype(np.float32)


def collect_rollout(agent, params, envs, wl, index, version, seed):
    """Algorithm 1's rollout phase for wl.T steps on `envs` with the given parameters: per step
    cache s_t and d_t, sample a_t ~ pi(.|s_t) with v_t, step the environments."""
    T, E, A = wl.T, wl.E, wl.net.num_actions
    shape = (envs.h, envs.w, envs.c)
    obs = np.empty((T + 1, E) + shape, np.uint8)
    act = np.empty((T, E), np.int32)
    logp = np.empty((T, E), np.float32)
    val = np.empty((T, E), np.float32)
    rew = np.empty((T, E), np.float32)
    dones = np.empty((T, E), np.uint8)
    s, d = envs.obs.copy(), envs.done.copy()
    for t in range(T):
        obs[t], dones[t] = s, d
        a, lp, v = agent.act(params, s, gumbel_noise(seed, index, t, (E, A)))
        act[t], logp[t], val[t] = a, lp, v
        s, rew[t], d = envs.step(a)
    obs[T] = s
    if wl.algo == "ppo":
        _, _, nv = agent.act(params, s, gumbel_noise(seed, index, T, (E, A)))
        return Rollout(index, version, obs[:T].reshape((T * E,) + shape), act.ravel(), logp.ravel(), rew, dones,
                       val, nv.astype(np.float32), d)
    return Rollout(index, version, obs.reshape(((T + 1) * E,) + shape), act.ravel(), logp.ravel(), rew, dones,
                   None, None, d)


# ----------------------------------------------------------------------------- the two loops


@dataclass
class PipelineRecord:
    rollouts: list = field(default_factory=list)      # (index, policy version, digest)
    updates: list = field(default_factory=list)       # (update k, rollout index, new version)
    stats: list = field(default_factory=list)         # per update: learner statistics rows
    actor_wait_s: float = 0.0                         # time in param_q.get
    learner_wait_s: float = 0.0                       # time in data_q.get
    wall_s: float = 0.0


class _Stop(Exception):
    pass


def _get(q, failed, timeout):
    t0 = time.perf_counter()
    while True:
        if failed.is_set():
            raise _Stop()
        try:
            return q.get(timeout=0.05)
        except queue.Empty:
            if timeout and time.perf_counter() - t0 > timeout:
                raise TimeoutError("pipeline queue get timed out")


def _put(q, item, failed, timeout):
    t0 = time.perf_counter()
    while True:
        if failed.is_set():
            raise _Stop()
        try:
            return q.put(item, timeout=0.05)
        except queue.Full:
            if timeout and time.perf_counter() - t0 > timeout:
                raise TimeoutError("pipeline queue put timed out")


def run_pipeline(agent, wl, iterations, seed=0, actor_delay=None, learner_delay=None, timeout=600.0):
    """Cleanba's architecture for `iterations` rollouts and as many updates. actor_delay and
    learner_delay, if given, are callables k -> seconds to sleep around rollout / update k
    (to vary the relative speed of the two threads). Returns (final parameters snapshot,
    PipelineRecord)."""
    data_q, param_q = queue.Queue(maxsize=1), queue.Queue(maxsize=1)
    rec = PipelineRecord()
    failed = threading.Event()
    errors = []
    envs = SyntheticAtari(wl.E, wl.net, seed, wl.reward_probs, wl.done_prob)
    param_q.put((1, agent.snapshot()))
    final = {}

    def actor():
        try:
            params, version = None, 0
            for k in range(1, iterations + 1):
                if k != 2:   # the second rollout reuses pi_1: it overlaps the first update
                    t0 = time.perf_counter()
                    version, params = _get(param_q, failed, timeout)
                    rec.actor_wait_s += time.perf_counter() - t0
                if actor_delay:
                    time.sleep(actor_delay(k))
                ro = collect_rollout(agent, params, envs, wl, k, version, seed)
                rec.rollouts.append((k, version, ro.digest()))
                _put(data_q, ro, failed, timeout)
        except _Stop:
            pass
        except BaseException as e:   # noqa: BLE001  (reported by the caller)
            errors.append(e)
            failed.set()

    def learner():
        try:
            for k in range(1, iterations + 1):
                t0 = time.perf_counter()
                ro = _get(data_q, failed, timeout)
                rec.learner_wait_s += time.perf_counter() - t0
                if learner_delay:
                    time.sleep(learner_delay(k))
                rec.stats.append(agent.learn(ro))
                rec.updates.append((k, ro.index, k + 1))
                if k + 2 <= iterations:   # rollout k + 2 is the one that takes pi_{k+1}
                    _put(param_q, (k + 1, agent.snapshot()), failed, timeout)
            final["params"] = agent.snapshot()
        except _Stop:
            pass
        except BaseException as e:   # noqa: BLE001
            errors.append(e)
            failed.set()

    t0 = time.perf_counter()
    threads = [threading.Thread(target=actor, name="cleanba-actor"),
               threading.Thread(target=learner, name="cleanba-learner")]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    rec.wall_s = time.perf_counter() - t0
    if errors:
        raise errors[0]
    return final["params"], rec


def run_sequential(agent, wl, iterations, seed=0):
    """The same composition in one thread: rollout 1 and 2 with pi_1, then for k = 1.. update k
    with rollout k and rollout k + 2 with pi_{k+1}."""
    rec = PipelineRecord()
    envs = SyntheticAtari(wl.E, wl.net, seed, wl.reward_probs, wl.done_prob)
    t0 = time.perf_counter()
    versions = {1: agent.snapshot()}
    pending = []
    for k in (1, 2):
        if k <= iterations:
            ro = collect_rollout(agent, versions[1], envs, wl, k, 1, seed)
            rec.rollouts.append((k, 1, ro.digest()))
            pending.append(ro)
    for k in range(1, iterations + 1):
        ro = pending.pop(0)
        rec.stats.append(agent.learn(ro))
        rec.updates.append((k, ro.index, k + 1))
        if k + 2 <= iterations:
            versions[k + 1] = agent.snapshot()
            nxt = collect_rollout(agent, versions[k + 1], envs, wl, k + 2, k + 1, seed)
            rec.rollouts.append((k + 2, k + 1, nxt.digest()))
            pending.append(nxt)
    rec.wall_s = time.perf_counter() - t0
    return agent.snapshot(), rec


# ----------------------------------------------------------------------------- the GPU agent


class LibraryAgent:
    """The agent on the GPU: actor inference and sampling with impala_actor_step on the actor's
    stream, learning phases with learner_step on the learner's stream. Parameters, optimiser
    state and step count live on the device; `snapshot` copies the parameters (the copy is
    finished before it is handed over)."""

    def __init__(self, wl, prec, params, device="cuda"):
        import torch
        self.torch = torch
        self.wl, self.prec, self.net = wl, prec, wl.net
        self.dev = device
        self.params = torch.as_tensor(np.asarray(params, np.float32)).to(device)
        self.m = torch.zeros_like(self.params)
        self.v = torch.zeros_like(self.params)
        self.step = 0
        self.cfg = L.learner_cfg(wl, prec)
        self.learner_stream = torch.cuda.Stream(device)
        self.actor_stream = torch.cuda.Stream(device)
        self.ws = torch.empty(L.learner_workspace_bytes(self.net, self.cfg), dtype=torch.uint8, device=device)
        E, A = wl.E, self.net.num_actions
        self.act_ws = torch.empty(L.impala_workspace_bytes(self.net, E, prec, 0) + (E * A * 4 + 255) // 256 * 256,
                                  dtype=torch.uint8, device=device)
        self.a = torch.empty(E, dtype=torch.int32, device=device)
        self.lp = torch.empty(E, dtype=torch.float32, device=device)
        self.val = torch.empty(E, dtype=torch.float32, device=device)
        self.stats = torch.zeros((wl.n_updates, 8), dtype=torch.float32, device=device)
        self.perm_rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, 104729])))

    def snapshot(self):
        torch = self.torch
        with torch.cuda.stream(self.learner_stream):
            p = self.params.clone()
        self.learner_stream.synchronize()
        return p

    def act(self, params, obs, gumbel):
        torch = self.torch
        with torch.cuda.stream(self.actor_stream):
            o = torch.from_numpy(np.ascontiguousarray(obs)).to(self.dev, non_blocking=False)
            g = torch.from_numpy(gumbel).to(self.dev)
            L.impala_actor_step(self.net, self.prec, params, o, obs.shape[0], g, self.act_ws, self.a, self.lp,
                                self.val, None, self.actor_stream)
            out = (self.a.cpu().numpy().copy(), self.lp.cpu().numpy().copy(), self.val.cpu().numpy().copy())
        return out

    def learn(self, ro):
        torch = self.torch
        wl = self.wl
        with torch.cuda.stream(self.learner_stream):
            t = lambda x, dt: (torch.from_numpy(np.ascontiguousarray(x).astype(dt)).to(self.dev)  # noqa: E731
                               if x is not None else None)
            d = dict(obs=t(ro.obs, np.uint8), actions=t(ro.actions, np.int32), logp=t(ro.logp, np.float32),
                     rewards=t(ro.rewards, np.float32), dones=t(ro.dones, np.uint8), values=t(ro.values, np.float32),
                     next_value=t(ro.next_value, np.float32), next_done=t(ro.next_done, np.uint8))
            rs = L.rollout_struct(d["obs"], d["actions"], d["logp"], d["rewards"], d["dones"], d["values"],
                                  d["next_value"], d["next_done"])
            perm = None
            if wl.algo == "ppo":
                perm = t(np.stack([self.perm_rng.permutation(wl.T * wl.E) for _ in range(wl.epochs)]), np.int32)
            self.step = L.learner_step(self.net, self.cfg, rs, self.params, self.m, self.v, self.step, perm, self.ws,
                                       self.stats, self.learner_stream)
            out = self.stats.cpu().numpy().copy()
        return out
