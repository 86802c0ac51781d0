"""Workload shapes and seeded random draws for Atari-shaped learner updates.

Shapes follow the paper's Atari setting (Section 5: 84x84 greyscale frames, 4 stacked, full
action space of 18) and the PPO / IMPALA hyperparameter tables of Appendix B. The random
streams stand in for EnvPool rollouts, which are not available: frames are i.i.d. uniform
bytes, rewards are clipped to {-1, 0, 1}, and episode ends are Bernoulli.

Every draw comes from numpy's PCG64 via ``SeedSequence(seed).spawn``, one child stream per
quantity, so each array is reproducible on its own.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class NetShape:
    """IMPALA-ResNet shape: input frame, three stage widths, dense width, action count."""
    in_h: int = 84
    in_w: int = 84
    in_c: int = 4
    ch: tuple = (16, 32, 32)
    hidden: int = 256
    num_actions: int = 18


@dataclass(frozen=True)
class Workload:
    """One learner-update workload (PPO, IMPALA/V-trace or actor inference)."""
    name: str
    algo: str                    # "ppo" | "impala" | "actor"
    T: int                       # rollout steps (num_steps); batch size for "actor"
    E: int                       # envs (local_num_envs); 1 for "actor"
    net: NetShape = NetShape()
    epochs: int = 1              # update_epochs
    num_minibatches: int = 1
    minibatch_size: int = 0      # m; 0 -> T*E / num_minibatches
    gamma: float = 0.99
    lam: float = 0.95
    clip_eps: float = 0.1
    vf_coef: float = 0.5
    ent_coef: float = 0.01
    pg_coef: float = 1.0
    rho_bar: float = 1.0
    c_bar: float = 1.0
    pg_rho_bar: float = 1.0
    lr: float = 2.5e-4
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-5
    max_grad_norm: float = 0.5
    optimizer: str = "adam"      # "adam" | "rmsprop"
    rms_decay: float = 0.99
    rms_eps: float = 0.01
    norm_adv: int = 1
    reward_probs: tuple = (0.05, 0.9, 0.05)   # P(r=-1), P(r=0), P(r=+1)
    done_prob: float = 0.02
    behav_logp_noise: float = 0.05            # PPO: N(0, s) on the behaviour log-prob
    behav_logit_noise: float = 0.0            # IMPALA: N(0, s) on every behaviour logit
    seed: int = 0

    @property
    def batch(self) -> int:
        return self.T * self.E

    @property
    def mb(self) -> int:
        return self.minibatch_size or self.batch // self.num_minibatches

    @property
    def n_updates(self) -> int:
        return self.epochs * self.num_minibatches if self.algo == "ppo" else self.num_minibatches

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


BASE_NET = NetShape()
WIDE_NET = NetShape(ch=(32, 64, 64), hidden=512)

WORKLOADS = {
    # Tiny PPO learner step: 4 envs x 8 steps, 6 actions, one full-batch update.
    0: Workload("ppo_tiny_4x8", "ppo", T=8, E=4, net=NetShape(num_actions=6),
                epochs=1, num_minibatches=1, seed=0),
    # PPO at a Cleanba-like shape: 64 envs x 128 steps, 4 minibatches of 2048, 2 epochs.
    1: Workload("ppo_64x128_mb2048x4_e2", "ppo", T=128, E=64, epochs=2, num_minibatches=4,
                seed=1),
    # IMPALA / V-trace: 64 envs x 20-step unroll (+1 bootstrap frame per env).
    2: Workload("impala_vtrace_64x20", "impala", T=20, E=64, lam=1.0, lr=6e-4,
                max_grad_norm=40.0, behav_logp_noise=0.0, behav_logit_noise=0.3, seed=2),
    # Actor-side inference: 128 frames per call with Gumbel-max sampling.
    3: Workload("actor_infer_b128", "actor", T=128, E=1, seed=3),
    # Widened learner: (32,64,64)/512, 128 envs x 128 steps, one minibatch of 8192.
    4: Workload("ppo_wide_128x128_mb8192", "ppo", T=128, E=128, net=WIDE_NET, epochs=1,
                num_minibatches=1, minibatch_size=8192, seed=4),
    # The paper's PPO shape (Appendix B, PPO table): 128 envs x 128 steps, 4 minibatches of
    # 4096, 4 epochs (16 updates); fixed learning rate (no annealing).
    5: Workload("ppo_paper_128x128_mb4096x4_e4", "ppo", T=128, E=128, epochs=4, num_minibatches=4,
                seed=5),
    # The paper's IMPALA shape (Appendix B, IMPALA table): 128 envs x 20 steps, 4 minibatches
    # of 32 envs, RMSprop (decay 0.99, eps 0.01), lr 6e-4, omega 40.
    6: Workload("impala_paper_128x20_mb4", "impala", T=20, E=128, num_minibatches=4, lam=1.0, lr=6e-4,
                max_grad_norm=40.0, optimizer="rmsprop", behav_logp_noise=0.0, behav_logit_noise=0.3,
                seed=6),
}


def workload(i: int) -> Workload:
    return WORKLOADS[i]


def _flat_after_stages(net: NetShape) -> tuple:
    h, w = net.in_h, net.in_w
    for _ in range(3):
        h, w = -(-h // 2), -(-w // 2)
    return h, w


def param_shapes(net: NetShape) -> list:
    """(name, shape, fan_in) of the 36 parameter tensors, in flat-buffer order.

    Conv weights are HWIO [3,3,Cin,Cout]; dense weights are [in, out]; biases follow their
    weight. The order is stage-major (entry conv, block0 conv0/conv1, block1 conv0/conv1),
    then dense, logits, value.
    """
    out = []
    cin = net.in_c
    for s, c in enumerate(net.ch):
        out.append((f"s{s}.conv.w", (3, 3, cin, c), 9 * cin))
        out.append((f"s{s}.conv.b", (c,), 0))
        for r in range(2):
            for k in range(2):
                out.append((f"s{s}.res{r}.conv{k}.w", (3, 3, c, c), 9 * c))
                out.append((f"s{s}.res{r}.conv{k}.b", (c,), 0))
        cin = c
    fh, fw = _flat_after_stages(net)
    flat = fh * fw * net.ch[2]
    out.append(("dense.w", (flat, net.hidden), flat))
    out.append(("dense.b", (net.hidden,), 0))
    out.append(("logits.w", (net.hidden, net.num_actions), net.hidden))
    out.append(("logits.b", (net.num_actions,), 0))
    out.append(("value.w", (net.hidden, 1), net.hidden))
    out.append(("value.b", (1,), 0))
    return out


def param_count(net: NetShape) -> int:
    return int(sum(np.prod(s) for _, s, _ in param_shapes(net)))


def _streams(seed: int, n: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


# stream indices
_S_PARAMS, _S_OBS, _S_REW, _S_DONE, _S_GUMBEL, _S_BNOISE, _S_PERM, _S_ACTOR = range(8)


def draw_params(net: NetShape, seed: int) -> np.ndarray:
    """He-normal weights N(0, 2/fan_in), zero biases, as one flat float32 buffer."""
    rng = _streams(seed, 8)[_S_PARAMS]
    parts = []
    for _, shape, fan_in in param_shapes(net):
        if fan_in:
            parts.append(rng.standard_normal(shape, dtype=np.float32).ravel()
                         * np.float32(np.sqrt(2.0 / fan_in)))
        else:
            parts.append(np.zeros(int(np.prod(shape)), np.float32))
    return np.concatenate(parts).astype(np.float32)


def draw_rollout(wl: Workload) -> dict:
    """Raw random arrays of one rollout, time-major [T, E] with E fastest.

    obs      uint8 [T+1, E, H, W, C]  (row T is s_next: the bootstrap frame)
    rewards  float32 [T, E] in {-1, 0, 1}
    dones    uint8 [T, E], next_done uint8 [E]  (d_t = 1: s_t starts a new episode)
    gumbel   float32 [(T+1)*E, A] standard Gumbel noise for behaviour sampling
    bnoise   float32 [T*E] (PPO log-prob noise) or [T*E, A] (IMPALA logit noise)
    perm     int32 [epochs, T*E], one permutation of the flattened batch per epoch
    """
    net = wl.net
    T, E, A = wl.T, wl.E, net.num_actions
    st = _streams(wl.seed, 8)
    obs = st[_S_OBS].integers(0, 256, size=(T + 1, E, net.in_h, net.in_w, net.in_c),
                              dtype=np.uint8)
    rewards = st[_S_REW].choice(np.array([-1.0, 0.0, 1.0], np.float32), size=(T, E),
                                p=list(wl.reward_probs)).astype(np.float32)
    dr = st[_S_DONE]
    dones = (dr.random((T, E)) < wl.done_prob).astype(np.uint8)
    next_done = (dr.random(E) < wl.done_prob).astype(np.uint8)
    gumbel = st[_S_GUMBEL].gumbel(size=((T + 1) * E, A)).astype(np.float32)
    if wl.behav_logit_noise > 0:
        bnoise = (st[_S_BNOISE].standard_normal((T * E, A)) * wl.behav_logit_noise)
    else:
        bnoise = st[_S_BNOISE].standard_normal(T * E) * wl.behav_logp_noise
    pr = st[_S_PERM]
    perm = np.stack([pr.permutation(T * E) for _ in range(max(wl.epochs, 1))]).astype(np.int32)
    return dict(obs=obs, rewards=rewards, dones=dones, next_done=next_done,
                gumbel=gumbel, bnoise=bnoise.astype(np.float32), perm=perm)


def draw_actor_batch(wl: Workload) -> dict:
    """Actor inference inputs: uint8 frames [B, H, W, C] and Gumbel noise [B, A]."""
    net = wl.net
    st = _streams(wl.seed, 8)
    obs = st[_S_OBS].integers(0, 256, size=(wl.T, net.in_h, net.in_w, net.in_c), dtype=np.uint8)
    gumbel = st[_S_ACTOR].gumbel(size=(wl.T, net.num_actions)).astype(np.float32)
    return dict(obs=obs, gumbel=gumbel)
