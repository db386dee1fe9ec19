"""Seeded synthetic inputs shaped like the paper's workloads.

This module draws random arrays and nothing else: it holds none of the
method's arithmetic, so that both the HIP path and the CPU oracle can take
their inputs from it.

The paper's LSTM input is the flattened observation of one hero (appendix
"Neural Network Architecture"); it is modelled as x ~ N(0, 1) of width D.
Rewards are modelled as N(0, 1) and episode ends as Bernoulli draws.  The
sizes follow the paper where it gives them: a 4096-unit LSTM, 16-step samples,
256-step segments, gamma/lambda/clip/entropy/Adam constants from Table
"Hyperparameters".

Generator: ``numpy.random.Generator(PCG64(seed))``.  Arrays are drawn in the
fixed order listed in ``make_inputs``; weights are U(-1/sqrt(H), 1/sqrt(H)).
"""
from dataclasses import dataclass, field
from typing import Tuple

import numpy as np


@dataclass(frozen=True)
class Config:
    name: str
    B: int                  # sequences (samples) in the minibatch
    T: int                  # BPTT length (timesteps per sample)
    D: int                  # LSTM input width
    H: int                  # LSTM hidden units
    head_sizes: Tuple[int, ...] = ()
    L: int = 0              # GAE segment length (0: no GAE)
    S: int = 0              # GAE segments
    done_p: float = 0.0
    state_std: float = 0.0  # h0, c0 ~ N(0, state_std); 0 means zeros
    dtype: str = "f32"
    gamma: float = 0.998
    lam: float = 0.95
    clip_eps: float = 0.2
    vf_coef: float = 1.0
    ent_coef: float = 0.01
    lr: float = 5e-5
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    clip_k: float = 5.0
    theta_noise: float = 1e-2   # behaviour-policy perturbation sigma
    extra: dict = field(default_factory=dict, compare=False, hash=False)


CONFIGS = {
    # Tiny LSTM-PPO step, fp32: each 16-step sample is its own GAE segment.
    "tiny": Config("tiny", B=8, T=16, D=64, H=128, head_sizes=(8,), L=16, S=8,
                   done_p=0.01, state_std=0.0, dtype="f32"),
    # Mid LSTM-PPO step: 256 samples = 16 segments of 256 steps.
    "mid": Config("mid", B=256, T=16, D=1024, H=1024, head_sizes=(30, 8, 32, 4),
                  L=256, S=16, done_p=0.005, state_std=0.1, dtype="f32"),
    "mid_bf16": Config("mid_bf16", B=256, T=16, D=1024, H=1024,
                       head_sizes=(30, 8, 32, 4), L=256, S=16, done_p=0.005,
                       state_std=0.1, dtype="bf16"),
    # Large bf16 step, small enough for the fp64 oracle in seconds, large
    # enough that the forward, recurrent and weight-gradient GEMMs all run on
    # the 256 x 256 MFMA engine: 2048 samples of 2 steps = 64 segments of 64.
    "big_bf16": Config("big_bf16", B=2048, T=2, D=2048, H=2048,
                       head_sizes=(30, 8, 32, 4), L=64, S=64, done_p=0.01,
                       state_std=0.1, dtype="bf16"),
    # Paper-scale LSTM forward + BPTT only.
    "lstm4096": Config("lstm4096", B=1024, T=16, D=4096, H=4096, state_std=0.1,
                       dtype="bf16"),
    # Rollout inference: one LSTM step + heads + sampling.
    "rollout4096": Config("rollout4096", B=4096, T=1, D=4096, H=4096,
                          head_sizes=(30, 8, 32, 4), state_std=0.1, dtype="bf16"),
    # Full paper-scale PPO step: 2048 samples = 128 segments of 256 steps.
    "full4096": Config("full4096", B=2048, T=16, D=4096, H=4096,
                       head_sizes=(30, 8, 32, 4), L=256, S=128, done_p=0.002,
                       state_std=0.1, dtype="bf16"),
}


def scaled(cfg: Config, **kw) -> Config:
    """A copy of ``cfg`` with some sizes replaced (for bounded samples)."""
    d = {k: getattr(cfg, k) for k in cfg.__dataclass_fields__}
    d.update(kw)
    return Config(**d)


def n_params(cfg: Config) -> int:
    A1 = sum(cfg.head_sizes) + 1 if cfg.head_sizes else 0
    return 4 * cfg.H * (cfg.D + cfg.H + 1) + A1 * (cfg.H + 1)


def _uniform(rng, shape, bound):
    return ((rng.random(shape, dtype=np.float32) * 2.0 - 1.0) * bound).astype(np.float32)


def _normal(rng, shape, std=1.0):
    a = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def make_inputs(cfg: Config, seed: int = 0, with_dh: bool = False) -> dict:
    """Draw every input of one step, in this order:

    Wx, Wh, b, Wp, bp (U(+-1/sqrt(H))), x [T,B,D], h0, c0 [B,H],
    theta' noise for Wx, Wh, b, Wp, bp (N(0, theta_noise^2)),
    rewards [L,S], dones [L,S], x_boot [B_boot, D] (the input one step after
    each segment, used for the bootstrap value), dh [T,B,H] (if with_dh).
    All float arrays are float32; dones are uint8.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    T, B, D, H = cfg.T, cfg.B, cfg.D, cfg.H
    bound = 1.0 / np.sqrt(H)
    out = {"cfg": cfg}
    out["Wx"] = _uniform(rng, (4 * H, D), bound)
    out["Wh"] = _uniform(rng, (4 * H, H), bound)
    out["b"] = _uniform(rng, (4 * H,), bound)
    if cfg.head_sizes:
        A1 = sum(cfg.head_sizes) + 1
        out["Wp"] = _uniform(rng, (A1, H), bound)
        out["bp"] = _uniform(rng, (A1,), bound)
    out["x"] = _normal(rng, (T, B, D))
    if cfg.state_std > 0:
        out["h0"] = _normal(rng, (B, H), cfg.state_std)
        out["c0"] = _normal(rng, (B, H), cfg.state_std)
    else:
        out["h0"] = np.zeros((B, H), np.float32)
        out["c0"] = np.zeros((B, H), np.float32)
    if cfg.head_sizes:
        for k in ("Wx", "Wh", "b", "Wp", "bp"):
            out["noise_" + k] = _normal(rng, out[k].shape, cfg.theta_noise)
    if cfg.L:
        out["rewards"] = _normal(rng, (cfg.L, cfg.S))
        out["dones"] = (rng.random((cfg.L, cfg.S)) < cfg.done_p).astype(np.uint8)
        out["x_boot"] = _normal(rng, (cfg.S, D))
    if with_dh:
        out["dh"] = _normal(rng, (T, B, H))
    return out


def uniform_ints(rng, shape, highs):
    """Integers in [0, highs[k]) along the last axis (e.g. actions per head)."""
    cols = [rng.integers(0, int(h), size=shape) for h in highs]
    return np.stack(cols, axis=-1).astype(np.int32)


# Minutes of game time per policy step: the game runs at 30 frames per
# second and the agent acts on every fourth frame (section "Dota 2"; section
# "Training System", subsection "Playing Dota using AI").
STEP_MINUTES = 4.0 / 30.0 / 60.0


def reward_inputs(L: int, G: int, seed: int = 0, outcome_p: float = 0.01) -> dict:
    """Raw rewards of G games of two teams of five over L steps, drawn in this
    order: shaped [L, 10G] ~ N(0, 1); outcome [L, 10G], +-1 with probability
    outcome_p each (else 0); the game minute at which each segment starts,
    U(0, 60) per game, from which game_time [L, G] advances STEP_MINUTES per
    step.  float32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shaped = _normal(rng, (L, 10 * G))
    u = rng.random((L, 10 * G))
    outcome = np.where(u < outcome_p, 1.0, np.where(u < 2 * outcome_p, -1.0, 0.0)).astype(np.float32)
    start = rng.random(G) * 60.0
    game_time = (start[None, :] + STEP_MINUTES * np.arange(L)[:, None]).astype(np.float32)
    return {"shaped": shaped, "outcome": outcome, "game_time": game_time}
