"""Seeded synthetic workloads for the PULSE patch codec.

This module only draws random numbers and lays out tensor shapes.  It holds
none of the codec's arithmetic (no BF16 cast, no comparison, no compaction, no
scatter): the snapshot each side needs is computed by that side.  Both the GPU
path's tests/benchmark and the CPU oracle's tests take their inputs from here,
so the two always see identical bytes.

What the synthetic streams stand in for.  The paper measures update sparsity on
Qwen2.5 / Llama-3.2 / Gemma-3 checkpoints trained with GRPO on MATH (Sec. 3,
App. F); none of those weights or datasets are used.  Instead:

* Weights: matrices w ~ N(0, 0.02) (variance), RMSNorm gains = 1.0 (exactly on
  the BF16 grid).  App. A.4's weight-magnitude table puts real median |w| at
  0.01-0.02; the synthetic sd of 0.141 is the configuration's stated law.
* Updates: an Adam-normalised direction u = clip(m / (sqrt(v) + 1e-8), -10, 10)
  with m ~ N(0, 1e-3), v = |N(0, 1e-6)|; the clip is the 10*eta one-step Adam
  bound of App. A.3 (Thm. "adam_bound", default betas).  New master
  w' = fl32(w - fl32(lr * u)), each op rounded separately in FP32.
* PULSELoCo pseudo-gradients: Delta = N(0, 1e-5) * |N(0, 1)|^2, fresh each round
  (heavy-tailed, standing in for H = 8 inner Adam steps, Sec. 4.3 / App. B).

``N(0, x)`` is read as variance x throughout (``reading="variance"``, the
default).  ``reading="std"`` reads it as standard deviation x instead: the
other reading of the configurations' notation, which gives about five times
the patch density (4.7% at lr 1e-6) and brackets the density range.

Parameter-set shapes follow the Qwen2.5 layout (no biases; per layer
input-norm, q, k, v, o, post-norm, gate, up, down; final norm):

* ``0.5b``: hidden 896, 24 layers, GQA k/v 128x896, MLP 4864, tied embedding
  151936x896 -> 494,005,120 params in 218 tensors.
* ``7b``:   hidden 3584, 28 layers, k/v 512x3584, MLP 18944, untied vocab
  152064 -> 7,615,487,488 params in 255 tensors.
* ``32b``:  hidden 5120, 64 layers, k/v 1024x5120, MLP 27648, untied vocab
  152064 -> 32,763,417,600 params in 579 tensors.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

W_VAR = 0.02          # matrices ~ N(0, 0.02)
M_VAR = 1e-3          # m ~ N(0, 1e-3)
V_VAR = 1e-6          # v = |N(0, 1e-6)|
ADAM_EPS = 1e-8
U_CLIP = 10.0         # 10 * eta one-step bound, App. A.3
LOCO_VAR = 1e-5       # Delta ~ N(0, 1e-5) * |N(0,1)|^2
LOCO_KEEP = 0.02      # tau chosen so ~2% of round-1 entries survive
READINGS = ("variance", "std")


def sd(x: float, reading: str = "variance") -> float:
    """Standard deviation of N(0, x) under a reading of the notation."""
    if reading == "variance":
        return math.sqrt(x)
    if reading == "std":
        return x
    raise ValueError(f"unknown reading {reading!r}; expected one of {READINGS}")


@dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: tuple
    is_norm: bool

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))


@dataclass(frozen=True)
class ModelShape:
    key: str
    hidden: int
    layers: int
    kv_dim: int
    inter: int
    vocab: int
    tied: bool

    def tensors(self) -> list[TensorSpec]:
        h, out = self.hidden, []
        out.append(TensorSpec("embed_tokens", (self.vocab, h), False))
        for i in range(self.layers):
            p = f"layers.{i}."
            out += [
                TensorSpec(p + "input_layernorm", (h,), True),
                TensorSpec(p + "q_proj", (h, h), False),
                TensorSpec(p + "k_proj", (self.kv_dim, h), False),
                TensorSpec(p + "v_proj", (self.kv_dim, h), False),
                TensorSpec(p + "o_proj", (h, h), False),
                TensorSpec(p + "post_attention_layernorm", (h,), True),
                TensorSpec(p + "gate_proj", (self.inter, h), False),
                TensorSpec(p + "up_proj", (self.inter, h), False),
                TensorSpec(p + "down_proj", (h, self.inter), False),
            ]
        out.append(TensorSpec("norm", (h,), True))
        if not self.tied:
            out.append(TensorSpec("lm_head", (self.vocab, h), False))
        return out

    def numel(self) -> int:
        return sum(t.numel for t in self.tensors())


SHAPES = {
    "0.5b": ModelShape("0.5b", 896, 24, 128, 4864, 151936, tied=True),
    "7b": ModelShape("7b", 3584, 28, 512, 18944, 152064, tied=False),
    "32b": ModelShape("32b", 5120, 64, 1024, 27648, 152064, tied=False),
}

SINGLE_N = 1 << 20


def mix_seed(*parts: int) -> int:
    """Deterministic 63-bit seed from integers (splitmix64 finaliser chain)."""
    x = 0x9E3779B97F4A7C15
    for p in parts:
        x = (x ^ (int(p) & 0xFFFFFFFFFFFFFFFF)) & 0xFFFFFFFFFFFFFFFF
        x = (x + 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF
        z = x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & 0xFFFFFFFFFFFFFFFF
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & 0xFFFFFFFFFFFFFFFF
        x = z ^ (z >> 31)
    return x & 0x7FFFFFFFFFFFFFFF


# --------------------------------------------------------------------------- numpy (CPU) draws

def adam_direction_np(rng: np.random.Generator, n: int, reading: str = "variance") -> np.ndarray:
    """u = clip(m / (sqrt(v) + eps), -10, 10) in FP32, draws in the order m, v."""
    m = rng.normal(0.0, sd(M_VAR, reading), n).astype(np.float32)
    v = np.abs(rng.normal(0.0, sd(V_VAR, reading), n)).astype(np.float32)
    u = m / (np.sqrt(v) + np.float32(ADAM_EPS))
    return np.clip(u, np.float32(-U_CLIP), np.float32(U_CLIP)).astype(np.float32)


def adam_step_np(w: np.ndarray, u: np.ndarray, lr: float) -> np.ndarray:
    """w' = fl32(w - fl32(lr * u)); two separately rounded FP32 ops."""
    step = (np.float32(lr) * u).astype(np.float32)
    return (w - step).astype(np.float32)


def single_tensor_inputs(lr: float = 1e-6, n: int = SINGLE_N, seed: int = 0,
                         reading: str = "variance"):
    """Single FP32 tensor: default_rng(seed), draws in the order w, m, v.

    Returns (w, w_new) as float32 arrays; the snapshot is bf16(w), computed by
    whichever side consumes these inputs.
    """
    rng = np.random.default_rng(seed)
    w = rng.normal(0.0, sd(W_VAR, reading), n).astype(np.float32)
    u = adam_direction_np(rng, n, reading)
    return w, adam_step_np(w, u, lr)


def loco_delta_np(rng: np.random.Generator, n: int) -> np.ndarray:
    """Delta = N(0, 1e-5) * |N(0,1)|^2 in FP32."""
    z1 = rng.normal(0.0, math.sqrt(LOCO_VAR), n).astype(np.float32)
    z2 = rng.normal(0.0, 1.0, n).astype(np.float32)
    return (z1 * (z2 * z2)).astype(np.float32)


def loco_tau(keep: float = LOCO_KEEP, sample: int = 1 << 22, seed: int = 5) -> float:
    """Threshold keeping ~`keep` of round-1 |Delta| (a fixed-seed sample quantile).

    tau is the caller's choice; it is fixed once and reused for every round, so
    the surviving fraction grows as the residual accumulates.
    """
    d = np.abs(loco_delta_np(np.random.default_rng(seed), sample))
    k = int(math.ceil((1.0 - keep) * sample)) - 1
    return float(np.partition(d, k)[k])


# --------------------------------------------------------------------------- torch (GPU) draws

def _gen(device, *seed_parts):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(mix_seed(*seed_parts))
    return g


def init_weights_(w, spec: TensorSpec, *seed_parts, reading: str = "variance"):
    """Fill an FP32 tensor in place: gains = 1.0, matrices ~ N(0, 0.02)."""
    if spec.is_norm:
        w.fill_(1.0)
    else:
        w.normal_(0.0, sd(W_VAR, reading), generator=_gen(w.device, 1, *seed_parts))
    return w


def adam_step_(w, lr: float, *seed_parts, reading: str = "variance"):
    """w <- fl32(w - fl32(lr * u)) in place with a fresh Adam-like direction u."""
    import torch
    g = _gen(w.device, 2, *seed_parts)
    m = torch.empty_like(w).normal_(0.0, sd(M_VAR, reading), generator=g)
    v = torch.empty_like(w).normal_(0.0, sd(V_VAR, reading), generator=g).abs_()
    v.sqrt_().add_(ADAM_EPS)
    m.div_(v).clamp_(-U_CLIP, U_CLIP).mul_(lr)
    del v
    w.sub_(m)
    return w


def loco_delta_(d, *seed_parts):
    """Fill d in place with Delta = N(0, 1e-5) * |N(0,1)|^2."""
    import torch
    g = _gen(d.device, 3, *seed_parts)
    d.normal_(0.0, math.sqrt(LOCO_VAR), generator=g)
    z = torch.empty_like(d).normal_(0.0, 1.0, generator=g)
    z.mul_(z)
    d.mul_(z)
    return d
