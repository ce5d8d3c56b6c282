"""Seeded synthetic workloads for the R-iKFAD optimiser step.

This module only produces inputs (shapes, initial parameters, gradient
streams); it holds none of the optimiser's arithmetic.  The parameter sets
are shaped like the models the paper trains (Section 4: GPT2-Nano, TinyViT,
DistilBERT, GPT2-S); the paper's datasets and trained weights are replaced by
random gradients g_ij = s_i t_j z_ij with z ~ N(0, 1) drawn fresh every step
and per-tensor row / column scales s, t fixed by the seed.

Every array is a deterministic function of (seed, tensor index, step), drawn
with numpy's PCG64 on the host, so that the GPU path and the oracle see the
same bits.  bf16 tensors are produced by rounding the fp32 draw to bf16 with
torch's CPU conversion; the values handed out are exactly representable.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class TensorSpec:
    name: str
    m: int
    n: int
    dtype: str = "fp32"          # storage type of x and g: "fp32" or "bf16"

    @property
    def numel(self):
        return self.m * self.n

    @property
    def is_vector(self):
        return self.m == 1 or self.n == 1


# ---------------------------------------------------------------- shapes

def single_matrix(m=256, n=512, dtype="fp32"):
    return [TensorSpec("w", m, n, dtype)]


def gpt2_nano(dtype="fp32"):
    """nanoGPT character-level model: 6 blocks, d = 384, vocab 65, context 256."""
    d = 384
    out = [TensorSpec("wte", 65, d, dtype), TensorSpec("wpe", 256, d, dtype)]
    for b in range(6):
        out += [TensorSpec(f"h{b}.ln_1.w", 1, d, dtype), TensorSpec(f"h{b}.ln_1.b", 1, d, dtype),
                TensorSpec(f"h{b}.attn.qkv", d, 3 * d, dtype),
                TensorSpec(f"h{b}.attn.proj", d, d, dtype),
                TensorSpec(f"h{b}.ln_2.w", 1, d, dtype), TensorSpec(f"h{b}.ln_2.b", 1, d, dtype),
                TensorSpec(f"h{b}.mlp.fc", d, 4 * d, dtype),
                TensorSpec(f"h{b}.mlp.proj", 4 * d, d, dtype)]
    out += [TensorSpec("ln_f.w", 1, d, dtype), TensorSpec("ln_f.b", 1, d, dtype)]
    return out


def gpt2_small(dtype="fp32"):
    """GPT-2 small: 12 blocks, d = 768, vocab 50257, context 1024, with the
    98 bias / LayerNorm vectors."""
    d = 768
    out = [TensorSpec("wte", 50257, d, dtype), TensorSpec("wpe", 1024, d, dtype)]
    for b in range(12):
        out += [TensorSpec(f"h{b}.ln_1.w", 1, d, dtype), TensorSpec(f"h{b}.ln_1.b", 1, d, dtype),
                TensorSpec(f"h{b}.attn.qkv", d, 3 * d, dtype),
                TensorSpec(f"h{b}.attn.qkv.b", 1, 3 * d, dtype),
                TensorSpec(f"h{b}.attn.proj", d, d, dtype),
                TensorSpec(f"h{b}.attn.proj.b", 1, d, dtype),
                TensorSpec(f"h{b}.ln_2.w", 1, d, dtype), TensorSpec(f"h{b}.ln_2.b", 1, d, dtype),
                TensorSpec(f"h{b}.mlp.fc", d, 4 * d, dtype),
                TensorSpec(f"h{b}.mlp.fc.b", 1, 4 * d, dtype),
                TensorSpec(f"h{b}.mlp.proj", 4 * d, d, dtype),
                TensorSpec(f"h{b}.mlp.proj.b", 1, d, dtype)]
    out += [TensorSpec("ln_f.w", 1, d, dtype), TensorSpec("ln_f.b", 1, d, dtype)]
    return out


def tinyvit_like(seed=0, count=150, dtype="bf16"):
    """Many small tensors: `count` matrices with m in {64,128,160,320,576} and
    n in {64,128,256,640,1280}, four 3x3 conv kernels flattened to
    (out, in*9), and one bias vector per matrix and per conv."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x7173])))
    ms = [64, 128, 160, 320, 576]
    ns = [64, 128, 256, 640, 1280]
    out = []
    for (o, i) in [(64, 3), (128, 64), (160, 128), (320, 160)]:
        out.append(TensorSpec(f"conv{o}x{i}", o, i * 9, dtype))
        out.append(TensorSpec(f"conv{o}x{i}.b", 1, o, dtype))
    for k in range(count):
        m = int(rng.choice(ms))
        n = int(rng.choice(ns))
        out.append(TensorSpec(f"lin{k}", m, n, dtype))
        out.append(TensorSpec(f"lin{k}.b", 1, m, dtype))
    return out


def distilbert_stress(big_dtype="bf16", big_count=32):
    """DistilBERT-shaped (6 blocks, d = 768, q/k/v separate, 30522 x 768
    embedding; fp32) plus big_count matrices of 4096 x 11008 / 11008 x 4096."""
    d = 768
    out = [TensorSpec("word_emb", 30522, d, "fp32")]
    for b in range(6):
        for nm in ("q", "k", "v"):
            out.append(TensorSpec(f"l{b}.{nm}", d, d, "fp32"))
        out += [TensorSpec(f"l{b}.ffn1", d, 4 * d, "fp32"),
                TensorSpec(f"l{b}.ffn2", 4 * d, d, "fp32")]
    for k in range(big_count):
        if k % 2 == 0:
            out.append(TensorSpec(f"big{k}", 4096, 11008, big_dtype))
        else:
            out.append(TensorSpec(f"big{k}", 11008, 4096, big_dtype))
    return out


# ------------------------------------------------------------ hyperparameters

# Parity configurations (h, gamma, alpha, mu, eps_stab).
HP_BASE = dict(h=1e-3, gamma=0.0, alpha=0.1, mu=1.0, eps_stab=1e-8)
# Friction strong enough to move the momentum visibly: the median (h/2) xi
# reaches ~0.1 within tens of steps, so the half-kicks are exercised.
HP_FRICTION = dict(h=0.1, gamma=0.0, alpha=0.1, mu=0.1, eps_stab=1e-8)
# Friction that is already active after a few steps (median (h/2) xi~
# about 0.065 after 5 steps of these gradients), for the full-size sets,
# which the oracle can follow for only a handful of steps.
HP_FRICTION_FULL = dict(h=0.1, gamma=0.0, alpha=0.1, mu=0.01, eps_stab=1e-8)
# The paper's tuned GPT2-S values for R-iKFAD0 (App. Optimal Hyperparameters,
# Table of optimised hyperparameters; eps_stab from Section 4).
HP_GPT2S_TUNED = dict(h=0.0918, gamma=0.0, alpha=0.0579, mu=1.3637e-6, eps_stab=1e-16)


# ---------------------------------------------------------------- values

def _rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def to_storage(a32, dtype):
    """Round an fp32 array to the storage type; returns fp32 values that are
    exactly representable in that type."""
    a32 = np.ascontiguousarray(a32, dtype=np.float32)
    if dtype == "fp32":
        return a32
    if dtype == "bf16":
        import torch
        t = torch.from_numpy(a32).to(torch.bfloat16).to(torch.float32)
        return t.numpy()
    raise ValueError(dtype)


class Workload:
    """Initial parameters and per-step gradients of a parameter list.

    scales: "lognormal" -> s_i, t_j ~ LogNormal(0, 0.5);
            "student_t" -> s_i = |T_i| with T ~ Student-t(3), t_j = 1.
    """

    def __init__(self, specs, seed=0, scales="lognormal", x_std=0.02):
        self.specs = list(specs)
        self.seed = int(seed)
        self.scales = scales
        self.x_std = float(x_std)
        self._st = {}

    @property
    def numel(self):
        return sum(s.numel for s in self.specs)

    def row_col_scales(self, i):
        if i not in self._st:
            sp = self.specs[i]
            rng = _rng(self.seed, i, 0x5CA1E)
            if self.scales == "lognormal":
                s = rng.lognormal(0.0, 0.5, sp.m).astype(np.float32)
                t = rng.lognormal(0.0, 0.5, sp.n).astype(np.float32)
            elif self.scales == "student_t":
                s = np.abs(rng.standard_t(3.0, sp.m)).astype(np.float32)
                t = np.ones(sp.n, dtype=np.float32)
            else:
                raise ValueError(self.scales)
            self._st[i] = (s, t)
        return self._st[i]

    def x0(self, i):
        sp = self.specs[i]
        z = _rng(self.seed, i, 0x10).standard_normal((sp.m, sp.n), dtype=np.float32)
        return to_storage(z * np.float32(self.x_std), sp.dtype)

    def grad(self, i, step):
        sp = self.specs[i]
        s, t = self.row_col_scales(i)
        z = _rng(self.seed, i, 0x20, step).standard_normal((sp.m, sp.n), dtype=np.float32)
        z *= s[:, None]
        z *= t[None, :]
        return to_storage(z, sp.dtype)


CONFIGS = {
    "single": lambda: single_matrix(),
    "gpt2_nano": lambda: gpt2_nano(),
    "tinyvit": lambda: tinyvit_like(),
    "gpt2_small": lambda: gpt2_small(),
    "gpt2_small_bf16": lambda: gpt2_small("bf16"),
    "distilbert_stress": lambda: distilbert_stress(),
}
