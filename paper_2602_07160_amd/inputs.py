"""Seeded synthetic inputs for the FEM read (shared by the tests, the bench and
the oracle-side checks).

This module only draws random numbers and rounds them to the storage dtype; it
holds none of the method's arithmetic, so that the oracle and the HIP path can
consume identical inputs without sharing any computation.

Workload recipe (all draws from ``numpy.random.default_rng(seed)``, in the
order q, k, v, [offset], beta; bf16 storage is round-to-nearest-even from the
float32 draw, and the oracle upcasts the stored bits exactly):

  1  softmax, fp32:  B=1,  H=1,  T=128,   d=32;  q,k,v ~ N(0,1); beta log-U[0.25, 4]
  2  softmax, bf16:  B=4,  H=8,  T=1024,  d=64;  q,k,v ~ N(0,1); beta log-U[0.1, 8]
  3  softmax, bf16:  B=8,  H=16, T=4096,  d=128; q,k,v ~ N(0,1); beta log-U[0.1, 8]
  4  softmax, bf16:  B=1,  H=8,  T=16384, d=64;  q,k ~ N(0,1);
                     v = clip(N(0,1) + offset, -5, 5), offset ~ N(0, 4) per (b,h,j);
                     beta log-U[1, 16]
  5  linear,  bf16:  B=4,  H=16, T=8192,  d_k=d_v=64, chunk 64;
                     q,k,v ~ N(0,1); beta log-U[0.1, 4]

Gates of the two-level gated read (``draw_gates``), per (b, h, t, j), from
their own generator: lam = sigmoid(z), z ~ N(0, 2^2), which puts mass near 0,
near 1 and in between; g = softplus(y), y ~ N(0, 1), divided by its root mean
square over the channels of the step (the paper's RMS-normalised positive
outer gate, with unit scale).

GLA log-decays (``draw_gla_decay``), per (b, h, t, c): g = log(sigmoid(z)) / 16,
z ~ N(0, 1) -- the gate parameterisation of gated linear attention with its
usual normaliser of 16, i.e. decay factors around 0.96 per step.

The paper's own speed measurements use randomly generated data, and its
language-model runs use T=4096 with head dimension 128; these shapes stand in
for those workloads.  beta has shape [H, d] (one inverse temperature per head
and channel, shared over batch and time).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

BASE_SEED = 42


@dataclass(frozen=True)
class Workload:
    no: int
    kind: str          # "softmax" or "linear"
    dtype: str         # "f32" or "bf16"
    B: int
    H: int
    T: int
    d: int             # d (softmax) or d_k (linear)
    dv: int            # value width (== d for softmax)
    beta_lo: float
    beta_hi: float
    offset_var: float = 0.0   # variance of the per-(b,h,j) value offset
    clip: float = 0.0         # |v| clip (0: none)
    chunk: int = 0            # linear-prior chunk length

    @property
    def name(self) -> str:
        return (f"fem_{self.kind}_{self.dtype}_B{self.B}_H{self.H}_T{self.T}"
                f"_d{self.d}" + (f"_dv{self.dv}" if self.dv != self.d else ""))


WORKLOADS = {
    1: Workload(1, "softmax", "f32", 1, 1, 128, 32, 32, 0.25, 4.0),
    2: Workload(2, "softmax", "bf16", 4, 8, 1024, 64, 64, 0.1, 8.0),
    3: Workload(3, "softmax", "bf16", 8, 16, 4096, 128, 128, 0.1, 8.0),
    4: Workload(4, "softmax", "bf16", 1, 8, 16384, 64, 64, 1.0, 16.0,
                offset_var=4.0, clip=5.0),
    5: Workload(5, "linear", "bf16", 4, 16, 8192, 64, 64, 0.1, 4.0, chunk=64),
}


def _store(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def draw(seed: int, B: int, H: int, T: int, d: int, dv: int | None = None, *,
         dtype: str = "bf16", beta_lo: float = 0.1, beta_hi: float = 8.0,
         offset_var: float = 0.0, clip: float = 0.0):
    """Draw (q, k, v, beta) as CPU torch tensors.

    q, k: [B, H, T, d]; v: [B, H, T, dv] in ``dtype`` ("bf16" or "f32");
    beta: [H, dv] float32, log-uniform in [beta_lo, beta_hi].
    """
    dv = d if dv is None else dv
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, T, d), dtype=np.float32)
    k = rng.standard_normal((B, H, T, d), dtype=np.float32)
    v = rng.standard_normal((B, H, T, dv), dtype=np.float32)
    if offset_var > 0.0:
        off = rng.normal(0.0, np.sqrt(offset_var), size=(B, H, 1, dv)).astype(np.float32)
        v = v + off
    if clip > 0.0:
        v = np.clip(v, -clip, clip)
    beta = np.exp(rng.uniform(np.log(beta_lo), np.log(beta_hi), size=(H, dv)))
    return (_store(q, dtype), _store(k, dtype), _store(v, dtype),
            torch.from_numpy(beta.astype(np.float32)))


def make_inputs(no: int, **override):
    """Inputs of workload ``no`` (1..5) with seed 42 + no; fields of the
    workload may be overridden (e.g. T=256 for a reduced parity case)."""
    w = WORKLOADS[no]
    f = dict(B=w.B, H=w.H, T=w.T, d=w.d, dv=w.dv, dtype=w.dtype,
             beta_lo=w.beta_lo, beta_hi=w.beta_hi,
             offset_var=w.offset_var, clip=w.clip)
    f.update(override)
    seed = f.pop("seed", BASE_SEED + no)
    return draw(seed, **f)


def toy_argmax_values(seed: int, T: int = 128, D: int = 512,
                      delta: float = 1.0, sigma: float = 0.05):
    """Values of the paper's single-layer channel-wise argmax toy (Appendix
    "Toy problem: single-layer channel-wise argmax"): per channel j one winner
    a_j drawn uniformly, V[a_j, j] = delta + eps_j and V[i != a_j, j] ~ N(0,
    sigma^2).  eps_j is read here as N(0, sigma^2), the same noise level as
    the other entries.  Returns (V [T, D] float64, winners [D] int64).
    """
    rng = np.random.default_rng(seed)
    a = rng.integers(0, T, size=D)
    v = rng.normal(0.0, sigma, size=(T, D))
    v[a, np.arange(D)] = delta + rng.normal(0.0, sigma, size=D)
    return v, a


def draw_gates(seed: int, B: int, H: int, T: int, d: int):
    """Draw (lam, gate) as CPU float32 tensors [B, H, T, d] (recipe above)."""
    rng = np.random.default_rng(seed)
    z = rng.normal(0.0, 2.0, size=(B, H, T, d)).astype(np.float32)
    lam = (1.0 / (1.0 + np.exp(-z))).astype(np.float32)
    y = rng.standard_normal((B, H, T, d), dtype=np.float32)
    g = np.logaddexp(np.float32(0.0), y)
    g = g / np.sqrt(np.mean(g * g, axis=-1, keepdims=True))
    return torch.from_numpy(np.ascontiguousarray(lam)), \
        torch.from_numpy(np.ascontiguousarray(g.astype(np.float32)))


def draw_gla_decay(seed: int, B: int, H: int, T: int, dk: int, scale: float = 1.0 / 16.0):
    """Draw GLA log-decays g = scale * log(sigmoid(z)), z ~ N(0, 1), as a CPU
    float32 tensor [B, H, T, dk] (recipe above)."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((B, H, T, dk))
    g = -np.logaddexp(0.0, -z) * scale
    return torch.from_numpy(np.ascontiguousarray(g.astype(np.float32)))
