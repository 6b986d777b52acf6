"""Seeded synthetic inputs for group attention.

This module only draws random numbers and rounds them to the storage dtype.
It holds none of the group-attention arithmetic, so both the GPU path and the
CPU oracle can be fed from it.

The paper's datasets (Table 1: sliding windows of length 200 / 2000 / 10000 over
3-21 channel sensor series) are not available, so the keys stand in for them as
a Gaussian mixture: the paper's premise (Section 4.1) is that periodic series
produce recurring, similar windows and hence clustered keys.  Per (b, h) slice:

  * M centres u_m = g_m / ||g_m||,  g_m ~ N(0, I_d)
  * a per-centre noise scale sigma_m ~ U[sigma_lo, sigma_hi] (per coordinate)
  * component z_i ~ U{0 .. M-1}
  * k_i = u_{z_i} + sigma_{z_i} * eps_i,  eps_i ~ N(0, I_d)
  * q_i, v_i ~ N(0, I_d) independently.

Everything is drawn in float32 from numpy's PCG64 and then rounded to the
storage dtype (bfloat16 with round-to-nearest-even, or kept as float32).

The attention block (projections around group attention) takes token
embeddings X [B, n, D] instead: per (batch, channel) the sum of four sinusoids
A sin(2 pi t / P + phi), A ~ U[0.5, 1.5], P log-uniform in [8, 1000],
phi ~ U[0, 2 pi), plus N(0, 0.1^2) noise (the periodic series of the paper's
premise), and weights W ~ N(0, 1/D), all rounded to bf16.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    """One group-attention workload: shapes, group count, iterations, key recipe."""

    name: str
    B: int
    H: int
    n: int
    d: int
    N: int | None          # None: drawn per call from N_choices
    dtype: str             # "f32" or "bf16"
    iters: int
    M: int                 # mixture components of the keys
    sigma_lo: float
    sigma_hi: float
    N_choices: tuple = ()

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


# Shapes follow the paper's workloads: window counts 200 / 2000 / 10000
# (Table 1), group counts 64..1024 (Table 4), hidden size 64 per head.
WORKLOADS = {
    "n512_N32_f32": Workload("n512_N32_f32", 1, 1, 512, 64, 32, "f32", 5, 32, 0.05, 0.05),
    "n2000_N64_bf16": Workload("n2000_N64_bf16", 8, 8, 2000, 64, 64, "bf16", 10, 64, 0.1, 0.1),
    "n8000_N128_bf16": Workload("n8000_N128_bf16", 16, 8, 8000, 64, 128, "bf16", 10, 128, 0.05, 0.3),
    "n20000_Nvar_bf16": Workload("n20000_Nvar_bf16", 4, 8, 20000, 64, None, "bf16", 10, 256, 0.05, 0.3,
                                 N_choices=(32, 64, 128, 256)),
}


@dataclasses.dataclass(frozen=True)
class BlockWorkload:
    """Attention block: projections of D = 64 H embeddings around group attention."""

    name: str
    B: int
    n: int
    H: int
    N: int
    iters: int

    @property
    def D(self) -> int:
        return 64 * self.H


BLOCK_WORKLOADS = {
    "encoder_n4000_N128_bf16": BlockWorkload("encoder_n4000_N128_bf16", 32, 4000, 8, 128, 10),
}


def to_storage(x: np.ndarray, dtype: str) -> torch.Tensor:
    """float32 numpy array -> CPU tensor in the storage dtype (bf16 uses RNE)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16) if dtype == "bf16" else t.clone()


def mixture_keys(rng: np.random.Generator, B: int, H: int, n: int, d: int, M: int,
                 sigma_lo: float, sigma_hi: float) -> np.ndarray:
    """Gaussian-mixture keys [B, H, n, d] float32 (recipe in the module docstring)."""
    g = rng.standard_normal((B, H, M, d), dtype=np.float32)
    centres = g / np.linalg.norm(g, axis=-1, keepdims=True)
    sig = rng.uniform(sigma_lo, sigma_hi, size=(B, H, M)).astype(np.float32)
    z = rng.integers(0, M, size=(B, H, n))
    eps = rng.standard_normal((B, H, n, d), dtype=np.float32)
    c = np.take_along_axis(centres, z[..., None], axis=2)
    s = np.take_along_axis(sig, z, axis=2)[..., None]
    return (c + s * eps).astype(np.float32)


def make_qkv(B: int, H: int, n: int, d: int, dtype: str, seed: int, M: int,
             sigma_lo: float, sigma_hi: float):
    """(Q, K, V) CPU tensors [B, H, n, d] in the storage dtype, from one seed."""
    rng = np.random.Generator(np.random.PCG64(seed))
    K = mixture_keys(rng, B, H, n, d, M, sigma_lo, sigma_hi)
    Q = rng.standard_normal((B, H, n, d), dtype=np.float32)
    V = rng.standard_normal((B, H, n, d), dtype=np.float32)
    return to_storage(Q, dtype), to_storage(K, dtype), to_storage(V, dtype)


def workload_inputs(w: Workload, seed: int, n: int | None = None, B: int | None = None,
                    H: int | None = None):
    """Inputs for a named workload; B/H/n may be shrunk for CPU-sized cases."""
    return make_qkv(B or w.B, H or w.H, n or w.n, w.d, w.dtype, seed, w.M, w.sigma_lo, w.sigma_hi)


def draw_group_count(w: Workload, seed: int, call: int) -> int:
    """Group count for call number `call` of a workload with a varying N."""
    if w.N is not None:
        return w.N
    rng = np.random.Generator(np.random.PCG64([seed, call]))
    return int(rng.choice(np.asarray(w.N_choices)))


def as_float64(t: torch.Tensor) -> np.ndarray:
    """Exact float64 copy of a bf16 / fp32 tensor (both widen exactly)."""
    return t.detach().to("cpu").to(torch.float64).contiguous().numpy()


def sha256(t: torch.Tensor) -> str:
    """Digest of the raw bytes of a tensor (to record which inputs were used)."""
    b = t.detach().to("cpu").contiguous().view(torch.uint8).numpy().tobytes()
    return hashlib.sha256(b).hexdigest()


def block_inputs(B: int, n: int, H: int, seed: int):
    """(X [B, n, D], Wqkv [3D, D], Wo [D, D]) bf16 CPU tensors, D = 64 H
    (recipe in the module docstring; weight rows are output features)."""
    D = 64 * H
    rng = np.random.Generator(np.random.PCG64(seed))
    t = np.arange(n, dtype=np.float32)[None, :, None]
    X = np.zeros((B, n, D), np.float32)
    for _ in range(4):
        A = rng.uniform(0.5, 1.5, size=(B, 1, D)).astype(np.float32)
        P = np.exp(rng.uniform(np.log(8.0), np.log(1000.0), size=(B, 1, D))).astype(np.float32)
        phi = rng.uniform(0.0, 2 * np.pi, size=(B, 1, D)).astype(np.float32)
        X += A * np.sin(np.float32(2 * np.pi) * t / P + phi)
    X += np.float32(0.1) * rng.standard_normal((B, n, D), dtype=np.float32)
    sd = np.float32(1.0 / np.sqrt(D))
    Wqkv = sd * rng.standard_normal((3 * D, D), dtype=np.float32)
    Wo = sd * rng.standard_normal((D, D), dtype=np.float32)
    return to_storage(X, "bf16"), to_storage(Wqkv, "bf16"), to_storage(Wo, "bf16")
