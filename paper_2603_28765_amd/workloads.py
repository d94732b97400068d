"""Seeded synthetic inputs for the five measured workloads.

Shapes and value distributions only: no quantization arithmetic lives here,
so both the HIP path and the CPU oracle can take their inputs from this
module.  Values are drawn in float64 with numpy's PCG64, then rounded to
bf16 (round to nearest even, via torch).  Seeds: the tiny case uses seed 0;
every other tensor uses 1000 * workload + tensor index; the 16-bit RHT sign
mask comes from seed + 100 and the stochastic-rounding seed is seed + 200.

They stand in for the paper's tensors (activations, weights and gradients
of the models it quantizes), which are not available here.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch


def to_bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)


def rht_mask(seed: int) -> int:
    return int(np.random.default_rng(seed + 100).integers(0, 1 << 16))


def sr_seed(seed: int) -> int:
    return seed + 200


@dataclass
class Workload:
    name: str
    tensors: dict = field(default_factory=dict)   # name -> bf16 CPU tensor
    seeds: dict = field(default_factory=dict)     # name -> generator seed
    info: dict = field(default_factory=dict)


def tiny(seed: int = 0, n: int = 256) -> Workload:
    """A and B, 256x256, N(0,1); IF4 RTN along K; GEMM 256^3 with fp32 out."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((n, n))
    b = rng.standard_normal((n, n))
    return Workload("tiny_256", {"A": to_bf16(a), "B": to_bf16(b)}, {"A": seed, "B": seed},
                    {"M": n, "N": n, "K": n})


def student_t_outlier_columns(rows: int, cols: int, seed: int, df: float = 3.0,
                              scale: float = 0.5, frac: float = 0.001, boost: float = 50.0):
    """Student-t(df) * scale with a seeded 0.1% of columns multiplied by 50."""
    rng = np.random.default_rng(seed)
    x = rng.standard_t(df, size=(rows, cols)) * scale
    n_out = int(np.floor(frac * cols))
    cols_out = rng.choice(cols, size=n_out, replace=False)
    x[:, cols_out] *= boost
    return x, np.sort(cols_out)


def quant_sweep(rows: int = 8192, cols: int = 8192) -> Workload:
    """Quantizer bandwidth workload: 8192x8192 t(3)*0.5 with 8 outlier columns
    (x50); quantized along rows, with and without the 16-point RHT."""
    seed = 2000
    x, oc = student_t_outlier_columns(rows, cols, seed)
    return Workload(f"quant_{rows}x{cols}", {"X": to_bf16(x)}, {"X": seed},
                    {"outlier_columns": oc.tolist(), "rht_signs": rht_mask(seed)})


def fwd_mlp(M: int = 8192, N: int = 14336, K: int = 4096) -> Workload:
    """Forward MLP up-projection: activations t(4) with a lognormal(0,1)
    scale per K channel, weights N(0, 0.02^2); Y = X W^T, bf16 out."""
    sa, sw = 3000, 3001
    rng = np.random.default_rng(sa)
    ch = rng.lognormal(0.0, 1.0, size=K)
    a = rng.standard_t(4.0, size=(M, K)) * ch[None, :]
    w = np.random.default_rng(sw).standard_normal((N, K)) * 0.02
    return Workload(f"fwd_mlp_{M}x{N}x{K}", {"A": to_bf16(a), "W": to_bf16(w)}, {"A": sa, "W": sw},
                    {"M": M, "N": N, "K": K})


def wgrad(T: int = 8192, N_out: int = 14336, N_in: int = 4096) -> Workload:
    """Weight gradient dW = dY^T X: dY [T, N_out] Laplace(0, 1e-3), X [T, N_in]
    N(0,1), both quantized along the token axis with RHT (shared mask),
    stochastic rounding and the 16/17 margin; fp32 out."""
    sd, sx = 4000, 4001
    dy = np.random.default_rng(sd).laplace(0.0, 1e-3, size=(T, N_out))
    x = np.random.default_rng(sx).standard_normal((T, N_in))
    return Workload(f"wgrad_{N_out}x{N_in}x{T}", {"dY": to_bf16(dy), "X": to_bf16(x)},
                    {"dY": sd, "X": sx},
                    {"M": N_out, "N": N_in, "K": T, "rht_signs": rht_mask(sd),
                     "sr_seed_dY": sr_seed(sd), "sr_seed_X": sr_seed(sx)})


def bitwidth(n: int = 8192) -> Workload:
    """A, B n x n N(0,1) with a seeded 0.05% of elements multiplied by 100;
    quantized to IF3, IF4, IF6 and NVFP4 along K."""
    out = {}
    seeds = {}
    for idx, name in enumerate(("A", "B")):
        seed = 5000 + idx
        rng = np.random.default_rng(seed)
        x = rng.standard_normal((n, n))
        k = int(np.floor(0.0005 * n * n))
        pos = rng.choice(n * n, size=k, replace=False)
        x.reshape(-1)[pos] *= 100.0
        out[name] = to_bf16(x)
        seeds[name] = seed
    return Workload(f"bitwidth_{n}", out, seeds, {"M": n, "N": n, "K": n})


def small_like(kind: str, scale: int = 16) -> Workload:
    """The same distributions at 1/scale of each dimension (parity tests)."""
    if kind == "quant_sweep":
        return quant_sweep(8192 // scale, 8192 // scale)
    if kind == "fwd_mlp":
        return fwd_mlp(8192 // scale, 14336 // scale, 4096 // scale)
    if kind == "wgrad":
        return wgrad(8192 // scale, 14336 // scale, 4096 // scale)
    if kind == "bitwidth":
        return bitwidth(8192 // scale)
    raise ValueError(kind)
