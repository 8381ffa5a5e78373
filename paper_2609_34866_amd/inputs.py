"""Seeded synthetic workloads for the JAB attention-block loss.

This module only draws numbers: it builds the calibration activations X and the
fused projection weights W = [W_Q | W_K | W_V] with the shapes and value
distributions of the workloads the library is measured on.  It holds none of the
method's arithmetic (no quantizer, projection, attention or loss) so that the
oracle and the GPU path can both consume its output without sharing code.

Shapes follow the paper's problem statement (Section "Layer-wise PTQ"): X is
[batch][seq_len][d_model] of independent sequences; the fused weight is stored
as [R][d_model] with R = (n_heads + 2 n_kv_heads) head_dim, i.e. one row per
output channel, Q rows first, then K, then V (the nn.Linear orientation; the
paper's Appendix on the full-model setup warns that quantizing along the wrong
axis of the transposed Conv1D layout is a silent error).

Recipes
-------
* ``gauss_outlier`` (tiny block): X ~ N(0,1); ``outliers`` channels, picked by a
  seeded permutation, are multiplied by ``outlier_scale``.
* ``rms_outlier`` (GPT-2 and Mistral shapes): each token is drawn N(0,1),
  divided by its root-mean-square over channels (no epsilon), then
  ceil(outlier_frac * d_model) channels picked by a seeded permutation are
  multiplied by ``outlier_scale``.  This stands in for the post-RMSNorm residual
  stream with heavy-tailed outlier channels that feeds a real QKV projection;
  the paper's WikiText-2 / C4 activations are not available.
* Weights: each of W_Q, W_K, W_V ~ N(0, w_std^2), drawn independently.

All draws are float32 from numpy's PCG64 and are rounded to the storage dtype
with round-to-nearest-even.  Every sequence and every matrix has its own
SeedSequence, so any subset of sequences can be regenerated alone:
X[b] <- SeedSequence([seed, 1, b]), W_m <- SeedSequence([seed, 2, m]),
outlier permutation <- SeedSequence([seed, 3]).
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from itertools import product
from typing import Optional, Sequence

import numpy as np
import torch

DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

# Candidate bit-widths of the knapsack sweep.  The paper's set also holds 16
# (= left in float), which is the teacher itself.
SWEEP_BITS = (2, 3, 4, 8)


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    seq_len: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    group_size: int
    dtype: str                      # "f32" | "f16" | "bf16"
    bits: tuple                     # tuple of (b_Q, b_K, b_V) triples evaluated
    op: str                         # "fwd" | "sweep" | "bwd" | "kl" | "curv" | "fisher" | "ft" | "bwd_kl"
    x_recipe: str                   # "gauss_outlier" | "rms_outlier"
    outliers: Optional[int] = None  # absolute outlier-channel count (gauss_outlier)
    outlier_frac: float = 0.01
    outlier_scale: float = 20.0
    w_std: float = 0.02
    seed: int = 0
    symmetric: bool = False
    lambda_kl: float = 0.0          # weight of the KL attention-map term in fine-tuning ("ft")
    rope_theta: float = 0.0         # RoPE base on Q and K (0: none; Mistral-7B-v0.1: 10000)
    probes: int = 0                 # Rademacher probes per curvature call ("curv"), Adam steps ("ft")

    @property
    def rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def tokens(self) -> int:
        return self.batch * self.seq_len

    @property
    def n_outliers(self) -> int:
        if self.outliers is not None:
            return self.outliers
        return int(math.ceil(self.outlier_frac * self.d_model))

    @property
    def torch_dtype(self) -> torch.dtype:
        return DTYPES[self.dtype]

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    # Tiny block in fp32: d=64, 4 heads x 16, 2 x 32 tokens, 4-bit, g=32.
    "tiny_fp32": Workload("tiny_fp32", 2, 32, 64, 4, 4, 16, 32, "f32", ((4, 4, 4),), "fwd",
                          "gauss_outlier", outliers=2, outlier_scale=10.0, w_std=0.05),
    # GPT-2-small-shaped block in fp16: d=768, 12 x 64 MHA, 32 x 1024 tokens.
    "gpt2_fp16": Workload("gpt2_fp16", 32, 1024, 768, 12, 12, 64, 128, "f16",
                          ((3, 3, 3), (4, 4, 4)), "fwd", "rms_outlier"),
    # Mistral-7B-shaped block in bf16: d=4096, 32 q / 8 kv heads x 128, 128 x 2048.
    "mistral_bf16": Workload("mistral_bf16", 128, 2048, 4096, 32, 8, 128, 128, "bf16",
                             ((3, 3, 3),), "fwd", "rms_outlier"),
    # Knapsack scoring sweep at the Mistral shape: all of {2,3,4,8}^3 at 32 x 2048.
    "mistral_sweep": Workload("mistral_sweep", 32, 2048, 4096, 32, 8, 128, 128, "bf16",
                              tuple(product(SWEEP_BITS, repeat=3)), "sweep", "rms_outlier"),
    # The joint objective with the KL attention-map term at the Mistral shape (the inputs of
    # mistral_bf16): squared error and D_KL(P || Q) from one student projection.
    "mistral_kl": Workload("mistral_kl", 128, 2048, 4096, 32, 8, 128, 128, "bf16",
                           ((3, 3, 3),), "kl", "rms_outlier"),
    # Curvature scores at the Mistral shape (the inputs of mistral_bf16): ten Rademacher probes
    # (the paper's count per layer), the exact Hutchinson terms of eq. gn with the KL term at the
    # paper's lambda_KL = 0.1 for each.
    "mistral_curv": Workload("mistral_curv", 128, 2048, 4096, 32, 8, 128, 128, "bf16",
                             ((0, 0, 0),), "curv", "rms_outlier", probes=10, lambda_kl=0.1),
    # The Mistral forward loss with Mistral's rotary embedding on Q and K (base 10000): the
    # block-faithful variant of mistral_bf16 (same inputs).
    "mistral_bf16_rope": Workload("mistral_bf16_rope", 128, 2048, 4096, 32, 8, 128, 128, "bf16",
                                  ((3, 3, 3),), "fwd", "rms_outlier", rope_theta=10000.0),
    # Joint STE fine-tuning at the STE-step shape: 200 Adam steps (the paper's count), a held-out
    # batch of 16 further sequences scored every 10 steps.
    "mistral_ft": Workload("mistral_ft", 16, 2048, 4096, 32, 8, 128, 128, "bf16",
                           ((3, 3, 3),), "ft", "rms_outlier", probes=200),
    # STE step of the paper's default objective (lambda_KL = 0.1) at the STE-step shape.
    "mistral_ste_kl": Workload("mistral_ste_kl", 16, 2048, 4096, 32, 8, 128, 128, "bf16",
                               ((3, 3, 3),), "bwd_kl", "rms_outlier"),
    # The same fine-tuning run with the paper's default objective, mse + 0.1 KL / B.
    "mistral_ft_kl": Workload("mistral_ft_kl", 16, 2048, 4096, 32, 8, 128, 128, "bf16",
                              ((3, 3, 3),), "ft", "rms_outlier", probes=200, lambda_kl=0.1),
    # Fisher-coupling scores at the shape of the STE step, at the 2-bit round-to-nearest probe.
    "mistral_fisher": Workload("mistral_fisher", 16, 2048, 4096, 32, 8, 128, 128, "bf16",
                               ((2, 2, 2),), "fisher", "rms_outlier"),
    # The quantizer alone over the W_Q, W_K, W_V of all 32 Mistral-7B layers at once: the layers'
    # rows stacked (every W_Q, then every W_K, then every W_V) as one problem of 32 x 32 query and
    # 32 x 8 key/value heads, 196608 x 4096 weights; codes, fp32 fake-quantized weights and the
    # eps^W sums at 3 bits.  The activations are not used.
    "mistral_quant32": Workload("mistral_quant32", 1, 32, 4096, 1024, 256, 128, 128, "bf16",
                                ((3, 3, 3),), "quant", "rms_outlier"),
    # STE fine-tuning step at the Mistral shape: 16 x 2048, 3-bit, fwd + bwd.
    "mistral_ste": Workload("mistral_ste", 16, 2048, 4096, 32, 8, 128, 128, "bf16",
                            ((3, 3, 3),), "bwd", "rms_outlier"),
}


def _seq_rng(seed: int, stream: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, index])))


def outlier_channels(wl: Workload) -> np.ndarray:
    """Indices of the channels scaled by ``outlier_scale``."""
    perm = _seq_rng(wl.seed, 3, 0).permutation(wl.d_model)
    return np.sort(perm[: wl.n_outliers])


def _draw_sequence(wl: Workload, b: int, chans: np.ndarray) -> np.ndarray:
    z = _seq_rng(wl.seed, 1, b).standard_normal((wl.seq_len, wl.d_model), dtype=np.float32)
    if wl.x_recipe == "rms_outlier":
        rms = np.sqrt(np.mean(z.astype(np.float64) ** 2, axis=1, keepdims=True))
        z = (z / rms).astype(np.float32)
    elif wl.x_recipe != "gauss_outlier":
        raise ValueError(f"unknown x recipe {wl.x_recipe!r}")
    z[:, chans] *= np.float32(wl.outlier_scale)
    return z


def make_x(wl: Workload, seqs: Optional[Sequence[int]] = None, threads: int = 8) -> torch.Tensor:
    """Calibration activations X[len(seqs)][seq_len][d_model] on the CPU, in the storage dtype."""
    if seqs is None:
        seqs = range(wl.batch)
    seqs = list(seqs)
    chans = outlier_channels(wl)
    out = torch.empty((len(seqs), wl.seq_len, wl.d_model), dtype=wl.torch_dtype)

    def fill(i: int) -> None:
        out[i].copy_(torch.from_numpy(_draw_sequence(wl, seqs[i], chans)))

    if len(seqs) > 1 and threads > 1:
        with ThreadPoolExecutor(min(threads, len(seqs))) as ex:
            list(ex.map(fill, range(len(seqs))))
    else:
        for i in range(len(seqs)):
            fill(i)
    return out


def make_w(wl: Workload) -> torch.Tensor:
    """Fused weight [R][d_model] = rows of W_Q, then W_K, then W_V, in the storage dtype."""
    d = wl.d_model
    parts = []
    for m, nrows in enumerate((wl.n_heads * wl.head_dim, wl.n_kv_heads * wl.head_dim,
                               wl.n_kv_heads * wl.head_dim)):
        w = _seq_rng(wl.seed, 2, m).standard_normal((nrows, d), dtype=np.float32)
        parts.append(torch.from_numpy(w * np.float32(wl.w_std)))
    return torch.cat(parts, 0).to(wl.torch_dtype)


def make_probes(wl: Workload, n: int, seed: int = 0) -> torch.Tensor:
    """n Rademacher probes over the fused weight, int8 [n][R][d_model] in {-1, +1} (CPU), probe i
    drawn from its own seeded stream."""
    out = torch.empty((n, wl.rows, wl.d_model), dtype=torch.int8)
    for i in range(n):
        bits = _seq_rng(wl.seed + 1000 * seed, 4, i).integers(0, 2, (wl.rows, wl.d_model), dtype=np.int8)
        out[i].copy_(torch.from_numpy(bits * np.int8(2) - np.int8(1)))
    return out


def matrix_rows(wl: Workload) -> tuple:
    """(start, stop) row ranges of W_Q, W_K, W_V inside the fused weight."""
    q = wl.n_heads * wl.head_dim
    kv = wl.n_kv_heads * wl.head_dim
    return ((0, q), (q, q + kv), (q + kv, q + 2 * kv))


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact widening of a storage-dtype tensor to a float64 numpy array."""
    return t.detach().to("cpu").to(torch.float64).numpy()
