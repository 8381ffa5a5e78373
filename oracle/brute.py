"""Brute-force numpy implementation for tiny inputs (second, independent oracle).

TEST INFRASTRUCTURE ONLY.  Shares nothing with ``jab_oracle.c`` except the
definitions in the paper:

* codes: exhaustive search of the grid for the nearest point (eq. quant), ties
  to the even integer offset, instead of a division and a rounding;
* attention: the full T x T score matrix with an explicit -inf causal mask M,
  softmax over each row, then P V (Method, A(X) = softmax(QK^T/sqrt(d_head)+M)V);
* the loss: || A - A_hat ||_F^2 over the whole batch at once (eq. joint_loss).
"""
from __future__ import annotations

import numpy as np


def nearest_codes(w: np.ndarray, s: np.ndarray, z: np.ndarray, bits: int, group: int) -> np.ndarray:
    """Asymmetric grid: argmin_c |w - (c - z) s| over c in 0..2^b-1; on an exact tie pick the
    code whose offset c - z is even (round-half-to-even of w/s)."""
    rows, cols = w.shape
    se = np.repeat(s, group, axis=1)
    ze = np.repeat(z, group, axis=1).astype(np.int64)
    best = np.zeros((rows, cols), np.int64)
    best_d = np.full((rows, cols), np.inf)
    for c in range(1 << bits):
        off = c - ze
        dist = np.abs(w - off * se)
        better = dist < best_d
        tie = (dist == best_d) & (off % 2 == 0)
        take = better | tie
        best = np.where(take, c, best)
        best_d = np.where(take, dist, best_d)
    return best


def nearest_codes_sym(w: np.ndarray, s: np.ndarray, bits: int, group: int) -> np.ndarray:
    """Symmetric grid q in -q_max..q_max, returned as q + q_max."""
    qmax = (1 << (bits - 1)) - 1
    se = np.repeat(s, group, axis=1)
    best = np.zeros(w.shape, np.int64)
    best_d = np.full(w.shape, np.inf)
    for q in range(-qmax, qmax + 1):
        dist = np.abs(w - q * se)
        take = (dist < best_d) | ((dist == best_d) & (q % 2 == 0))
        best = np.where(take, q, best)
        best_d = np.where(take, dist, best_d)
    return best + qmax


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int, n_kv_heads: int):
    """q [T][Hq][dh], k/v [T][Hkv][dh] -> A [T][Hq*dh], P [Hq][T][T]."""
    T, _, dh = q.shape
    rep = n_heads // n_kv_heads
    kk = np.repeat(k, rep, axis=1)          # GQA: head h uses kv head h // rep
    vv = np.repeat(v, rep, axis=1)
    S = np.einsum("ihc,jhc->hij", q, kk) / np.sqrt(dh)
    M = np.triu(np.full((T, T), -np.inf), k=1)
    S = S + M[None]
    S = S - S.max(axis=2, keepdims=True)
    P = np.exp(S)
    P = P / P.sum(axis=2, keepdims=True)
    A = np.einsum("hij,jhc->ihc", P, vv)
    return A.reshape(T, n_heads * dh), P


def block_output(x: np.ndarray, w: np.ndarray, n_heads: int, n_kv_heads: int, head_dim: int):
    """x [B][T][d], fused w [R][d] -> A [B][T][Hq*dh]."""
    y = x @ w.T
    hq, hk = n_heads * head_dim, n_kv_heads * head_dim
    out = []
    for b in range(x.shape[0]):
        T = x.shape[1]
        q = y[b, :, :hq].reshape(T, n_heads, head_dim)
        k = y[b, :, hq:hq + hk].reshape(T, n_kv_heads, head_dim)
        v = y[b, :, hq + hk:].reshape(T, n_kv_heads, head_dim)
        out.append(attention(q, k, v, n_heads, n_kv_heads)[0])
    return np.stack(out)


def sse(x, w, w_hat, n_heads, n_kv_heads, head_dim) -> float:
    a = block_output(x, w, n_heads, n_kv_heads, head_dim)
    ah = block_output(x, w_hat, n_heads, n_kv_heads, head_dim)
    return float(np.sum((a - ah) ** 2))
