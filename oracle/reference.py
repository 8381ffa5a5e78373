"""Composition of the fp64 oracle routines into the JAB loss, sweep and gradients.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The loss is the mean-squared-error term of the joint attention-block loss
(Method, eq. joint_loss, with lambda_KL = 0, the paper's "no KL" arm):

    L(w) = || A(X) - A_hat(X; w) ||_F^2,   reported both as the sum (sse) and as
    mse = sse / (B * T * n_heads * head_dim)   (the element-wise mean of the
    Appendix on the effective weight of the KL term),

where A is the causal attention output of the block with its float weights and
A_hat the same computation with W_Q, W_K, W_V fake-quantized (eq. quant) --
teacher and student see the same X (Appendix "Joint STE fine-tuning", (3)).
The backward follows eq. lsq: straight-through on the weights (dW = dW_hat) and
the LSQ factor on the per-(row, group) scales.

Two precision modes:
* ``fmt=None`` ("exact"): every quantity in float64, w_hat = (q - z) s exactly.
* ``fmt in {"f32","f16","bf16"}`` ("contract"): the roundings that belong to a
  computation in that storage dtype: w_hat = RN_dtype(RN_fp32((q - z) s)), and
  the projections Q, K, V are rounded to the dtype before attention.  Everything
  else (sums, softmax, attention, loss) stays in float64.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

from . import build as _build

FMT = {None: 0, "none": 0, "f32": 1, "f16": 2, "bf16": 3}
ASYM, SYM = 0, 1

_LIB = None
_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.POINTER(ctypes.c_int32)


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        path = _build.build(force=False)
        L = ctypes.CDLL(path)
        ci, c64, cd = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.orc_round.argtypes = [_D, c64, ci]
        L.orc_quant_params.argtypes = [_D, ci, ci, ci, ci, ci, _D, _I]
        L.orc_fake_quant.argtypes = [_D, ci, ci, ci, ci, ci, _D, _I, _I, _D, _D]
        L.orc_project.argtypes = [_D, ci, ci, _D, ci, _D]
        L.orc_attention.argtypes = [_D, ci, ci, ci, ci, ci, _D, _D, _D]
        L.orc_attention_bwd.argtypes = [_D, ci, ci, ci, ci, ci, _D, _D]
        L.orc_attention_kl.argtypes = [_D, _D, ci, ci, ci, ci, ci, _D, _D]
        L.orc_attention_jvp.argtypes = [_D, _D, ci, ci, ci, ci, ci, _D]
        L.orc_weight_grad.argtypes = [_D, _D, ci, ci, ci, _D]
        L.orc_scale_grad.argtypes = [_D, _D, ci, ci, ci, cd, _D]
        for f in ("orc_round", "orc_quant_params", "orc_fake_quant", "orc_project", "orc_attention",
                  "orc_attention_bwd", "orc_attention_kl", "orc_attention_jvp", "orc_weight_grad",
                  "orc_scale_grad"):
            getattr(L, f).restype = ci
        _LIB = L
    return _LIB


def _dp(a: np.ndarray):
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(_D)


def _ip(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.int32 and a.flags.c_contiguous
    return a.ctypes.data_as(_I)


def _c64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ok(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


# --------------------------------------------------------------------------- steps
def round_fmt(x, fmt) -> np.ndarray:
    """Round to the storage format ``fmt`` (ties to even); fmt None leaves float64."""
    y = _c64(x).copy()
    _ok(lib().orc_round(_dp(y), y.size, FMT[fmt]), "round")
    return y


def quant_params(w, group: int, bits: int, scheme: int = ASYM) -> Tuple[np.ndarray, np.ndarray]:
    """Per-(row, group) scale and zero-point of eq. quant (min-max init, 0 in range)."""
    w = _c64(w)
    rows, cols = w.shape
    s = np.zeros((rows, cols // group), np.float64)
    z = np.zeros((rows, cols // group), np.int32)
    _ok(lib().orc_quant_params(_dp(w), rows, cols, group, bits, scheme, _dp(s), _ip(z)), "quant_params")
    return s, z


def fake_quant(w, group: int, bits: int, s, z, scheme: int = ASYM):
    """Codes, fake-quantized weights w_hat and the LSQ factor phi (eq. quant, eq. lsq)."""
    w = _c64(w)
    rows, cols = w.shape
    codes = np.zeros((rows, cols), np.int32)
    w_hat = np.zeros((rows, cols), np.float64)
    phi = np.zeros((rows, cols), np.float64)
    s = _c64(s)
    z = None if z is None else np.ascontiguousarray(z, dtype=np.int32)
    _ok(lib().orc_fake_quant(_dp(w), rows, cols, group, bits, scheme, _dp(s), _ip(z), _ip(codes),
                             _dp(w_hat), _dp(phi)), "fake_quant")
    return codes, w_hat, phi


def project(x_seq, w) -> np.ndarray:
    """y = x W^T for one sequence: x [T][d], W [R][d] -> y [T][R] (Method, Layer-wise PTQ)."""
    x_seq, w = _c64(x_seq), _c64(w)
    T, d = x_seq.shape
    R = w.shape[0]
    y = np.zeros((T, R), np.float64)
    _ok(lib().orc_project(_dp(x_seq), T, d, _dp(w), R, _dp(y)), "project")
    return y


def attention(y, n_heads: int, n_kv_heads: int, head_dim: int):
    """Causal GQA softmax attention of one sequence -> (A [T][Hq*dh], lse [Hq][T], max|rowsum(P)-1|)."""
    y = _c64(y)
    T, R = y.shape
    a = np.zeros((T, n_heads * head_dim), np.float64)
    lse = np.zeros((n_heads, T), np.float64)
    dev = np.zeros(1, np.float64)
    _ok(lib().orc_attention(_dp(y), T, R, n_heads, n_kv_heads, head_dim, _dp(a), _dp(lse), _dp(dev)),
        "attention")
    return a, lse, float(dev[0])


def attention_kl(yt, ys, n_heads: int, n_kv_heads: int, head_dim: int):
    """D_KL(P || Q) of one sequence's causal attention maps (eq. joint_loss): P from the teacher
    projection ``yt``, Q from the student projection ``ys`` -> (kl [Hq][T] per query row, sum)."""
    yt, ys = _c64(yt), _c64(ys)
    T, R = yt.shape
    assert ys.shape == yt.shape
    kl = np.zeros((n_heads, T), np.float64)
    tot = np.zeros(1, np.float64)
    _ok(lib().orc_attention_kl(_dp(yt), _dp(ys), T, R, n_heads, n_kv_heads, head_dim, _dp(kl), _dp(tot)),
        "attention_kl")
    return kl, float(tot[0])


def attention_jvp(y, yd, n_heads: int, n_kv_heads: int, head_dim: int) -> np.ndarray:
    """Directional derivatives of one sequence's causal attention at the projection y along the
    tangent yd (eq. gn's J_A v and J_Q v, split by the unit the tangent moves) -> the nine sums
    [<aQ,aQ>, <aK,aK>, <aV,aV>, <aQ,aK>, <aQ,aV>, <aK,aV>, zQ.I(P).zQ, zK.I(P).zK, zQ.I(P).zK]
    over heads and query rows (see orc_attention_jvp)."""
    y, yd = _c64(y), _c64(yd)
    T, R = y.shape
    assert yd.shape == y.shape
    out = np.zeros(9, np.float64)
    _ok(lib().orc_attention_jvp(_dp(y), _dp(yd), T, R, n_heads, n_kv_heads, head_dim, _dp(out)), "attention_jvp")
    return out


def attention_bwd(y, n_heads: int, n_kv_heads: int, head_dim: int, g) -> np.ndarray:
    """dLoss/d[Q|K|V] of one sequence given g = dLoss/dA."""
    y, g = _c64(y), _c64(g)
    T, R = y.shape
    dy = np.zeros((T, R), np.float64)
    _ok(lib().orc_attention_bwd(_dp(y), T, R, n_heads, n_kv_heads, head_dim, _dp(g), _dp(dy)),
        "attention_bwd")
    return dy


def weight_grad_acc(dy, x_seq, dw_hat: np.ndarray) -> None:
    """dw_hat += dY^T X for one sequence."""
    dy, x_seq = _c64(dy), _c64(x_seq)
    T, R = dy.shape
    d = x_seq.shape[1]
    _ok(lib().orc_weight_grad(_dp(dy), _dp(x_seq), T, d, R, _dp(dw_hat)), "weight_grad")


def scale_grad(dw_hat, phi, group: int, gamma: float) -> np.ndarray:
    dw_hat, phi = _c64(dw_hat), _c64(phi)
    rows, cols = dw_hat.shape
    ds = np.zeros((rows, cols // group), np.float64)
    _ok(lib().orc_scale_grad(_dp(dw_hat), _dp(phi), rows, cols, group, float(gamma), _dp(ds)), "scale_grad")
    return ds


# --------------------------------------------------------------------------- problem
@dataclass(frozen=True)
class Problem:
    batch: int
    seq_len: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    group_size: int
    scheme: int = ASYM
    rope_theta: float = 0.0         # RoPE base on Q and K; 0: no rotary embedding

    @property
    def rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def matrix_rows(self):
        q = self.n_heads * self.head_dim
        kv = self.n_kv_heads * self.head_dim
        return ((0, q), (q, q + kv), (q + kv, q + 2 * kv))

    @property
    def n_out(self) -> int:
        """Elements of the merged attention output per token."""
        return self.n_heads * self.head_dim


def default_gamma(bits: int, group: int, scheme: int = ASYM) -> float:
    """LSQ gradient factor (n_w q_max)^(-1/2) of eq. lsq, with n_w = the weights that
    share one scale (a group) and q_max = the largest code magnitude of the grid
    (2^b - 1 steps for the asymmetric grid, 2^(b-1) - 1 for the symmetric one)."""
    if bits == 0:
        return 0.0
    qmax = (1 << bits) - 1 if scheme == ASYM else (1 << (bits - 1)) - 1
    return float((group * qmax) ** -0.5)


def init_scales(w, prob: Problem, bits3) -> Tuple[np.ndarray, Optional[np.ndarray]]:
    """Min-max scales (and zero-points) of the fused weight, each matrix at its own bit-width."""
    w = _c64(w)
    ng = prob.d_model // prob.group_size
    s = np.ones((prob.rows, ng), np.float64)
    z = np.zeros((prob.rows, ng), np.int32)
    for (r0, r1), b in zip(prob.matrix_rows(), bits3):
        if b:
            sm, zm = quant_params(w[r0:r1], prob.group_size, b, prob.scheme)
            s[r0:r1], z[r0:r1] = sm, zm
    return s, (z if prob.scheme == ASYM else None)


def student_weight(w, prob: Problem, bits3, s, z, fmt) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Fake-quantized fused weight as the student uses it -> (w_eff, codes, phi).

    Contract mode rounds w_hat = (q - z) s to fp32 and then to the storage dtype;
    a matrix with b = 0 keeps its float weights."""
    w = _c64(w)
    w_eff = w.copy()
    codes = np.zeros(w.shape, np.int32)
    phi = np.zeros(w.shape, np.float64)
    for (r0, r1), b in zip(prob.matrix_rows(), bits3):
        if not b:
            continue
        zm = None if z is None else z[r0:r1]
        c, wh, ph = fake_quant(w[r0:r1], prob.group_size, b, s[r0:r1], zm, prob.scheme)
        if fmt is not None:
            wh = round_fmt(round_fmt(wh, "f32"), fmt)
        w_eff[r0:r1], codes[r0:r1], phi[r0:r1] = wh, c, ph
    return w_eff, codes, phi


def rope_angles(seq_len: int, head_dim: int, theta: float) -> Tuple[np.ndarray, np.ndarray]:
    """Rotary position embedding (the RoPE Mistral applies to queries and keys): at position t the
    pair j < head_dim/2 turns by the angle t * theta^(-2j / head_dim).  -> (cos, sin) [T][head_dim/2]"""
    j = np.arange(head_dim // 2, dtype=np.float64)
    inv = np.power(float(theta), -2.0 * j / head_dim)
    ang = np.arange(seq_len, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope_qk(y, prob: Problem, inverse: bool = False) -> np.ndarray:
    """Rotate the query and key columns of one sequence's projection y [T][R] in fp64 (the value
    columns pass through).  Each head pairs its element j with element j + head_dim/2 (the
    half-split layout of the Hugging Face Mistral checkpoints):
        (a, b) -> (a cos - b sin, b cos + a sin)
    ``inverse`` turns the other way (the transpose, for the gradient)."""
    if not prob.rope_theta:
        return y
    T, dh = y.shape[0], prob.head_dim
    c, s = rope_angles(T, dh, prob.rope_theta)
    if inverse:
        s = -s
    out = np.array(y, dtype=np.float64, copy=True)
    nqk = (prob.n_heads + prob.n_kv_heads) * dh
    h = out[:, :nqk].reshape(T, -1, dh)
    a, b = h[..., :dh // 2].copy(), h[..., dh // 2:].copy()
    h[..., :dh // 2] = a * c[:, None, :] - b * s[:, None, :]
    h[..., dh // 2:] = b * c[:, None, :] + a * s[:, None, :]
    out[:, :nqk] = h.reshape(T, nqk)
    return out


def qkv_operands(y, prob: Problem, fmt) -> np.ndarray:
    """What the attention consumes from one sequence's projection y (exact): Q and K rotated when
    the problem has RoPE, then everything rounded once to the storage dtype in contract mode (the
    rotation acts on the projection as accumulated, before its rounding)."""
    y = rope_qk(y, prob)
    return y if fmt is None else round_fmt(y, fmt)


def block_forward(x_seq, w_eff, prob: Problem, fmt):
    """Projection (Q and K rotated when the problem has RoPE) then causal attention for one
    sequence -> (y, A, lse, rowsum deviation); y is what the attention consumes."""
    y = qkv_operands(project(x_seq, w_eff), prob, fmt)
    a, lse, dev = attention(y, prob.n_heads, prob.n_kv_heads, prob.head_dim)
    return y, a, lse, dev


def attn_ref(x, w, prob: Problem, fmt, seqs: Optional[Iterable[int]] = None) -> Dict[int, np.ndarray]:
    """Teacher output A(X) with the float weights, per sequence."""
    seqs = range(len(x)) if seqs is None else seqs
    return {b: block_forward(x[b], w, prob, fmt)[1] for b in seqs}


def loss_fwd(x, w, prob: Problem, bits3, s, z, fmt, a_ref: Optional[Dict[int, np.ndarray]] = None,
             seqs: Optional[Iterable[int]] = None) -> dict:
    """Squared-error JAB loss.  ``x`` holds the sequences listed in ``seqs`` (default: all of
    the batch).  Returns sse / mse / sum A^2 over those sequences and sse per sequence; mse
    divides by the full-batch element count B*T*Hq*dh."""
    seqs = list(range(len(x))) if seqs is None else list(seqs)
    w_eff, _, _ = student_weight(w, prob, bits3, s, z, fmt)
    sse_seq, suma2 = {}, 0.0
    for i, b in enumerate(seqs):
        a = a_ref[b] if a_ref is not None else block_forward(x[i], w, prob, fmt)[1]
        ahat = block_forward(x[i], w_eff, prob, fmt)[1]
        sse_seq[b] = float(np.sum((a - ahat) ** 2))
        suma2 += float(np.sum(a ** 2))
    sse = float(sum(sse_seq.values()))
    n = prob.batch * prob.seq_len * prob.n_out
    return {"sse": sse, "mse": sse / n, "sum_a2": suma2, "sse_seq": sse_seq}


def loss_kl(x, w, prob: Problem, bits3, s, z, fmt, seqs: Optional[Iterable[int]] = None) -> dict:
    """KL attention-map term of eq. joint_loss, D_KL(P || Q(w)), with the reduction of the
    Appendix on the effective weight of the KL term (``batchmean``: summed over heads, queries
    and keys of every sequence, divided by B only).  ``x`` holds the sequences in ``seqs``
    (default: all); kl_batchmean divides the sum over them by the full batch size B.  Both maps
    come from projections rounded to the storage dtype in contract mode."""
    seqs = list(range(len(x))) if seqs is None else list(seqs)
    w_eff, _, _ = student_weight(w, prob, bits3, s, z, fmt)
    kl_seq = {}
    for i, b in enumerate(seqs):
        yt = qkv_operands(project(x[i], w), prob, fmt)
        ys = qkv_operands(project(x[i], w_eff), prob, fmt)
        kl_seq[b] = attention_kl(yt, ys, prob.n_heads, prob.n_kv_heads, prob.head_dim)[1]
    kl = float(sum(kl_seq.values()))
    return {"kl": kl, "kl_batchmean": kl / prob.batch, "kl_seq": kl_seq}


CURVATURE_FORMS = ("t_Q", "t_K", "t_V", "pooled", "h_QQ", "h_KK", "h_VV")


def curvature_parts(x, w, prob: Problem, probes, fmt, seqs: Optional[Iterable[int]] = None) -> np.ndarray:
    """The nine tangent sums of attention_jvp per probe, over the sequences: [n_probes][9].  The
    tangent of the projection along probe v is X v^T (a probe over the fused weight's rows: its
    W_Q rows move Q, its W_K rows K, its W_V rows V); with RoPE it turns with Q and K.  Contract
    mode rounds the projection and its tangent to the storage dtype, as the device forms them."""
    seqs = list(range(len(x))) if seqs is None else list(seqs)
    w = _c64(w)
    probes = np.asarray(probes, dtype=np.float64)
    out = np.zeros((len(probes), 9))
    for i, b in enumerate(seqs):
        y = block_forward(x[i], w, prob, fmt)[0]
        for p in range(len(probes)):
            yd = qkv_operands(project(x[i], probes[p]), prob, fmt)
            out[p] += attention_jvp(y, yd, prob.n_heads, prob.n_kv_heads, prob.head_dim)
    return out


def curvature_forms(parts, lambda_kl: float) -> np.ndarray:
    """Quadratic forms of eq. gn's Hessian H = 2 J_A^T J_A + lambda_KL J_Q^T I(P) J_Q from the tangent
    sums -> [n][7]:
      t_u     = v_u^T (H v)_u for u = Q, K, V: the paper's per-unit partition of v^T H v over the
                unit's coordinates (Appendix on per-unit traces; unbiased for Tr(H_uu)),
      pooled  = v^T H v = t_Q + t_K + t_V (the pooled Hutchinson term),
      h_uu    = v_u^T H_uu v_u: the diagonal block alone (the probe restricted to unit u).
    With J_A v = aQ + aK + aV and J_Q v = zQ + zK (W_V does not move the map):
      t_Q = 2 <aQ, aQ + aK + aV> + lambda (zQ.I.zQ + zQ.I.zK), t_K alike, t_V = 2 <aV, aQ + aK + aV>."""
    e = np.asarray(parts, dtype=np.float64)
    lam = float(lambda_kl)
    qq, kk, vv, qk, qv, kv, fqq, fkk, fqk = (e[:, i] for i in range(9))
    tq = 2.0 * (qq + qk + qv) + lam * (fqq + fqk)
    tk = 2.0 * (qk + kk + kv) + lam * (fqk + fkk)
    tv = 2.0 * (qv + kv + vv)
    return np.stack([tq, tk, tv, tq + tk + tv, 2.0 * qq + lam * fqq, 2.0 * kk + lam * fkk, 2.0 * vv], axis=1)


def curvature_gn(x, w, prob: Problem, probes, fmt, lambda_kl: float = 0.0,
                 seqs: Optional[Iterable[int]] = None) -> np.ndarray:
    """Hutchinson terms of the curvature of eq. gn at the float point, per probe: [n][7] in the order
    of CURVATURE_FORMS.  The loss is eq. joint_loss as printed, ||A - A_hat||_F^2 + lambda_KL
    D_KL(P || Q(w)) with the KL summed over every query row; it is 0 at the float point, so its
    Hessian there is exactly H = 2 J_A^T J_A + lambda_KL J_Q^T I(P) J_Q (the residual terms multiply
    A - A_hat = 0 and the KL's gradient, 0 at Q = P).  The objective as implemented, mse + lambda
    kl / B, has the Hessian (1/N) H with lambda_KL = lambda N / B (N = B T Hq d_head)."""
    return curvature_forms(curvature_parts(x, w, prob, probes, fmt, seqs), lambda_kl)


TRACE_BLOCK, TRACE_UNIT = 0, 1
OMEGA_C1, OMEGA_C2 = 0, 1


def omega_table(curv, werr, trace: int = TRACE_BLOCK, criterion: int = OMEGA_C1) -> np.ndarray:
    """The allocator's sensitivity table of eq. omega for L attention blocks -> [3 L][n_widths].
    Row 3 l + m is matrix m (W_Q, W_K, W_V) of block l (depth order, l from 0).
      C1: Omega_i(b) = Tr(H_i) ||Q_b(W_i) - W_i||_F^2
      C2: Omega_i(b) = (L - l) Omega_i(b), the layers an error of block l passes through, its own
          included (the paper's i as a 0-based depth: the last block keeps weight 1).
    Tr(H_i) is Hutchinson's estimate, the mean over the block's probes (Section "Sensitivity and
    allocation"): of the pooled v^T H v for one trace per block, shared by its three matrices, or of
    the matrix's own partition term t_u (Appendix on per-unit traces).
    curv [L][n_probes][7] in the order of CURVATURE_FORMS; werr [L][n_widths][3][2], entry
    [l][k][m][0] the squared Frobenius error of matrix m of block l at width k."""
    curv = np.asarray(curv, dtype=np.float64)
    werr = np.asarray(werr, dtype=np.float64)
    n_layers, n_widths = curv.shape[0], werr.shape[1]
    out = np.zeros((3 * n_layers, n_widths))
    for layer in range(n_layers):
        for m in range(3):
            col = CURVATURE_FORMS.index("pooled") if trace == TRACE_BLOCK else m
            tr = sum(float(t) for t in curv[layer, :, col]) / curv.shape[1]
            weight = float(n_layers - layer) if criterion == OMEGA_C2 else 1.0
            for k in range(n_widths):
                out[3 * layer + m, k] = weight * (tr * werr[layer, k, m, 0])
    return out


def curvature_fd(x, w, prob: Problem, probes, eps: float, fmt, seqs: Optional[Iterable[int]] = None,
                 lambda_kl: float = 0.0) -> np.ndarray:
    """Finite-difference check of eq. gn at the float point: per (probe, unit) the symmetric
    difference of the joint loss,

        (L(w + eps v) + L(w - eps v)) / eps^2 = v^T H v + O(eps^2),
        L(w') = ||A(X; w) - A(X; w')||_F^2 + lambda_KL sum over rows of D_KL(P(w) || Q(w')),

    built only from the pinned forward routines.  Unit u = 0, 1, 2 restricts the probe to the rows
    of W_Q, W_K, W_V (the diagonal block h_uu of curvature_gn); u = 3 uses the whole probe (the
    pooled form).  In contract mode the perturbed weights are rounded as RN_dtype(RN_fp32(w +- eps v)).
    probes [n][R][d] in {-1, +1} -> [n][4]."""
    seqs = list(range(len(x))) if seqs is None else list(seqs)
    w = _c64(w)
    probes = np.asarray(probes, dtype=np.float64)
    teacher = {b: block_forward(x[i], w, prob, fmt) for i, b in enumerate(seqs)}
    units = list(prob.matrix_rows()) + [(0, prob.rows)]
    out = np.zeros((len(probes), 4))
    for p in range(len(probes)):
        for u, (r0, r1) in enumerate(units):
            tot = 0.0
            for sign in (1.0, -1.0):
                w2 = w.copy()
                w2[r0:r1] = w[r0:r1] + sign * eps * probes[p][r0:r1]
                if fmt is not None:
                    w2[r0:r1] = round_fmt(round_fmt(w2[r0:r1], "f32"), fmt)
                for i, b in enumerate(seqs):
                    y2, a2 = block_forward(x[i], w2, prob, fmt)[:2]
                    tot += float(np.sum((teacher[b][1] - a2) ** 2))
                    if lambda_kl:
                        tot += lambda_kl * attention_kl(teacher[b][0], y2, prob.n_heads, prob.n_kv_heads,
                                                        prob.head_dim)[1]
            out[p, u] = tot / (eps * eps)
    return out


def sweep(x, w, prob: Problem, triples: Sequence[Tuple[int, int, int]], scales_by_bits: dict, fmt,
          seqs: Optional[Iterable[int]] = None) -> dict:
    """Loss for every (b_Q, b_K, b_V) triple.  ``scales_by_bits[b] = (s, z)`` holds the fused
    weight's scales at bit-width b.  Each matrix's projection at each bit-width is computed
    once and reused by every triple that contains it (columns of y are independent)."""
    seqs = list(range(len(x))) if seqs is None else list(seqs)
    bits_used = sorted({b for t in triples for b in t})
    w = _c64(w)
    w_eff_b = {}
    for b in bits_used:
        s, z = scales_by_bits[b]
        w_eff_b[b] = student_weight(w, prob, (b, b, b), s, z, fmt)[0]
    (q0, q1), (k0, k1), (v0, v1) = prob.matrix_rows()
    out = {t: {"sse_seq": {}} for t in triples}
    for i, b in enumerate(seqs):
        a = block_forward(x[i], w, prob, fmt)[1]
        ys = {bb: qkv_operands(project(x[i], w_eff_b[bb]), prob, fmt) for bb in bits_used}
        for t in triples:
            y = np.concatenate([ys[t[0]][:, q0:q1], ys[t[1]][:, k0:k1], ys[t[2]][:, v0:v1]], axis=1)
            ahat = attention(y, prob.n_heads, prob.n_kv_heads, prob.head_dim)[0]
            out[t]["sse_seq"][b] = float(np.sum((a - ahat) ** 2))
    n = prob.batch * prob.seq_len * prob.n_out
    for t in triples:
        out[t]["sse"] = float(sum(out[t]["sse_seq"].values()))
        out[t]["mse"] = out[t]["sse"] / n
    return out


def attention_kl_grad(yt, ys, n_heads: int, n_kv_heads: int, head_dim: int, coef: float) -> np.ndarray:
    """Gradient of coef * sum over heads and query rows of D_KL(P_i || Q_i) with respect to the
    student's projection ys (its query and key columns; the value columns get 0).  P and Q are
    the causal softmax maps of the teacher's yt and the student's ys.  With z_ij = q_i . k_j /
    sqrt(d_head) and sum_j P_ij = 1, d KL_i / d z_ij = Q_ij - P_ij, so
        dq_i = coef / sqrt(d_head) sum_j (Q_ij - P_ij) k_j,
        dk_j = coef / sqrt(d_head) sum_i (Q_ij - P_ij) q_i   (summed over a key head's query heads)."""
    T = ys.shape[0]
    dh = head_dim
    mask = np.tril(np.ones((T, T), dtype=bool))
    d = np.zeros_like(np.asarray(ys, dtype=np.float64))
    k0 = n_heads * dh

    def smax(q, k):
        sc = (q @ k.T) / math.sqrt(dh)
        sc = np.where(mask, sc, -np.inf)
        sc = sc - sc.max(axis=1, keepdims=True)
        e = np.exp(sc)
        return e / e.sum(axis=1, keepdims=True)

    for h in range(n_heads):
        g = h * n_kv_heads // n_heads
        qs, ks = ys[:, h * dh:(h + 1) * dh], ys[:, k0 + g * dh:k0 + (g + 1) * dh]
        qt, kt = yt[:, h * dh:(h + 1) * dh], yt[:, k0 + g * dh:k0 + (g + 1) * dh]
        ds = coef / math.sqrt(dh) * (smax(qs, ks) - smax(qt, kt))
        d[:, h * dh:(h + 1) * dh] += ds @ ks
        d[:, k0 + g * dh:k0 + (g + 1) * dh] += ds.T @ qs
    return d


def loss_bwd(x, w, prob: Problem, bits3, s, z, fmt, gammas=None,
             a_ref: Optional[Dict[int, np.ndarray]] = None, lambda_kl: float = 0.0, w_teacher=None) -> dict:
    """mse loss and its gradients over the whole batch ``x`` [B][T][d]:
    dW = dW_hat (straight-through, no case split) and ds[r][j] = gamma_m sum_{k in j} dW_hat phi
    (eq. lsq).  ``gammas`` per matrix; default :func:`default_gamma`.  The teacher is the block
    with the float weights ``w`` unless ``a_ref`` (per sequence) is given, as in fine-tuning,
    where the float teacher stays fixed while the latent weights move.  ``lambda_kl`` > 0 adds
    the KL attention-map term of eq. joint_loss to the objective, mse + lambda_kl * kl / B
    (batchmean), its gradient from :func:`attention_kl_grad` against the float block's map (the
    block with ``w_teacher``, default ``w``)."""
    assert len(x) == prob.batch
    if gammas is None:
        gammas = [default_gamma(b, prob.group_size, prob.scheme) for b in bits3]
    w = _c64(w)
    w_eff, codes, phi = student_weight(w, prob, bits3, s, z, fmt)
    n = prob.batch * prob.seq_len * prob.n_out
    dw_hat = np.zeros(w.shape, np.float64)
    sse_seq, suma2 = {}, 0.0
    for b in range(prob.batch):
        a = a_ref[b] if a_ref is not None else block_forward(x[b], w, prob, fmt)[1]
        y, ahat, _, _ = block_forward(x[b], w_eff, prob, fmt)
        sse_seq[b] = float(np.sum((a - ahat) ** 2))
        suma2 += float(np.sum(a ** 2))
        g = 2.0 * (ahat - a) / n
        dy = attention_bwd(y, prob.n_heads, prob.n_kv_heads, prob.head_dim, g)
        if lambda_kl:
            yt = block_forward(x[b], w if w_teacher is None else w_teacher, prob, fmt)[0]
            dy = dy + attention_kl_grad(yt, y, prob.n_heads, prob.n_kv_heads, prob.head_dim, lambda_kl / prob.batch)
        dy = rope_qk(dy, prob, inverse=True)     # through the rotation: its transpose
        weight_grad_acc(dy, x[b], dw_hat)
    ds = np.zeros(s.shape, np.float64)
    for (r0, r1), b, gm in zip(prob.matrix_rows(), bits3, gammas):
        if b:
            ds[r0:r1] = scale_grad(dw_hat[r0:r1], phi[r0:r1], prob.group_size, gm)
    sse = float(sum(sse_seq.values()))
    return {"sse": sse, "mse": sse / n, "sum_a2": suma2, "sse_seq": sse_seq, "dw": dw_hat, "ds": ds,
            "codes": codes, "w_eff": w_eff}


def fisher(x, w, prob: Problem, bits3, s, z, fmt, lambda_kl: float = 0.0) -> dict:
    """Fisher-coupling scores (Appendix on Fisher-coupling): the squared norm of the loss
    gradient per unit, taken off the float point at a coarse round-to-nearest probe (the paper's
    is 2-bit; ``bits3`` and the scales ``s``, ``z`` define it).  The gradient is the
    straight-through one of :func:`loss_bwd` (dW = dW_hat, gradient of mse), restricted to the
    rows of W_Q, W_K, W_V: ``sq[u] = sum over unit u's rows of dW^2``.  ``lambda_kl`` > 0 takes
    the gradient of the joint objective mse + lambda_kl kl / B (L_JAB with its KL term)."""
    out = loss_bwd(x, w, prob, bits3, s, z, fmt, lambda_kl=lambda_kl)
    dw = out["dw"]
    sq = [float(np.sum(dw[r0:r1] ** 2)) for (r0, r1) in prob.matrix_rows()]
    return {"sq": sq, "mse": out["mse"], "dw": dw}


# ----------------------------------------------------------------------------- fine-tuning
def adam_update(theta, g, m, v, t: int, lr: float, beta1: float, beta2: float, eps: float):
    """One Adam step (Kingma and Ba): biased moments, their bias corrections at step t, and
    theta - lr * m_hat / (sqrt(v_hat) + eps).  -> (theta, m, v)"""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    return theta - lr * m_hat / (np.sqrt(v_hat) + eps), m, v


def cosine_factor(t: int, n_steps: int) -> float:
    """Cosine annealing of the rate over the run (Appendix "Joint STE fine-tuning", (2)): the
    factor for step t = 1..n_steps, 1 at the first step, falling towards 0."""
    return 0.5 * (1.0 + math.cos(math.pi * (t - 1) / n_steps))


def ste_finetune(x, a_ref, x_held, a_ref_held, w_master, prob: Problem, bits3, s, z, fmt, n_steps: int,
                 eval_every: int, alpha_w: float, alpha_s: float, gammas, beta1=0.9, beta2=0.999,
                 adam_eps=1e-8, scale_floor=1e-12, lambda_kl: float = 0.0) -> dict:
    """Joint STE fine-tuning (Appendix "Joint STE fine-tuning"), the steps in the paper's order:

    (1) gradients by STE on the weights and LSQ on the scales (eq. lsq; :func:`loss_bwd` with the
        fixed float teacher ``a_ref``), at the latent weights rounded to the storage dtype;
    (2) Adam with grid-relative rates eta = alpha * sbar (eq. lr), sbar the mean starting scale
        over the quantized matrices, cosine-annealed over ``n_steps``;
    (4) every ``eval_every`` steps (and after the last) the held-out batch is scored and the best
        checkpoint kept; the start is the first checkpoint, so it is returned unless beaten;
    (5) the flip rate per matrix (eq. flip): the fraction of codes that differ between the start
        and the returned weights, both on the returned grid.

    With ``lambda_kl`` > 0 the objective is the joint loss mse + lambda_kl * kl / B (eq.
    joint_loss, the paper's default lambda 0.1): its gradient drives the steps, and the training
    log and the held-out scores are that objective, the maps taken against the float block.
    The latent weights are kept in fp32 (each update rounded to fp32), the scales too; the
    scales are kept >= ``scale_floor``.  Returns the stats array in the library's layout
    ([held start, held best, best step, flip Q, K, V, train mse per step, held mse per
    evaluation]), the returned fp32 weights and scales."""
    import dataclasses
    held = dataclasses.replace(prob, batch=len(x_held))
    master = round_fmt(np.asarray(w_master, np.float64), "f32")
    s = np.asarray(s, np.float64).copy()

    def dtype_w(wm):
        return wm if fmt in (None, "f32") else round_fmt(wm, fmt)

    w_float = np.asarray(w_master, np.float64)

    def kl_of(xs, wd, sc, pr):
        we = student_weight(wd, pr, bits3, sc, z, fmt)[0]
        tot = 0.0
        for i in range(len(xs)):
            yt = block_forward(xs[i], w_float, pr, fmt)[0]
            ys = block_forward(xs[i], we, pr, fmt)[0]
            tot += attention_kl(yt, ys, pr.n_heads, pr.n_kv_heads, pr.head_dim)[1]
        return tot / pr.batch

    def held_mse(wm, sc):
        m = loss_fwd(x_held, dtype_w(wm), held, bits3, sc, z, fmt, a_ref=a_ref_held)["mse"]
        return m + lambda_kl * kl_of(x_held, dtype_w(wm), sc, held) if lambda_kl else m

    rows = prob.matrix_rows()
    sel = [np.arange(r0, r1) for (r0, r1), b in zip(rows, bits3) if b]
    sbar = float(np.mean(s[np.concatenate(sel)])) if sel else 0.0
    w0 = dtype_w(master)
    mw, vw = np.zeros_like(master), np.zeros_like(master)
    ms, vs = np.zeros_like(s), np.zeros_like(s)
    start = held_mse(master, s)
    best, best_step, best_w, best_s = start, 0, master.copy(), s.copy()
    train, evals = [], []
    for t in range(1, n_steps + 1):
        out = loss_bwd(x, dtype_w(master), prob, bits3, s, z, fmt, gammas=gammas, a_ref=a_ref, lambda_kl=lambda_kl,
                       w_teacher=w_float)
        train.append(out["mse"] + (lambda_kl * kl_of(x, dtype_w(master), s, prob) if lambda_kl else 0.0))
        c = cosine_factor(t, n_steps)
        master, mw, vw = adam_update(master, out["dw"], mw, vw, t, alpha_w * sbar * c, beta1, beta2, adam_eps)
        master = round_fmt(master, "f32")
        s, ms, vs = adam_update(s, out["ds"], ms, vs, t, alpha_s * sbar * c, beta1, beta2, adam_eps)
        s = np.maximum(round_fmt(s, "f32"), scale_floor)
        if t % eval_every == 0 or t == n_steps:
            h = held_mse(master, s)
            evals.append(h)
            if h < best:
                best, best_step, best_w, best_s = h, t, master.copy(), s.copy()
    w_out = dtype_w(best_w)
    c0 = student_weight(w0, prob, bits3, best_s, z, fmt)[1]
    c1 = student_weight(w_out, prob, bits3, best_s, z, fmt)[1]
    flips = [float(np.mean(c0[r0:r1] != c1[r0:r1])) if b else 0.0 for (r0, r1), b in zip(rows, bits3)]
    stats = np.array([start, best, best_step] + flips + train + evals, np.float64)
    return {"stats": stats, "w_master": best_w, "scale": best_s, "w": w_out}
