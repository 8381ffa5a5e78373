"""Python binding of libjab (the MI355X JAB-loss library).

Argument marshalling only: tensors provide device memory (``data_ptr``) and the
current HIP stream; every step of the computation runs in the library's HIP
kernels.  Importing this module does not touch the GPU; the first call loads
``libjab.so`` and raises if it was not built -- there is no fallback path.

Function names follow the C ABI in ``include/jab.h``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence, Tuple

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libjab.so")

JAB_OK, JAB_E_INVALID, JAB_E_UNSUPPORTED, JAB_E_WORKSPACE, JAB_E_HIP = 0, -1, -2, -3, -4
F32, F16, BF16 = 0, 1, 2
ASYM, SYM = 0, 1
OP_FWD, OP_SWEEP, OP_BWD, OP_REF, OP_QUANTIZE, OP_PROJECT, OP_FWD_KL, OP_CURVATURE, OP_FISHER, OP_STE = range(10)
KT_NAMES = ("quant", "gemm", "attn", "reduce", "attn_bwd", "dw_gemm", "misc", "gemm_vt", "kl")

_DTYPE_CODE = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}
_CODE_DTYPE = {v: k for k, v in _DTYPE_CODE.items()}


class JabError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seq_len", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("dtype", ctypes.c_int32), ("scheme", ctypes.c_int32),
                ("rope_theta", ctypes.c_float)]

    @property
    def rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def torch_dtype(self) -> torch.dtype:
        return _CODE_DTYPE[self.dtype]

    def with_batch(self, batch: int) -> "Problem":
        p = Problem()
        ctypes.pointer(p)[0] = self
        p.batch = batch
        return p


class Quant(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32 * 3), ("scale", ctypes.c_void_p), ("zero", ctypes.c_void_p)]


class SteConfig(ctypes.Structure):
    _fields_ = [("n_steps", ctypes.c_int32), ("eval_every", ctypes.c_int32), ("alpha_w", ctypes.c_float),
                ("alpha_s", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("adam_eps", ctypes.c_float), ("scale_floor", ctypes.c_float), ("lambda_kl", ctypes.c_float)]


def problem(batch, seq_len, d_model, n_heads, n_kv_heads, head_dim, group_size, dtype,
            scheme: int = ASYM, rope_theta: float = 0.0) -> Problem:
    code = _DTYPE_CODE[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return Problem(batch, seq_len, d_model, n_heads, n_kv_heads, head_dim, group_size, code, scheme, rope_theta)


def problem_of(wl, batch: Optional[int] = None) -> Problem:
    """Problem for a workload of ``paper_2609_34866_amd.inputs``."""
    return problem(wl.batch if batch is None else batch, wl.seq_len, wl.d_model, wl.n_heads,
                   wl.n_kv_heads, wl.head_dim, wl.group_size, wl.torch_dtype,
                   SYM if wl.symmetric else ASYM, wl.rope_theta)


_LIB = None


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libjab.so is not built ({LIB_PATH}); run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    vp, sz, i32, P = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.POINTER(Problem)
    Q = ctypes.POINTER(Quant)
    sig = {
        "jab_workspace_size": (sz, [P, i32, i32]),
        "jab_quant_init": (i32, [P, vp, vp, vp, vp, vp]),
        "jab_quantize": (i32, [P, vp, Q, vp, vp, vp, vp, sz, vp]),
        "jab_attn_ref": (i32, [P, vp, vp, vp, vp, sz, vp]),
        "jab_loss_fwd": (i32, [P, vp, vp, Q, vp, vp, vp, sz, vp]),
        "jab_loss_fwd_noalloc": (i32, [P, vp, vp, Q, vp, vp, vp]),
        "jab_attn_ref_kl": (i32, [P, vp, vp, vp, vp, vp, vp, sz, vp]),
        "jab_loss_fwd_kl": (i32, [P, vp, vp, Q, vp, vp, vp, vp, vp, sz, vp]),
        "jab_loss_sweep": (i32, [P, vp, vp, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp, sz, vp]),
        "jab_loss_bwd": (i32, [P, vp, vp, Q, vp, vp, vp, vp, vp, vp, sz, vp]),
        "jab_project": (i32, [P, vp, vp, Q, vp, vp, sz, vp]),
        "jab_allocate": (i32, [i32, i32, vp, vp, vp, ctypes.c_double, i32, i32, vp, vp]),
        "jab_omega": (i32, [i32, i32, vp, i32, vp, i32, i32, vp]),
        "jab_curvature": (i32, [P, vp, vp, ctypes.c_float, i32, vp, vp, vp, sz, vp]),
        "jab_fisher": (i32, [P, vp, vp, Q, vp, vp, vp, ctypes.c_float, vp, vp, sz, vp]),
        "jab_loss_bwd_kl": (i32, [P, vp, vp, Q, vp, vp, vp, vp, ctypes.c_float, vp, vp, vp, vp, sz, vp]),
        "jab_ste_stats_len": (i32, [i32, i32]),
        "jab_ste_finetune": (i32, [P, ctypes.POINTER(SteConfig), vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   vp, vp, vp, vp, vp, sz, vp]),
        "jab_status_string": (ctypes.c_char_p, [i32]),
        "jab_last_error": (ctypes.c_char_p, []),
        "jab_set_bwd_ds_limit": (i32, [ctypes.c_size_t]),
        "jab_timing_enable": (i32, [i32]),
        "jab_timing_read": (i32, [vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    _LIB = L
    return L


EXPORTED = ("jab_workspace_size", "jab_quant_init", "jab_quantize", "jab_attn_ref", "jab_loss_fwd",
            "jab_loss_fwd_noalloc",
            "jab_attn_ref_kl", "jab_loss_fwd_kl", "jab_loss_sweep", "jab_loss_bwd", "jab_project",
            "jab_allocate", "jab_omega", "jab_curvature", "jab_fisher", "jab_loss_bwd_kl", "jab_ste_stats_len", "jab_ste_finetune", "jab_status_string", "jab_last_error", "jab_set_bwd_ds_limit", "jab_timing_enable",
            "jab_timing_read")
ALLOC_GREEDY, ALLOC_PARETO = 0, 1
TRACE_BLOCK, TRACE_UNIT = 0, 1
OMEGA_C1, OMEGA_C2 = 0, 1


def _check(status: int) -> None:
    if status != JAB_OK:
        L = lib()
        raise JabError(status, f"{L.jab_status_string(status).decode()}: {L.jab_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream() -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _quant(bits: Sequence[int], scale: Optional[torch.Tensor], zero: Optional[torch.Tensor]) -> Quant:
    q = Quant()
    for i in range(3):
        q.bits[i] = int(bits[i])
    q.scale = None if scale is None else scale.data_ptr()
    q.zero = None if zero is None else zero.data_ptr()
    return q


def workspace_size(p: Problem, op: int, n_bits: int = 0) -> int:
    return int(lib().jab_workspace_size(ctypes.byref(p), op, n_bits))


def workspace(p: Problem, op: int, n_bits: int = 0, device="cuda") -> torch.Tensor:
    n = workspace_size(p, op, n_bits)
    if n == 0:
        raise JabError(JAB_E_INVALID, "invalid problem for workspace_size")
    return torch.empty(n, dtype=torch.uint8, device=device)


# --------------------------------------------------------------------------- entry points
def quant_init(p: Problem, w: torch.Tensor, bits: Sequence[int]) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    ng = p.d_model // p.group_size
    scale = torch.empty((p.rows, ng), dtype=torch.float32, device=w.device)
    zero = torch.empty((p.rows, ng), dtype=torch.uint8, device=w.device) if p.scheme == ASYM else None
    b = (ctypes.c_int32 * 3)(*[int(v) for v in bits])
    _check(lib().jab_quant_init(ctypes.byref(p), _ptr(w), ctypes.cast(b, ctypes.c_void_p), _ptr(scale),
                                _ptr(zero), _stream()))
    return scale, zero


def quantize(p: Problem, w: torch.Tensor, bits, scale, zero, want_codes=True, want_w_hat=True,
             want_werr=True, out: Optional[dict] = None, ws: Optional[torch.Tensor] = None) -> dict:
    """Codes, fake-quantized fp32 weights and eps^W sums; `out` may hold preallocated "codes",
    "w_hat" and "werr" tensors (then the want_* flags are ignored)."""
    dev = w.device
    if out is not None:
        codes, w_hat, werr = out.get("codes"), out.get("w_hat"), out.get("werr")
    else:
        codes = torch.empty((p.rows, p.d_model), dtype=torch.uint8, device=dev) if want_codes else None
        w_hat = torch.empty((p.rows, p.d_model), dtype=torch.float32, device=dev) if want_w_hat else None
        werr = torch.empty((3, 2), dtype=torch.float64, device=dev) if want_werr else None
    if werr is not None and ws is None:
        ws = workspace(p, OP_QUANTIZE, device=dev)
    q = _quant(bits, scale, zero)
    _check(lib().jab_quantize(ctypes.byref(p), _ptr(w), ctypes.byref(q), _ptr(codes), _ptr(w_hat), _ptr(werr),
                              _ptr(ws), 0 if ws is None else ws.numel(), _stream()))
    return {"codes": codes, "w_hat": w_hat, "werr": werr}


def project(p: Problem, x: torch.Tensor, w: torch.Tensor, bits=None, scale=None, zero=None,
            ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    y = torch.empty((p.batch, p.seq_len, p.rows), dtype=x.dtype, device=x.device)
    q = None if bits is None else _quant(bits, scale, zero)
    if q is not None and ws is None:
        ws = workspace(p, OP_PROJECT, device=x.device)
    _check(lib().jab_project(ctypes.byref(p), _ptr(x), _ptr(w), None if q is None else ctypes.byref(q), _ptr(y),
                             _ptr(ws), 0 if ws is None else ws.numel(), _stream()))
    return y


def attn_ref(p: Problem, x: torch.Tensor, w: torch.Tensor, ws: Optional[torch.Tensor] = None,
             out: Optional[torch.Tensor] = None) -> torch.Tensor:
    a = out if out is not None else torch.empty((p.batch, p.seq_len, p.n_heads * p.head_dim),
                                                dtype=torch.float32, device=x.device)
    if ws is None:
        ws = workspace(p, OP_REF, device=x.device)
    _check(lib().jab_attn_ref(ctypes.byref(p), _ptr(x), _ptr(w), _ptr(a), _ptr(ws), ws.numel(), _stream()))
    return a


def loss_fwd(p: Problem, x, w, bits, scale, zero, a_ref, ws: Optional[torch.Tensor] = None,
             out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """-> float64 [3 + B]: sse, mse, sum a_ref^2, sse per sequence."""
    if out is None:
        out = torch.empty(3 + p.batch, dtype=torch.float64, device=x.device)
    if ws is None:
        ws = workspace(p, OP_FWD, device=x.device)
    q = _quant(bits, scale, zero)
    _check(lib().jab_loss_fwd(ctypes.byref(p), _ptr(x), _ptr(w), ctypes.byref(q), _ptr(a_ref), _ptr(out),
                              _ptr(ws), ws.numel(), _stream()))
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20      # JAB_NOALLOC_SCRATCH_BYTES


def loss_fwd_noalloc(p: Problem, x, w, bits, scale, zero, a_ref, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """jab_loss_fwd on the library's own device scratch (no workspace argument) -> float64 [3 + B]."""
    if out is None:
        out = torch.empty(3 + p.batch, dtype=torch.float64, device=x.device)
    q = _quant(bits, scale, zero)
    _check(lib().jab_loss_fwd_noalloc(ctypes.byref(p), _ptr(x), _ptr(w), ctypes.byref(q), _ptr(a_ref), _ptr(out),
                                      _stream()))
    return out


def attn_ref_kl(p: Problem, x: torch.Tensor, w: torch.Tensor, ws: Optional[torch.Tensor] = None):
    """Teacher pass keeping the KL term's inputs -> (a_ref fp32 [B][T][Hq*dh], qk_ref dtype
    [B*T][(Hq+Hkv)*dh], lse_ref fp32 [B][Hq][T], base 2)."""
    a = torch.empty((p.batch, p.seq_len, p.n_heads * p.head_dim), dtype=torch.float32, device=x.device)
    qk = torch.empty((p.batch * p.seq_len, (p.n_heads + p.n_kv_heads) * p.head_dim), dtype=x.dtype,
                     device=x.device)
    lse = torch.empty((p.batch, p.n_heads, p.seq_len), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = workspace(p, OP_REF, device=x.device)
    _check(lib().jab_attn_ref_kl(ctypes.byref(p), _ptr(x), _ptr(w), _ptr(a), _ptr(qk), _ptr(lse), _ptr(ws),
                                 ws.numel(), _stream()))
    return a, qk, lse


def loss_fwd_kl(p: Problem, x, w, bits, scale, zero, a_ref, qk_ref, lse_ref, ws: Optional[torch.Tensor] = None,
                out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """-> float64 [2 (3 + B)]: loss_fwd's [3 + B], then kl, kl / B, teacher map mass defect,
    kl per sequence."""
    if out is None:
        out = torch.empty(2 * (3 + p.batch), dtype=torch.float64, device=x.device)
    if ws is None:
        ws = workspace(p, OP_FWD_KL, device=x.device)
    q = _quant(bits, scale, zero)
    _check(lib().jab_loss_fwd_kl(ctypes.byref(p), _ptr(x), _ptr(w), ctypes.byref(q), _ptr(a_ref), _ptr(qk_ref),
                                 _ptr(lse_ref), _ptr(out), _ptr(ws), ws.numel(), _stream()))
    return out


def loss_sweep(p: Problem, x, w, bits: Sequence[int], scales: Sequence[torch.Tensor],
               zeros: Optional[Sequence[Optional[torch.Tensor]]], triples: Sequence[Sequence[int]], a_ref,
               ws: Optional[torch.Tensor] = None, per_seq: bool = True):
    """-> (loss [n_triples] float64, loss_per_seq [n_triples][B] float64 or None)."""
    nb, nt = len(bits), len(triples)
    loss = torch.empty(nt, dtype=torch.float64, device=x.device)
    lps = torch.empty((nt, p.batch), dtype=torch.float64, device=x.device) if per_seq else None
    if ws is None:
        ws = workspace(p, OP_SWEEP, nb, device=x.device)
    cb = (ctypes.c_int32 * nb)(*[int(b) for b in bits])
    cs = (ctypes.c_void_p * nb)(*[s.data_ptr() for s in scales])
    cz = None
    if zeros is not None:
        cz = (ctypes.c_void_p * nb)(*[None if z is None else z.data_ptr() for z in zeros])
    flat = [int(v) for t in triples for v in t]
    ct = (ctypes.c_int32 * len(flat))(*flat)
    _check(lib().jab_loss_sweep(ctypes.byref(p), _ptr(x), _ptr(w), nb, ctypes.cast(cb, ctypes.c_void_p),
                                ctypes.cast(cs, ctypes.c_void_p),
                                None if cz is None else ctypes.cast(cz, ctypes.c_void_p), nt,
                                ctypes.cast(ct, ctypes.c_void_p), _ptr(a_ref), _ptr(loss), _ptr(lps), _ptr(ws),
                                ws.numel(), _stream()))
    return loss, lps


def loss_bwd(p: Problem, x, w, bits, scale, zero, a_ref, gscale: Sequence[float],
             ws: Optional[torch.Tensor] = None):
    """-> (out [3 + B] float64, dw [R][d] fp32, dscale [R][d/g] fp32)."""
    dev = x.device
    out = torch.empty(3 + p.batch, dtype=torch.float64, device=dev)
    dw = torch.empty((p.rows, p.d_model), dtype=torch.float32, device=dev)
    ds = torch.empty((p.rows, p.d_model // p.group_size), dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(p, OP_BWD, device=dev)
    g = (ctypes.c_float * 3)(*[float(v) for v in gscale])
    q = _quant(bits, scale, zero)
    _check(lib().jab_loss_bwd(ctypes.byref(p), _ptr(x), _ptr(w), ctypes.byref(q), _ptr(a_ref),
                              ctypes.cast(g, ctypes.c_void_p), _ptr(out), _ptr(dw), _ptr(ds), _ptr(ws),
                              ws.numel(), _stream()))
    return out, dw, ds


def fisher(p: Problem, x, w, bits, scale, zero, a_ref, ws: Optional[torch.Tensor] = None,
           out: Optional[torch.Tensor] = None, lambda_kl: float = 0.0, kl_cache=None) -> torch.Tensor:
    """Fisher-coupling scores at the probe (bits, scale, zero) -> float64 [4]: the squared
    straight-through gradient norms of W_Q, W_K, W_V and the mse."""
    if out is None:
        out = torch.empty(4, dtype=torch.float64, device=x.device)
    if ws is None:
        ws = workspace(p, OP_FISHER, device=x.device)
    q = _quant(bits, scale, zero)
    qk_t, lse_t = kl_cache if kl_cache is not None else (None, None)
    _check(lib().jab_fisher(ctypes.byref(p), _ptr(x), _ptr(w), ctypes.byref(q), _ptr(a_ref), _ptr(qk_t), _ptr(lse_t),
                            float(lambda_kl), _ptr(out), _ptr(ws), ws.numel(), _stream()))
    return out


def ste_finetune(p: Problem, x, a_ref, x_held, a_ref_held, bits, w_master, scale, zero, gscale=None,
                 n_steps: int = 200, eval_every: int = 10, alpha_w: float = 0.05, alpha_s: float = 0.02,
                 beta1: float = 0.9, beta2: float = 0.999, adam_eps: float = 1e-8, scale_floor: float = 1e-12,
                 ws: Optional[torch.Tensor] = None, w: Optional[torch.Tensor] = None, lambda_kl: float = 0.0,
                 kl_cache=None, kl_cache_held=None):
    """Joint STE fine-tuning; w_master (fp32) and scale are updated in place to the best
    checkpoint -> (w in the dtype, stats float64; see jab_ste_stats_len for the layout)."""
    dev = x.device
    cfg = SteConfig(n_steps, eval_every, alpha_w, alpha_s, beta1, beta2, adam_eps, scale_floor, lambda_kl)
    qk_t, lse_t = kl_cache if kl_cache is not None else (None, None)
    qk_h, lse_h = kl_cache_held if kl_cache_held is not None else (None, None)
    n = lib().jab_ste_stats_len(n_steps, eval_every)
    if n <= 0:
        raise JabError(JAB_E_INVALID, "invalid n_steps / eval_every")
    stats = torch.empty(n, dtype=torch.float64, device=dev)
    if w is None:
        w = torch.empty((p.rows, p.d_model), dtype=x.dtype, device=dev)
    if ws is None:
        ws = workspace(p, OP_STE, device=dev)
    if gscale is None:
        gscale = lsq_gscale(bits, p.group_size)
    b = (ctypes.c_int32 * 3)(*[int(v) for v in bits])
    g = (ctypes.c_float * 3)(*[float(v) for v in gscale])
    _check(lib().jab_ste_finetune(ctypes.byref(p), ctypes.byref(cfg), _ptr(x), _ptr(a_ref), int(x_held.shape[0]),
                                  _ptr(x_held), _ptr(a_ref_held), _ptr(qk_t), _ptr(lse_t), _ptr(qk_h), _ptr(lse_h),
                                  ctypes.cast(b, ctypes.c_void_p),
                                  ctypes.cast(g, ctypes.c_void_p), _ptr(w_master), _ptr(w), _ptr(scale),
                                  _ptr(zero), _ptr(stats), _ptr(ws), ws.numel(),
                                  _stream()))
    return w, stats


def loss_bwd_kl(p: Problem, x, w, bits, scale, zero, a_ref, qk_ref, lse_ref, gscale: Sequence[float],
                lambda_kl: float, ws: Optional[torch.Tensor] = None):
    """Backward of mse + lambda_kl * kl / B -> (out [2 (3 + B)] float64, dw, dscale)."""
    dev = x.device
    out = torch.empty(2 * (3 + p.batch), dtype=torch.float64, device=dev)
    dw = torch.empty((p.rows, p.d_model), dtype=torch.float32, device=dev)
    ds = torch.empty((p.rows, p.d_model // p.group_size), dtype=torch.float32, device=dev)
    if ws is None:
        ws = workspace(p, OP_BWD, device=dev)
    g = (ctypes.c_float * 3)(*[float(v) for v in gscale])
    q = _quant(bits, scale, zero)
    _check(lib().jab_loss_bwd_kl(ctypes.byref(p), _ptr(x), _ptr(w), ctypes.byref(q), _ptr(a_ref), _ptr(qk_ref),
                                 _ptr(lse_ref), ctypes.cast(g, ctypes.c_void_p), float(lambda_kl), _ptr(out),
                                 _ptr(dw), _ptr(ds), _ptr(ws), ws.numel(), _stream()))
    return out, dw, ds


CURVATURE_FORMS = ("t_Q", "t_K", "t_V", "pooled", "h_QQ", "h_KK", "h_VV")


def curvature(p: Problem, x, w, probes: torch.Tensor, lambda_kl: float = 0.0, ws: Optional[torch.Tensor] = None,
              out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Hutchinson terms of eq. gn's Hessian at the float point -> float64 [n_probes][7] in the order of
    CURVATURE_FORMS (per-unit partition t_u, pooled v^T H v, diagonal blocks h_uu).
    probes: int8 [n_probes][R][d_model] in {-1, +1}."""
    n_probes = probes.shape[0]
    if out is None:
        out = torch.empty((n_probes, 7), dtype=torch.float64, device=x.device)
    if ws is None:
        ws = workspace(p, OP_CURVATURE, device=x.device)
    _check(lib().jab_curvature(ctypes.byref(p), _ptr(x), _ptr(w), float(lambda_kl), n_probes, _ptr(probes),
                               _ptr(out), _ptr(ws), ws.numel(), _stream()))
    return out


def allocate(omega, widths: Sequence[int], params: Sequence[float], budget_bits: float, min_bits: int = 0,
             method: int = ALLOC_GREEDY) -> Tuple[list, float]:
    """Bit allocation of eq. mckp (host-only) -> (width index per unit, objective)."""
    rows = [list(map(float, r)) for r in omega]
    n, k = len(rows), len(widths)
    if any(len(r) != k for r in rows) or len(params) != n:
        raise JabError(JAB_E_INVALID, "omega must be [n_units][n_widths] and params [n_units]")
    om = (ctypes.c_double * (n * k))(*[v for r in rows for v in r])
    wd = (ctypes.c_int32 * k)(*[int(v) for v in widths])
    pr = (ctypes.c_double * n)(*[float(v) for v in params])
    ch = (ctypes.c_int32 * n)()
    obj = ctypes.c_double(0.0)
    _check(lib().jab_allocate(n, k, ctypes.addressof(wd), ctypes.addressof(om), ctypes.addressof(pr),
                              float(budget_bits), int(min_bits), int(method), ctypes.addressof(ch),
                              ctypes.addressof(obj)))
    return list(ch), obj.value


def omega(curv, werr, trace: int = TRACE_BLOCK, criterion: int = OMEGA_C1) -> torch.Tensor:
    """Sensitivity table of eq. omega (host-only): curv [n_layers][n_probes][7] (jab_curvature's
    output per block), werr [n_layers][n_widths][3][2] (jab_quantize's per width) ->
    omega [3 n_layers][n_widths] (float64, host) for jab_allocate."""
    c = torch.as_tensor(curv, dtype=torch.float64).cpu().contiguous()
    e = torch.as_tensor(werr, dtype=torch.float64).cpu().contiguous()
    if c.dim() != 3 or c.shape[2] != 7 or e.dim() != 4 or e.shape[0] != c.shape[0] or tuple(e.shape[2:]) != (3, 2):
        raise JabError(JAB_E_INVALID, "curv must be [n_layers][n_probes][7] and werr [n_layers][n_widths][3][2]")
    out = torch.empty((3 * c.shape[0], e.shape[1]), dtype=torch.float64)
    _check(lib().jab_omega(c.shape[0], c.shape[1], c.data_ptr(), e.shape[1], e.data_ptr(), int(trace),
                           int(criterion), out.data_ptr()))
    return out


def set_bwd_ds_limit(max_bytes: int) -> None:
    """Largest stored-dS buffer the attention backward keeps in its workspace (default
    8 GiB; 0 recomputes dS in the dQ pass).  Set before sizing workspaces."""
    _check(lib().jab_set_bwd_ds_limit(int(max_bytes)))


def timing_enable(on: bool = True) -> None:
    _check(lib().jab_timing_enable(1 if on else 0))


def timing_read() -> dict:
    """Per kernel family: (summed milliseconds, launches) since the last read."""
    ms = (ctypes.c_double * len(KT_NAMES))()
    n = (ctypes.c_int64 * len(KT_NAMES))()
    _check(lib().jab_timing_read(ctypes.cast(ms, ctypes.c_void_p), ctypes.cast(n, ctypes.c_void_p)))
    return {k: (ms[i], n[i]) for i, k in enumerate(KT_NAMES)}


def lsq_gscale(bits: Sequence[int], group: int, scheme: int = ASYM):
    """LSQ's gradient factor (n_w q_max)^(-1/2) per matrix, n_w = weights sharing a scale."""
    out = []
    for b in bits:
        if b == 0:
            out.append(0.0)
            continue
        qmax = (1 << b) - 1 if scheme == ASYM else (1 << (b - 1)) - 1
        out.append(float((group * qmax) ** -0.5))
    return out
