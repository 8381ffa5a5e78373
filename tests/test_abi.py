"""The C-ABI library loads, exports what include/jab.h declares, and validates its
arguments on the host before any device work (these calls never reach HIP)."""
import ctypes
import os
import re

import pytest

from paper_2609_34866_amd import jab

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000      # aligned, never dereferenced: validation fails before any use


def _header_symbols():
    txt = open(os.path.join(ROOT, "include", "jab.h")).read()
    return sorted(set(re.findall(r"\b(jab_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    L = jab.lib()
    syms = _header_symbols()
    assert len(syms) >= 12
    for s in syms:
        assert hasattr(L, s), s
    assert set(syms) == set(jab.EXPORTED)


def _prob(**kw):
    base = dict(batch=2, seq_len=32, d_model=64, n_heads=4, n_kv_heads=4, head_dim=16, group_size=32,
                dtype=jab.F32, scheme=jab.ASYM, rope_theta=0.0)
    base.update(kw)
    return jab.Problem(*[base[k] for k, _ in jab.Problem._fields_])


def _loss_fwd(p, x=FAKE, w=FAKE, bits=(4, 4, 4), scale=FAKE, zero=FAKE, a_ref=FAKE, out=FAKE, ws=FAKE,
              ws_bytes=1 << 40):
    q = jab.Quant()
    for i in range(3):
        q.bits[i] = bits[i]
    q.scale, q.zero = scale, zero
    return jab.lib().jab_loss_fwd(ctypes.byref(p), x, w, ctypes.byref(q), a_ref, out, ws, ws_bytes, None)


def _last():
    return jab.lib().jab_last_error().decode()


def test_status_strings():
    L = jab.lib()
    assert L.jab_status_string(0) == b"JAB_OK"
    assert L.jab_status_string(-3) == b"JAB_E_WORKSPACE"


def test_backward_workspace_counts_the_stored_ds():
    """The backward's workspace holds 2 bytes per causal (sequence, query head, query,
    key) entry, in 32 x 32 tiles, for the 16-bit dtypes at head_dim 64 / 128 while that
    fits the limit; none for fp32 or head_dim 16, or under a limit of 0."""
    def ds_bytes(b, h, t):
        nq = (t + 31) // 32
        return b * h * nq * (nq + 1) // 2 * 2048

    cases = [(dict(batch=2, seq_len=70, d_model=256, n_heads=8, n_kv_heads=2, head_dim=64, group_size=64,
                   dtype=jab.BF16), True),
             (dict(batch=1, seq_len=2048, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128, group_size=128,
                   dtype=jab.F16), True),
             (dict(batch=2, seq_len=70, d_model=256, n_heads=8, n_kv_heads=2, head_dim=64, group_size=64,
                   dtype=jab.F32), False),
             (dict(batch=2, seq_len=70, d_model=64, n_heads=4, n_kv_heads=4, head_dim=16, group_size=32,
                   dtype=jab.BF16), False)]
    try:
        for kw, stores in cases:
            p = _prob(**kw)
            for op in (jab.OP_BWD, jab.OP_FISHER, jab.OP_STE):
                jab.set_bwd_ds_limit(8 << 30)
                full = jab.workspace_size(p, op)
                jab.set_bwd_ds_limit(0)
                none = jab.workspace_size(p, op)
                want = ds_bytes(p.batch, p.n_heads, p.seq_len) if stores else 0
                assert full - none == (want + 255) // 256 * 256, (kw, op)
                # a limit just below the buffer drops it
                jab.set_bwd_ds_limit(max(want - 1, 0))
                assert jab.workspace_size(p, op) == none
    finally:
        jab.set_bwd_ds_limit(8 << 30)


def test_workspace_size():
    p = _prob()
    for op in (jab.OP_FWD, jab.OP_REF, jab.OP_QUANTIZE, jab.OP_PROJECT):
        assert jab.workspace_size(p, op) > 0
    assert jab.workspace_size(p, jab.OP_SWEEP, 4) > jab.workspace_size(p, jab.OP_FWD)
    assert jab.workspace_size(p, jab.OP_SWEEP, 0) == 0
    assert jab.workspace_size(p, 99) == 0
    assert jab.workspace_size(_prob(head_dim=32), jab.OP_FWD) == 0
    # the forward workspace holds W_hat and the projection at least
    wl = _prob(batch=128, seq_len=2048, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
               group_size=128, dtype=jab.BF16)
    assert jab.workspace_size(wl, jab.OP_FWD) >= 2 * (6144 * 4096 + 128 * 2048 * 6144)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=0), jab.JAB_E_INVALID),
    (dict(n_heads=6, n_kv_heads=4), jab.JAB_E_INVALID),
    (dict(group_size=48), jab.JAB_E_INVALID),            # 64 % 48 != 0
    (dict(scheme=7), jab.JAB_E_INVALID),
    (dict(head_dim=32), jab.JAB_E_UNSUPPORTED),
    (dict(group_size=16), jab.JAB_E_UNSUPPORTED),
    (dict(dtype=5), jab.JAB_E_UNSUPPORTED),
    (dict(n_heads=12, n_kv_heads=4), jab.JAB_E_UNSUPPORTED),   # ratio 3
])
def test_problem_validation(kw, status):
    assert _loss_fwd(_prob(**kw)) == status
    assert _last()


@pytest.mark.parametrize("args,status", [
    (dict(x=None), jab.JAB_E_INVALID),
    (dict(x=FAKE + 8), jab.JAB_E_INVALID),                   # misaligned
    (dict(a_ref=None), jab.JAB_E_INVALID),
    (dict(out=FAKE + 4), jab.JAB_E_INVALID),
    (dict(bits=(1, 4, 4)), jab.JAB_E_INVALID),
    (dict(bits=(4, 9, 4)), jab.JAB_E_INVALID),
    (dict(scale=None), jab.JAB_E_INVALID),
    (dict(zero=None), jab.JAB_E_INVALID),                    # asymmetric needs zero-points
    (dict(ws=None), jab.JAB_E_INVALID),
    (dict(ws=FAKE + 16), jab.JAB_E_INVALID),                 # workspace must be 256-aligned
    (dict(ws_bytes=16), jab.JAB_E_WORKSPACE),
])
def test_argument_validation(args, status):
    assert _loss_fwd(_prob(), **args) == status


def test_symmetric_rejects_zero_points():
    assert _loss_fwd(_prob(scheme=jab.SYM)) == jab.JAB_E_INVALID
    assert "NULL" in _last()


def test_sweep_validation():
    L = jab.lib()
    p = _prob()
    bits = (ctypes.c_int32 * 2)(2, 4)
    ptrs = (ctypes.c_void_p * 2)(FAKE, FAKE)

    def call(triples, n_triples=None, bits_arr=bits, nb=2):
        flat = (ctypes.c_int32 * len(triples))(*triples)
        return L.jab_loss_sweep(ctypes.byref(p), FAKE, FAKE, nb, ctypes.cast(bits_arr, ctypes.c_void_p),
                                ctypes.cast(ptrs, ctypes.c_void_p), ctypes.cast(ptrs, ctypes.c_void_p),
                                n_triples or len(triples) // 3, ctypes.cast(flat, ctypes.c_void_p), FAKE,
                                FAKE, None, FAKE, 1 << 40, None)

    assert call([2, 4, 3]) == jab.JAB_E_INVALID                       # 3 not a candidate
    assert call([2, 4, 4], n_triples=9) == jab.JAB_E_INVALID           # more than n_bits^3
    dup = (ctypes.c_int32 * 2)(4, 4)
    assert call([4, 4, 4], bits_arr=dup) == jab.JAB_E_INVALID          # candidates must be distinct


def test_quant_init_validation():
    L = jab.lib()
    p = _prob()
    bits = (ctypes.c_int32 * 3)(4, 4, 10)
    assert L.jab_quant_init(ctypes.byref(p), FAKE, ctypes.cast(bits, ctypes.c_void_p), FAKE, FAKE,
                            None) == jab.JAB_E_INVALID
    bits = (ctypes.c_int32 * 3)(4, 4, 4)
    assert L.jab_quant_init(ctypes.byref(p), FAKE, ctypes.cast(bits, ctypes.c_void_p), FAKE, None,
                            None) == jab.JAB_E_INVALID


def test_no_cpu_fallback():
    """The binding has no path that computes without the HIP library."""
    src = open(os.path.join(ROOT, "paper_2609_34866_amd", "jab.py")).read()
    assert "oracle" not in src
    assert "numpy" not in src


def _curv(p, x=FAKE, w=FAKE, lam=0.1, n_probes=1, probes=FAKE, out=FAKE, ws=FAKE, ws_bytes=1 << 40):
    return jab.lib().jab_curvature(ctypes.byref(p), x, w, ctypes.c_float(lam), n_probes, probes, out, ws, ws_bytes,
                                   None)


@pytest.mark.parametrize("kw,msg", [
    (dict(x=None), "x / w"),
    (dict(w=FAKE + 4), "x / w"),
    (dict(n_probes=0), "probe"),
    (dict(probes=None), "probe"),
    (dict(lam=-0.1), "lambda"),
    (dict(lam=float("inf")), "lambda"),
    (dict(lam=float("nan")), "lambda"),
    (dict(out=FAKE + 4), "out"),
    (dict(ws=FAKE + 16), "workspace"),
])
def test_curvature_validation(kw, msg):
    assert _curv(_prob(), **kw) == jab.JAB_E_INVALID
    assert msg in _last()


def test_curvature_workspace():
    p = _prob()
    need = jab.workspace_size(p, jab.OP_CURVATURE)
    # the projection at the float point and its tangent are held at once
    assert need > jab.workspace_size(p, jab.OP_FWD) + jab.workspace_size(p, jab.OP_REF) // 2
    assert _curv(p, ws_bytes=need - 1) == jab.JAB_E_WORKSPACE


def test_fisher_validation_and_workspace():
    p = _prob()
    q = jab.Quant()
    for i in range(3):
        q.bits[i] = 2
    q.scale, q.zero = FAKE, FAKE
    L = jab.lib()
    need = jab.workspace_size(p, jab.OP_FISHER)
    # the backward's workspace plus dW, ds and the partial sums
    assert need > jab.workspace_size(p, jab.OP_BWD) + 4 * p.rows * p.d_model
    assert L.jab_fisher(ctypes.byref(p), FAKE, FAKE, ctypes.byref(q), FAKE, None, None, ctypes.c_float(0.0), FAKE, FAKE, need - 1, None) \
        == jab.JAB_E_WORKSPACE
    assert L.jab_fisher(ctypes.byref(p), FAKE, FAKE, ctypes.byref(q), None, None, None, ctypes.c_float(0.0), FAKE, FAKE, need, None) \
        == jab.JAB_E_INVALID
    assert "a_ref" in _last()
    assert L.jab_fisher(ctypes.byref(p), FAKE, FAKE, ctypes.byref(q), FAKE, None, None, ctypes.c_float(0.0), FAKE + 4, FAKE, need, None) \
        == jab.JAB_E_INVALID
    assert L.jab_fisher(ctypes.byref(p), FAKE, FAKE, ctypes.byref(q), FAKE, None, None, ctypes.c_float(0.1), FAKE,
                        FAKE, need, None) == jab.JAB_E_INVALID and "teacher cache" in _last()
    q.bits[0] = 9
    assert L.jab_fisher(ctypes.byref(p), FAKE, FAKE, ctypes.byref(q), FAKE, None, None, ctypes.c_float(0.0), FAKE, FAKE, need, None) \
        == jab.JAB_E_INVALID


def test_ste_validation_and_stats_len():
    L = jab.lib()
    assert L.jab_ste_stats_len(200, 10) == 6 + 200 + 20
    assert L.jab_ste_stats_len(7, 3) == 6 + 7 + 3
    assert L.jab_ste_stats_len(0, 1) == 6 and L.jab_ste_stats_len(5, 0) == 0
    p = _prob()
    need = jab.workspace_size(p, jab.OP_STE)
    assert need > jab.workspace_size(p, jab.OP_BWD) + 16 * p.rows * p.d_model
    b = (ctypes.c_int32 * 3)(3, 3, 3)
    g = (ctypes.c_float * 3)(1.0, 1.0, 1.0)

    def call(cfg=None, held=2, bits=b, ws_bytes=need, a_ref=FAKE):
        cfg = cfg or jab.SteConfig(10, 5, 0.05, 0.02, 0.9, 0.999, 1e-8, 1e-12, 0.0)
        return L.jab_ste_finetune(ctypes.byref(p), ctypes.byref(cfg), FAKE, a_ref, held, FAKE, FAKE, None, None, None,
                                  None,
                                  ctypes.cast(bits, ctypes.c_void_p), ctypes.cast(g, ctypes.c_void_p), FAKE, FAKE,
                                  FAKE, FAKE, FAKE, FAKE, ws_bytes, None)

    assert call(ws_bytes=need - 1) == jab.JAB_E_WORKSPACE
    assert call(held=3) == jab.JAB_E_INVALID and "held_batch" in _last()
    assert call(held=0) == jab.JAB_E_INVALID
    assert call(a_ref=None) == jab.JAB_E_INVALID
    assert call(cfg=jab.SteConfig(10, 0, 0.05, 0.02, 0.9, 0.999, 1e-8, 1e-12)) == jab.JAB_E_INVALID
    assert call(cfg=jab.SteConfig(10, 5, -1.0, 0.02, 0.9, 0.999, 1e-8, 1e-12)) == jab.JAB_E_INVALID
    assert call(cfg=jab.SteConfig(10, 5, 0.05, 0.02, 1.0, 0.999, 1e-8, 1e-12)) == jab.JAB_E_INVALID
    assert call(bits=(ctypes.c_int32 * 3)(3, 9, 3)) == jab.JAB_E_INVALID
    # the KL term needs the teacher caches
    assert call(cfg=jab.SteConfig(10, 5, 0.05, 0.02, 0.9, 0.999, 1e-8, 1e-12, 0.1)) == jab.JAB_E_INVALID
    assert "teacher caches" in _last()


@pytest.mark.parametrize("theta", [-1.0, float("nan"), float("inf")])
def test_rope_theta_validation(theta):
    assert _loss_fwd(_prob(rope_theta=theta)) == jab.JAB_E_INVALID
    assert "rope_theta" in _last()


def test_rope_workspace_holds_the_table():
    assert jab.workspace_size(_prob(rope_theta=10000.0), jab.OP_FWD) > jab.workspace_size(_prob(), jab.OP_FWD)


def test_loss_bwd_kl_validation():
    p = _prob()
    q = jab.Quant()
    for i in range(3):
        q.bits[i] = 3
    q.scale, q.zero = FAKE, FAKE
    g = (ctypes.c_float * 3)(1.0, 1.0, 1.0)
    L = jab.lib()
    need = jab.workspace_size(p, jab.OP_BWD)

    def call(qk=FAKE, lam=0.1, ws_bytes=need):
        return L.jab_loss_bwd_kl(ctypes.byref(p), FAKE, FAKE, ctypes.byref(q), FAKE, qk, FAKE,
                                 ctypes.cast(g, ctypes.c_void_p), ctypes.c_float(lam), FAKE, FAKE, FAKE, FAKE,
                                 ws_bytes, None)

    assert call(qk=None) == jab.JAB_E_INVALID and "qk_ref" in _last()
    assert call(lam=-0.1) == jab.JAB_E_INVALID and "lambda_kl" in _last()
    assert call(lam=float("nan")) == jab.JAB_E_INVALID
    assert call(ws_bytes=need - 1) == jab.JAB_E_WORKSPACE


def test_noalloc_validates_on_the_host():
    """jab_loss_fwd_noalloc rejects a problem whose workspace exceeds its device scratch
    (JAB_NOALLOC_SCRATCH_BYTES) and bad pointers before it touches the GPU."""
    L = jab.lib()
    q = jab.Quant()
    for i in range(3):
        q.bits[i] = 3
    q.scale, q.zero = FAKE, FAKE
    big = _prob(batch=64, seq_len=2048, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128, group_size=128,
                dtype=jab.BF16)
    assert jab.workspace_size(big, jab.OP_FWD) > jab.NOALLOC_SCRATCH_BYTES
    assert L.jab_loss_fwd_noalloc(ctypes.byref(big), FAKE, FAKE, ctypes.byref(q), FAKE, FAKE, None) == \
        jab.JAB_E_WORKSPACE
    assert "scratch" in _last()
    small_p = _prob()
    assert jab.workspace_size(small_p, jab.OP_FWD) <= jab.NOALLOC_SCRATCH_BYTES
    assert L.jab_loss_fwd_noalloc(ctypes.byref(small_p), None, FAKE, ctypes.byref(q), FAKE, FAKE, None) == \
        jab.JAB_E_INVALID
    assert L.jab_loss_fwd_noalloc(ctypes.byref(small_p), FAKE, FAKE, ctypes.byref(q), FAKE, FAKE + 4, None) == \
        jab.JAB_E_INVALID
