"""GPU parity of the backward of the joint objective mse + lambda_KL kl / B (eq. joint_loss with
its KL attention-map term; jab_loss_bwd_kl) against the oracle (``oracle.reference.loss_bwd`` with
``lambda_kl``) in contract mode.

Tolerances are the backward's (relative L2 per matrix: 2e-2 for 16-bit, 1e-4 for fp32): the KL
term enters dS before the same dtype rounding as the squared-error term.  The KL value is bound
as in the forward KL test."""
import numpy as np
import pytest
import torch

from oracle import reference as ref
from paper_2609_34866_amd import inputs, jab

from gpu_helpers import device_inputs, oracle_problem, rel, small

pytestmark = pytest.mark.gpu

GRAD_TOL = {"f32": 1e-4, "f16": 2e-2, "bf16": 2e-2}
LOSS_TOL = {"f32": 1e-5, "f16": 1e-2, "bf16": 1e-2}
KL_TOL = {"f32": 1e-3, "f16": 1e-2, "bf16": 1e-2}

SHAPES = [
    # (B, T, d, Hq, Hkv, dh, g, dtype, rope, lambda_KL)
    (2, 33, 128, 4, 4, 16, 32, "f32", 0.0, 0.1),
    (2, 70, 256, 8, 2, 64, 64, "bf16", 0.0, 0.1),
    (1, 130, 256, 4, 1, 128, 128, "f16", 0.0, 0.1),
    (1, 97, 256, 8, 2, 128, 64, "f32", 0.0, 0.1),
    (1, 300, 256, 8, 2, 128, 64, "bf16", 10000.0, 0.1),
    # several key blocks of 128 (paired per workgroup) and ragged query tiles on the DMA kernels
    (2, 200, 256, 4, 2, 64, 64, "f16", 0.0, 0.1),
    (1, 520, 256, 4, 4, 64, 128, "bf16", 0.0, 0.1),
    (3, 1, 64, 2, 2, 16, 32, "bf16", 0.0, 0.1),
    # fp16 with the KL weight kappa = (N / 2) lambda / B = 6.7e5 far above 65504: the backward keeps
    # dS and dV scaled by a power of two and divides it out of the weight gradient
    (1, 130, 256, 4, 1, 128, 128, "f16", 0.0, 20.0),
    (2, 64, 256, 8, 2, 16, 32, "f16", 0.0, 20.0),
]


@pytest.mark.parametrize("shape", SHAPES)
def test_kl_backward_matches_oracle(shape):
    _check_kl_backward(shape)


# the 16-bit shapes at head_dim 64 / 128 once more with the dQ pass recomputing dS (no stored dS)
@pytest.mark.parametrize("shape", [s for s in SHAPES if s[7] != "f32" and s[5] in (64, 128)])
def test_kl_backward_recomputing_dq_matches_oracle(shape):
    jab.set_bwd_ds_limit(0)
    try:
        _check_kl_backward(shape)
    finally:
        jab.set_bwd_ds_limit(8 << 30)


def _check_kl_backward(shape):
    B, T, d, hq, hkv, dh, g, dtype, rope, lam = shape
    wl = small(batch=B, seq_len=T, d_model=d, n_heads=hq, n_kv_heads=hkv, head_dim=dh, group_size=g, dtype=dtype,
               rope_theta=rope)
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    bits = (3, 4, 2)
    scale, zero = jab.quant_init(p, w, bits)
    a, qk, lse = jab.attn_ref_kl(p, x, w)
    gam = jab.lsq_gscale(bits, wl.group_size)
    out, dw, ds = jab.loss_bwd_kl(p, x, w, bits, scale, zero, a, qk, lse, gam, lam)
    out, dw, ds = out.cpu().numpy(), dw.cpu().numpy().astype(np.float64), ds.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(dw)) and np.all(np.isfinite(ds))
    prob = oracle_problem(wl)
    x64, w64 = inputs.to_f64(x.cpu()), inputs.to_f64(w.cpu())
    s, z = ref.init_scales(w64, prob, bits)
    want = ref.loss_bwd(x64, w64, prob, bits, s, z, wl.dtype, gammas=gam, lambda_kl=lam)
    plain = ref.loss_bwd(x64, w64, prob, bits, s, z, wl.dtype, gammas=gam)
    want_kl = ref.loss_kl(x64, w64, prob, bits, s, z, wl.dtype)
    assert rel(out[1], want["mse"]) < LOSS_TOL[dtype]
    if T > 1:
        assert rel(out[3 + B], want_kl["kl"]) < KL_TOL[dtype]
    else:   # one key per row: the KL is 0; the single-pass form leaves a few 2^-24 of the scores
        assert want_kl["kl"] == 0.0 and abs(out[3 + B]) < 1e-4
    tol = GRAD_TOL[dtype]
    # a matrix whose exact gradient is 0 (W_Q and W_K of one-token sequences: the output does not
    # depend on the scores) is held against the whole gradient's norm: the GPU keeps the rounding
    # residual of P - P_t there (a few 2^-24 of the scores)
    floor_dw = 1e-5 * np.linalg.norm(want["dw"])
    floor_ds = 1e-5 * np.linalg.norm(want["ds"])
    for (r0, r1) in prob.matrix_rows():
        ref_dw = want["dw"][r0:r1]
        assert np.linalg.norm(dw[r0:r1] - ref_dw) / max(np.linalg.norm(ref_dw), floor_dw) < tol
        ref_ds = want["ds"][r0:r1]
        assert np.linalg.norm(ds[r0:r1] - ref_ds) / max(np.linalg.norm(ref_ds), floor_ds) < tol
    # the KL term is a visible part of the gradient at this lambda (beyond the tolerance); a single
    # token has one key per row, where the map is 1 whatever the weights
    (q0, q1) = prob.matrix_rows()[0]
    if T > 1:
        assert np.linalg.norm(want["dw"][q0:q1] - plain["dw"][q0:q1]) > 3 * tol * np.linalg.norm(want["dw"][q0:q1])


def test_kl_backward_lambda_zero_is_the_plain_backward_and_float_point_is_zero():
    wl = small(batch=2, seq_len=70, d_model=256, n_heads=8, n_kv_heads=2, head_dim=64, group_size=64, dtype="bf16")
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    bits = (3, 3, 3)
    scale, zero = jab.quant_init(p, w, bits)
    a, qk, lse = jab.attn_ref_kl(p, x, w)
    gam = jab.lsq_gscale(bits, wl.group_size)
    out0, dw0, ds0 = jab.loss_bwd_kl(p, x, w, bits, scale, zero, a, qk, lse, gam, 0.0)
    outp, dwp, dsp = jab.loss_bwd(p, x, w, bits, scale, zero, a, gam)
    # lambda = 0 adds exactly 0 to every dS entry on the same kernels: the same gradient
    assert float(out0[1]) == float(outp[1])
    assert torch.equal(dw0, dwp) and torch.equal(ds0, dsp)
    outf, dwf, dsf = jab.loss_bwd_kl(p, x, w, (0, 0, 0), scale, zero, a, qk, lse, (1.0, 1.0, 1.0), 0.1)
    assert float(outf[0]) == 0.0 and not torch.any(dwf) and not torch.any(dsf)
