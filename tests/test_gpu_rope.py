"""GPU parity with the rotary position embedding on Q and K (jab_problem.rope_theta > 0: the RoPE
Mistral applies) against the oracle (``oracle.reference.rope_qk`` inside the forward, the KL maps,
the sweep and the backward) in contract mode.

The device rotates the projection as accumulated (fp32) with fp32 cosines and sines of fp64
angles and rounds the result once to the dtype; the oracle rotates the exact projection in fp64
and rounds once.  The two differ by at most one unit in the last place of a rotated entry (away
from cancellation), as the projections themselves do, so the bars of the plain path hold: loss 1e-2 (16-bit) / 1e-5 (fp32), gradients 2e-2 / 1e-4,
KL 1e-2 / 1e-3."""
import itertools

import numpy as np
import pytest
import torch

from oracle import reference as ref
from paper_2609_34866_amd import inputs, jab

from gpu_helpers import device_inputs, oracle_problem, rel, small, ulp_diff_16bit

pytestmark = pytest.mark.gpu

THETA = 10000.0
LOSS_TOL = {"f32": 1e-5, "f16": 1e-2, "bf16": 1e-2}
GRAD_TOL = {"f32": 1e-4, "f16": 2e-2, "bf16": 2e-2}
KL_TOL = {"f32": 1e-3, "f16": 1e-2, "bf16": 1e-2}

SHAPES = [
    # (B, T, d, Hq, Hkv, dh, g, dtype)
    (2, 33, 128, 4, 2, 16, 32, "f32"),
    (2, 70, 256, 8, 2, 64, 64, "bf16"),
    (1, 130, 256, 4, 1, 128, 128, "f16"),
    (1, 300, 256, 8, 2, 128, 64, "bf16"),
]


def _wl(B, T, d, hq, hkv, dh, g, dtype, theta=THETA):
    return small(batch=B, seq_len=T, d_model=d, n_heads=hq, n_kv_heads=hkv, head_dim=dh, group_size=g,
                 dtype=dtype, rope_theta=theta)


@pytest.mark.parametrize("shape", SHAPES)
def test_rope_forward_and_backward_match_oracle(shape):
    wl = _wl(*shape)
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    bits = (3, 4, 2)
    scale, zero = jab.quant_init(p, w, bits)
    a = jab.attn_ref(p, x, w)
    fwd = jab.loss_fwd(p, x, w, bits, scale, zero, a).cpu().numpy()
    gam = jab.lsq_gscale(bits, wl.group_size)
    out, dw, ds = jab.loss_bwd(p, x, w, bits, scale, zero, a, gam)
    out, dw, ds = out.cpu().numpy(), dw.cpu().numpy().astype(np.float64), ds.cpu().numpy().astype(np.float64)
    prob = oracle_problem(wl)
    x64, w64 = inputs.to_f64(x.cpu()), inputs.to_f64(w.cpu())
    s, z = ref.init_scales(w64, prob, bits)
    want = ref.loss_bwd(x64, w64, prob, bits, s, z, wl.dtype, gammas=gam)
    assert rel(fwd[0], want["sse"]) < LOSS_TOL[wl.dtype]
    assert rel(out[1], want["mse"]) < LOSS_TOL[wl.dtype]
    for (r0, r1) in prob.matrix_rows():
        assert np.linalg.norm(dw[r0:r1] - want["dw"][r0:r1]) / np.linalg.norm(want["dw"][r0:r1]) < GRAD_TOL[wl.dtype]
        assert np.linalg.norm(ds[r0:r1] - want["ds"][r0:r1]) / np.linalg.norm(want["ds"][r0:r1]) < GRAD_TOL[wl.dtype]


def test_rope_changes_the_loss_and_keeps_it_zero_unquantized():
    wl = _wl(2, 70, 256, 8, 2, 64, 64, "bf16")
    x, w = device_inputs(wl)
    p, p0 = jab.problem_of(wl), jab.problem_of(_wl(2, 70, 256, 8, 2, 64, 64, "bf16", theta=0.0))
    scale, zero = jab.quant_init(p, w, (3, 3, 3))
    a, a0 = jab.attn_ref(p, x, w), jab.attn_ref(p0, x, w)
    assert not torch.equal(a, a0)
    assert float(jab.loss_fwd(p, x, w, (0, 0, 0), scale, zero, a)[0]) == 0.0
    l1 = float(jab.loss_fwd(p, x, w, (3, 3, 3), scale, zero, a)[0])
    l0 = float(jab.loss_fwd(p0, x, w, (3, 3, 3), scale, zero, a0)[0])
    assert l1 > 0 and l1 != l0


def test_rope_sweep_matches_oracle():
    wl = _wl(2, 70, 256, 8, 2, 64, 64, "bf16")
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    bits = [2, 4, 8]
    triples = list(itertools.product(bits, repeat=3))
    sc = [jab.quant_init(p, w, (b, b, b)) for b in bits]
    a = jab.attn_ref(p, x, w)
    loss, _ = jab.loss_sweep(p, x, w, bits, [s for s, _ in sc], [z for _, z in sc], triples, a)
    loss = loss.cpu().numpy()
    prob = oracle_problem(wl)
    x64, w64 = inputs.to_f64(x.cpu()), inputs.to_f64(w.cpu())
    sb = {b: ref.init_scales(w64, prob, (b, b, b)) for b in bits}
    want = ref.sweep(x64, w64, prob, triples, sb, "bf16")
    for i, t in enumerate(triples):
        assert rel(loss[i], want[t]["sse"]) < 1e-2, (t, loss[i], want[t]["sse"])


@pytest.mark.parametrize("shape", [(2, 40, 128, 4, 2, 16, 32, "f32"), (2, 64, 256, 8, 2, 64, 64, "bf16")])
def test_rope_kl_matches_oracle(shape):
    wl = _wl(*shape)
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    bits = (3, 3, 3)
    scale, zero = jab.quant_init(p, w, bits)
    a, qk, lse = jab.attn_ref_kl(p, x, w)
    out = jab.loss_fwd_kl(p, x, w, bits, scale, zero, a, qk, lse).cpu().numpy()
    prob = oracle_problem(wl)
    x64, w64 = inputs.to_f64(x.cpu()), inputs.to_f64(w.cpu())
    s, z = ref.init_scales(w64, prob, bits)
    want = ref.loss_kl(x64, w64, prob, bits, s, z, wl.dtype)
    B = wl.batch
    assert rel(out[3 + B], want["kl"]) < KL_TOL[wl.dtype], (out[3 + B], want["kl"])


@pytest.mark.parametrize("shape", [
    # the [Q|K] GEMM takes the rotation in its epilogue (rows and columns at least 256, d a multiple
    # of 64): head_dim 128 and 64, bf16 and fp16, a ragged last row tile, several sequences
    (2, 300, 256, 8, 2, 128, 64, "bf16"),
    (3, 200, 512, 8, 2, 64, 64, "f16"),
    (1, 520, 256, 4, 4, 64, 128, "bf16"),
    # a separate pass over an fp32 projection (too few rows for the persistent GEMM), head_dim 16
    (2, 70, 256, 8, 2, 64, 64, "bf16"),
    (2, 40, 128, 4, 2, 16, 32, "f16"),
])
def test_rope_projection_matches_oracle_to_an_ulp(shape):
    """The rotated [Q|K] the teacher cache keeps (jab_attn_ref_kl's qk_ref) against the oracle's:
    the exact projection turned in fp64 and rounded once to the dtype.  The device turns its fp32
    accumulators with fp32 (cos, sin) and rounds once, so the two agree to one unit in the last
    place, except where the pair's accumulation error (<= K 2^-24 sum|x w| per entry) or the fp32
    turn (2^-22 (|a| + |b|)) exceeds an ulp of a small result."""
    wl = _wl(*shape)
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    _, qk, _ = jab.attn_ref_kl(p, x, w)
    torch.cuda.synchronize()
    prob = oracle_problem(wl)
    B, T, hq, hkv, dh = wl.batch, wl.seq_len, wl.n_heads, wl.n_kv_heads, wl.head_dim
    nqk = (hq + hkv) * dh
    got = qk.cpu().reshape(B, T, nqk)
    x64, w64 = inputs.to_f64(x.cpu()), inputs.to_f64(w.cpu())
    for b in range(B):
        y = ref.project(x64[b], w64)
        want = ref.qkv_operands(y, prob, wl.dtype)[:, :nqk]
        want_t = torch.from_numpy(want).to(got.dtype)
        u = ulp_diff_16bit(got[b], want_t).numpy()
        err = np.abs(got[b].double().numpy() - want)
        acc = wl.d_model * 2.0 ** -24 * (np.abs(x64[b]) @ np.abs(w64[:nqk]).T)
        yq = np.abs(y[:, :nqk])
        # each output mixes an entry with its pair partner (dh/2 apart inside the head)
        part = lambda a: a.reshape(T, -1, 2, dh // 2)[:, :, ::-1].reshape(T, nqk)
        bound = np.abs(want) * 2.0 ** -(8 if wl.dtype == "bf16" else 11) + acc + part(acc) + \
            2.0 ** -22 * (yq + part(yq))
        assert np.all((u <= 1) | (err <= bound))
        assert float((u > 0).mean()) < 0.05
