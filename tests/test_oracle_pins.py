"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these compares the oracle with a retyped copy of itself: each checks it
against a different computation (hardware fp32 / numpy / torch conversions, an
exhaustive grid search, the materialised attention matrix, finite differences,
torch autograd) or against an exact property stated in the paper.
"""
import math

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import reference as ref
from paper_2609_34866_amd import inputs

RNG = np.random.default_rng(1234)


def _wide_values(n, rng):
    mant = rng.uniform(-2, 2, n)
    exp = rng.integers(-140, 120, n)
    return np.ldexp(mant, exp)


# ----------------------------------------------------------------------------- rounding
def test_round_fp32_matches_hardware_cast():
    x = _wide_values(200000, RNG)
    got = ref.round_fmt(x, "f32")
    want = x.astype(np.float32).astype(np.float64)
    assert np.array_equal(got, want)


def test_round_fp16_matches_numpy_cast():
    x = np.concatenate([_wide_values(100000, RNG) * 1e-30, RNG.normal(0, 1000, 100000),
                        RNG.normal(0, 1e-6, 10000), np.array([65504.0, 65519.99, 65520.0, -65520.0])])
    got = ref.round_fmt(x, "f16")
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).astype(np.float64)
    assert np.array_equal(got, want)


def test_round_bf16_matches_torch_cast_and_ties():
    x32 = _wide_values(200000, RNG).astype(np.float32)
    got = ref.round_fmt(x32.astype(np.float64), "bf16")
    want = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(got, want)
    # exact ties go to the even significand
    ties = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 2 ** -130 * (1 + 2 ** -8)])
    assert np.array_equal(ref.round_fmt(ties, "bf16"), [1.0, 1 + 2 ** -6, -1.0, 2 ** -130])


# ----------------------------------------------------------------------------- quantizer
@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("group", [32, 128])
def test_codes_are_the_nearest_grid_point(bits, group):
    rows, cols = 64, 256
    w = RNG.normal(0, 0.02, (rows, cols)).astype(np.float32).astype(np.float64)
    s, z = ref.quant_params(w, group, bits)
    codes, w_hat, _ = ref.fake_quant(w, group, bits, s, z)
    want = brute.nearest_codes(w, s, z, bits, group)
    mismatch = codes != want
    if mismatch.any():
        # only near-ties of the fp32 quotient may differ (reading of "round")
        v = w / np.repeat(s, group, axis=1)
        frac = np.abs(np.abs(v - np.floor(v)) - 0.5)
        assert np.all(frac[mismatch] < 2.0 ** -22 * np.maximum(1, np.abs(v[mismatch])))
    assert mismatch.mean() < 1e-3
    assert codes.min() >= 0 and codes.max() <= (1 << bits) - 1
    ze = np.repeat(z, group, axis=1)
    assert np.array_equal(w_hat, (codes - ze) * np.repeat(s, group, axis=1))


def test_exact_ties_round_to_even():
    s = np.full((1, 1), 2.0 ** -6)
    z = np.full((1, 1), 4, np.int32)
    k = np.arange(-4, 4)
    w = ((k + 0.5) * 2.0 ** -6)[None, :]
    w = np.pad(w, ((0, 0), (0, 0)))
    codes, _, _ = ref.fake_quant(w, 8, 3, s, z)
    u = np.where(k % 2 == 0, k, k + 1)                 # round half to even of k + 1/2
    assert np.array_equal(codes[0], np.clip(u + 4, 0, 7))
    assert np.array_equal(codes, brute.nearest_codes(w, s, z, 3, 8))


@pytest.mark.parametrize("bits", [2, 3, 4, 5, 6, 7, 8])
def test_scale_and_zero_point(bits):
    rows, cols, g = 128, 256, 128
    w = RNG.normal(0, 0.02, (rows, cols)).astype(np.float32).astype(np.float64)
    w[0, :g] = 0.0                                      # degenerate group
    w[1, :g] = np.abs(w[1, :g])                         # all non-negative -> z = 0
    s, z = ref.quant_params(w, g, bits)
    L = (1 << bits) - 1
    # fp32 arithmetic of the min-max rule, evaluated by numpy's float32 hardware ops
    grp = w.reshape(rows, cols // g, g)
    lo = np.minimum(grp.min(-1), 0).astype(np.float32)
    hi = np.maximum(grp.max(-1), 0).astype(np.float32)
    s32 = (hi - lo) / np.float32(L)
    s32 = np.where(s32 == 0, np.float32(1), s32)
    z32 = np.clip(np.rint(-lo / s32), 0, L)
    assert np.array_equal(s, s32.astype(np.float64))
    assert np.array_equal(z, z32.astype(np.int32))
    assert s[0, 0] == 1.0 and z[0, 0] == 0 and z[1, 0] == 0
    codes, w_hat, _ = ref.fake_quant(w, g, bits, s, z)
    assert np.all(w_hat[0, :g] == 0.0)
    # the group minimum lands on code 0
    amin = grp.argmin(-1)
    rr, jj = np.nonzero(grp.min(-1) < 0)
    assert np.all(codes[rr, jj * g + amin[rr, jj]] == 0)


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_quantizer_idempotent(bits):
    g = 32
    w = RNG.normal(0, 0.05, (64, 128)).astype(np.float32).astype(np.float64)
    s, z = ref.quant_params(w, g, bits)
    c1, wh1, _ = ref.fake_quant(w, g, bits, s, z)
    wh32 = ref.round_fmt(wh1, "f32")
    c2, wh2, _ = ref.fake_quant(wh32, g, bits, s, z)
    assert np.array_equal(c1, c2)
    assert np.array_equal(wh1, wh2)


def test_symmetric_two_bit_is_ternary():
    g = 32
    w = RNG.normal(0, 0.05, (16, 64))
    s, _ = ref.quant_params(w, g, 2, ref.SYM)
    codes, w_hat, _ = ref.fake_quant(w, g, 2, s, None, ref.SYM)
    se = np.repeat(s, g, axis=1)
    assert set(np.unique(np.round(w_hat / se)).tolist()) <= {-1.0, 0.0, 1.0}
    assert np.array_equal(codes, brute.nearest_codes_sym(w, s, 2, g))


@pytest.mark.parametrize("bits,group,expected", [(3, 128, 0.215), (4, 128, 0.101), (8, 128, 0.0059),
                                                 (3, 32, 0.173), (4, 32, 0.081)])
def test_weight_error_matches_rounding_noise_model(bits, group, expected):
    """eps^W = ||W - W_hat||_F / ||W||_F against the uniform rounding-noise model
    sigma^2 = s^2 / 12 used in the paper's variance argument."""
    w = RNG.normal(0, 0.02, (512, 1024))
    s, z = ref.quant_params(w, group, bits)
    _, w_hat, _ = ref.fake_quant(w, group, bits, s, z)
    eps = np.linalg.norm(w - w_hat) / np.linalg.norm(w)
    model = math.sqrt(np.mean(s ** 2) / 12) / np.sqrt(np.mean(w ** 2))
    assert abs(eps / model - 1) < 0.03
    assert abs(eps / expected - 1) < 0.03


def test_lsq_factor_branches():
    """phi of eq. lsq: u - v inside the representable range, the clipped offset outside."""
    s = np.full((1, 1), 0.5)
    z = np.full((1, 1), 2, np.int32)            # 3-bit: codes 0..7, offsets -2..5
    w = np.array([[-2.0, -1.2, -1.05, -0.2, 0.26, 2.5, 2.7, 3.0]])
    _, _, phi = ref.fake_quant(w, 8, 3, s, z)
    v = w[0] / 0.5
    u = np.rint(v)
    want = np.where(v < -2, -2.0, np.where(v > 5, 5.0, u - v))
    assert np.allclose(phi[0], want, rtol=0, atol=1e-6)
    # symmetric: |v| <= q_max -> q - v, else sign(v) q_max
    s2, _ = np.full((1, 1), 0.5), None
    w2 = np.array([[-2.0, -1.6, -0.7, 0.0, 0.74, 1.4, 1.6, 4.0]])
    _, _, phi2 = ref.fake_quant(w2, 8, 3, s2, None, ref.SYM)
    v2 = w2[0] / 0.5
    q2 = np.clip(np.rint(v2), -3, 3)
    want2 = np.where(np.abs(v2) <= 3, q2 - v2, np.sign(v2) * 3)
    assert np.allclose(phi2[0], want2, rtol=0, atol=1e-6)


# ----------------------------------------------------------------------------- projection / attention
def test_projection_matches_numpy_matmul():
    x = RNG.normal(size=(33, 96))
    w = RNG.normal(size=(80, 96))
    y = ref.project(x, w)
    np.testing.assert_allclose(y, x @ w.T, rtol=1e-12, atol=1e-12)


ATTN_SHAPES = [(1, 1, 1, 16), (2, 2, 1, 16), (7, 4, 1, 16), (33, 4, 2, 16), (33, 4, 4, 64),
               (20, 8, 2, 128), (17, 2, 2, 64)]


@pytest.mark.parametrize("T,hq,hkv,dh", ATTN_SHAPES)
def test_attention_matches_brute_force(T, hq, hkv, dh):
    R = (hq + 2 * hkv) * dh
    y = RNG.normal(0, 1.5, (T, R))
    a, lse, dev = ref.attention(y, hq, hkv, dh)
    q = y[:, :hq * dh].reshape(T, hq, dh)
    k = y[:, hq * dh:(hq + hkv) * dh].reshape(T, hkv, dh)
    v = y[:, (hq + hkv) * dh:].reshape(T, hkv, dh)
    ab, P = brute.attention(q, k, v, hq, hkv)
    np.testing.assert_allclose(a, ab, rtol=1e-12, atol=1e-12)
    assert dev < 1e-14
    # lse = log sum_j exp(S_ij)
    S = np.einsum("ihc,jhc->hij", q, np.repeat(k, hq // hkv, axis=1)) / np.sqrt(dh)
    S = np.where(np.tril(np.ones((T, T), bool))[None], S, -np.inf)
    np.testing.assert_allclose(lse, np.log(np.exp(S).sum(-1)), rtol=1e-12)


def test_token_zero_sees_only_itself():
    T, hq, hkv, dh = 9, 4, 2, 16
    y = RNG.normal(size=(T, (hq + 2 * hkv) * dh))
    a, _, _ = ref.attention(y, hq, hkv, dh)
    voff = (hq + hkv) * dh
    for h in range(hq):
        kv = h * hkv // hq
        assert np.array_equal(a[0, h * dh:(h + 1) * dh], y[0, voff + kv * dh: voff + (kv + 1) * dh])


def test_causality():
    T, hq, hkv, dh, t = 24, 4, 1, 16, 10
    y = RNG.normal(size=(T, (hq + 2 * hkv) * dh))
    a1, _, _ = ref.attention(y, hq, hkv, dh)
    y2 = y.copy()
    y2[t + 1:] = RNG.normal(size=y2[t + 1:].shape)
    a2, _, _ = ref.attention(y2, hq, hkv, dh)
    assert np.array_equal(a1[:t + 1], a2[:t + 1])
    assert not np.array_equal(a1[t + 1:], a2[t + 1:])


# ----------------------------------------------------------------------------- KL term
def _maps(y, T, hq, hkv, dh):
    q = y[:, :hq * dh].reshape(T, hq, dh)
    k = y[:, hq * dh:(hq + hkv) * dh].reshape(T, hkv, dh)
    v = y[:, (hq + hkv) * dh:].reshape(T, hkv, dh)
    return brute.attention(q, k, v, hq, hkv)[1]


@pytest.mark.parametrize("T,hq,hkv,dh", ATTN_SHAPES)
def test_kl_matches_scipy_rel_entr_on_materialised_maps(T, hq, hkv, dh):
    """D_KL(P || Q) of eq. joint_loss: P the teacher's map, Q the student's, summed over keys per
    query row; scipy's rel_entr(p, q) = p log(p / q) (0 for p = 0) on the brute-force maps."""
    from scipy.special import rel_entr
    R = (hq + 2 * hkv) * dh
    yt = RNG.normal(0, 1.5, (T, R))
    ys = yt + RNG.normal(0, 0.3, (T, R))
    kl, tot = ref.attention_kl(yt, ys, hq, hkv, dh)
    P, Q = _maps(yt, T, hq, hkv, dh), _maps(ys, T, hq, hkv, dh)
    want = rel_entr(P, Q).sum(axis=2)                  # [Hq][T]
    np.testing.assert_allclose(kl, want, rtol=1e-9, atol=1e-13)
    assert abs(tot - want.sum()) <= 1e-9 * abs(want.sum()) + 1e-13
    assert np.all(kl >= -1e-15)                        # Gibbs' inequality
    assert np.all(kl[:, 0] == 0.0)                     # query 0 sees one key: both maps are 1


def test_kl_two_keys_is_bernoulli_kl():
    """T = 2, one head, d_head 1: query 1's maps over keys (0, 1) are Bernoulli(sigma(a1 - a0))
    and Bernoulli(sigma(b1 - b0)); D_KL(P || Q) = p log(p/q) + (1-p) log((1-p)/(1-q))."""
    a, b = (0.5, 2.0), (1.0, 1.5)                     # teacher and student scores of query 1
    yt = np.array([[0.0, a[0], 0.0], [1.0, a[1], 0.0]])   # columns: q, k, v (d_head 1)
    ys = np.array([[0.0, b[0], 0.0], [1.0, b[1], 0.0]])
    kl, tot = ref.attention_kl(yt, ys, 1, 1, 1)
    p = 1.0 / (1.0 + math.exp(-(a[1] - a[0])))
    q = 1.0 / (1.0 + math.exp(-(b[1] - b[0])))
    want = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
    assert kl[0, 0] == 0.0
    assert abs(kl[0, 1] - want) <= 1e-14
    assert abs(tot - want) <= 1e-14
    # the direction is P || Q (teacher first): the reverse divergence differs here
    rev = q * math.log(q / p) + (1 - q) * math.log((1 - q) / (1 - p))
    assert abs(want - rev) > 1e-3


def test_kl_is_zero_for_identical_maps():
    T, hq, hkv, dh = 19, 4, 2, 16
    y = RNG.normal(0, 2.0, (T, (hq + 2 * hkv) * dh))
    kl, tot = ref.attention_kl(y, y, hq, hkv, dh)
    assert tot == 0.0 and np.all(kl == 0.0)


def test_kl_loss_is_batchmean_of_the_full_maps():
    """The Appendix on the effective weight of the KL term: the KL sum runs over B * Hq * T^2
    map entries and is divided by B only.  Brute force over the materialised maps of the
    quantized and float blocks."""
    from scipy.special import rel_entr
    prob = _tiny_problem(B=3, T=12)
    x, w = _tiny_inputs(prob, seed=5)
    bits = (3, 2, 4)
    s, z = ref.init_scales(w, prob, bits)
    out = ref.loss_kl(x, w, prob, bits, s, z, None)
    w_hat = w.copy()
    for (r0, r1), bb in zip(prob.matrix_rows(), bits):
        c = brute.nearest_codes(w[r0:r1], s[r0:r1], z[r0:r1], bb, prob.group_size)
        w_hat[r0:r1] = (c - np.repeat(z[r0:r1], prob.group_size, 1)) * np.repeat(s[r0:r1], prob.group_size, 1)
    total = 0.0
    for b in range(prob.batch):
        P = _maps(x[b] @ w.T, prob.seq_len, prob.n_heads, prob.n_kv_heads, prob.head_dim)
        Q = _maps(x[b] @ w_hat.T, prob.seq_len, prob.n_heads, prob.n_kv_heads, prob.head_dim)
        kb = rel_entr(P, Q).sum()
        assert abs(out["kl_seq"][b] - kb) <= 1e-9 * kb
        total += kb
    assert total > 0
    assert abs(out["kl"] - total) <= 1e-9 * total
    assert abs(out["kl_batchmean"] - total / prob.batch) <= 1e-9 * total
    # no quantization: both maps are the same
    assert ref.loss_kl(x, w, prob, (0, 0, 0), s, z, None)["kl"] == 0.0


# ----------------------------------------------------------------------------- curvature
def _torch_block(x, w, prob):
    """A(X; W) of every sequence in torch fp64 (projection, causal GQA softmax attention)."""
    hq, hkv, dh = prob.n_heads, prob.n_kv_heads, prob.head_dim
    T = x.shape[1]
    y = x @ w.T
    q = y[..., :hq * dh].reshape(-1, T, hq, dh)
    k = y[..., hq * dh:(hq + hkv) * dh].reshape(-1, T, hkv, dh).repeat_interleave(hq // hkv, dim=2)
    v = y[..., (hq + hkv) * dh:].reshape(-1, T, hkv, dh).repeat_interleave(hq // hkv, dim=2)
    s = torch.einsum("bihc,bjhc->bhij", q, k) / math.sqrt(dh)
    mask = torch.triu(torch.ones(T, T, dtype=torch.bool), 1)
    p = torch.softmax(s.masked_fill(mask, float("-inf")), dim=-1)
    return torch.einsum("bhij,bjhc->bihc", p, v).reshape(x.shape[0], T, hq * dh)


def test_curvature_is_the_gauss_newton_form():
    """eq. gn at the float point: v^T H v = 2 ||J_A v||^2 (lambda_KL = 0).  The oracle's symmetric
    difference against the exact directional derivative J_A v from torch forward-mode autodiff
    in fp64, per unit (the probe restricted to W_Q, W_K, W_V rows) and pooled."""
    prob = _tiny_problem(B=2, T=12, d=32, hq=4, hkv=2, dh=8, g=16)
    x, w = _tiny_inputs(prob, seed=9, wstd=0.2)
    r = np.random.default_rng(4)
    probes = r.choice([-1.0, 1.0], size=(3, prob.rows, prob.d_model))
    eps = 1e-4
    got = ref.curvature_fd(x, w, prob, probes, eps, None)
    xt, wt = torch.from_numpy(x), torch.from_numpy(w)
    units = list(prob.matrix_rows()) + [(0, prob.rows)]
    for p in range(len(probes)):
        for u, (r0, r1) in enumerate(units):
            v = torch.zeros_like(wt)
            v[r0:r1] = torch.from_numpy(probes[p][r0:r1])
            _, jv = torch.func.jvp(lambda ww: _torch_block(xt, ww, prob), (wt,), (v,))
            want = 2.0 * float((jv ** 2).sum())
            assert want > 0
            assert abs(got[p, u] - want) <= 1e-6 * want, (p, u, got[p, u], want)
    # quadratic in the probe: 2v gives four times the form
    twice = ref.curvature_fd(x, w, prob, 2.0 * probes[:1], eps, None)
    np.testing.assert_allclose(twice[0], 4.0 * got[0], rtol=1e-6)


def _torch_logits_and_output(x, w, prob):
    """Masked logits z = Q K^T / sqrt(d_head) (-1e9 above the diagonal) and A(X; W) in torch fp64,
    with the half-split rotary embedding on Q and K when the problem has one (written from its
    definition: pair (j, j + d_head/2) of each head turns by t theta^(-2j/d_head))."""
    hq, hkv, dh = prob.n_heads, prob.n_kv_heads, prob.head_dim
    T = x.shape[1]
    y = x @ w.T
    q = y[..., :hq * dh].reshape(-1, T, hq, dh)
    k = y[..., hq * dh:(hq + hkv) * dh].reshape(-1, T, hkv, dh)
    v = y[..., (hq + hkv) * dh:].reshape(-1, T, hkv, dh)
    if prob.rope_theta:
        j = torch.arange(dh // 2, dtype=torch.float64)
        ang = torch.arange(T, dtype=torch.float64)[:, None] * prob.rope_theta ** (-2.0 * j / dh)
        c, sn = torch.cos(ang)[None, :, None, :], torch.sin(ang)[None, :, None, :]

        def turn(t):
            a, b = t[..., :dh // 2], t[..., dh // 2:]
            return torch.cat([a * c - b * sn, b * c + a * sn], dim=-1)
        q, k = turn(q), turn(k)
    k = k.repeat_interleave(hq // hkv, dim=2)
    v = v.repeat_interleave(hq // hkv, dim=2)
    z = torch.einsum("bihc,bjhc->bhij", q, k) / math.sqrt(dh)
    mask = torch.triu(torch.ones(T, T, dtype=torch.bool), 1)
    z = z.masked_fill(mask, -1e9)
    p = torch.softmax(z, dim=-1)
    a = torch.einsum("bhij,bjhc->bihc", p, v).reshape(x.shape[0], T, hq * dh)
    return z, a


@pytest.mark.parametrize("hq,hkv,rope,lam", [(4, 2, 0.0, 0.0), (4, 2, 0.0, 0.3), (4, 4, 0.0, 2.0),
                                             (4, 1, 10000.0, 0.3)])
def test_curvature_forms_are_hessian_vector_products_of_the_joint_loss(hq, hkv, rope, lam):
    """eq. gn at the float point against the paper's own construction: H v from two chained
    backward passes (torch.autograd.functional.hvp, fp64) of the joint loss written independently,
    ||A(w*) - A(w)||_F^2 + lambda sum_rows KL(P(w*) || Q(w)).  The per-unit terms are the partition
    t_u = sum over unit u's coordinates of v_j (H v)_j (their sum the pooled v^T H v), and the
    diagonal blocks h_uu = v_u^T H v_u with the probe restricted to unit u."""
    prob = ref.Problem(2, 11, 32, hq, hkv, 8, 16, ref.ASYM, rope)
    x, w = _tiny_inputs(prob, seed=21, wstd=0.25)
    r = np.random.default_rng(8)
    probes = r.choice([-1.0, 1.0], size=(2, prob.rows, prob.d_model))
    got = ref.curvature_gn(x, w, prob, probes, None, lam)
    xt, wt = torch.from_numpy(x), torch.from_numpy(w)
    with torch.no_grad():
        z0, a0 = _torch_logits_and_output(xt, wt, prob)
        logp0 = torch.log_softmax(z0, dim=-1)
        p0 = logp0.exp()

    def joint(ww):
        z, a = _torch_logits_and_output(xt, ww, prob)
        kl = (p0 * (logp0 - torch.log_softmax(z, dim=-1))).sum()
        return ((a0 - a) ** 2).sum() + lam * kl

    units = prob.matrix_rows()
    for pi in range(len(probes)):
        v = torch.from_numpy(probes[pi])
        hv = torch.autograd.functional.hvp(joint, wt, v)[1]
        want_t = [float((v[r0:r1] * hv[r0:r1]).sum()) for (r0, r1) in units]
        want_pooled = float((v * hv).sum())
        want_h = []
        for (r0, r1) in units:
            vu = torch.zeros_like(v)
            vu[r0:r1] = v[r0:r1]
            want_h.append(float((vu * torch.autograd.functional.hvp(joint, wt, vu)[1]).sum()))
        want = np.array(want_t + [want_pooled] + want_h)
        scale = np.abs(want).max()
        np.testing.assert_allclose(got[pi], want, rtol=1e-8, atol=1e-10 * scale)
        assert abs(sum(want_t) - want_pooled) <= 1e-10 * scale
        assert np.all(got[pi, 4:] > 0)


def test_hutchinson_mean_over_a_hadamard_probe_set_is_the_exact_trace():
    """Section "Sensitivity and allocation": Tr(H) ~ (1/n) sum_i v_i^T H v_i; the Appendix on
    per-unit traces: t_u is unbiased for Tr(H_uu) because E[v_j v_k] = delta_jk.  Over the rows of a
    Hadamard matrix (sign vectors with sum_i v_i v_i^T = n I exactly) the mean is the trace itself, so
    the oracle's curvature terms, averaged by eq. omega's table, must give the traces of the explicit
    Hessian of the joint loss written independently in torch (fp64, lambda_KL 0.3)."""
    from scipy.linalg import hadamard
    prob = ref.Problem(1, 6, 32, 2, 1, 8, 16, ref.ASYM, 0.0)
    n = prob.rows * prob.d_model
    assert n == 1024
    x, w = _tiny_inputs(prob, seed=31, wstd=0.3)
    lam = 0.3
    probes = hadamard(n).astype(np.float64).reshape(n, prob.rows, prob.d_model)
    curv = ref.curvature_gn(x, w, prob, probes, None, lam)
    werr = np.ones((1, 1, 3, 2))
    block = ref.omega_table(curv[None], werr, ref.TRACE_BLOCK)[:, 0]
    unit = ref.omega_table(curv[None], werr, ref.TRACE_UNIT)[:, 0]

    xt, wt = torch.from_numpy(x), torch.from_numpy(w)
    with torch.no_grad():
        z0, a0 = _torch_logits_and_output(xt, wt, prob)
        logp0 = torch.log_softmax(z0, dim=-1)
        p0 = logp0.exp()

    def joint(flat):
        z, a = _torch_logits_and_output(xt, flat.reshape(wt.shape), prob)
        kl = (p0 * (logp0 - torch.log_softmax(z, dim=-1))).sum()
        return ((a0 - a) ** 2).sum() + lam * kl

    diag = torch.diagonal(torch.autograd.functional.hessian(joint, wt.reshape(-1))).reshape(wt.shape).numpy()
    tr = diag.sum()
    tr_u = [diag[r0:r1].sum() for (r0, r1) in prob.matrix_rows()]
    assert tr > 0 and min(tr_u) > 0
    np.testing.assert_allclose(block, tr, rtol=1e-9)
    np.testing.assert_allclose(unit, tr_u, rtol=1e-9, atol=1e-12 * tr)


def test_omega_table_worked_example():
    """eq. omega on a two-block example worked by hand.  Block 0: pooled terms 3 and 5 (trace 4),
    partition terms (1, 2, 1) and (2, 2, 1) (traces 1.5, 2, 1); block 1: pooled 2 and 2 (trace 2),
    partition (1, 0.5, 0.5) twice.  Squared errors at widths (2, 16): 10 and 0 for every matrix of
    block 0; 3, 6, 9 and 0 for block 1.  C1 = trace x error; C2 multiplies block 0 by 2 (the errors
    of the first of two blocks pass through both) and block 1 by 1."""
    curv = np.zeros((2, 2, 7))
    curv[0, 0, :4] = [1, 2, 1, 3]
    curv[0, 1, :4] = [2, 2, 1, 5]
    curv[1, :, :4] = [1, 0.5, 0.5, 2]
    werr = np.zeros((2, 2, 3, 2))
    werr[0, 0, :, 0] = 10
    werr[1, 0, :, 0] = [3, 6, 9]
    werr[..., 1] = 99.0                                # sum w^2: not part of the score
    c1_block = ref.omega_table(curv, werr, ref.TRACE_BLOCK, ref.OMEGA_C1)
    np.testing.assert_array_equal(c1_block, [[40, 0], [40, 0], [40, 0], [6, 0], [12, 0], [18, 0]])
    c2_block = ref.omega_table(curv, werr, ref.TRACE_BLOCK, ref.OMEGA_C2)
    np.testing.assert_array_equal(c2_block, [[80, 0], [80, 0], [80, 0], [6, 0], [12, 0], [18, 0]])
    c1_unit = ref.omega_table(curv, werr, ref.TRACE_UNIT, ref.OMEGA_C1)
    np.testing.assert_array_equal(c1_unit, [[15, 0], [20, 0], [10, 0], [3, 0], [3, 0], [4.5, 0]])
    c2_unit = ref.omega_table(curv, werr, ref.TRACE_UNIT, ref.OMEGA_C2)
    np.testing.assert_array_equal(c2_unit, [[30, 0], [40, 0], [20, 0], [3, 0], [3, 0], [4.5, 0]])


def test_curvature_matches_finite_differences_of_the_pinned_losses():
    """The diagonal blocks and the pooled form equal the symmetric second difference of the joint
    loss built from the pinned forward routines (squared error and the KL of the attention maps)
    up to O(eps^2); the value unit is exact (the output is linear in W_V, the map does not move)."""
    prob = _tiny_problem(B=2, T=12, d=32, hq=4, hkv=2, dh=8, g=16)
    x, w = _tiny_inputs(prob, seed=5, wstd=0.2)
    probes = np.random.default_rng(6).choice([-1.0, 1.0], size=(2, prob.rows, prob.d_model))
    for lam in (0.0, 0.5):
        gn = ref.curvature_gn(x, w, prob, probes, None, lam)
        fd = ref.curvature_fd(x, w, prob, probes, 1e-4, None, lambda_kl=lam)
        np.testing.assert_allclose(gn[:, [4, 5, 6, 3]], fd, rtol=1e-6)
        np.testing.assert_allclose(gn[:, 6], fd[:, 2], rtol=1e-11)
    # quadratic in the probe, and the KL part is a positive semi-definite form (Fisher information)
    twice = ref.curvature_gn(x, w, prob, 2.0 * probes[:1], None, 0.5)
    np.testing.assert_allclose(twice[0], 4.0 * ref.curvature_gn(x, w, prob, probes[:1], None, 0.5)[0], rtol=1e-12)
    parts = ref.curvature_parts(x, w, prob, probes, None)
    fqq, fkk, fqk = parts[:, 6], parts[:, 7], parts[:, 8]
    assert np.all(fqq > 0) and np.all(fkk > 0) and np.all(fqk ** 2 <= fqq * fkk)


def _tiny_problem(B=2, T=16, d=64, hq=4, hkv=2, dh=16, g=32, scheme=ref.ASYM):
    return ref.Problem(B, T, d, hq, hkv, dh, g, scheme)


def _tiny_inputs(prob, seed=0, xstd=1.0, wstd=0.05):
    r = np.random.default_rng(seed)
    x = r.normal(0, xstd, (prob.batch, prob.seq_len, prob.d_model))
    w = r.normal(0, wstd, (prob.rows, prob.d_model))
    return x, w


def _block(prob, x, w, fmt=None):
    return np.stack([ref.block_forward(x[b], w, prob, fmt)[1] for b in range(len(x))])


def test_invariance_power_of_two_rescale_is_exact():
    """W_Q -> 2 W_Q, W_K -> W_K / 2 per head is the paper's d_head=1 rescaling toy
    made exact in floating point: the attention output is bitwise unchanged."""
    prob = _tiny_problem()
    x, w = _tiny_inputs(prob)
    (q0, q1), (k0, k1), _ = prob.matrix_rows()
    w2 = w.copy()
    w2[q0:q1] *= 2.0
    w2[k0:k1] *= 0.5
    assert np.array_equal(_block(prob, x, w), _block(prob, x, w2))


def test_invariance_orthogonal_rotation():
    """L is invariant under W_Q -> W_Q R, W_K -> W_K R^-T per head (Section 'Why one
    joint objective'); R is shared by the query heads of one key/value group."""
    prob = _tiny_problem(hq=4, hkv=2, dh=16)
    x, w = _tiny_inputs(prob)
    (q0, _), (k0, _), _ = prob.matrix_rows()
    dh, per = prob.head_dim, prob.n_heads // prob.n_kv_heads
    w2 = w.copy()
    r = np.random.default_rng(7)
    for g in range(prob.n_kv_heads):
        Rm, _ = np.linalg.qr(r.normal(size=(dh, dh)))
        for hh in range(per):
            h = g * per + hh
            rows = slice(q0 + h * dh, q0 + (h + 1) * dh)
            w2[rows] = Rm.T @ w[rows]            # Q_h -> Q_h R
        rows = slice(k0 + g * dh, k0 + (g + 1) * dh)
        w2[rows] = Rm.T @ w[rows]                # K -> K R (= K R^-T for orthogonal R)
    a1, a2 = _block(prob, x, w), _block(prob, x, w2)
    assert np.sum((a1 - a2) ** 2) < 1e-24 * np.sum(a1 ** 2)
    assert not np.array_equal(w, w2)


def test_gqa_equals_mha_with_repeated_kv_weights():
    prob = _tiny_problem(hq=4, hkv=2, dh=16)
    x, w = _tiny_inputs(prob)
    (q0, q1), (k0, k1), (v0, v1) = prob.matrix_rows()
    dh = prob.head_dim
    rep = lambda blk: np.concatenate([blk[(h // 2) * dh:(h // 2 + 1) * dh] for h in range(4)])
    w_mha = np.concatenate([w[q0:q1], rep(w[k0:k1]), rep(w[v0:v1])])
    mha = ref.Problem(prob.batch, prob.seq_len, prob.d_model, 4, 4, dh, prob.group_size)
    assert np.array_equal(_block(prob, x, w), _block(mha, x, w_mha))


# ----------------------------------------------------------------------------- loss
@pytest.mark.parametrize("fmt", [None, "f32", "bf16"])
def test_loss_is_zero_without_quantization(fmt):
    prob = _tiny_problem()
    x, w = _tiny_inputs(prob)
    w = ref.round_fmt(w, fmt) if fmt else w
    x = ref.round_fmt(x, fmt) if fmt else x
    s, z = ref.init_scales(w, prob, (4, 4, 4))
    out = ref.loss_fwd(x, w, prob, (0, 0, 0), s, z, fmt)
    assert out["sse"] == 0.0 and out["mse"] == 0.0 and out["sum_a2"] > 0


def test_loss_matches_brute_force_on_tiny_block():
    wl = inputs.WORKLOADS["tiny_fp32"]
    prob = ref.Problem(wl.batch, wl.seq_len, wl.d_model, wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.group_size)
    x = inputs.to_f64(inputs.make_x(wl))
    w = inputs.to_f64(inputs.make_w(wl))
    s, z = ref.init_scales(w, prob, (4, 4, 4))
    out = ref.loss_fwd(x, w, prob, (4, 4, 4), s, z, None)
    # brute force: nearest-grid-point codes, materialised attention
    w_hat = w.copy()
    for (r0, r1) in prob.matrix_rows():
        c = brute.nearest_codes(w[r0:r1], s[r0:r1], z[r0:r1], 4, prob.group_size)
        w_hat[r0:r1] = (c - np.repeat(z[r0:r1], prob.group_size, 1)) * np.repeat(s[r0:r1], prob.group_size, 1)
    want = brute.sse(x, w, w_hat, prob.n_heads, prob.n_kv_heads, prob.head_dim)
    assert out["sse"] > 0
    assert abs(out["sse"] - want) <= 1e-12 * want
    assert abs(out["mse"] - want / (wl.tokens * wl.n_heads * wl.head_dim)) <= 1e-12 * out["mse"]


def test_sweep_diagonal_equals_forward():
    prob = _tiny_problem()
    x, w = _tiny_inputs(prob)
    sb = {b: ref.init_scales(w, prob, (b, b, b)) for b in (2, 3, 4, 8)}
    triples = [(2, 3, 4), (4, 4, 4), (8, 2, 8), (3, 3, 3)]
    sw = ref.sweep(x, w, prob, triples, sb, "bf16")
    for t in triples:
        s = np.concatenate([sb[t[0]][0][:64], sb[t[1]][0][64:96], sb[t[2]][0][96:]])
        z = np.concatenate([sb[t[0]][1][:64], sb[t[1]][1][64:96], sb[t[2]][1][96:]])
        f = ref.loss_fwd(x, w, prob, t, s, z, "bf16")
        assert sw[t]["sse"] == f["sse"]


def test_loss_ratio_follows_grid_step_squared():
    """Small-noise regime: the loss is quadratic in the rounding residual whose variance is
    s^2/12, and min-max scales at 8 and 4 bits differ by exactly 15/255 -> L8/L4 ~ (15/255)^2."""
    prob = _tiny_problem(B=4, T=64, d=128, hq=4, hkv=2, dh=32, g=32)
    x, w = _tiny_inputs(prob, seed=3, wstd=0.1)
    L = {}
    for b in (8, 4, 3, 2):
        s, z = ref.init_scales(w, prob, (b, b, b))
        L[b] = ref.loss_fwd(x, w, prob, (b, b, b), s, z, None)["sse"]
    assert abs((L[8] / L[4]) / (15 / 255) ** 2 - 1) < 0.15
    assert 2.5 < L[3] / L[4] < 8 and 2.5 < L[2] / L[3] < 9


# ----------------------------------------------------------------------------- gradients
def test_gradient_is_zero_at_the_float_point():
    prob = _tiny_problem()
    x, w = _tiny_inputs(prob)
    s, z = ref.init_scales(w, prob, (3, 3, 3))
    out = ref.loss_bwd(x, w, prob, (0, 0, 0), s, z, None)
    assert out["mse"] == 0.0
    assert not np.any(out["dw"])


def test_weight_gradient_matches_finite_differences():
    prob = _tiny_problem(B=2, T=8, d=32, hq=2, hkv=1, dh=16, g=32)
    x, w = _tiny_inputs(prob, seed=5)
    s, z = ref.init_scales(w, prob, (3, 3, 3))
    out = ref.loss_bwd(x, w, prob, (3, 3, 3), s, z, None)
    w_eff = out["w_eff"]
    teacher = _block(prob, x, w)
    n = prob.batch * prob.seq_len * prob.n_out

    def mse(we):
        return np.sum((teacher - _block(prob, x, we)) ** 2) / n

    r = np.random.default_rng(11)
    idx = [(int(r.integers(prob.rows)), int(r.integers(prob.d_model))) for _ in range(40)]
    h = 1e-5
    for (i, j) in idx:
        wp, wm = w_eff.copy(), w_eff.copy()
        wp[i, j] += h
        wm[i, j] -= h
        fd = (mse(wp) - mse(wm)) / (2 * h)
        assert abs(fd - out["dw"][i, j]) <= 1e-6 * np.abs(out["dw"]).max()


def _torch_pipeline(x, w, prob, bits3, s, z):
    """STE + LSQ through torch autograd in float64: d w_hat/d w = 1, d w_hat/d s from
    differentiating (round_ste(clip(w/s + z, 0, 2^b-1)) - z) s."""
    xt = torch.tensor(x)
    wt = torch.tensor(w, requires_grad=True)
    st = torch.tensor(s, requires_grad=True)
    g = prob.group_size
    parts = []
    for (r0, r1), b in zip(prob.matrix_rows(), bits3):
        wm = wt[r0:r1]
        se = st[r0:r1].repeat_interleave(g, 1)
        ze = torch.tensor(z[r0:r1], dtype=torch.float64).repeat_interleave(g, 1)
        # LSQ's form: clip the unrounded v to the grid, then round straight-through,
        # so the branch is decided by v itself as in eq. lsq
        # (the quotient w/s is taken in fp32, as the quantizer computes it)
        v = wm.detach() / se
        v = v + (v.float().double() - v).detach()
        vc = torch.clamp(v + ze, 0, (1 << b) - 1)
        q = vc + (torch.round(vc) - vc).detach()
        parts.append((q - ze) * se + (wm - wm.detach()))
    w_hat = torch.cat(parts)
    wf = torch.tensor(w)

    def attn(weight):
        y = xt @ weight.T
        B, T, _ = y.shape
        hq, hk, dh = prob.n_heads, prob.n_kv_heads, prob.head_dim
        q = y[..., :hq * dh].reshape(B, T, hq, dh).transpose(1, 2)
        k = y[..., hq * dh:(hq + hk) * dh].reshape(B, T, hk, dh).transpose(1, 2)
        vv = y[..., (hq + hk) * dh:].reshape(B, T, hk, dh).transpose(1, 2)
        k = k.repeat_interleave(hq // hk, 1)
        vv = vv.repeat_interleave(hq // hk, 1)
        S = q @ k.transpose(-1, -2) / math.sqrt(dh)
        S = S.masked_fill(~torch.tril(torch.ones(T, T, dtype=torch.bool)), float("-inf"))
        return (torch.softmax(S, -1) @ vv).transpose(1, 2).reshape(B, T, hq * dh)

    mse = ((attn(wf) - attn(w_hat)) ** 2).mean()
    mse.backward()
    return mse.item(), wt.grad.numpy(), st.grad.numpy()


def test_fisher_is_the_squared_autograd_gradient_per_unit():
    """Appendix on Fisher-coupling: ||grad L||^2 per unit at a 2-bit round-to-nearest probe
    equals the squared norm of torch autograd's straight-through gradient over that unit's rows
    (an independent formulation); at the float point it is exactly 0."""
    prob = _tiny_problem(B=2, T=12, d=64, hq=4, hkv=2, dh=16, g=32)
    x, w = _tiny_inputs(prob, seed=13)
    s, z = ref.init_scales(w, prob, (2, 2, 2))
    got = ref.fisher(x, w, prob, (2, 2, 2), s, z, None)
    mse, dw, _ = _torch_pipeline(x, w, prob, (2, 2, 2), s, z)
    assert abs(got["mse"] - mse) <= 1e-12 * mse
    for u, (r0, r1) in enumerate(prob.matrix_rows()):
        want = float(np.sum(dw[r0:r1] ** 2))
        assert want > 0
        assert abs(got["sq"][u] - want) <= 1e-9 * want, (u, got["sq"][u], want)
    zero = ref.fisher(x, w, prob, (0, 0, 0), s, z, None)
    assert zero["sq"] == [0.0, 0.0, 0.0]
    # quantizing only W_V: W_Q and W_K still receive gradient (the output depends on them),
    # and the scores differ from the all-2-bit probe
    only_v = ref.fisher(x, w, prob, (0, 0, 2), s, z, None)
    assert all(v > 0 for v in only_v["sq"]) and only_v["sq"] != got["sq"]


def test_gradients_match_torch_autograd_ste_lsq():
    prob = _tiny_problem(B=2, T=12, d=64, hq=4, hkv=2, dh=16, g=32)
    x, w = _tiny_inputs(prob, seed=9)
    bits3 = (3, 4, 2)
    s, z = ref.init_scales(w, prob, bits3)
    out = ref.loss_bwd(x, w, prob, bits3, s, z, None, gammas=[1.0, 1.0, 1.0])
    mse, dw, ds = _torch_pipeline(x, w, prob, bits3, s, z)
    assert abs(out["mse"] - mse) <= 1e-12 * mse
    np.testing.assert_allclose(out["dw"], dw, rtol=1e-9, atol=1e-12 * np.abs(dw).max())
    # autograd differentiates -w/s in float64 where eq. lsq's phi uses the fp32 quotient v:
    # |delta phi| <= 2^-24 |v| per weight, which bounds the scale-gradient difference
    g = prob.group_size
    v = w / np.repeat(s, g, 1)
    bound = (np.abs(out["dw"]) * np.abs(v)).reshape(prob.rows, -1, g).sum(-1) * 2.0 ** -23
    assert np.all(np.abs(out["ds"] - ds) <= bound + 1e-13 * np.abs(ds).max())
    assert np.linalg.norm(out["ds"] - ds) <= 1e-4 * np.linalg.norm(ds)
    # gamma only multiplies
    out2 = ref.loss_bwd(x, w, prob, bits3, s, z, None, gammas=[0.5, 2.0, 3.0])
    (q0, q1), (k0, k1), (v0, v1) = prob.matrix_rows()
    np.testing.assert_allclose(out2["ds"][q0:q1], 0.5 * out["ds"][q0:q1], rtol=1e-15)
    np.testing.assert_allclose(out2["ds"][v0:v1], 3.0 * out["ds"][v0:v1], rtol=1e-15)


# ----------------------------------------------------------------------------- fine-tuning
def test_adam_update_matches_torch_adam():
    """The oracle's Adam step against torch.optim.Adam (an independent implementation), five
    steps on a quadratic with a changing rate."""
    r = np.random.default_rng(21)
    theta0 = r.normal(size=50)
    target = r.normal(size=50)
    p = torch.nn.Parameter(torch.tensor(theta0))
    opt = torch.optim.Adam([p], lr=0.1, betas=(0.9, 0.999), eps=1e-8)
    theta, m, v = theta0.copy(), np.zeros(50), np.zeros(50)
    for t in range(1, 6):
        lr = 0.1 / t
        for grp in opt.param_groups:
            grp["lr"] = lr
        g = 2.0 * (theta - target)
        p.grad = torch.tensor(2.0 * (p.detach().numpy() - target))
        opt.step()
        theta, m, v = ref.adam_update(theta, g, m, v, t, lr, 0.9, 0.999, 1e-8)
        np.testing.assert_allclose(theta, p.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_cosine_factor_matches_torch_schedule():
    """eq. lr's cosine annealing: the factor per step equals torch's CosineAnnealingLR (T_max =
    n_steps, eta_min = 0) at the step's index; 1 at the first step, decreasing."""
    n = 20
    p = torch.nn.Parameter(torch.zeros(1))
    opt = torch.optim.SGD([p], lr=1.0)
    sched = torch.optim.lr_scheduler.CosineAnnealingLR(opt, T_max=n, eta_min=0.0)
    f = []
    for t in range(1, n + 1):
        f.append(ref.cosine_factor(t, n))
        assert abs(f[-1] - opt.param_groups[0]["lr"]) < 1e-12, t
        opt.step()
        sched.step()
    assert f[0] == 1.0 and all(a > b for a, b in zip(f, f[1:])) and f[-1] > 0


def _ft_case(bits=(3, 3, 3), seed=31, held_is_train=False):
    prob = _tiny_problem(B=2, T=12, d=64, hq=4, hkv=2, dh=16, g=32)
    x, w = _tiny_inputs(prob, seed=seed, wstd=0.1)
    xh = x.copy() if held_is_train else _tiny_inputs(prob, seed=seed + 1)[0]
    s, z = ref.init_scales(w, prob, bits)
    teach = {b: ref.block_forward(x[b], w, prob, None)[1] for b in range(2)}
    teach_h = {b: ref.block_forward(xh[b], w, prob, None)[1] for b in range(2)}
    return prob, x, w, xh, s, z, teach, teach_h


def test_finetune_without_movement_returns_the_start():
    """alpha = 0: nothing moves, the start is kept (best step 0), no code flips, every training
    loss equals the start's training loss."""
    prob, x, w, xh, s, z, teach, teach_h = _ft_case()
    out = ref.ste_finetune(x, teach, xh, teach_h, w, prob, (3, 3, 3), s, z, None, 6, 3, 0.0, 0.0,
                           [1.0, 1.0, 1.0])
    st = out["stats"]
    assert st[2] == 0 and list(st[3:6]) == [0.0, 0.0, 0.0]
    assert np.all(st[6:12] == st[6]) and st[0] == st[1]
    assert np.array_equal(out["w_master"], ref.round_fmt(w, "f32")) and np.array_equal(out["scale"], s)


def test_finetune_lowers_the_loss_and_keeps_the_best_checkpoint():
    """With the paper's rates the training loss falls, codes flip, and the gate returns the best
    evaluated checkpoint: its held-out loss (recomputed) is the logged minimum, below the start.
    The held-out batch is the training batch here, so that fine-tuning can beat the start (on
    an independent batch this tiny block overfits: see the next test)."""
    prob, x, w, xh, s, z, teach, teach_h = _ft_case(held_is_train=True)
    g = [ref.default_gamma(3, prob.group_size)] * 3
    n, every = 30, 5
    out = ref.ste_finetune(x, teach, xh, teach_h, w, prob, (3, 3, 3), s, z, None, n, every, 0.05, 0.02, g)
    st = out["stats"]
    train, evals = st[6:6 + n], st[6 + n:]
    assert len(evals) == 6
    assert train[-1] < 0.8 * train[0]
    assert 0 < st[1] < st[0] and st[1] == evals.min()
    assert st[2] == every * (1 + int(np.argmin(evals)))
    assert all(0 < f < 0.5 for f in st[3:6])
    import dataclasses
    held = dataclasses.replace(prob, batch=2)
    again = ref.loss_fwd(xh, out["w"], held, (3, 3, 3), out["scale"], z, None, a_ref=teach_h)["mse"]
    assert again == st[1]
    # the flip rate is the brute-force fraction of differing codes
    c0 = ref.student_weight(ref.round_fmt(w, "f32"), prob, (3, 3, 3), out["scale"], z, None)[1]
    c1 = ref.student_weight(out["w"], prob, (3, 3, 3), out["scale"], z, None)[1]
    (q0, q1) = prob.matrix_rows()[0]
    assert st[3] == np.count_nonzero(c0[q0:q1] != c1[q0:q1]) / c0[q0:q1].size


def test_finetune_gate_keeps_the_start_when_no_checkpoint_beats_it():
    """On an independent held-out batch the tiny block overfits (training loss falls, every
    held-out score is above the start's): the commit gate returns the start, bit for bit."""
    prob, x, w, xh, s, z, teach, teach_h = _ft_case()
    g = [ref.default_gamma(3, prob.group_size)] * 3
    out = ref.ste_finetune(x, teach, xh, teach_h, w, prob, (3, 3, 3), s, z, None, 30, 5, 0.05, 0.02, g)
    st = out["stats"]
    assert st[6 + 29] < st[6] and np.all(st[36:] > st[0])
    assert st[2] == 0 and st[1] == st[0] and list(st[3:6]) == [0.0, 0.0, 0.0]
    assert np.array_equal(out["w_master"], ref.round_fmt(w, "f32")) and np.array_equal(out["scale"], s)


# ----------------------------------------------------------------------------- RoPE
def _rope_problem(theta=10000.0):
    return ref.Problem(2, 24, 64, 4, 2, 16, 32, ref.ASYM, theta)


def test_rope_is_complex_multiplication_by_the_position_phase():
    """RoPE on each half-split pair (a_j, b_j) is multiplication of a_j + i b_j by
    exp(i t theta^(-2j/d_head)) (numpy complex arithmetic, an independent formulation); position
    0 is the identity and the value columns pass through."""
    prob = _rope_problem()
    r = np.random.default_rng(3)
    y = r.normal(size=(24, prob.rows))
    got = ref.rope_qk(y, prob)
    dh = prob.head_dim
    t = np.arange(24)[:, None]
    for h in range(prob.n_heads + prob.n_kv_heads):
        a, b = y[:, h * dh:h * dh + dh // 2], y[:, h * dh + dh // 2:(h + 1) * dh]
        j = np.arange(dh // 2)[None, :]
        z = (a + 1j * b) * np.exp(1j * t * 10000.0 ** (-2.0 * j / dh))
        np.testing.assert_allclose(got[:, h * dh:h * dh + dh // 2], z.real, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(got[:, h * dh + dh // 2:(h + 1) * dh], z.imag, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(got[0], y[0])
    v0 = (prob.n_heads + prob.n_kv_heads) * dh
    np.testing.assert_array_equal(got[:, v0:], y[:, v0:])
    np.testing.assert_allclose(ref.rope_qk(got, prob, inverse=True), y, rtol=1e-12, atol=1e-12)


def test_rope_scores_depend_only_on_the_relative_position():
    """The defining property of rotary embeddings: a query at position m and a key at n give a
    score that depends on m - n only."""
    prob = _rope_problem()
    r = np.random.default_rng(5)
    q, k = r.normal(size=prob.head_dim), r.normal(size=prob.head_dim)
    y = np.zeros((24, prob.rows))
    y[:, :prob.head_dim] = q                                    # query head 0 at every position
    y[:, prob.n_heads * prob.head_dim:][:, :prob.head_dim] = k  # key head 0 at every position
    yr = ref.rope_qk(y, prob)
    qr, kr = yr[:, :prob.head_dim], yr[:, prob.n_heads * prob.head_dim:][:, :prob.head_dim]
    for m, n, shift in ((5, 2, 7), (20, 20, -13), (9, 0, 11)):
        assert abs(qr[m] @ kr[n] - qr[m + shift] @ kr[n + shift]) < 1e-12


def test_rope_loss_zero_unquantized_and_gradient_matches_finite_differences():
    prob = ref.Problem(2, 8, 32, 2, 1, 16, 32, ref.ASYM, 10000.0)
    x, w = _tiny_inputs(prob, seed=5)
    s, z = ref.init_scales(w, prob, (3, 3, 3))
    assert ref.loss_bwd(x, w, prob, (0, 0, 0), s, z, None)["mse"] == 0.0
    out = ref.loss_bwd(x, w, prob, (3, 3, 3), s, z, None)
    w_eff = out["w_eff"]
    teacher = _block(prob, x, w)
    n = prob.batch * prob.seq_len * prob.n_out
    # the rotation changes the loss (positions matter) ...
    plain = ref.Problem(*[getattr(prob, f) for f in ("batch", "seq_len", "d_model", "n_heads", "n_kv_heads",
                                                      "head_dim", "group_size", "scheme")])
    assert abs(ref.loss_bwd(x, w, plain, (3, 3, 3), s, z, None)["mse"] - out["mse"]) > 1e-6 * out["mse"]

    def mse(we):
        return np.sum((teacher - _block(prob, x, we)) ** 2) / n

    r = np.random.default_rng(11)
    h = 1e-5
    for _ in range(30):
        i, j = int(r.integers(prob.rows)), int(r.integers(prob.d_model))
        wp, wm = w_eff.copy(), w_eff.copy()
        wp[i, j] += h
        wm[i, j] -= h
        fd = (mse(wp) - mse(wm)) / (2 * h)
        assert abs(fd - out["dw"][i, j]) <= 1e-6 * np.abs(out["dw"]).max()


# ----------------------------------------------------------------------------- KL gradient
def test_kl_gradient_matches_finite_differences_of_the_kl_forward():
    """attention_kl_grad against central differences of the KL forward (attention_kl, itself
    pinned against scipy's rel_entr) in the student's query and key columns; value columns get
    nothing."""
    prob = _tiny_problem(B=1, T=10, d=32, hq=4, hkv=2, dh=16, g=32)
    r = np.random.default_rng(17)
    yt = r.normal(size=(10, prob.rows))
    ys = yt + 0.3 * r.normal(size=yt.shape)
    coef = 0.7
    got = ref.attention_kl_grad(yt, ys, 4, 2, 16, coef)
    kv_end = (prob.n_heads + prob.n_kv_heads) * prob.head_dim
    assert not np.any(got[:, kv_end:])
    h = 1e-6
    for _ in range(40):
        i, j = int(r.integers(10)), int(r.integers(kv_end))
        yp, ym = ys.copy(), ys.copy()
        yp[i, j] += h
        ym[i, j] -= h
        fd = coef * (ref.attention_kl(yt, yp, 4, 2, 16)[1] - ref.attention_kl(yt, ym, 4, 2, 16)[1]) / (2 * h)
        assert abs(fd - got[i, j]) <= 1e-6 * np.abs(got).max() + 1e-9, (i, j, fd, got[i, j])


def test_joint_objective_gradient_matches_finite_differences():
    """loss_bwd with lambda_kl: the weight gradient of mse + lambda kl / B against central
    differences of that objective in the effective weights; lambda = 0 is the plain gradient."""
    prob = _tiny_problem(B=2, T=8, d=32, hq=2, hkv=1, dh=16, g=32)
    x, w = _tiny_inputs(prob, seed=7)
    s, z = ref.init_scales(w, prob, (3, 3, 3))
    lam = 0.5
    out = ref.loss_bwd(x, w, prob, (3, 3, 3), s, z, None, lambda_kl=lam)
    plain = ref.loss_bwd(x, w, prob, (3, 3, 3), s, z, None)
    assert not np.allclose(out["dw"], plain["dw"])
    w_eff = out["w_eff"]
    teacher = _block(prob, x, w)
    yts = [ref.block_forward(x[b], w, prob, None)[0] for b in range(2)]
    n = prob.batch * prob.seq_len * prob.n_out

    def objective(we):
        mse = np.sum((teacher - _block(prob, x, we)) ** 2) / n
        kl = sum(ref.attention_kl(yts[b], ref.block_forward(x[b], we, prob, None)[0], 2, 1, 16)[1] for b in range(2))
        return mse + lam * kl / prob.batch

    r = np.random.default_rng(12)
    h = 1e-5
    for _ in range(30):
        i, j = int(r.integers(prob.rows)), int(r.integers(prob.d_model))
        wp, wm = w_eff.copy(), w_eff.copy()
        wp[i, j] += h
        wm[i, j] -= h
        fd = (objective(wp) - objective(wm)) / (2 * h)
        assert abs(fd - out["dw"][i, j]) <= 1e-6 * np.abs(out["dw"]).max()


def test_finetune_with_the_kl_term():
    """lambda_KL > 0: the logged training objective is mse + lambda kl / B (recomputed here from
    the pinned forward pieces at the start), the trajectory differs from the squared error
    alone, and the gate still returns the lowest held-out objective."""
    prob, x, w, xh, s, z, teach, teach_h = _ft_case(held_is_train=True)
    w = ref.round_fmt(w, "f32")               # the fp32 latent start is the float block itself
    teach = teach_h = {b: ref.block_forward(x[b], w, prob, None)[1] for b in range(2)}
    s, z = ref.init_scales(w, prob, (3, 3, 3))
    g = [ref.default_gamma(3, prob.group_size)] * 3
    lam = 0.1
    out = ref.ste_finetune(x, teach, xh, teach_h, w, prob, (3, 3, 3), s, z, None, 10, 5, 0.05, 0.02, g,
                           lambda_kl=lam)
    plain = ref.ste_finetune(x, teach, xh, teach_h, w, prob, (3, 3, 3), s, z, None, 10, 5, 0.05, 0.02, g)
    st = out["stats"]
    wf = ref.round_fmt(w, "f32")
    mse0 = ref.loss_fwd(x, wf, prob, (3, 3, 3), s, z, None, a_ref=teach)["mse"]
    kl0 = ref.loss_kl(x, wf, prob, (3, 3, 3), s, z, None)["kl_batchmean"]
    assert kl0 > 0 and abs(st[6] - (mse0 + lam * kl0)) <= 1e-12 * st[6]
    assert st[0] == st[6]                      # held-out batch = training batch, same start
    assert not np.array_equal(st[6:16], plain["stats"][6:16])
    assert st[1] == min(st[0], st[16:].min()) and st[1] < st[0]
