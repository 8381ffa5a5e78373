"""GPU quantizer parity: scales, zero-points and codes bit-exact against the oracle."""
import numpy as np
import pytest
import torch

from oracle import reference as ref
from paper_2609_34866_amd import inputs, jab

from gpu_helpers import oracle_problem, small

pytestmark = pytest.mark.gpu


def _check_quant(wl, bits, w=None):
    p = jab.problem_of(wl)
    prob = oracle_problem(wl)
    if w is None:
        w = inputs.make_w(wl)
    wd = w.cuda()
    scale, zero = jab.quant_init(p, wd, bits)
    res = jab.quantize(p, wd, bits, scale, zero)
    torch.cuda.synchronize()
    w64 = inputs.to_f64(w)
    s, z = ref.init_scales(w64, prob, bits)
    assert np.array_equal(scale.cpu().numpy().astype(np.float64), s)
    if z is not None:
        assert np.array_equal(zero.cpu().numpy().astype(np.int32), z)
    _, codes, _ = ref.student_weight(w64, prob, bits, s, z, None)
    w_eff, _, _ = ref.student_weight(w64, prob, bits, s, z, "f32")
    got_codes = res["codes"].cpu().numpy().astype(np.int32)
    for (r0, r1), b in zip(prob.matrix_rows(), bits):
        if b:
            assert np.array_equal(got_codes[r0:r1], codes[r0:r1]), f"codes differ (bits {b})"
    assert np.array_equal(res["w_hat"].cpu().numpy().astype(np.float64), w_eff)
    # eps^W sums (metric M3)
    werr = res["werr"].cpu().numpy()
    for m, ((r0, r1), b) in enumerate(zip(prob.matrix_rows(), bits)):
        e = float(np.sum((w_eff[r0:r1] - w64[r0:r1]) ** 2))
        n = float(np.sum(w64[r0:r1] ** 2))
        assert abs(werr[m, 1] - n) <= 1e-12 * n
        assert abs(werr[m, 0] - e) <= 1e-12 * max(e, 1e-300) + (0.0 if b else 0.0)


@pytest.mark.parametrize("name", ["tiny_fp32", "gpt2_fp16", "mistral_bf16"])
@pytest.mark.parametrize("bits", [(2, 3, 4), (8, 8, 8), (3, 3, 3), (0, 4, 0)])
def test_quantizer_bit_exact_on_workload_weights(name, bits):
    _check_quant(inputs.WORKLOADS[name], bits)


@pytest.mark.parametrize("group", [32, 64, 128])
def test_quantizer_symmetric(group):
    wl = small(d_model=256, group_size=group, symmetric=True, dtype="f16")
    _check_quant(wl, (2, 4, 8))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_quantizer_exact_ties_and_degenerate_groups(dtype):
    """Weights on exact half-steps of a power-of-two grid (ties to even), groups of zeros
    (scale 1, zero-point 0) and all-positive groups (zero-point 0)."""
    wl = small(d_model=128, group_size=32, dtype=dtype)
    p = jab.problem_of(wl)
    R, d, g = p.rows, wl.d_model, wl.group_size
    rng = np.random.default_rng(5)
    w = rng.normal(0, 0.05, (R, d)).astype(np.float32)
    s = 2.0 ** -6
    for r in range(0, R, 3):                      # 4-bit grid: lo = -7 s, hi = 8 s -> s exact
        grp = np.array([-7, 8] + list(rng.integers(-7, 8, g - 2) + 0.5)) * s
        w[r, :g] = grp
    w[1, 32:64] = 0.0
    w[2, 64:96] = np.abs(w[2, 64:96])
    wt = torch.from_numpy(w).to(wl.torch_dtype)
    _check_quant(wl, (4, 4, 4), w=wt)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_quantizer_bit_exact_for_caller_scales(dtype):
    """Scales a caller may pass (fine-tuned, far from the min-max init): random magnitudes
    2^-70 .. 2^70, on both sides of the range where the device forms the quotient from one
    reciprocal per group, and scales that put a weight's quotient on a half-integer (a tie) or one
    ulp from it, with random zero-points.  Codes and w_hat bit-exact against the oracle."""
    wl = small(d_model=256, group_size=32, dtype=dtype)
    p = jab.problem_of(wl)
    prob = oracle_problem(wl)
    w = inputs.make_w(wl)
    w64 = inputs.to_f64(w)
    R, g = wl.rows, wl.group_size
    ng = wl.d_model // g
    rng = np.random.default_rng(11)
    s = (rng.uniform(1.0, 2.0, (R, ng)) * np.exp2(rng.integers(-70, 71, (R, ng)))).astype(np.float32)
    bits = (4, 8, 3)
    row_bits = np.concatenate([np.full(r1 - r0, b) for (r0, r1), b in zip(prob.matrix_rows(), bits)])
    for r in range(R):
        levels = 2 ** int(row_bits[r]) - 1
        for j in range(0, ng, 2):                       # every other group: a quotient at k + 1/2
            wv = abs(float(w64[r, j * g + (r % g)]))
            if wv == 0.0:
                continue
            t = np.float32(wv / (int(rng.integers(0, levels // 2 + 1)) + 0.5))
            s[r, j] = [np.nextafter(t, np.float32(0)), t, np.nextafter(t, np.float32(np.inf))][(r + j) % 3]
    z = np.concatenate([rng.integers(0, 2 ** b, (r1 - r0, ng)) for (r0, r1), b in zip(prob.matrix_rows(), bits)])
    wd = w.cuda()
    res = jab.quantize(p, wd, bits, torch.from_numpy(s).cuda(), torch.from_numpy(z.astype(np.uint8)).cuda())
    torch.cuda.synchronize()
    s64, z32 = s.astype(np.float64), z.astype(np.int32)
    _, codes, _ = ref.student_weight(w64, prob, bits, s64, z32, None)
    w_eff, _, _ = ref.student_weight(w64, prob, bits, s64, z32, "f32")
    assert np.array_equal(res["codes"].cpu().numpy().astype(np.int32), codes)
    assert np.array_equal(res["w_hat"].cpu().numpy().astype(np.float64), w_eff)
