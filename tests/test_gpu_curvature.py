"""GPU parity of the curvature scores (Method, eq. gn with lambda_KL = 0; jab_curvature) against
the oracle's difference quotient (``oracle.reference.curvature_fd``) in contract mode: the same
perturbed weights RN_dtype(RN_fp32(w +- eps v)), the same symmetric quotient.

Tolerance: each quotient is a sum of two squared-error losses of a perturbed block against the
teacher, so it inherits the loss's precision: for the 16-bit dtypes the device rounds the softmax
probabilities to the dtype for the value product (2^-9 relative in each output, not emulated by
the oracle) while the perturbation moves the outputs by a few tens of per cent (eps is a quarter of
the weights' RMS), so about 1e-2 of the quotient; fp32, 1e-4.
"""
import numpy as np
import pytest
import torch

from oracle import reference as ref
from paper_2609_34866_amd import inputs, jab

from gpu_helpers import device_inputs, oracle_problem, small

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "f16": 3e-2, "bf16": 3e-2}

SHAPES = [
    # (T, d, Hq, Hkv, dh, g, dtype)
    (33, 128, 4, 4, 16, 32, "bf16"),
    (40, 128, 4, 2, 16, 32, "f32"),
    (64, 256, 8, 2, 64, 64, "f16"),
    (96, 256, 8, 2, 128, 64, "bf16"),
]


def _wl(T, d, hq, hkv, dh, g, dtype, batch=2):
    return small(batch=batch, seq_len=T, d_model=d, n_heads=hq, n_kv_heads=hkv, head_dim=dh,
                 group_size=g, dtype=dtype)


def _probes(n, rows, cols, seed):
    g = torch.Generator().manual_seed(seed)
    return (torch.randint(0, 2, (n, rows, cols), generator=g, dtype=torch.int8) * 2 - 1)


@pytest.mark.parametrize("shape", SHAPES)
def test_curvature_matches_oracle(shape):
    wl = _wl(*shape)
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    probes = _probes(2, wl.rows, wl.d_model, seed=17)
    eps = float(np.float32(0.25 * float(w.float().pow(2).mean().sqrt())))
    a = jab.attn_ref(p, x, w)
    got = jab.curvature(p, x, w, a, probes.cuda(), eps).cpu().numpy()
    prob = oracle_problem(wl)
    want = ref.curvature_fd(inputs.to_f64(x.cpu()), inputs.to_f64(w.cpu()), prob, probes.numpy(), eps, wl.dtype)
    assert np.all(want > 0)
    err = np.abs(got - want) / want
    assert err.max() < TOL[wl.dtype], (err.max(), got, want)


def test_curvature_quadratic_in_the_probe_and_deterministic():
    """Halving eps leaves the quotient nearly unchanged (O(eps^2) truncation, a few 1e-2 at this
    eps); repeated calls are bitwise identical."""
    wl = _wl(64, 256, 8, 2, 64, 64, "f32")
    x, w = device_inputs(wl)
    p = jab.problem_of(wl)
    probes = _probes(1, wl.rows, wl.d_model, seed=3).cuda()
    rms = float(w.float().pow(2).mean().sqrt())
    a = jab.attn_ref(p, x, w)
    o1 = jab.curvature(p, x, w, a, probes, 0.1 * rms).cpu().numpy()
    o2 = jab.curvature(p, x, w, a, probes, 0.1 * rms).cpu().numpy()
    o3 = jab.curvature(p, x, w, a, probes, 0.05 * rms).cpu().numpy()
    assert np.array_equal(o1, o2)
    assert np.all(np.abs(o3 - o1) / o3 < 0.1)
