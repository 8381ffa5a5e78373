"""The precision contract's deviation from the exact loss (eq. joint_loss's squared-error term),
from the oracle alone: tests/golden/make_golden.py stores, for the sampled sequences of the
GPT-2 fp16, Mistral bf16 and Mistral sweep workloads, the per-sequence sums in contract mode
(W_hat = RN_dtype(RN_fp32((q - z) s)), the projection rounded to the dtype) and in exact mode
(float64 throughout).  The GPU is held to the contract; this is how far the contract itself is
from the exact value.

Bars: 1e-2 for the single-triple workloads and for every sweep triple of widths at most 4; the
triples with 8-bit matrices are reported (the dtype rounding of Q, K, V is then as large as the
quantization error: 0.28 at (8, 8, 8)); with one 8-bit matrix they stay below 1e-2, with two below
2e-2 (worst (8, 8, 4), 1.5e-2).

CPU only: reads stored values."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "oracle_samples.json")


def _entries():
    if not os.path.exists(GOLDEN):
        pytest.skip("golden oracle samples not generated")
    data = json.load(open(GOLDEN))
    out = {}
    for name in ("gpt2_fp16", "mistral_bf16", "mistral_sweep"):
        e = data.get(name)
        if e is None or "exact_sse_seq" not in e["results"][0]:
            pytest.skip(f"no exact-mode values for {name}")
        out[name] = [(tuple(r["bits"]), np.abs(np.array(r["sse_seq"]) - np.array(r["exact_sse_seq"])) /
                      np.array(r["exact_sse_seq"])) for r in e["results"]]
    return out


def test_contract_deviation_of_the_single_triple_workloads():
    dev = _entries()
    for name in ("gpt2_fp16", "mistral_bf16"):
        for bits, d in dev[name]:
            assert np.all(d < 1e-2), (name, bits, d)
            assert np.all(d > 0)          # the two modes are distinct computations


def test_contract_deviation_of_the_sweep_triples():
    rows = _entries()["mistral_sweep"]
    assert len(rows) == 64
    by_eights = {}
    for bits, d in rows:
        by_eights.setdefault(sum(b == 8 for b in bits), []).append((float(d.max()), bits))
    assert max(by_eights[0])[0] < 1e-2            # every width at most 4
    assert max(by_eights[1])[0] < 1e-2            # one 8-bit matrix
    assert max(by_eights[2])[0] < 2e-2            # two 8-bit matrices
    assert by_eights[3][0][0] > 0.1               # (8, 8, 8): rounding as large as the quantization error
