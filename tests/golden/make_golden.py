"""Write the oracle's values for sampled sequences of the full-size workloads.

Runs only the fp64 oracle (``oracle/``) on the seeded inputs of
``paper_2609_34866_amd.inputs``; nothing here calls the GPU library.  The GPU
parity tests regenerate the same inputs from the same seeds, run the whole
workload on the device, and compare the per-sequence values stored here.

Mode: "contract" in the workload's storage dtype (W_hat = RN_dtype(RN_fp32((q-z) s)),
Q/K/V rounded to the dtype, everything else float64).  With --exact, the loss workloads'
entries also get the same sums in exact mode (float64 throughout: W_hat = (q-z) s, the
teacher, projection and attention unrounded), "exact_sse_seq" beside each "sse_seq": the
deviation of the precision contract from the exact loss.

usage: python tests/golden/make_golden.py [workload ...]
       python tests/golden/make_golden.py --exact [workload ...]
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import reference as ref  # noqa: E402
from paper_2609_34866_amd import inputs  # noqa: E402

OUT = os.path.join(HERE, "oracle_samples.json")

# sequences sampled per workload (first and last of the batch); the STE step's
# gradient sums over the whole batch, so it runs in full and stores sampled rows
SAMPLES = {"gpt2_fp16": [0, 31], "mistral_bf16": [0, 127], "mistral_sweep": [0], "mistral_ste": None,
           "mistral_kl": [0, 127], "mistral_curv": [0]}
CURV_PROBES = 2          # Rademacher probes (inputs.make_probes, seed 0) of the stored curvature sums
# gradient rows stored for the STE step: one row of each of W_Q, W_K, W_V
STE_ROWS = [100, 4096 + 517, 5120 + 1000]
STE_COLS = 512           # leading columns of each stored dW row


def oracle_problem(wl):
    return ref.Problem(wl.batch, wl.seq_len, wl.d_model, wl.n_heads, wl.n_kv_heads, wl.head_dim,
                       wl.group_size, ref.SYM if wl.symmetric else ref.ASYM)


def run(name):
    wl = inputs.WORKLOADS[name]
    prob = oracle_problem(wl)
    seqs = SAMPLES[name]
    if seqs is None:
        return run_full_backward(wl, prob)
    x = inputs.to_f64(inputs.make_x(wl, seqs))
    w = inputs.to_f64(inputs.make_w(wl))
    fmt = wl.dtype
    t0 = time.time()
    entry = {"seqs": seqs, "mode": f"contract-{fmt}", "results": []}
    if wl.op == "curv":
        probes = inputs.make_probes(wl, CURV_PROBES, seed=0).numpy()
        parts = ref.curvature_parts(x, w, prob, probes, fmt, seqs=seqs)
        entry["results"].append({"probes": CURV_PROBES, "probe_seed": 0, "parts": parts.tolist()})
    elif wl.op == "kl":
        for bits in wl.bits:
            s, z = ref.init_scales(w, prob, bits)
            out = ref.loss_kl(x, w, prob, bits, s, z, fmt, seqs=seqs)
            entry["results"].append({"bits": list(bits), "kl_seq": [out["kl_seq"][b] for b in seqs]})
    elif wl.op == "sweep":
        sb = {b: ref.init_scales(w, prob, (b, b, b)) for b in inputs.SWEEP_BITS}
        sw = ref.sweep(x, w, prob, list(wl.bits), sb, fmt, seqs=seqs)
        for t in wl.bits:
            entry["results"].append({"bits": list(t), "sse_seq": [sw[t]["sse_seq"][b] for b in seqs]})
    else:
        teacher = ref.attn_ref(x, w, prob, fmt, seqs=range(len(seqs)))
        for bits in wl.bits:
            s, z = ref.init_scales(w, prob, bits)
            out = ref.loss_fwd(x, w, prob, bits, s, z, fmt,
                               a_ref={b: teacher[i] for i, b in enumerate(seqs)}, seqs=seqs)
            entry["results"].append({"bits": list(bits), "sse_seq": [out["sse_seq"][b] for b in seqs],
                                     "sum_a2_seq": [float(np.sum(teacher[i] ** 2)) for i in range(len(seqs))]})
    entry["oracle_seconds"] = time.time() - t0
    return entry


EXACT = ["gpt2_fp16", "mistral_bf16", "mistral_sweep"]


def add_exact(name, entry):
    """Exact-mode sums (fmt None) for the stored sequences and bit-widths of a loss entry."""
    wl = inputs.WORKLOADS[name]
    prob = oracle_problem(wl)
    seqs = entry["seqs"]
    x = inputs.to_f64(inputs.make_x(wl, seqs))
    w = inputs.to_f64(inputs.make_w(wl))
    t0 = time.time()
    if wl.op == "sweep":
        sb = {b: ref.init_scales(w, prob, (b, b, b)) for b in inputs.SWEEP_BITS}
        triples = [tuple(r["bits"]) for r in entry["results"]]
        sw = ref.sweep(x, w, prob, triples, sb, None, seqs=seqs)
        for r, t in zip(entry["results"], triples):
            r["exact_sse_seq"] = [sw[t]["sse_seq"][b] for b in seqs]
    else:
        teacher = ref.attn_ref(x, w, prob, None, seqs=range(len(seqs)))
        for r in entry["results"]:
            bits = tuple(r["bits"])
            s, z = ref.init_scales(w, prob, bits)
            out = ref.loss_fwd(x, w, prob, bits, s, z, None,
                               a_ref={b: teacher[i] for i, b in enumerate(seqs)}, seqs=seqs)
            r["exact_sse_seq"] = [out["sse_seq"][b] for b in seqs]
    entry["exact_oracle_seconds"] = time.time() - t0


def run_full_backward(wl, prob):
    t0 = time.time()
    bits = wl.bits[0]
    x = inputs.to_f64(inputs.make_x(wl))
    w = inputs.to_f64(inputs.make_w(wl))
    s, z = ref.init_scales(w, prob, bits)
    gammas = [ref.default_gamma(b, wl.group_size, prob.scheme) for b in bits]
    out = ref.loss_bwd(x, w, prob, bits, s, z, wl.dtype, gammas=gammas)
    entry = {"mode": f"contract-{wl.dtype}", "bits": list(bits), "gammas": gammas, "mse": out["mse"],
             "sse": out["sse"], "rows": [], "cols": STE_COLS}
    for (r0, r1), name in zip(prob.matrix_rows(), "QKV"):
        entry[f"norm_dw_{name}"] = float(np.linalg.norm(out["dw"][r0:r1]))
        entry[f"norm_ds_{name}"] = float(np.linalg.norm(out["ds"][r0:r1]))
    for r in STE_ROWS:
        entry["rows"].append({"row": r, "dw": out["dw"][r, :STE_COLS].tolist(), "ds": out["ds"][r].tolist()})
    entry["oracle_seconds"] = time.time() - t0
    return entry


def main(names):
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    for n in names:
        print(f"[golden] {n} ...", flush=True)
        data[n] = run(n)
        print(f"[golden] {n} done in {data[n]['oracle_seconds']:.1f} s", flush=True)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1)


def main_exact(names):
    data = json.load(open(OUT))
    for n in names:
        print(f"[golden] exact {n} ...", flush=True)
        add_exact(n, data[n])
        print(f"[golden] exact {n} done in {data[n]['exact_oracle_seconds']:.1f} s", flush=True)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1)


if __name__ == "__main__":
    if sys.argv[1:2] == ["--exact"]:
        main_exact(sys.argv[2:] or EXACT)
    else:
        main(sys.argv[1:] or list(SAMPLES))
