"""Benchmark of the JAB forward loss at the Mistral-7B attention-block shape.

One step = one jab_loss_fwd call over the whole batch (quantize W_Q/W_K/W_V,
fused QKV projection, causal GQA attention with the fused squared-error
epilogue, deterministic reduction), inputs resident in HBM, teacher output
cached beforehand (computed once per (X, W) and reported separately).

Prints one JSON line: tokens/s, the roofline of the dominant kernel (its
algorithmic flops per launch over its average HIP-event-timed duration, against
the MI355X dense bf16 peak) and the fp64 CPU oracle timed on a bounded sample.
The timed steps run as a caller runs them; the per-kernel durations come from the
same number of steps run right after with the library's per-launch HIP events on
the stream the kernels run on (those events hold each next kernel back by ~8 us).

usage: python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload mistral_bf16]
                       [--no-cpu-baseline] [--calib-copy-mib N]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}   # MI355X dense matrix-core peaks
HBM_GBS = 8000.0
METRIC = "JAB loss evals: calibration tokens/sec at Mistral-7B attn shape; % bf16 MFMA peak"
METRIC_OP = {"fwd": METRIC,
             "sweep": "JAB sweep: calibration triple-tokens/sec (one loss per bit-width triple) at Mistral-7B attn shape",
             "bwd": "JAB STE step (loss, dW, d_scale): calibration tokens/sec at Mistral-7B attn shape",
             "kl": "JAB joint objective (squared error + KL attention-map term): calibration tokens/sec at Mistral-7B attn shape",
             "bwd_kl": "JAB STE step of the joint objective (squared error + KL attention-map term, lambda 0.1): calibration tokens/sec at Mistral-7B attn shape",
             "fisher": "JAB Fisher-coupling scores (squared STE gradient norm per unit at a 2-bit probe): calibration tokens/sec at Mistral-7B attn shape",
             "ft": "JAB joint STE fine-tuning (Adam steps with held-out commit gate): calibration tokens/sec at Mistral-7B attn shape",
             "quant": "JAB quantizer (codes, fp32 fake-quantized weights, eps^W sums) over W_Q/W_K/W_V of 32 Mistral-7B layers: weights/sec",
             "curv": "JAB Gauss-Newton curvature of eq. gn with its KL term (exact Hutchinson terms per Rademacher probe): calibration token-probes/sec at Mistral-7B attn shape"}


def algorithmic_flops(wl):
    """Flops the method needs per step, by kernel family: the projection of Q and K, the
    projection of V (written transposed), and only the unmasked causal products
    (T(T+1)/2 pairs per head) of the attention.  Sweep: each distinct projection once
    (one per candidate bit-width), the scores once per (b_Q, b_K) and the value product
    once per triple.  STE step: the forward, the attention backward (scores recomputed,
    dP, dV, dK, dQ: 10 d_head flops per pair) and the weight-gradient GEMM.  Joint objective:
    the forward and the KL term's two score products (teacher and student) per pair.
    Curvature: one projection of the weights per call and one of each probe (the tangent X v^T);
    per probe one forward-mode attention pass with three score products (Q K^T, Qd K^T, Q Kd^T) and
    four value products (P V, (P zQ) V, (P zK) V, P Vd)."""
    M = wl.batch * wl.seq_len
    qk = 2.0 * M * (wl.n_heads + wl.n_kv_heads) * wl.head_dim * wl.d_model
    vt = 2.0 * M * wl.n_kv_heads * wl.head_dim * wl.d_model
    pairs = wl.seq_len * (wl.seq_len + 1) / 2.0
    half = 2.0 * wl.batch * wl.n_heads * pairs * wl.head_dim          # one of QK^T or PV
    if wl.op == "sweep":
        nb = len(inputs_sweep_bits())
        nqk = len({(t[0], t[1]) for t in wl.bits})
        return {"gemm": nb * qk, "gemm_vt": nb * vt, "attn": (nqk + len(wl.bits)) * half}
    out = {"gemm": qk, "gemm_vt": vt, "attn": 2.0 * half}
    if wl.op in ("kl", "bwd_kl"):
        out["kl"] = 2.0 * half                                          # teacher and student scores
    if wl.op == "curv":
        n = wl.probes
        out = {"gemm": (1 + n) * qk, "gemm_vt": (1 + n) * vt, "attn": n * 7 * half}
    if wl.op in ("bwd", "fisher", "ft", "bwd_kl"):
        out["attn_bwd"] = (6.0 if wl.op == "bwd_kl" else 5.0) * half   # KL: the teacher's scores too
        out["dw_gemm"] = 2.0 * M * wl.rows * wl.d_model
    if wl.op == "ft":                                                   # Adam steps + held-out scores
        n_eval = -(-wl.probes // 10)
        fwd = {"gemm": qk, "gemm_vt": vt, "attn": 2.0 * half}
        if wl.lambda_kl > 0:                                            # the KL term: forward and backward
            out["kl"] = 2.0 * half
            out["attn_bwd"] = 6.0 * half
            fwd["kl"] = 2.0 * half
        out = {k: wl.probes * v + n_eval * fwd.get(k, 0.0) for k, v in out.items()}
    return out


def inputs_sweep_bits():
    from paper_2609_34866_amd import inputs
    return inputs.SWEEP_BITS


def timed_steps(step, steps):
    """Times `steps` calls of `step` between two events on the current stream, as a caller runs
    them (no per-kernel events: each recorded event holds the next kernel back by about 8 us),
    then `steps` more with the library's per-kernel-family events for the kernel durations.
    Returns (ms per step, wall ms of the first set, {family: (ms, launches)} of the second)."""
    import torch

    from paper_2609_34866_amd import jab

    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    ms = e0.elapsed_time(e1) / steps
    jab.timing_enable(True)
    jab.timing_read()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    kern = jab.timing_read()
    jab.timing_enable(False)
    return ms, wall_ms, kern


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary, or None
    when the kernel's source has changed since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hbm_traffic_mistral_bf16.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        if not line.startswith("traffic-record:"):
            continue
        rec = json.loads(line.split(":", 1)[1])
        if rec["kernel"] != kernel:
            continue
        src = os.path.join(ROOT, "paper_2609_34866_amd", "csrc", rec["source"])
        if hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] != rec["sha256_16"]:
            return None
        return rec["bytes"]
    return None


def cpu_baseline(wl, bits, budget_s):
    """The fp64 oracle on a bounded sample of the same workload: whole sequences, student
    path (quantize, project, attend, squared error) with the teacher precomputed."""
    import numpy as np

    from oracle import reference as ref
    from paper_2609_34866_amd import inputs

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    prob = ref.Problem(wl.batch, wl.seq_len, wl.d_model, wl.n_heads, wl.n_kv_heads, wl.head_dim,
                       wl.group_size)
    w = inputs.to_f64(inputs.make_w(wl))
    s, z = ref.init_scales(w, prob, bits)
    done, t_total, seqs = 0, 0.0, []
    while done < wl.batch:
        x = inputs.to_f64(inputs.make_x(wl, [done]))
        teacher = ref.attn_ref(x, w, prob, wl.dtype)
        t0 = time.perf_counter()
        ref.loss_fwd(x, w, prob, bits, s, z, wl.dtype, a_ref={done: teacher[0]}, seqs=[done])
        t_total += time.perf_counter() - t0
        seqs.append(done)
        done += 1
        if t_total * (len(seqs) + 1) / len(seqs) > budget_s:
            break
    tokens = len(seqs) * wl.seq_len
    return {"value": tokens / t_total, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(seqs)} of {wl.batch} sequences x {wl.seq_len} tokens, student path with "
                      f"teacher precomputed, fp64 contract mode ({wl.dtype}), {t_total:.1f} s"}


def bench_quant(wl, bits, dev, args):
    """The quantizer alone (jab_quantize: codes, fp32 w_hat, eps^W sums) on a stacked weight batch.
    Algorithmic bytes per weight: the bf16 weight in, its code (1 B) and fp32 w_hat (4 B) out, and
    per group of g weights its fp32 scale and 8-bit zero-point in; bound by HBM bandwidth."""
    import torch

    from paper_2609_34866_amd import inputs, jab

    print(f"[bench] workload {wl.name}: generating weights", file=sys.stderr, flush=True)
    w = inputs.make_w(wl).to(dev)
    p = jab.problem_of(wl)
    scale, zero = jab.quant_init(p, w, bits)
    n = wl.rows * wl.d_model
    out = {"codes": torch.empty((wl.rows, wl.d_model), dtype=torch.uint8, device=dev),
           "w_hat": torch.empty((wl.rows, wl.d_model), dtype=torch.float32, device=dev),
           "werr": torch.empty((3, 2), dtype=torch.float64, device=dev)}
    ws = jab.workspace(p, jab.OP_QUANTIZE)

    def step():
        jab.quantize(p, w, bits, scale, zero, out=out, ws=ws)

    for _ in range(args.warmup):
        step()
    ms, wall_ms, kern = timed_steps(step, args.steps)
    kernels = {k: {"avg_ms": tms / c, "launches_per_step": c / args.steps, "ms_per_step": tms / args.steps}
               for k, (tms, c) in kern.items() if c}
    bytes_launch = n * (2 + 1 + 4) + (n // wl.group_size) * (4 + 1)
    gbs = bytes_launch / (kernels["quant"]["avg_ms"] * 1e-3) / 1e9
    kernels["quant"]["gb_s"] = gbs
    rec = {"metric": METRIC_OP["quant"], "value": n / (ms * 1e-3), "unit": "weights/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
           "data": "synthetic (seeded Gaussian weights)",
           "config": {"workload": wl.name, "rows": wl.rows, "d_model": wl.d_model, "layers": 32,
                      "group_size": wl.group_size, "bits": list(bits), "scheme": "asym", "parallelism": "single GPU"},
           "roofline": {"bound": "hbm", "kernel": "quant", "achieved": gbs, "peak": HBM_GBS, "unit": "GB/s",
                        "frac": gbs / HBM_GBS, "traffic": None},
           "algorithmic_bytes_per_launch": bytes_launch, "kernels": kernels, "wall_ms_timed_region": wall_ms,
           "cpu_baseline": None}
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mistral_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="only run 3 plain device copies of this many MiB (calibrates the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes": n, "copies": 3}), flush=True)
        return

    from paper_2609_34866_amd import inputs, jab

    wl = inputs.WORKLOADS[args.workload]
    bits = wl.bits[0]
    dev = torch.device("cuda:0")
    if wl.op == "quant":
        bench_quant(wl, bits, dev, args)
        return
    print(f"[bench] workload {wl.name}: generating inputs", file=sys.stderr, flush=True)
    x = inputs.make_x(wl, threads=16).to(dev)
    w = inputs.make_w(wl).to(dev)
    p = jab.problem_of(wl)
    scale, zero = jab.quant_init(p, w, bits)
    ws = jab.workspace(p, {"fwd": jab.OP_FWD, "sweep": jab.OP_SWEEP, "bwd": jab.OP_BWD, "kl": jab.OP_FWD_KL,
                           "curv": jab.OP_CURVATURE, "fisher": jab.OP_FISHER, "bwd_kl": jab.OP_BWD,
                           "ft": jab.OP_STE}[wl.op],
                       len(inputs.SWEEP_BITS) if wl.op == "sweep" else 0)
    ws_ref = jab.workspace(p, jab.OP_REF)
    use_kl_cache = wl.op in ("kl", "bwd_kl") or (wl.op == "ft" and wl.lambda_kl > 0)
    a_ref = None if use_kl_cache else torch.empty((wl.batch, wl.seq_len, wl.n_heads * wl.head_dim),
                                                    dtype=torch.float32, device=dev)
    out = torch.empty((2 if wl.op == "kl" else 1) * (3 + wl.batch), dtype=torch.float64, device=dev)

    # teacher (cached once per (X, W); timed on its own)
    def teacher():
        if use_kl_cache:
            return jab.attn_ref_kl(p, x, w, ws=ws_ref)
        jab.attn_ref(p, x, w, ws=ws_ref, out=a_ref)
        return None

    teacher()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    kl_cache = teacher()
    torch.cuda.synchronize()
    teacher_ms = (time.perf_counter() - t0) * 1e3
    if kl_cache is not None:
        a_ref = kl_cache[0]
    del ws_ref

    if wl.op == "sweep":
        sb = [jab.quant_init(p, w, (b, b, b)) for b in inputs.SWEEP_BITS]

        def step():
            jab.loss_sweep(p, x, w, inputs.SWEEP_BITS, [s_ for s_, _ in sb], [z_ for _, z_ in sb], wl.bits, a_ref,
                           ws=ws, per_seq=False)
    elif wl.op == "bwd":
        gammas = jab.lsq_gscale(bits, wl.group_size)

        def step():
            jab.loss_bwd(p, x, w, bits, scale, zero, a_ref, gammas, ws=ws)
    elif wl.op == "ft":
        # held-out batch: the next wl.batch sequences of the same generator; each timed run restarts
        # from the same latent weights and scales (two device copies, ~0.05 ms)
        x_held = inputs.make_x(wl, seqs=range(wl.batch, 2 * wl.batch), threads=16).to(dev)
        kl_kw = {}
        if wl.lambda_kl > 0:
            a_held, qk_held, lse_held = jab.attn_ref_kl(p, x_held, w)
            kl_kw = dict(lambda_kl=wl.lambda_kl, kl_cache=(kl_cache[1], kl_cache[2]), kl_cache_held=(qk_held, lse_held))
        else:
            a_held = jab.attn_ref(p, x_held, w)
        wm0, s0 = w.float(), scale.clone()
        wm, sc = torch.empty_like(wm0), torch.empty_like(s0)
        w_cur = torch.empty_like(w)
        ft_stats = []

        def step():
            wm.copy_(wm0)
            sc.copy_(s0)
            ft_stats[:] = [jab.ste_finetune(p, x, a_ref, x_held, a_held, bits, wm, sc, zero, n_steps=wl.probes,
                                            eval_every=10, ws=ws, w=w_cur, **kl_kw)[1]]
    elif wl.op == "bwd_kl":
        gammas = jab.lsq_gscale(bits, wl.group_size)

        def step():
            jab.loss_bwd_kl(p, x, w, bits, scale, zero, a_ref, kl_cache[1], kl_cache[2], gammas, 0.1, ws=ws)
    elif wl.op == "fisher":
        fisher_out = torch.empty(4, dtype=torch.float64, device=dev)

        def step():
            jab.fisher(p, x, w, bits, scale, zero, a_ref, ws=ws, out=fisher_out)
    elif wl.op == "curv":
        probes = inputs.make_probes(wl, wl.probes, seed=1).to(dev)
        # the paper's lambda_KL = 0.1 on the objective as implemented (mse + lambda kl / B) is
        # lambda N / B in the printed form the curvature takes
        lam = wl.lambda_kl * wl.seq_len * wl.n_heads * wl.head_dim
        curv_out = torch.empty((wl.probes, 7), dtype=torch.float64, device=dev)

        def step():
            jab.curvature(p, x, w, probes, lam, ws=ws, out=curv_out)
    elif wl.op == "kl":
        def step():
            jab.loss_fwd_kl(p, x, w, bits, scale, zero, a_ref, kl_cache[1], kl_cache[2], ws=ws, out=out)
    else:
        def step():
            jab.loss_fwd(p, x, w, bits, scale, zero, a_ref, ws=ws, out=out)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ms, wall_ms, kern = timed_steps(step, args.steps)
    print(f"[bench] {ms:.3f} ms/step", file=sys.stderr, flush=True)

    loss = out.cpu().numpy() if wl.op in ("fwd", "kl") else None
    flops = algorithmic_flops(wl)
    step_flops = sum(flops.values())
    peak = PEAK_TFLOPS[wl.dtype]
    kernels = {}
    for k, (tms, n) in kern.items():
        if n:
            kernels[k] = {"avg_ms": tms / n, "launches_per_step": n / args.steps, "ms_per_step": tms / args.steps}
    for k, f in flops.items():
        if k in kernels:
            # algorithmic flops of one launch: the family's share of a step over its launches
            kernels[k]["tflops"] = f / kernels[k]["launches_per_step"] / (kernels[k]["avg_ms"] * 1e-3) / 1e12
            kernels[k]["frac_peak"] = kernels[k]["tflops"] / peak
    # dominant kernel: the largest share of the step among the matrix-core kernels
    dom = max(flops, key=lambda k: kernels.get(k, {"ms_per_step": 0.0})["ms_per_step"])
    achieved = kernels[dom]["tflops"]
    tokens = wl.batch * wl.seq_len * (len(wl.bits) if wl.op == "sweep" else wl.probes if wl.op == "curv"
                                      else wl.probes if wl.op == "ft" else 1)
    rec = {
        "metric": METRIC_OP[wl.op],
        "value": tokens / (ms * 1e-3),
        "unit": "triple-tokens/s" if wl.op == "sweep" else "token-probes/s" if wl.op == "curv" else "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded RMS-normalised activations with outlier channels, Gaussian weights)",
        "config": {"workload": wl.name, "batch": wl.batch, "seq_len": wl.seq_len, "d_model": wl.d_model,
                   "n_heads": wl.n_heads, "n_kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim,
                   "group_size": wl.group_size, "bits": list(bits), "scheme": "asym",
                   "parallelism": "single GPU", **({"probes": wl.probes} if wl.op == "curv" else {}),
                   **({"adam_steps": wl.probes, "eval_every": 10, "held_out_batch": wl.batch, "lambda_kl": wl.lambda_kl}
                      if wl.op == "ft" else {})},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak,
                     "traffic": measured_traffic(dom) if wl.name == "mistral_bf16" else None},
        "step_frac_of_peak": step_flops / (ms * 1e-3) / 1e12 / peak,
        "algorithmic_tflop_per_step": step_flops / 1e12,
        "kernels": kernels,
        "teacher_ms": teacher_ms,
        "wall_ms_timed_region": wall_ms,
        "loss": None if loss is None else dict(
            {"sse": float(loss[0]), "mse": float(loss[1]), "eps_A": float((loss[0] / loss[2]) ** 0.5)},
            **({"kl_batchmean": float(loss[4 + wl.batch])} if wl.op == "kl" else {})),
        "cpu_baseline": None,
    }
    del x, a_ref, ws, kl_cache
    torch.cuda.empty_cache()
    if wl.op == "ft":
        fs = ft_stats[0].cpu().numpy()
        n = wl.probes
        rec["finetune"] = {"held_mse_start": float(fs[0]), "held_mse_best": float(fs[1]), "best_step": int(fs[2]),
                           "flip_rate_qkv": [float(v) for v in fs[3:6]], "train_mse_first": float(fs[6]),
                           "train_mse_last": float(fs[5 + n])}
    if not args.no_cpu_baseline and wl.op == "fwd":
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(wl, bits, args.cpu_budget)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
