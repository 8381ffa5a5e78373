"""Shared helpers of the GPU parity tests: seeded inputs on the device and the
matching oracle problem.  Inputs come from ``paper_2609_34866_amd.inputs`` (draws
only); expected values come from ``oracle`` alone."""
import numpy as np
import torch

from oracle import reference as ref
from paper_2609_34866_amd import inputs, jab

FMT = {"f32": "f32", "f16": "f16", "bf16": "bf16"}


def oracle_problem(wl):
    return ref.Problem(wl.batch, wl.seq_len, wl.d_model, wl.n_heads, wl.n_kv_heads, wl.head_dim,
                       wl.group_size, ref.SYM if wl.symmetric else ref.ASYM, wl.rope_theta)


def small(name="tiny", **kw):
    """A small workload for shape sweeps."""
    base = dict(name=name, batch=2, seq_len=33, d_model=128, n_heads=4, n_kv_heads=4, head_dim=16,
                group_size=32, dtype="bf16", bits=((4, 4, 4),), op="fwd", x_recipe="rms_outlier",
                outlier_frac=0.02, w_std=0.05)
    base.update(kw)
    return inputs.Workload(**base)


def device_inputs(wl, seqs=None):
    x = inputs.make_x(wl, seqs).cuda()
    w = inputs.make_w(wl).cuda()
    return x, w


def rel(a, b):
    return abs(a - b) / max(abs(b), 1e-300)


def ulp_diff_16bit(a: torch.Tensor, b: torch.Tensor) -> torch.Tensor:
    """Distance in units in the last place between two tensors of the same 16-bit dtype."""
    ia = a.view(torch.int16).to(torch.int32)
    ib = b.view(torch.int16).to(torch.int32)
    # map sign-magnitude to a monotone integer line
    ia = torch.where(ia < 0, -(ia & 0x7FFF), ia)
    ib = torch.where(ib < 0, -(ib & 0x7FFF), ib)
    return (ia - ib).abs()
