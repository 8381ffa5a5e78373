"""Build libjab.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

Every translation unit is compiled with
  -ffp-contract=off                      products and sums rounded as written
                                         (fused multiply-adds are explicit)
  -fhip-fp32-correctly-rounded-divide-sqrt   IEEE division for the quantizer
  -Xclang -target-feature -Xclang -packed-fp32-ops   no packed fp32 VALU ops
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libjab.so")
SOURCES = ["quant.hip", "gemm.hip", "attn_fwd.hip", "attn_fwd_nv2.hip", "attn_fwd_fast_multi.hip", "attn_kl.hip", "attn_bwd.hip",
           "attn_bwd_mfma.hip", "attn_jvp.hip", "reduce.hip", "ste.hip", "rope.hip", "alloc.cpp", "api.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-ffp-contract=off",
         "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-fast-math",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include")]
# per-source additions: the attention kernels keep their MFMA accumulators in the
# architectural registers, which leaves the accumulation registers for operands
_VGPR_MFMA = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
EXTRA = {"attn_fwd.hip": _VGPR_MFMA, "attn_fwd_nv2.hip": _VGPR_MFMA, "attn_kl.hip": _VGPR_MFMA}


def _compile(src: str) -> str:
    obj = os.path.join(OUT_DIR, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = [HIPCC] + FLAGS + EXTRA.get(src, []) + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-6000:]}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-4000:]}")
    os.replace(tmp, LIB)
    if verbose:
        print(LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
