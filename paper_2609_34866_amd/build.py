"""Build libjab.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

Every translation unit is compiled with
  -ffp-contract=off                      products and sums rounded as written
                                         (fused multiply-adds are explicit)
  -fhip-fp32-correctly-rounded-divide-sqrt   IEEE division for the quantizer
  -Xclang -target-feature -Xclang -packed-fp32-ops   no packed fp32 VALU ops
"""
import os
import re
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


# Translation units with matrix products written as inline asm (attn_fwd_fast.h's mma_v): their
# device assembly is generated and checked for the hazards the compiler does not see.
ASM_CHECKED = ["attn_fwd_fast_multi.hip"]
MFMA_WINDOW = 19        # wait states between a product and any other access to its result


def _device_asm(src: str) -> str:
    out = os.path.join(OUT_DIR, os.path.basename(src) + ".s")
    cmd = [HIPCC] + FLAGS + EXTRA.get(src, []) + ["--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stderr[-6000:]}")
    return out


def _vgprs(text: str) -> set:
    regs = set()
    for lo, hi in re.findall(r"\bv\[(\d+):(\d+)\]", text):
        regs |= set(range(int(lo), int(hi) + 1))
    regs |= {int(r) for r in re.findall(r"\bv(\d+)\b", text)}
    return regs


def mfma_result_hazards(asm: str, window: int = MFMA_WINDOW) -> list:
    """Accesses to the result of a v_mfma whose destination is architectural registers (v[...])
    within `window` wait states of it: an instruction counts one wait state, s_nop N counts N + 1.
    The next product of a chain (destination and accumulator input both exactly the same
    registers) ends the window; a label or a branch inside the window counts as an access (the
    code that follows is not known).  Returns (product, offending line) pairs."""
    lines = []
    for raw in asm.splitlines():
        t = raw.split(";")[0].strip()
        if not t or (t.startswith(".") and not t.endswith(":")):
            continue
        lines.append(t)
    bad = []
    for i, t in enumerate(lines):
        m = re.match(r"v_mfma\S*\s+v\[(\d+):(\d+)\]", t)
        if not m:
            continue
        dst = set(range(int(m.group(1)), int(m.group(2)) + 1))
        dtext = f"v[{m.group(1)}:{m.group(2)}]"
        ws = 0
        for u in lines[i + 1:]:
            if ws >= window:
                break
            n = re.match(r"s_nop\s+(\d+)", u)
            if n:
                ws += int(n.group(1)) + 1
                continue
            if u.endswith(":") or u.startswith("s_branch") or u.startswith("s_cbranch") or u.startswith("s_setpc"):
                bad.append((t, u))
                break
            ops = [o.strip() for o in u.split(None, 1)[1].split(",")] if " " in u else []
            if u.startswith("v_mfma") and ops and ops[0] == dtext and ops[-1] == dtext:
                break                                    # the chain's next product
            if _vgprs(" ".join(ops)) & dst:
                bad.append((t, u))
                break
            ws += 1
    return bad


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES) + len(ASM_CHECKED))) as ex:
        asm_jobs = [ex.submit(_device_asm, s) for s in ASM_CHECKED]
        objs = list(ex.map(_compile, SOURCES))
        for src, job in zip(ASM_CHECKED, asm_jobs):
            bad = mfma_result_hazards(open(job.result()).read())
            if bad:
                raise RuntimeError(f"{src}: {len(bad)} access(es) to a matrix product's result within "
                                   f"{MFMA_WINDOW} wait states, first: {bad[0]}")
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
