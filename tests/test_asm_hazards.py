"""The build's check of the inline-asm matrix products (attn_fwd_fast.h's mma_v): no instruction may
access a product's architectural-register result within the hazard window, except the next product
of its chain.  The checker against hand-written cases, and the generated assembly of the last build."""
import os
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(os.path.dirname(HERE), "paper_2609_34866_amd"))
import build  # noqa: E402

P = "v_mfma_f32_32x32x16_bf16 v[16:31], v[60:63], v[64:67], v[16:31]"
DRAIN = ["s_nop 7", "s_nop 7", "s_nop 2"]


def test_copy_of_result_right_after_product_is_flagged():
    asm = "\n".join([P, "s_nop 0", "v_mov_b64_e32 v[158:159], v[30:31]"])
    assert len(build.mfma_result_hazards(asm)) == 1


def test_write_into_result_is_flagged():
    asm = "\n".join([P, "v_exp_f32_e32 v20, v2"])
    assert len(build.mfma_result_hazards(asm)) == 1


def test_chain_and_drain_pass():
    asm = "\n".join([P, "v_exp_f32_e32 v1, v2", "ds_read_b128 v[4:7], v85 offset:4096", P, *DRAIN,
                     "v_mov_b64_e32 v[158:159], v[30:31]"])
    assert build.mfma_result_hazards(asm) == []


def test_short_drain_is_flagged():
    asm = "\n".join([P, "s_nop 7", "s_nop 7", "v_fma_f32 v0, s80, v31, v1"])
    assert len(build.mfma_result_hazards(asm)) == 1


def test_branch_inside_window_is_flagged():
    asm = "\n".join([P, "s_cbranch_scc0 .LBB0_3"])
    assert len(build.mfma_result_hazards(asm)) == 1


def test_accumulation_register_products_are_not_checked():
    asm = "\n".join(["v_mfma_f32_32x32x16_bf16 a[0:15], v[60:63], v[64:67], a[0:15]", "v_accvgpr_read_b32 v0, a15"])
    assert build.mfma_result_hazards(asm) == []


def test_last_build_is_clean():
    found = False
    for src in build.ASM_CHECKED:
        path = os.path.join(build.OUT_DIR, os.path.basename(src) + ".s")
        if not os.path.exists(path):
            continue
        found = True
        text = open(path).read()
        assert "v_mfma_f32_32x32x16_bf16 v[" in text       # the asm products are there
        assert build.mfma_result_hazards(text) == []
    if not found:
        pytest.skip("no generated assembly (build() not run here)")
