"""Host-side logic of bench.py: the LM head's launch plan and algorithmic
bytes, the counter-figure digest, and the refusal of several GPUs."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import L2_7B_BS1, L3_70B_BS32, L3_8B_BS1, L3_8B_BS16, L3_8B_TREE  # noqa: E402


def test_lm_workgroups_follow_the_launch_plan():
    # one row: 4 tiles per wave when 1024 such waves remain, else 1; 2-32
    # rows: 8 tiles per wave
    assert bench.lm_workgroups(L3_8B_BS1, 1) == 8016 // 16
    assert bench.lm_workgroups(L2_7B_BS1, 1) == 2000 // 4
    assert bench.lm_workgroups(L3_8B_BS16, 16) == (8016 // 8 + 3) // 4
    assert bench.lm_workgroups(L3_8B_TREE, 32) == (8016 // 8 + 3) // 4
    assert bench.lm_workgroups(L3_70B_BS32, 32) == (8016 // 8 + 3) // 4


def test_lm_head_bytes():
    # weights + the row's hi/lo planes + (max, sum, value, id) per workgroup
    assert bench.lm_head_bytes(L3_8B_BS1, 1) == 128256 * 4096 * 2 + 4096 * 4 + 501 * 16
    # top-1 on 16 rows: partials of 251 workgroups
    assert bench.lm_head_bytes(L3_8B_BS16, 16) == 128256 * 4096 * 2 + 16 * 4096 * 4 + 16 * 251 * 16
    # tree levels (top-8 on 32 rows): the launch stores the fp32 logits rows
    assert bench.lm_topk_pass(L3_8B_TREE, 32) and not bench.lm_topk_pass(L3_8B_BS16, 16)
    assert bench.lm_head_bytes(L3_8B_TREE, 32) == 128256 * 4096 * 2 + 32 * 4096 * 4 + 32 * 128256 * 4


def test_streamed_bytes_with_the_embedding_table():
    # batch 1: the FC streams its feature columns plus one fp32 table row
    full = bench.step_weight_bytes(L3_8B_BS1, 1)
    assert bench.uses_embed_table(L3_8B_BS1, 1)
    assert bench.step_streamed_bytes(L3_8B_BS1, 1, 1) == full - 2 * 4096 * 4096 + 4096 * 4
    # batched rows too: one table row per row
    assert bench.uses_embed_table(L3_8B_BS16, 16)
    assert (bench.step_streamed_bytes(L3_8B_BS16, 1, 16)
            == bench.step_weight_bytes(L3_8B_BS16, 1) - 2 * 4096 * 4096 + 16 * 4096 * 4)
    # fp32 contexts keep the whole FC
    from synth import TINY_F32
    assert not bench.uses_embed_table(TINY_F32, 1)


def _digest_with(edit):
    base = os.path.join(ROOT, "paper_2602_01762_amd", "csrc")

    def read(f):
        with open(os.path.join(base, f)) as fh:
            text = fh.read()
        return edit(f, text)
    return bench.kernel_source_digest(read)


def test_digest_ignores_comments_but_not_code():
    ref = bench.kernel_source_digest()
    assert _digest_with(lambda f, t: t) == ref
    assert _digest_with(lambda f, t: t + "\n// a new comment\n\n") == ref
    assert _digest_with(lambda f, t: t.replace("constexpr int UV = 16;", "constexpr int UV = 16;  // batch")
                        if f == "gemm.hip" else t) == ref
    assert _digest_with(lambda f, t: t.replace("constexpr int UV = 16;", "constexpr int UV = 8;")
                        if f == "gemm.hip" else t) != ref


def test_several_gpus_are_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "single-GPU" in r.stdout + r.stderr


def test_mfma_figures():
    # streaming each weight once: rows flop per byte at 8 TB/s over 2.5 PF
    assert abs(bench.mfma_ceiling(32) - 32 * 8e12 / 2.5e15) < 1e-12
    assert abs(bench.mfma_ceiling(32) - 0.1024) < 1e-12
    # 2 flops per weight element per row; a later step's FC is [H, 2H]
    H, I, V = 8192, 28672, 128256
    params = H * 2 * H + (64 + 16) * 128 * H + H * 64 * 128 + 3 * H * I + V * H
    assert bench.product_flops(L3_70B_BS32, 1, 32) == 2 * 32 * params
