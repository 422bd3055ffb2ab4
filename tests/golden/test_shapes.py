"""Shapes of the stored oracle runs (shared by make_golden.py and the test)."""
from synth import DraftConfig

_TINY = DraftConfig(name="golden_tiny", hidden=32, n_q_heads=4, n_kv_heads=2, head_dim=8, ffn=48,
                    vocab=64, n_steps=3, feat_width=48, rope_theta=10000.0, dtype="f32",
                    batch=2, ctx_len=0, ctx_range=(3, 9), kv_block_size=4, shuffle_blocks=True)

GOLDEN_SHAPES = {
    "greedy_f32": (_TINY, "greedy"),
    "greedy_bf16": (_TINY.with_(dtype="bf16"), "greedy"),
    "catchup_f32": (_TINY.with_(batch=3, n_new=(1, 3)), "catchup"),
    "sampled_bf16": (_TINY.with_(dtype="bf16", temperature=1.0), "sampled"),
}
