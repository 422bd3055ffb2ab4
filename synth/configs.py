"""Workload shapes for the PRISM drafting hot path.

This module is shared by the oracle and the GPU path.  It only describes
shapes and seeds; it contains none of the drafting arithmetic.

The drafter follows the paper's architecture (Sec. 3.2, Table 2): a frozen
token embedding E, a frozen LM head, and M processing modules, each a fusion
FC plus one transformer layer.  A surjection f_map sends draft step k to the
module that computes it.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class DraftConfig:
    name: str
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    n_steps: int                 # K for a chain, D (forward passes) for a tree
    feat_width: int              # F_t: width of the target feature fed at step 1
    rope_theta: float
    dtype: str                   # "f32" or "bf16": weights, embeddings, features, KV
    batch: int
    ctx_len: int = 0             # fixed prior context (used when ctx_range is None)
    ctx_range: Optional[Tuple[int, int]] = None   # ragged prior context, inclusive
    kv_block_size: int = 16
    shuffle_blocks: bool = False  # physical KV blocks in seeded random order
    mode: str = "chain"          # "chain" or "tree"
    tree_width: int = 0          # w
    tree_nodes: int = 0          # v (output nodes, root excluded)
    rms_eps: float = 1e-5
    seed: int = 0
    f_map: Optional[Tuple[int, ...]] = None   # 0-based; None = identity
    n_sets: Optional[int] = None              # M; None = n_steps
    # chain whose step 1 catches up on n_b accepted tokens per sequence,
    # n_b uniform on this inclusive range (None: step 1 takes the last one)
    n_new: Optional[Tuple[int, int]] = None
    # stochastic drafting: tokens drawn from softmax(logits / T) with seeded
    # uniforms (None: greedy)
    temperature: Optional[float] = None
    # KV slots appended after the prior context, when not those of the
    # chain or tree (a target model scoring a tree of v nodes needs 1 + v)
    draft_slots: Optional[int] = None

    # ---- derived -------------------------------------------------------
    @property
    def M(self) -> int:
        return self.n_sets if self.n_sets is not None else self.n_steps

    @property
    def fmap(self) -> Tuple[int, ...]:
        if self.f_map is not None:
            return tuple(self.f_map)
        return tuple(range(self.n_steps))

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def set_feat_width(self, s: int) -> int:
        """Feature width F_s of parameter set s.

        The set that serves step 1 fuses the target feature (width F_t); sets
        serving later steps fuse the draft's own previous hidden state
        (width H).  A set serving both kinds needs F_t == H.
        """
        fm = self.fmap
        first = fm[0] == s
        later = any(fm[k] == s for k in range(1, len(fm)))
        if first and later and self.feat_width != self.hidden:
            raise ValueError("set %d serves step 1 and later steps but F_t != H" % s)
        if first:
            return self.feat_width
        return self.hidden

    @property
    def n_draft_slots(self) -> int:
        """KV slots the drafting call appends after the prior context."""
        if self.draft_slots is not None:
            return self.draft_slots
        if self.mode == "chain":
            return self.n_steps + (self.n_new[1] - 1 if self.n_new else 0)
        return 1 + (self.n_steps - 1) * self.tree_width

    @property
    def max_new_rows(self) -> int:
        """Largest total of catch-up rows (0 without catch-up)."""
        return self.batch * self.n_new[1] if self.n_new else 0

    @property
    def max_ctx(self) -> int:
        return self.ctx_range[1] if self.ctx_range else self.ctx_len

    @property
    def blocks_per_seq(self) -> int:
        return -(-(self.max_ctx + self.n_draft_slots) // self.kv_block_size)

    @property
    def rows(self) -> int:
        """Largest number of rows one forward step processes."""
        if self.mode == "chain":
            return self.batch
        return self.batch * self.tree_width

    @property
    def n_candidates(self) -> int:
        return self.tree_width + (self.n_steps - 1) * self.tree_width ** 2

    def with_(self, **kw) -> "DraftConfig":
        return replace(self, **kw)


# The five workloads.  Shapes follow the Llama-3 8B/70B targets the paper
# evaluates against (Sec. 4 "Target LLMs"); the tree shape follows the
# depth/width/verified-node topology of Sec. 4.3.
TINY_F32 = DraftConfig(
    name="tiny_f32_chain", hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
    ffn=688, vocab=4096, n_steps=3, feat_width=256, rope_theta=10000.0,
    dtype="f32", batch=1, ctx_len=128)

L3_8B_BS1 = DraftConfig(
    name="llama3_8b_bf16_chain_bs1", hidden=4096, n_q_heads=32, n_kv_heads=8,
    head_dim=128, ffn=14336, vocab=128256, n_steps=5, feat_width=12288,
    rope_theta=500000.0, dtype="bf16", batch=1, ctx_len=2048)

L3_8B_BS16 = L3_8B_BS1.with_(
    name="llama3_8b_bf16_chain_bs16_paged", batch=16, ctx_len=0,
    ctx_range=(512, 4096), shuffle_blocks=True)

L3_8B_TREE = L3_8B_BS1.with_(
    name="llama3_8b_bf16_tree_bs4", batch=4, ctx_len=1024, mode="tree",
    n_steps=6, tree_width=8, tree_nodes=60)

L3_70B_BS32 = DraftConfig(
    name="llama3_70b_bf16_chain_bs32", hidden=8192, n_q_heads=64, n_kv_heads=8,
    head_dim=128, ffn=28672, vocab=128256, n_steps=7, feat_width=24576,
    rope_theta=500000.0, dtype="bf16", batch=32, ctx_len=4096)

# Catch-up chains: step 1 prefills every token accepted in the last
# verification (the paper's S_acc; with K = 5 drafts, up to K + 1 = 6 tokens
# can be accepted per cycle, so batch 16 brings up to 96 rows).
L3_8B_BS1_CATCHUP = L3_8B_BS1.with_(name="llama3_8b_bf16_chain_bs1_catchup4", n_new=(4, 4))
L3_8B_BS16_CATCHUP = L3_8B_BS16.with_(name="llama3_8b_bf16_chain_bs16_paged_catchup",
                                      n_new=(1, 6))

# The paper's second target family (Sec. 4 "Target LLMs": Llama-2 7B; MHA,
# vocabulary 32000).  The draft fuses only the target's last-layer hidden
# state here (F_t = H, the paper's own design), so one parameter set can
# serve every step: M = 1, 2 (the paper's evaluated instance: module 1 for
# step 1, module 2 for the rest) and 5 are all valid step maps.
L2_7B_BS1 = DraftConfig(
    name="llama2_7b_bf16_chain_bs1", hidden=4096, n_q_heads=32, n_kv_heads=32,
    head_dim=128, ffn=11008, vocab=32000, n_steps=5, feat_width=4096,
    rope_theta=10000.0, dtype="bf16", batch=1, ctx_len=2048)
L2_7B_BS1_M1 = L2_7B_BS1.with_(name="llama2_7b_bf16_chain_bs1_m1", f_map=(0, 0, 0, 0, 0), n_sets=1)
L2_7B_BS1_M2 = L2_7B_BS1.with_(name="llama2_7b_bf16_chain_bs1_m2", f_map=(0, 1, 1, 1, 1), n_sets=2)

# Stochastic drafting at T = 1 (the paper's T = 1 rows, Tables 4-5).
L3_8B_BS1_T1 = L3_8B_BS1.with_(name="llama3_8b_bf16_chain_bs1_t1", temperature=1.0)

# A target model for tree verification (Sec. 2: the target scores every
# candidate of a draft tree in one pass under a tree attention mask): one
# transformer layer of the drafter's shape with its own weights, fed the
# token embeddings (its feature input is zero, width H), scoring the root
# and the v nodes of each drafted tree.
def scoring_target(cfg: DraftConfig) -> DraftConfig:
    return cfg.with_(name=cfg.name + "_target1", n_steps=1, feat_width=cfg.hidden, mode="chain",
                     tree_width=0, tree_nodes=0, f_map=None, n_sets=1,
                     draft_slots=1 + cfg.tree_nodes)


CONFIGS = {c.name: c for c in (TINY_F32, L3_8B_BS1, L3_8B_BS16, L3_8B_TREE, L3_70B_BS32,
                               L3_8B_BS1_CATCHUP, L3_8B_BS16_CATCHUP, L3_8B_BS1_T1,
                               L2_7B_BS1, L2_7B_BS1_M1, L2_7B_BS1_M2)}

# Reduced shapes for element-by-element parity: small enough for the oracle to
# finish in seconds, large enough to span several tiles of every kernel and to
# leave ragged tails (vocab not a multiple of the LM-head tile, contexts not a
# multiple of the KV chunk or block).
SMALL_BF16_CHAIN = DraftConfig(
    name="small_bf16_chain", hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=64,
    ffn=1376, vocab=5008, n_steps=4, feat_width=1536, rope_theta=500000.0,
    dtype="bf16", batch=3, ctx_len=0, ctx_range=(37, 700), shuffle_blocks=True)

SMALL_BF16_TREE = SMALL_BF16_CHAIN.with_(
    name="small_bf16_tree", batch=2, ctx_range=(200, 333), mode="tree", n_steps=4,
    tree_width=4, tree_nodes=20)

SMALL_F32_CHAIN = TINY_F32.with_(name="small_f32_chain_ragged", batch=3, ctx_len=0,
                                 ctx_range=(1, 300), shuffle_blocks=True)
