"""Convenience wrapper that owns a context and marshals torch tensors.

Marshalling only: allocation of output tensors, struct filling, and calls
into the HIP library.  Nothing here computes any part of the drafting path.
"""
from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import binding as B


def _dtype_code(dtype: str) -> int:
    return B.PRISM_BF16 if dtype == "bf16" else B.PRISM_F32


class Drafter:
    """One drafting context on the current GPU.

    `shape` is any object with the model/capacity attributes of
    prism_config (hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab,
    feat_width, rope_theta, rms_eps, dtype ("f32"/"bf16"), kv_block_size,
    batch, tree_width, tree_nodes) plus n_sets (M), n_steps and
    blocks_per_seq.
    """

    def __init__(self, shape, max_batch: Optional[int] = None, max_steps: Optional[int] = None,
                 max_blocks_per_seq: Optional[int] = None, max_new_rows: Optional[int] = None):
        self.shape = shape
        cfg = B.prism_config()
        cfg.hidden = shape.hidden
        cfg.n_q_heads = shape.n_q_heads
        cfg.n_kv_heads = shape.n_kv_heads
        cfg.head_dim = shape.head_dim
        cfg.ffn = shape.ffn
        cfg.vocab = shape.vocab
        cfg.n_sets = shape.M
        cfg.max_steps = max_steps or shape.n_steps
        cfg.feat_width = shape.feat_width
        cfg.rope_theta = shape.rope_theta
        cfg.rms_eps = shape.rms_eps
        cfg.dtype = _dtype_code(shape.dtype)
        cfg.kv_block_size = shape.kv_block_size
        cfg.max_batch = max_batch or shape.batch
        cfg.max_blocks_per_seq = max_blocks_per_seq or shape.blocks_per_seq
        cfg.tree_width = shape.tree_width
        cfg.tree_nodes = shape.tree_nodes
        cfg.max_new_rows = (max_new_rows if max_new_rows is not None
                            else getattr(shape, "max_new_rows", 0))
        self.cfg = cfg
        self.ctx = B.prism_create(cfg)
        self.device = torch.device("cuda", torch.cuda.current_device())

    def close(self):
        if self.ctx:
            B.prism_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # weights ------------------------------------------------------------------
    def load(self, weights, sets: Optional[Sequence[int]] = None):
        B.prism_draft_load_shared(self.ctx, weights.embed, weights.lm_head, weights.final_norm)
        ids = range(len(weights.sets)) if sets is None else sets
        for s, ps in zip(ids, weights.sets):
            self.load_set(s, ps)

    def load_set(self, s: int, ps):
        p = B.prism_param_set()
        for name in ("w_fc", "g1", "w_q", "w_k", "w_v", "w_o", "g2", "w_gate", "w_up", "w_down"):
            setattr(p, "d_" + name, B.ptr(getattr(ps, name)))
        p.feat_width = ps.feat_width
        B.prism_draft_load_params(self.ctx, s, p)

    def set_step_map(self, f_map):
        B.prism_set_step_map(self.ctx, f_map)

    # batches ------------------------------------------------------------------
    def batch(self, inp) -> B.prism_batch:
        b = B.prism_batch()
        b.batch = int(inp.tokens.shape[0])
        b.d_tokens = B.ptr(inp.tokens)
        b.d_features = B.ptr(inp.features)
        b.d_ctx_lens = B.ptr(inp.ctx_lens)
        b.d_k_pool = B.ptr(inp.k_pool)
        b.d_v_pool = B.ptr(inp.v_pool)
        b.d_block_table = B.ptr(inp.block_table)
        b.n_pool_blocks = int(inp.k_pool.shape[0])
        return b

    # calls --------------------------------------------------------------------
    def chain_buffers(self, nb: int, K: int, logits=False, hidden=False):
        dev = self.device
        out = {"tokens": torch.full((nb, K), -1, dtype=torch.int32, device=dev)}
        out["logits"] = (torch.empty((nb, K, self.shape.vocab), dtype=torch.float32, device=dev)
                         if logits else None)
        out["hidden"] = (torch.empty((nb, K, self.shape.hidden), dtype=torch.float32, device=dev)
                         if hidden else None)
        return out

    def chain(self, inp, K: Optional[int] = None, logits=False, hidden=False, out=None,
              batch=None):
        K = K or self.shape.n_steps
        b = batch if batch is not None else self.batch(inp)
        if out is None:
            out = self.chain_buffers(b.batch, K, logits, hidden)
        B.prism_draft_chain(self.ctx, b, K, out["tokens"], out["logits"], out["hidden"])
        return out

    def chain_sample(self, inp, temperature: float, K: Optional[int] = None, logits=False,
                     hidden=False, out=None, batch=None):
        """Stochastic chain: tokens drawn from softmax(logits / T) with the
        uniforms inp.uniforms [B, K]; out["logp"] holds log p_draft."""
        K = K or self.shape.n_steps
        b = batch if batch is not None else self.batch(inp)
        if out is None:
            out = self.chain_buffers(b.batch, K, logits, hidden)
            out["logp"] = torch.full((b.batch, K), float("nan"), dtype=torch.float32,
                                     device=self.device)
        B.prism_draft_chain_sample(self.ctx, b, K, temperature, inp.uniforms, out["tokens"],
                                   out.get("logp"), out["logits"], out["hidden"])
        return out

    def chain_catchup(self, inp, K: Optional[int] = None, logits=False, hidden=False, out=None,
                      batch=None):
        """Chain whose step 1 is the prefill over inp.new_tokens / new_features
        (rows delimited by inp.new_offsets)."""
        K = K or self.shape.n_steps
        b = batch if batch is not None else self.batch(inp)
        if out is None:
            out = self.chain_buffers(b.batch, K, logits, hidden)
        cu = B.prism_catchup()
        cu.total_rows = int(inp.new_tokens.shape[0])
        cu.d_offsets = B.ptr(inp.new_offsets)
        cu.d_tokens = B.ptr(inp.new_tokens)
        cu.d_features = B.ptr(inp.new_features)
        B.prism_draft_chain_catchup(self.ctx, b, cu, K, out["tokens"], out["logits"],
                                    out["hidden"])
        return out

    def tree_buffers(self, nb: int, depth: int, debug=True, logits=False):
        dev = self.device
        w, v = self.shape.tree_width, self.shape.tree_nodes
        C = w + (depth - 1) * w * w
        i32 = dict(dtype=torch.int32, device=dev)
        out = {"tokens": torch.full((nb, v), -1, **i32), "parent": torch.full((nb, v), -2, **i32),
               "depth": torch.zeros((nb, v), **i32),
               "score": torch.zeros((nb, v), dtype=torch.float32, device=dev),
               "mask": torch.zeros((nb, v), dtype=torch.int64, device=dev)}
        if debug:
            out["cand_tokens"] = torch.full((nb, C), -1, **i32)
            out["cand_parent"] = torch.full((nb, C), -2, **i32)
            out["cand_score"] = torch.zeros((nb, C), dtype=torch.float32, device=dev)
            out["frontier"] = torch.full((nb, max(depth - 1, 1), w), -1, **i32)
        if logits:
            out["logits"] = torch.full((depth, nb, w, self.shape.vocab), float("nan"),
                                       dtype=torch.float32, device=dev)
        return out

    def tree(self, inp, depth: Optional[int] = None, debug=True, logits=False, out=None,
             batch=None):
        depth = depth or self.shape.n_steps
        b = batch if batch is not None else self.batch(inp)
        if out is None:
            out = self.tree_buffers(b.batch, depth, debug, logits)
        t = B.prism_tree_out()
        for k in ("tokens", "parent", "depth", "score", "mask"):
            setattr(t, "d_" + k, B.ptr(out[k]))
        for k in ("cand_tokens", "cand_parent", "cand_score", "frontier", "logits"):
            setattr(t, "d_" + k, B.ptr(out.get(k)))
        B.prism_draft_tree(self.ctx, b, depth, t)
        return out

    def score_tree(self, inp, tokens, depth, mask, out=None, batch=None):
        """Target-side scoring of B draft trees (this context holds the
        scoring model): logits [B, v+1, V] of the root and every node under
        the tree mask.  inp describes the scoring model's own sequences
        (root tokens, features, prior KV)."""
        b = batch if batch is not None else self.batch(inp)
        Bn, v = int(tokens.shape[0]), int(tokens.shape[1])
        if out is None:
            out = torch.empty((Bn, v + 1, self.shape.vocab), dtype=torch.float32,
                              device=self.device)
        B.prism_score_tree(self.ctx, b, v, tokens, depth, mask, out)
        return out

    def verify_chain(self, target_logits, draft_tokens, temperature: float = 0.0,
                     draft_logits=None, uniforms=None):
        """Sec. 2 verification of B chains of K drafts; returns kept counts
        and next tokens [B]."""
        Bn, K = int(draft_tokens.shape[0]), int(draft_tokens.shape[1])
        n = torch.empty(Bn, dtype=torch.int32, device=self.device)
        nxt = torch.empty(Bn, dtype=torch.int32, device=self.device)
        B.prism_verify_chain(self.ctx, Bn, K, temperature, target_logits, draft_logits,
                             draft_tokens, uniforms, n, nxt)
        return {"n": n, "next": nxt}

    def verify_tree(self, target_logits, tokens, parent):
        """Greedy verification of B draft trees; returns kept counts, kept
        node paths [B, nodes] (-1 padded) and next tokens."""
        Bn, v = int(tokens.shape[0]), int(tokens.shape[1])
        n = torch.empty(Bn, dtype=torch.int32, device=self.device)
        path = torch.empty((Bn, v), dtype=torch.int32, device=self.device)
        nxt = torch.empty(Bn, dtype=torch.int32, device=self.device)
        B.prism_verify_tree(self.ctx, Bn, v, target_logits, tokens, parent, n, path, nxt)
        return {"n": n, "path": path, "next": nxt}

    def step(self, k: int, inp, rows: dict, topk: int = 1, logits=False, batch=None):
        """One pass of step k on explicit rows.  `rows` holds device tensors:
        tokens, feat, seq, pos, slot and optionally feat_rows, tree_bits;
        feat is fp32 (hidden states) or the context dtype (target features)."""
        b = batch if batch is not None else self.batch(inp)
        R = int(rows["tokens"].shape[0])
        dev = self.device
        io = B.prism_step_io()
        io.rows = R
        io.d_tokens = B.ptr(rows["tokens"])
        io.d_feat = B.ptr(rows["feat"])
        io.feat_dtype = B.PRISM_BF16 if rows["feat"].dtype == torch.bfloat16 else B.PRISM_F32
        io.d_feat_rows = B.ptr(rows.get("feat_rows"))
        io.d_seq = B.ptr(rows["seq"])
        io.d_pos = B.ptr(rows["pos"])
        io.d_slot = B.ptr(rows["slot"])
        io.d_tree_bits = B.ptr(rows.get("tree_bits"))
        io.kv = __import__("ctypes").pointer(b)
        io.topk = topk
        out = {"hidden": torch.empty((R, self.shape.hidden), dtype=torch.float32, device=dev),
               "ids": torch.empty((R, topk), dtype=torch.int32, device=dev),
               "logp": torch.empty((R, topk), dtype=torch.float32, device=dev),
               "logits": (torch.empty((R, self.shape.vocab), dtype=torch.float32, device=dev)
                          if logits else None)}
        io.d_hidden_out = B.ptr(out["hidden"])
        io.d_topk_ids = B.ptr(out["ids"])
        io.d_topk_logp = B.ptr(out["logp"])
        io.d_logits = B.ptr(out["logits"])
        B.prism_draft_step(self.ctx, k, io)
        return out

    def device_status(self) -> int:
        return B.prism_device_status(self.ctx)
