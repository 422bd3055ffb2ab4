"""Seeded synthetic weights and inputs for the drafting hot path.

Shared by the oracle and the GPU path; it holds no drafting arithmetic, only
random draws and data placement (scattering the prior-context KV into a paged
pool).  Everything is drawn with torch generators on the requested device, so
a GPU run draws its tensors in HBM and the oracle receives exact host copies
of the same bytes.

Recipe (the paper trains real drafters; no weights are available, so every
tensor is synthetic):
  * matrices, E and the LM head: N(0, 0.02), rounded to the storage dtype (RNE)
  * RMSNorm gains: 1 + N(0, 0.02)
  * target features: N(0, 1); tokens uniform on [0, V)
  * prior-context K (already rotated, as stored) and V: N(0, 1)
  * ragged contexts: L_b uniform on the configured inclusive range, per sequence
  * paged KV: blocks of `kv_block_size` slots; the block table is a seeded
    permutation of the physical blocks when `shuffle_blocks` is set; slots that
    hold no prior context are NaN so that a read of them shows up.
  * stochastic drafting: one uniform on [0, 1) per (sequence, step), the
    draw that picks the token by inverse CDF
  * catch-up chains: n_b accepted tokens per sequence, uniform on the
    configured inclusive range; the earlier n_b - 1 tokens uniform on [0, V)
    and their target features N(0, 1); the newest one is the sequence's
    `tokens[b]` / `features[b]`, so n_b = 1 is the plain chain.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np
import torch

from .configs import DraftConfig

# tensor ids used to derive per-tensor seeds
T_EMBED, T_LMHEAD, T_FNORM = 0, 1, 2
T_FC, T_G1, T_WQ, T_WK, T_WV, T_WO, T_G2, T_WGATE, T_WUP, T_WDOWN = range(10, 20)
T_TOK, T_FEAT, T_CTX, T_KPOOL, T_VPOOL, T_BTAB, T_NNEW, T_NTOK, T_NFEAT, T_UNIF = range(100, 110)

SET_TENSORS = ("w_fc", "g1", "w_q", "w_k", "w_v", "w_o", "g2", "w_gate", "w_up", "w_down")


def derive_seed(*ids: int) -> int:
    st = np.random.SeedSequence([int(i) for i in ids]).generate_state(2, dtype=np.uint32)
    return int((int(st[0]) << 31) ^ int(st[1])) & ((1 << 63) - 1)


def torch_dtype(cfg: DraftConfig) -> torch.dtype:
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def _gen(device, *ids) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(derive_seed(*ids))
    return g


def _normal(shape, std, mean, dtype, device, *ids) -> torch.Tensor:
    t = torch.randn(shape, generator=_gen(device, *ids), device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(dtype)


@dataclass
class ParamSet:
    w_fc: torch.Tensor      # [H, H + F_s]   input order [embedding ; feature]
    g1: torch.Tensor        # [H]
    w_q: torch.Tensor       # [n_q*d, H]
    w_k: torch.Tensor       # [n_kv*d, H]
    w_v: torch.Tensor       # [n_kv*d, H]
    w_o: torch.Tensor       # [H, n_q*d]
    g2: torch.Tensor        # [H]
    w_gate: torch.Tensor    # [I, H]
    w_up: torch.Tensor      # [I, H]
    w_down: torch.Tensor    # [H, I]
    feat_width: int


@dataclass
class Weights:
    embed: torch.Tensor       # [V, H]
    lm_head: torch.Tensor     # [V, H]
    final_norm: torch.Tensor  # [H]
    sets: List[ParamSet]


@dataclass
class Inputs:
    tokens: torch.Tensor        # int32 [B]   last accepted token per sequence
    features: torch.Tensor      # [B, F_t]    target hidden-state feature of that token
    ctx_lens: torch.Tensor      # int32 [B]   prior context length L_b
    k_pool: torch.Tensor        # [n_blocks, n_kv, block, d]
    v_pool: torch.Tensor        # [n_blocks, n_kv, block, d]
    block_table: torch.Tensor   # int32 [B, blocks_per_seq]
    # catch-up chains only: rows new_offsets[b] .. new_offsets[b+1]-1 of
    # new_tokens / new_features are sequence b's accepted tokens, oldest first
    new_offsets: Optional[torch.Tensor] = None   # int32 [B + 1]
    new_tokens: Optional[torch.Tensor] = None    # int32 [T]
    new_features: Optional[torch.Tensor] = None  # [T, F_t]
    # stochastic drafting only: the uniform in [0, 1) of each (sequence, step)
    uniforms: Optional[torch.Tensor] = None      # fp32 [B, K]


def make_param_set(cfg: DraftConfig, s: int, device="cpu") -> ParamSet:
    H, d, I = cfg.hidden, cfg.head_dim, cfg.ffn
    F = cfg.set_feat_width(s)
    dt = torch_dtype(cfg)
    sd = cfg.seed
    mk = lambda shape, tid: _normal(shape, 0.02, 0.0, dt, device, sd, tid, s)
    gain = lambda tid: _normal((H,), 0.02, 1.0, dt, device, sd, tid, s)
    return ParamSet(
        w_fc=mk((H, H + F), T_FC), g1=gain(T_G1),
        w_q=mk((cfg.n_q_heads * d, H), T_WQ), w_k=mk((cfg.n_kv_heads * d, H), T_WK),
        w_v=mk((cfg.n_kv_heads * d, H), T_WV), w_o=mk((H, cfg.n_q_heads * d), T_WO),
        g2=gain(T_G2), w_gate=mk((I, H), T_WGATE), w_up=mk((I, H), T_WUP),
        w_down=mk((H, I), T_WDOWN), feat_width=F)


def make_weights(cfg: DraftConfig, device="cpu", sets: Optional[List[int]] = None) -> Weights:
    H, V = cfg.hidden, cfg.vocab
    dt = torch_dtype(cfg)
    sd = cfg.seed
    ids = range(cfg.M) if sets is None else sets
    return Weights(
        embed=_normal((V, H), 0.02, 0.0, dt, device, sd, T_EMBED),
        lm_head=_normal((V, H), 0.02, 0.0, dt, device, sd, T_LMHEAD),
        final_norm=_normal((H,), 0.02, 1.0, dt, device, sd, T_FNORM),
        sets=[make_param_set(cfg, s, device) for s in ids])


def ctx_lengths(cfg: DraftConfig) -> np.ndarray:
    if cfg.ctx_range is None:
        return np.full(cfg.batch, cfg.ctx_len, dtype=np.int32)
    lo, hi = cfg.ctx_range
    out = np.empty(cfg.batch, dtype=np.int32)
    for b in range(cfg.batch):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, T_CTX, b])))
        out[b] = rng.integers(lo, hi + 1)
    return out


def new_counts(cfg: DraftConfig) -> np.ndarray:
    """Accepted tokens n_b per sequence of a catch-up chain."""
    lo, hi = cfg.n_new
    out = np.empty(cfg.batch, dtype=np.int32)
    for b in range(cfg.batch):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, T_NNEW, b])))
        out[b] = rng.integers(lo, hi + 1)
    return out


def make_inputs(cfg: DraftConfig, device="cpu", extra_blocks: int = 0) -> Inputs:
    B, H, d, nkv, bs = cfg.batch, cfg.hidden, cfg.head_dim, cfg.n_kv_heads, cfg.kv_block_size
    dt = torch_dtype(cfg)
    sd = cfg.seed
    toks = []
    feats = []
    for b in range(B):
        toks.append(torch.randint(0, cfg.vocab, (1,), generator=_gen(device, sd, T_TOK, b),
                                  device=device, dtype=torch.int64))
        feats.append(_normal((1, cfg.feat_width), 1.0, 0.0, dt, device, sd, T_FEAT, b))
    tokens = torch.cat(toks).to(torch.int32)
    features = torch.cat(feats, 0)

    lens = ctx_lengths(cfg)
    nbps = cfg.blocks_per_seq
    n_blocks = B * nbps + extra_blocks
    if cfg.shuffle_blocks:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([sd, T_BTAB])))
        perm = rng.permutation(n_blocks)[: B * nbps]
    else:
        perm = np.arange(B * nbps)
    btab = perm.reshape(B, nbps).astype(np.int32)

    shape = (n_blocks, nkv, bs, d)
    k_pool = _normal(shape, 1.0, 0.0, dt, device, sd, T_KPOOL)
    v_pool = _normal(shape, 1.0, 0.0, dt, device, sd, T_VPOOL)
    # poison every slot that holds no prior context
    live = torch.zeros((n_blocks, bs), dtype=torch.bool)
    for b in range(B):
        L = int(lens[b])
        for blk in range(nbps):
            lo = blk * bs
            n = max(0, min(bs, L - lo))
            if n:
                live[int(btab[b, blk]), :n] = True
    dead = (~live).to(device)[:, None, :, None].expand(shape)
    k_pool.masked_fill_(dead, float("nan"))
    v_pool.masked_fill_(dead, float("nan"))
    inp = Inputs(tokens=tokens, features=features,
                 ctx_lens=torch.from_numpy(lens).to(device),
                 k_pool=k_pool, v_pool=v_pool,
                 block_table=torch.from_numpy(btab).to(device))
    if cfg.n_new:
        counts = new_counts(cfg)
        nt, nf = [], []
        for b in range(B):
            n = int(counts[b])
            if n > 1:
                nt.append(torch.randint(0, cfg.vocab, (n - 1,), generator=_gen(device, sd, T_NTOK, b),
                                        device=device, dtype=torch.int64).to(torch.int32))
                nf.append(_normal((n - 1, cfg.feat_width), 1.0, 0.0, dt, device, sd, T_NFEAT, b))
            nt.append(tokens[b:b + 1])
            nf.append(features[b:b + 1])
        offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
        inp.new_offsets = torch.from_numpy(offs).to(device)
        inp.new_tokens = torch.cat(nt).contiguous()
        inp.new_features = torch.cat(nf, 0).contiguous()
    if cfg.temperature is not None:
        inp.uniforms = torch.rand((B, cfg.n_steps), generator=_gen(device, sd, T_UNIF),
                                  device=device, dtype=torch.float32)
    return inp


T_VLOG, T_VTGT, T_VTOK, T_VAGR, T_VUNI, T_VPATH = range(200, 206)


def make_verify_chain(V: int, B: int, K: int, seed: int = 0, device="cpu", noise: float = 0.5):
    """Synthetic inputs of chain verification: draft logits N(0, 2) [B, K, V];
    draft tokens uniform on [0, V), placed as each draft row's maximum; target
    logits = the draft rows plus N(0, noise) (row K: N(0, 2)), with the
    target's maximum placed on the draft for the first a_b positions and
    away from it at position a_b (a_b uniform on 0..K per sequence); the
    uniforms [B, K+1] of the rejection rule."""
    g = lambda tid: _gen(device, seed, tid)
    dl = torch.randn((B, K, V), generator=g(T_VLOG), device=device) * 2.0
    tok = torch.randint(0, V, (B, K), generator=g(T_VTOK), device=device, dtype=torch.int64)
    dl.scatter_(2, tok[..., None], dl.amax(dim=2, keepdim=True) + 1.0)
    tl = torch.randn((B, K + 1, V), generator=g(T_VTGT), device=device) * noise
    tl[:, :K] += dl
    tl[:, K] *= 2.0 / noise
    agree = torch.randint(0, K + 1, (B,), generator=g(T_VAGR), device=device)
    for b in range(B):
        a = int(agree[b])
        for i in range(K):
            row = tl[b, i]
            if i < a:
                row[tok[b, i]] = row.max() + 1.0
            elif i == a:
                row[tok[b, i]] = row.min() - 1.0
    u = torch.rand((B, K + 1), generator=g(T_VUNI), device=device)
    return {"target_logits": tl.contiguous(), "draft_logits": dl.contiguous(),
            "draft_tokens": tok.to(torch.int32).contiguous(), "uniforms": u}


def make_verify_tree_targets(tokens: torch.Tensor, parent: torch.Tensor, V: int, seed: int = 0):
    """Synthetic target logits [B, v+1, V] N(0, 2) for draft trees
    (tokens / parent [B, v]): along a random root path of each tree (a
    random child at each level, random length) the target's maximum is
    placed on the path's next token."""
    device = tokens.device
    B, v = tokens.shape
    g = _gen(device, seed, T_VTGT)
    tl = torch.randn((B, v + 1, V), generator=g, device=device) * 2.0
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, T_VPATH])))
    tk, pa = tokens.cpu().numpy(), parent.cpu().numpy()
    for b in range(B):
        at = -1
        for _ in range(int(rng.integers(0, v + 1))):
            kids = [j for j in range(v) if pa[b, j] == at]
            if not kids:
                break
            j = int(kids[rng.integers(0, len(kids))])
            row = tl[b, at + 1]
            row[int(tk[b, j])] = row.max() + 1.0
            at = j
    return tl.contiguous()


def logical_prior_kv(kp: torch.Tensor, vp: torch.Tensor, btab: torch.Tensor, L: int,
                     cfg: DraftConfig):
    """Prior-context K and V of one sequence as [L, n_kv, d] host arrays.

    A gather through the block table row `btab` from host copies of the
    pools: data placement only.
    """
    bs = cfg.kv_block_size
    t = torch.arange(L)
    blk = btab.long()[t // bs]
    off = t % bs
    return to_host(kp[blk, :, off, :]), to_host(vp[blk, :, off, :])


def to_host(t: torch.Tensor) -> np.ndarray:
    """Exact host copy: bf16 as its uint16 bit pattern, others as numpy."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def host_weights(w: Weights) -> dict:
    """Host copies in the dict layout the oracle takes."""
    out = {"embed": to_host(w.embed), "lm_head": to_host(w.lm_head),
           "final_norm": to_host(w.final_norm), "sets": []}
    for ps in w.sets:
        d = {k: to_host(getattr(ps, k)) for k in SET_TENSORS}
        d["feat_width"] = ps.feat_width
        out["sets"].append(d)
    return out


def host_inputs(inp: Inputs, cfg: DraftConfig, seqs=None) -> dict:
    """Host copies in the dict layout the oracle takes.

    `seqs` restricts the (large) prior-KV gather to the listed sequences; the
    others get None.
    """
    kp, vp = inp.k_pool.cpu(), inp.v_pool.cpu()
    btab = inp.block_table.cpu()
    lens = inp.ctx_lens.cpu()
    ks, vs = [], []
    for b in range(cfg.batch):
        if seqs is not None and b not in seqs:
            ks.append(None)
            vs.append(None)
            continue
        k, v = logical_prior_kv(kp, vp, btab[b], int(lens[b]), cfg)
        ks.append(k)
        vs.append(v)
    out = {"tokens": to_host(inp.tokens), "features": to_host(inp.features),
           "ctx_lens": to_host(inp.ctx_lens), "prior_k": ks, "prior_v": vs}
    if inp.new_offsets is not None:
        out["new_offsets"] = to_host(inp.new_offsets)
        out["new_tokens"] = to_host(inp.new_tokens)
        out["new_features"] = to_host(inp.new_features)
    if inp.uniforms is not None:
        out["uniforms"] = to_host(inp.uniforms).astype(np.float64)
    return out
