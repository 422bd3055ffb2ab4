"""GPU parity: the HIP drafting path (through the C ABI) against the oracle.

Small configurations are compared element by element (every sequence, every
step); the full-size workloads are compared on sampled sequences, which the
oracle computes exactly because sequences are independent.
"""
import numpy as np
import pytest
import torch

from synth import (L2_7B_BS1, L2_7B_BS1_M1, L2_7B_BS1_M2, L3_8B_BS1, L3_8B_BS1_CATCHUP,
                   L3_8B_BS1_T1, L3_8B_BS16, L3_8B_BS16_CATCHUP, L3_8B_TREE,
                   L3_70B_BS32, SMALL_BF16_CHAIN, SMALL_BF16_TREE, SMALL_F32_CHAIN, TINY_F32)
from harness import (check_chain, check_draft_kv, check_sampled_chain, check_tree, gpu_setup,
                     log, oracle_for)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def run_chain_parity(cfg, seqs=None):
    log("chain parity", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    out = dr.chain(inp, logits=True, hidden=True)
    plain = dr.chain(inp)                      # the launch the benchmark times
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    assert torch.equal(out["tokens"], plain["tokens"])
    seqs = list(range(cfg.batch)) if seqs is None else seqs
    orc, hi = oracle_for(cfg, w, inp, seqs)
    log("oracle", cfg.name, "seqs", seqs)
    res = check_chain(cfg, out, orc, hi, seqs, inp=inp)
    log(cfg.name, res)
    dr.close()
    return res


@pytest.mark.parametrize("cfg", [TINY_F32, SMALL_F32_CHAIN, SMALL_BF16_CHAIN], ids=lambda c: c.name)
def test_chain_parity_small(cfg):
    run_chain_parity(cfg)


# Row counts that select different product paths: 1 and 2 rows take the
# VALU GEMV main loop (1 row also the GEMV LM head), 3-16 rows one 16-row
# MFMA group, 17-32 rows two groups and eight tiles per wave where the tile
# count allows (vocabulary 5120 = 320 tiles), more than 32 rows four groups;
# every sequence is compared.
@pytest.mark.parametrize("cfg", [
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs1", batch=1),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs2", batch=2),
    # H = 480: no embedding table (H % 64 != 0), so the GEMV fusion FC gathers
    # [E(x) ; f] itself, and the one-row LM head takes the MFMA tiles (its
    # GEMV streams whole batches of 16 k-blocks, H % 512 == 0)
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs1_h480", batch=1, hidden=480),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs24", batch=24, vocab=5120),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs40", batch=40, ctx_range=(20, 300)),
    # H = 2048 at 24 rows: the fusion FC's K-split grid (80 workgroups) has one
    # per row, so steps >= 2 take their feature operand from the previous
    # down product and resolve their tokens in the K-split kernel (no prep
    # pass), with two row tiles
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs24_h2048", batch=24, hidden=2048,
                           ctx_range=(20, 200)),
], ids=lambda c: c.name)
def test_chain_parity_row_counts(cfg):
    run_chain_parity(cfg)


# A wide FFN gives the gate/up product at least 200 groups of 4 (16 rows) or
# 8 (24 rows) tiles, which takes the unsplit batched path (K shared by the
# waves of a workgroup, epilogue in the kernel).  At the 8B FFN width (1792
# gate/up tiles) it runs 7 tiles per wave, at 16 and 32 rows.
@pytest.mark.parametrize("cfg", [
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs16_ffn6400", batch=16, ffn=6400),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs24_ffn12800", batch=24, ffn=12800, vocab=5120),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs16_ffn14336", batch=16, ffn=14336),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs32_ffn14336", batch=32, ffn=14336,
                           ctx_range=(20, 200)),
], ids=lambda c: c.name)
def test_chain_parity_unsplit_products(cfg):
    run_chain_parity(cfg)


# Catch-up chains: step 1 is the prefill over every accepted token of a
# sequence (ragged n_b), then the chain continues from the last one.  The
# draft KV written for the accepted rows and the chain steps is compared slot
# by slot.  n_b = 2 at one sequence keeps the front on the GEMV path; larger
# totals take the MFMA path, and the back of step 1 runs on B rows.
@pytest.mark.parametrize("cfg", [
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs1_n2", batch=1, n_new=(2, 2)),
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs1_n5", batch=1, n_new=(5, 5)),
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs3", batch=3, n_new=(1, 5)),
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs12", batch=12, n_new=(1, 4)),
    SMALL_F32_CHAIN.with_(name="small_f32_catchup", n_new=(1, 4)),
    # more accepted rows than one pass takes: the front runs in chunks of 64
    # rows, a sequence's rows may straddle two chunks
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs16_n1to6", batch=16, n_new=(1, 6)),
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs1_n70", batch=1, n_new=(70, 70),
                           ctx_range=(37, 100)),
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs5_n30to40", batch=5, n_new=(30, 40)),
], ids=lambda c: c.name)
def test_chain_catchup_parity(cfg):
    log("catch-up parity", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    out = dr.chain_catchup(inp, logits=True, hidden=True)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    seqs = list(range(cfg.batch))
    orc, hi = oracle_for(cfg, w, inp, seqs)
    res = check_chain(cfg, out, orc, hi, seqs, catchup=True, inp=inp)
    log(cfg.name, "n_b", np.diff(hi["new_offsets"]).tolist(), res)
    dr.close()


# Stochastic drafting: tokens drawn from softmax(logits / T) by inverse CDF
# with seeded uniforms, through the MFMA LM head (batch 3) and the GEMV one
# (batch 1), in bf16 and fp32.
@pytest.mark.parametrize("cfg", [
    SMALL_BF16_CHAIN.with_(name="small_bf16_sample_t1", temperature=1.0),
    SMALL_BF16_CHAIN.with_(name="small_bf16_sample_bs1_t07", batch=1, temperature=0.7),
    SMALL_F32_CHAIN.with_(name="small_f32_sample_t15", temperature=1.5),
], ids=lambda c: c.name)
def test_chain_sample_parity(cfg):
    log("sampled chain parity", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    out = dr.chain_sample(inp, cfg.temperature, logits=True, hidden=True)
    again = dr.chain_sample(inp, cfg.temperature)        # the launch the benchmark times
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    assert torch.equal(out["tokens"], again["tokens"])
    assert torch.equal(out["logp"], again["logp"])
    seqs = list(range(cfg.batch))
    orc, hi = oracle_for(cfg, w, inp, seqs)
    res = check_sampled_chain(cfg, out, orc, hi, seqs, cfg.temperature)
    check_draft_kv(cfg, inp, orc.chain(hi, forced=out["tokens"].cpu().numpy().astype(np.int64),
                                       temperature=cfg.temperature,
                                       uniforms=hi["uniforms"])["draft_kv"], seqs)
    log(cfg.name, res)
    assert res["draw_agreement"] == 1.0
    dr.close()


# The ends of the unit interval: u = 0 draws the first id of nonzero
# probability; u = 1 (and u just below 1, where rounding can leave the running
# sum short of u * S) takes the last one, the id the inverse CDF reaches at
# the top of the distribution.
def test_chain_sample_extreme_uniforms():
    cfg = SMALL_BF16_CHAIN.with_(name="small_bf16_sample_edges", temperature=1.0)
    log("sampled chain, extreme uniforms", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    B, K = inp.uniforms.shape
    edges = torch.tensor([0.0, 1.0, 0.99999994, 1e-7, 0.5], dtype=torch.float32)
    u = torch.stack([edges[(torch.arange(K) + b) % len(edges)] for b in range(B)])
    inp.uniforms = u.to(inp.uniforms.device).contiguous()
    out = dr.chain_sample(inp, cfg.temperature, logits=True)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    toks = out["tokens"].cpu().numpy()
    for b in range(B):
        for k in range(K):
            if float(u[b, k]) == 0.0:
                assert toks[b, k] == 0, (b, k, toks[b, k])
    # every draw (u = 1 included) lies in its token's CDF interval
    seqs = list(range(B))
    orc, hi = oracle_for(cfg, w, inp, seqs)
    res = check_sampled_chain(cfg, out, orc, hi, seqs, cfg.temperature)
    log(cfg.name, res)
    dr.close()


def test_catchup_of_one_token_equals_chain():
    cfg = SMALL_BF16_CHAIN.with_(n_new=(1, 1))
    dr, w, inp = gpu_setup(cfg)
    a = dr.chain_catchup(inp, logits=True, hidden=True)
    b = dr.chain(inp, logits=True, hidden=True)
    torch.cuda.synchronize()
    assert torch.equal(a["tokens"], b["tokens"])
    assert torch.equal(a["logits"], b["logits"])
    assert torch.equal(a["hidden"], b["hidden"])
    dr.close()


def test_chain_deterministic_and_poison_free():
    cfg = SMALL_BF16_CHAIN
    dr, w, inp = gpu_setup(cfg)
    a = dr.chain(inp, logits=True, hidden=True)
    b = dr.chain(inp, logits=True, hidden=True)
    torch.cuda.synchronize()
    assert torch.equal(a["tokens"], b["tokens"])
    assert torch.equal(a["logits"], b["logits"])
    assert torch.isfinite(a["logits"]).all() and torch.isfinite(a["hidden"]).all()
    dr.close()


def test_chain_fmap_surjection():
    # the paper's evaluated instance: module 1 for step 1, module 2 for the rest
    cfg = SMALL_BF16_CHAIN.with_(f_map=(0, 1, 1, 1), n_sets=2)
    run_chain_parity(cfg)


def test_step_api_matches_chain_first_step():
    cfg = SMALL_BF16_CHAIN
    dr, w, inp = gpu_setup(cfg)
    ref = dr.chain(inp, K=1, logits=True, hidden=True)
    B = cfg.batch
    dev = inp.tokens.device
    # the chain wrote slot L_b; the explicit step rewrites the same slot
    rows = {"tokens": inp.tokens, "feat": inp.features,
            "seq": torch.arange(B, dtype=torch.int32, device=dev),
            "pos": inp.ctx_lens.clone(), "slot": inp.ctx_lens.clone()}
    st = dr.step(1, inp, rows, topk=1, logits=True)
    torch.cuda.synchronize()
    assert torch.equal(st["ids"][:, 0], ref["tokens"][:, 0])
    assert torch.equal(st["logits"], ref["logits"][:, 0])
    assert torch.equal(st["hidden"], ref["hidden"][:, 0])
    dr.close()


@pytest.mark.parametrize("lm", ["random", "zero", "pairs"])
def test_step_topk_matches_its_logits(lm):
    """Top-k > 1 on batched rows: the LM head stores the logits and a separate
    pass reduces them to the top-k partials.  Its filtered path (random
    logits, and exact ties between id pairs) and its plain path (every logit
    0) must give the exact top-k of the logits the same call returns, ordered
    by (value desc, id asc), with log-probabilities logit - logsumexp."""
    from synth import make_inputs, make_weights
    from paper_2602_01762_amd import Drafter
    cfg = SMALL_BF16_CHAIN.with_(tree_width=4, tree_nodes=12)
    w = make_weights(cfg, "cuda")
    if lm == "zero":
        w.lm_head.zero_()
    elif lm == "pairs":
        w.lm_head[1::2] = w.lm_head[0::2]
    inp = make_inputs(cfg, "cuda")
    dr = Drafter(cfg)
    dr.load(w)
    B, k = cfg.batch, 4
    dev = inp.tokens.device
    rows = {"tokens": inp.tokens, "feat": inp.features,
            "seq": torch.arange(B, dtype=torch.int32, device=dev),
            "pos": inp.ctx_lens.clone(), "slot": inp.ctx_lens.clone()}
    st = dr.step(1, inp, rows, topk=k, logits=True)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    lg = st["logits"].cpu().numpy().astype(np.float64)
    ids = st["ids"].cpu().numpy()
    logp = st["logp"].cpu().numpy()
    V = lg.shape[1]
    for r in range(B):
        order = np.lexsort((np.arange(V), -lg[r]))[:k]
        assert ids[r].tolist() == order.tolist(), (lm, r)
        m = lg[r].max()
        lse = m + np.log(np.exp(lg[r] - m).sum())
        np.testing.assert_allclose(logp[r], lg[r, order] - lse, atol=1e-4, rtol=0)
    if lm == "zero":
        assert (ids == np.arange(k)).all()
    dr.close()


def run_tree_parity(cfg, seqs=None):
    log("tree parity", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    out = dr.tree(inp, debug=True, logits=True)
    plain = dr.tree(inp, debug=False)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    for k in ("tokens", "parent", "depth", "score", "mask"):
        assert torch.equal(out[k], plain[k]), k
    seqs = list(range(cfg.batch)) if seqs is None else seqs
    orc, hi = oracle_for(cfg, w, inp, seqs)
    res = check_tree(cfg, out, orc, hi, seqs, cfg.n_steps)
    log(cfg.name, res)
    dr.close()


# An empty prior context (L_b = 0: the first pass starts from an empty KV
# cache, Sec. 3.2): the first row attends to its own slot only.  All
# sequences empty at one row (GEMV) and three rows (MFMA), a ragged batch
# with one empty sequence among short ones, catch-up prefills from an empty
# cache, and a tree.
CTX0 = dict(ctx_range=None, ctx_len=0)


@pytest.mark.parametrize("cfg", [
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_ctx0", **CTX0),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_bs1_ctx0", batch=1, **CTX0),
    SMALL_BF16_CHAIN.with_(name="small_bf16_chain_ctx0_mixed", batch=6, ctx_range=(0, 3)),
    SMALL_F32_CHAIN.with_(name="small_f32_chain_ctx0", **CTX0),
], ids=lambda c: c.name)
def test_chain_parity_empty_context(cfg):
    from synth import ctx_lengths
    assert (ctx_lengths(cfg) == 0).any()
    run_chain_parity(cfg)


@pytest.mark.parametrize("cfg", [
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs1_n4_ctx0", batch=1, n_new=(4, 4), **CTX0),
    SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs3_ctx0", batch=3, n_new=(2, 5), **CTX0),
], ids=lambda c: c.name)
def test_chain_catchup_parity_empty_context(cfg):
    test_chain_catchup_parity(cfg)


def test_tree_parity_empty_context():
    run_tree_parity(SMALL_BF16_TREE.with_(name="small_bf16_tree_ctx0", **CTX0))


def test_tree_parity_small():
    run_tree_parity(SMALL_BF16_TREE)


def test_tree_parity_small_f32():
    """fp32 weights and KV: ungrouped tree attention (the VALU kernel), fp32
    products and LM head."""
    run_tree_parity(SMALL_BF16_TREE.with_(name="small_f32_tree", dtype="f32"))


# Head geometries of the grouped tree attention (a workgroup takes the
# largest divisor of w whose rows x query heads fit 16 score columns): 6 rows
# of 2 heads, 2 rows of 8 heads, 4 rows of 4 heads at head_dim 128, and a
# width with no such divisor (ungrouped).
@pytest.mark.parametrize("cfg", [
    SMALL_BF16_TREE.with_(name="small_bf16_tree_g2_w6", n_q_heads=8, n_kv_heads=4,
                          tree_width=6, n_steps=3, tree_nodes=20),
    SMALL_BF16_TREE.with_(name="small_bf16_tree_g8_w4", n_q_heads=8, n_kv_heads=1),
    SMALL_BF16_TREE.with_(name="small_bf16_tree_d128", n_q_heads=4, n_kv_heads=1, head_dim=128),
    SMALL_BF16_TREE.with_(name="small_bf16_tree_w5", tree_width=5, n_steps=3, tree_nodes=14),
], ids=lambda c: c.name)
def test_tree_parity_head_geometries(cfg):
    run_tree_parity(cfg)


# The most rows a tree level takes in one pass: batch 8 x width 8 = 64 rows
# (four 16-row tiles in every batched product and in the LM head).
def test_tree_parity_max_rows():
    run_tree_parity(SMALL_BF16_TREE.with_(name="small_bf16_tree_b8_w8", batch=8, tree_width=8,
                                          n_steps=3, tree_nodes=20, ctx_range=(40, 200)))


def test_tree_width_one_equals_chain():
    tcfg = SMALL_BF16_TREE.with_(tree_width=1, tree_nodes=SMALL_BF16_TREE.n_steps)
    dr, w, inp = gpu_setup(tcfg)
    t = dr.tree(inp)
    c = dr.chain(inp, K=tcfg.n_steps)
    torch.cuda.synchronize()
    assert torch.equal(t["tokens"], c["tokens"])
    dr.close()


# ---------------------------------------------------------------- full size
@pytest.mark.slow
def test_full_8b_bs1_chain():
    run_chain_parity(L3_8B_BS1)


@pytest.mark.slow
def test_full_8b_bs16_paged_chain():
    from synth import ctx_lengths
    lens = ctx_lengths(L3_8B_BS16)
    run_chain_parity(L3_8B_BS16, seqs=[int(np.argmin(lens)), int(np.argmax(lens))])


@pytest.mark.slow
def test_full_8b_tree():
    run_tree_parity(L3_8B_TREE, seqs=[0])


@pytest.mark.slow
def test_full_70b_bs32_chain():
    run_chain_parity(L3_70B_BS32, seqs=[0, 31])


def run_catchup_parity(cfg, seqs):
    log("catch-up parity", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    out = dr.chain_catchup(inp, logits=True, hidden=True)
    plain = dr.chain_catchup(inp)                # the launch the benchmark times
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    assert torch.equal(out["tokens"], plain["tokens"])
    orc, hi = oracle_for(cfg, w, inp, seqs)
    res = check_chain(cfg, out, orc, hi, seqs, catchup=True, inp=inp)
    log(cfg.name, "seqs", seqs, res)
    dr.close()


@pytest.mark.slow
@pytest.mark.parametrize("cfg", [L2_7B_BS1, L2_7B_BS1_M1, L2_7B_BS1_M2], ids=lambda c: c.name)
def test_full_llama2_7b_chain(cfg):
    run_chain_parity(cfg)


@pytest.mark.slow
def test_full_8b_bs1_sample():
    cfg = L3_8B_BS1_T1
    dr, w, inp = gpu_setup(cfg)
    out = dr.chain_sample(inp, 1.0, logits=True)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    orc, hi = oracle_for(cfg, w, inp, [0])
    res = check_sampled_chain(cfg, out, orc, hi, [0], 1.0)
    log(cfg.name, res)
    dr.close()


@pytest.mark.slow
def test_full_8b_bs1_catchup():
    run_catchup_parity(L3_8B_BS1_CATCHUP, [0])


def test_catchup_at_the_row_limit():
    """4096 accepted rows (64 sequences x 64 tokens, the largest catch-up
    call): 64 front chunks of 64 rows, every sequence in a chunk of its own
    at a chunk border."""
    cfg = SMALL_BF16_CHAIN.with_(name="small_bf16_catchup_bs64_n64", batch=64, n_new=(64, 64),
                                 ctx_range=(37, 100))
    assert cfg.max_new_rows == 4096
    test_chain_catchup_parity(cfg)


@pytest.mark.slow
def test_full_8b_bs1_catchup_two_chunks():
    """The 8B shape with 70 accepted tokens: the front runs in two chunks
    (64 + 6 rows), the last row in the second."""
    run_catchup_parity(L3_8B_BS1.with_(name="llama3_8b_bf16_chain_bs1_catchup70", n_new=(70, 70)),
                       [0])


@pytest.mark.slow
def test_full_8b_bs16_catchup():
    from synth import new_counts
    n = new_counts(L3_8B_BS16_CATCHUP)
    run_catchup_parity(L3_8B_BS16_CATCHUP, sorted({int(np.argmin(n)), int(np.argmax(n)), 15}))
