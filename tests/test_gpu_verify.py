"""GPU parity of the verification step (Sec. 2) through the C ABI against the
CPU oracle, on synthetic target logits: greedy and sampled chain
verification, greedy verification of trees drafted by the GPU path.  The
inputs are the same fp32 logits on both sides, so the decisions are compared
exactly; a sampled decision that falls within rounding of its threshold is
reported and checked only for validity."""
import numpy as np
import pytest
import torch

from oracle import softmax_t, verify_chain_greedy, verify_chain_sample, verify_tree_greedy
from synth import (L3_8B_BS16, L3_8B_TREE, SMALL_BF16_CHAIN, SMALL_BF16_TREE, host_inputs,
                   host_weights, make_inputs, make_verify_chain, make_verify_tree_targets,
                   make_weights, scoring_target)
from harness import LOGIT_TOL, MARGIN, check_draft_kv, check_token, gpu_setup, log

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _drafter(cfg):
    from paper_2602_01762_amd import Drafter
    return Drafter(cfg)


def _near_threshold(tl, dl, drafts, T, r, n_gpu):
    """True when the oracle's decision at the first differing position is
    within rounding of its threshold (fp32 on the GPU, fp64 here)."""
    for i in range(min(n_gpu + 1, len(drafts))):
        pt, pd = softmax_t(tl[i], T), softmax_t(dl[i], T)
        x = int(drafts[i])
        if abs(r[i] - min(1.0, pt[x] / pd[x])) < 1e-5:
            return True
    return False


def run_chain_verify(cfg, B, K, T, seed):
    dr = _drafter(cfg)
    d = make_verify_chain(cfg.vocab, B, K, seed=seed, device="cuda")
    out = dr.verify_chain(d["target_logits"], d["draft_tokens"], T,
                          d["draft_logits"] if T > 0 else None, d["uniforms"] if T > 0 else None)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    n, nxt = out["n"].cpu().numpy(), out["next"].cpu().numpy()
    tl = d["target_logits"].cpu().numpy().astype(np.float64)
    dl = d["draft_logits"].cpu().numpy().astype(np.float64)
    tok = d["draft_tokens"].cpu().numpy()
    u = d["uniforms"].cpu().numpy().astype(np.float64)
    near, same = 0, 0
    for b in range(B):
        if T == 0:
            ref = verify_chain_greedy(tl[b], tok[b])
            assert (int(n[b]), int(nxt[b])) == (ref["n"], ref["next"]), b
            continue
        ref = verify_chain_sample(tl[b], dl[b], tok[b], T, u[b])
        if int(n[b]) != ref["n"]:
            assert _near_threshold(tl[b], dl[b], tok[b], T, u[b], int(n[b])), (
                "seq %d: gpu kept %d, oracle %d" % (b, n[b], ref["n"]))
            near += 1
            continue
        # the final draw: u_K must fall in the drawn id's interval of the
        # oracle's CDF, up to fp32 summation over V terms (1e-4 of the total)
        k = int(n[b])
        pt = softmax_t(tl[b, k], T)
        wts = np.maximum(0.0, pt - softmax_t(dl[b, k], T)) if k < K else pt
        if wts.sum() <= 0.0:
            wts = pt
        cdf = np.cumsum(wts)
        t = int(nxt[b])
        goal, tot = u[b, K] * cdf[-1], cdf[-1]
        lo = cdf[t - 1] if t > 0 else 0.0
        assert wts[t] > 0.0 and lo - 1e-4 * tot <= goal < cdf[t] + 1e-4 * tot, (
            "seq %d: drawn %d, oracle %d" % (b, t, ref["next"]))
        same += int(t == ref["next"])
    dr.close()
    return {"accepted": n.tolist(), "near_threshold": near, "draws_equal_oracle": same}


@pytest.mark.parametrize("T", [0.0, 1.0, 0.8])
def test_verify_chain_small(T):
    res = run_chain_verify(SMALL_BF16_CHAIN.with_(batch=8), 8, 4, T, seed=3)
    log("verify chain T=%g" % T, res)
    assert len(set(res["accepted"])) > 1


def test_verify_tree_of_drafted_tree():
    cfg = SMALL_BF16_TREE
    dr, w, inp = gpu_setup(cfg)
    tr = dr.tree(inp)
    tl = make_verify_tree_targets(tr["tokens"], tr["parent"], cfg.vocab, seed=4)
    out = dr.verify_tree(tl, tr["tokens"], tr["parent"])
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    tln = tl.cpu().numpy().astype(np.float64)
    tk, pa = tr["tokens"].cpu().numpy(), tr["parent"].cpu().numpy()
    lens = []
    for b in range(cfg.batch):
        ref = verify_tree_greedy(tln[b], tk[b], pa[b])
        assert int(out["n"][b]) == ref["n"]
        got = out["path"][b].cpu().numpy()
        assert list(got[:ref["n"]]) == ref["path"] and np.all(got[ref["n"]:] == -1)
        assert int(out["next"][b]) == ref["next"]
        lens.append(ref["n"])
    log("verify tree accepted", lens)
    dr.close()


@pytest.mark.slow
@pytest.mark.parametrize("T", [0.0, 1.0])
def test_verify_chain_full_vocab(T):
    res = run_chain_verify(L3_8B_BS16, 16, 5, T, seed=7)
    log("verify chain 8B vocab T=%g" % T, res)


@pytest.mark.slow
def test_verify_tree_full_vocab():
    cfg = L3_8B_TREE
    dr = _drafter(cfg)
    B, v = cfg.batch, cfg.tree_nodes
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    # a random tree in the drafter's output order (every parent precedes its children)
    parent = torch.full((B, v), -1, dtype=torch.int32)
    for b in range(B):
        for j in range(v):
            parent[b, j] = int(torch.randint(-1, j, (1,), generator=torch.Generator().manual_seed(b * 97 + j))) if j else -1
    tokens = torch.randint(0, cfg.vocab, (B, v), generator=g, device="cuda", dtype=torch.int32)
    parent = parent.cuda()
    tl = make_verify_tree_targets(tokens, parent, cfg.vocab, seed=6)
    out = dr.verify_tree(tl, tokens, parent)
    torch.cuda.synchronize()
    tln = tl.cpu().numpy().astype(np.float64)
    for b in range(B):
        ref = verify_tree_greedy(tln[b], tokens[b].cpu().numpy(), parent[b].cpu().numpy())
        assert int(out["n"][b]) == ref["n"] and int(out["next"][b]) == ref["next"]
    dr.close()


def run_score_tree(cfg, seqs=None):
    """Draft a tree with the GPU drafter, score it with a GPU target model
    (one layer of the drafter's shape with its own weights, its feature input
    zero) under the tree mask, verify it greedily, and compare with the
    oracle: the target's logits of every row (root and nodes), the target KV
    it wrote, and the accepted path."""
    from oracle import Oracle
    from paper_2602_01762_amd import Drafter
    log("score tree", cfg.name)
    dr, w, inp = gpu_setup(cfg)
    tr = dr.tree(inp, debug=False)
    torch.cuda.synchronize()
    assert dr.device_status() == 0
    tcfg = scoring_target(cfg)
    wt = make_weights(tcfg.with_(seed=7), "cuda")
    it = make_inputs(tcfg, "cuda")
    it.features.zero_()
    assert torch.equal(it.tokens, inp.tokens) and torch.equal(it.ctx_lens, inp.ctx_lens)
    tdr = Drafter(tcfg, max_batch=64)        # bf16: passes of whole trees, up to 256 rows
    tdr.load(wt)
    lg = tdr.score_tree(it, tr["tokens"], tr["depth"], tr["mask"])
    again = tdr.score_tree(it, tr["tokens"], tr["depth"], tr["mask"])
    ver = tdr.verify_tree(lg, tr["tokens"], tr["parent"])
    torch.cuda.synchronize()
    assert tdr.device_status() == 0
    assert torch.equal(lg, again)
    seqs = list(range(cfg.batch)) if seqs is None else seqs
    toks, depth = tr["tokens"].cpu().numpy(), tr["depth"].cpu().numpy()
    mask, parent = tr["mask"].cpu().numpy(), tr["parent"].cpu().numpy()
    ref = Oracle(tcfg, host_weights(wt)).score_tree(host_inputs(it, tcfg, seqs), toks, depth,
                                                    mask, seqs)
    g = lg.cpu().numpy().astype(np.float64)
    err, lens = 0.0, []
    for b in seqs:
        e = float(np.max(np.abs(g[b] - ref["logits"][b])))
        assert e <= LOGIT_TOL[cfg.dtype], "seq %d: logits max-abs %.3g" % (b, e)
        err = max(err, e)
        for r in range(cfg.tree_nodes + 1):
            check_token(ref["logits"][b, r], int(np.argmax(g[b, r])), "seq %d row %d" % (b, r))
        # verification of the GPU's logits is exact; on the oracle's logits it
        # agrees unless a choice on the path is a near tie
        mine = verify_tree_greedy(g[b], toks[b], parent[b])
        n = int(ver["n"][b])
        assert (n, int(ver["next"][b])) == (mine["n"], mine["next"])
        assert list(ver["path"][b].cpu().numpy()[:n]) == mine["path"]
        theirs = verify_tree_greedy(ref["logits"][b], toks[b], parent[b])
        if theirs["path"] != mine["path"]:
            at = -1
            for node in mine["path"] + [None]:
                row = ref["logits"][b, at + 1]
                top = np.sort(row)[::-1]
                if top[0] - top[1] <= MARGIN:
                    break
                assert node is not None, "seq %d: paths differ without a near tie" % b
                at = node
        lens.append(n)
    check_draft_kv(tcfg, it, ref["draft_kv"], seqs)
    log(cfg.name, "target logits max-abs %.3g, accepted %s" % (err, lens))
    tdr.close()
    dr.close()
    return lens


def test_score_tree_and_verify_small():
    lens = run_score_tree(SMALL_BF16_TREE)
    assert len(lens) == SMALL_BF16_TREE.batch


def test_score_tree_and_verify_small_empty_context():
    run_score_tree(SMALL_BF16_TREE.with_(name="small_bf16_tree_ctx0", ctx_range=None, ctx_len=0))


def test_score_tree_and_verify_small_two_passes():
    """4 trees x 21 rows = 84 rows: one scoring pass of more than 64 rows
    (the row-group products over a full and a ragged row group, the trees'
    rows grouped by 4 in the attention, 5 groups per tree, the last of one
    row)."""
    lens = run_score_tree(SMALL_BF16_TREE.with_(name="small_bf16_tree_b4", batch=4))
    assert len(lens) == 4


def test_score_tree_and_verify_small_two_groups():
    """13 trees x 21 rows = 273 rows: two scoring passes of whole trees (12
    trees in 252 rows, then one in 21), the second one's nodes attending to
    KV that the first one wrote."""
    lens = run_score_tree(SMALL_BF16_TREE.with_(name="small_bf16_tree_b13", batch=13))
    assert len(lens) == 13


def test_score_tree_and_verify_small_f32():
    """fp32: 4 trees x 21 rows = 84 rows in passes of up to 64 rows (64, then
    20, the second one's nodes attending to KV the first one wrote), each pass
    with its own LM head; the attention ungrouped."""
    lens = run_score_tree(SMALL_BF16_TREE.with_(name="small_f32_tree_b4", dtype="f32", batch=4))
    assert len(lens) == 4


@pytest.mark.parametrize("nodes", [1, 2])
def test_score_tree_and_verify_one_tiny_tree(nodes):
    """One tree of 1 or 2 nodes: a scoring pass of 2 or 3 rows (the 2-row
    one on the GEMV products), an attention group smaller than its 4-row
    group size, and the LM head over a partial row tile."""
    cfg = SMALL_BF16_TREE.with_(name="small_bf16_tree_v%d" % nodes, batch=1, n_steps=2,
                                tree_width=2, tree_nodes=nodes)
    lens = run_score_tree(cfg)
    assert len(lens) == 1


def test_score_tree_and_verify_small_h480():
    """Hidden size 480: 15 k-blocks per row (odd, so the LM head's single K
    slice ends with a k-block of zero activations), 30 output tiles in the
    480-wide products (a tile group with waves past the last tile), no
    embedding table; 5 trees = 105 rows in one row-group pass."""
    lens = run_score_tree(SMALL_BF16_TREE.with_(name="small_bf16_tree_h480_b5", batch=5,
                                                hidden=480, feat_width=1440))
    assert len(lens) == 5


def test_score_tree_and_verify_small_mha():
    """One query head per KV head: 16 rows per attention workgroup, so each
    21-row tree is a group of 16 and one of 5; 5 trees = 105 rows in one
    row-group pass."""
    lens = run_score_tree(SMALL_BF16_TREE.with_(name="small_bf16_tree_mha_b5", batch=5,
                                                n_kv_heads=8))
    assert len(lens) == 5


def test_score_tree_graph_replay_reads_new_tokens():
    """A second scoring call on the same buffers replays the captured graph;
    with new token ids written into the tree buffers in place, its logits
    follow the new tokens (the oracle scores the changed tree), and the
    call count of captured graphs does not grow."""
    from oracle import Oracle
    from paper_2602_01762_amd import Drafter
    cfg = SMALL_BF16_TREE.with_(name="small_bf16_tree_b4_replay", batch=4)
    dr, w, inp = gpu_setup(cfg)
    tr = dr.tree(inp, debug=False)
    tcfg = scoring_target(cfg)
    wt = make_weights(tcfg.with_(seed=7), "cuda")
    it = make_inputs(tcfg, "cuda")
    it.features.zero_()
    tdr = Drafter(tcfg, max_batch=64)
    tdr.load(wt)
    lg = tdr.score_tree(it, tr["tokens"], tr["depth"], tr["mask"])
    torch.cuda.synchronize()
    from paper_2602_01762_amd import binding as B
    n_graphs = B.prism_graph_cache(tdr.ctx)[0]
    tr["tokens"].copy_((tr["tokens"] * 7 + 3) % cfg.vocab)     # a valid tree with other tokens
    lg2 = tdr.score_tree(it, tr["tokens"], tr["depth"], tr["mask"], out=lg)
    torch.cuda.synchronize()
    assert tdr.device_status() == 0
    assert B.prism_graph_cache(tdr.ctx)[0] == n_graphs
    seqs = list(range(cfg.batch))
    ref = Oracle(tcfg, host_weights(wt)).score_tree(
        host_inputs(it, tcfg, seqs), tr["tokens"].cpu().numpy(), tr["depth"].cpu().numpy(),
        tr["mask"].cpu().numpy(), seqs)
    g = lg2.cpu().numpy().astype(np.float64)
    for b in seqs:
        e = float(np.max(np.abs(g[b] - ref["logits"][b])))
        assert e <= LOGIT_TOL[cfg.dtype], "seq %d: logits max-abs %.3g" % (b, e)
    tdr.close()
    dr.close()


def test_score_tree_rows_are_checked():
    """A mask that names a later node or lacks the node's own bit, and a
    depth out of range, are clamped to well-formed rows and reported."""
    from paper_2602_01762_amd import Drafter
    cfg = SMALL_BF16_TREE
    tcfg = scoring_target(cfg)
    it = make_inputs(tcfg, "cuda")
    tdr = Drafter(tcfg, max_batch=64)
    tdr.load(make_weights(tcfg.with_(seed=7), "cuda"))
    v = cfg.tree_nodes
    toks = torch.zeros((cfg.batch, v), dtype=torch.int32, device="cuda")
    depth = torch.ones((cfg.batch, v), dtype=torch.int32, device="cuda")
    mask = (torch.ones((cfg.batch, v), dtype=torch.int64, device="cuda")
            << torch.arange(v, device="cuda"))
    tdr.score_tree(it, toks, depth, mask)
    torch.cuda.synchronize()
    assert tdr.device_status() == 0
    for bad in ("mask_later", "mask_self", "depth"):
        m, dp = mask.clone(), depth.clone()
        if bad == "mask_later":
            m[0, 3] |= 1 << 5
        elif bad == "mask_self":
            m[1, 4] = 1
        else:
            dp[0, 2] = v + 1
        tdr.score_tree(it, toks, dp, m)
        torch.cuda.synchronize()
        assert tdr.device_status() == -1, bad
    tdr.close()


@pytest.mark.slow
def test_score_tree_and_verify_full_8b():
    run_score_tree(L3_8B_TREE, seqs=[0])
