"""Pins of the CPU oracle against facts fixed by the mathematics.

The paper prints no worked example or intermediate values, so every pin here
is a closed form, an invariant, a special case that reduces to a simpler
computation, brute force on tiny inputs, or an independent library
formulation.  Each is chosen so that a plausible mistake (dropped term, wrong
sign or index, transposed operand, wrong head mapping, wrong position or slot,
wrong parameter set) fails at least one test.
"""
import copy

import numpy as np
import pytest
import torch

import oracle
from oracle import Oracle, brute_chain, round_bf16, rmsnorm, silu, rope, softmax_attend
from oracle import logsumexp, topk_ids, widen, sample_inverse_cdf
from synth import DraftConfig, make_weights, make_inputs, host_weights, host_inputs

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

TINY = DraftConfig(name="pin_tiny", hidden=32, n_q_heads=4, n_kv_heads=2, head_dim=8, ffn=48,
                   vocab=64, n_steps=3, feat_width=48, rope_theta=10000.0, dtype="f32",
                   batch=2, ctx_len=0, ctx_range=(3, 9), kv_block_size=4, shuffle_blocks=True)
TINY_BF16 = TINY.with_(name="pin_tiny_bf16", dtype="bf16")


def build(cfg):
    w = make_weights(cfg)
    i = make_inputs(cfg)
    return host_weights(w), host_inputs(i, cfg)


# ------------------------------------------------------------------ T0 closed forms
def test_round_bf16_matches_ieee_rne():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(100000).astype(np.float32)
    x = np.concatenate([x, x * 1e-30, x * 1e30]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(round_bf16(x.astype(np.float64)), ref)


def test_round_bf16_ties_to_even():
    one = 1.0
    ulp = 2.0 ** -7                       # bf16 spacing in [1, 2)
    assert round_bf16(np.array([one + ulp / 2]))[0] == one             # tie -> even (1.0)
    assert round_bf16(np.array([one + 3 * ulp / 2]))[0] == one + 2 * ulp  # tie -> even
    assert round_bf16(np.array([one + ulp / 2 + 1e-12]))[0] == one + ulp
    assert round_bf16(np.array([-(one + ulp / 2)]))[0] == -one
    assert np.isnan(round_bf16(np.array([np.nan]))[0])
    assert round_bf16(np.array([0.0]))[0] == 0.0


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(1)
    d, T = 16, 37
    q = rng.standard_normal(d)
    K = rng.standard_normal((T, d)) * 3
    # V = identity rows: the output is the probability vector itself
    V = np.eye(T)
    p = softmax_attend(q, K, V)
    assert abs(p.sum() - 1.0) < 1e-12
    s = K @ q / np.sqrt(d)
    assert np.allclose(p, np.exp(s) / np.exp(s).sum(), rtol=1e-12, atol=0)


def test_single_key_attention_returns_value():
    rng = np.random.default_rng(2)
    v = rng.standard_normal((1, 8))
    assert np.array_equal(softmax_attend(rng.standard_normal(8), rng.standard_normal((1, 8)), v), v[0])


def test_logsumexp_normalises():
    x = np.random.default_rng(3).standard_normal(1000) * 5
    lp = x - logsumexp(x)
    assert abs(logsumexp(lp)) < 1e-12
    assert abs(np.exp(lp).sum() - 1) < 1e-12


def test_rmsnorm_unit_rms():
    x = np.random.default_rng(4).standard_normal((3, 64)) * 7
    y = rmsnorm(x, np.ones(64), 0.0)
    assert np.allclose(np.sqrt((y * y).mean(-1)), 1.0, atol=1e-14)
    g = np.arange(64) / 10.0
    assert np.allclose(rmsnorm(x, g, 0.0), y * g, atol=1e-14)
    # eps enters under the root: constant rows c give c / sqrt(c^2 + eps)
    c = np.full((1, 8), 0.01)
    assert np.allclose(rmsnorm(c, np.ones(8), 1e-4), 0.01 / np.sqrt(1e-4 + 1e-4))


def test_silu_closed_forms():
    y = np.linspace(-20, 20, 101)
    assert silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(silu(y) - silu(-y), y, atol=1e-12)
    assert np.allclose(silu(np.array([1.0])), 1 / (1 + np.exp(-1)))


def test_rope_rotation_convention():
    # d = 2: one pair, frequency theta^0 = 1, so position p rotates by p radians
    x = np.array([1.0, 0.0])
    for p in (0, 1, 5, 4000):
        y = rope(x, p, 10000.0)
        assert np.allclose(y, [np.cos(p), np.sin(p)], atol=1e-7)
    # d = 4, second pair (i=1) turns at theta^(-2/4)
    x = np.array([0.0, 1.0, 0.0, 0.0])   # x_1 pairs with x_3
    p, th = 7, 100.0
    phi = p * th ** -0.5
    assert np.allclose(rope(x, p, th), [0, np.cos(phi), 0, np.sin(phi)], atol=1e-7)


def test_rope_invariants():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 64))
    assert np.array_equal(rope(x, 0, 5e5), x)
    y = rope(x, 123, 5e5)
    n0 = x[:, :32] ** 2 + x[:, 32:] ** 2
    n1 = y[:, :32] ** 2 + y[:, 32:] ** 2
    assert np.allclose(n0, n1, rtol=1e-6)
    # relative position: <R(p)q, R(t)k> depends only on p - t
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    a = rope(q, 50, 1e4) @ rope(k, 20, 1e4)
    b = rope(q, 130, 1e4) @ rope(k, 100, 1e4)
    assert abs(a - b) < 1e-5 * (abs(a) + 1)


def test_topk_tie_break_lowest_index():
    v = np.array([1.0, 3.0, 3.0, 2.0, 3.0])
    assert list(topk_ids(v, 3)) == [1, 2, 4]


def test_native_linear_matches_numpy():
    rng = np.random.default_rng(6)
    W32 = rng.standard_normal((37, 50)).astype(np.float32)
    Wbf = (torch.from_numpy(W32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))
    X = rng.standard_normal((3, 50))
    for W in (W32, Wbf):
        ref = X @ widen(W).T
        assert np.allclose(oracle.linear(W, X, use_c=True), ref, rtol=1e-13, atol=1e-13)
        assert np.allclose(oracle.linear(W, X, use_c=False), ref, rtol=1e-13, atol=1e-13)


# ------------------------------------------------------------------ T1 brute force
@pytest.mark.parametrize("cfg", [TINY, TINY_BF16], ids=lambda c: c.dtype)
def test_chain_equals_brute_force(cfg):
    hw, hi = build(cfg)
    orc = Oracle(cfg, hw)
    inc = orc.chain(hi)
    bf = brute_chain(orc, hi, cfg.n_steps)
    assert np.array_equal(inc["tokens"], bf["tokens"])
    assert np.max(np.abs(inc["hidden"] - bf["hidden"])) < 1e-12


# ------------------------------------------------------------------ T1b catch-up prefill
TINY_CU = TINY.with_(name="pin_tiny_catchup", batch=4, n_new=(1, 4))


@pytest.mark.parametrize("cfg", [TINY_CU, TINY_CU.with_(dtype="bf16")], ids=lambda c: c.dtype)
def test_catchup_chain_equals_brute_force(cfg):
    hw, hi = build(cfg)
    n = np.diff(hi["new_offsets"])
    assert n.min() == 1 and n.max() > 2        # ragged, including a single-token sequence
    orc = Oracle(cfg, hw)
    inc = orc.chain(hi, catchup=True)
    bf = brute_chain(orc, hi, cfg.n_steps, catchup=True)
    assert np.array_equal(inc["tokens"], bf["tokens"])
    assert np.max(np.abs(inc["hidden"] - bf["hidden"])) < 1e-12


def test_catchup_of_one_token_is_plain_chain():
    cfg = TINY_CU.with_(n_new=(1, 1))
    hw, hi = build(cfg)
    orc = Oracle(cfg, hw)
    a, b = orc.chain(hi, catchup=True), orc.chain(hi)
    assert np.array_equal(a["tokens"], b["tokens"])
    assert np.array_equal(a["logits"], b["logits"])


def test_catchup_block_prefill_equals_row_by_row():
    # one pass over all accepted rows (causal among them) equals feeding the
    # rows one at a time, each after the previous one's KV is written
    cfg = TINY_CU
    hw, hi = build(cfg)
    orc = Oracle(cfg, hw)
    ref = orc.chain(hi, catchup=True)
    s1 = cfg.fmap[0]
    for b in range(cfg.batch):
        cache = {b: orc.new_cache(hi, b)}
        L = cache[b]["L"]
        o0, o1 = int(hi["new_offsets"][b]), int(hi["new_offsets"][b + 1])
        for i in range(o1 - o0):
            f = widen(hi["new_features"][o0 + i])[None]
            h, lg = orc.forward(s1, [int(hi["new_tokens"][o0 + i])], f, [L + i], cache, [b],
                                [L + i], [list(range(L + i + 1))])
        p = L + o1 - o0
        for k in range(1, cfg.n_steps + 1):
            if k > 1:
                h, lg = orc.forward(cfg.fmap[k - 1], [x], h, [p], cache, [b], [p],
                                    [list(range(p + 1))])
                p += 1
            assert np.max(np.abs(lg[0] - ref["logits"][b, k - 1])) < 1e-12
            x = int(np.argmax(lg[0]))
        assert sorted(cache[b]["draft"]) == sorted(ref["draft_kv"][b])
        for slot, (kk, vv) in cache[b]["draft"].items():
            rk, rv = ref["draft_kv"][b][slot]
            assert np.array_equal(kk, rk) and np.array_equal(vv, rv)


# ------------------------------------------------------------------ T1c stochastic drafting
def test_inverse_cdf_frequencies_match_softmax():
    # u on a regular grid: the share of grid points mapped to token t is its
    # probability up to the grid step; the returned log-prob is log p_t
    lg = np.random.default_rng(3).standard_normal(7) * 2.0
    N = 20000
    for T in (0.5, 1.0, 2.0):
        p = np.exp(lg / T - (lg / T).max())
        p /= p.sum()
        counts = np.zeros(len(lg))
        for i in range(N):
            t, lp = sample_inverse_cdf(lg, T, (i + 0.5) / N)
            counts[t] += 1
            assert abs(lp - np.log(p[t])) < 1e-12
        assert np.max(np.abs(counts / N - p)) <= 1.0 / N + 1e-12


def test_inverse_cdf_edges():
    lg = np.array([0.3, -1.0, 2.0, 0.5])
    assert sample_inverse_cdf(lg, 1.0, 0.0)[0] == 0
    assert sample_inverse_cdf(lg, 1.0, float(np.nextafter(1.0, 0.0)))[0] == 3
    for u in (0.01, 0.5, 0.99):      # a cold temperature puts the mass on the argmax
        assert sample_inverse_cdf(lg, 1e-3, u)[0] == 2


@pytest.mark.parametrize("cfg", [TINY, TINY_BF16], ids=lambda c: c.dtype)
def test_sampled_chain_equals_brute_force(cfg):
    scfg = cfg.with_(temperature=1.0)
    hw, hi = build(scfg)
    orc = Oracle(scfg, hw)
    inc = orc.chain(hi, temperature=1.0, uniforms=hi["uniforms"])
    bf = brute_chain(orc, hi, scfg.n_steps, temperature=1.0, uniforms=hi["uniforms"])
    assert np.array_equal(inc["tokens"], bf["tokens"])
    assert np.max(np.abs(inc["hidden"] - bf["hidden"])) < 1e-12
    greedy = orc.chain(hi)
    assert not np.array_equal(inc["tokens"], greedy["tokens"])   # the draws matter
    lse = np.array([[logsumexp(inc["logits"][b, k]) for k in range(scfg.n_steps)]
                    for b in range(scfg.batch)])
    picked = np.take_along_axis(inc["logits"], inc["tokens"][..., None], axis=2)[..., 0]
    assert np.max(np.abs(inc["logp"] - (picked - lse))) < 1e-12


# ------------------------------------------------------------------ T1d empty prior context
# The prefill from an initial KV cache that holds nothing yet (Sec. 3.2: the
# first draft pass starts from KV_(0)): every sequence, or some of a ragged
# batch, has L_b = 0, so its first row attends to its own slot only.
TINY_EMPTY = TINY.with_(name="pin_tiny_empty", ctx_range=None, ctx_len=0)
TINY_MIXED = TINY.with_(name="pin_tiny_mixed", batch=6, ctx_range=(0, 3))   # L_b = 1 2 3 1 3 0


@pytest.mark.parametrize("cfg", [TINY_EMPTY, TINY_EMPTY.with_(dtype="bf16"), TINY_MIXED],
                         ids=["f32", "bf16", "mixed"])
def test_empty_prior_context_chain_equals_brute_force(cfg):
    hw, hi = build(cfg)
    assert (hi["ctx_lens"] == 0).any()
    orc = Oracle(cfg, hw)
    inc = orc.chain(hi)
    bf = brute_chain(orc, hi, cfg.n_steps)
    assert np.array_equal(inc["tokens"], bf["tokens"])
    assert np.max(np.abs(inc["hidden"] - bf["hidden"])) < 1e-12


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_empty_prior_context_catchup_equals_brute_force(dtype):
    cfg = TINY_EMPTY.with_(batch=3, n_new=(2, 4), dtype=dtype)
    hw, hi = build(cfg)
    orc = Oracle(cfg, hw)
    inc = orc.chain(hi, catchup=True)
    bf = brute_chain(orc, hi, cfg.n_steps, catchup=True)
    assert np.array_equal(inc["tokens"], bf["tokens"])
    assert np.max(np.abs(inc["hidden"] - bf["hidden"])) < 1e-12
    # the accepted rows sit at slots 0 .. n_b - 1, the chain right after them
    for b in range(cfg.batch):
        n = int(hi["new_offsets"][b + 1] - hi["new_offsets"][b])
        assert sorted(inc["draft_kv"][b]) == list(range(n + cfg.n_steps - 1))


def test_empty_prior_context_first_step_attends_to_itself():
    # with L_b = 0 the first row sees one key, its own, so each head's
    # attention output is its KV head's stored value: o_h = v_(h // g), and
    # the first step equals a forward pass whose attention is replaced by
    # that copy (a different computation of the same quantity)
    cfg = TINY_EMPTY
    hw, hi = build(cfg)
    orc = Oracle(cfg, hw)
    ch = orc.chain(hi, K=1)
    P = hw["sets"][cfg.fmap[0]]
    g = cfg.n_q_heads // cfg.n_kv_heads
    for b in range(cfg.batch):
        x = np.concatenate([widen(hw["embed"][int(hi["tokens"][b])]), widen(hi["features"][b])])
        u = widen(P["w_fc"]) @ x
        a = rmsnorm(u, widen(P["g1"]), cfg.rms_eps)
        v = orc.store(widen(P["w_v"]) @ a).reshape(cfg.n_kv_heads, cfg.head_dim)
        o = np.concatenate([v[h // g] for h in range(cfg.n_q_heads)])
        r1 = u + widen(P["w_o"]) @ o
        m = rmsnorm(r1, widen(P["g2"]), cfg.rms_eps)
        hid = r1 + widen(P["w_down"]) @ (silu(widen(P["w_gate"]) @ m) * (widen(P["w_up"]) @ m))
        assert np.max(np.abs(hid - ch["hidden"][b, 0])) < 1e-12


@pytest.mark.parametrize("cfg", [TINY_EMPTY, TINY_EMPTY.with_(dtype="bf16")], ids=["f32", "bf16"])
def test_empty_prior_context_tree_nodes_equal_forced_chains(cfg):
    tcfg = cfg.with_(mode="tree", n_steps=3, tree_width=3, tree_nodes=10)
    hw, hi = build(tcfg)
    orc = Oracle(tcfg, hw)
    tr = orc.tree(hi)
    for b in range(tcfg.batch):
        c = tr[b]["cand"]
        for ps in tr[b]["passes"]:
            d, n, path = ps["depth"], ps["cand"], []
            while n >= 0:
                path.append(int(c["token"][n]))
                n = int(c["parent"][n])
            forced = np.zeros((tcfg.batch, d + 1), dtype=np.int64)
            forced[b, :d] = path[::-1]
            ch = orc.chain(hi, K=d + 1, forced=forced, seqs=[b])
            assert np.max(np.abs(ch["logits"][b, d] - ps["logits"])) < 1e-12


# ------------------------------------------------------------------ T2 tree = chains
@pytest.mark.parametrize("cfg", [TINY, TINY_BF16], ids=lambda c: c.dtype)
def test_tree_nodes_equal_forced_chains(cfg):
    tcfg = cfg.with_(mode="tree", n_steps=3, tree_width=3, tree_nodes=10)
    hw, hi = build(tcfg)
    orc = Oracle(tcfg, hw)
    tr = orc.tree(hi)
    for b in range(tcfg.batch):
        c = tr[b]["cand"]
        for ps in tr[b]["passes"]:
            d = ps["depth"]
            path = []
            n = ps["cand"]
            while n >= 0:
                path.append(int(c["token"][n]))
                n = int(c["parent"][n])
            path = path[::-1]
            assert len(path) == d
            forced = np.zeros((tcfg.batch, d + 1), dtype=np.int64)
            forced[b, :d] = path
            ch = orc.chain(hi, K=d + 1, forced=forced, seqs=[b])
            assert np.max(np.abs(ch["logits"][b, d] - ps["logits"])) < 1e-12
            assert np.max(np.abs(ch["hidden"][b, d] - ps["hidden"])) < 1e-12


def test_tree_width_one_is_chain():
    tcfg = TINY.with_(mode="tree", n_steps=3, tree_width=1, tree_nodes=3)
    hw, hi = build(tcfg)
    orc = Oracle(tcfg, hw)
    tr = orc.tree(hi)
    ch = orc.chain(hi, K=3)
    for b in range(tcfg.batch):
        assert list(tr[b]["tokens"]) == list(ch["tokens"][b])
        lp = [ch["logits"][b, k, ch["tokens"][b, k]] - logsumexp(ch["logits"][b, k]) for k in range(3)]
        assert np.allclose(tr[b]["score"], np.cumsum(lp), atol=1e-12)
        assert list(tr[b]["parent"]) == [-1, 0, 1]
        assert [int(m) for m in tr[b]["mask"]] == [1, 3, 7]


def test_tree_all_candidates_when_v_large():
    tcfg = TINY.with_(mode="tree", n_steps=3, tree_width=2, tree_nodes=2 + 2 * 4)
    hw, hi = build(tcfg)
    tr = Oracle(tcfg, hw).tree(hi)
    for b in range(tcfg.batch):
        assert sorted(tr[b]["nodes"]) == list(range(tcfg.n_candidates))
        sc = tr[b]["score"]
        assert np.all(np.diff(sc) <= 0)
        # ancestor closure: every parent precedes its child and is in the set
        for i, p in enumerate(tr[b]["parent"]):
            assert p < i
            if p >= 0:
                assert tr[b]["depth"][p] == tr[b]["depth"][i] - 1


def test_tree_frontier_is_topw_of_children():
    tcfg = TINY.with_(mode="tree", n_steps=3, tree_width=3, tree_nodes=8)
    hw, hi = build(tcfg)
    tr = Oracle(tcfg, hw).tree(hi)
    w = 3
    for b in range(tcfg.batch):
        c = tr[b]["cand"]
        f1 = tr[b]["frontiers"][1]
        kids = np.arange(w, w + w * w)
        best = kids[np.argsort(-c["score"][kids], kind="stable")[:w]]
        assert list(f1) == list(best)
        # every child score is parent score + a log-prob (<= parent score)
        for n in kids:
            assert c["score"][n] <= c["score"][c["parent"][n]] + 1e-15


# ------------------------------------------------------------------ T2b the final cut
def _cut_by_brute_force(c, v):
    """The final top-v of a candidate list, from the definitions alone.

    Rank = number of candidates that come first under (score desc, creation
    index asc), counted pair by pair.  Each kept candidate's path is walked
    explicitly through the candidate parents; its output parent is the
    output position of the path's second node, its depth the path's length,
    its mask the output positions of the whole path.  Returns the kept
    candidates in rank order and, for each, (token, parent, depth, score,
    mask), plus whether every kept node's ancestors were kept."""
    n = len(c["score"])
    sc = [float(x) for x in c["score"]]
    rank = [sum(1 for j in range(n) if sc[j] > sc[i] or (sc[j] == sc[i] and j < i))
            for i in range(n)]
    kept = sorted((i for i in range(n) if rank[i] < v), key=lambda i: rank[i])
    pos = {cand: k for k, cand in enumerate(kept)}
    rows, closed = [], True
    for cand in kept:
        path = []
        x = cand
        while x >= 0:
            path.append(x)
            x = int(c["parent"][x])
        closed &= all(a in pos for a in path)
        parent = pos.get(path[1], -99) if len(path) > 1 else -1
        mask = sum(1 << pos[a] for a in path if a in pos)
        rows.append((int(c["token"][cand]), parent, len(path), sc[cand], mask))
    return kept, rows, closed


@pytest.mark.parametrize("cfg", [TINY, TINY_BF16, TINY_EMPTY], ids=["f32", "bf16", "empty"])
@pytest.mark.parametrize("v", [5, 8, 17])
def test_tree_cut_equals_brute_force(cfg, v):
    # w = 3, D = 3: 3 + 2 * 9 = 21 candidates, cut to v < 21
    tcfg = cfg.with_(mode="tree", n_steps=3, tree_width=3, tree_nodes=v)
    hw, hi = build(tcfg)
    orc = Oracle(tcfg, hw)
    tr = orc.tree(hi)
    for b in range(tcfg.batch):
        c = tr[b]["cand"]
        assert len(c["score"]) == tcfg.n_candidates == 21
        kept, rows, closed = _cut_by_brute_force(c, v)
        assert closed, "the cut must keep every ancestor of a kept node"
        assert [int(x) for x in tr[b]["nodes"]] == kept
        got = list(zip([int(x) for x in tr[b]["tokens"]], [int(x) for x in tr[b]["parent"]],
                       [int(x) for x in tr[b]["depth"]], [float(x) for x in tr[b]["score"]],
                       [int(x) for x in tr[b]["mask"]]))
        assert got == rows
        # the cut reaches below depth 1 and is not the whole list
        assert max(r[2] for r in rows) >= 2 and len(kept) < 21
        # every candidate's score is the sum of its path's log-probs, each
        # taken from a chain forced along the path
        for cand in range(21):
            path, x = [], cand
            while x >= 0:
                path.append(x)
                x = int(c["parent"][x])
            path = path[::-1]
            toks = [int(c["token"][a]) for a in path]
            forced = np.zeros((tcfg.batch, len(path)), dtype=np.int64)
            forced[b, :] = toks
            ch = orc.chain(hi, K=len(path), forced=forced, seqs=[b])
            lp = sum(ch["logits"][b, k, toks[k]] - logsumexp(ch["logits"][b, k])
                     for k in range(len(path)))
            assert abs(lp - c["score"][cand]) < 1e-12


# ------------------------------------------------------------------ T2c target-side tree scoring
@pytest.mark.parametrize("cfg", [TINY, TINY_BF16, TINY_EMPTY], ids=["f32", "bf16", "empty"])
def test_scored_tree_rows_equal_causal_paths(cfg):
    # the scoring model's row for node j equals a plain causal pass over the
    # root and the path to j (positions L_b, L_b + 1, ...), and its root row a
    # one-row pass at L_b: the tree mask, slots and positions reproduce every
    # branch run on its own
    tcfg = cfg.with_(mode="tree", n_steps=4, tree_width=2, tree_nodes=12)
    hw, hi = build(tcfg)
    tr = Oracle(tcfg, hw).tree(hi)
    assert max(int(x) for b in range(tcfg.batch) for x in tr[b]["depth"]) >= 3
    scfg = tcfg.with_(mode="chain", n_steps=1, feat_width=tcfg.hidden, tree_width=0,
                      tree_nodes=0, draft_slots=1 + tcfg.tree_nodes)
    hs = host_weights(make_weights(scfg.with_(seed=5)))
    feats = np.random.default_rng(2).standard_normal((tcfg.batch, tcfg.hidden))
    his = dict(hi, features=feats)
    sc = Oracle(scfg, hs)
    toks = np.stack([tr[b]["tokens"] for b in range(tcfg.batch)])
    depth = np.stack([tr[b]["depth"] for b in range(tcfg.batch)])
    mask = np.stack([tr[b]["mask"] for b in range(tcfg.batch)])
    got = sc.score_tree(his, toks, depth, mask)["logits"]
    for b in range(tcfg.batch):
        L = int(hi["ctx_lens"][b])
        for j in range(-1, tcfg.tree_nodes):
            path = [] if j < 0 else [a for a in range(j + 1) if (int(mask[b, j]) >> a) & 1]
            rows = [int(hi["tokens"][b])] + [int(toks[b, a]) for a in path]
            n = len(rows)
            assert j < 0 or n - 1 == int(depth[b, j])
            cache = {b: sc.new_cache(his, b)}
            pos = [L + i for i in range(n)]
            _, lg = sc.forward(0, rows, np.stack([feats[b]] * n), pos, cache, [b] * n, pos,
                               [list(range(p + 1)) for p in pos])
            assert np.max(np.abs(lg[-1] - got[b, j + 1])) < 1e-12, (b, j)


# ------------------------------------------------------------------ T3 set isolation
def test_step_k_uses_only_set_k():
    hw, hi = build(TINY)
    base = Oracle(TINY, hw).chain(hi)
    hw2 = copy.deepcopy(hw)
    rng = np.random.default_rng(9)
    for key in ("w_fc", "w_q", "w_down"):
        hw2["sets"][2][key] = (rng.standard_normal(hw2["sets"][2][key].shape) * 0.02).astype(np.float32)
    alt = Oracle(TINY, hw2).chain(hi)
    assert np.array_equal(base["logits"][:, :2], alt["logits"][:, :2])
    assert not np.allclose(base["logits"][:, 2], alt["logits"][:, 2])
    # a set no step maps to may hold NaN without effect
    hw3 = copy.deepcopy(hw)
    cfg2 = TINY.with_(n_steps=2)
    for key in hw3["sets"][2]:
        if key != "feat_width":
            hw3["sets"][2][key] = np.full_like(hw3["sets"][2][key], np.nan)
    two = Oracle(cfg2, hw3).chain(hi)
    assert np.array_equal(two["logits"], base["logits"][:, :2])


# ------------------------------------------------------------------ T4 reductions
def test_identical_sets_equal_single_module():
    cfg = TINY.with_(feat_width=32)              # one set serves every step: F_t = H
    one = cfg.with_(f_map=(0, 0, 0), n_sets=1)
    hw1, hi = build(one)
    hwM = copy.deepcopy(hw1)
    hwM["sets"] = [copy.deepcopy(hw1["sets"][0]) for _ in range(3)]
    a = Oracle(one, hw1).chain(hi)
    b = Oracle(cfg, hwM).chain(hi)
    assert np.array_equal(a["tokens"], b["tokens"])
    assert np.array_equal(a["logits"], b["logits"])


def test_gqa_equals_mha_with_repeated_kv():
    cfg = TINY
    g = cfg.n_q_heads // cfg.n_kv_heads
    hw, hi = build(cfg)
    mha = cfg.with_(n_kv_heads=cfg.n_q_heads)
    hw2 = copy.deepcopy(hw)
    d = cfg.head_dim
    for P in hw2["sets"]:
        for key in ("w_k", "w_v"):
            W = P[key].reshape(cfg.n_kv_heads, d, -1)
            P[key] = np.repeat(W, g, axis=0).reshape(cfg.n_q_heads * d, -1)
    hi2 = dict(hi)
    hi2["prior_k"] = [np.repeat(k, g, axis=1) for k in hi["prior_k"]]
    hi2["prior_v"] = [np.repeat(v, g, axis=1) for v in hi["prior_v"]]
    a = Oracle(cfg, hw).chain(hi)
    b = Oracle(mha, hw2).chain(hi2)
    assert np.max(np.abs(a["logits"] - b["logits"])) < 1e-12


def test_duplicated_lm_rows_tie_to_lowest_id():
    hw, hi = build(TINY)
    orc = Oracle(TINY, hw)
    base = orc.chain(hi, K=1)
    t = int(base["tokens"][0, 0])
    hw2 = copy.deepcopy(hw)
    lo = max(0, t - 5)
    hw2["lm_head"] = hw2["lm_head"].copy()
    hw2["lm_head"][lo] = hw2["lm_head"][t]     # exact tie at a lower id
    r = Oracle(TINY, hw2).chain(hi, K=1)
    assert r["tokens"][0, 0] == lo
    assert r["logits"][0, 0, lo] == r["logits"][0, 0, t]


# ------------------------------------------------------------------ T8 torch fp64
def _torch_step(cfg, P, hw, tok, feat, Kp, Vp, pos):
    """The decoder block with torch fp64 library ops (independent formulation):
    rms_norm, complex rotation for RoPE, scaled_dot_product_attention with
    GQA, silu."""
    F = torch.nn.functional
    t = lambda a: torch.from_numpy(widen(a))
    H, d, nq, nkv = cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    x = torch.cat([t(hw["embed"][tok]), torch.from_numpy(feat)])
    u = t(P["w_fc"]) @ x
    a = F.rms_norm(u, (H,), t(P["g1"]), cfg.rms_eps)
    q = (t(P["w_q"]) @ a).view(nq, d)
    k = (t(P["w_k"]) @ a).view(nkv, d)
    v = (t(P["w_v"]) @ a).view(nkv, d)
    i = torch.arange(d // 2, dtype=torch.float64)
    ang = pos * torch.pow(torch.tensor(cfg.rope_theta, dtype=torch.float64), -2 * i / d)
    rot = torch.complex(torch.cos(ang).float().double(), torch.sin(ang).float().double())

    def rotate(z):
        c = torch.complex(z[..., : d // 2], z[..., d // 2:]) * rot
        return torch.cat([c.real, c.imag], -1)
    q, k = rotate(q), rotate(k)
    k = k.float().double()       # fp32 cache
    v = v.float().double()
    Ks = torch.cat([t(Kp), k[None]], 0).transpose(0, 1)   # [nkv, T, d]
    Vs = torch.cat([t(Vp), v[None]], 0).transpose(0, 1)
    o = F.scaled_dot_product_attention(q[:, None, :], Ks, Vs, enable_gqa=True)[:, 0, :]
    r1 = u + t(P["w_o"]) @ o.reshape(-1)
    m = F.rms_norm(r1, (H,), t(P["g2"]), cfg.rms_eps)
    z = F.silu(t(P["w_gate"]) @ m) * (t(P["w_up"]) @ m)
    h = r1 + t(P["w_down"]) @ z
    lg = t(hw["lm_head"]) @ F.rms_norm(h, (H,), t(hw["final_norm"]), cfg.rms_eps)
    return h.numpy(), lg.numpy()


def test_step_matches_torch_fp64():
    cfg = TINY.with_(batch=1, ctx_range=None, ctx_len=6)
    hw, hi = build(cfg)
    orc = Oracle(cfg, hw)
    res = orc.chain(hi, K=1)
    L = int(hi["ctx_lens"][0])
    h, lg = _torch_step(cfg, hw["sets"][0], hw, int(hi["tokens"][0]),
                        widen(hi["features"][0]), hi["prior_k"][0], hi["prior_v"][0], L)
    assert np.max(np.abs(res["hidden"][0, 0] - h)) < 1e-11
    assert np.max(np.abs(res["logits"][0, 0] - lg)) < 1e-11
