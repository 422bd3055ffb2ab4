"""Pins of the verification oracle against facts fixed by the mathematics:
the lossless property of the rejection rule (Sec. 2: the emitted token is
distributed exactly as the target's own draw), greedy verification as the
zero-temperature limit of it, and tree acceptance as the best of the chain
acceptances along every root-to-leaf path."""
import numpy as np
import pytest

from oracle import softmax_t, verify_chain_greedy, verify_chain_sample, verify_tree_greedy


@pytest.mark.parametrize("T", [0.7, 1.0, 1.6])
def test_rejection_rule_is_lossless(T):
    rng = np.random.default_rng(11)
    V = 6
    tl = rng.standard_normal((2, V)) * 1.5      # target rows: after 0 and 1 drafts
    dl = rng.standard_normal((1, V)) * 1.5      # draft row of the one draft
    pt, pd = softmax_t(tl[0], T), softmax_t(dl[0], T)
    N = 4000
    grid = (np.arange(N) + 0.5) / N
    # acceptance share of each possible draft token over a grid of r
    acc = np.array([np.mean([verify_chain_sample(tl, dl, np.array([t]), T,
                                                 np.array([r, 0.5]))["n"] == 1 for r in grid])
                    for t in range(V)])
    assert np.max(np.abs(acc - np.minimum(1.0, pt / pd))) <= 1.0 / N
    # distribution of the correction token (a draft the target never keeps)
    t_rej = int(np.argmin(pt / pd))
    corr = np.zeros(V)
    for u in grid:
        out = verify_chain_sample(tl, dl, np.array([t_rej]), T, np.array([1.0 - 1e-15, u]))
        assert out["n"] == 0
        corr[out["next"]] += 1.0 / N
    emit = pd * acc + (1.0 - np.sum(pd * acc)) * corr
    assert np.max(np.abs(emit - pt)) <= 3.0 / N


def test_greedy_is_the_cold_limit_of_sampling():
    rng = np.random.default_rng(5)
    V, K = 50, 6
    for trial in range(40):
        tl = rng.standard_normal((K + 1, V))
        dl = rng.standard_normal((K, V))
        drafts = np.argmax(dl, axis=1)
        # let the target agree with the first few drafts
        m = trial % (K + 1)
        for i in range(m):
            tl[i, drafts[i]] = tl[i].max() + 0.5
        g = verify_chain_greedy(tl, drafts)
        s = verify_chain_sample(tl, dl, drafts, 1e-3, rng.uniform(0.0, 1.0, K + 1))
        assert g == s
        assert g["n"] >= m


def test_tree_acceptance_is_best_path():
    rng = np.random.default_rng(9)
    V, w = 30, 3
    for trial in range(30):
        # a random tree: each node's parent is an earlier node or the root,
        # siblings carry distinct tokens
        v = 12
        parent = np.full(v, -1)
        tokens = np.zeros(v, dtype=np.int64)
        used = {}
        for j in range(v):
            p = int(rng.integers(-1, j)) if j else -1
            while len(used.setdefault(p, set())) >= w:
                p = int(rng.integers(-1, j)) if j else -1
            t = int(rng.integers(0, V))
            while t in used[p]:
                t = int(rng.integers(0, V))
            used[p].add(t)
            parent[j], tokens[j] = p, t
        tl = rng.standard_normal((v + 1, V))
        for j in range(v):                   # the target often agrees with a child
            if rng.uniform() < 0.6:
                tl[int(parent[j]) + 1, tokens[j]] = tl[int(parent[j]) + 1].max() + 1.0
        got = verify_tree_greedy(tl, tokens, parent)
        # brute force: greedy chain verification along every root path
        best = (0, [], int(np.argmax(tl[0])))
        for leaf in range(v):
            path = []
            j = leaf
            while j >= 0:
                path.append(j)
                j = int(parent[j])
            path = path[::-1]
            rows = np.stack([tl[0]] + [tl[j + 1] for j in path])
            c = verify_chain_greedy(rows, tokens[path])
            if c["n"] > best[0]:
                best = (c["n"], path[:c["n"]], c["next"])
        assert got["n"] == best[0] and got["path"] == best[1] and got["next"] == best[2]
