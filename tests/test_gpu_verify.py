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
from synth import (L3_8B_BS16, L3_8B_TREE, SMALL_BF16_CHAIN, SMALL_BF16_TREE, make_verify_chain,
                   make_verify_tree_targets)
from harness import gpu_setup, log

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
