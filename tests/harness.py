"""Parity harness: GPU drafting (through the C ABI) against the CPU oracle.

Several results can be correct when logits nearly tie, so the oracle is
replayed teacher-forced on the GPU's own choices and then:
  * logits of every step agree within the dtype's tolerance;
  * the GPU token equals the oracle argmax wherever the oracle's top-1 margin
    exceeds 1e-2, and elsewhere is within 1e-2 of the oracle maximum;
  * tree children, frontiers and the final node set are valid top-w / top-v
    choices under the oracle's scores (1e-2 slack at the cut), and the
    GPU's tree structure follows exactly from its own candidate list.
"""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

from oracle import Oracle
from synth import host_inputs, host_weights, make_inputs, make_weights

LOGIT_TOL = {"bf16": 2e-2, "f32": 1e-4}
MARGIN = 1e-2


def log(*a):
    print("[%s]" % time.strftime("%H:%M:%S"), *a, file=sys.stderr, flush=True)


def gpu_setup(cfg, device="cuda"):
    from paper_2602_01762_amd import Drafter
    w = make_weights(cfg, device)
    inp = make_inputs(cfg, device)
    dr = Drafter(cfg)
    if cfg.f_map is not None:
        dr.set_step_map(cfg.fmap)
    dr.load(w)
    torch.cuda.synchronize()
    return dr, w, inp


def oracle_for(cfg, w, inp, seqs=None):
    return Oracle(cfg, host_weights(w)), host_inputs(inp, cfg, seqs)


def check_token(lg_oracle: np.ndarray, tok: int, what: str):
    order = np.argsort(-lg_oracle, kind="stable")
    top1, top2 = lg_oracle[order[0]], lg_oracle[order[1]]
    if top1 - top2 > MARGIN:
        assert tok == order[0], "%s: token %d, oracle argmax %d (margin %.4g)" % (
            what, tok, order[0], top1 - top2)
    else:
        assert lg_oracle[tok] >= top1 - MARGIN, "%s: token %d logit %.5f vs max %.5f" % (
            what, tok, lg_oracle[tok], top1)


def check_chain(cfg, out: dict, orc: Oracle, hi: dict, seqs, hidden_tol=None, catchup=False,
                inp=None):
    """Teacher-forced comparison of a GPU chain; with `inp` also the draft KV
    the chain wrote into the paged pools."""
    tol = LOGIT_TOL[cfg.dtype]
    hidden_tol = tol if hidden_tol is None else hidden_tol
    toks = out["tokens"].cpu().numpy().astype(np.int64)
    K = toks.shape[1]
    ref = orc.chain(hi, K=K, forced=toks, seqs=seqs, catchup=catchup)
    if inp is not None:
        check_draft_kv(cfg, inp, ref["draft_kv"], seqs)
    lg = out["logits"].cpu().numpy() if out.get("logits") is not None else None
    hd = out["hidden"].cpu().numpy() if out.get("hidden") is not None else None
    worst = 0.0
    for b in seqs:
        for k in range(K):
            what = "seq %d step %d" % (b, k + 1)
            assert 0 <= toks[b, k] < cfg.vocab, what
            check_token(ref["logits"][b, k], int(toks[b, k]), what)
            if lg is not None:
                e = float(np.max(np.abs(lg[b, k] - ref["logits"][b, k])))
                worst = max(worst, e)
                assert e <= tol, "%s: logits max-abs %.3g > %.3g" % (what, e, tol)
            if hd is not None:
                e = float(np.max(np.abs(hd[b, k] - ref["hidden"][b, k])))
                assert e <= hidden_tol, "%s: hidden max-abs %.3g" % (what, e)
    agree = np.mean([toks[b, k] == np.argmax(ref["logits"][b, k]) for b in seqs for k in range(K)])
    return {"max_logit_err": worst, "argmax_agreement": float(agree)}


CDF_SLACK = {"bf16": 1e-4, "f32": 1e-6}


def check_sampled_chain(cfg, out: dict, orc: Oracle, hi: dict, seqs, temperature: float):
    """Stochastic chain: with the oracle replayed on the GPU's draws, each
    drawn token's cumulative-probability interval [F(t-1), F(t)) (oracle, id
    order) contains its uniform up to a slack for the logit error, and the
    returned log p_draft matches the oracle's."""
    tol = LOGIT_TOL[cfg.dtype]
    toks = out["tokens"].cpu().numpy().astype(np.int64)
    K = toks.shape[1]
    u = hi["uniforms"]
    ref = orc.chain(hi, K=K, forced=toks, seqs=seqs, temperature=temperature, uniforms=u)
    lp = out["logp"].cpu().numpy()
    lg = out["logits"].cpu().numpy() if out.get("logits") is not None else None
    worst, same = 0.0, []
    for b in seqs:
        for k in range(K):
            what = "seq %d step %d" % (b, k + 1)
            t = int(toks[b, k])
            assert 0 <= t < cfg.vocab, what
            z = ref["logits"][b, k] / temperature
            p = np.exp(z - z.max())
            p /= p.sum()
            lo = float(p[:t].sum())
            hi_ = lo + float(p[t])
            sl = CDF_SLACK[cfg.dtype] / temperature
            assert lo - sl <= u[b, k] < hi_ + sl, "%s: u %.7f outside [%.7f, %.7f)" % (
                what, u[b, k], lo, hi_)
            e = abs(float(lp[b, k]) - float(np.log(p[t])))
            assert e <= tol / temperature, "%s: log p %.5f vs %.5f" % (what, lp[b, k], np.log(p[t]))
            if lg is not None:
                worst = max(worst, float(np.max(np.abs(lg[b, k] - ref["logits"][b, k]))))
                assert worst <= tol, "%s: logits max-abs %.3g" % (what, worst)
            same.append(t == int(ref["tokens"][b, k]))
    return {"max_logit_err": worst, "draw_agreement": float(np.mean(same))}


def check_draft_kv(cfg, inp, draft_kv: dict, seqs):
    """The K and V rows the GPU stored at every draft slot equal the oracle's
    stored values.  fp32 caches: to fp32 accumulation order.  bf16: within one
    rounding step of the value plus 2^-12 of the row's RMS; the two sides
    round an fp32 (activations carried to 2^-17) and an fp64 value of the
    same quantity, whose difference scales with the row, not the element."""
    from synth import to_host
    from oracle import widen
    bs = cfg.kv_block_size
    kp, vp = inp.k_pool.cpu(), inp.v_pool.cpu()
    btab = inp.block_table.cpu().numpy()
    for b in seqs:
        for slot, (kr, vr) in sorted(draft_kv[b].items()):
            blk = int(btab[b, slot // bs])
            kg = widen(to_host(kp[blk, :, slot % bs, :]))
            vg = widen(to_host(vp[blk, :, slot % bs, :]))
            for got, want, what in ((kg, kr, "k"), (vg, vr, "v")):
                if cfg.dtype == "f32":
                    assert np.max(np.abs(got - want)) <= 1e-5 * (1 + np.max(np.abs(want))), (b, slot, what)
                else:
                    rms = np.sqrt(np.mean(want * want, axis=-1, keepdims=True))
                    lim = 2.0 ** -7 * np.abs(want) + 2.0 ** -12 * rms
                    assert np.all(np.abs(got - want) <= lim), (
                        "seq %d slot %d %s: max diff %.3g" % (b, slot, what, np.max(np.abs(got - want))))


def _valid_cut(chosen_vals: np.ndarray, all_vals: np.ndarray, slack: float, what: str):
    """chosen are a valid top-n of all_vals up to `slack` at the cut."""
    n = len(chosen_vals)
    srt = np.sort(all_vals)[::-1]
    if len(srt) > n:
        assert chosen_vals.min() >= srt[n] - slack, "%s: chosen min %.5f < next best %.5f" % (
            what, chosen_vals.min(), srt[n])


def tree_forced(out: dict, b: int, D: int, w: int) -> dict:
    ct = out["cand_tokens"][b].cpu().numpy()
    fr = out["frontier"][b].cpu().numpy()
    children = [list(ct[:w])]
    for d in range(1, D):
        base = w + (d - 1) * w * w
        for r in range(w):
            children.append(list(ct[base + r * w: base + (r + 1) * w]))
    return {"children": children, "frontier": [list(fr[d]) for d in range(D - 1)]}


def check_tree_structure(out: dict, b: int, D: int, w: int, v: int):
    """The GPU's final output follows exactly from its own candidate list."""
    cs = out["cand_score"][b].cpu().numpy()
    cp = out["cand_parent"][b].cpu().numpy()
    ct = out["cand_tokens"][b].cpu().numpy()
    C = len(cs)
    order = sorted(range(C), key=lambda i: (-cs[i], i))[:v]
    pos = {n: i for i, n in enumerate(order)}
    tok = out["tokens"][b].cpu().numpy()
    par = out["parent"][b].cpu().numpy()
    dep = out["depth"][b].cpu().numpy()
    msk = out["mask"][b].cpu().numpy().astype(np.uint64)
    for i, n in enumerate(order):
        assert tok[i] == ct[n]
        p = int(cp[n])
        assert par[i] == (pos[p] if p >= 0 else -1), "parent of node %d" % i
        assert dep[i] == (1 if n < w else 2 + (n - w) // (w * w))
        bits, j = 0, i
        while j >= 0:
            bits |= 1 << j
            j = int(par[j])
        assert int(msk[i]) == bits
    # frontiers: top-w of each depth's candidates by (score desc, index asc)
    fr = out["frontier"][b].cpu().numpy()
    for d in range(D - 1):
        lo = 0 if d == 0 else w + (d - 1) * w * w
        hi = w if d == 0 else lo + w * w
        exp = sorted(range(lo, hi), key=lambda i: (-cs[i], i))[:w]
        assert list(fr[d]) == exp, "frontier at depth %d" % (d + 1)


def check_tree(cfg, out: dict, orc: Oracle, hi: dict, seqs, D: int):
    tol = LOGIT_TOL[cfg.dtype]
    w, v = cfg.tree_width, cfg.tree_nodes
    forced = {b: tree_forced(out, b, D, w) for b in seqs}
    ref = orc.tree(hi, forced=forced, seqs=seqs)
    lg = out["logits"].cpu().numpy() if out.get("logits") is not None else None
    worst = 0.0
    for b in seqs:
        check_tree_structure(out, b, D, w, v)
        R = ref[b]
        for i, ps in enumerate(R["passes"]):
            d = ps["depth"]
            r = 0 if d == 0 else (i - 1) % w
            what = "seq %d pass %d (depth %d rank %d)" % (b, i, d, r)
            if lg is not None:
                e = float(np.max(np.abs(lg[d, b, r] - ps["logits"])))
                worst = max(worst, e)
                assert e <= tol, "%s: logits max-abs %.3g" % (what, e)
            kids = np.asarray(forced[b]["children"][i])
            _valid_cut(ps["lp"][kids], ps["lp"], MARGIN, what + " children")
            assert len(set(kids.tolist())) == w
        cs_gpu = out["cand_score"][b].cpu().numpy()
        cs_orc = R["cand"]["score"]
        e = float(np.max(np.abs(cs_gpu - cs_orc)))
        assert e <= tol * cfg.n_steps, "seq %d: candidate scores max-abs %.3g" % (b, e)
        for d, f in enumerate(R["frontiers"]):
            lo = 0 if d == 0 else w + (d - 1) * w * w
            hi_ = w if d == 0 else lo + w * w
            _valid_cut(cs_orc[np.asarray(f)], cs_orc[lo:hi_], 2 * MARGIN, "seq %d frontier %d" % (b, d))
        nodes = out["tokens"].shape[1]
        gsel = sorted(range(len(cs_gpu)), key=lambda i: (-cs_gpu[i], i))[:nodes]
        _valid_cut(cs_orc[np.asarray(gsel)], cs_orc, 2 * MARGIN, "seq %d final" % b)
    return {"max_logit_err": worst}
