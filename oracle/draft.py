"""Plain CPU oracle of PRISM's drafting hot path, in fp64.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path
(the HIP library and its binding) never does, and shares no code with it.

What is computed (PRISM, Sec. 3.2 "Draft with PRISM"; notation of Table 2):

  * a frozen embedding E and a frozen LM head shared by every module
    (Sec. 3.2 architecture paragraph, Table 2);
  * M processing modules, each a fusion FC F_i and one transformer layer L_i;
    draft step k runs module f_map(k) (Sec. 3.2, the surjection paragraph);
  * step 1 fuses E(x_i) of every accepted token with the target's hidden
    state for it, runs L_{f(1)} over the fused rows in one pass (causal
    among them), and predicts x_1 = argmax LM_head(h_0) from the last row
    (Sec. 3.2, the prefill equations); the plain chain has one accepted
    token per sequence;
  * step k >= 2 fuses E(x_{k-1}) with the draft's own previous hidden state
    h_{k-2}, runs L_{f(k)} against the KV cache shared by all modules, and
    predicts x_k = argmax LM_head(h_{k-1}) (Sec. 3.2, decoding equations;
    Fig. 3(b) caption: the KV cache passes from one module to the next);
  * the same steps laid out as a draft tree with a tree attention mask
    (Sec. 2 "SoTA Draft Models"; Sec. 3.2 says PRISM is compatible with tree
    drafts; Sec. 4.1 and 4.3 give the depth / width / verified-node topology);
  * the target's side of tree verification: one pass of a scoring model
    over the root and every node of a drafted tree under its ancestor mask
    (Sec. 2, speculative decoding with tree attention).

Readings where the paper is silent:
the decode equation is read as H_in = F(E(x_{k-1}), h_{k-2})
with the transformer updating the KV; FC input order is [E(x) ; feature],
no biases; Llama pre-norm block (RMSNorm, RoPE GQA attention, residual,
RMSNorm, SwiGLU, residual) with the residual stream starting at the FC
output u; a shared final RMSNorm before the LM head, h fed back un-normed;
rotate-half RoPE with angles in fp64 and cos/sin rounded to fp32; chain
step k at position L+k-1; tree depth-d nodes at position L+d; ties broken by
lowest token id.

Precision: the paper fixes none.  Everything here is fp64.  Stored tensors
are exact in their storage type (bf16 or fp32 weights, embeddings, target
features), and the one value the drafting step itself stores, the new k and
v of the KV cache, is rounded to the cache type.  Activations that feed a
matrix product are used exactly (the kernels carry them at fp32 precision),
so no other rounding is emulated.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

from ._native import linear as _linear, widen


# ---------------------------------------------------------------- primitives
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bf16 value, ties to even.

    bf16 keeps 8 significant bits.  frexp gives x = m * 2**e with
    0.5 <= |m| < 1, so m * 2**8 rounded half-to-even to an integer and
    scaled back is the RNE result (exact in fp64).  NaN and inf pass through.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    r = np.ldexp(np.round(m * 256.0), e - 8)
    return np.where(np.isfinite(x), r, x)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(y: np.ndarray) -> np.ndarray:
    return y / (1.0 + np.exp(-y))


def rope_cos_sin(pos: int, d: int, theta: float):
    """cos/sin of the rotate-half angles p * theta^(-2i/d), i < d/2.

    Angles in fp64, cos/sin rounded to fp32 (the kernel's table precision).
    """
    i = np.arange(d // 2, dtype=np.float64)
    phi = float(pos) * np.power(float(theta), -2.0 * i / d)
    c = np.cos(phi).astype(np.float32).astype(np.float64)
    s = np.sin(phi).astype(np.float32).astype(np.float64)
    return c, s


def rope(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate pairs (x_i, x_{i+d/2}) of every head by the angle for `pos`.

    x: [..., d].
    """
    d = x.shape[-1]
    c, s = rope_cos_sin(pos, d, theta)
    a, b = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def softmax_attend(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """softmax(q . K_t / sqrt(d)) weighted sum of V_t (max-subtracted).

    q: [d]; K, V: [T, d].
    """
    d = q.shape[-1]
    s = K @ q / np.sqrt(d)
    p = np.exp(s - s.max())
    return (p @ V) / p.sum()


def logsumexp(x: np.ndarray) -> float:
    m = x.max()
    return float(m + np.log(np.exp(x - m).sum()))


def topk_ids(v: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest values; ties broken by lower index."""
    return np.argsort(-v, kind="stable")[:k]


def sample_inverse_cdf(logits: np.ndarray, temperature: float, u: float):
    """Draw from p = softmax(logits / T) with the uniform u in [0, 1): the
    smallest token id t whose cumulative probability (ids 0..t, in id order)
    exceeds u.  Returns (t, log p_t).  This is the draft distribution whose
    probabilities the rejection rule of Sec. 2 compares with the target's.
    """
    z = logits / temperature
    m = z.max()
    e = np.exp(z - m)
    S = e.sum()
    cdf = np.cumsum(e) / S
    t = int(np.searchsorted(cdf, u, side="right"))
    t = min(t, len(cdf) - 1)
    return t, float(z[t] - m - np.log(S))


# --------------------------------------------------------------------- model
class Oracle:
    """The drafter on host arrays (see module docstring)."""

    def __init__(self, cfg, hw: dict, use_c: bool = True):
        self.cfg = cfg
        self.hw = hw
        self.use_c = use_c
        self.bf16 = cfg.dtype == "bf16"
        self.g_f = widen(hw["final_norm"])

    def store(self, x):
        """A value written to the KV cache (rounded to the cache dtype)."""
        return round_bf16(x) if self.bf16 else x.astype(np.float32).astype(np.float64)

    def lin(self, W, X):
        return _linear(W, X, self.use_c)

    # one forward pass for a set of rows ----------------------------------
    def forward(self, s: int, tokens: Sequence[int], feats: np.ndarray,
                pos: Sequence[int], caches: List[dict], seq: Sequence[int],
                slots: Sequence[int], visible: Sequence[Sequence[int]],
                want_logits: bool = True):
        """Run parameter set s on R rows.

        Row r: token tokens[r], feature feats[r] (target feature or a
        previous hidden state), RoPE position pos[r], sequence seq[r]; its k/v
        go to slot slots[r] of caches[seq[r]] and it attends to the slots in
        visible[r] (increasing order, own slot included).
        Returns (h [R,H], logits [R,V]).
        """
        cfg, P = self.cfg, self.hw["sets"][s]
        H, d, nq, nkv = cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
        g = nq // nkv
        R = len(tokens)
        assert feats.shape == (R, P["feat_width"]), (feats.shape, P["feat_width"])
        e = widen(self.hw["embed"][np.asarray(tokens)])
        u = self.lin(P["w_fc"], np.concatenate([e, feats], axis=1))
        a = rmsnorm(u, widen(P["g1"]), cfg.rms_eps)
        q = self.lin(P["w_q"], a).reshape(R, nq, d)
        k = self.lin(P["w_k"], a).reshape(R, nkv, d)
        v = self.lin(P["w_v"], a).reshape(R, nkv, d)
        for r in range(R):
            q[r] = rope(q[r], pos[r], cfg.rope_theta)
            k[r] = self.store(rope(k[r], pos[r], cfg.rope_theta))
            v[r] = self.store(v[r])
            caches[seq[r]]["draft"][slots[r]] = (k[r].copy(), v[r].copy())
        o = np.empty((R, nq, d))
        for r in range(R):
            Kv, Vv = self.gather(caches[seq[r]], visible[r])
            for h in range(nq):
                o[r, h] = softmax_attend(q[r, h], Kv[:, h // g, :], Vv[:, h // g, :])
        r1 = u + self.lin(P["w_o"], o.reshape(R, nq * d))
        m = rmsnorm(r1, widen(P["g2"]), cfg.rms_eps)
        z = silu(self.lin(P["w_gate"], m)) * self.lin(P["w_up"], m)
        hid = r1 + self.lin(P["w_down"], z)
        logits = None
        if want_logits:
            logits = self.lin(self.hw["lm_head"], rmsnorm(hid, self.g_f, cfg.rms_eps))
        return hid, logits

    @staticmethod
    def gather(cache: dict, visible: Sequence[int]):
        L = cache["L"]
        ks, vs = [], []
        prior = [t for t in visible if t < L]
        if prior:
            idx = np.asarray(prior)
            ks.append(cache["k"][idx])
            vs.append(cache["v"][idx])
        for t in visible:
            if t >= L:
                kt, vt = cache["draft"][t]
                ks.append(kt[None])
                vs.append(vt[None])
        return np.concatenate(ks, 0), np.concatenate(vs, 0)

    def new_cache(self, hi: dict, b: int) -> dict:
        return {"L": int(hi["ctx_lens"][b]), "k": widen(hi["prior_k"][b]),
                "v": widen(hi["prior_v"][b]), "draft": {}}

    # chain ------------------------------------------------------------------
    def chain(self, hi: dict, K: Optional[int] = None, forced: Optional[np.ndarray] = None,
              seqs: Optional[Sequence[int]] = None, catchup: bool = False,
              temperature: Optional[float] = None,
              uniforms: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
        """Greedy K-step chain for the sequences in `seqs` (default all).

        Step 1 is the drafter's prefill (Sec. 3.2, "Draft with PRISM"): each
        accepted token x_i of the sequence is fused with the target's hidden
        state h_{i-1}, and the fused rows run through module f_map(1) in one
        pass at positions L_b .. L_b + n_b - 1, each attending to the prior
        context and to the new rows up to itself.  The last row's output is
        h_0 and x_1 = argmax LM_head(h_0).  Without `catchup` the accepted
        tokens are just the last one (hi["tokens"] / hi["features"], n_b = 1);
        with it they are the rows of hi["new_tokens"] / hi["new_features"]
        delimited by hi["new_offsets"].  Step k >= 2 fuses E(x_{k-1}) with
        h_{k-2} at position L_b + n_b + k - 2.

        Greedy by default (x_k = argmax, ties to the lowest id).  With a
        `temperature` T > 0, x_k is drawn from softmax(logits / T) by
        sample_inverse_cdf with the uniform uniforms[b, k-1] (stochastic
        drafting, Sec. 2; Sec. 3.2 notes PRISM works with it), and
        "logp"[b, k-1] holds log p_draft(x_k).

        forced[b, k]: token fed to step k+2 instead of the oracle's own
        choice at step k+1 (teacher forcing on another drafter's choices).
        Returns tokens [B,K], logits [B,K,V], hidden [B,K,H] (rows of
        sequences not computed are left at -1 / NaN; step 1 holds the last
        row's values) and, per computed sequence, the draft KV it wrote
        ("draft_kv": {b: {slot: (k, v)}}).
        """
        cfg = self.cfg
        K = cfg.n_steps if K is None else K
        B = len(hi["tokens"])
        seqs = list(range(B)) if seqs is None else list(seqs)
        fm = cfg.fmap
        toks = np.full((B, K), -1, dtype=np.int64)
        logits = np.full((B, K, cfg.vocab), np.nan)
        hidden = np.full((B, K, cfg.hidden), np.nan)
        logp = np.full((B, K), np.nan)

        def choose(b, k, lg):       # the token of step k (1-based) from its logits
            if temperature is None:
                return int(np.argmax(lg))
            t, lp = sample_inverse_cdf(lg, temperature, float(uniforms[b, k - 1]))
            logp[b, k - 1] = lp
            return t

        caches = {b: self.new_cache(hi, b) for b in seqs}
        # the accepted rows of each sequence, oldest first
        acc = {}
        for b in seqs:
            if catchup:
                o0, o1 = int(hi["new_offsets"][b]), int(hi["new_offsets"][b + 1])
                acc[b] = ([int(t) for t in hi["new_tokens"][o0:o1]],
                          [widen(hi["new_features"][i]) for i in range(o0, o1)])
            else:
                acc[b] = ([int(hi["tokens"][b])], [widen(hi["features"][b])])
        # step 1: one pass of set f_map(1) over every accepted row
        rows_b, tk, ft, pos = [], [], [], []
        for b in seqs:
            L = caches[b]["L"]
            for i, (t, f) in enumerate(zip(*acc[b])):
                rows_b.append(b)
                tk.append(t)
                ft.append(f)
                pos.append(L + i)
        h, lg = self.forward(fm[0], tk, np.stack(ft), pos, caches, rows_b, pos,
                             [list(range(p + 1)) for p in pos])
        last = {b: max(i for i, rb in enumerate(rows_b) if rb == b) for b in seqs}
        x_in, f_in, start = {}, {}, {}
        for b in seqs:
            i = last[b]
            toks[b, 0] = choose(b, 1, lg[i])
            logits[b, 0] = lg[i]
            hidden[b, 0] = h[i]
            x_in[b] = int(forced[b, 0]) if forced is not None else toks[b, 0]
            f_in[b] = h[i]
            start[b] = pos[i] + 1          # position of step 2
        # steps k >= 2: decoding
        for k in range(2, K + 1):
            s = fm[k - 1]
            pos = [start[b] + k - 2 for b in seqs]
            h, lg = self.forward(s, [x_in[b] for b in seqs], np.stack([f_in[b] for b in seqs]),
                                 pos, caches, seqs, pos, [list(range(p + 1)) for p in pos])
            for i, b in enumerate(seqs):
                toks[b, k - 1] = choose(b, k, lg[i])
                logits[b, k - 1] = lg[i]
                hidden[b, k - 1] = h[i]
                x_in[b] = int(forced[b, k - 1]) if forced is not None else toks[b, k - 1]
                f_in[b] = h[i]
        return {"tokens": toks, "logits": logits, "hidden": hidden, "logp": logp,
                "draft_kv": {b: caches[b]["draft"] for b in seqs}}

    # tree -------------------------------------------------------------------
    def tree(self, hi: dict, forced: Optional[dict] = None,
             seqs: Optional[Sequence[int]] = None) -> dict:
        """Dynamic draft tree: depth D = n_steps passes, width w, v output nodes.

        Root pass (set f(1)) at position L_b; its top-w log-probs are the
        depth-1 candidates.  The frontier at each depth is the top-w of that
        depth's candidates by cumulative log-prob; each frontier node runs one
        pass with set f(d+1) at position L_b + d, attending to the prior
        context, the root and its ancestors, and yields its top-w children
        (score = parent score + log-prob).  The output is the top-v candidates.
        Order keys: (score desc, creation order asc); creation order is depth,
        then parent rank, then child rank.

        forced[b] = {"children": [pass][w] tokens, "frontier": [D-1][w]
        candidate ids} replays another drafter's choices; the scores are
        still the oracle's own.
        """
        cfg = self.cfg
        D, w, v = cfg.n_steps, cfg.tree_width, cfg.tree_nodes
        B = len(hi["tokens"])
        seqs = list(range(B)) if seqs is None else list(seqs)
        fm = cfg.fmap
        out = {}
        caches = {b: self.new_cache(hi, b) for b in seqs}
        cand = {b: {"token": [], "parent": [], "depth": [], "score": []} for b in seqs}
        passes = {b: [] for b in seqs}

        def add_children(b, lg, parent, score0, depth, forced_toks):
            lp = lg - logsumexp(lg)
            kids = topk_ids(lp, w) if forced_toks is None else np.asarray(forced_toks)
            for t in kids:
                c = cand[b]
                c["token"].append(int(t))
                c["parent"].append(parent)
                c["depth"].append(depth)
                c["score"].append(score0 + float(lp[t]))
            return lp

        # root pass
        pos = [caches[b]["L"] for b in seqs]
        h, lg = self.forward(fm[0], [int(hi["tokens"][b]) for b in seqs],
                             np.stack([widen(hi["features"][b]) for b in seqs]),
                             pos, caches, seqs, pos, [list(range(p + 1)) for p in pos])
        front = {}
        for i, b in enumerate(seqs):
            ft = forced[b]["children"][0] if forced else None
            lp = add_children(b, lg[i], -1, 0.0, 1, ft)
            passes[b].append({"cand": -1, "depth": 0, "slot": pos[i], "pos": pos[i],
                              "logits": lg[i], "lp": lp, "hidden": h[i]})
            front[b] = self._frontier(cand[b], 0, w, forced[b]["frontier"][0] if forced else None)
        frontiers = {b: [front[b]] for b in seqs}
        # pass hidden / ancestor slots of every expanded candidate
        node_hidden = {b: {} for b in seqs}
        node_slots = {b: {} for b in seqs}
        for i, b in enumerate(seqs):
            for c in range(w):
                node_hidden[b][c] = h[i]          # depth-1 nodes: parent is the root
                node_slots[b][c] = [caches[b]["L"]]

        for d in range(1, D):
            rows_b, rows_c, toks, feats, pos, slots, vis = [], [], [], [], [], [], []
            for b in seqs:
                L = caches[b]["L"]
                for r, c in enumerate(front[b]):
                    slot = L + 1 + (d - 1) * w + r
                    rows_b.append(b)
                    rows_c.append(c)
                    toks.append(cand[b]["token"][c])
                    feats.append(node_hidden[b][c])
                    pos.append(L + d)
                    slots.append(slot)
                    anc = node_slots[b][c]
                    vis.append(list(range(L)) + anc + [slot])
            h, lg = self.forward(fm[d], toks, np.stack(feats), pos, caches, rows_b, slots, vis)
            base_rank = {}
            for i, b in enumerate(rows_b):
                c = rows_c[i]
                r = base_rank.get(b, 0)
                base_rank[b] = r + 1
                ft = forced[b]["children"][1 + (d - 1) * w + r] if forced else None
                first_child = len(cand[b]["token"])
                lp = add_children(b, lg[i], c, cand[b]["score"][c], d + 1, ft)
                passes[b].append({"cand": c, "depth": d, "slot": slots[i], "pos": pos[i],
                                  "logits": lg[i], "lp": lp, "hidden": h[i]})
                for j in range(w):
                    node_hidden[b][first_child + j] = h[i]
                    node_slots[b][first_child + j] = vis[i][caches[b]["L"]:]
            if d < D - 1:
                for b in seqs:
                    lo = w + (d - 1) * w * w
                    front[b] = self._frontier(cand[b], lo, w,
                                              forced[b]["frontier"][d] if forced else None)
                    frontiers[b].append(front[b])

        for b in seqs:
            c = {k: np.asarray(vv) for k, vv in cand[b].items()}
            order = np.argsort(-c["score"], kind="stable")[:v]
            where = {int(n): i for i, n in enumerate(order)}
            par = np.array([where.get(int(c["parent"][n]), -1) if c["parent"][n] >= 0 else -1
                            for n in order], dtype=np.int64)
            mask = np.zeros(len(order), dtype=np.uint64)
            for i, n in enumerate(order):
                bits = 0
                j = i
                while j >= 0:
                    bits |= 1 << j
                    j = int(par[j])
                mask[i] = np.uint64(bits)
            out[b] = {"cand": c, "frontiers": frontiers[b], "passes": passes[b],
                      "nodes": order, "tokens": c["token"][order], "parent": par,
                      "depth": c["depth"][order], "score": c["score"][order], "mask": mask}
        return out

    # target-side tree scoring ------------------------------------------------
    def score_tree(self, hi: dict, tokens: np.ndarray, depth: np.ndarray, mask: np.ndarray,
                   seqs: Optional[Sequence[int]] = None) -> dict:
        """The target model's pass over draft trees (Sec. 2: the target
        scores every candidate of the tree in one forward pass under a tree
        attention mask), with this oracle's weights as the scoring model
        (set f_map(1), every row fusing the sequence's feature row).

        Sequence b: row 0 is the root (hi["tokens"][b]) at position and slot
        L_b; row 1 + j is node j (tokens[b, j]) at position L_b + depth[b, j]
        and slot L_b + 1 + j, seeing the prior context, the root and the
        slots of the nodes in mask[b, j] (its ancestors and itself).
        Returns logits [B, n+1, V] (sequences not in `seqs` left NaN) and the
        KV each sequence wrote ("draft_kv")."""
        cfg = self.cfg
        B, n = tokens.shape
        seqs = list(range(B)) if seqs is None else list(seqs)
        logits = np.full((B, n + 1, cfg.vocab), np.nan)
        kv = {}
        for b in seqs:
            cache = self.new_cache(hi, b)
            L = cache["L"]
            toks, pos, slots, vis = [int(hi["tokens"][b])], [L], [L], [list(range(L + 1))]
            for j in range(n):
                m = int(mask[b, j]) & ((1 << 64) - 1)
                nodes = [a for a in range(n) if (m >> a) & 1]
                toks.append(int(tokens[b, j]))
                pos.append(L + int(depth[b, j]))
                slots.append(L + 1 + j)
                vis.append(list(range(L + 1)) + [L + 1 + a for a in nodes])
            feats = np.stack([widen(hi["features"][b])] * (n + 1))
            _, lg = self.forward(cfg.fmap[0], toks, feats, pos, {b: cache}, [b] * (n + 1), slots,
                                 vis)
            logits[b] = lg
            kv[b] = cache["draft"]
        return {"logits": logits, "draft_kv": kv}

    @staticmethod
    def _frontier(c: dict, lo: int, w: int, forced) -> List[int]:
        """Top-w of the candidates created from index lo on (one depth)."""
        if forced is not None:
            return [int(x) for x in forced]
        sc = np.asarray(c["score"][lo:])
        return [lo + int(i) for i in np.argsort(-sc, kind="stable")[:w]]


# ------------------------------------------------------------ brute force
def brute_chain(orc: Oracle, hi: dict, K: int, seqs: Optional[Sequence[int]] = None,
                catchup: bool = False, temperature: Optional[float] = None,
                uniforms: Optional[np.ndarray] = None):
    """Greedy chain recomputed from scratch at every step, for tiny shapes.

    No cache object survives between steps: for step k all draft positions
    are re-run in order -- the n_b - 1 earlier accepted tokens (with
    `catchup`; set f(1), their own tokens and target features), then the k
    chain positions (set f(j), its token, and the hidden state this same
    recomputation produced for the position before) -- attention is an
    explicit causal mask over the full key matrix, and the token is the
    first entry of a full sort of the logits, or with a temperature the
    first id at which a running sum of exp(logit / T - max) passes u times
    the total.  Returns tokens [B,K] and hidden [B,K,H].
    """
    cfg = orc.cfg
    H, d, nq, nkv = cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    g = nq // nkv
    B = len(hi["tokens"])
    seqs = list(range(B)) if seqs is None else list(seqs)
    toks = np.full((B, K), -1, dtype=np.int64)
    hidden = np.full((B, K, H), np.nan)
    for b in seqs:
        L = int(hi["ctx_lens"][b])
        Kp, Vp = widen(hi["prior_k"][b]), widen(hi["prior_v"][b])
        if catchup:
            o0, o1 = int(hi["new_offsets"][b]), int(hi["new_offsets"][b + 1])
            pre = [(int(hi["new_tokens"][i]), widen(hi["new_features"][i])) for i in range(o0, o1 - 1)]
            first = (int(hi["new_tokens"][o1 - 1]), widen(hi["new_features"][o1 - 1]))
        else:
            pre, first = [], (int(hi["tokens"][b]), widen(hi["features"][b]))
        n0 = len(pre)
        chosen: List[int] = []
        for k in range(1, K + 1):
            n = n0 + k                      # draft positions recomputed for this step
            Ks = np.zeros((L + n, nkv, d))
            Vs = np.zeros((L + n, nkv, d))
            Ks[:L], Vs[:L] = Kp, Vp
            mask = np.zeros((n, L + n), dtype=bool)
            for j in range(n):
                mask[j, : L + j + 1] = True
            tok, feat = pre[0] if n0 else first
            for j in range(n):
                step = max(j - n0, 0)       # 0-based chain step of position j
                P = orc.hw["sets"][cfg.fmap[step]]
                e = widen(orc.hw["embed"][tok])[None]
                u = orc.lin(P["w_fc"], np.concatenate([e, feat[None]], 1))
                a = rmsnorm(u, widen(P["g1"]), cfg.rms_eps)
                q = orc.lin(P["w_q"], a).reshape(nq, d)
                kk = orc.lin(P["w_k"], a).reshape(nkv, d)
                vv = orc.lin(P["w_v"], a).reshape(nkv, d)
                q = rope(q, L + j, cfg.rope_theta)
                Ks[L + j] = orc.store(rope(kk, L + j, cfg.rope_theta))
                Vs[L + j] = orc.store(vv)
                o = np.empty((nq, d))
                for hh in range(nq):
                    sc = Ks[:, hh // g, :] @ q[hh] / np.sqrt(d)
                    sc = np.where(mask[j], sc, -np.inf)
                    p = np.exp(sc - sc.max())
                    o[hh] = (p @ Vs[:, hh // g, :]) / p.sum()
                r1 = u + orc.lin(P["w_o"], o.reshape(1, nq * d))
                m = rmsnorm(r1, widen(P["g2"]), cfg.rms_eps)
                z = silu(orc.lin(P["w_gate"], m)) * orc.lin(P["w_up"], m)
                hj = (r1 + orc.lin(P["w_down"], z))[0]
                if j == n - 1:
                    lg = orc.lin(orc.hw["lm_head"],
                                 rmsnorm(hj[None], orc.g_f, cfg.rms_eps))[0]
                    if temperature is None:
                        order = np.argsort(-lg, kind="stable")
                        chosen.append(int(order[0]))
                    else:
                        w = [float(np.exp((x - lg.max()) / temperature)) for x in lg]
                        goal, run, pick = float(uniforms[b, k - 1]) * sum(w), 0.0, len(w) - 1
                        for t, wt in enumerate(w):
                            run += wt
                            if run > goal:
                                pick = t
                                break
                        chosen.append(pick)
                    hidden[b, k - 1] = hj
                elif j < n0 - 1:
                    tok, feat = pre[j + 1]  # the next accepted token, its target feature
                elif j == n0 - 1:
                    tok, feat = first
                else:
                    tok, feat = chosen[j - n0], hj
        toks[b] = chosen
    return {"tokens": toks, "hidden": hidden}
