"""Plain CPU oracle of the verification step that follows drafting, in fp64.

TEST INFRASTRUCTURE (see the package docstring): only tests, the smoke check
and the benchmark's CPU-baseline leg use it.

What is computed (PRISM, Sec. 2 "Speculative Decoding"): the target model
scores the drafted tokens in one pass; greedy drafts are kept while they
match the target's own choice, and sampled drafts go through the modified
rejection rule -- draft token x_i is accepted when a uniform r satisfies
r < min(1, p_target(x_i) / p_draft(x_i)); at the first rejection a token is
drawn from p' proportional to max(0, p_target - p_draft) at that position,
and when every draft is accepted one extra token is drawn from p_target at
the next position.  The target's scores come in as logits (a synthetic
target stands in for the target model).  Trees (Sec. 2, tree verification):
the accepted drafts are the longest root path whose every node is the
target's choice at its parent.

Draws use the same inverse CDF in token-id order as the drafter
(oracle.draft.sample_inverse_cdf); ties in arg-max go to the lowest id.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from .draft import sample_inverse_cdf


def softmax_t(logits: np.ndarray, temperature: float) -> np.ndarray:
    z = logits / temperature
    e = np.exp(z - z.max())
    return e / e.sum()


def draw_from(weights: np.ndarray, u: float) -> int:
    """Smallest id whose cumulative weight (id order) exceeds u times the total."""
    cdf = np.cumsum(weights)
    t = int(np.searchsorted(cdf, u * cdf[-1], side="right"))
    return min(t, len(weights) - 1)


def verify_chain_greedy(target_logits: np.ndarray, drafts: np.ndarray) -> Dict[str, int]:
    """target_logits [K+1, V] (row i scores the token after i drafts), drafts [K].
    Returns the accepted count n and the next token: the target's choice after
    the n accepted drafts."""
    K = len(drafts)
    n = 0
    while n < K and int(np.argmax(target_logits[n])) == int(drafts[n]):
        n += 1
    return {"n": n, "next": int(np.argmax(target_logits[n]))}


def verify_chain_sample(target_logits: np.ndarray, draft_logits: np.ndarray, drafts: np.ndarray,
                        temperature: float, r: np.ndarray) -> Dict[str, int]:
    """The rejection rule of Sec. 2 at temperature T.  r [K+1]: r[i] decides
    draft i, r[K] draws the final token (the correction or the extra one)."""
    K = len(drafts)
    for i in range(K):
        pt = softmax_t(target_logits[i], temperature)
        pd = softmax_t(draft_logits[i], temperature)
        x = int(drafts[i])
        if not r[i] < min(1.0, pt[x] / pd[x]):
            resid = np.maximum(0.0, pt - pd)
            if resid.sum() <= 0.0:          # p_target == p_draft: nothing to correct
                resid = pt
            return {"n": i, "next": draw_from(resid, float(r[K]))}
    return {"n": K, "next": sample_inverse_cdf(target_logits[K], temperature, float(r[K]))[0]}


def verify_tree_greedy(target_logits: np.ndarray, tokens: np.ndarray,
                       parent: np.ndarray) -> Dict[str, object]:
    """target_logits [v+1, V]: row 0 scores the token after the root, row 1+j
    the token after node j.  tokens / parent [v] (parent -1 = the root).
    Walks from the root: at each accepted position the child whose token is
    the target's choice there is accepted (children of a node carry distinct
    tokens; the first in node order if not).  Returns the accepted count, the
    accepted node indices in depth order, and the next token."""
    choice = [int(np.argmax(target_logits[j])) for j in range(len(tokens) + 1)]
    path: List[int] = []
    at = -1                                  # current position: the root
    while True:
        want = choice[at + 1]
        nxt = [j for j in range(len(tokens)) if int(parent[j]) == at and int(tokens[j]) == want]
        if not nxt:
            break
        at = nxt[0]
        path.append(at)
    return {"n": len(path), "path": path, "next": choice[at + 1]}
