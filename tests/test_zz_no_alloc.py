"""prism_verify_chain_static: chain verification with no context and no
device allocation (its scratch is a fixed device array of the library).

Checked against prism_verify_chain (the context's entry point, same kernels)
on the same inputs, bit for bit, over two calls in a row whose second input
is smaller, greedy and sampled, at a small and the 8B vocabulary; and its
size limit is refused on the host before anything is launched.
"""
import pytest
import torch

from synth import SMALL_BF16_CHAIN, make_verify_chain

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _static(V, d, T):
    from paper_2602_01762_amd import binding as B
    Bn, K = d["draft_tokens"].shape
    n = torch.full((Bn,), -7, dtype=torch.int32, device="cuda")
    nxt = torch.full((Bn,), -7, dtype=torch.int32, device="cuda")
    B.prism_verify_chain_static(V, Bn, K, T, d["target_logits"],
                                d["draft_logits"] if T > 0 else None, d["draft_tokens"],
                                d["uniforms"] if T > 0 else None, n, nxt)
    return n, nxt


def _with_context(dr, d, T):
    r = dr.verify_chain(d["target_logits"], d["draft_tokens"], T,
                        d["draft_logits"] if T > 0 else None, d["uniforms"] if T > 0 else None)
    return r["n"], r["next"]


@pytest.mark.parametrize("vocab", [5008, 128256])
@pytest.mark.parametrize("T", [0.0, 1.0, 0.8])
def test_static_verify_matches_the_context_call(vocab, T):
    from paper_2602_01762_amd import Drafter
    cfg = SMALL_BF16_CHAIN.with_(batch=16, n_steps=6, vocab=vocab)
    # the static call first: on a fresh process its first call resolves the
    # scratch address itself (no context exists yet)
    calls = [(16, 6, 0), (5, 3, 1)]          # the second call is smaller
    data = [make_verify_chain(vocab, Bn, K, seed=seed, device="cuda") for Bn, K, seed in calls]
    got = []
    for d in data:
        got.append(_static(vocab, d, T))
    torch.cuda.synchronize()
    dr = Drafter(cfg)
    for d, (n, nxt) in zip(data, got):
        rn, rnxt = _with_context(dr, d, T)
        torch.cuda.synchronize()
        assert torch.equal(n, rn) and torch.equal(nxt, rnxt)
        assert (n >= 0).all() and (nxt >= 0).all() and (nxt < vocab).all()
    # and again after the context exists, in the other order (large after small)
    for d in data[::-1]:
        n, nxt = _static(vocab, d, T)
        rn, rnxt = _with_context(dr, d, T)
        torch.cuda.synchronize()
        assert torch.equal(n, rn) and torch.equal(nxt, rnxt)
    assert dr.device_status() == 0
    dr.close()


def test_static_verify_refuses_more_rows_than_its_scratch():
    from paper_2602_01762_amd import PrismError, binding as B
    d = make_verify_chain(5008, 2, 2, seed=0, device="cuda")
    n = torch.zeros(2, dtype=torch.int32, device="cuda")
    # 700 sequences of 6 sampled drafts: 700 * 7 + 700 * 6 = 9100 rows > 8192
    with pytest.raises(PrismError) as e:
        B.prism_verify_chain_static(5008, 700, 6, 1.0, d["target_logits"], d["draft_logits"],
                                    d["draft_tokens"], d["uniforms"], n, n)
    assert e.value.status == -2 and "8192" in str(e.value)
    with pytest.raises(PrismError) as e:
        B.prism_verify_chain_static(5000, 2, 2, 0.0, d["target_logits"], None,
                                    d["draft_tokens"], None, n, n)
    assert e.value.status == -2
