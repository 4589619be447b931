"""Draft top-K and DyTC decoding through the library (GPU).

- cas_topk against numpy on the very logits the library produced: ids
  bit-exact (stable descending order, ties to the lower id), probabilities
  against an fp64 softmax of the same row.
- DyTC speculative decoding through the library (tree-parallel draft calls
  that append nodes, over layer-skip, W8A8 and W4A4 levels and prompt
  lookup; top-K candidates, full-depth verify, commit) equals
  greedy autoregressive decoding of the oracle and of the library, token for
  token.  The models are the tiny fp32 decoder and a small bf16 GQA decoder;
  bf16 mismatches are excused only where the oracle's top-1/top-2 margin is
  at most 0.05.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2510_26843_amd import cas, decode, dytc, synth

pytestmark = pytest.mark.gpu

GQA = synth.ModelShape("gqa_small", 4, 256, 4, 2, 64, 688, 512, 5e5, 1e-6, "bf16")


@pytest.fixture(scope="module")
def weights():
    return {"tiny": synth.gen_weights(synth.SHAPES["tiny"], seed=0), "gqa": synth.gen_weights(GQA, seed=0)}


@pytest.mark.parametrize("name,n,K", [("tiny", 15, 4), ("tiny", 1, 1), ("gqa", 9, 16), ("gqa", 32, 7)])
def test_topk_matches_numpy_on_the_same_logits(weights, name, n, K):
    shape = synth.SHAPES["tiny"] if name == "tiny" else GQA
    g = cas.Model(shape, max_ctx=256)
    g.load_weights(weights[name])
    prompt = [int(x) for x in synth.gen_prompt(shape.vocab, 30, seed=3)]
    g.prefill(prompt)
    parents = synth.balanced_tree(n)
    toks = synth.gen_tree_tokens(parents, shape.vocab, seed=4)
    skip = [l % 2 for l in range(shape.n_layers)]
    lg = g.forward(toks, parents, 0, skip=skip)
    ids, probs = g.topk(K, n)
    for r in range(n):
        row = lg[r].astype(np.float64)
        want = np.argsort(-lg[r], kind="stable")[:K]
        assert np.array_equal(ids[r], want), (r, ids[r], want)
        p = np.exp(row - row.max())
        p /= p.sum()
        np.testing.assert_allclose(probs[r], p[want], rtol=2e-5, atol=1e-9)
    g.close()


def test_topk_errors(weights):
    shape = synth.SHAPES["tiny"]
    g = cas.Model(shape, max_ctx=64, max_tree=16)
    g.load_weights(weights["tiny"])
    with pytest.raises(cas.CasError, match="CAS_ERR_STATE"):
        g.topk(4, 1)
    g.forward([1, 2], [-1, 0], 0, logits=False)
    with pytest.raises(cas.CasError, match="CAS_ERR_ARG"):
        g.topk(4, 3)
    with pytest.raises(cas.CasError, match="CAS_ERR_ARG"):
        g.topk(17, 2)
    with pytest.raises(cas.CasError, match="CAS_ERR_ARG"):
        g.topk(0, 2)
    g.close()


def _cfgs(L):
    q3 = tuple(1 if l % 4 == 3 else 0 for l in range(L))
    odd = tuple(l % 2 for l in range(L))
    return [dytc.DraftConfig("q3", q3), dytc.DraftConfig("odd", odd), dytc.DraftConfig("odd_i8", odd, 1),
            dytc.DraftConfig("odd_i4", odd, 2), dytc.DraftConfig("pld", pld=True)]


@pytest.mark.parametrize("name", ["tiny", "gqa"])
def test_dytc_decoding_through_the_library_is_lossless(weights, name):
    shape = synth.SHAPES["tiny"] if name == "tiny" else GQA
    w = weights[name]
    base = [int(x) for x in synth.gen_prompt(shape.vocab, 24, seed=1)]
    prompt = base + base
    n_new = 32
    ref = O.ar_decode(O.OracleModel(shape, w, max_ctx=256), prompt, n_new)
    g = cas.Model(shape, max_ctx=256, max_tree=64)
    g.load_weights(w)
    g.build_int8()
    g.build_int4()
    cfgs = _cfgs(shape.n_layers)
    params = dytc.DytcParams(max_tree=24, k_max=3, t_min=1.1, top_k=3, top_p=0.5)
    out, excused = [], 0
    stats = {}
    while len(out) < n_new:
        est = dytc.AcceptanceEstimator({"q3": 0.9, "odd": 0.8, "odd_i8": 0.75, "odd_i4": 0.72, "pld": 0.05})
        cost = {"q3": 0.3, "odd": 0.2, "odd_i8": 0.18, "odd_i4": 0.15, "pld": 0.01}
        seg = dytc.cas_decode_dytc(dytc.LibraryBackend(g), prompt + out, n_new - len(out), cfgs, cfgs[-1], est,
                                   cost, params, shape.n_layers, stats)
        i = next((k for k, (a, b) in enumerate(zip(seg, ref[len(out):])) if a != b), None)
        if i is None:
            out += seg
            break
        pos = len(out) + i
        seq = prompt + ref[:pos]
        m = O.OracleModel(shape, w, max_ctx=256)
        m.prefill(seq[:-1])
        lg = np.sort(m.forward([seq[-1]], [-1])[0])
        margin = lg[-1] - lg[-2]
        assert shape.dtype == "bf16" and margin <= 0.05, f"divergence at token {pos}, oracle margin {margin}"
        excused += 1
        out = ref[:pos + 1]
    assert out[:n_new] == ref
    assert sum(stats["expansions"].get(c, 0) for c in ("q3", "odd", "odd_i8", "odd_i4")) > 0
    # the library's own greedy decoding agrees with its speculative decoding
    if excused == 0:
        assert decode.ar_decode(g, prompt, n_new) == ref
    g.close()
