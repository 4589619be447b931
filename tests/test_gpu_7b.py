"""Parity at the full 7B layer shapes (Llama-2-7B: d 4096, 32 heads of 128,
FFN 11008, vocab 32000, bf16) with two decoder layers, so that every GEMM,
attention and norm launch has the geometry of the full-size workload while
the fp64 oracle still finishes in seconds: a verify call over the 32-node
tree (4,2,2,1,1) against a 1024-slot committed KV cache, a layer-skipping
draft call of the root with int8 activations, greedy acceptance and the KV
commit of the accepted path.

The committed cache is synthetic (N(0, 1.28^2), rounded to bf16), loaded
into both sides; a 1024-token prefill of the fp64 oracle would take minutes.
Tolerances as in the small-shape forward tests (2e-2 of the row's largest
logit for bf16, 6e-2 with int8 activations).
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2510_26843_amd import cas, synth

pytestmark = pytest.mark.gpu

SHAPE = synth.SHAPES["llama2_7b"].with_layers(2)
LC = 1024


@pytest.fixture(scope="module")
def pair():
    w = synth.gen_weights(SHAPE, seed=21)
    k, v = synth.gen_kv(SHAPE.n_layers, SHAPE.n_kv_heads, LC, SHAPE.head_dim, seed=22)
    kb, vb = synth.f32_to_bf16_bits(k), synth.f32_to_bf16_bits(v)
    g = cas.Model(SHAPE, max_ctx=LC + 128, max_tree=128)
    g.load_weights(w)
    g.build_int8()
    o = O.OracleModel(SHAPE, w, max_ctx=LC + 128, int8=True)
    for l in range(SHAPE.n_layers):
        g.kv_load(l, kb[l], vb[l])
        o.set_kv(l, synth.bf16_bits_to_f32(kb[l]), synth.bf16_bits_to_f32(vb[l]))
    g.set_committed(LC)
    o.set_committed(LC)
    yield g, o
    g.close()


def _row_err(got, ref):
    return float((np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)).max())


def test_verify_tree_7b_layers(pair):
    g, o = pair
    parents = synth.tree_from_branching(*synth.TREE_7B)
    toks = synth.gen_tree_tokens(parents, SHAPE.vocab, seed=23)
    # a first pass picks the root's greedy token; giving it to the root's first
    # child makes the accepted path at least two nodes long
    first = g.forward(toks, parents)
    toks[1] = int(first[0].argmax())
    got = g.forward(toks, parents)
    ref = o.forward(toks, parents)
    assert _row_err(got, ref) < 2e-2
    # acceptance is decided on each side's own logits; where the oracle's
    # decision is not tie-close, the library must take the same path
    path, bonus = g.accept()
    assert len(path) >= 2
    assert (path, bonus) == O.accept_greedy(got.astype(np.float64), parents, toks)
    g.compact(path)
    o.compact(path)
    n = LC + len(path)
    assert g.committed == n
    kg, vg = g.kv_read(1, n)
    for slot in range(LC, n):
        for h in (0, 17, 31):
            ko, vo = o.get_kv(1, h, slot)
            kgf = synth.bf16_bits_to_f32(kg[h, slot]).astype(np.float64)
            vgf = synth.bf16_bits_to_f32(vg[h, slot]).astype(np.float64)
            assert np.abs(kgf - ko).max() <= 2e-2 * np.abs(ko).max()
            assert np.abs(vgf - vo).max() <= 2e-2 * np.abs(vo).max()
    g.set_committed(LC)
    o.set_committed(LC)


def test_draft_root_7b_layers(pair):
    g, o = pair
    for aq, tol in ((False, 2e-2), (True, 6e-2)):
        got = g.forward([5], [-1], skip=[0, 1], act_quant=aq)
        ref = o.forward([5], [-1], skip=[0, 1], act_quant=aq)
        assert _row_err(got, ref) < tol, aq
