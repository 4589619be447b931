"""A draft that computes the target's function gives the verify's bits.

Self-speculative drafting skips layers; where a skipped layer contributes
nothing to the residual stream (here layer 1 of a two-layer decoder at the
full 7B layer shapes, with its W_o and W_down set to zero), the skip draft
computes exactly the target's function.  The library's one-row draft then
returns the root row of a 32-node verify bit for bit (MFMA tiles, the
default): the row reductions do not depend on the call's row count, the
skipped layer adds exact zeros, and the O projection's merge-on-load gives
the merge kernel's bits.  With the GEMV-style tiles switched on
(`cas_set_gemv`) the draft's wide GEMMs sum in another order: the row
moves by rounding only (well inside the bf16 parity bar), and switching
them off again restores the verify's bits.
"""
import numpy as np
import pytest

from paper_2510_26843_amd import cas, synth

pytestmark = pytest.mark.gpu

SHAPE = synth.SHAPES["llama2_7b"].with_layers(2)
LC = 1024


@pytest.fixture(scope="module")
def model():
    w = synth.gen_weights(SHAPE, seed=31)
    for n in ("wo", "w_down"):
        w["layers"][1][n] = np.zeros_like(w["layers"][1][n])
    k, v = synth.gen_kv(SHAPE.n_layers, SHAPE.n_kv_heads, LC, SHAPE.head_dim, seed=32)
    g = cas.Model(SHAPE, max_ctx=LC + 128, max_tree=128)
    g.load_weights(w)
    for l in range(SHAPE.n_layers):
        g.kv_load(l, synth.f32_to_bf16_bits(k[l]), synth.f32_to_bf16_bits(v[l]))
    g.set_committed(LC)
    yield g
    g.close()


def _tree():
    parents = synth.tree_from_branching(*synth.TREE_7B)
    return synth.gen_tree_tokens(parents, SHAPE.vocab, seed=33), parents


def test_skip_draft_of_a_zero_layer_gives_the_verify_bits(model):
    toks, parents = _tree()
    ref = model.forward(toks, parents)[0]
    for skip in ([0, 1], None):  # the exact draft, and a one-row verify
        got = model.forward(toks[:1], parents[:1], skip=skip)[0]
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), skip
    # the attention-window draft with a window covering the whole context
    got = model.forward(toks[:1], parents[:1], skip=[0, 1], attn_window=(4, LC))[0]
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_gemv_tiles_move_the_draft_by_rounding_only(model):
    toks, parents = _tree()
    ref = model.forward(toks, parents)[0]
    model.set_gemv(True)
    try:
        got = model.forward(toks[:1], parents[:1], skip=[0, 1])[0]
    finally:
        model.set_gemv(False)
    err = float(np.abs(got - ref).max() / np.abs(ref).max())
    print(f"[gemv] one-row draft with GEMV tiles vs the verify's root row: {err:.2e} of max |logit|")
    assert 0 < err < 2e-2, err
    back = model.forward(toks[:1], parents[:1], skip=[0, 1])[0]
    assert np.array_equal(back.view(np.uint32), ref.view(np.uint32))
