"""How far an fp32 implementation of the bf16 numerics contract lands from the
fp64 oracle: the basis of the full-depth tolerance of the bf16 parity tests.

`fp32_contract.Fp32ContractModel` implements the decoder step in fp32 with
bf16 rounding at the contract's points (weights; the inputs of every linear
layer; q, k and v after RoPE), written independently of the oracle and of the
HIP library.  It is a second correct implementation of the same definition,
so its distance from the oracle is what any fp32 implementation of the
contract may show.

What the tests establish (CPU, Llama-2-7B shapes with the benchmark's seeded
weights, the 32-node (4,2,2,1,1) tree over a seeded synthetic bf16 cache):
- one layer: the emulation agrees with the oracle to 1e-6 on rows where no
  bf16 rounding decision differs; where one does (an fp32 sum a hair on the
  other side of a rounding boundary), the row moves by about 1e-3 of max
  |logit|, because one changed bf16 input moves every output of the next
  linear layer and so flips further roundings downstream;
- the spread is intrinsic: two fp32 implementations that differ only in the
  summation order of their linear layers differ from each other by about as
  much as each differs from the oracle;
- at full depth (32 layers) on the benchmark's configuration the emulation
  lands 2.3e-2 (max row) from the oracle, above 2e-2; the bf16 parity tests of
  the library therefore hold full-depth rows to 4e-2;
- with quantised activations (W8A8, W4A4) a code that lands on the other
  side of a grid boundary moves a row far more than a bf16 step does: the
  emulation agrees with the oracle to fp32 accuracy on some drafts and moves
  by about 2e-2 on others (small decoders, below), and by 8.6e-2 on the
  level-1 rows of the 13B W8A8 draft of 20 layers (the library: 8.7e-2).
"""
import concurrent.futures as fut

import numpy as np
import pytest

from oracle import oracle as O
from paper_2510_26843_amd import synth

from fp32_contract import Fp32ContractModel

pytestmark = pytest.mark.slow

SHAPE = synth.SHAPES["llama2_7b"]


def _row_err(got, ref):
    return (np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1))


def _cache(layers, ctx):
    """The committed cache of the 7B full-size tests: per layer the first ctx
    slots of the seeded 8192-slot synthetic cache, rounded to bf16."""
    def one(l):
        k, v = synth.gen_kv(1, SHAPE.n_kv_heads, 8192, SHAPE.head_dim, seed=1000 + l)
        kb = synth.f32_to_bf16_bits(np.ascontiguousarray(k[0][:, :ctx]))
        vb = synth.f32_to_bf16_bits(np.ascontiguousarray(v[0][:, :ctx]))
        return synth.bf16_bits_to_f32(kb), synth.bf16_bits_to_f32(vb)
    with fut.ThreadPoolExecutor(max_workers=8) as ex:
        return list(ex.map(one, layers))


def _models(shape, w, ctx, layers, k_chunks=(1,)):
    kv = _cache(layers, ctx)
    ems = [Fp32ContractModel(shape, w, ctx + 64, k_chunks=kc) for kc in k_chunks]
    o = O.OracleModel(shape, w, max_ctx=ctx + 64)
    for l, (kf, vf) in zip(layers, kv):
        for e in ems:
            e.set_kv(l, kf, vf)
        o.set_kv(l, kf, vf)
    for e in ems:
        e.Lc = ctx
    o.set_committed(ctx)
    return ems, o


def _tree():
    parents = synth.tree_from_branching(*synth.TREE_7B)
    return parents, synth.gen_tree_tokens(parents, SHAPE.vocab, seed=1024 + len(parents))


def test_one_layer_flips_only():
    shape = SHAPE.with_layers(1)
    w = synth.gen_weights(shape, seed=0)
    (em,), o = _models(shape, w, 256, [0])
    parents, toks = _tree()
    err = _row_err(em.forward(toks, parents), o.forward(toks, parents))
    print(f"[contract] one layer, fp32 emulation vs oracle: rows {np.array2string(err, precision=1)}")
    # rows without a differing rounding decision agree to fp32 accuracy,
    # the others move by about 1e-3 of max |logit|
    assert err.min() < 1e-5, err.min()
    assert err.max() < 6e-3, err.max()


def test_spread_is_the_contract_not_an_implementation():
    shape = SHAPE.with_layers(4)
    w = synth.gen_weights(shape, seed=0)
    (e1, e4), o = _models(shape, w, 256, range(4), k_chunks=(1, 4))
    parents, toks = _tree()
    a, b, r = e1.forward(toks, parents), e4.forward(toks, parents), o.forward(toks, parents)
    ea, eb, eab = _row_err(a, r).max(), _row_err(b, r).max(), _row_err(a, b).max()
    print(f"[contract] 4 layers: emulation vs oracle {ea:.2e}, 4-range summation vs oracle {eb:.2e}, "
          f"the two emulations {eab:.2e}")
    # two fp32 implementations differ from each other by about as much as
    # each differs from the oracle
    assert eab > 0.3 * min(ea, eb), (ea, eb, eab)
    assert max(ea, eb) < 2e-2


@pytest.mark.timeout(900)
def test_full_depth_benchmark_configuration():
    """32 layers, context 1024: the configuration of the benchmark and of the
    library's full-depth parity test (same weights, tree, tokens and cache)."""
    w = synth.gen_weights(SHAPE, seed=0)
    (em,), o = _models(SHAPE, w, 1024, range(SHAPE.n_layers))
    parents, toks = _tree()
    err = _row_err(em.forward(toks, parents), o.forward(toks, parents))
    print(f"[contract] 32 layers, ctx 1024: fp32 emulation vs oracle max {err.max():.3e}, "
          f"median {np.median(err):.3e}, min {err.min():.3e}")
    # the library's full-depth bar (4e-2) covers what a correct fp32
    # implementation shows; the emulation itself lands above 2e-2
    assert err.max() < 4e-2, err.max()
    assert np.median(err) > 5e-3, "the contract's spread at depth has vanished: revisit the bar"


GQA = synth.ModelShape("gqa_small", 2, 512, 8, 2, 64, 1376, 1024, 5e5, 1e-6, "bf16")
MHA = synth.ModelShape("mha_small", 2, 1024, 8, 8, 128, 2752, 4096, 1e4, 1e-6, "bf16")


@pytest.mark.parametrize("shape,skip,aq,exact", [(GQA, [0, 1], 1, True), (GQA, [0, 1], 2, True),
                                                 (MHA, [0, 0], 1, False)])
def test_quantised_drafts_spread(shape, skip, aq, exact):
    """The W8A8 (aq 1) and W4A4 (aq 2) contract in fp32 against the oracle on
    the small decoders of the library's draft parity tests: a 33-token
    prefill by each side, then a 15-node tree drafted depth by depth.  Where
    no code lands differently the two agree to fp32 accuracy (the one-layer
    GQA drafts); where the prefill's fp32 sums move an activation across a
    boundary of the 255-level grid, the rows move by about 2e-2 of max |logit|
    (the two-layer MHA draft), which the library's 6e-2 bar for these drafts
    covers."""
    w = synth.gen_weights(shape, seed=9)
    prompt = [int(x) for x in synth.gen_prompt(shape.vocab, 33, seed=3)]
    em = Fp32ContractModel(shape, w, 512)
    o = O.OracleModel(shape, w, 512, int8=aq == 1, int4=aq == 2)
    z = np.zeros((shape.n_kv_heads, 0, shape.head_dim), np.float32)
    for l in range(shape.n_layers):
        em.set_kv(l, z, z)
    em.prefill(prompt)
    o.prefill(prompt)
    parents = synth.tree_from_branching((3, 2, 1), 15)
    toks = synth.gen_tree_tokens(parents, shape.vocab, seed=4)
    errs = []
    for a, b in ((0, 1), (1, 4), (4, 10), (10, 15)):
        errs.append(_row_err(em.forward(toks[a:b], parents[a:b], a, skip=skip, act_quant=aq),
                             o.forward(toks[a:b], parents[a:b], a, skip=skip, act_quant=aq)).max())
    print(f"[contract] {shape.name} skip {skip} act_quant {aq}: fp32 emulation vs oracle per level "
          f"{['%.2e' % e for e in errs]}")
    if exact:
        assert max(errs) < 1e-5, errs
    else:
        assert 1e-3 < max(errs) < 6e-2, errs
