"""The build with device checks (libcas_debug.so, -DCAS_DEBUG) and the
per-kernel profile switch.

- With valid inputs no device check fails, and the debug build's logits,
  acceptance, top-K and committed KV are the release build's, bit for bit:
  the checks guard accesses without changing any arithmetic.
- A slot-capacity check made to fail from the host (the checks are told to
  allow fewer slots than the cache holds, so every access stays inside the
  real cache) is reported: the check word holds its code and the
  synchronising call returns CAS_ERR_DEVICE; after the limit is lifted the
  next round is the release build's again.
- CAS_PROFILE=1 prints per-kernel-class totals when the Model closes.
"""
import numpy as np
import pytest

from paper_2510_26843_amd import cas, synth

pytestmark = pytest.mark.gpu

TINY = synth.SHAPES["tiny"]
GQA = synth.ModelShape("gqa_small", 2, 512, 8, 2, 64, 1376, 1024, 5e5, 1e-6, "bf16")
SLOT_CHECKS = {4, 6, 7}  # slot capacity (embedding), KV write slot, attention slots


def _pair(shape, seed):
    w = synth.gen_weights(shape, seed=seed)
    ms = []
    for debug in (False, True):
        m = cas.Model(shape, max_ctx=512, max_tree=128, debug=debug)
        m.load_weights(w)
        m.build_int8()
        m.build_int4()
        ms.append(m)
    return ms


def _session(m, shape, seed):
    """Prefill, then three rounds of drafts (skip + W8A8, W4A4 with a window,
    an appended level), verify, top-K, acceptance and compaction; returns
    everything the calls produced."""
    rng = np.random.default_rng(seed)
    prompt = synth.gen_prompt(shape.vocab, 70, seed=seed)
    m.prefill(prompt)
    skip = [l % 2 for l in range(shape.n_layers)]
    out = []
    for r, (br, n) in enumerate((((3, 2, 1), 15), ((4, 2, 2, 1, 1), 32), ((2,) * 6, 100))):
        parents = synth.tree_from_branching(br, n)
        toks = [int(t) for t in rng.integers(0, shape.vocab, n)]
        out.append(m.forward(toks[:1], parents[:1], skip=skip, act_quant=1))
        out.append(m.forward(toks[1:4], parents[1:4], node_offset=1, act_quant=2, attn_window=(4, 32)))
        out.append(m.topk(4, 3)[0])
        out.append(m.forward(toks, parents))
        ids, probs = m.topk(5, n)
        out += [ids, probs]
        path, bonus = m.accept()
        out.append(np.array(path + [bonus]))
        m.compact(path if r != 1 else [0, 1])
        assert m.debug_check() == 0
    k, v = m.kv_read(1, m.committed)
    return out + [k, v]


@pytest.mark.parametrize("shape", [TINY, GQA], ids=["tiny_f32", "gqa_bf16"])
def test_debug_build_matches_release_bitwise(shape):
    rel, dbg = _pair(shape, seed=5)
    assert rel._L.cas_debug_build() == 0 and dbg._L.cas_debug_build() == 1
    a = _session(rel, shape, 11)
    b = _session(dbg, shape, 11)
    assert len(a) == len(b)
    for i, (x, y) in enumerate(zip(a, b)):
        assert x.shape == y.shape and np.array_equal(x.view(np.uint8), y.view(np.uint8)), f"output {i} differs"
    assert dbg.debug_check() == 0
    # release build: the word is never written and the limit is refused
    assert rel.debug_check() == 0
    with pytest.raises(cas.CasError) as e:
        rel.debug_limit_slots(64)
    assert e.value.status == cas.ERR_UNSUPPORTED
    rel.close()
    dbg.close()


def test_slot_check_reports_and_recovers():
    shape = GQA
    rel, dbg = _pair(shape, seed=6)
    prompt = synth.gen_prompt(shape.vocab, 40, seed=2)
    for m in (rel, dbg):
        m.prefill(prompt)
    parents = synth.tree_from_branching((2, 2), 7)
    toks = [int(t) for t in synth.gen_tree_tokens(parents, shape.vocab, seed=3)]
    # the checks now allow slots < 42: the 7-node round needs slots 40..46,
    # all inside the real 512-slot cache
    dbg.debug_limit_slots(42)
    dbg.forward(toks, parents, logits=False)
    code = dbg.debug_check()
    assert code in SLOT_CHECKS, code
    assert dbg.debug_check() == 0  # read clears it
    # a synchronising call reports a failed check as CAS_ERR_DEVICE
    with pytest.raises(cas.CasError) as e:
        dbg.forward(toks, parents)
    assert e.value.status == cas.ERR_DEVICE and "device check failed" in str(e.value)
    assert dbg.debug_check() == 0
    with pytest.raises(cas.CasError) as e:
        dbg.debug_limit_slots(513)  # beyond max_ctx
    assert e.value.status == cas.ERR_ARG
    # lifted: the next round is the release build's, bit for bit
    dbg.debug_limit_slots(0)
    a = rel.forward(toks, parents)
    b = dbg.forward(toks, parents)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    pa, pb = rel.accept(), dbg.accept()
    assert pa == pb
    rel.compact(pa[0])
    dbg.compact(pb[0])
    ka, va = rel.kv_read(0, rel.committed)
    kb, vb = dbg.kv_read(0, dbg.committed)
    assert np.array_equal(ka, kb) and np.array_equal(va, vb)
    assert dbg.debug_check() == 0
    rel.close()
    dbg.close()


def test_profile_switch_prints_kernel_table(monkeypatch, capsys):
    monkeypatch.setenv("CAS_PROFILE", "1")
    w = synth.gen_weights(TINY, seed=1)
    m = cas.Model(TINY, max_ctx=256, max_tree=32)
    m.load_weights(w)
    m.prefill(synth.gen_prompt(TINY.vocab, 20, seed=1))
    parents = synth.tree_from_branching((3, 2), 9)
    m.forward(synth.gen_tree_tokens(parents, TINY.vocab, seed=2), parents)
    m.close()
    err = capsys.readouterr().err
    assert "kernel class" in err and "gemm_qkv" in err and "attn" in err, err
