"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Every check here is chosen so that a plausible slip in the oracle (a dropped
term, a wrong sign or index, a transposed operand, a wrong position or mask)
fails at least one of them:
  - a chain tree is ordinary causal decoding, which reduces to library routines
    (torch rms_norm, scaled_dot_product_attention with a causal mask, silu,
    complex-number rotation for RoPE): the textbook model;
  - tree verification equals independent causal forwards along each
    root-to-node path (the exactness of tree attention, Sec. 4.2);
  - greedy speculative decoding equals greedy autoregressive decoding token
    for token (lossless decoding, Sec. 5.1);
  - closed forms: skip-all logits, one-key attention, RoPE relative-position
    identity, RMSNorm output scale, exact integer dot products;
  - structural invariants: skip-layer-l equals deleting layer l, GQA equals
    MHA with repeated KV projections, per-row independence.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import oracle as O
from paper_2510_26843_amd import synth

TINY = synth.SHAPES["tiny"]
# a small bf16 GQA decoder (2 query heads per kv head), for bf16 and GQA paths
SMALL_BF16 = synth.ModelShape("small_bf16", 3, 128, 4, 2, 32, 320, 512, 1e4, 1e-6, "bf16")


@pytest.fixture(scope="module")
def tiny():
    return synth.gen_weights(TINY, seed=0)


@pytest.fixture(scope="module")
def small():
    return synth.gen_weights(SMALL_BF16, seed=5)


# ---------------------------------------------------------------- textbook model

def _w64(a, bf16):
    if bf16:
        return torch.from_numpy(synth.bf16_bits_to_f32(a).astype(np.float64))
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def _rope_complex(x, pos, theta):
    """RoPE as multiplication of the complex numbers x[i] + j x[i+hd/2] by
    exp(j pos theta^(-2i/hd)).  x: [S, heads, hd] float64."""
    hd = x.shape[-1]
    half = hd // 2
    z = torch.complex(x[..., :half], x[..., half:])
    inv = theta ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)
    ang = pos.to(torch.float64)[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    z = z * rot
    return torch.cat([z.real, z.imag], dim=-1)


def _qlin(x, w, bf16, qmax):
    """x @ W^T as a quantised linear layer: per-row codes of x and
    per-output-channel codes of W (the oracle's pinned quantisers), an exact
    int64 product, then (fp32(acc) * s_x) * s_w in float32."""
    xq, sx = O.quant_rows(x.numpy().astype(np.float32), qmax)
    wq, sw = O.quant_weight(w, bf16, qmax)
    acc = xq.astype(np.int64) @ wq.astype(np.int64).T
    y = (acc.astype(np.float32) * sx[:, None]) * sw[None, :]
    return torch.from_numpy(y.astype(np.float64))


def textbook_logits(shape, w, tokens, round_bf16=False, mask=None, qmax=None):
    """Causal decoder over `tokens` from library routines, float64.  With
    round_bf16 the storage points round through torch's bfloat16 cast; mask
    ([S][S] bool, True = visible) replaces the causal mask; qmax (127 or 7)
    makes the seven projections of every layer quantised linear layers."""
    bf16 = shape.dtype == "bf16"
    if qmax is None:
        mm = lambda x, a: x @ _w64(a, bf16).T
    else:
        mm = lambda x, a: _qlin(x, a, bf16, qmax)
    rb = (lambda t: t.to(torch.float32).to(torch.bfloat16).to(torch.float64)) if round_bf16 else (lambda t: t)
    S = len(tokens)
    H, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    pos = torch.arange(S)
    x = _w64(w["embed"], bf16)[torch.as_tensor(np.asarray(tokens, dtype=np.int64))]
    for lw in w["layers"]:
        xn = rb(F.rms_norm(x, (shape.d_model,), weight=torch.from_numpy(lw["attn_norm"]).double(), eps=shape.rms_eps))
        q = mm(xn, lw["wq"]).view(S, H, hd)
        k = mm(xn, lw["wk"]).view(S, Hkv, hd)
        v = mm(xn, lw["wv"]).view(S, Hkv, hd)
        q = rb(_rope_complex(q, pos, shape.rope_theta))
        k = rb(_rope_complex(k, pos, shape.rope_theta))
        v = rb(v)
        if mask is None:
            o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                               v.transpose(0, 1)[None], is_causal=True, enable_gqa=True)
        else:
            o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                               v.transpose(0, 1)[None], attn_mask=torch.as_tensor(mask),
                                               enable_gqa=True)
        o = rb(o[0].transpose(0, 1).reshape(S, H * hd))
        x = x + mm(o, lw["wo"])
        xn = rb(F.rms_norm(x, (shape.d_model,), weight=torch.from_numpy(lw["ffn_norm"]).double(), eps=shape.rms_eps))
        s = rb(F.silu(mm(xn, lw["w_gate"])) * mm(xn, lw["w_up"]))
        x = x + mm(s, lw["w_down"])
    xn = rb(F.rms_norm(x, (shape.d_model,), weight=torch.from_numpy(w["final_norm"]).double(), eps=shape.rms_eps))
    return (xn @ _w64(w["lm_head"], bf16).T).numpy()


def test_chain_equals_textbook_fp32(tiny):
    toks = synth.gen_prompt(TINY.vocab, 24, seed=11)
    m = O.OracleModel(TINY, tiny, max_ctx=64)
    got = m.forward(toks, synth.chain_parents(len(toks)))
    ref = textbook_logits(TINY, tiny, toks)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 1e-12, err


def test_chain_equals_textbook_bf16_gqa(small):
    toks = synth.gen_prompt(SMALL_BF16.vocab, 20, seed=12)
    m = O.OracleModel(SMALL_BF16, small, max_ctx=64)
    got = m.forward(toks, synth.chain_parents(len(toks)))
    # without storage rounding the textbook model differs by bf16 rounding noise only
    ref_exact = textbook_logits(SMALL_BF16, small, toks, round_bf16=False)
    err0 = np.abs(got - ref_exact).max() / np.abs(ref_exact).max()
    assert err0 < 3e-2, err0
    # with the same storage points rounded, the two agree far more closely
    ref = textbook_logits(SMALL_BF16, small, toks, round_bf16=True)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 2e-3, err
    assert err < err0 / 4


@pytest.mark.parametrize("sink,win", [(4, 8), (0, 5), (3, 100), (30, 4)])
def test_attention_window_equals_masked_textbook(tiny, sink, win):
    """Efficient-attention draft (StreamingLLM-style): after a 24-token
    prefix is committed with full attention, a 6-token chain that sees only
    the first `sink` and the last `win` committed slots (plus its own chain)
    equals the textbook decoder under that explicit mask.  A sink or window
    covering the prefix gives plain causal attention."""
    P, C = 24, 6
    toks = synth.gen_prompt(TINY.vocab, P + C, seed=13)
    m = O.OracleModel(TINY, tiny, max_ctx=64)
    m.prefill(list(toks[:P]))
    got = m.forward(toks[P:], synth.chain_parents(C), attn_window=(sink, win))
    S = P + C
    mask = np.tril(np.ones((S, S), dtype=bool))
    lo = min(sink, P)
    hi = max(lo, P - win)
    for i in range(P, S):
        mask[i, :P] = False
        mask[i, :lo] = True
        mask[i, hi:P] = True
    ref = textbook_logits(TINY, tiny, toks, mask=mask)[P:]
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 1e-12, err
    if lo == P or hi == lo:
        full = textbook_logits(TINY, tiny, toks)[P:]
        assert np.abs(full - ref).max() / np.abs(full).max() < 1e-12
    else:
        full = m.forward(toks[P:], synth.chain_parents(C))
        assert np.abs(full - got).max() > 1e-6  # the window changes the result


# ---------------------------------------------------------------- tree exactness

def _fresh(shape, w, prompt, max_ctx=128, int8=False):
    m = O.OracleModel(shape, w, max_ctx=max_ctx, int8=int8)
    if len(prompt):
        m.prefill(list(prompt))
    return m


@pytest.mark.parametrize("which", ["tiny", "small"])
def test_tree_equals_per_path_forward(which, tiny, small):
    shape, w = (TINY, tiny) if which == "tiny" else (SMALL_BF16, small)
    prompt = synth.gen_prompt(shape.vocab, 9, seed=13)
    parents = synth.tree_from_branching((3, 2, 1), 15)
    toks = synth.gen_tree_tokens(parents, shape.vocab, seed=14)
    m = _fresh(shape, w, prompt)
    tree = m.forward(toks, parents)
    depth, anc = O.tree_metadata(parents)
    for i in range(len(parents)):
        path = [j for j in range(len(parents)) if (anc[i] >> j) & 1]
        ref_m = _fresh(shape, w, prompt)
        lg = ref_m.forward([int(toks[j]) for j in path], synth.chain_parents(len(path)))
        assert np.array_equal(lg[-1], tree[i]), f"node {i} path {path}"


def test_row_independence(tiny):
    prompt = synth.gen_prompt(TINY.vocab, 5, seed=15)
    parents = synth.tree_from_branching((4, 2, 2, 1, 1), 32)
    toks = synth.gen_tree_tokens(parents, TINY.vocab, seed=16)
    full = _fresh(TINY, tiny, prompt).forward(toks, parents)
    need = [i in (7, 30) for i in range(32)]
    part = _fresh(TINY, tiny, prompt).forward(toks, parents, need=need)
    assert np.array_equal(full[7], part[7]) and np.array_equal(full[30], part[30])


def test_split_calls_equal_one_call(tiny):
    """Feeding the tree depth by depth in appended calls gives the same rows."""
    prompt = synth.gen_prompt(TINY.vocab, 6, seed=17)
    parents = synth.tree_from_branching((3, 2, 1), 15)
    toks = synth.gen_tree_tokens(parents, TINY.vocab, seed=18)
    one = _fresh(TINY, tiny, prompt).forward(toks, parents)
    m = _fresh(TINY, tiny, prompt)
    rows = [m.forward(toks[a:b], parents[a:b], a) for a, b in ((0, 1), (1, 4), (4, 10), (10, 15))]
    assert np.array_equal(np.concatenate(rows), one)


# ---------------------------------------------------------------- closed forms

def test_skip_all_closed_form(small):
    sh = SMALL_BF16
    prompt = synth.gen_prompt(sh.vocab, 4, seed=19)
    parents = synth.tree_from_branching((2, 2), 5)
    toks = synth.gen_tree_tokens(parents, sh.vocab, seed=20)
    m = _fresh(sh, small, prompt)
    got = m.forward(toks, parents, skip=[1] * sh.n_layers)
    E = synth.bf16_bits_to_f32(small["embed"]).astype(np.float64)[toks]
    xn = E / np.sqrt((E * E).mean(axis=1, keepdims=True) + sh.rms_eps)
    xn = np.vectorize(O.round_bf16)(xn)
    ref = xn @ synth.bf16_bits_to_f32(small["lm_head"]).astype(np.float64).T
    assert np.allclose(got, ref, rtol=0, atol=1e-12 * np.abs(ref).max())


def test_skip_layer_equals_deleted_layer(tiny):
    keep = [0, 2, 3]
    sh3 = dataclasses.replace(TINY, n_layers=3)
    w3 = dict(tiny)
    w3["layers"] = [tiny["layers"][l] for l in keep]
    parents = synth.tree_from_branching((3, 2, 1), 15)
    toks = synth.gen_tree_tokens(parents, TINY.vocab, seed=21)
    a = O.OracleModel(TINY, tiny, max_ctx=64).forward(toks, parents, skip=[0, 1, 0, 0])
    b = O.OracleModel(sh3, w3, max_ctx=64).forward(toks, parents)
    assert np.array_equal(a, b)


def test_gqa_equals_mha_with_repeated_kv(small):
    sh = SMALL_BF16
    G = sh.n_heads // sh.n_kv_heads
    mha = dataclasses.replace(sh, n_kv_heads=sh.n_heads)
    wm = {k: v for k, v in small.items() if k != "layers"}
    wm["layers"] = []
    for lw in small["layers"]:
        d = dict(lw)
        for n in ("wk", "wv"):
            blocks = lw[n].reshape(sh.n_kv_heads, sh.head_dim, sh.d_model)
            d[n] = np.repeat(blocks, G, axis=0).reshape(sh.n_heads * sh.head_dim, sh.d_model)
        wm["layers"].append(d)
    prompt = synth.gen_prompt(sh.vocab, 7, seed=22)
    parents = synth.tree_from_branching((2, 2, 1), 7)
    toks = synth.gen_tree_tokens(parents, sh.vocab, seed=23)
    a = _fresh(sh, small, prompt).forward(toks, parents)
    b = _fresh(mha, wm, prompt).forward(toks, parents)
    assert np.array_equal(a, b)


def test_attention_one_key_and_uniform_scores():
    rng = np.random.default_rng(0)
    q = rng.standard_normal(64)
    k = rng.standard_normal((1, 64))
    v = rng.standard_normal((1, 64))
    assert np.array_equal(O.attend(q, k, v), v[0])
    # equal keys give equal weights: the output is the mean of the values
    ks = np.repeat(k, 5, axis=0)
    vs = rng.standard_normal((5, 64))
    assert np.allclose(O.attend(q, ks, vs), vs.mean(axis=0), atol=1e-14)
    # weights sum to one: constant values come back unchanged
    kk = rng.standard_normal((9, 64))
    assert np.allclose(O.attend(q, kk, np.full((9, 64), 2.5)), 2.5, atol=1e-14)
    # the weights are softmax of the scaled scores (one coordinate at a time)
    vv = np.eye(9, 64)
    w = O.attend(q, kk, vv)[:9]
    s = kk @ q / 8.0
    ref = np.exp(s - s.max()) / np.exp(s - s.max()).sum()
    assert np.allclose(w, ref, atol=1e-15)


def test_rope_properties():
    rng = np.random.default_rng(1)
    hd, theta = 128, 1e4
    q, k = rng.standard_normal(hd), rng.standard_normal(hd)
    for m_, n_ in ((5, 3), (1000, 17), (40, 40)):
        lhs = O.rope(q, m_, theta) @ O.rope(k, n_, theta)
        rhs = O.rope(q, m_ - n_, theta) @ k
        assert abs(lhs - rhs) < 1e-9 * (1 + abs(lhs))
    assert np.array_equal(O.rope(q, 0, theta), q)
    assert abs(np.linalg.norm(O.rope(q, 777, theta)) - np.linalg.norm(q)) < 1e-12
    # agrees with the complex-number rotation
    ref = _rope_complex(torch.from_numpy(q)[None, None, :], torch.tensor([321]), theta)[0, 0].numpy()
    assert np.allclose(O.rope(q, 321, theta), ref, atol=1e-12)


def test_rmsnorm_scale_and_library():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(4096) * 3.0
    g = np.ones(4096, dtype=np.float32)
    y = O.rmsnorm_row(x, g, 1e-6)
    assert abs(np.sqrt((y * y).mean()) - 1.0) < 1e-6
    g2 = rng.standard_normal(4096).astype(np.float32)
    ref = F.rms_norm(torch.from_numpy(x), (4096,), weight=torch.from_numpy(g2).double(), eps=1e-6).numpy()
    assert np.allclose(O.rmsnorm_row(x, g2, 1e-6), ref, rtol=1e-13, atol=1e-13)


def test_round_bf16_matches_library_cast():
    rng = np.random.default_rng(3)
    xs = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                         # exact halfway points between neighbouring bf16 values
                         np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(2.0 + 2 ** -7), 2 ** -130 * 1.5], np.float32)])
    xs = xs.astype(np.float32)
    ref = torch.from_numpy(xs).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([O.round_bf16(float(x)) for x in xs])
    assert np.array_equal(got, ref)


# ---------------------------------------------------------------- int8

def test_quant_rows_properties():
    x = synth.gen_activations(64, 688, seed=3)
    q, s = O.quant_rows(x)
    for r in range(x.shape[0]):
        amax = np.abs(x[r]).max()
        if amax == 0:
            assert s[r] == 0 and not q[r].any()
            continue
        assert s[r] == np.float32(amax) / np.float32(127.0)
        assert np.abs(q[r]).max() == 127
        assert q[r][np.argmax(np.abs(x[r]))] == np.sign(x[r][np.argmax(np.abs(x[r]))]) * 127
        err = np.abs(x[r].astype(np.float64) - q[r].astype(np.float64) * np.float64(s[r]))
        assert (err <= 0.5 * np.float64(s[r]) * (1 + 1e-6)).all()


def test_int8_dot_exact():
    rng = np.random.default_rng(4)
    a = rng.integers(-127, 128, (5, 1000)).astype(np.int8)
    b = rng.integers(-127, 128, (7, 1000)).astype(np.int8)
    got = O.dot_i8_matrix(a, b)
    ref = a.astype(np.int64) @ b.astype(np.int64).T
    assert np.array_equal(got.astype(np.int64), ref)


def test_int8_draft_approximates_full(tiny):
    """The int8-activation draft is an approximation of the same model: its
    logits stay close to the full-precision ones (a transposed or unscaled
    operand would not)."""
    parents = synth.tree_from_branching((3, 2, 1), 15)
    toks = synth.gen_tree_tokens(parents, TINY.vocab, seed=24)
    m = O.OracleModel(TINY, tiny, max_ctx=64, int8=True)
    full = m.forward(toks, parents)
    q8 = m.forward(toks, parents, act_quant=True)
    err = np.abs(full - q8).max() / np.abs(full).max()
    assert 0 < err < 0.1, err


# ---------------------------------------------------------------- int4 (W4A4)

def test_quant_rows_int4_properties():
    x = synth.gen_activations(64, 688, seed=13)
    x[5] = 0.0
    q, s = O.quant_rows(x, 7)
    for r in range(x.shape[0]):
        amax = np.abs(x[r]).max()
        if amax == 0:
            assert s[r] == 0 and not q[r].any()
            continue
        assert s[r] == np.float32(amax) / np.float32(7.0)
        assert np.abs(q[r]).max() == 7
        i = np.argmax(np.abs(x[r]))
        assert q[r][i] == np.sign(x[r][i]) * 7
        err = np.abs(x[r].astype(np.float64) - q[r].astype(np.float64) * np.float64(s[r]))
        assert (err <= 0.5 * np.float64(s[r]) * (1 + 1e-6)).all()


def test_quant_int4_worked_example():
    """amax 3.5 gives the scale 0.5 exactly; x / s = 7, -3.5, 0.5, 0, -7, 2.5,
    1.5 round half to even: 7, -4, 0, 0, -7, 2, 2."""
    x = np.array([[3.5, -1.75, 0.25, 0.0, -3.5, 1.25, 0.75]], dtype=np.float32)
    q, s = O.quant_rows(x, 7)
    assert s[0] == np.float32(0.5)
    assert q[0].tolist() == [7, -4, 0, 0, -7, 2, 2]


@pytest.mark.parametrize("bf16", [False, True])
def test_quant_weight_int4_recovers_representable_rows(bf16):
    """Rows that are a power-of-two scale 2^-e times integer codes in [-7, 7]
    (each row with a +-7) quantise back to exactly those codes, with the scale
    amax / 7 = 2^-e."""
    rng = np.random.default_rng(14)
    codes = rng.integers(-7, 8, (48, 200))
    codes[np.arange(48), rng.integers(0, 200, 48)] = rng.choice([-7, 7], 48)
    scale = 2.0 ** -rng.integers(3, 9, 48)
    w = (codes * scale[:, None]).astype(np.float32)
    arr = synth.f32_to_bf16_bits(w) if bf16 else w
    q, s = O.quant_weight(arr, bf16, 7)
    assert np.array_equal(q.astype(np.int64), codes)
    assert np.array_equal(s.astype(np.float64), scale)


@pytest.mark.parametrize("which,qmax", [("tiny", 127), ("tiny", 7), ("small", 127), ("small", 7)])
def test_quantised_forward_equals_textbook(which, qmax, tiny, small):
    """The oracle's act_quant forward (1: W8A8, 2: W4A4) over a chain equals the
    textbook decoder whose seven projections per layer are quantised linear
    layers (codes of the rounded inputs and of the weights, exact integer
    products, fp32 dequantisation); the LM head stays full precision."""
    shape, w = (TINY, tiny) if which == "tiny" else (SMALL_BF16, small)
    bf16 = shape.dtype == "bf16"
    toks = [int(t) for t in synth.gen_prompt(shape.vocab, 9, seed=15)]
    m = O.OracleModel(shape, w, max_ctx=32, int8=qmax == 127, int4=qmax == 7)
    got = m.forward(toks, list(range(-1, len(toks) - 1)), act_quant=1 if qmax == 127 else 2)
    ref = textbook_logits(shape, w, toks, round_bf16=bf16, qmax=qmax)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 1e-9, err


def test_int4_draft_is_coarser_than_int8(tiny):
    """Both quantised drafts approximate the same model, int4 less closely."""
    parents = synth.tree_from_branching((3, 2, 1), 15)
    toks = synth.gen_tree_tokens(parents, TINY.vocab, seed=24)
    m = O.OracleModel(TINY, tiny, max_ctx=64, int8=True, int4=True)
    full = m.forward(toks, parents)
    e8 = np.abs(full - m.forward(toks, parents, act_quant=1)).max() / np.abs(full).max()
    e4 = np.abs(full - m.forward(toks, parents, act_quant=2)).max() / np.abs(full).max()
    assert 0 < e8 < e4 < 1.0, (e8, e4)


def test_int4_forward_needs_its_copy(tiny):
    m = O.OracleModel(TINY, tiny, max_ctx=32, int8=True)
    with pytest.raises(ValueError):
        m.forward([1, 2], [-1, 0], act_quant=2)
    with pytest.raises(ValueError):
        m.forward([1, 2], [-1, 0], act_quant=3)


# ---------------------------------------------------------------- acceptance, compaction, losslessness

def test_acceptance_main_path_and_decoys(tiny):
    prompt = synth.gen_prompt(TINY.vocab, 12, seed=25)
    ar = O.ar_decode(O.OracleModel(TINY, tiny, max_ctx=64), prompt, 4)
    # root = last prompt token; main path = next 3 greedy tokens; decoy siblings
    parents = [-1, 0, 0, 1, 1, 3, 3]
    toks = [int(prompt[-1]), ar[0], (ar[0] + 1) % TINY.vocab, ar[1], (ar[1] + 7) % TINY.vocab,
            (ar[2] + 3) % TINY.vocab, ar[2]]
    m = _fresh(TINY, tiny, prompt[:-1])
    lg = m.forward(toks, parents)
    path, bonus = O.accept_greedy(lg, parents, toks)
    assert path == [0, 1, 3, 6] and bonus == ar[3]
    # all decoys: nothing accepted, bonus is the plain greedy step
    toks2 = [int(prompt[-1]), (ar[0] + 1) % TINY.vocab, (ar[0] + 2) % TINY.vocab, 5, 6, 7, 8]
    m2 = _fresh(TINY, tiny, prompt[:-1])
    path2, bonus2 = O.accept_greedy(m2.forward(toks2, parents), parents, toks2)
    assert path2 == [0] and bonus2 == ar[0]


def test_compaction_equals_ar_cache(small):
    sh = SMALL_BF16
    prompt = synth.gen_prompt(sh.vocab, 10, seed=26)
    ar = O.ar_decode(O.OracleModel(sh, small, max_ctx=64), prompt, 3)
    parents = [-1, 0, 0, 2, 2, 4]
    toks = [int(prompt[-1]), 3, ar[0], 9, ar[1], ar[2]]
    m = _fresh(sh, small, prompt[:-1], max_ctx=64)
    path, bonus = O.accept_greedy(m.forward(toks, parents), parents, toks)
    assert path == [0, 2, 4, 5]
    m.compact(path)
    ref = _fresh(sh, small, list(prompt) + ar[:3], max_ctx=64)
    assert m.committed == ref.committed == len(prompt) + 3
    for l in range(sh.n_layers):
        for h in range(sh.n_kv_heads):
            for s in range(m.committed):
                a, b = m.get_kv(l, h, s), ref.get_kv(l, h, s)
                assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), (l, h, s)


def test_cas_equals_ar_tiny_config(tiny):
    """Greedy CAS decode with two draft levels and the static 15-node tree
    equals plain greedy decoding on the tiny fp32 decoder (64-token prompt,
    32 new tokens)."""
    prompt = synth.gen_prompt(TINY.vocab, 64, seed=1)
    ar = O.ar_decode(O.OracleModel(TINY, tiny, max_ctx=256), prompt, 32)
    parents = synth.tree_from_branching(*synth.TREE_TINY)
    skip = [0, 1, 1, 0]
    levels = {0: (skip, False), 1: (skip, True), 2: (skip, True)}
    st = {}
    cas = O.cas_decode_static(O.OracleModel(TINY, tiny, max_ctx=256, int8=True), prompt, 32, parents, levels, st)
    assert cas == ar
    assert st["rounds"] < 32


def test_cas_equals_ar_bf16_gqa(small):
    sh = SMALL_BF16
    prompt = synth.gen_prompt(sh.vocab, 16, seed=27)
    ar = O.ar_decode(O.OracleModel(sh, small, max_ctx=128), prompt, 20)
    parents = synth.tree_from_branching((4, 2, 2, 1, 1), 32)
    levels = {d: ([0, 1, 0], d > 0) for d in range(5)}
    cas = O.cas_decode_static(O.OracleModel(sh, small, max_ctx=128, int8=True), prompt, 20, parents, levels)
    assert cas == ar


def test_tree_metadata_brute_force():
    parents = synth.tree_from_branching((4, 2, 2, 1, 1), 32)
    depth, anc = O.tree_metadata(parents)
    for i in range(32):
        chain, a = [], i
        while a >= 0:
            chain.append(a)
            a = parents[a]
        assert depth[i] == len(chain) - 1
        assert anc[i] == sum(1 << c for c in chain)


def test_forward_rejects_bad_trees(tiny):
    m = O.OracleModel(TINY, tiny, max_ctx=32)
    with pytest.raises(ValueError):
        m.forward([1, 2], [-1, 1])           # parent not before child
    with pytest.raises(ValueError):
        m.forward([1, 2], [0, 0])            # root with a parent
    with pytest.raises(ValueError):
        m.forward([1, TINY.vocab], [-1, 0])  # token out of range
    with pytest.raises(ValueError):
        m.forward(list(range(40)), synth.chain_parents(40))  # beyond the cache
