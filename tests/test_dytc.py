"""DyTC host scheduler pinned against the paper and brute force (CPU).

- The EWIF formulas against explicit enumeration of Bernoulli acceptance
  outcomes, and against the paper's worked example (tests/golden).
- FindBestConfigurationForStep against an exhaustive search.
- The acceptance EMA against a hand-computed sequence; prompt lookup on
  constructed sequences; the Bayesian linear regression against least
  squares.
- Tree construction invariants with a scripted backend.
- End to end on the oracle: DyTC speculative decoding equals greedy
  autoregressive decoding token for token (lossless, Sec. 5.1).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2510_26843_amd import dytc, synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "dytc_worked_example.json")


# ---------------------------------------------------------------- EWIF by enumeration

def _enum_sd(alpha, c, k):
    """E[tokens per verify] / cost by enumerating which of the k drafted
    tokens are accepted (i.i.d. Bernoulli, the run stops at the first miss);
    the verify always yields one more token."""
    e = 0.0
    for bits in itertools.product([0, 1], repeat=k):
        p = 1.0
        for b in bits:
            p *= alpha if b else 1 - alpha
        run = 0
        for b in bits:
            if not b:
                break
            run += 1
        e += p * (run + 1)
    return e / (1 + c * k)


def _enum_hc(a1, c1, k1, a2, c2, k2):
    e = 0.0
    for bits in itertools.product([0, 1], repeat=k1 + k2):
        p = 1.0
        for i, b in enumerate(bits):
            a = a1 if i < k1 else a2
            p *= a if b else 1 - a
        run = 0
        for b in bits:
            if not b:
                break
            run += 1
        e += p * (run + 1)
    return e / (1 + k1 * c1 + k2 * c2)


@pytest.mark.parametrize("alpha,c,k", [(0.8, 0.3, 3), (0.5, 0.1, 1), (0.95, 0.05, 6), (0.2, 0.6, 4)])
def test_ewif_sd_matches_enumeration(alpha, c, k):
    assert dytc.ewif_sd(alpha, c, k) == pytest.approx(_enum_sd(alpha, c, k), rel=1e-12)


@pytest.mark.parametrize("args", [(0.9, 0.4, 2, 0.8, 0.3, 2), (0.7, 0.2, 1, 0.4, 0.01, 5), (0.6, 0.3, 3, 0.9, 0.1, 2)])
def test_ewif_hc_matches_enumeration(args):
    assert dytc.ewif_hc(*args) == pytest.approx(_enum_hc(*args), rel=1e-12)


def test_step_objective_by_enumeration():
    """T_s counts the expected accepted tokens of k draft steps plus, when all
    k are accepted, one bottom-draft token accepted with alpha_n."""
    for a, c, k, an, cn in [(0.8, 0.3, 3, 0.4, 0.01), (0.6, 0.2, 1, 0.3, 0.05), (1.0, 0.5, 4, 0.2, 0.1)]:
        e = 0.0
        for bits in itertools.product([0, 1], repeat=k + 1):
            p = 1.0
            for i, b in enumerate(bits):
                q = a if i < k else an
                p *= q if b else 1 - q
            run = 0
            for b in bits:
                if not b:
                    break
                run += 1
            e += p * run
        assert dytc.step_objective(a, c, k, an, cn) == pytest.approx(e / (c * k + cn), rel=1e-12)


def test_worked_example_from_the_paper():
    g = json.load(open(GOLDEN))
    d1, d2 = g["d1"], g["d2"]
    # local speedups of one draft step (k_s = 1, no accumulated factor)
    for name, d in (("d1", d1), ("d2", d2)):
        t = dytc.expected_accepted(d["alpha"], 1) / (d["c"] * 1)
        assert round(t, 2) == g["local_speedup_k1"][name]
    greedy = max(dytc.ewif_sd(d2["alpha"], d2["c"], k) for k in range(1, 20))
    hc = max(dytc.ewif_hc(d1["alpha"], d1["c"], k1, d2["alpha"], d2["c"], k2)
             for k1 in range(1, 12) for k2 in range(1, 12))
    assert round(greedy, g["printed_decimals"]) == g["greedy_ewif"]
    assert round(hc, g["printed_decimals"]) == g["hc_ewif"]
    assert hc > greedy


# ---------------------------------------------------------------- Alg. 2

def test_find_best_config_is_the_argmax():
    rng = np.random.default_rng(0)
    for trial in range(50):
        cands = {f"s{i}": (float(rng.uniform(0.05, 0.99)), float(rng.uniform(0.01, 0.8))) for i in range(4)}
        an, cn, kmax = float(rng.uniform(0.05, 0.9)), float(rng.uniform(0.005, 0.1)), int(rng.integers(1, 8))
        best = max(((dytc.step_objective(a, c, k, an, cn), -i, -k, name, k)
                    for i, (name, (a, c)) in enumerate(cands.items()) for k in range(1, kmax + 1)))
        assert dytc.find_best_config(cands, an, cn, kmax) == (best[3], best[4])


def test_find_best_config_none_when_nothing_pays():
    assert dytc.find_best_config({"a": (0.0, 0.5)}, 0.0, 0.01, 5) == (None, 0)
    assert dytc.find_best_config({}, 0.5, 0.01, 5) == (None, 0)
    # alpha = 1 uses E[accepted] = k
    assert dytc.expected_accepted(1.0, 4) == 4.0


# ---------------------------------------------------------------- estimates, PLD, BLR

def test_acceptance_estimator_ema_by_hand():
    est = dytc.AcceptanceEstimator({"a": 0.5, "b": 0.2}, H=3, lam=0.7)
    seq = [1, 0, 1, 1, 1]
    want = 0.5
    window = []
    for o in seq:
        est.record("a", bool(o))
        est.end_step()
        window = (window + [o])[-3:]
        want = 0.7 * want + 0.3 * (sum(window) / len(window))
        assert est.alpha("a") == pytest.approx(want, abs=1e-15)
    assert est.alpha("b") == 0.2  # not drafting: no decay


def test_pld_propose():
    seq = [5, 6, 7, 8, 1, 2, 5, 6, 7]
    assert dytc.pld_propose(seq, 3) == ([8, 1, 2], 3)
    assert dytc.pld_propose(seq, 1) == ([8], 3)
    # the most recent earlier occurrence wins
    assert dytc.pld_propose([1, 2, 9, 1, 2, 4, 1, 2], 2, n_max=2) == ([4, 1], 2)
    # falls back to shorter n-grams, then nothing
    assert dytc.pld_propose([3, 4, 5, 9, 4], 2) == ([5, 9], 1)
    assert dytc.pld_propose([1, 2, 3], 2) == ([], 0)


def test_latency_model_recovers_linear_law():
    rng = np.random.default_rng(1)
    F = np.column_stack([np.ones(30), rng.uniform(1, 30, 30), rng.uniform(0, 3, 30), rng.uniform(0, 2, 30),
                         rng.integers(8, 41, 30)])
    w = np.array([0.05, 0.17, 0.15, 0.6, 0.004])
    y = F @ w
    m = dytc.LatencyModel(prior_precision=1e-8, noise_precision=1e6).fit(F, y)
    ls = np.linalg.lstsq(F, y, rcond=None)[0]
    assert np.allclose(m.mean, ls, rtol=1e-5, atol=1e-7)
    f = np.array([1.0, 13.5, 0.5, 0.9, 32.0])
    mu, var = m.predict(f)
    assert mu == pytest.approx(float(f @ w), rel=1e-6)
    # a strong prior shrinks the weights toward zero
    m0 = dytc.LatencyModel(prior_precision=1e9, noise_precision=1.0).fit(F, y)
    assert np.abs(m0.mean).max() < 1e-3
    # more data, less predictive variance
    v_small = dytc.LatencyModel(1e-2, 1e2).fit(F[:6], y[:6]).predict(f)[1]
    v_big = dytc.LatencyModel(1e-2, 1e2).fit(F, y).predict(f)[1]
    assert v_big < v_small


def test_roofline_features_match_latency_byte_model():
    from paper_2510_26843_amd import latency
    shape = synth.SHAPES["llama2_7b"]
    f = dytc.roofline_features(shape, 32, 1, 1024)
    b = latency.algorithmic_bytes(shape, 1, 1024, 32)
    # weights + head + KV reads of ctx + the new row: the byte model less its KV write, embedding row and logits
    extra = 32 * 2 * shape.n_kv_heads * shape.head_dim * 2 * 1 + shape.d_model * 2 + shape.vocab * 4
    assert (f[1] + f[2]) * 1e9 == pytest.approx(b - extra, rel=1e-12)


# ---------------------------------------------------------------- tree construction

class ScriptedBackend:
    """Draft calls return deterministic pseudo-random candidates per fed
    (node id, token); checks the library's feeding rules on every call."""

    def __init__(self, vocab=50, K=4):
        self.vocab, self.calls, self.n_fed = vocab, [], 0

    def reset(self, prompt):
        self.n_fed = 0

    def draft(self, tokens, parents, node_offset, cfg, K):
        assert node_offset == (0 if node_offset == 0 else self.n_fed)
        if node_offset == 0:
            assert parents[0] == -1 and self.n_fed == 0
        for i, p in enumerate(parents):
            assert p < node_offset + i
        self.n_fed = node_offset + len(tokens)
        self.calls.append((list(tokens), list(parents), node_offset, cfg.name))
        ids = np.zeros((len(tokens), K), dtype=np.int32)
        pr = np.zeros((len(tokens), K), dtype=np.float32)
        for r, t in enumerate(tokens):
            g = np.random.default_rng(t * 131 + node_offset + r)
            ids[r] = g.choice(self.vocab, K, replace=False)
            p = np.sort(g.dirichlet(np.ones(K) * 0.5))[::-1]
            pr[r] = p * 0.9
        return ids, pr


def _configs(n_layers=8):
    q3 = tuple(1 if l % 4 == 3 else 0 for l in range(n_layers))
    odd = tuple(l % 2 for l in range(n_layers))
    return [dytc.DraftConfig("q3", q3), dytc.DraftConfig("odd", odd), dytc.DraftConfig("odd_i8", odd, True),
            dytc.DraftConfig("pld", pld=True)]


def test_build_tree_invariants():
    cfgs = _configs()
    pld = cfgs[-1]
    est = dytc.AcceptanceEstimator({"q3": 0.7, "odd": 0.5, "odd_i8": 0.45, "pld": 0.3})
    cost = {"q3": 0.75, "odd": 0.5, "odd_i8": 0.42, "pld": 0.01}
    for M in (8, 17, 64):
        be = ScriptedBackend()
        params = dytc.DytcParams(max_tree=M, k_max=4, t_min=1.1, top_k=4, top_p=0.9)
        ctx = [1, 2, 3, 1, 2]
        tree = dytc.build_tree(be, 3, ctx, cfgs, pld, est, cost, params, 8, stats={})
        assert 1 <= len(tree) <= M
        order = tree.ordering()
        assert sorted(order) == list(range(len(tree)))
        rid = {n: j for j, n in enumerate(order)}
        for i, n in enumerate(tree.nodes):
            if n.parent >= 0:
                assert rid[n.parent] < rid[i]
                assert n.p_acc <= tree.nodes[n.parent].p_acc + 1e-12
            if n.fed_id >= 0:
                assert order[n.fed_id] == i
                # R4: the draft that fed it reads only KV its ancestors have
                for a in tree.path(i)[:-1]:
                    assert tree.nodes[a].fed_id >= 0 and n.run <= tree.nodes[a].run
            if n.pld_made:
                assert n.fed_id < 0 and all(tree.nodes[c].pld_made for c in n.children)
        assert [c[2] for c in be.calls] == sorted(c[2] for c in be.calls)


def test_build_tree_prefers_the_cheap_bottom_when_drafts_are_poor():
    cfgs = _configs()
    est = dytc.AcceptanceEstimator({"q3": 0.05, "odd": 0.05, "odd_i8": 0.05, "pld": 0.6})
    cost = {"q3": 0.75, "odd": 0.5, "odd_i8": 0.42, "pld": 0.01}
    be = ScriptedBackend()
    st = {}
    tree = dytc.build_tree(be, 2, [7, 2, 9, 4, 7], cfgs, cfgs[-1], est, cost, dytc.DytcParams(max_tree=16), 8, st)
    assert be.calls == [] and set(st["expansions"]) == {"pld"}
    # prompt lookup keeps following the repeating context as one chain
    assert [n.token for n in tree.nodes] == ([2, 9, 4, 7] * 8)[: len(tree)]
    assert [n.parent for n in tree.nodes] == list(range(-1, len(tree) - 1))


# ---------------------------------------------------------------- end to end on the oracle

class OracleBackend:
    """The oracle behind the calls DyTC makes (top-K from fp64 logits with
    ties to the lower id, probabilities from an fp64 softmax)."""

    def __init__(self, model):
        self.m = model

    def reset(self, prompt):
        self.m.set_committed(0)
        if len(prompt) > 1:
            self.m.prefill(list(prompt[:-1]))

    def draft(self, tokens, parents, node_offset, cfg, K):
        lg = self.m.forward(tokens, parents, node_offset, skip=list(cfg.skip) if cfg.skip else None,
                            act_quant=cfg.act_quant, attn_window=cfg.window)
        ids = np.stack([np.argsort(-r, kind="stable")[:K] for r in lg]).astype(np.int32)
        e = np.exp(lg - lg.max(axis=1, keepdims=True))
        p = e / e.sum(axis=1, keepdims=True)
        return ids, np.take_along_axis(p, ids, axis=1)

    def verify(self, tokens, parents):
        lg = self.m.forward(tokens, parents, 0)
        return O.accept_greedy(lg, parents, tokens)

    def commit(self, path):
        self.m.compact(path)


@pytest.mark.parametrize("name", ["tiny", "gqa"])
def test_dytc_decoding_is_lossless_on_the_oracle(name):
    if name == "tiny":
        shape = synth.SHAPES["tiny"]
        n_new, plen = 24, 48
    else:
        shape = synth.ModelShape("gqa_small", 4, 256, 4, 2, 64, 688, 512, 5e5, 1e-6, "bf16")
        n_new, plen = 16, 40
    w = synth.gen_weights(shape, seed=0)
    # a prompt with repeats, so prompt lookup finds matches
    base = [int(x) for x in synth.gen_prompt(shape.vocab, plen // 2, seed=1)]
    prompt = base + base
    ref = O.ar_decode(O.OracleModel(shape, w, max_ctx=256), prompt, n_new)
    L = shape.n_layers
    q3 = tuple(1 if l % 4 == 3 else 0 for l in range(L))
    odd = tuple(l % 2 for l in range(L))
    cfgs = [dytc.DraftConfig("q3", q3), dytc.DraftConfig("odd", odd), dytc.DraftConfig("odd_i8", odd, True),
            dytc.DraftConfig("pld", pld=True)]
    # priors under which the neural levels win the first rounds (with a
    # near-free bottom draft the step objective otherwise prefers prompt lookup)
    est = dytc.AcceptanceEstimator({"q3": 0.9, "odd": 0.8, "odd_i8": 0.75, "pld": 0.05})
    cost = {"q3": 0.3, "odd": 0.2, "odd_i8": 0.18, "pld": 0.01}
    params = dytc.DytcParams(max_tree=24, k_max=3, t_min=1.1, top_k=3, top_p=0.5)
    st = {}
    got = dytc.cas_decode_dytc(OracleBackend(O.OracleModel(shape, w, max_ctx=256, int8=True)), prompt, n_new,
                               cfgs, cfgs[-1], est, cost, params, L, st)
    assert got == ref
    assert sum(st["expansions"].get(c, 0) for c in ("q3", "odd", "odd_i8")) > 0
    assert max(st["tree_sizes"]) <= params.max_tree
