"""End-to-end greedy decoding on one GPU: plain autoregressive decoding
against CAS-Spec with DyTC trees, through the library.

    python -m paper_2510_26843_amd.e2e --shape llama3_8b --prompt 4096 --new 256 --max-tree 64

The draft levels are the cascade of DSIA variants of the target: skip a
quarter of the layers (l % 4 == 3), skip every other layer, and skip every
other layer with per-token int8 activations.  Prompt lookup is the bottom
draft.  Their cost coefficients come from a Bayesian linear regression of
forward latency on roofline features, fitted to forwards timed at the
prompt's context before decoding (Sec. 4.2, "Hardware-Aware Latency
Prediction").  Acceptance estimates start from priors ordered by how many
layers a level skips (App. D, cold start) and follow the EMA of Sec. 4.2.
Weights are random N(0, 0.02^2), so acceptance rates say nothing about
trained models; the run reports what happens with these weights.

Timing covers the decoding loops only (the prompt is prefilled before the
clock starts).  The output line is one JSON object; the script also checks
that the two decodings produced the same tokens.
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from typing import Dict, List

import numpy as np

from . import cas, dytc, synth
from .latency import skip_mask


def calibrate(model, shape, ctx: int, levels: List[dytc.DraftConfig], log) -> Dict:
    """Time verify forwards and draft steps at context ctx, fit the latency
    model, and return the cost coefficients c-hat (R6 of dytc)."""
    L = shape.n_layers
    F, y, pts = [], [], []
    model.set_committed(ctx)

    def timed(tokens, parents, skip, aq, reps=6):
        for _ in range(2):
            model.forward(tokens, parents, 0, skip=skip, act_quant=aq, logits=False)
        model.sync()
        t0 = time.perf_counter()
        for _ in range(reps):
            model.forward(tokens, parents, 0, skip=skip, act_quant=aq, logits=False)
        model.sync()
        return (time.perf_counter() - t0) / reps * 1e3

    for n in (1, 4, 16, 32, 64):
        par = synth.balanced_tree(n)
        toks = synth.gen_tree_tokens(par, shape.vocab, seed=n)
        ms = timed(toks, par, None, False)
        F.append(dytc.roofline_features(shape, L, n, ctx))
        y.append(ms)
        pts.append(("verify", n, ms))
    for c in levels:
        run = len(c.run_layers(L))
        for n in (1, 2, 4, 8):
            par = synth.balanced_tree(n)
            toks = synth.gen_tree_tokens(par, shape.vocab, seed=n)
            ms = timed(toks, par, list(c.skip), c.act_quant)
            F.append(dytc.roofline_features(shape, run, n, ctx, c.act_quant))
            y.append(ms)
            pts.append((c.name, n, ms))
    model.set_committed(0)
    lm = dytc.LatencyModel(prior_precision=1e-3, noise_precision=1e2).fit(np.array(F), np.array(y))
    base = lm.predict(dytc.roofline_features(shape, L, 1, ctx))[0]
    cost = {c.name: lm.predict(dytc.roofline_features(shape, len(c.run_layers(L)), 1, ctx, c.act_quant))[0] / base
            for c in levels}
    resid = float(np.sqrt(np.mean((np.array(F) @ lm.mean - np.array(y)) ** 2)))
    log(f"[e2e] latency model: rms residual {resid:.3f} ms over {len(y)} points; c-hat {cost}")
    return {"cost": cost, "points": pts, "rms_residual_ms": resid, "target_ms": base}


class TimedBackend(dytc.LibraryBackend):
    """Starts the clock once the prompt is prefilled."""

    def reset(self, prompt):
        super().reset(prompt)
        self.m.sync()
        self.t0 = time.perf_counter()


def main(argv=None) -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--shape", default="llama3_8b")
    ap.add_argument("--prompt", type=int, default=4096)
    ap.add_argument("--new", type=int, default=256)
    ap.add_argument("--max-tree", type=int, default=64)
    ap.add_argument("--k-max", type=int, default=5)
    ap.add_argument("--top-k", type=int, default=4)
    ap.add_argument("--top-p", type=float, default=0.9)
    ap.add_argument("--t-min", type=float, default=1.1)
    ap.add_argument("--out", default="")
    args = ap.parse_args(argv)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    shape = synth.SHAPES[args.shape]
    L = shape.n_layers
    t0 = time.perf_counter()
    w = synth.gen_weights(shape, seed=0)
    m = cas.Model(shape, max_ctx=args.prompt + args.new + args.max_tree + 8, max_tree=max(64, args.max_tree))
    m.load_weights(w)
    m.build_int8()
    del w
    log(f"[e2e] {args.shape} loaded with its int8 copy in {time.perf_counter() - t0:.1f} s")
    prompt = [int(x) for x in synth.gen_prompt(shape.vocab, args.prompt, seed=1)]

    q3 = tuple(skip_mask(L, "q3"))
    odd = tuple(skip_mask(L, "odd"))
    levels = [dytc.DraftConfig("skip25", q3), dytc.DraftConfig("skip50", odd),
              dytc.DraftConfig("skip50_int8", odd, True)]
    pld = dytc.DraftConfig("pld", pld=True)
    m.prefill(prompt[:-1])
    cal = calibrate(m, shape, len(prompt) - 1, levels, log)
    cost = dict(cal["cost"])
    cost["pld"] = 0.01  # host-side lookup: negligible next to a forward (Sec. 3 takes c = 0.01)

    # plain greedy decoding
    m.set_committed(0)
    m.prefill(prompt[:-1])
    m.sync()
    t0 = time.perf_counter()
    ar, root = [], prompt[-1]
    while len(ar) < args.new:
        m.forward([root], [-1], 0, logits=False)
        acc, bonus = m.accept()
        m.compact(acc)
        ar.append(bonus)
        root = bonus
    m.sync()
    t_ar = time.perf_counter() - t0
    log(f"[e2e] greedy AR: {args.new} tokens in {t_ar:.3f} s")

    # CAS-Spec with DyTC
    est = dytc.AcceptanceEstimator({"skip25": 0.6, "skip50": 0.45, "skip50_int8": 0.4, "pld": 0.3})
    params = dytc.DytcParams(max_tree=args.max_tree, k_max=args.k_max, t_min=args.t_min, top_k=args.top_k,
                             top_p=args.top_p)
    be = TimedBackend(m)
    stats: Dict = {}
    out = dytc.cas_decode_dytc(be, prompt, args.new, levels + [pld], pld, est, cost, params, L, stats)
    m.sync()
    t_cas = time.perf_counter() - be.t0
    log(f"[e2e] CAS-Spec (DyTC): {args.new} tokens in {t_cas:.3f} s, {len(stats['accepted'])} rounds")
    first_diff = next((i for i, (a, b) in enumerate(zip(out, ar)) if a != b), None)
    res = {
        "shape": args.shape, "prompt": args.prompt, "new_tokens": args.new,
        "ar_tokens_per_s": round(args.new / t_ar, 2), "cas_tokens_per_s": round(args.new / t_cas, 2),
        "speedup_vs_ar": round(t_ar / t_cas, 4),
        "outputs_equal": first_diff is None, "first_difference": first_diff,
        "rounds": len(stats["accepted"]), "mean_accepted_per_round": round(float(np.mean(stats["accepted"])), 3),
        "mean_tree_size": round(float(np.mean(stats["tree_sizes"])), 2),
        "expansions": stats.get("expansions", {}), "alpha_final": {k: round(v, 4) for k, v in est.a.items()},
        "c_hat": {k: round(v, 4) for k, v in cost.items()}, "latency_model_rms_ms": round(cal["rms_residual_ms"], 4),
        "params": vars(params),
        "data": "synthetic: random N(0,0.02^2) bf16 weights, uniform-random prompt",
    }
    m.close()
    line = json.dumps(res)
    if args.out:
        with open(args.out, "w") as f:
            f.write(line + "\n")
    print(line)


if __name__ == "__main__":
    main()
