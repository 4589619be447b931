"""End-to-end greedy decoding on one GPU: plain autoregressive decoding
against CAS-Spec with DyTC trees, through the library.

    python -m paper_2510_26843_amd.e2e --shape llama3_8b --prompt 4096 --new 256 --max-tree 64

The draft levels are the cascade of DSIA variants of the target: skip a
quarter of the layers (l % 4 == 3), skip every other layer, and skip every
other layer with per-token int8 (W8A8) or int4 (W4A4) activations.  Prompt
lookup is the bottom draft.  Their cost coefficients come from a Bayesian linear regression of
forward latency on roofline features, fitted to forwards timed at the
prompt's context before decoding (Sec. 4.2, "Hardware-Aware Latency
Prediction").  Acceptance estimates start from priors ordered by how many
layers a level skips (App. D, cold start) and follow the EMA of Sec. 4.2.
Weights are random N(0, 0.02^2), so acceptance rates say nothing about
trained models; the run reports what happens with these weights.  With
--damp-odd e the output projections (W_o, W_down) of the odd layers are
scaled by e: a synthetic model whose odd layers barely move the residual
stream, the layer redundancy that layer-skip drafting relies on in trained
models.  With e = 0 the odd layers add exactly zero, so the skip-50% draft
computes the target's own logits: its acceptance is 1 and the run measures
the ceiling of the mechanism (draft cost, tree verify, acceptance) on the
hardware.  --prior sets the cold-start acceptance estimates (App. D).

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


def divergence_report(m, prompt: List[int], ar: List[int], levels, pld, prior, cost, params, L, log) -> Dict:
    """Tie analysis of CAS against AR (untimed): decode with CAS from the
    prompt; at the first token that differs from AR, record the top-1/top-2
    margin of AR's own logits at that position (absolute, and relative to the
    row's largest |logit|), then continue from the AR sequence up to and
    including that token.  A divergence at a margin of the order of fp32
    rounding of the attention sums is a near-tie, not a wrong acceptance."""
    out, divs = [], []
    n_new = len(ar)
    while len(out) < n_new:
        est = dytc.AcceptanceEstimator(dict(prior))
        seg = dytc.cas_decode_dytc(dytc.LibraryBackend(m), prompt + out, n_new - len(out), levels + [pld], pld, est,
                                   cost, params, L, {})
        i = next((k for k, (a, b) in enumerate(zip(seg, ar[len(out):])) if a != b), None)
        if i is None:
            break
        pos = len(out) + i
        seq = prompt + ar[:pos]
        m.set_committed(0)
        m.prefill(seq[:-1])
        lg = m.forward([seq[-1]], [-1], 0)[0].astype(np.float64)
        top = np.sort(lg)[-2:]
        divs.append({"token": pos, "margin": float(top[1] - top[0]), "rel_margin": float((top[1] - top[0]) / np.abs(lg).max())})
        log(f"[e2e] divergence at token {pos}: AR top-1/top-2 margin {divs[-1]['margin']:.3e} "
            f"({divs[-1]['rel_margin']:.2e} of max |logit|)")
        out = ar[:pos + 1]
    return {"divergences": divs, "max_rel_margin": max((d["rel_margin"] for d in divs), default=0.0)}


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
    ap.add_argument("--prior", default="skip25=0.6,skip50=0.45,skip50_int8=0.4,skip50_int4=0.3,pld=0.3",
                    help="cold-start acceptance estimates, name=value pairs")
    ap.add_argument("--ties", action="store_true",
                    help="after timing, locate every CAS/AR divergence and report AR's logit margin there")
    ap.add_argument("--damp-odd", type=float, default=None,
                    help="scale the odd layers' W_o and W_down by this factor (unset: unchanged)")
    ap.add_argument("--gemv", type=int, choices=(0, 1), default=None,
                    help="GEMV-style tiles for one-row drafts (default: the library's)")
    ap.add_argument("--out", default="")
    args = ap.parse_args(argv)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    shape = synth.SHAPES[args.shape]
    L = shape.n_layers
    t0 = time.perf_counter()
    w = synth.gen_weights(shape, seed=0)
    if args.damp_odd is not None:
        e = np.float32(args.damp_odd)
        for l in range(1, L, 2):
            for n in ("wo", "w_down"):
                a = w["layers"][l][n]
                w["layers"][l][n] = synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(a) * e) if a.dtype == np.uint16 \
                    else (a * e).astype(np.float32)
    m = cas.Model(shape, max_ctx=args.prompt + args.new + args.max_tree + 8, max_tree=max(64, args.max_tree))
    m.load_weights(w)
    m.build_int8()
    m.build_int4()
    if args.gemv is not None:
        m.set_gemv(bool(args.gemv))
    del w
    log(f"[e2e] {args.shape} loaded with its int8 and int4 copies in {time.perf_counter() - t0:.1f} s")
    prompt = [int(x) for x in synth.gen_prompt(shape.vocab, args.prompt, seed=1)]

    q3 = tuple(skip_mask(L, "q3"))
    odd = tuple(skip_mask(L, "odd"))
    levels = [dytc.DraftConfig("skip25", q3), dytc.DraftConfig("skip50", odd),
              dytc.DraftConfig("skip50_int8", odd, 1), dytc.DraftConfig("skip50_int4", odd, 2)]
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
    prior = {k: float(v) for k, v in (kv.split("=") for kv in args.prior.split(","))}
    est = dytc.AcceptanceEstimator(prior)
    params = dytc.DytcParams(max_tree=args.max_tree, k_max=args.k_max, t_min=args.t_min, top_k=args.top_k,
                             top_p=args.top_p)
    be = TimedBackend(m)
    stats: Dict = {}
    out = dytc.cas_decode_dytc(be, prompt, args.new, levels + [pld], pld, est, cost, params, L, stats)
    m.sync()
    t_cas = time.perf_counter() - be.t0
    log(f"[e2e] CAS-Spec (DyTC): {args.new} tokens in {t_cas:.3f} s, {len(stats['accepted'])} rounds")
    first_diff = next((i for i, (a, b) in enumerate(zip(out, ar)) if a != b), None)
    ties = divergence_report(m, prompt, ar, levels, pld, prior, cost, params, L, log) if args.ties else None
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
        "damp_odd": args.damp_odd, "gemv": args.gemv, "prior": prior, "ties": ties,
        "data": ("synthetic: random N(0,0.02^2) bf16 weights" +
                 (f", odd layers' W_o and W_down scaled by {args.damp_odd}" if args.damp_odd is not None else "") +
                 ", uniform-random prompt"),
    }
    m.close()
    line = json.dumps(res)
    if args.out:
        with open(args.out, "w") as f:
            f.write(line + "\n")
    print(line)


if __name__ == "__main__":
    main()
