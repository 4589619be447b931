"""Latency table of the decoder step on one GPU.

Times the library's forward (HIP graphs replayed, inputs resident) over
token trees of several sizes T and committed context lengths, at full depth
(the verify pass) and for draft configurations (a layer-skip set, optionally
with per-token int8 activations).  Each point carries the forward's
algorithmic HBM bytes and FLOPs, so the table reads directly as achieved
bandwidth and MFMA use.  The table is what a DyTC-style cost predictor is
fitted on (Sec. 4.2: the cost coefficient of a draft configuration is
predicted from the platform's roofline latency).

    python -m paper_2510_26843_amd.latency --shape llama2_7b --T 1,8,16,32,64,128 \\
        --ctx 512,2048,8192 --out table.json

KV contents do not change the timing of any kernel, so the committed length
is set directly instead of prefilling.
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys
import time
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

HBM_PEAK_GBPS = 8000.0      # MI355X HBM3E
MFMA_PEAK_TFLOPS = 2500.0   # MI355X dense bf16


def skip_mask(n_layers: int, rule: str) -> Optional[List[int]]:
    """Layer-skip sets of the draft levels: 'none'; 'odd' (every other
    layer, layer 0 always runs: 50%); 'q3' (l % 4 == 3: 25%); or an explicit
    comma-separated list of layer indices."""
    if rule in ("none", ""):
        return None
    if rule == "odd":
        return [l % 2 for l in range(n_layers)]
    if rule == "q3":
        return [1 if l % 4 == 3 else 0 for l in range(n_layers)]
    ids = {int(x) for x in rule.split(",")}
    return [1 if l in ids else 0 for l in range(n_layers)]


def parse_draft(spec: str, n_layers: int):
    """A draft configuration from '<skip rule>[+int8|+int4][@sink:window]'
    -> (skip mask, act_quant 0/1/2, window)."""
    window = None
    if "@" in spec:
        spec, w = spec.split("@")
        sink, win = w.split(":")
        window = (int(sink), int(win))
    aq = 1 if spec.endswith("+int8") else 2 if spec.endswith("+int4") else 0
    return skip_mask(n_layers, spec.split("+")[0]), aq, window


def algorithmic_bytes(shape, T: int, Lc: int, run_layers: int, int8: int = 0,
                      window: Optional[Tuple[int, int]] = None) -> int:
    """Bytes one forward must move: the weights of the layers that run (bf16
    or fp32; int8 = 1: int8 codes, 2: 4-bit codes, plus fp32 per-channel
    scales) and the LM head once, the KV reads of all visible slots (only
    the sink and the window of the committed ones under a window) and the
    writes of the new ones, the embedding rows and the fp32 logits."""
    if window and window[1] > 0:
        Lc = min(Lc, window[0] + window[1])
    es = 2 if shape.dtype == "bf16" else 4
    kv_row = shape.n_kv_heads * shape.head_dim * es
    if int8:
        d, q, kv, f = shape.d_model, shape.n_heads * shape.head_dim, shape.n_kv_heads * shape.head_dim, shape.ffn_dim
        rows = (q + 2 * kv) + d + 2 * f + d
        b = run_layers * (shape.layer_params() // (2 if int(int8) == 2 else 1) + 4 * rows)
    else:
        b = run_layers * shape.layer_params() * es
    b += shape.vocab * shape.d_model * es
    b += run_layers * 2 * kv_row * (Lc + T)
    b += run_layers * 2 * kv_row * T
    b += T * shape.d_model * es + T * shape.vocab * 4
    return b


def algorithmic_flops(shape, T: int, Lc: int, run_layers: int, mean_depth: float) -> float:
    """2 T (parameters of the run layers + LM head) plus the attention's QK^T
    and PV over the visible keys (Lc + ancestors-or-self of each row)."""
    f = 2.0 * T * (run_layers * shape.layer_params() + shape.vocab * shape.d_model)
    f += run_layers * 4.0 * T * (Lc + mean_depth + 1) * shape.n_heads * shape.head_dim
    return f


def tree_for(T: int) -> List[int]:
    """The balanced tree of T nodes (the n-node cut of a full binary tree)."""
    from .synth import balanced_tree
    return balanced_tree(T)


def time_forward(model, toks, parents, skip, aq: bool, reps: int, warmup: int = 3,
                 window: Optional[Tuple[int, int]] = None) -> Dict[str, float]:
    """Wall time per forward over `reps` back-to-back calls (logits stay on
    the device), median of three such batches."""
    for _ in range(warmup):
        model.forward(toks, parents, 0, skip=skip, act_quant=aq, logits=False, attn_window=window)
    model.sync()
    runs = []
    for _ in range(3):
        t0 = time.perf_counter()
        for _ in range(reps):
            model.forward(toks, parents, 0, skip=skip, act_quant=aq, logits=False, attn_window=window)
        model.sync()
        runs.append((time.perf_counter() - t0) / reps * 1e3)
    return {"ms": statistics.median(runs), "ms_min": min(runs), "ms_max": max(runs)}


def sweep(model, shape, Ts: Sequence[int], ctxs: Sequence[int], drafts: Sequence[str], reps: int = 20,
          log=None) -> List[Dict]:
    """One record per (configuration, T, ctx): 'verify' at full depth for
    every T, and each draft configuration ('<rule>', '<rule>+int8', '<rule>+int4') for
    every T as well (tree-parallel drafting runs drafts over several rows)."""
    from .synth import gen_tree_tokens
    out = []
    configs = [("verify", None, 0, None)] + [(d,) + parse_draft(d, shape.n_layers) for d in drafts]
    for ctx in ctxs:
        for T in Ts:
            parents = tree_for(T)
            toks = gen_tree_tokens(parents, shape.vocab, seed=ctx + T)
            depth = [0] * T
            for i, p in enumerate(parents):
                depth[i] = 0 if p < 0 else depth[p] + 1
            for name, skip, aq, window in configs:
                model.set_committed(ctx)
                run = shape.n_layers - (sum(skip) if skip else 0)
                r = time_forward(model, toks, parents, skip, aq, reps, window=window)
                b = algorithmic_bytes(shape, T, ctx, run, int8=aq, window=window)
                ctx_vis = min(ctx, window[0] + window[1]) if window and window[1] > 0 else ctx
                fl = algorithmic_flops(shape, T, ctx_vis, run, float(np.mean(depth)))
                rec = {"config": name, "T": T, "ctx": ctx, "run_layers": run, "act_quant": aq,
                       "ms": round(r["ms"], 4), "ms_min": round(r["ms_min"], 4), "ms_max": round(r["ms_max"], 4),
                       "tokens_per_s": round(T / (r["ms"] * 1e-3), 1), "bytes": b,
                       "hbm_gbps": round(b / (r["ms"] * 1e-3) / 1e9, 1),
                       "hbm_frac": round(b / (r["ms"] * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                       "mfma_frac": round(fl / (r["ms"] * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS, 4)}
                out.append(rec)
                if log:
                    log(f"[latency] {name:>10} T {T:4d} ctx {ctx:5d}: {rec['ms']:.3f} ms, "
                        f"{rec['hbm_gbps']:.0f} GB/s ({rec['hbm_frac']:.1%}), MFMA {rec['mfma_frac']:.1%}")
    model.set_committed(0)
    return out


def markdown(records: List[Dict]) -> str:
    lines = ["| config | T | ctx | layers run | ms | tokens/s | algorithmic GB | GB/s | of 8 TB/s | MFMA of 2.5 PF |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for r in records:
        lines.append(f"| {r['config']} | {r['T']} | {r['ctx']} | {r['run_layers']} | {r['ms']:.3f} | "
                     f"{r['tokens_per_s']:.0f} | {r['bytes'] / 1e9:.3f} | {r['hbm_gbps']:.0f} | "
                     f"{r['hbm_frac']:.1%} | {r['mfma_frac']:.1%} |")
    return "\n".join(lines)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--shape", default="llama2_7b")
    ap.add_argument("--T", default="1,8,16,32,64,128")
    ap.add_argument("--ctx", default="512,2048,8192")
    ap.add_argument("--drafts", default="",
                    help="draft configurations separated by ';', e.g. 'odd;q3;odd+int8;odd+int4;odd@4:1024' "
                         "(skip rule, +int8 or +int4 activations, @sink:window attention)")
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--out", default="")
    ap.add_argument("--md", default="")
    args = ap.parse_args(argv)
    from . import cas, synth
    shape = synth.SHAPES[args.shape]
    Ts = [int(x) for x in args.T.split(",")]
    ctxs = [int(x) for x in args.ctx.split(",")]
    drafts = [d for d in args.drafts.split(";") if d]
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    w = synth.gen_weights(shape, seed=0)
    m = cas.Model(shape, max_ctx=max(ctxs) + max(Ts), max_tree=max(128, max(Ts)), device=0)
    m.load_weights(w)
    if any(d.split("@")[0].endswith("+int8") for d in drafts):
        m.build_int8()
    if any(d.split("@")[0].endswith("+int4") for d in drafts):
        m.build_int4()
    del w
    log(f"[latency] {args.shape} ready in {time.perf_counter() - t0:.1f} s")
    recs = sweep(m, shape, Ts, ctxs, drafts, args.reps, log)
    m.close()
    res = {"shape": args.shape, "records": recs}
    if args.out:
        with open(args.out, "w") as f:
            json.dump(res, f, indent=1)
    if args.md:
        with open(args.md, "w") as f:
            f.write(markdown(recs) + "\n")
    print(json.dumps({"shape": args.shape, "points": len(recs)}))


if __name__ == "__main__":
    main()
