"""Benchmark of the CAS-Spec tree-verify hot path on one MI355X.

Workload (Llama-2-7B-shaped decoder, bf16, random N(0, 0.02^2) weights, batch
1): the KV cache is prefilled from a 1024-token uniform-random prompt; one
step is
  - one draft forward of the root skipping every other layer (16 of 32),
  - one verify forward over a fixed 32-node token tree (branching 4,2,2,1,1,
    depth 5) at full depth,
  - greedy acceptance of the tree and the KV commit of the accepted path,
  - a rollback of the committed length to 1024 so every step is identical.
value = verified tree tokens per second over the whole step (32 per step).

Per-kernel durations come from HIP events recorded on the library's own
stream (cas_profile); the dominant kernel's achieved HBM rate is its
algorithmic bytes per launch over its mean duration.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
KERNELS_SRC = os.path.join(ROOT, "paper_2510_26843_amd", "csrc", "kernels.hip")
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "gemm_gateup_7b_t32_traffic.json")


def kernels_sha256():
    with open(KERNELS_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per gate/up launch from the stored rocprofv3 counter record,
    or None when the record is missing or the kernel source has changed since
    the counters were taken."""
    try:
        with open(TRAFFIC_RECORD) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernels_sha256") != kernels_sha256():
        return None
    return rec.get("hbm_bytes_per_launch")


def gemm_bytes(N, K, T, out_bytes):
    return N * K * 2 + T * K * 2 + out_bytes


def cpu_baseline(shape, weights, parents, toks, Lc, min_s=10.0, max_reps=3):
    """The oracle's verify forward on the host cores: whole 32-layer forwards
    of the same tree over a synthetic 1024-slot committed KV cache, repeated
    until at least min_s seconds of work (at most max_reps forwards)."""
    from oracle import oracle as O
    from paper_2510_26843_amd import synth
    O.set_threads(min(16, os.cpu_count() or 1))
    om = O.OracleModel(shape, weights, max_ctx=Lc + len(parents))
    k, v = synth.gen_kv(shape.n_layers, shape.n_kv_heads, Lc, shape.head_dim, seed=4)
    for l in range(shape.n_layers):
        om.set_kv(l, synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(k[l])),
                  synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(v[l])))
    del k, v
    om.set_committed(Lc)
    reps, t = 0, 0.0
    while reps < max_reps and (reps == 0 or t < min_s):
        t0 = time.perf_counter()
        om.forward(toks, parents, 0)
        t += time.perf_counter() - t0
        reps += 1
    return {"value": round(len(parents) * reps / t, 3), "unit": "tree tokens/s", "cores": O.threads(),
            "host_cpus": os.cpu_count(), "kind": "oracle",
            "sample": (f"{reps} fp64 oracle verify forward(s) of the full {shape.n_layers}-layer model, "
                       f"T={len(parents)} tree (4,2,2,1,1), over a synthetic {Lc}-slot KV cache: {t:.1f} s")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layers", type=int, default=0, help="(testing only) fewer layers; invalidates the metric")
    ap.add_argument("--counter-pass", action="store_true",
                    help="profiling pass for hardware counters: verify steps only, direct launches (no graphs), "
                         "then a copy of --copy-mib MiB; prints no metric")
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--counter-T", type=int, default=32,
                    help="counter pass only: verify tree size (32: the benchmark's tree; else a balanced tree)")
    ap.add_argument("--counter-ctx", type=int, default=0, help="counter pass only: committed length (0: 1024)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus above 1 is not supported",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    from paper_2510_26843_amd import cas, synth
    from paper_2510_26843_amd.latency import algorithmic_bytes

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    shape = synth.SHAPES["llama2_7b"]
    if args.layers:
        shape = shape.with_layers(args.layers)
    Lc = 1024
    T = 32
    log = lambda *a: print(*a, file=sys.stderr, flush=True)

    t0 = time.perf_counter()
    weights = synth.gen_weights(shape, seed=0)
    log(f"[bench] weights generated in {time.perf_counter() - t0:.1f} s")
    # the library enqueues on this stream, so per-call events can bracket its graph replays
    stream = torch.cuda.Stream(device=0)
    m = cas.Model(shape, max_ctx=Lc + 128, max_tree=128, device=0, stream=stream.cuda_stream)
    t0 = time.perf_counter()
    m.load_weights(weights)
    log(f"[bench] weights uploaded in {time.perf_counter() - t0:.1f} s")
    prompt = synth.gen_prompt(shape.vocab, Lc, seed=1)
    t0 = time.perf_counter()
    m.prefill(prompt)
    m.sync()
    log(f"[bench] prefill of {Lc} tokens in {time.perf_counter() - t0:.2f} s")
    parents = synth.tree_from_branching(*synth.TREE_7B)
    toks = synth.gen_tree_tokens(parents, shape.vocab, seed=2)
    odd = [l % 2 for l in range(shape.n_layers)]

    if args.counter_pass:
        m.set_graphs(False)
        cp, ct, cL = parents, toks, Lc
        if args.counter_T != T:
            cp = synth.balanced_tree(args.counter_T)
            ct = synth.gen_tree_tokens(cp, shape.vocab, seed=2)
        if args.counter_ctx:
            cL = args.counter_ctx
        m.set_committed(cL)
        for _ in range(args.warmup + args.steps):
            m.forward(ct, cp, 0, logits=False)
            acc, _ = m.accept()
            m.compact(acc)
            m.set_committed(cL)
        m.sync()
        m.close()
        del m
        nbytes = args.copy_mib << 20
        src = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda:0").random_()
        dst = torch.empty_like(src)
        for _ in range(3):
            cas.op_copy(dst, src, nbytes)
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
        log(f"[bench] counter pass: {args.warmup + args.steps} verify steps (T={len(cp)}, ctx {cL}), "
            f"3 copies of {nbytes} bytes")
        return

    def step():
        m.forward(toks[:1], [-1], 0, skip=odd, logits=False)
        m.forward(toks, parents, 0, logits=False)
        acc, _ = m.accept()
        m.compact(acc)
        m.set_committed(Lc)

    for _ in range(args.warmup):
        step()
    m.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    m.sync()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = elapsed / args.steps * 1e3
    value = T * args.steps / elapsed
    log(f"[bench] {args.steps} steps in {elapsed:.3f} s: {ms_step:.3f} ms/step")

    # per-kernel durations: the same steps, each launch bracketed by events on the library's stream
    m.profile(True)
    m.profile_read(reset=True)
    n_prof = min(args.steps, 10)
    for _ in range(n_prof):
        step()
    prof = m.profile_read(reset=True)
    m.profile(False)
    d, ffn, V = shape.d_model, shape.ffn_dim, shape.vocab
    n_run = shape.n_layers
    # gate/up launches per step: verify (all layers) + draft (odd layers skipped)
    gu_ms, gu_n = prof["gemm_gateup"]
    gu_avg_ms = gu_ms / max(gu_n, 1)
    # the two forwards have T=32 and T=1; take the mean over the verify launches only from a verify-only pass
    m.profile(True)
    m.profile_read(reset=True)
    for _ in range(n_prof):
        m.forward(toks, parents, 0, logits=False)
    pv = m.profile_read(reset=True)
    m.profile(False)
    v_gu_ms, v_gu_n = pv["gemm_gateup"]
    v_gu_avg = v_gu_ms / max(v_gu_n, 1)
    gu_bytes = gemm_bytes(2 * ffn, d, T, T * ffn * 2)
    achieved = gu_bytes / (v_gu_avg * 1e-3) / 1e9
    verify_ms = sum(x[0] for x in pv.values()) / n_prof
    kernels_verify = {k: {"ms_per_call": round(v[0] / n_prof, 4), "launches_per_call": v[1] // n_prof}
                      for k, v in pv.items() if v[1]}

    # verify-only and draft-only times (graph replays, no profiling): the
    # median of at least 50 calls, each bracketed by events on the library's
    # stream, and the mean wall time of back-to-back calls
    def per_call_ms(fn, n):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        m.sync()
        t0 = time.perf_counter()
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
        m.sync()
        wall = (time.perf_counter() - t0) / n * 1e3
        return float(np.median([a.elapsed_time(b) for a, b in ev])), wall

    n_calls = max(50, args.steps)
    verify_ms_med, verify_wall_ms = per_call_ms(lambda: m.forward(toks, parents, 0, logits=False), n_calls)
    draft_ms_med, draft_wall_ms = per_call_ms(lambda: m.forward(toks[:1], [-1], 0, skip=odd, logits=False), n_calls)
    m.set_committed(Lc)

    vbytes = algorithmic_bytes(shape, T, Lc, n_run)
    dbytes = algorithmic_bytes(shape, 1, Lc, n_run - sum(odd))
    res = {
        "metric": "tree-verify tokens/sec + achieved HBM GB/s, 7B-shape bf16, T=32, ctx 1024",
        "value": round(value, 2),
        "unit": "tree tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: random N(0,0.02^2) bf16 weights, uniform-random 1024-token prompt and tree tokens",
        "config": {"workload": ("llama2-7b-shape bf16 decoder, batch 1, ctx 1024: draft forward of the root "
                                "skipping 16/32 layers + verify forward of a 32-node tree (4,2,2,1,1) + greedy "
                                "accept + KV commit"),
                   "tree_nodes": T, "ctx": Lc, "layers": shape.n_layers},
        "verify_ms": round(verify_ms_med, 4),
        "verify_timing": f"median of {n_calls} event-timed verify calls (graph replays)",
        "verify_wall_ms_mean": round(verify_wall_ms, 4),
        "verify_hbm_gbps": round(vbytes / (verify_ms_med * 1e-3) / 1e9, 1),
        "verify_frac_of_peak": round(vbytes / (verify_ms_med * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "verify_tokens_per_s": round(T / (verify_ms_med * 1e-3), 1),
        "verify_algorithmic_bytes": vbytes,
        "draft_ms": round(draft_ms_med, 4),
        "draft_wall_ms_mean": round(draft_wall_ms, 4),
        "draft_hbm_gbps": round(dbytes / (draft_ms_med * 1e-3) / 1e9, 1),
        "step_hbm_gbps": round((vbytes + dbytes) / (ms_step * 1e-3) / 1e9, 1),
        "verify_kernel_sum_ms": round(verify_ms, 4),
        "verify_kernels": kernels_verify,
        "roofline": {"bound": "hbm", "kernel": "gemm_gateup (bf16 MFMA, N=22016 K=4096 T=32, fused SwiGLU)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(),
                     "bytes_per_launch": gu_bytes, "avg_ms": round(v_gu_avg, 5)},
    }
    if args.layers:
        res["invalid"] = "reduced layer count (testing only)"
    m.close()
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        res["cpu_baseline"] = cpu_baseline(shape, weights, parents, toks, Lc)
        log(f"[bench] cpu baseline in {time.perf_counter() - t0:.1f} s")
    print(json.dumps(res))


if __name__ == "__main__":
    main()
