"""Writes greedy_paths.json: for each full-size decoder of the parity tests, a
root token and the oracle's greedy continuation from it, over that test's
seeded synthetic committed cache.

The full-size tests put this continuation on the main branch (the first-child
chain) of their verify tree, so greedy verification (Sec. 5.1) accepts a path
longer than the root.  A root qualifies when the oracle's top-1/top-2 logit
margin at every node of its continuation, the last one included (its argmax
is the bonus token), is at least MIN_MARGIN; the acceptance criterion itself
is a margin above 0.05, and the extra room keeps the library's bf16 logit
error at depth from deciding the test.  Candidate roots are drawn from a
seeded generator and tried in order.

Only the oracle computes anything here; the inputs come from the seeded
generators.  Run from the repository root:
    python tests/golden/make_greedy_paths.py
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2510_26843_amd import synth  # noqa: E402

MIN_MARGIN = 0.1
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "greedy_paths.json")

# (model, context, cache seed base, slots the cache is drawn with, tree)
CASES = [
    ("llama2_7b", 1024, 1000, 8192, ("branching", synth.TREE_7B)),
    ("llama2_13b", 2048, 2000, 2048, ("branching", synth.TREE_13B)),
    ("llama3_8b", 4096, 3000, 4096, ("balanced", 64)),
]


def tree(kind, arg):
    return synth.balanced_tree(arg) if kind == "balanced" else synth.tree_from_branching(*arg)


def main_path(parents):
    """The first-child chain from the root (node ids)."""
    path = [0]
    while True:
        kids = [i for i, p in enumerate(parents) if p == path[-1]]
        if not kids:
            return path
        path.append(min(kids))


def margin(row):
    top2 = np.sort(row)[-2:]
    return float(top2[1] - top2[0])


def search(name, ctx, seed0, slots, tspec):
    shape = synth.SHAPES[name]
    depth = len(main_path(tree(*tspec))) - 1
    t0 = time.time()
    w = synth.gen_weights(shape, seed=0)
    o = O.OracleModel(shape, w, max_ctx=ctx + 16)
    for l in range(shape.n_layers):
        k, v = synth.gen_kv(1, shape.n_kv_heads, slots, shape.head_dim, seed=seed0 + l)
        kf = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(np.ascontiguousarray(k[0][:, :ctx])))
        vf = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(np.ascontiguousarray(v[0][:, :ctx])))
        o.set_kv(l, kf, vf)
    print(f"{name}: model and cache in {time.time() - t0:.0f} s; path depth {depth}", flush=True)
    rng = np.random.Generator(np.random.PCG64(7))
    tried = 0
    while True:
        root = int(rng.integers(0, shape.vocab))
        tried += 1
        o.set_committed(ctx)
        toks, margins = [root], []
        ok = True
        for d in range(depth + 1):
            row = o.forward([toks[-1]], [-1 if d == 0 else d - 1], d)[0]
            margins.append(margin(row))
            if margins[-1] < MIN_MARGIN:
                ok = False
                break
            toks.append(int(np.argmax(row)))
        print(f"  root {root}: margins {[round(m, 3) for m in margins]}", flush=True)
        if ok:
            return {"ctx": ctx, "cache_seed0": seed0, "cache_slots": slots, "depth": depth,
                    "path": toks[:-1], "bonus": toks[-1], "margins": [round(m, 6) for m in margins],
                    "roots_tried": tried}


def main():
    want = sys.argv[1:] or [c[0] for c in CASES]
    out = json.load(open(OUT)) if os.path.exists(OUT) else {}
    out["_about"] = ("oracle greedy continuations (root first, then depth tokens, then the bonus) "
                     f"with every top-1/top-2 margin >= {MIN_MARGIN}; written by make_greedy_paths.py")
    for case in CASES:
        if case[0] in want:
            out[case[0]] = search(*case)
            with open(OUT, "w") as f:
                json.dump(out, f, indent=1)
                f.write("\n")


if __name__ == "__main__":
    main()
