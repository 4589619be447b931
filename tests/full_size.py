"""Helpers of the full-size parity tests (7B, 13B and 8B shapes): row errors,
sampled sub-trees, and the check of greedy acceptance against the oracle's
own decision (Sec. 5.1: the accepted tokens must be the target's greedy
continuation)."""
import json
import os

import numpy as np

from paper_2510_26843_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "greedy_paths.json")
MARGIN = 0.05   # the acceptance criterion: identical decisions wherever the oracle's margin exceeds it


def row_err(got, ref):
    """Per-row max |got - ref| relative to the row's max |ref|, worst row."""
    return float((np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)).max())


def subtree(parents, nodes):
    """Node ids on the root paths of `nodes` (ascending, so parents first)
    and their parent list renumbered to positions in that id list."""
    keep = set()
    for n in nodes:
        while n != -1:
            keep.add(n)
            n = parents[n]
    ids = sorted(keep)
    pos = {old: i for i, old in enumerate(ids)}
    return ids, [-1 if parents[i] == -1 else pos[parents[i]] for i in ids]


def main_path(parents):
    """The first-child chain from the root (node ids)."""
    path = [0]
    while True:
        kids = [i for i, p in enumerate(parents) if p == path[-1]]
        if not kids:
            return path
        path.append(min(kids))


def greedy_record(model_name):
    with open(GOLDEN) as f:
        return json.load(f)[model_name]


def tree_tokens_on_greedy_path(parents, vocab, seed, path_tokens):
    """Seeded random tokens with distinct siblings, the main branch carrying
    the given tokens (the oracle's greedy continuation of its root)."""
    toks = synth.gen_tree_tokens(parents, vocab, seed=seed)
    mp = main_path(parents)
    assert len(path_tokens) == len(mp), (len(path_tokens), len(mp))
    for node, t in zip(mp, path_tokens):
        toks[node] = t
    for node in mp[1:]:
        sibs = [i for i, p in enumerate(parents) if p == parents[node] and i != node]
        for s in sibs:
            while toks[s] == toks[node] or any(toks[s] == toks[o] for o in sibs if o != s):
                toks[s] = (toks[s] + 1) % vocab
    return toks


def oracle_acceptance(rows, parents, toks):
    """The oracle's greedy walk over the rows it computed ({node: logits}):
    accepted node ids (root first), bonus token, and the top-1/top-2 margin
    at every accepted node."""
    children = {}
    for i, p in enumerate(parents):
        children.setdefault(p, []).append(i)
    path, margins = [0], []
    while True:
        cur = path[-1]
        assert cur in rows, f"the walk reached node {cur}, whose row the oracle did not compute"
        row = np.asarray(rows[cur], dtype=np.float64)
        g = int(np.argmax(row))
        top = np.sort(row)[-2:]
        margins.append(float(top[1] - top[0]))
        nxt = [c for c in children.get(cur, []) if int(toks[c]) == g]
        if not nxt:
            return path, g, margins
        path.append(nxt[0])


def check_acceptance(lib_result, rows, parents, toks, tag):
    """The library's acceptance equals the oracle's wherever every margin on
    the oracle's accepted path exceeds MARGIN (else the case is reported as
    tie-excused).  Returns the oracle's (path, bonus)."""
    path, bonus, margins = oracle_acceptance(rows, parents, toks)
    print(f"[full] {tag}: oracle accepts {len(path)} nodes (bonus {bonus}), margins "
          f"{[round(m, 3) for m in margins]}; library accepts {len(lib_result[0])} (bonus {lib_result[1]})",
          flush=True)
    if min(margins) > MARGIN:
        assert (list(lib_result[0]), int(lib_result[1])) == (path, bonus), (lib_result, path, bonus)
    else:
        print(f"[full] {tag}: tie-excused (oracle margin {min(margins):.3e} <= {MARGIN})", flush=True)
    return path, bonus
