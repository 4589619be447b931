"""Host decoding loops over the library: plain greedy decoding and greedy
speculative decoding with a static token tree drafted by DSIA levels.

Routing (which draft level fills which tree depth, how many children a node
gets) is host logic; every forward, the acceptance and the KV commit run in
the library's kernels.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .cas import Model


def _top(row: np.ndarray, b: int) -> List[int]:
    order = np.argsort(-row, kind="stable")  # ties to the lower token id
    return [int(x) for x in order[:b]]


def ar_decode(model: Model, prompt: Sequence[int], n_new: int) -> List[int]:
    """Greedy autoregressive decoding: a one-node tree per step."""
    model.set_committed(0)
    if len(prompt) > 1:
        model.prefill(list(prompt[:-1]))
    root = int(prompt[-1])
    out: List[int] = []
    while len(out) < n_new:
        model.forward([root], [-1], 0, logits=False)
        acc, bonus = model.accept()
        model.compact(acc)
        out.append(bonus)
        root = bonus
    return out


def cas_decode_static(model: Model, prompt: Sequence[int], n_new: int, tree_parents: Sequence[int],
                      level_of_depth: Dict[int, Tuple[Optional[Sequence[int]], bool]],
                      stats: Optional[Dict] = None) -> List[int]:
    """Greedy CAS decoding with a static tree: the draft level of depth d
    (skip mask, act_quant) runs over the nodes at depth d in one tree-parallel
    call and its top-b tokens become their children; then one full-depth
    verify of the tree, greedy acceptance and the KV commit."""
    T = len(tree_parents)
    depth = [0] * T
    for i, p in enumerate(tree_parents):
        depth[i] = 0 if p < 0 else depth[p] + 1
    max_d = max(depth)
    by_depth = [[i for i in range(T) if depth[i] == d] for d in range(max_d + 1)]
    for ids in by_depth:
        if ids != list(range(ids[0], ids[-1] + 1)):
            raise ValueError("tree nodes must be numbered depth by depth")
    children: Dict[int, List[int]] = {}
    for i, p in enumerate(tree_parents):
        children.setdefault(p, []).append(i)
    model.set_committed(0)
    if len(prompt) > 1:
        model.prefill(list(prompt[:-1]))
    root = int(prompt[-1])
    out: List[int] = []
    rounds = 0
    toks = np.zeros(T, dtype=np.int32)
    while len(out) < n_new:
        toks[:] = 0
        toks[0] = root
        for d in range(max_d):
            ids = by_depth[d]
            skip, aq = level_of_depth[d]
            lg = model.forward(toks[ids[0]:ids[-1] + 1], [tree_parents[i] for i in ids], ids[0], skip=skip,
                               act_quant=aq)
            for r, i in enumerate(ids):
                ch = children.get(i, [])
                for c, t in zip(ch, _top(lg[r], len(ch))):
                    toks[c] = t
        model.forward(toks, tree_parents, 0, logits=False)
        path, bonus = model.accept()
        model.compact(path)
        out.extend(int(toks[i]) for i in path[1:])
        out.append(bonus)
        root = bonus
        rounds += 1
        if stats is not None:
            stats.setdefault("accepted", []).append(len(path) - 1)
    if stats is not None:
        stats["rounds"] = rounds
    return out[:n_new]
