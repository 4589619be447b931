"""Dynamic Tree Cascade (DyTC): the host-side scheduler of CAS-Spec.

DyTC (Sec. 4.2, Alg. 1; the functions of Alg. 2 in App. D) grows a draft
token tree one expansion at a time.  It picks the active leaf with the
highest accumulated acceptance rate, chooses a draft configuration and a
draft length by the step objective, and drafts.  The objective adds the
expected speedup of the step to the least future speedup of the bottom
draft.  The whole tree then goes through one full-depth verify.  Everything
here is host logic over the library's calls:
  - cas_forward with a skip mask / int8 activations is a draft step over a
    leaf and its sibling leaves (tree-parallel draft generation);
  - cas_topk returns the K candidates of every drafted position with their
    normalised probabilities;
  - cas_forward at full depth + cas_accept_tree + cas_kv_compact verify and
    commit the tree.

Contents:
  - the EWIF formulas of speculative decoding and of the horizontal cascade
    (Sec. 3) and the DyTC step objective (Sec. 4.2);
  - find_best_config: FindBestConfigurationForStep (Alg. 2);
  - AcceptanceEstimator: the per-configuration EMA of first-token acceptance
    (Sec. 4.2, "Acceptance Rate for Draft Configurations"; App. D);
  - pld_propose: prompt-lookup drafting, the bottom draft model;
  - LatencyModel: Bayesian linear regression of forward latency on roofline
    features, which gives the cost coefficients c-hat (Sec. 4.2,
    "Hardware-Aware Latency Prediction");
  - build_tree / cas_decode_dytc: Alg. 1 and the decoding loop.

Readings where Alg. 1 is ambiguous or silent:
  R1 A leaf is a node without children.  An expanded leaf stops being one,
     so the argmax over active leaves never picks it again.
  R2 Expanding a leaf with a neural configuration for k steps feeds the leaf
     (and, tree-parallel, its unexpanded sibling leaves) through the draft
     model, then the chain heads step by step.  At each step the top-1
     candidate continues the chain.  On the leaf's own chain only, the other
     candidates inside the top-P nucleus (cumulative probability of the
     better candidates below P_tree) become sibling leaves of that chain node.
  R3 P_acc(child) = P_acc(parent) * alpha-hat_S for the top-1 candidate
     (Alg. 1).  For the other candidates it is further scaled by p_j / p_0,
     their normalised probability relative to the top-1 (the token-level
     refinement of Sec. 4.2).
  R4 A neural configuration may extend a leaf only if every ancestor on the
     path was fed by a draft call that ran a superset of its layers.  These
     are the only KV entries the draft's attention reads.  The cascade's
     skip sets nest (the 25% set inside the 50% set), so better drafts fill
     shallow depths and cheaper ones deeper: the Tree Cascade of Sec. 4.2.
     Prompt-lookup nodes are never fed; only prompt lookup extends them.
  R5 The acceptance outcome of an expansion is whether its first drafted
     token (the top-1 child of the expanded leaf) was accepted.  It counts
     only when the expanded leaf itself was accepted: alpha is a conditional
     probability.
  R6 The cost coefficient c-hat_S is the predicted latency of one draft
     step over one row divided by the predicted latency of one target
     forward over one row (Sec. 3: ratio of single-step inference times).
  R7 The candidates at a leaf are the configurations that can draft there:
     neural ones under R4, prompt lookup only when the leaf's sequence has
     an n-gram match.  Alg. 1 stops the round when no configuration is
     chosen; with leaf-dependent candidates, a leaf that has none is
     retired and the next best leaf is tried.
  R8 t_min, the minimum local speedup, also bounds the chosen step: the
     round stops when T_s(S*, k*) * P_acc(leaf) < t_min, not only when the
     bottom draft's alpha/c * P_acc is below it.  Drafting that yields fewer
     tokens per unit of target-forward cost than t_min is not started.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# EWIF formulas (Sec. 3, from the cascade speculative decoding analysis)
# ----------------------------------------------------------------------------


def expected_accepted(alpha: float, k: int) -> float:
    """Expected number of accepted tokens among k drafted ones whose
    acceptances are i.i.d. Bernoulli(alpha), stopping at the first miss:
    alpha (1 - alpha^k) / (1 - alpha), or k when alpha is 1."""
    if abs(1.0 - alpha) < 1e-12:
        return float(k)
    return alpha * (1.0 - alpha ** k) / (1.0 - alpha)


def ewif_sd(alpha: float, c: float, k: int) -> float:
    """Expected walltime improvement factor of speculative decoding with one
    draft model of acceptance rate alpha and cost coefficient c drafting k
    tokens: (1 - alpha^(k+1)) / ((1 - alpha)(c k + 1))."""
    return (1.0 + expected_accepted(alpha, k)) / (c * k + 1.0)


def ewif_hc(a1: float, c1: float, k1: int, a2: float, c2: float, k2: int) -> float:
    """EWIF of the horizontal cascade: k1 tokens from draft 1, then k2 from
    draft 2, one verification: ((1 - a1^(k1+1)) / (1 - a1) + a1^k1 a2 (1 -
    a2^k2) / (1 - a2)) / (1 + k1 c1 + k2 c2)."""
    num = 1.0 + expected_accepted(a1, k1) + a1 ** k1 * expected_accepted(a2, k2)
    return num / (1.0 + k1 * c1 + k2 * c2)


def step_objective(alpha: float, c: float, k: int, alpha_n: float, c_n: float) -> float:
    """DyTC's per-step objective T_s(M_s, k): the expected accepted tokens of
    k draft steps of configuration (alpha, c), plus the least future
    speedup of one bottom-draft step, over their cost:
    (E[accepted] + alpha^k alpha_n) / (c k + c_n)."""
    den = c * k + c_n
    if den <= 1e-12:
        return -math.inf
    return (expected_accepted(alpha, k) + alpha ** k * alpha_n) / den


def find_best_config(candidates: Dict[str, Tuple[float, float]], alpha_n: float, c_n: float,
                     k_max: int) -> Tuple[Optional[str], int]:
    """FindBestConfigurationForStep (Alg. 2): the configuration and draft
    length k in [1, k_max] with the largest step objective; (None, 0) when
    no objective is positive.  candidates maps a configuration name to its
    (alpha-hat, c-hat); iteration follows the mapping's order and a later
    candidate must be strictly better to win."""
    best, best_k, best_val = None, 0, -math.inf
    for name, (a, c) in candidates.items():
        for k in range(1, k_max + 1):
            v = step_objective(a, c, k, alpha_n, c_n)
            if v > best_val:
                best, best_k, best_val = name, k, v
    if best_val <= 0.0:
        return None, 0
    return best, best_k


# ----------------------------------------------------------------------------
# acceptance-rate estimates
# ----------------------------------------------------------------------------

class AcceptanceEstimator:
    """Per-configuration acceptance-rate estimates (Sec. 4.2, App. D).
    Each configuration keeps the first-token outcomes of its most recent H
    expansions.  After every generation step in which a configuration drafted,
    alpha-new = lambda * alpha-prev + (1 - lambda) * (mean of the window).
    Configurations that did not draft keep their estimate (no decay).  Cold
    start: the given priors."""

    def __init__(self, priors: Dict[str, float], H: int = 20, lam: float = 0.7):
        self.H, self.lam = int(H), float(lam)
        self.a = {k: float(v) for k, v in priors.items()}
        self.window: Dict[str, List[int]] = {k: [] for k in priors}
        self._fresh: Dict[str, bool] = {k: False for k in priors}

    def alpha(self, name: str) -> float:
        return self.a[name]

    def record(self, name: str, accepted: bool) -> None:
        w = self.window.setdefault(name, [])
        w.append(1 if accepted else 0)
        if len(w) > self.H:
            del w[0]
        self._fresh[name] = True

    def end_step(self) -> None:
        for name, fresh in self._fresh.items():
            if fresh:
                w = self.window[name]
                self.a[name] = self.lam * self.a[name] + (1.0 - self.lam) * (sum(w) / len(w))
                self._fresh[name] = False


# ----------------------------------------------------------------------------
# prompt lookup (the bottom draft model)
# ----------------------------------------------------------------------------

def pld_propose(seq: Sequence[int], k: int, n_max: int = 3, n_min: int = 1) -> Tuple[List[int], int]:
    """Prompt-lookup drafting: for n = n_max down to n_min, find the most
    recent earlier occurrence of the last n tokens of seq; propose the (up
    to k) tokens that followed it.  Returns (tokens, n); ([], 0) when no
    n-gram recurs.  The match length n is the draft's token-level
    confidence (Sec. 4.2).  The search is vectorised over start positions."""
    a = np.asarray(seq, dtype=np.int64)
    L = a.shape[0]
    for n in range(min(n_max, L - 1), n_min - 1, -1):
        S = L - n  # candidate starts 0 .. L-n-1 (the last n tokens themselves excluded)
        hit = np.ones(S, dtype=bool)
        for j in range(n):
            hit &= a[j:j + S] == a[L - n + j]
        idx = np.flatnonzero(hit)
        if idx.size:
            start = int(idx[-1])
            return [int(x) for x in a[start + n:start + n + k]], n
    return [], 0


# ----------------------------------------------------------------------------
# latency prediction (cost coefficients)
# ----------------------------------------------------------------------------

def roofline_features(shape, run_layers: int, n_rows: int, ctx: int, act_quant: int = 0) -> np.ndarray:
    """Roofline features of one forward: [1, weight GB of the layers that run
    (+ LM head), KV GB read, dense TFLOP, layers run].  The constant and the
    layer count absorb launch and latency floors, the byte terms the HBM
    time, the FLOP term the matrix-core time.  act_quant 1 (W8A8) reads one
    byte per weight of the run layers, 2 (W4A4) half a byte."""
    es = 2 if shape.dtype == "bf16" else 4
    wb = {0: es, 1: 1, 2: 0.5}[int(act_quant)]
    wbytes = run_layers * shape.layer_params() * wb + shape.vocab * shape.d_model * es
    kv = run_layers * 2 * shape.n_kv_heads * shape.head_dim * es * (ctx + n_rows)
    flops = 2.0 * n_rows * (run_layers * shape.layer_params() + shape.vocab * shape.d_model)
    return np.array([1.0, wbytes / 1e9, kv / 1e9, flops / 1e12, float(run_layers)])


class LatencyModel:
    """Bayesian linear regression of forward latency (ms) on roofline
    features, with prior w ~ N(0, I / prior_precision) and Gaussian noise of
    precision noise_precision: posterior precision A = a I + b F^T F, mean
    m = b A^-1 F^T y; a prediction is f^T m with variance 1/b + f^T A^-1 f."""

    def __init__(self, prior_precision: float = 1e-2, noise_precision: float = 1e2):
        self.a, self.b = float(prior_precision), float(noise_precision)
        self.mean: Optional[np.ndarray] = None
        self.cov: Optional[np.ndarray] = None

    def fit(self, F: np.ndarray, y: np.ndarray) -> "LatencyModel":
        F = np.asarray(F, dtype=np.float64)
        y = np.asarray(y, dtype=np.float64)
        A = self.a * np.eye(F.shape[1]) + self.b * F.T @ F
        self.cov = np.linalg.inv(A)
        self.mean = self.b * self.cov @ F.T @ y
        return self

    def predict(self, f: np.ndarray) -> Tuple[float, float]:
        if self.mean is None:
            raise RuntimeError("LatencyModel.predict before fit")
        f = np.asarray(f, dtype=np.float64)
        return float(f @ self.mean), float(1.0 / self.b + f @ self.cov @ f)


# ----------------------------------------------------------------------------
# draft configurations and the tree
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class DraftConfig:
    """A draft model: a DSIA variant of the target (skip mask over the
    layers, optional quantised activations: 1 = W8A8, 2 = W4A4, optional sink
    + window attention) or prompt lookup (skip is None and pld is True)."""
    name: str
    skip: Optional[Tuple[int, ...]] = None
    act_quant: int = 0
    pld: bool = False
    window: Optional[Tuple[int, int]] = None  # efficient attention: (sink, window) committed slots

    def run_layers(self, n_layers: int) -> frozenset:
        if self.pld:
            return frozenset()
        return frozenset(l for l in range(n_layers) if not (self.skip and self.skip[l]))


@dataclasses.dataclass
class Node:
    token: int
    parent: int                     # index into the tree's node list, -1 for the root
    config: Optional[str]           # the configuration that drafted it (None: root)
    p_acc: float                    # accumulated acceptance rate of the path to it
    children: List[int] = dataclasses.field(default_factory=list)
    active: bool = True
    fed_id: int = -1                # round node id when a draft call fed it
    run: frozenset = frozenset()    # layers whose KV a draft call wrote for it
    pld_made: bool = False          # drafted by prompt lookup (never fed)
    first_of: Optional[str] = None  # first drafted token of an expansion by this config


@dataclasses.dataclass
class DytcParams:
    max_tree: int = 64      # M_tree_max
    k_max: int = 5          # maximum draft length per expansion
    t_min: float = 1.1      # minimum local speedup to keep drafting
    top_k: int = 4          # K candidates per drafted position
    top_p: float = 0.9      # P_tree nucleus for the extra candidates
    pld_n_max: int = 3


class DraftTree:
    """The draft token tree of one round and the draft calls that fed it."""

    def __init__(self, root_token: int):
        self.nodes: List[Node] = [Node(int(root_token), -1, None, 1.0)]
        self.fed: List[int] = []  # node indices in feed order (= round node ids)

    def __len__(self) -> int:
        return len(self.nodes)

    def add(self, parent: int, token: int, config: str, p_acc: float, pld: bool = False) -> int:
        self.nodes.append(Node(int(token), parent, config, p_acc, pld_made=pld))
        i = len(self.nodes) - 1
        self.nodes[parent].children.append(i)
        return i

    def path(self, i: int) -> List[int]:
        out = []
        while i >= 0:
            out.append(i)
            i = self.nodes[i].parent
        return out[::-1]

    def best_leaf(self) -> Optional[int]:
        best, bv = None, -1.0
        for i, n in enumerate(self.nodes):
            if n.active and not n.children and n.p_acc > bv:
                best, bv = i, n.p_acc
        return best

    def neural_ok(self, leaf: int, run: frozenset) -> bool:
        """R4: every ancestor of the leaf was fed with KV in all of run, and
        the leaf itself is not fed yet (nothing is fed when the leaf is the
        root)."""
        if self.nodes[leaf].fed_id >= 0 or self.nodes[leaf].pld_made:
            return False
        if leaf == 0:
            return not self.fed
        for a in self.path(leaf)[:-1]:
            n = self.nodes[a]
            if n.fed_id < 0 or not run <= n.run:
                return False
        return True

    def ordering(self) -> List[int]:
        """Round node ids for the verify: fed nodes in feed order, then the
        rest in creation order (parents always precede children)."""
        fed = set(self.fed)
        return list(self.fed) + [i for i in range(len(self.nodes)) if i not in fed]


# ----------------------------------------------------------------------------
# Alg. 1 and the decoding loop
# ----------------------------------------------------------------------------

class LibraryBackend:
    """The library's calls as DyTC uses them (cas.Model)."""

    def __init__(self, model):
        self.m = model

    def reset(self, prompt: Sequence[int]) -> None:
        self.m.set_committed(0)
        if len(prompt) > 1:
            self.m.prefill(list(prompt[:-1]))

    def draft(self, tokens, parents, node_offset: int, cfg: DraftConfig, K: int):
        self.m.forward(tokens, parents, node_offset, skip=list(cfg.skip) if cfg.skip else None,
                       act_quant=cfg.act_quant, logits=False, attn_window=cfg.window)
        return self.m.topk(K, len(tokens))

    def verify(self, tokens, parents) -> Tuple[List[int], int]:
        self.m.forward(tokens, parents, 0, logits=False)
        return self.m.accept()

    def commit(self, path: Sequence[int]) -> None:
        self.m.compact(path)


def _feed(tree: DraftTree, backend, rows: List[int], cfg: DraftConfig, K: int, n_layers: int):
    """One draft call over the given unfed nodes: they get the next round ids."""
    off = len(tree.fed)
    toks, pars = [], []
    for i in rows:
        n = tree.nodes[i]
        toks.append(n.token)
        pars.append(-1 if n.parent < 0 else tree.nodes[n.parent].fed_id)
    ids, probs = backend.draft(toks, pars, off, cfg, K)
    run = cfg.run_layers(n_layers)
    for j, i in enumerate(rows):
        tree.nodes[i].fed_id = off + j
        tree.nodes[i].run = run
        tree.fed.append(i)
    return ids, probs


def build_tree(backend, root_token: int, context: Sequence[int], configs: Sequence[DraftConfig],
               bottom: DraftConfig, est: AcceptanceEstimator, cost: Dict[str, float], params: DytcParams,
               n_layers: int, stats: Optional[Dict] = None) -> DraftTree:
    """Alg. 1: grow the draft tree of one round (readings R1-R6 above)."""
    tree = DraftTree(root_token)
    ctx = np.asarray(context, dtype=np.int64)
    by_name = {c.name: c for c in configs}
    a_n, c_n = est.alpha(bottom.name), cost[bottom.name]
    M = params.max_tree
    while len(tree) < M:
        leaf = tree.best_leaf()
        if leaf is None:
            break
        if c_n > 0 and a_n / c_n * tree.nodes[leaf].p_acc < params.t_min:
            break
        cands = {}
        lookup: List[int] = []
        for c in configs:
            if c.pld:
                seq = np.concatenate([ctx, np.array([tree.nodes[i].token for i in tree.path(leaf)], dtype=np.int64)])
                lookup, _ = pld_propose(seq, params.k_max, params.pld_n_max)
                if lookup:
                    cands[c.name] = (est.alpha(c.name), cost[c.name])
            elif tree.neural_ok(leaf, c.run_layers(n_layers)):
                cands[c.name] = (est.alpha(c.name), cost[c.name])
        name, k = find_best_config(cands, a_n, c_n, params.k_max)
        if name is None:
            tree.nodes[leaf].active = False
            continue
        a_b, c_b = cands[name]
        if step_objective(a_b, c_b, k, a_n, c_n) * tree.nodes[leaf].p_acc < params.t_min:
            break
        cfg = by_name[name]
        a_s = est.alpha(name)
        if stats is not None:
            stats.setdefault("expansions", {}).setdefault(name, 0)
            stats["expansions"][name] += 1
        if cfg.pld:
            prop = lookup[:min(k, M - len(tree))]
            cur = leaf
            for j, t in enumerate(prop):
                cur = tree.add(cur, t, name, tree.nodes[cur].p_acc * a_s, pld=True)
                if j == 0:
                    tree.nodes[cur].first_of = name
            continue
        # neural: the leaf plus its unexpanded, unfed sibling leaves, fed together
        rows = [leaf]
        par = tree.nodes[leaf].parent
        if par >= 0:
            sibs = [s for s in tree.nodes[par].children
                    if s != leaf and not tree.nodes[s].children and tree.nodes[s].active
                    and tree.nodes[s].fed_id < 0 and not tree.nodes[s].pld_made]
            sibs.sort(key=lambda s: -tree.nodes[s].p_acc)
            rows += sibs
        heads = rows[:max(1, min(len(rows), M - len(tree)))]
        for step in range(k):
            if len(tree) >= M:
                break
            ids, probs = _feed(tree, backend, heads, cfg, params.top_k, n_layers)
            new_heads = []
            for r, h in enumerate(heads):
                if len(tree) >= M:
                    break
                p0 = float(probs[r][0])
                c0 = tree.add(h, int(ids[r][0]), name, tree.nodes[h].p_acc * a_s)
                if step == 0 and r == 0:
                    tree.nodes[c0].first_of = name
                new_heads.append(c0)
                if r == 0:
                    cum = p0
                    for j in range(1, params.top_k):
                        if cum >= params.top_p or len(tree) >= M or int(ids[r][j]) < 0:
                            break
                        pj = float(probs[r][j])
                        tree.add(h, int(ids[r][j]), name,
                                 tree.nodes[h].p_acc * a_s * (pj / p0 if p0 > 0 else 0.0))
                        cum += pj
            heads = new_heads
            if not heads:
                break
    return tree


def cas_decode_dytc(backend, prompt: Sequence[int], n_new: int, configs: Sequence[DraftConfig],
                    bottom: DraftConfig, est: AcceptanceEstimator, cost: Dict[str, float],
                    params: DytcParams, n_layers: int, stats: Optional[Dict] = None) -> List[int]:
    """Greedy CAS decoding with DyTC trees: per round, Alg. 1 builds the
    tree, one full-depth verify checks it, the accepted path is committed and
    the acceptance estimates take the round's first-token outcomes.  The
    output equals greedy autoregressive decoding (Sec. 5.1)."""
    backend.reset(prompt)
    # the sequence so far, kept in one buffer (the context prompt lookup scans)
    seq = np.empty(len(prompt) + n_new + params.max_tree + 1, dtype=np.int64)
    seq[:len(prompt)] = prompt
    n_seq = len(prompt)
    out: List[int] = []
    root = int(prompt[-1])
    while len(out) < n_new:
        tree = build_tree(backend, root, seq[:n_seq - 1], configs, bottom, est, cost, params, n_layers, stats)
        order = tree.ordering()
        rid = {node: j for j, node in enumerate(order)}
        toks = [tree.nodes[i].token for i in order]
        pars = [-1 if tree.nodes[i].parent < 0 else rid[tree.nodes[i].parent] for i in order]
        path_ids, bonus = backend.verify(toks, pars)
        backend.commit(path_ids)
        accepted = {order[j] for j in path_ids}
        for i, n in enumerate(tree.nodes):
            if n.first_of is not None and n.parent in accepted:
                est.record(n.first_of, i in accepted)
        est.end_step()
        new = [tree.nodes[order[j]].token for j in path_ids[1:]] + [int(bonus)]
        out.extend(new)
        seq[n_seq:n_seq + len(new)] = new
        n_seq += len(new)
        root = int(bonus)
        if stats is not None:
            stats.setdefault("accepted", []).append(len(path_ids) - 1)
            stats.setdefault("tree_sizes", []).append(len(tree))
    return out[:n_new]
