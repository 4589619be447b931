"""Seeded synthetic inputs for the token-tree decoder step.

This module draws random numbers and builds tree *shapes*; it holds none of the
method's arithmetic (no norm, projection, attention, masking or acceptance).
Both the CPU oracle's tests and the HIP path's tests, bench and smoke take their
inputs from here, so the two sides see identical bytes.

Stand-ins (the paper's workloads use trained Vicuna/Llama-2 weights and
Spec-Bench prompts, neither of which is available): Llama-shaped decoders with
random N(0, 0.02^2) weights, RMSNorm gains of one, uniform-random prompts and
uniform-random tree tokens with distinct siblings.
"""
from __future__ import annotations

import concurrent.futures as _fut
import dataclasses
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# tensor codes used to derive one independent seed per weight tensor
_TENSOR_CODE = {"embed": 0, "lm_head": 1, "wq": 2, "wk": 3, "wv": 4,
                "wo": 5, "w_gate": 6, "w_up": 7, "w_down": 8}
LAYER_TENSORS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float
    rms_eps: float
    dtype: str  # "f32" or "bf16": storage type of weights and activations

    def tensor_shape(self, name: str) -> Tuple[int, int]:
        d, hd = self.d_model, self.head_dim
        return {
            "embed": (self.vocab, d),
            "lm_head": (self.vocab, d),
            "wq": (self.n_heads * hd, d),
            "wk": (self.n_kv_heads * hd, d),
            "wv": (self.n_kv_heads * hd, d),
            "wo": (d, self.n_heads * hd),
            "w_gate": (self.ffn_dim, d),
            "w_up": (self.ffn_dim, d),
            "w_down": (d, self.ffn_dim),
        }[name]

    def layer_params(self) -> int:
        return sum(int(np.prod(self.tensor_shape(t))) for t in LAYER_TENSORS)

    def with_layers(self, n_layers: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n_layers,
                                   name=f"{self.name}[{n_layers}L]")


# The decoder shapes of the workloads: a tiny fp32 decoder, and the
# Llama-2-7B / Llama-2-13B / Llama-3-8B (GQA) shapes in bf16.
SHAPES: Dict[str, ModelShape] = {
    "tiny": ModelShape("tiny", 4, 256, 4, 4, 64, 688, 2048, 1e4, 1e-6, "f32"),
    "llama2_7b": ModelShape("llama2_7b", 32, 4096, 32, 32, 128, 11008, 32000, 1e4, 1e-6, "bf16"),
    "llama2_13b": ModelShape("llama2_13b", 40, 5120, 40, 40, 128, 13824, 32000, 1e4, 1e-6, "bf16"),
    "llama3_8b": ModelShape("llama3_8b", 32, 4096, 32, 8, 128, 14336, 128256, 5e5, 1e-6, "bf16"),
}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even) and return the uint16 bit patterns."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _rng(seed: int, layer: int, code: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, layer + 1, code])))


def gen_tensor(shape: ModelShape, name: str, layer: int = -1, seed: int = 0,
               std: float = 0.02) -> np.ndarray:
    """One weight tensor, N(0, std^2), row-major [out][in].

    fp32 models get float32 values; bf16 models get uint16 bf16 bit patterns
    (float32 draw rounded once, RNE).  Each tensor has its own seed stream, so any
    single tensor can be regenerated alone.
    """
    rows, cols = shape.tensor_shape(name)
    g = _rng(seed, layer, _TENSOR_CODE[name])
    a = g.standard_normal((rows, cols), dtype=np.float32)
    a *= np.float32(std)
    if shape.dtype == "bf16":
        return f32_to_bf16_bits(a)
    return a


def gen_weights(shape: ModelShape, seed: int = 0, threads: Optional[int] = None,
                layers: Optional[Sequence[int]] = None) -> Dict:
    """All weights of a model: {"embed", "lm_head", "final_norm", "layers": [ {name: array} ]}.

    Norm gains are ones (float32).  `layers` restricts which layers are drawn
    (others are None); drawing runs on a thread pool (numpy releases the GIL).
    """
    if threads is None:
        threads = min(16, os.cpu_count() or 1)
    want = list(range(shape.n_layers)) if layers is None else list(layers)
    jobs = [("embed", -1), ("lm_head", -1)] + [(t, l) for l in want for t in LAYER_TENSORS]
    out: Dict = {"layers": [None] * shape.n_layers}
    with _fut.ThreadPoolExecutor(max_workers=threads) as ex:
        futs = {ex.submit(gen_tensor, shape, n, l, seed): (n, l) for n, l in jobs}
        for f in _fut.as_completed(futs):
            n, l = futs[f]
            if l < 0:
                out[n] = f.result()
            else:
                if out["layers"][l] is None:
                    out["layers"][l] = {}
                out["layers"][l][n] = f.result()
    ones = np.ones(shape.d_model, dtype=np.float32)
    out["final_norm"] = ones
    for l in want:
        out["layers"][l]["attn_norm"] = ones
        out["layers"][l]["ffn_norm"] = ones
    return out


def gen_prompt(vocab: int, n: int, seed: int = 1) -> np.ndarray:
    """Uniform-random prompt tokens in [0, vocab)."""
    return np.random.Generator(np.random.PCG64(seed)).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def gen_activations(rows: int, cols: int, seed: int = 3, edge_rows: bool = True) -> np.ndarray:
    """float32 N(0,1) activations for isolated kernel tests, with edge rows
    (all zeros, one-hot, +-largest finite bf16-representable value, ties) mixed in."""
    a = np.random.Generator(np.random.PCG64(seed)).standard_normal((rows, cols), dtype=np.float32)
    if edge_rows and rows >= 4:
        a[1, :] = 0.0
        a[2, :] = 0.0
        a[2, cols // 3] = -3.5
        a[3, :] = np.float32(1.0)
        a[3, ::2] = np.float32(-1.0)
    return a


def gen_kv(n_layers: int, n_kv_heads: int, n_slots: int, head_dim: int, seed: int = 4,
           std: float = 1.28) -> Tuple[np.ndarray, np.ndarray]:
    """A synthetic committed KV cache, N(0, std^2) float32, [layer][kv_head][slot][head_dim].

    Stands in for a prefilled prompt when a full-size prefill is too slow for
    the CPU side; std matches the scale of k and v for RMS-normalised inputs
    times N(0, 0.02^2) weights at d=4096 (0.02 * 64 = 1.28).
    """
    g = np.random.Generator(np.random.PCG64(seed))
    k = g.standard_normal((n_layers, n_kv_heads, n_slots, head_dim), dtype=np.float32) * np.float32(std)
    v = g.standard_normal((n_layers, n_kv_heads, n_slots, head_dim), dtype=np.float32) * np.float32(std)
    return k, v


# ----------------------------------------------------------------------------
# tree shapes
# ----------------------------------------------------------------------------

def tree_from_branching(branching: Sequence[int], n_nodes: int) -> List[int]:
    """Parent list (BFS order, root parent -1) of an n-node tree cut from the
    full product tree of `branching` (children per node at each depth).

    Cut rule: a node whose rank path is (r1..rd) costs d + sum(r); keep the
    n_nodes cheapest (ties: shallower, then lexicographically smaller path),
    which keeps every kept node's parent.  Nodes are numbered breadth-first with
    children in rank order, so every parent id is below its children's ids.
    """
    paths: List[Tuple[int, ...]] = [()]
    frontier: List[Tuple[int, ...]] = [()]
    for b in branching:
        nxt = [p + (r,) for p in frontier for r in range(b)]
        paths.extend(nxt)
        frontier = nxt
    if n_nodes > len(paths):
        raise ValueError(f"branching {tuple(branching)} has only {len(paths)} nodes, asked {n_nodes}")
    kept = sorted(paths, key=lambda p: (len(p) + sum(p), len(p), p))[:n_nodes]
    kept.sort(key=lambda p: (len(p), p))
    index = {p: i for i, p in enumerate(kept)}
    parents = []
    for p in kept:
        if len(p) == 0:
            parents.append(-1)
        else:
            if p[:-1] not in index:
                raise AssertionError("cut tree lost a parent")
            parents.append(index[p[:-1]])
    return parents


def chain_parents(n: int) -> List[int]:
    """A chain 0 <- 1 <- ... <- n-1 (a plain causal sequence)."""
    return [-1] + list(range(n - 1))


def balanced_tree(n_nodes: int) -> List[int]:
    """The n-node cut of a full binary tree of depth 7 (up to 255 nodes)."""
    return tree_from_branching((2,) * 7, n_nodes)


def gen_tree_tokens(parents: Sequence[int], vocab: int, seed: int = 2,
                    root_token: Optional[int] = None) -> np.ndarray:
    """Uniform-random tokens for a tree with distinct tokens among siblings."""
    g = np.random.Generator(np.random.PCG64(seed))
    toks = np.zeros(len(parents), dtype=np.int32)
    used: Dict[int, set] = {}
    for i, p in enumerate(parents):
        s = used.setdefault(p, set())
        while True:
            t = int(g.integers(0, vocab))
            if t not in s:
                break
        s.add(t)
        toks[i] = t
    if root_token is not None:
        toks[0] = root_token
    return toks


# Workload trees of the measured configurations (n counts the root).
TREE_TINY = ((3, 2, 1), 15)          # 15-node tree, depth 3
TREE_7B = ((4, 2, 2, 1, 1), 32)      # 32-node tree, depth 5
TREE_13B = ((4, 4, 4, 4), 64)        # 64-node tree, depth 4
