"""CPU oracle of the CAS-Spec token-tree decoder step: Python side.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg use it; the product path never imports it.  It shares no code
with the HIP library (the only thing both sides share is the seeded input
module, which holds no arithmetic of the method).

The heavy decoder step lives in `cas_oracle.c` (plain C, fp64, OpenMP over
output features).  This file adds the pieces that are pure bookkeeping:
tree metadata, the greedy acceptance walk, and the autoregressive and static
tree-cascade decoding drivers built on the step.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cas_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

W_ORDER = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (OpenMP, no fast-math, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
                               "-fno-fast-math", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB_PATH)
        P, I, D, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_double, ctypes.c_float
        L.om_create.restype = P
        L.om_create.argtypes = [I, I, I, I, I, I, I, D, D, I, I]
        L.om_destroy.argtypes = [P]
        L.om_set_global.argtypes = [P, P, P, P]
        L.om_set_layer.argtypes = [P, I, P, P, P]
        L.om_set_layer_i8.argtypes = [P, I, P, P]
        L.om_set_layer_i4.argtypes = [P, I, P, P]
        L.om_set_threads.argtypes = [I]
        L.om_threads.restype = I
        L.om_set_kv.argtypes = [P, I, I, P, P]
        L.om_set_kv.restype = I
        L.om_get_kv.argtypes = [P, I, I, I, P, P]
        L.om_get_kv.restype = I
        L.om_set_committed.argtypes = [P, I]
        L.om_set_committed.restype = I
        L.om_committed.argtypes = [P]
        L.om_committed.restype = I
        L.om_forward.argtypes = [P, P, P, I, I, P, I, P, P]
        L.om_forward.restype = I
        L.om_set_window.argtypes = [P, I, I]
        L.om_set_window.restype = I
        L.om_compact.argtypes = [P, P, I]
        L.om_compact.restype = I
        L.om_round_bf16.argtypes = [D]
        L.om_round_bf16.restype = D
        L.om_quant_row.argtypes = [P, I, P, P]
        L.om_quant_weight.argtypes = [P, I, I, I, P, P]
        L.om_quant_row_q.argtypes = [P, I, I, P, P]
        L.om_quant_weight_q.argtypes = [P, I, I, I, I, P, P]
        L.om_dot_i8.argtypes = [P, P, I, P]
        L.om_dot_i8.restype = I
        L.om_rmsnorm_row.argtypes = [P, P, I, D, P]
        L.om_rope.argtypes = [P, I, I, D]
        L.om_attend.argtypes = [P, P, P, I, I, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def set_threads(n: int) -> None:
    lib().om_set_threads(int(n))


def threads() -> int:
    return int(lib().om_threads())


# ----------------------------------------------------------------------------
# op-level entry points (used by the pins and by kernel parity tests)
# ----------------------------------------------------------------------------

def round_bf16(x: float) -> float:
    return float(lib().om_round_bf16(float(x)))


def quant_rows(x: np.ndarray, qmax: int = 127) -> Tuple[np.ndarray, np.ndarray]:
    """Per-row symmetric quantisation of float32 rows to codes in [-qmax, qmax]
    (127: int8, 7: int4) -> (int8 q, float32 scale)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    rows, cols = x.shape
    q = np.zeros((rows, cols), dtype=np.int8)
    s = np.zeros(rows, dtype=np.float32)
    for r in range(rows):
        lib().om_quant_row_q(_ptr(x[r]), cols, int(qmax), _ptr(q[r]), s[r:].ctypes.data)
    return q, s


def quant_weight(w: np.ndarray, bf16: bool, qmax: int = 127) -> Tuple[np.ndarray, np.ndarray]:
    """Per-output-channel copy of W[out][in] (uint16 bf16 bits or float32),
    codes in [-qmax, qmax]."""
    w = np.ascontiguousarray(w)
    out, inn = w.shape
    q = np.zeros((out, inn), dtype=np.int8)
    s = np.zeros(out, dtype=np.float32)
    lib().om_quant_weight_q(_ptr(w), 1 if bf16 else 0, out, inn, int(qmax), _ptr(q), _ptr(s))
    return q, s


def dot_i8_matrix(qx: np.ndarray, qw: np.ndarray) -> np.ndarray:
    """acc[t][n] = sum_k qx[t][k] * qw[n][k] exactly (int32, overflow-checked)."""
    qx = np.ascontiguousarray(qx, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    out = np.zeros((qx.shape[0], qw.shape[0]), dtype=np.int32)
    v = np.zeros(1, dtype=np.int32)
    for t in range(qx.shape[0]):
        for n in range(qw.shape[0]):
            if lib().om_dot_i8(_ptr(qx[t]), _ptr(qw[n]), qx.shape[1], _ptr(v)):
                raise OverflowError("int8 dot product exceeds int32")
            out[t, n] = v[0]
    return out


def rmsnorm_row(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    g = np.ascontiguousarray(g, dtype=np.float32)
    y = np.zeros_like(x)
    lib().om_rmsnorm_row(_ptr(x), _ptr(g), x.shape[0], float(eps), _ptr(y))
    return y


def rope(v: np.ndarray, pos: int, theta: float) -> np.ndarray:
    v = np.array(v, dtype=np.float64, copy=True)
    lib().om_rope(_ptr(v), v.shape[0], int(pos), float(theta))
    return v


def attend(q: np.ndarray, keys: np.ndarray, vals: np.ndarray) -> np.ndarray:
    """Softmax attention of one query over an ordered list of keys (fp64)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    keys = np.ascontiguousarray(keys, dtype=np.float64)
    vals = np.ascontiguousarray(vals, dtype=np.float64)
    nk, hd = keys.shape
    kp = (ctypes.c_void_p * max(nk, 1))(*[keys[j].ctypes.data for j in range(nk)])
    vp = (ctypes.c_void_p * max(nk, 1))(*[vals[j].ctypes.data for j in range(nk)])
    o = np.zeros(hd, dtype=np.float64)
    lib().om_attend(_ptr(q), ctypes.cast(kp, ctypes.c_void_p), ctypes.cast(vp, ctypes.c_void_p), nk, hd, _ptr(o))
    return o


def matmul_rows(x: np.ndarray, w: np.ndarray, bf16: bool) -> np.ndarray:
    """y[t][n] = sum_k x[t][k] W[n][k] in fp64, W given as bf16 bits or float32.

    A plain library product of exact fp64 widenings (no rounding of the inputs)."""
    wf = (np.ascontiguousarray(w, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32) if bf16 else w
    return np.asarray(x, dtype=np.float64) @ np.asarray(wf, dtype=np.float64).T


# ----------------------------------------------------------------------------
# the model
# ----------------------------------------------------------------------------

class OracleModel:
    """A decoder with its own fp64 KV cache, mirroring the tree-forward API."""

    def __init__(self, shape, weights: Dict, max_ctx: int, int8: bool = False, int4: bool = False):
        self.shape = shape
        self.bf16 = shape.dtype == "bf16"
        self.max_ctx = int(max_ctx)
        self._keep: List[np.ndarray] = []
        L = lib()
        self.h = L.om_create(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                             shape.head_dim, shape.ffn_dim, shape.vocab, float(shape.rope_theta),
                             float(shape.rms_eps), 1 if self.bf16 else 0, self.max_ctx)
        if not self.h:
            raise MemoryError("oracle model allocation failed")
        emb = self._hold(weights["embed"])
        head = self._hold(weights["lm_head"])
        fn = self._hold(np.asarray(weights["final_norm"], dtype=np.float32))
        L.om_set_global(self.h, _ptr(emb), _ptr(head), _ptr(fn))
        self.int8 = False
        self._layers_set = [False] * shape.n_layers
        for l, lw in enumerate(weights["layers"]):
            if lw is None:
                continue
            ptrs = (ctypes.c_void_p * 7)(*[_ptr(self._hold(lw[n])) for n in W_ORDER])
            an = self._hold(np.asarray(lw["attn_norm"], dtype=np.float32))
            fn_ = self._hold(np.asarray(lw["ffn_norm"], dtype=np.float32))
            L.om_set_layer(self.h, l, ctypes.cast(ptrs, ctypes.c_void_p), _ptr(an), _ptr(fn_))
            self._layers_set[l] = True
            for on, qmax, setter in ((int8, 127, L.om_set_layer_i8), (int4, 7, L.om_set_layer_i4)):
                if not on:
                    continue
                qs, ss = [], []
                for n in W_ORDER:
                    q, s = quant_weight(lw[n], self.bf16, qmax)
                    qs.append(self._hold(q))
                    ss.append(self._hold(s))
                qp = (ctypes.c_void_p * 7)(*[_ptr(a) for a in qs])
                sp = (ctypes.c_void_p * 7)(*[_ptr(a) for a in ss])
                setter(self.h, l, ctypes.cast(qp, ctypes.c_void_p), ctypes.cast(sp, ctypes.c_void_p))
        self.int8 = bool(int8)
        self.int4 = bool(int4)

    def _hold(self, a: np.ndarray) -> np.ndarray:
        a = np.ascontiguousarray(a)
        self._keep.append(a)
        return a

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            lib().om_destroy(h)
            self.h = None

    # state ------------------------------------------------------------------
    @property
    def committed(self) -> int:
        return int(lib().om_committed(self.h))

    def set_committed(self, n: int) -> None:
        if lib().om_set_committed(self.h, int(n)):
            raise ValueError("bad committed length")

    def set_kv(self, layer: int, k: np.ndarray, v: np.ndarray) -> None:
        """Committed KV of one layer, [Hkv][n][hd] float32 values."""
        k = np.ascontiguousarray(k, dtype=np.float32)
        v = np.ascontiguousarray(v, dtype=np.float32)
        if lib().om_set_kv(self.h, int(layer), int(k.shape[1]), _ptr(k), _ptr(v)):
            raise ValueError("bad kv")

    def get_kv(self, layer: int, kvh: int, slot: int) -> Tuple[np.ndarray, np.ndarray]:
        k = np.zeros(self.shape.head_dim)
        v = np.zeros(self.shape.head_dim)
        if lib().om_get_kv(self.h, layer, kvh, slot, _ptr(k), _ptr(v)):
            raise IndexError("bad kv slot")
        return k, v

    # the step ----------------------------------------------------------------
    def forward(self, tokens: Sequence[int], parents: Sequence[int], node_offset: int = 0,
                skip: Optional[Sequence[int]] = None, act_quant: int = 0,
                need: Optional[Sequence[bool]] = None,
                attn_window: Optional[Tuple[int, int]] = None) -> np.ndarray:
        """act_quant: 0, 1 (or True) = int8 activations against the int8 copy,
        2 = int4 activations against the int4 copy.  attn_window = (sink,
        window): efficient-attention draft that sees only the first sink and
        the last window committed slots."""
        sink, win = attn_window if attn_window else (0, 0)
        if lib().om_set_window(self.h, int(sink), int(win)):
            raise ValueError("bad attention window")
        try:
            return self._forward(tokens, parents, node_offset, skip, act_quant, need)
        finally:
            lib().om_set_window(self.h, 0, 0)

    def _forward(self, tokens, parents, node_offset, skip, act_quant, need) -> np.ndarray:
        toks = np.ascontiguousarray(tokens, dtype=np.int32)
        par = np.ascontiguousarray(parents, dtype=np.int32)
        n = toks.shape[0]
        skip_a = None if skip is None else np.ascontiguousarray(
            [1 if x else 0 for x in skip], dtype=np.uint8)
        if skip_a is not None and skip_a.shape[0] != self.shape.n_layers:
            raise ValueError("skip mask length")
        for l in range(self.shape.n_layers):
            if (skip_a is None or not skip_a[l]) and not self._layers_set[l]:
                raise ValueError(f"layer {l} has no weights")
        need_a = None if need is None else np.ascontiguousarray([1 if x else 0 for x in need], dtype=np.uint8)
        logits = np.zeros((n, self.shape.vocab), dtype=np.float64)
        rc = lib().om_forward(self.h, _ptr(toks), _ptr(par), int(node_offset), n,
                              None if skip_a is None else _ptr(skip_a), int(act_quant),
                              None if need_a is None else _ptr(need_a), _ptr(logits))
        if rc == -2:
            raise OverflowError("int8 accumulator overflow")
        if rc:
            raise ValueError("invalid forward arguments")
        return logits

    def compact(self, accepted: Sequence[int]) -> None:
        acc = np.ascontiguousarray(accepted, dtype=np.int32)
        if lib().om_compact(self.h, _ptr(acc), int(acc.shape[0])):
            raise ValueError("invalid compaction")

    def prefill(self, tokens: Sequence[int]) -> np.ndarray:
        """Commit tokens as a causal chain; returns the last token's logits."""
        n = len(tokens)
        need = [False] * (n - 1) + [True]
        lg = self.forward(tokens, [-1] + list(range(n - 1)), 0, need=need)
        self.compact(list(range(n)))
        return lg[-1]


# ----------------------------------------------------------------------------
# tree bookkeeping, acceptance and the decoding drivers
# ----------------------------------------------------------------------------

def tree_metadata(parents: Sequence[int]) -> Tuple[List[int], List[int]]:
    """Depth of every node and its ancestor-or-self set as an integer bitmask."""
    depth: List[int] = []
    anc: List[int] = []
    for i, p in enumerate(parents):
        if p < 0:
            depth.append(0)
            anc.append(1 << i)
        else:
            depth.append(depth[p] + 1)
            anc.append(anc[p] | (1 << i))
    return depth, anc


def greedy_argmax(logits: np.ndarray) -> np.ndarray:
    """Per-row argmax, lowest index on ties; NaN rows are an error."""
    if np.isnan(logits).any():
        raise FloatingPointError("NaN logits")
    return np.argmax(logits, axis=1).astype(np.int64)


def accept_greedy(logits: np.ndarray, parents: Sequence[int], tokens: Sequence[int]) -> Tuple[List[int], int]:
    """Greedy tree verification: from the root, keep moving to the child whose
    token equals the target's argmax at the current node (lowest id if several).
    Returns the accepted node ids (root first) and the bonus token, the
    target's argmax at the last accepted node."""
    g = greedy_argmax(logits)
    children: Dict[int, List[int]] = {}
    for i, p in enumerate(parents):
        children.setdefault(p, []).append(i)
    path = [0]
    cur = 0
    while True:
        nxt = [c for c in children.get(cur, []) if int(tokens[c]) == int(g[cur])]
        if not nxt:
            break
        cur = nxt[0]
        path.append(cur)
    return path, int(g[cur])


def top_tokens(row: np.ndarray, b: int) -> List[int]:
    """The b highest-scoring tokens, ties to the lower index."""
    order = np.argsort(-row, kind="stable")
    return [int(x) for x in order[:b]]


def ar_decode(model: OracleModel, prompt: Sequence[int], n_new: int) -> List[int]:
    """Plain greedy autoregressive decoding: the losslessness reference."""
    model.set_committed(0)
    if len(prompt) > 1:
        model.prefill(list(prompt[:-1]))
    root = int(prompt[-1])
    out: List[int] = []
    while len(out) < n_new:
        lg = model.forward([root], [-1], 0)
        nxt = int(greedy_argmax(lg)[0])
        model.compact([0])
        out.append(nxt)
        root = nxt
    return out


def cas_decode_static(model: OracleModel, prompt: Sequence[int], n_new: int,
                      tree_parents: Sequence[int], level_of_depth: Dict[int, Tuple[Sequence[int], bool]],
                      stats: Optional[Dict] = None) -> List[int]:
    """Greedy speculative decoding with a static token tree filled depth by
    depth by draft levels (tree cascade: level_of_depth[d] = (skip mask,
    act_quant) drafts the tokens at depth d+1 from the nodes at depth d), then
    one full-depth verify of the whole tree, greedy acceptance and commit."""
    depth, _ = tree_metadata(tree_parents)
    T = len(tree_parents)
    max_d = max(depth)
    by_depth = [[i for i in range(T) if depth[i] == d] for d in range(max_d + 1)]
    children: Dict[int, List[int]] = {}
    for i, p in enumerate(tree_parents):
        children.setdefault(p, []).append(i)
    model.set_committed(0)
    if len(prompt) > 1:
        model.prefill(list(prompt[:-1]))
    root = int(prompt[-1])
    out: List[int] = []
    rounds = 0
    while len(out) < n_new:
        toks = np.zeros(T, dtype=np.int32)
        toks[0] = root
        for d in range(max_d):
            ids = by_depth[d]
            skip, aq = level_of_depth[d]
            lg = model.forward(toks[ids[0]:ids[-1] + 1], [tree_parents[i] for i in ids], ids[0],
                               skip=skip, act_quant=aq)
            for r, i in enumerate(ids):
                ch = children.get(i, [])
                for c, t in zip(ch, top_tokens(lg[r], len(ch))):
                    toks[c] = t
        lg = model.forward(toks, tree_parents, 0)
        path, bonus = accept_greedy(lg, tree_parents, toks)
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
