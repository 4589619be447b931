"""ctypes binding of libcas.so (include/cas.h, include/cas_ops.h).

Argument marshalling only: every step of the decoder forward, acceptance and
compaction runs in the library's HIP kernels.  The binding refuses to run
without the built library; there is no fallback of any kind.

Environment switches read when a Model is created:
- CAS_DEBUG=1: use libcas_debug.so, the build with device checks (failed
  checks surface as CAS_ERR_DEVICE from the synchronising calls);
- CAS_PROFILE=1: launch kernel by kernel with per-kernel event timing, and
  print the per-kernel-class totals to stderr when the Model is closed.
"""
from __future__ import annotations

import ctypes
import os
import sys
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcas.so")
LIB_DEBUG_PATH = os.path.join(_PKG, "libcas_debug.so")
_lib = None
_lib_debug = None

# status codes (cas_status)
OK, ERR_ARG, ERR_TREE, ERR_CAPACITY, ERR_UNSUPPORTED, ERR_OOM, ERR_DEVICE, ERR_STATE = range(8)
STATUS_NAMES = ["CAS_OK", "CAS_ERR_ARG", "CAS_ERR_TREE", "CAS_ERR_CAPACITY", "CAS_ERR_UNSUPPORTED",
                "CAS_ERR_OOM", "CAS_ERR_DEVICE", "CAS_ERR_STATE"]
F32, BF16 = 0, 1
W_F32, W_BF16, W_I8, W_I4 = 0, 1, 2, 3
EPI_STORE, EPI_RESID, EPI_RAW_I32 = 0, 1, 2
TENSOR = {"embed": 0, "lm_head": 1, "final_norm": 2, "attn_norm": 3, "ffn_norm": 4, "wq": 5, "wk": 6,
          "wv": 7, "wo": 8, "w_gate": 9, "w_up": 10, "w_down": 11}
KCLASS = ["embed", "rmsnorm", "gemm_qkv", "attn", "gemm_o", "gemm_gateup", "gemm_down", "gemm_head", "quant",
          "accept", "compact", "topk"]

# every symbol the two headers declare
EXPORTS = ("cas_create", "cas_destroy", "cas_last_error", "cas_create_error", "cas_load_tensor", "cas_build_int8",
           "cas_build_int4",
           "cas_prefill", "cas_kv_load", "cas_kv_read", "cas_set_committed", "cas_committed_len", "cas_forward",
           "cas_logits_device", "cas_forward_draft", "cas_accept_tree", "cas_topk", "cas_kv_compact", "cas_tree_info", "cas_set_graphs",
           "cas_profile", "cas_profile_read", "cas_sync", "cas_op_gemm", "cas_op_gemm_work_bytes",
           "cas_op_quant_rows", "cas_op_quant_rows_q", "cas_op_quant_weight", "cas_op_quant_weight_i4",
           "cas_op_quant_weight_work_bytes", "cas_op_attention",
           "cas_op_attention_work_bytes", "cas_op_copy", "cas_op_rmsnorm", "cas_op_rmsnorm_work_bytes",
           "cas_op_attn_merge", "cas_op_attn_merge_work_bytes", "cas_op_gemm_qx", "cas_op_gemm_qx_splits",
           "cas_op_gemm_qx_work_bytes", "cas_op_attention_noalloc", "cas_op_attention_noalloc_max_bytes",
           "cas_debug_build", "cas_debug_check", "cas_debug_limit_slots", "cas_set_gemv")
# device check codes (cas_debug_check)
DEVICE_CHECKS = ["none", "tree size", "token id", "parent order", "slot capacity", "RoPE position",
                 "KV write slot", "attention slots", "compaction path", "acceptance parent"]


class CasError(RuntimeError):
    def __init__(self, status: int, msg: str):
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"{name}: {msg}")
        self.status = status


class DraftOpts(ctypes.Structure):
    _fields_ = [("skip_mask", ctypes.c_void_p), ("act_quant", ctypes.c_int32), ("attn_sink", ctypes.c_int32),
                ("attn_window", ctypes.c_int32)]


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("max_ctx", ctypes.c_int32), ("max_tree", ctypes.c_int32)]


def lib(debug: bool = False):
    """Load libcas.so (debug: libcas_debug.so, the build with device checks);
    raises if it has not been built."""
    global _lib, _lib_debug
    if (_lib_debug if debug else _lib) is None:
        path = LIB_DEBUG_PATH if debug else LIB_PATH
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(path)
        P, I, Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        sig = {
            "cas_create": ([P, ctypes.c_int, P, P], I),
            "cas_destroy": ([P], None),
            "cas_last_error": ([P], ctypes.c_char_p),
            "cas_create_error": ([], ctypes.c_char_p),
            "cas_load_tensor": ([P, I, I, P, Z], I),
            "cas_build_int8": ([P], I),
            "cas_build_int4": ([P], I),
            "cas_prefill": ([P, P, I], I),
            "cas_kv_load": ([P, I, P, P, I], I),
            "cas_kv_read": ([P, I, P, P, I], I),
            "cas_set_committed": ([P, I], I),
            "cas_committed_len": ([P, P], I),
            "cas_forward": ([P, P, P, I, I, P, I, P], I),
            "cas_logits_device": ([P, P, P], I),
            "cas_accept_tree": ([P, I, P, P, P], I),
            "cas_kv_compact": ([P, P, I], I),
            "cas_forward_draft": ([P, P, P, I, I, P, P], I),
            "cas_topk": ([P, I, I, P, P], I),
            "cas_tree_info": ([P, I, P, P], I),
            "cas_set_graphs": ([P, I], I),
            "cas_set_gemv": ([P, I], I),
            "cas_profile": ([P, I], I),
            "cas_profile_read": ([P, P, P, I], I),
            "cas_sync": ([P], I),
            "cas_op_gemm": ([I, P, P, I, I, I, P, P, I, P, I, P, Z, P], I),
            "cas_op_gemm_work_bytes": ([I, I, I, I], Z),
            "cas_op_quant_rows": ([I, P, I, I, P, P, P], I),
            "cas_op_quant_rows_q": ([I, P, I, I, I, P, P, P], I),
            "cas_op_quant_weight": ([I, P, I, I, P, P, P, Z, P], I),
            "cas_op_quant_weight_i4": ([I, P, I, I, P, P, P, Z, P], I),
            "cas_op_quant_weight_work_bytes": ([I, I, I], Z),
            "cas_op_attention": ([P, P, P, I, I, I, I, I, I, I, P, P, P, Z, P], I),
            "cas_op_attention_work_bytes": ([I, I, I, I, I, I, I], Z),
            "cas_op_copy": ([P, P, Z, P], I),
            "cas_op_rmsnorm": ([I, P, P, I, I, ctypes.c_float, P, I, I, P, P, P, P, Z, P], I),
            "cas_op_rmsnorm_work_bytes": ([I, I, I, I], Z),
            "cas_op_attn_merge": ([P, P, I, I, I, I, I, P, P, P, P, Z, P], I),
            "cas_op_attn_merge_work_bytes": ([I, I, I, I], Z),
            "cas_op_gemm_qx": ([I, P, P, P, I, I, I, I, P, P, Z, P], I),
            "cas_op_gemm_qx_splits": ([I, I, I, I], I),
            "cas_op_gemm_qx_work_bytes": ([I, I, I, I], Z),
            "cas_op_attention_noalloc": ([P, P, P, I, I, I, I, I, I, I, P, P, P], I),
            "cas_op_attention_noalloc_max_bytes": ([], Z),
            "cas_debug_build": ([], I),
            "cas_debug_check": ([P, P], I),
            "cas_debug_limit_slots": ([P, I], I),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        if debug:
            _lib_debug = L
        else:
            _lib = L
    return _lib_debug if debug else _lib


def _p(a: np.ndarray) -> int:
    return a.ctypes.data


def tree_info(parents: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Depth and 128-bit ancestor-or-self masks ([n][2] uint64) as the library computes them."""
    par = np.ascontiguousarray(parents, dtype=np.int32)
    n = par.shape[0]
    depth = np.zeros(n, dtype=np.int32)
    anc = np.zeros((n, 2), dtype=np.uint64)
    st = lib().cas_tree_info(_p(par), n, _p(depth), _p(anc))
    if st:
        raise CasError(st, "invalid parent list")
    return depth, anc


class Model:
    """One decoder context (weights, KV cache, round state) on one GPU."""

    def __init__(self, shape, max_ctx: int, max_tree: int = 128, device: int = 0, stream: Optional[int] = None,
                 debug: Optional[bool] = None):
        """debug: use the build with device checks (default: the CAS_DEBUG
        environment switch)."""
        if debug is None:
            debug = os.environ.get("CAS_DEBUG", "0") == "1"
        self.debug = bool(debug)
        self._L = lib(self.debug)
        self.shape = shape
        self.bf16 = shape.dtype == "bf16"
        cfg = Config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim,
                     shape.vocab, float(shape.rope_theta), float(shape.rms_eps), BF16 if self.bf16 else F32,
                     int(max_ctx), int(max_tree))
        self.max_ctx, self.max_tree = int(max_ctx), int(max_tree)
        h = ctypes.c_void_p()
        st = self._L.cas_create(ctypes.byref(cfg), int(device), stream, ctypes.byref(h))
        if st:
            raise CasError(st, self._L.cas_create_error().decode())
        self.h = h.value
        self._acc = np.zeros(self.max_tree, dtype=np.int32)
        self._print_profile = os.environ.get("CAS_PROFILE", "0") == "1"
        if self._print_profile:
            self.profile(True)

    def close(self) -> None:
        if getattr(self, "h", None):
            if getattr(self, "_print_profile", False):
                self._print_profile = False
                self.print_profile()
            self._L.cas_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _chk(self, st: int) -> None:
        if st:
            raise CasError(st, self._L.cas_last_error(self.h).decode())

    # weights ------------------------------------------------------------------
    def load_tensor(self, name: str, layer: int, arr: np.ndarray) -> None:
        a = np.ascontiguousarray(arr)
        self._chk(self._L.cas_load_tensor(self.h, TENSOR[name], int(layer), _p(a), a.nbytes))

    def load_weights(self, w: Dict, layers: Optional[Sequence[int]] = None) -> None:
        self.load_tensor("embed", 0, w["embed"])
        self.load_tensor("lm_head", 0, w["lm_head"])
        self.load_tensor("final_norm", 0, np.asarray(w["final_norm"], dtype=np.float32))
        for l, lw in enumerate(w["layers"]):
            if lw is None or (layers is not None and l not in layers):
                continue
            for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
                self.load_tensor(n, l, lw[n])
            self.load_tensor("attn_norm", l, np.asarray(lw["attn_norm"], dtype=np.float32))
            self.load_tensor("ffn_norm", l, np.asarray(lw["ffn_norm"], dtype=np.float32))

    def build_int8(self) -> None:
        self._chk(self._L.cas_build_int8(self.h))

    def build_int4(self) -> None:
        """The int4 weight copy behind act_quant = 2 (W4A4 drafts)."""
        self._chk(self._L.cas_build_int4(self.h))

    # state ----------------------------------------------------------------------
    @property
    def committed(self) -> int:
        n = ctypes.c_int32()
        self._chk(self._L.cas_committed_len(self.h, ctypes.byref(n)))
        return n.value

    def set_committed(self, n: int) -> None:
        self._chk(self._L.cas_set_committed(self.h, int(n)))

    def kv_load(self, layer: int, k: np.ndarray, v: np.ndarray) -> None:
        """Committed KV of one layer, [n_kv_heads][n][head_dim] in the storage type."""
        k = np.ascontiguousarray(k)
        v = np.ascontiguousarray(v)
        self._chk(self._L.cas_kv_load(self.h, int(layer), _p(k), _p(v), int(k.shape[1])))

    def kv_read(self, layer: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
        """KV slots 0..n-1 of one layer as [n_kv_heads][n][head_dim] (bf16 bits or float32)."""
        dt = np.uint16 if self.bf16 else np.float32
        k = np.zeros((self.shape.n_kv_heads, n, self.shape.head_dim), dtype=dt)
        v = np.zeros_like(k)
        self._chk(self._L.cas_kv_read(self.h, int(layer), _p(k), _p(v), int(n)))
        return k, v

    def prefill(self, tokens: Sequence[int]) -> None:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        self._chk(self._L.cas_prefill(self.h, _p(t), t.shape[0]))

    # the step -------------------------------------------------------------------
    def forward(self, tokens: Sequence[int], parents: Sequence[int], node_offset: int = 0,
                skip: Optional[Sequence[int]] = None, act_quant: int = 0,
                logits: bool = True, attn_window: Optional[Tuple[int, int]] = None) -> Optional[np.ndarray]:
        """act_quant: 0, 1 (or True) = W8A8, 2 = W4A4.  attn_window = (sink,
        window): efficient-attention draft."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        p = np.ascontiguousarray(parents, dtype=np.int32)
        n = t.shape[0]
        if p.shape[0] != n:
            raise ValueError("tokens and parents differ in length")
        sk = None
        if skip is not None:
            sk = np.ascontiguousarray(skip, dtype=np.uint8)  # the library validates the values
            if sk.shape[0] != self.shape.n_layers:
                raise ValueError("skip mask length")
        out = np.empty((n, self.shape.vocab), dtype=np.float32) if logits else None
        if attn_window:
            o = DraftOpts(None if sk is None else _p(sk), int(act_quant), int(attn_window[0]),
                          int(attn_window[1]))
            self._chk(self._L.cas_forward_draft(self.h, _p(t), _p(p), n, int(node_offset), ctypes.byref(o),
                                              None if out is None else _p(out)))
        else:
            self._chk(self._L.cas_forward(self.h, _p(t), _p(p), n, int(node_offset), None if sk is None else _p(sk),
                                        int(act_quant), None if out is None else _p(out)))
        return out

    def logits_device(self) -> Tuple[int, int]:
        ptr = ctypes.c_void_p()
        n = ctypes.c_int32()
        self._chk(self._L.cas_logits_device(self.h, ctypes.byref(ptr), ctypes.byref(n)))
        return ptr.value, n.value

    def accept(self) -> Tuple[List[int], int]:
        n = ctypes.c_int32()
        b = ctypes.c_int32()
        self._chk(self._L.cas_accept_tree(self.h, 1, _p(self._acc), ctypes.byref(n), ctypes.byref(b)))
        return [int(x) for x in self._acc[: n.value]], int(b.value)

    def topk(self, K: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
        """Top-K token ids and their softmax probabilities for the n rows of
        the last forward ([n][K] int32 and float32)."""
        ids = np.zeros((n, K), dtype=np.int32)
        probs = np.zeros((n, K), dtype=np.float32)
        self._chk(self._L.cas_topk(self.h, int(n), int(K), _p(ids), _p(probs)))
        return ids, probs

    def compact(self, accepted: Sequence[int]) -> None:
        a = np.ascontiguousarray(accepted, dtype=np.int32)
        self._chk(self._L.cas_kv_compact(self.h, _p(a), a.shape[0]))

    def sync(self) -> None:
        self._chk(self._L.cas_sync(self.h))

    def set_graphs(self, on: bool) -> None:
        self._chk(self._L.cas_set_graphs(self.h, 1 if on else 0))

    def set_gemv(self, on: bool) -> None:
        """GEMV-style tiles for one-row drafts (default off: the MFMA tiles,
        whose rows carry the verify's bits)."""
        self._chk(self._L.cas_set_gemv(self.h, 1 if on else 0))

    def profile(self, on: bool) -> None:
        self._chk(self._L.cas_profile(self.h, 1 if on else 0))

    def profile_read(self, reset: bool = True) -> Dict[str, Tuple[float, int]]:
        ms = np.zeros(len(KCLASS), dtype=np.float64)
        cnt = np.zeros(len(KCLASS), dtype=np.int32)
        self._chk(self._L.cas_profile_read(self.h, _p(ms), _p(cnt), 1 if reset else 0))
        return {k: (float(ms[i]), int(cnt[i])) for i, k in enumerate(KCLASS)}

    def print_profile(self, file=None) -> None:
        """Per-kernel-class totals since the last read, as a table."""
        rows = [(k, ms, n) for k, (ms, n) in self.profile_read(reset=True).items() if n]
        out = file or sys.stderr
        total = sum(ms for _, ms, _ in rows)
        print(f"{'kernel class':<14}{'launches':>10}{'ms':>12}{'us/launch':>12}{'share':>8}", file=out)
        for k, ms, n in sorted(rows, key=lambda r: -r[1]):
            print(f"{k:<14}{n:>10}{ms:>12.3f}{1e3 * ms / n:>12.2f}{ms / total if total else 0:>8.1%}", file=out)

    # device checks (CAS_DEBUG build) --------------------------------------------
    def debug_check(self) -> int:
        """Synchronise and return the code of a failed device check since the
        last read (0: none; always 0 in the release build), clearing it."""
        code = ctypes.c_int32()
        self._chk(self._L.cas_debug_check(self.h, ctypes.byref(code)))
        return code.value

    def debug_limit_slots(self, cap: int) -> None:
        """Make the device checks allow only KV slots < cap (0: the whole
        cache).  Debug build only."""
        self._chk(self._L.cas_debug_limit_slots(self.h, int(cap)))


# ----------------------------------------------------------------------------
# kernel-level entry points on device tensors (torch tensors on a HIP device)
# ----------------------------------------------------------------------------

def _dp(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    return int(stream)


def _ochk(st: int, what: str) -> None:
    if st:
        raise CasError(st, what)


def _work(nbytes: int):
    import torch
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device="cuda")


def op_gemm(wtype: int, W, X, N: int, K: int, T: int, out, ldo: int, epi: int = EPI_STORE,
            xs=None, ws=None, stream=None, work=None) -> None:
    need = int(lib().cas_op_gemm_work_bytes(wtype, N, K, T))
    work = _work(need) if work is None else work
    _ochk(lib().cas_op_gemm(wtype, _dp(W), _dp(X), N, K, T, _dp(xs), _dp(ws), epi, _dp(out), ldo, _dp(work),
                            int(work.numel() * work.element_size()), _stream(stream)), "cas_op_gemm")


def op_quant_rows(atype: int, x, T: int, K: int, q, s, stream=None, qmax: int = 127) -> None:
    if qmax == 127:
        _ochk(lib().cas_op_quant_rows(atype, _dp(x), T, K, _dp(q), _dp(s), _stream(stream)), "cas_op_quant_rows")
    else:
        _ochk(lib().cas_op_quant_rows_q(atype, _dp(x), T, K, int(qmax), _dp(q), _dp(s), _stream(stream)),
              "cas_op_quant_rows_q")


def op_quant_weight(wtype: int, W, N: int, K: int, q, s, stream=None, qmax: int = 127) -> None:
    """Per-output-channel copy of W; qmax 127 (int8) or 7 (int4, packed by the
    library and returned unpacked)."""
    work = _work(lib().cas_op_quant_weight_work_bytes(wtype, N, K))
    fn = lib().cas_op_quant_weight if qmax == 127 else lib().cas_op_quant_weight_i4
    _ochk(fn(wtype, _dp(W), N, K, _dp(q), _dp(s), _dp(work), int(work.numel()), _stream(stream)),
          "cas_op_quant_weight" if qmax == 127 else "cas_op_quant_weight_i4")


def op_attention(q, k, v, ctx_cap: int, Lc: int, n_tree: int, T: int, H: int, Hkv: int, hd: int, anc, out,
                 stream=None) -> None:
    """k, v: [Hkv][ctx_cap][hd] bf16 row-major device tensors."""
    work = _work(lib().cas_op_attention_work_bytes(Lc, n_tree, T, H, hd, Hkv, ctx_cap))
    _ochk(lib().cas_op_attention(_dp(q), _dp(k), _dp(v), ctx_cap, Lc, n_tree, T, H, Hkv, hd, _dp(anc), _dp(out),
                                 _dp(work), int(work.numel()), _stream(stream)), "cas_op_attention")


def op_attention_noalloc(q, k, v, ctx_cap: int, Lc: int, n_tree: int, T: int, H: int, Hkv: int, hd: int, anc,
                         out, stream=None) -> int:
    """op_attention on the library's own scratch (no device allocation);
    returns the status (CAS_ERR_CAPACITY beyond the scratch size)."""
    return int(lib().cas_op_attention_noalloc(_dp(q), _dp(k), _dp(v), ctx_cap, Lc, n_tree, T, H, Hkv, hd, _dp(anc),
                                              _dp(out), _stream(stream)))


def op_copy(dst, src, nbytes: int, stream=None) -> None:
    _ochk(lib().cas_op_copy(_dp(dst), _dp(src), nbytes, _stream(stream)), "cas_op_copy")


def op_rmsnorm(atype: int, h, gain, T: int, d: int, eps: float, out=None, q=None, qs=None, parts=None,
               nparts: int = 0, qmax: int = 0, stream=None) -> None:
    """RMSNorm of the residual rows h [T][d] (updated in place by pending
    split-K sums when nparts > 0): the normalised rows in the model type
    (qmax 0) or their per-token codes and scales (qmax 127 or 7)."""
    work = _work(lib().cas_op_rmsnorm_work_bytes(atype, T, d, qmax))
    _ochk(lib().cas_op_rmsnorm(atype, _dp(h), _dp(gain), T, d, float(eps), _dp(parts), int(nparts), int(qmax),
                               _dp(out), _dp(q), _dp(qs), _dp(work), int(work.numel()), _stream(stream)),
          "cas_op_rmsnorm")


def op_attn_merge(part_o, part_ml, S: int, T: int, H: int, hd: int, out=None, q=None, qs=None, qmax: int = 0,
                  stream=None) -> None:
    """Merge of S attention split partials into bf16 rows (qmax 0) or their
    per-token codes and scales (qmax 127 or 7)."""
    work = _work(lib().cas_op_attn_merge_work_bytes(T, H, hd, qmax))
    _ochk(lib().cas_op_attn_merge(_dp(part_o), _dp(part_ml), S, T, H, hd, int(qmax), _dp(out), _dp(q), _dp(qs),
                                  _dp(work), int(work.numel()), _stream(stream)), "cas_op_attn_merge")


def op_gemm_qx_splits(wtype: int, N: int, K: int, T: int) -> int:
    return int(lib().cas_op_gemm_qx_splits(wtype, N, K, T))


def op_gemm_qx(wtype: int, W, ws, x, N: int, K: int, T: int, qmax: int, parts, stream=None) -> None:
    """Split-K integer projection that quantises its bf16 rows on load; parts
    [splits][T][N] fp32 receives each split's dequantised sums."""
    work = _work(lib().cas_op_gemm_qx_work_bytes(wtype, N, K, T))
    _ochk(lib().cas_op_gemm_qx(wtype, _dp(W), _dp(ws), _dp(x), N, K, T, int(qmax), _dp(parts), _dp(work),
                               int(work.numel()), _stream(stream)), "cas_op_gemm_qx")
