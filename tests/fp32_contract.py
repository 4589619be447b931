"""An fp32 implementation of the bf16 numerics contract of the decoder step,
written independently of the fp64 oracle and of the HIP library.

It exists to measure how far ANY correct fp32 implementation of the contract
lands from the fp64 oracle at full depth, which is what the tolerance of the
full-depth bf16 parity tests has to cover.  It imports nothing from `oracle/`
or from the HIP path; only the seeded inputs come from `synth`.

The contract (bf16 models): weights bf16; residual stream fp32; the inputs of
every linear layer (the RMSNorm outputs, the attention output, the SwiGLU
output) rounded to bf16; q, k and v rounded to bf16 after RoPE (the KV cache
is bf16); products accumulate in fp32; scores, softmax and logits in fp32.
The decoder is Llama-style: RMSNorm with eps inside the square root, rotate-
half RoPE at position committed-length + depth with inv_freq_i =
theta^(-2i/hd) (the angles in fp64, cos and sin rounded once to fp32), GQA
head h -> kv head h / (H / Hkv), SwiGLU, no biases.  A tree node attends to
every committed slot and to its ancestors and itself (tree attention,
Sec. 4.2); a skipped layer is the identity on the residual (layer sparsity,
Sec. 4.1).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np
import torch


def _bf16(x: torch.Tensor) -> torch.Tensor:
    """Round fp32 to the nearest bf16 value (ties to even), kept as fp32."""
    return x.to(torch.bfloat16).to(torch.float32)


def _w(bits: np.ndarray) -> torch.Tensor:
    """bf16 bit patterns -> fp32 tensor (exact)."""
    return torch.from_numpy((np.ascontiguousarray(bits).astype(np.uint32) << 16).view(np.float32))


def _rmsnorm_bf16(h: torch.Tensor, g: torch.Tensor, eps: float) -> torch.Tensor:
    ms = (h * h).mean(dim=1, keepdim=True)
    return _bf16(h * torch.rsqrt(ms + eps) * g)


def _rope(x: torch.Tensor, pos: torch.Tensor, theta: float) -> torch.Tensor:
    """x: [n][heads][hd]; rotate-half at per-row positions."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = pos.numpy().astype(np.float64)[:, None] * inv[None, :]
    c = torch.from_numpy(np.cos(ang).astype(np.float32))[:, None, :]
    s = torch.from_numpy(np.sin(ang).astype(np.float32))[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return torch.cat([a * c - b * s, a * s + b * c], dim=-1)


def _mm(x: torch.Tensor, w: torch.Tensor, k_chunks: int) -> torch.Tensor:
    """x @ w.T in fp32.  k_chunks > 1 sums that many contiguous K ranges in
    order, each a separate fp32 product: another valid fp32 summation order."""
    if k_chunks <= 1:
        return x @ w.T
    K = x.shape[1]
    step = -(-K // k_chunks)
    y = None
    for k0 in range(0, K, step):
        part = x[:, k0:k0 + step] @ w[:, k0:k0 + step].T
        y = part if y is None else y + part
    return y


def _quant_rows(x: torch.Tensor, qmax: int):
    """Per-row symmetric codes in [-qmax, qmax]: s = amax / qmax (fp32),
    q = clamp(round-half-even(x / s)); a zero row gives s = 0, q = 0."""
    amax = x.abs().amax(dim=1, keepdim=True)
    s = amax / np.float32(qmax)
    safe = torch.where(s == 0, torch.ones_like(s), s)
    q = torch.clamp(torch.round(x / safe), -qmax, qmax)
    q = torch.where(s == 0, torch.zeros_like(q), q)
    return q, s


def _qlinear(x: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor, qmax: int) -> torch.Tensor:
    """Quantised-activation linear layer: exact integer sums (fp64 products of
    small integers), then y = (fp32(acc) * s_x) * s_w in fp32."""
    q, s = _quant_rows(x, qmax)
    acc = (q.double() @ qw.double().T).float()
    return (acc * s) * sw[None, :]


class Fp32ContractModel:
    """A bf16-weight decoder with an fp32 KV cache holding bf16 values.

    k_chunks selects the fp32 summation order of the linear layers (1: one
    library product; n: n K ranges summed in order)."""

    def __init__(self, shape, weights: Dict, max_ctx: int, k_chunks: int = 1):
        if shape.dtype != "bf16":
            raise ValueError("the contract emulated here is the bf16 one")
        self.s = shape
        self.wts = weights
        self.max_ctx = max_ctx
        self.K = [None] * shape.n_layers   # [Hkv][max_ctx][hd] fp32
        self.V = [None] * shape.n_layers
        self.Lc = 0
        self.k_chunks = k_chunks
        self.qcopy = {}           # (layer, tensor, qmax) -> (codes, scales)
        self.round = None         # the open round: parents, depths, ancestor sets

    def set_kv(self, layer: int, k: np.ndarray, v: np.ndarray) -> None:
        """k, v: [Hkv][n][hd] float32 (bf16 values), placed at slots 0..n-1."""
        s = self.s
        K = torch.zeros(s.n_kv_heads, self.max_ctx, s.head_dim)
        V = torch.zeros(s.n_kv_heads, self.max_ctx, s.head_dim)
        n = k.shape[1]
        K[:, :n] = torch.from_numpy(np.ascontiguousarray(k, dtype=np.float32))
        V[:, :n] = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
        self.K[layer], self.V[layer] = K, V

    def _qweight(self, l: int, name: str, qmax: int):
        key = (l, name, qmax)
        if key not in self.qcopy:
            w = _w(self.wts["layers"][l][name])
            s = w.abs().amax(dim=1) / np.float32(qmax)
            safe = torch.where(s == 0, torch.ones_like(s), s)
            q = torch.clamp(torch.round(w / safe[:, None]), -qmax, qmax)
            q = torch.where(s[:, None] == 0, torch.zeros_like(q), q)
            self.qcopy[key] = (q.to(torch.int8), s)
        return self.qcopy[key]

    def prefill(self, tokens: Sequence[int]) -> None:
        """Commit tokens as a causal chain after the committed prefix."""
        n = len(tokens)
        self.forward(tokens, [-1] + list(range(n - 1)))
        self.Lc += n
        self.round = None

    def forward(self, tokens: Sequence[int], parents: Sequence[int], node_offset: int = 0,
                skip: Optional[Sequence[int]] = None, act_quant: int = 0,
                window: Optional[Sequence[int]] = None) -> np.ndarray:
        """Forward over the nodes node_offset .. node_offset+n-1 of the round
        (node_offset 0 opens a new round; parents are round node ids) ->
        fp32 logits [n][vocab].  act_quant 1 / 2: per-token int8 / int4
        codes for the seven linear layers of every layer that runs, against
        per-output-channel copies of the weights (the LM head, attention and
        KV cache keep bf16).  window = (sink, window): of the committed slots
        only the first sink and the last window are visible."""
        s = self.s
        n = len(tokens)
        d, H, Hkv, hd = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim
        G = H // Hkv
        kc = self.k_chunks
        if node_offset == 0:
            self.round = {"depth": [], "anc": []}
        rd = self.round
        for i, p in enumerate(parents):
            node = node_offset + i
            if p < 0:
                rd["depth"].append(0)
                rd["anc"].append({node})
            else:
                rd["depth"].append(rd["depth"][p] + 1)
                rd["anc"].append(rd["anc"][p] | {node})
        depth = np.array(rd["depth"][node_offset:node_offset + n], dtype=np.int64)
        pos = torch.from_numpy(self.Lc + depth)
        Lc = self.Lc
        nk = node_offset + n                      # round slots that exist now
        vis = torch.zeros(n, Lc + nk, dtype=torch.bool)
        if window and window[1] > 0:
            sink, win = window
            vis[:, :min(sink, Lc)] = True
            vis[:, max(Lc - win, min(sink, Lc)):Lc] = True
        else:
            vis[:, :Lc] = True
        for i in range(n):
            for a in rd["anc"][node_offset + i]:
                vis[i, Lc + a] = True
        neg = torch.zeros(n, Lc + nk)
        neg[~vis] = float("-inf")
        qmax = {1: 127, 2: 7}.get(int(act_quant), 0)

        def lin(x, l, name):
            if qmax:
                qw, sw = self._qweight(l, name, qmax)
                return _qlinear(x, qw, sw, qmax)
            return _mm(x, _w(self.wts["layers"][l][name]), kc)

        h = _w(self.wts["embed"][np.asarray(tokens)]).clone()
        for l in range(s.n_layers):
            if skip is not None and skip[l]:
                continue
            lw = self.wts["layers"][l]
            x = _rmsnorm_bf16(h, torch.from_numpy(np.asarray(lw["attn_norm"], np.float32)), s.rms_eps)
            q = lin(x, l, "wq").view(n, H, hd)
            k = lin(x, l, "wk").view(n, Hkv, hd)
            v = lin(x, l, "wv").view(n, Hkv, hd)
            q = _bf16(_rope(q, pos, s.rope_theta))
            k = _bf16(_rope(k, pos, s.rope_theta))
            v = _bf16(v)
            self.K[l][:, Lc + node_offset:Lc + nk] = k.transpose(0, 1)
            self.V[l][:, Lc + node_offset:Lc + nk] = v.transpose(0, 1)
            Kl = self.K[l][:, :Lc + nk]
            Vl = self.V[l][:, :Lc + nk]
            o = torch.empty(n, H, hd)
            for kh in range(Hkv):
                qh = q[:, kh * G:(kh + 1) * G, :].transpose(0, 1)
                sc = (qh @ Kl[kh].T) * np.float32(1.0 / np.sqrt(hd)) + neg
                p = torch.softmax(sc, dim=-1)
                o[:, kh * G:(kh + 1) * G, :] = (p @ Vl[kh]).transpose(0, 1)
            o = _bf16(o.reshape(n, H * hd))
            h = h + lin(o, l, "wo")
            x = _rmsnorm_bf16(h, torch.from_numpy(np.asarray(lw["ffn_norm"], np.float32)), s.rms_eps)
            g = lin(x, l, "w_gate")
            u = lin(x, l, "w_up")
            a = _bf16(torch.nn.functional.silu(g) * u)
            h = h + lin(a, l, "w_down")
        x = _rmsnorm_bf16(h, torch.from_numpy(np.asarray(self.wts["final_norm"], np.float32)), s.rms_eps)
        return _mm(x, _w(self.wts["lm_head"]), kc).numpy()
