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

    def set_kv(self, layer: int, k: np.ndarray, v: np.ndarray) -> None:
        """k, v: [Hkv][n][hd] float32 (bf16 values), placed at slots 0..n-1."""
        s = self.s
        K = torch.zeros(s.n_kv_heads, self.max_ctx, s.head_dim)
        V = torch.zeros(s.n_kv_heads, self.max_ctx, s.head_dim)
        n = k.shape[1]
        K[:, :n] = torch.from_numpy(np.ascontiguousarray(k, dtype=np.float32))
        V[:, :n] = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
        self.K[layer], self.V[layer] = K, V

    def forward(self, tokens: Sequence[int], parents: Sequence[int],
                skip: Optional[Sequence[int]] = None) -> np.ndarray:
        """Verify-style forward of a whole round (node ids 0..n-1) -> fp32 logits [n][vocab]."""
        s = self.s
        n = len(tokens)
        d, H, Hkv, hd = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim
        G = H // Hkv
        kc = self.k_chunks
        depth = np.zeros(n, dtype=np.int64)
        anc = np.zeros((n, n), dtype=bool)
        for i, p in enumerate(parents):
            if p >= 0:
                depth[i] = depth[p] + 1
                anc[i] = anc[p]
            anc[i, i] = True
        pos = torch.from_numpy(self.Lc + depth)
        Lc = self.Lc
        # visibility of the Lc committed slots and the n tree slots
        vis = torch.ones(n, Lc + n, dtype=torch.bool)
        vis[:, Lc:] = torch.from_numpy(anc)
        neg = torch.zeros(n, Lc + n)
        neg[~vis] = float("-inf")
        h = _w(self.wts["embed"][np.asarray(tokens)]).clone()
        for l in range(s.n_layers):
            if skip is not None and skip[l]:
                continue
            lw = self.wts["layers"][l]
            x = _rmsnorm_bf16(h, torch.from_numpy(np.asarray(lw["attn_norm"], np.float32)), s.rms_eps)
            q = _mm(x, _w(lw["wq"]), kc).view(n, H, hd)
            k = _mm(x, _w(lw["wk"]), kc).view(n, Hkv, hd)
            v = _mm(x, _w(lw["wv"]), kc).view(n, Hkv, hd)
            q = _bf16(_rope(q, pos, s.rope_theta))
            k = _bf16(_rope(k, pos, s.rope_theta))
            v = _bf16(v)
            self.K[l][:, Lc:Lc + n] = k.transpose(0, 1)
            self.V[l][:, Lc:Lc + n] = v.transpose(0, 1)
            Kl = self.K[l][:, :Lc + n]            # [Hkv][Lc+n][hd]
            Vl = self.V[l][:, :Lc + n]
            o = torch.empty(n, H, hd)
            for kh in range(Hkv):
                qh = q[:, kh * G:(kh + 1) * G, :].transpose(0, 1)      # [G][n][hd]
                sc = (qh @ Kl[kh].T) * np.float32(1.0 / np.sqrt(hd)) + neg
                p = torch.softmax(sc, dim=-1)
                o[:, kh * G:(kh + 1) * G, :] = (p @ Vl[kh]).transpose(0, 1)
            o = _bf16(o.reshape(n, H * hd))
            h = h + _mm(o, _w(lw["wo"]), kc)
            x = _rmsnorm_bf16(h, torch.from_numpy(np.asarray(lw["ffn_norm"], np.float32)), s.rms_eps)
            g = _mm(x, _w(lw["w_gate"]), kc)
            u = _mm(x, _w(lw["w_up"]), kc)
            a = _bf16(torch.nn.functional.silu(g) * u)
            h = h + _mm(a, _w(lw["w_down"]), kc)
        x = _rmsnorm_bf16(h, torch.from_numpy(np.asarray(self.wts["final_norm"], np.float32)), s.rms_eps)
        return _mm(x, _w(self.wts["lm_head"]), kc).numpy()
