"""Kernel-level parity of the HIP library against the CPU oracle, through the
C ABI (include/cas_ops.h), on identical seeded inputs.

Bars: int8 and int4 codes, scales and integer accumulators bit-exact; the fp32/bf16
GEMM within the rigorous fp32 summation bound K * 2^-23 * sum_k |x_k w_k|; the
bf16 attention output within half a bf16 step of the fp64 value (2^-8 |ref|,
the output's own rounding) plus 4e-5 of max |v| (the two-term bf16
probabilities of the PV product, 2^-17 relative per weight, and fp32 sums).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2510_26843_amd import cas, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _bf16_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV)


def _f32_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def _i8_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int8)).to(DEV)


def _gemm_bound(x64, w64):
    K = x64.shape[1]
    return K * 2.0 ** -23 * (np.abs(x64) @ np.abs(w64).T) + 1e-30


# N >= 8192 with N/16 a multiple of 3 or 4 takes the multi-tile workgroup
# variant: 4 waves x 1 tile (8192, 8256), 3 x 1 (8208, 12288), 4 x 2 (16512),
# 3 x 2 (24480); 8240 and smaller N split K inside a one-tile workgroup.  At
# any row count, a tile count whose equal split gives a workgroup more than
# six (seven) tiles spreads evenly over fewer than 256 workgroups of six
# (seven) one-tile waves (22016: 230 workgroups of 5-6 tiles; 27648: 247 of
# 6-7); 28672 keeps the equal split, as do the smaller matrices above
@pytest.mark.parametrize("N,K,T", [(64, 4096, 32), (48, 688, 5), (32, 256, 1), (16, 1376, 17), (64, 512, 128),
                                   (80, 11008, 64), (32, 128, 100), (8192, 512, 32), (8256, 256, 5),
                                   (8192, 384, 128), (8208, 256, 9), (8320, 128, 1), (16512, 256, 32),
                                   (16512, 128, 100), (12288, 256, 32), (24480, 128, 20), (8240, 128, 3),
                                   (22016, 256, 32), (27648, 128, 7), (28672, 128, 20), (22016, 256, 64),
                                   (22016, 128, 100), (27648, 128, 128),
                                   # one row: the GEMV-style tiles (4x1, 3x2, 3x1 and 4x2 workgroups)
                                   (16512, 256, 1), (12288, 512, 1), (22016, 4096, 1)])
def test_gemm_bf16(N, K, T):
    w = synth.f32_to_bf16_bits(synth.gen_activations(N, K, seed=N + K, edge_rows=False) * 0.02)
    x = synth.f32_to_bf16_bits(synth.gen_activations(T, K, seed=T + 7))
    out = torch.zeros((T, N), dtype=torch.float32, device=DEV)
    cas.op_gemm(cas.W_BF16, _bf16_dev(w), _bf16_dev(x), N, K, T, out, N)
    torch.cuda.synchronize()
    x64 = synth.bf16_bits_to_f32(x).astype(np.float64)
    w64 = synth.bf16_bits_to_f32(w).astype(np.float64)
    ref = O.matmul_rows(x64, w, bf16=True)
    got = out.cpu().numpy()
    assert (np.abs(got - ref) <= _gemm_bound(x64, w64)).all()


@pytest.mark.parametrize("N,K,T", [(32, 256, 15), (16, 688, 3), (2048, 256, 7), (64, 4096, 33), (8192, 256, 20),
                                   (8256, 128, 1), (16512, 128, 3)])
def test_gemm_f32_and_residual(N, K, T):
    w = synth.gen_activations(N, K, seed=11, edge_rows=False) * np.float32(0.02)
    x = synth.gen_activations(T, K, seed=12)
    base = synth.gen_activations(T, N, seed=13, edge_rows=False)
    out = _f32_dev(base)
    cas.op_gemm(cas.W_F32, _f32_dev(w), _f32_dev(x), N, K, T, out, N, epi=cas.EPI_RESID)
    torch.cuda.synchronize()
    ref = base.astype(np.float64) + O.matmul_rows(x, w, bf16=False)
    bound = _gemm_bound(x.astype(np.float64), w.astype(np.float64)) + np.abs(ref) * 2.0 ** -23
    assert (np.abs(out.cpu().numpy() - ref) <= bound).all()


@pytest.mark.parametrize("N,K,T", [(64, 4096, 32), (48, 688, 5), (16, 13824, 3), (32, 256, 100), (16, 5120, 64),
                                   (8192, 512, 32), (8256, 256, 1), (8192, 256, 65), (16512, 256, 17),
                                   (12288, 128, 5), (24480, 128, 33), (22016, 256, 17), (27648, 128, 32),
                                   (22016, 256, 40),
                                   # one row: the GEMV-style tiles (exact int32 dot4 sums)
                                   (16512, 256, 1), (12288, 512, 1), (22016, 4096, 1)])
def test_gemm_int8_bit_exact(N, K, T):
    rng = np.random.default_rng(N * 7 + K + T)
    qw = rng.integers(-127, 128, (N, K)).astype(np.int8)
    qx = rng.integers(-127, 128, (T, K)).astype(np.int8)
    qx[0, :] = 127
    qw[0, :] = 127  # largest accumulator magnitude
    if T > 1:
        qx[1, :] = 0
    acc = torch.zeros((T, N), dtype=torch.int32, device=DEV)
    cas.op_gemm(cas.W_I8, _i8_dev(qw), _i8_dev(qx), N, K, T, acc, N, epi=cas.EPI_RAW_I32)
    xs = (rng.random(T).astype(np.float32) + np.float32(0.01)) / np.float32(127)
    ws = (rng.random(N).astype(np.float32) + np.float32(0.01)) / np.float32(127)
    y = torch.zeros((T, N), dtype=torch.float32, device=DEV)
    cas.op_gemm(cas.W_I8, _i8_dev(qw), _i8_dev(qx), N, K, T, y, N, epi=cas.EPI_STORE, xs=_f32_dev(xs), ws=_f32_dev(ws))
    torch.cuda.synchronize()
    ref = O.dot_i8_matrix(qx, qw)
    assert np.array_equal(acc.cpu().numpy(), ref)
    # dequantisation in fp32: (float(acc) * s_x) * s_w
    want = (ref.astype(np.float32) * xs[:, None]).astype(np.float32) * ws[None, :]
    assert np.array_equal(y.cpu().numpy().view(np.uint32), want.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("N,K,T", [(64, 4096, 32), (48, 688, 5), (16, 13824, 3), (32, 256, 100), (16, 5120, 64),
                                   (8192, 512, 32), (8256, 256, 1), (8192, 256, 65), (16512, 256, 17),
                                   (12288, 128, 5), (24480, 128, 33), (64, 272, 128), (8208, 4096, 1)])
def test_gemm_int4_bit_exact(N, K, T):
    """Packed int4 weights (codes in [-7, 7]) against int8-held int4
    activation codes: exact int32 accumulators on every kernel path (one-tile
    workgroups, multi-tile, all column-tile counts, K not a multiple of the
    256-wide chunk), and the fp32 dequantisation."""
    rng = np.random.default_rng(N * 5 + K + T)
    qw = rng.integers(-7, 8, (N, K)).astype(np.int8)
    qx = rng.integers(-7, 8, (T, K)).astype(np.int8)
    qx[0, :] = -7
    qw[0, :] = 7  # largest accumulator magnitude
    qw[1, ::2] = -7
    if T > 1:
        qx[1, :] = 0
    acc = torch.zeros((T, N), dtype=torch.int32, device=DEV)
    cas.op_gemm(cas.W_I4, _i8_dev(qw), _i8_dev(qx), N, K, T, acc, N, epi=cas.EPI_RAW_I32)
    xs = (rng.random(T).astype(np.float32) + np.float32(0.01)) / np.float32(7)
    ws = (rng.random(N).astype(np.float32) + np.float32(0.01)) / np.float32(7)
    y = torch.zeros((T, N), dtype=torch.float32, device=DEV)
    cas.op_gemm(cas.W_I4, _i8_dev(qw), _i8_dev(qx), N, K, T, y, N, epi=cas.EPI_STORE, xs=_f32_dev(xs), ws=_f32_dev(ws))
    torch.cuda.synchronize()
    ref = O.dot_i8_matrix(qx, qw)
    assert np.array_equal(acc.cpu().numpy(), ref)
    want = (ref.astype(np.float32) * xs[:, None]).astype(np.float32) * ws[None, :]
    assert np.array_equal(y.cpu().numpy().view(np.uint32), want.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("T,K,bf16", [(64, 4096, True), (9, 688, False), (3, 11008, True)])
def test_quant_rows_int4_bit_exact(T, K, bf16):
    x = synth.gen_activations(T, K, seed=T + K + 1)
    if bf16:
        xb = synth.f32_to_bf16_bits(x)
        xf = synth.bf16_bits_to_f32(xb)
        xd = _bf16_dev(xb)
    else:
        xf = x
        xd = _f32_dev(x)
    q = torch.zeros((T, K), dtype=torch.int8, device=DEV)
    s = torch.zeros(T, dtype=torch.float32, device=DEV)
    cas.op_quant_rows(cas.W_BF16 if bf16 else cas.W_F32, xd, T, K, q, s, qmax=7)
    torch.cuda.synchronize()
    qr, sr = O.quant_rows(xf, 7)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), sr.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), qr)


@pytest.mark.parametrize("rows,cols", [(96, None), (48, 688)])
def test_quant_weight_int4_bit_exact(rows, cols):
    """The packed int4 copy, unpacked by the library: codes and scales equal
    the oracle's (K = 4096, and K = 688 with a partial last chunk)."""
    shape = synth.SHAPES["llama2_7b"]
    w = synth.gen_tensor(shape.with_layers(1), "wo", 0, seed=4)[:rows]
    if cols:
        w = np.ascontiguousarray(w[:, :cols])
    q = torch.zeros(w.shape, dtype=torch.int8, device=DEV)
    s = torch.zeros(w.shape[0], dtype=torch.float32, device=DEV)
    cas.op_quant_weight(cas.W_BF16, _bf16_dev(w), w.shape[0], w.shape[1], q, s, qmax=7)
    torch.cuda.synchronize()
    qr, sr = O.quant_weight(w, bf16=True, qmax=7)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), sr.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), qr)


@pytest.mark.parametrize("T,K,bf16", [(64, 4096, True), (9, 688, False), (3, 11008, True), (128, 256, False)])
def test_quant_rows_bit_exact(T, K, bf16):
    x = synth.gen_activations(T, K, seed=T + K)
    x[min(4, T - 1), 5] = 1e-30  # tiny values next to a large one
    if bf16:
        xb = synth.f32_to_bf16_bits(x)
        xf = synth.bf16_bits_to_f32(xb)
        xd = _bf16_dev(xb)
    else:
        xf = x
        xd = _f32_dev(x)
    q = torch.zeros((T, K), dtype=torch.int8, device=DEV)
    s = torch.zeros(T, dtype=torch.float32, device=DEV)
    cas.op_quant_rows(cas.W_BF16 if bf16 else cas.W_F32, xd, T, K, q, s)
    torch.cuda.synchronize()
    qr, sr = O.quant_rows(xf)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), sr.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), qr)


def test_quant_weight_bit_exact():
    shape = synth.SHAPES["llama2_7b"]
    w = synth.gen_tensor(shape.with_layers(1), "wo", 0, seed=3)[:96]
    q = torch.zeros(w.shape, dtype=torch.int8, device=DEV)
    s = torch.zeros(w.shape[0], dtype=torch.float32, device=DEV)
    cas.op_quant_weight(cas.W_BF16, _bf16_dev(w), w.shape[0], w.shape[1], q, s)
    torch.cuda.synchronize()
    qr, sr = O.quant_weight(w, bf16=True)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), sr.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), qr)


def _attention_case(H, Hkv, hd, Lc, parents, seed):
    T = len(parents)
    ctx_cap = ((Lc + T + 127) // 128) * 128
    rng = np.random.default_rng(seed)
    q = synth.f32_to_bf16_bits(rng.standard_normal((T, H, hd)).astype(np.float32) * np.float32(1.28))
    kc = synth.f32_to_bf16_bits(rng.standard_normal((Hkv, ctx_cap, hd)).astype(np.float32) * np.float32(1.28))
    vv = synth.f32_to_bf16_bits(rng.standard_normal((Hkv, ctx_cap, hd)).astype(np.float32))
    _, anc = O.tree_metadata(parents)
    anc_np = np.array([[a & (2 ** 64 - 1), a >> 64] for a in anc], dtype=np.uint64)
    out = torch.zeros((T, H * hd), dtype=torch.int16, device=DEV)
    cas.op_attention(_bf16_dev(q), _bf16_dev(kc), _bf16_dev(vv), ctx_cap, Lc, T, T, H, Hkv, hd,
                     torch.from_numpy(anc_np.view(np.int64)).to(DEV), out)
    torch.cuda.synchronize()
    got = synth.bf16_bits_to_f32(out.cpu().numpy().view(np.uint16)).reshape(T, H, hd)
    qf = synth.bf16_bits_to_f32(q)
    kf = synth.bf16_bits_to_f32(kc)
    vf = synth.bf16_bits_to_f32(vv)
    G = H // Hkv
    worst = 0.0
    for t in range(T):
        vis = list(range(Lc)) + [Lc + j for j in range(T) if (anc[t] >> j) & 1]
        for h in range(H):
            ref = O.attend(qf[t, h], kf[h // G, vis], vf[h // G, vis])
            # the output's bf16 rounding explains half a step, 2^-8 |ref|; the
            # rest (two-term bf16 probabilities, 2^-17 relative per weight,
            # i.e. up to 7.6e-6 of max |v|, plus fp32 sums) below 4e-5 of max |v|
            vmax = np.abs(vf[h // G, vis]).max()
            excess = np.abs(got[t, h] - ref) - 2.0 ** -8 * np.abs(ref)
            worst = max(worst, excess.max() / vmax)
    return worst


@pytest.mark.parametrize("H,Hkv,hd,Lc,tree", [
    (4, 4, 128, 1000, ((4, 2, 2, 1, 1), 32)),
    (8, 2, 64, 77, ((3, 2, 1), 15)),
    (4, 1, 128, 0, ((2, 2, 2), 9)),
    (2, 2, 128, 0, ((), 1)),
    (4, 2, 128, 300, ((2,) * 7, 128)),
    (8, 8, 64, 129, ((4, 4, 4), 20)),
    # several 16-row query tiles per workgroup sharing one load of K/V
    # (GQA 4:1, 64 nodes, 9 KV splits: 3 tiles per workgroup, the last
    # workgroup of each head group with one), and an MHA 128-node tree
    (32, 8, 128, 2000, ((4, 4, 4, 4), 64)),
    (8, 8, 128, 3000, ((2,) * 7, 128)),
    # grids of at most 256 such workgroups stage a whole split at once: a
    # 64-wide head (MHA, 128 nodes, 3 splits) and a 4:1 group (64 nodes, 2 splits)
    (8, 8, 64, 500, ((2,) * 7, 128)),
    (8, 2, 128, 400, ((2,) * 6, 64)),
    # two query tiles per workgroup (large grids of MHA heads): an even and an
    # odd tile count (the last workgroup of each head then has one tile)
    (16, 16, 128, 3000, ((2,) * 7, 128)),
    (16, 16, 128, 7000, ((2,) * 7, 40)),
    (32, 32, 64, 2500, ((2,) * 7, 64)),
    # grouped heads packed into shared query tiles (calls of up to 16 tokens):
    # the 8B layout at one and four tokens (one tile per kv head), seven
    # tokens (two tiles, a head's rows straddling them) and an 8-head group
    (32, 8, 128, 4000, ((), 1)),
    (32, 8, 128, 1500, ((3,), 4)),
    (8, 2, 128, 600, ((2, 2), 7)),
    (16, 2, 64, 200, ((2, 2), 5)),
])
def test_attention_tree_mask(H, Hkv, hd, Lc, tree):
    parents = synth.tree_from_branching(*tree) if tree[0] else [-1]
    worst = _attention_case(H, Hkv, hd, Lc, parents, seed=Lc + hd + H)
    assert worst < 4e-5, worst


def test_copy_kernel():
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (1 << 20,), dtype=torch.int32, device=DEV)
    dst = torch.zeros_like(src)
    cas.op_copy(dst, src, src.numel() * 4)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
