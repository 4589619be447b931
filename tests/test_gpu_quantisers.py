"""Bit-exactness of the quantisers fused into the forward's kernels.

Activation quantisation (Sec. 4.1, App. C) runs inside three kernels of the
forward rather than as a pass of its own:
- the RMSNorm writes the codes of the QKV and gate/up inputs;
- the attention's split merge writes the codes of the O projection's input
  (quantised drafts with more than one node);
- the split-K O and down projections of one-node drafts quantise their bf16
  input on load.
Each is run alone through `include/cas_ops.h` and compared, code for code and
scale bit for bit, with the oracle's row quantiser (`O.quant_rows`) applied to
the exact values the kernel quantised.

Inputs mix seeded random rows with designed rows whose values are
representable and whose scale is a power of two, so that x / s lands exactly
on .5 for some elements (round half to even is then observable) and the
row's largest element maps to +-qmax.  For the norm, the designed rows have
a mean square of exactly 4^m and eps = 0, so the normalisation itself is
exact; zero rows (eps > 0) give s = 0 and all-zero codes.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2510_26843_amd import cas, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _dev(a, dtype=None):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _bf16_bits_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV)


def _designed_row(d, qmax, rng, sumsq_exact):
    """A row whose amax element is qmax * u, with a scale s = u exactly: u =
    2^-4 (qmax 127) or 2^-2 (qmax 7).  Half the designed elements sit on
    (k + 0.5) u (ties, both parities of k, both signs).  With sumsq_exact the
    remaining elements are multiples of u/2 chosen so that the row's sum of
    squares is exactly d (mean square 1, every partial sum exact in fp32)."""
    u = 2.0 ** -4 if qmax == 127 else 2.0 ** -2
    half = u / 2
    n_max = 2 * qmax                       # filler |n| * half <= amax
    row = np.zeros(d, dtype=np.float64)
    row[0] = qmax * u
    row[1] = -qmax * u
    used = 2
    budget = d / 2 if sumsq_exact else np.inf   # leave room for the filler
    sq = 2 * (qmax * u) ** 2
    while used < min(66, d // 8):
        k = int(rng.integers(0, qmax))
        v = (k + 0.5) * u
        if sq + v * v > budget:
            k = int(rng.integers(0, max(1, qmax // 8)))
            v = (k + 0.5) * u
            if sq + v * v > budget:
                break
        row[used] = v if rng.random() < 0.5 else -v
        sq += v * v
        used += 1
    if sumsq_exact:
        # units of half: value n * half, square n^2 * half^2
        target = int(round(d / half ** 2))
        have = int(round(float(np.sum((row[:used] / half) ** 2))))
        rest = target - have
        assert rest >= 0
        i = used
        while rest > 0:
            n = min(int(np.sqrt(rest)), n_max)
            row[i] = (n if rng.random() < 0.5 else -n) * half
            rest -= n * n
            i += 1
            assert i <= d, "row too short for the filler"
        assert float(np.sum((row / half) ** 2)) == target
    else:
        row[used:] = rng.integers(-n_max, n_max + 1, size=d - used) * half
    rng.shuffle(row)
    return row.astype(np.float32)


def _check_codes(q_got, s_got, x_f32, qmax, tag):
    q_ref, s_ref = O.quant_rows(x_f32, qmax)
    assert np.array_equal(s_got.view(np.uint32), s_ref.view(np.uint32)), f"{tag}: scales"
    bad = np.argwhere(q_got != q_ref)
    assert bad.size == 0, f"{tag}: {len(bad)} codes differ, first {bad[:4].tolist()}"
    return q_ref, s_ref


# ---------------------------------------------------------------- RMSNorm codes

@pytest.mark.parametrize("atype", [cas.W_BF16, cas.W_F32])
@pytest.mark.parametrize("qmax", [127, 7])
@pytest.mark.parametrize("d,T,nparts", [(4096, 5, 0), (4096, 33, 4), (5120, 17, 2), (688, 3, 0)])
def test_rmsnorm_codes(atype, qmax, d, T, nparts):
    rng = np.random.default_rng(d + T + qmax)
    gain = np.ones(d, dtype=np.float32)
    # (a) random residual rows (one of them zero), eps 1e-6, with pending split-K sums
    h0 = (rng.standard_normal((T, d)) * 2.0).astype(np.float32)
    h0[min(1, T - 1)] = 0.0
    parts = (rng.standard_normal((max(nparts, 1), T, d)) * 0.5).astype(np.float32)
    if nparts:
        parts[:, min(1, T - 1)] = 0.0
    # (b) designed rows: mean square exactly 4^m, eps 0
    hd = np.stack([_designed_row(d, qmax, rng, True) * np.float32(2.0 ** (i % 3)) for i in range(T)])
    for tag, h_in, eps, np_ in (("random", h0, 1e-6, nparts), ("designed", hd, 0.0, 0)):
        vals = torch.zeros((T, d), dtype=torch.int16 if atype == cas.W_BF16 else torch.float32, device=DEV)
        h1 = _dev(h_in)
        cas.op_rmsnorm(atype, h1, _dev(gain), T, d, eps, out=vals, parts=_dev(parts) if np_ else None,
                       nparts=np_, qmax=0)
        q = torch.zeros((T, d), dtype=torch.int8, device=DEV)
        s = torch.zeros(T, dtype=torch.float32, device=DEV)
        h2 = _dev(h_in)
        cas.op_rmsnorm(atype, h2, _dev(gain), T, d, eps, q=q, qs=s, parts=_dev(parts) if np_ else None,
                       nparts=np_, qmax=qmax)
        torch.cuda.synchronize()
        # both calls fold the same partial sums into the residual
        assert torch.equal(h1, h2)
        if np_:
            # the pending sums are added up in split order, then to the residual (fp32)
            pend = parts[0].copy()
            for p in range(1, np_):
                pend = pend + parts[p]
            assert np.array_equal(h1.cpu().numpy(), h_in + pend)
        x = vals.cpu().numpy()
        x = synth.bf16_bits_to_f32(x.view(np.uint16)) if atype == cas.W_BF16 else x
        # the values quantised are the normalised rows (within one rounding of fp64)
        hx = h1.cpu().numpy().astype(np.float64)
        ref = np.stack([O.rmsnorm_row(hx[t], gain, eps) for t in range(T)])
        if tag == "designed":
            assert np.array_equal(x, hd / np.float32(2.0) ** (np.arange(T) % 3)[:, None])
        else:
            # bf16: half a step of the output rounding plus the fp32 norm's own error
            step = 2.0 ** -8 + 1e-5 if atype == cas.W_BF16 else 1e-5
            assert np.all(np.abs(x - ref) <= step * np.abs(ref) + 1e-30)
        q_ref, s_ref = _check_codes(q.cpu().numpy(), s.cpu().numpy(), x, qmax, f"rmsnorm {tag}")
        if tag == "designed":
            assert np.all(np.abs(q_ref).max(axis=1) == qmax)
            ties = np.abs(x / s_ref[:, None] - np.trunc(x / s_ref[:, None])) == 0.5
            assert ties.sum() >= T * 4, "designed rows lost their ties"
        else:
            z = min(1, T - 1)
            assert s_ref[z] == 0 and not q_ref[z].any()


# ---------------------------------------------------------------- merge codes

def _partials(S, T, H, hd, rng):
    m = rng.uniform(-6.0, 6.0, size=(S, H, T)).astype(np.float32)
    l = rng.uniform(0.5, 40.0, size=(S, H, T)).astype(np.float32)
    o = (rng.standard_normal((S, H, T, hd)) * l[..., None]).astype(np.float32)
    ml = np.stack([m, l], axis=-1).astype(np.float32)
    return o, ml


@pytest.mark.parametrize("qmax", [127, 7])
@pytest.mark.parametrize("S,T,H,hd", [(5, 3, 32, 128), (9, 33, 40, 128), (1, 2, 8, 64), (17, 64, 32, 128)])
def test_attn_merge_codes(qmax, S, T, H, hd):
    rng = np.random.default_rng(S * 100 + T + qmax)
    K = H * hd
    o, ml = _partials(S, T, H, hd, rng)
    o[:, :, min(1, T - 1)] = 0.0      # a zero output row
    cases = [("random", S, o, ml)]
    # designed: one split with (m, l) = (0, 1), so the merged row is part_o itself
    od = np.stack([_designed_row(K, qmax, rng, False) for _ in range(T)])     # [T][K]
    od = od.reshape(T, H, hd).transpose(1, 0, 2)[None].copy()                 # [1][H][T][hd]
    mld = np.zeros((1, H, T, 2), dtype=np.float32)
    mld[..., 1] = 1.0
    cases.append(("designed", 1, od, mld))
    for tag, S_, po, pml in cases:
        bf = torch.zeros((T, K), dtype=torch.int16, device=DEV)
        cas.op_attn_merge(_dev(po), _dev(pml), S_, T, H, hd, out=bf, qmax=0)
        q = torch.zeros((T, K), dtype=torch.int8, device=DEV)
        s = torch.zeros(T, dtype=torch.float32, device=DEV)
        cas.op_attn_merge(_dev(po), _dev(pml), S_, T, H, hd, q=q, qs=s, qmax=qmax)
        torch.cuda.synchronize()
        x = synth.bf16_bits_to_f32(bf.cpu().numpy().view(np.uint16))
        # the merged rows against an fp64 merge of the same partials
        mm = pml[..., 0].astype(np.float64)
        M = mm.max(axis=0)
        wgt = np.exp2(mm - M)                                             # [S][H][T]
        num = (po.astype(np.float64) * wgt[..., None]).sum(axis=0)        # [H][T][hd]
        den = (pml[..., 1].astype(np.float64) * wgt).sum(axis=0)
        ref = (num / den[..., None]).transpose(1, 0, 2).reshape(T, K)
        if tag == "designed":
            assert np.array_equal(x, od[0].transpose(1, 0, 2).reshape(T, K))
        else:
            assert np.all(np.abs(x - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-5 * np.abs(ref).max())
        q_ref, s_ref = _check_codes(q.cpu().numpy(), s.cpu().numpy(), x, qmax, f"merge {tag}")
        if tag == "designed":
            assert np.all(np.abs(q_ref).max(axis=1) == qmax)
        else:
            z = min(1, T - 1)
            assert s_ref[z] == 0 and not q_ref[z].any()


# ---------------------------------------------------------------- quantise on load

@pytest.mark.parametrize("wtype,qmax", [(cas.W_I8, 127), (cas.W_I4, 7)])
@pytest.mark.parametrize("N,K", [(4096, 4096), (4096, 11008), (5120, 13824), (4096, 14336)])
def test_gemm_quantise_on_load_codes(wtype, qmax, N, K):
    """Weights W[n][sigma(n)] = qmax (one-hot rows, sigma injective), so each
    output's integer sum is qmax times one code of the row and lands in
    exactly one split; the other splits hold +0.  The sum of the splits then
    equals (fp32(qmax * q[sigma(n)]) * s) * ws[n] exactly, which fixes every
    code and the scale."""
    T = 1
    splits = cas.op_gemm_qx_splits(wtype, N, K, T)
    assert splits >= 2, "this shape runs the quantise-on-load form in the forward"
    rng = np.random.default_rng(N + K + qmax)
    sigma = rng.permutation(K)[:N]
    W = np.zeros((N, K), dtype=np.int8)
    W[np.arange(N), sigma] = qmax
    ws = rng.uniform(0.5, 2.0, size=N).astype(np.float32)
    rows = {
        "random": synth.f32_to_bf16_bits(rng.standard_normal((1, K)).astype(np.float32) * np.float32(1.7)),
        "designed": synth.f32_to_bf16_bits(_designed_row(K, qmax, rng, False)[None]),
        "zero": np.zeros((1, K), dtype=np.uint16),
    }
    for tag, xb in rows.items():
        parts = torch.full((splits, T, N), float("nan"), dtype=torch.float32, device=DEV)
        cas.op_gemm_qx(wtype, _dev(W), _dev(ws), _bf16_bits_dev(xb), N, K, T, qmax, parts)
        torch.cuda.synchronize()
        p = parts.cpu().numpy()
        assert not np.isnan(p).any()
        nz = (p != 0).sum(axis=0)
        assert nz.max() <= 1, f"{tag}: an output has sums in two splits"
        got = p.sum(axis=0)[0]                      # one nonzero term: exact
        x = synth.bf16_bits_to_f32(xb)
        q_ref, s_ref = O.quant_rows(x, qmax)
        acc = (qmax * q_ref[0, sigma].astype(np.int32)).astype(np.float32)
        want = (acc * s_ref[0]) * ws
        bad = np.argwhere(got.view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, f"{tag}: {len(bad)} outputs differ, first {bad[:4].ravel().tolist()}"
        if tag == "zero":
            assert s_ref[0] == 0 and not got.any()
        if tag == "designed":
            assert np.abs(q_ref).max() == qmax
