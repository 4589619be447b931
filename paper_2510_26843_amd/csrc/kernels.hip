// gfx950 (MI355X, CDNA4) kernels of the CAS-Spec token-tree decoder step.
//
// Hot path (Sec. 4.2: one target forward verifies a whole draft tree with tree
// attention; Def. 4.1 / Sec. 4.1: the same forward with layers skipped or
// int8 activations is a draft model):
//   k_gemm       weight-streaming linear layer on MFMA (bf16 16x16x32, int8
//                16x16x64, fp32 16x16x4) with fused epilogues: RoPE + KV
//                write (QKV), SwiGLU (gate/up), residual add (O, down),
//                fp32 logits (LM head)
//   k_attn_bf16  tree-masked attention: QK^T and PV on MFMA, ancestor masks
//                in registers, fp32 online softmax, split over KV slots
//   k_attn_merge merge of the KV splits
//   k_rmsnorm    RMSNorm (optionally straight to per-token int8)
//   k_accept_*   greedy acceptance (argmax + tree walk)
//   k_compact    KV compaction of the accepted path
//
// Wave64 throughout.  MFMA fragments: lane l holds row (l % 16) of the A
// operand and column (l % 16) of B, for the k-group l / 16; the four 16-byte
// loads of a lane in a chunk are contiguous in memory (64 B per lane, 256 B per
// row), so weight rows are read in whole cache lines without any swizzle.  A
// contraction only needs A and B to agree on which k sits in which register
// element, so this k-order is free.
#include "cas_internal.h"
#include <algorithm>
#include <type_traits>

#include <hip/hip_runtime.h>
#include <math.h>

namespace cas {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

template <typename AT> struct Act;
template <> struct Act<float> {
    static __device__ __forceinline__ float ld(const float* p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void st(float* p, size_t i, float v) { p[i] = v; }
    static __device__ __forceinline__ float round(float v) { return v; }
};
template <> struct Act<uint16_t> {
    static __device__ __forceinline__ float ld(const uint16_t* p, size_t i) { return bf2f(p[i]); }
    static __device__ __forceinline__ void st(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }
    static __device__ __forceinline__ float round(float v) { return bf2f(f2bf(v)); }
};

// ---------------------------------------------------------------- reductions

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
// Block-wide reductions for 256 threads; fixed combination order.
__device__ __forceinline__ float block_sum256(float v, float* sh) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[w] = v;
    __syncthreads();
    return ((sh[0] + sh[1]) + sh[2]) + sh[3];
}
__device__ __forceinline__ float block_max256(float v, float* sh) {
    v = wave_max(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[w] = v;
    __syncthreads();
    return fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]));
}

// Reductions over a workgroup of W waves (sh: W floats of LDS); the wave
// partials are combined in wave order, so every thread gets the same value.
template <int W>
__device__ __forceinline__ float block_sum(float v, float* sh) {
    v = wave_sum(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    float r = sh[0];
#pragma unroll
    for (int w = 1; w < W; ++w) r += sh[w];
    return r;
}
template <int W>
__device__ __forceinline__ float block_max(float v, float* sh) {
    v = wave_max(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    float r = sh[0];
#pragma unroll
    for (int w = 1; w < W; ++w) r = fmaxf(r, sh[w]);
    return r;
}

// Code of x at scale sc in [-qm, qm] (qm 127: int8, 7: int4).
__device__ __forceinline__ float qcode(float x, float sc, float qm) {
    return sc != 0.f ? fminf(fmaxf(rintf(x / sc), -qm), qm) : 0.f;
}
// Largest magnitude of 8 bf16 values (16 bytes).
__device__ __forceinline__ float amax_bf8(const i32x4 v) {
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t w = (uint32_t)v[i];
        m = fmaxf(m, fmaxf(fabsf(__uint_as_float(w << 16)), fabsf(__uint_as_float(w & 0xffff0000u))));
    }
    return m;
}

// The attention output of one query row of one head at 4 consecutive d: the
// KV splits' partial states merged in split order with a running max
// (online softmax), eight splits' (m, l) pairs and partial outputs loaded at
// a time (one round of loads for contexts up to 2048 slots), then
// normalised.  row = head * T + t.
__device__ __forceinline__ f32x4 attn_merge_row_hd(const AttnArgs& a, int S, size_t row, int d4, int HD) {
#pragma clang fp contract(off)
    const size_t sstride = (size_t)a.H * a.T;  // rows between splits
    float M = -1e30f, L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < S; s0 += 8) {
        float2 ml[8];
        f32x4 po[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const size_t r = row + (size_t)min(s0 + k, S - 1) * sstride;
            ml[k] = *(const float2*)(a.part_ml + r * 2);
            po[k] = *(const f32x4*)(a.part_o + r * HD + d4);
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            if (s0 + k < S) {
                const float mn = fmaxf(M, ml[k].x);
                const float fo = exp2f(M - mn), fn = exp2f(ml[k].x - mn);
                acc = acc * fo + po[k] * fn;
                L = L * fo + ml[k].y * fn;
                M = mn;
            }
        }
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    return acc * inv;
}
template <int HD>
__device__ __forceinline__ f32x4 attn_merge_row(const AttnArgs& a, int S, size_t row, int d4) {
    return attn_merge_row_hd(a, S, row, d4, HD);
}

// ---------------------------------------------------------------- GEMM

template <int WT> struct WTr;
template <> struct WTr<ET_F32> { static constexpr int E = 4, EB = 4; using acc_t = f32x4; };
template <> struct WTr<ET_BF16> { static constexpr int E = 8, EB = 2; using acc_t = f32x4; };
template <> struct WTr<ET_I8> { static constexpr int E = 16, EB = 1; using acc_t = i32x4; };
// int4 weights run on the int8 MFMA: same steps (16 k per lane), half the bytes
template <> struct WTr<ET_I4> { static constexpr int E = 16, EB = 1; using acc_t = i32x4; };
template <int WT> constexpr bool is_int() { return WT == ET_I8 || WT == ET_I4; }
// 1 KB weight blocks per 16-row tile and chunk (int4: two steps per block)
template <int WT> constexpr int wblocks() { return WT == ET_I4 ? FRAG_U / 2 : FRAG_U; }
// steps per stage: int4 stages hold whole blocks
template <int WT, int UC> constexpr int stage_uc() { return WT == ET_I4 && UC < 2 ? 2 : UC; }

// Four packed nibbles-with-offset (q + 8, one per byte) -> four int8 codes q:
// ((u | 0x80) - 8) ^ 0x80 per byte, no borrow crosses a byte.
__device__ __forceinline__ uint32_t sext_nib4(uint32_t x) { return ((x | 0x80808080u) - 0x08080808u) ^ 0x80808080u; }
// The int8 A-fragment of step h (0, 1) of a packed int4 block (wt4_byte layout).
__device__ __forceinline__ i32x4 i4_step(const i32x4 blk, int h) {
    const uint32_t w0 = (uint32_t)(h ? blk[2] : blk[0]), w1 = (uint32_t)(h ? blk[3] : blk[1]);
    return i32x4{(int)sext_nib4(w0 & 0x0f0f0f0fu), (int)sext_nib4(w1 & 0x0f0f0f0fu),
                 (int)sext_nib4((w0 >> 4) & 0x0f0f0f0fu), (int)sext_nib4((w1 >> 4) & 0x0f0f0f0fu)};
}

// GEMV-style step of one activation row: the lane's 16 weight bytes (8 bf16
// or 16 int8 k of one weight row) times the same k of the row, accumulated in
// the lane (fp32 fma, or exact int32 dot4).  The four lanes of a weight row
// (one per k-group) are summed once, at the end of the stream.
__device__ __forceinline__ float gv_dot(const i32x4 w, const i32x4 x, float acc) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t a = (uint32_t)w[i], b = (uint32_t)x[i];
        acc = fmaf(__uint_as_float(a << 16), __uint_as_float(b << 16), acc);
        acc = fmaf(__uint_as_float(a & 0xffff0000u), __uint_as_float(b & 0xffff0000u), acc);
    }
    return acc;
}
__device__ __forceinline__ int gv_dot(const i32x4 w, const i32x4 x, int acc) {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc = __builtin_amdgcn_sdot4(w[i], x[i], acc, false);
    return acc;
}

// A VALU read of an MFMA result needs a number of wait states after the MFMA
// (8 for the bf16 and int8 16x16 forms, 10 for the fp32 one).  The compiler
// pads straight-line code, but a drain that branches right after its MFMAs
// has been compiled with the accumulators read back at the join two
// instructions later (the last stage's contribution lost for part of a
// tile).  16 wait states after each conditional MFMA group close every such
// path; they cost a few cycles per drain stage.
__device__ __forceinline__ void mfma_result_pad() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7");
    __builtin_amdgcn_sched_barrier(0);
}

template <int WT>
__device__ __forceinline__ typename WTr<WT>::acc_t mfma_step(i32x4 a, i32x4 b, typename WTr<WT>::acc_t c) {
    if constexpr (WT == ET_BF16) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                        __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    } else if constexpr (is_int<WT>()) {
        return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
    } else {
        const f32x4 fa = __builtin_bit_cast(f32x4, a), fb = __builtin_bit_cast(f32x4, b);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[0], fb[0], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[1], fb[1], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[2], fb[2], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[3], fb[3], c, 0, 0, 0);
        return c;
    }
}

// Per-lane operands of the QKV epilogue of one weight tile, loaded at kernel
// start so that they sit in registers when the weight stream ends: each
// row's KV slot and, for q and k rows, the RoPE cos/sin of the lane's two
// rotation pairs at the row's position.  Loads are unconditional (indices
// clamped into their arrays).
template <int NT>
struct QkvPre {
    int slot[NT];
    float cs[NT][2], sn[NT][2];
    __device__ __forceinline__ void load(const GemmArgs& a, int tile, int lane) {
        const int r = lane & 15, g = lane >> 4, nb = tile * 16 + 4 * g;
        const int hd = a.hd, qrows = a.H * hd, krows = a.Hkv * hd, half = hd / 2;
        const bool rot = nb < qrows + krows;
        const int p0 = ((nb - (nb < qrows ? 0 : qrows)) % hd) / 2;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int t = min(16 * j + r, a.T - 1);
            slot[j] = a.row_slot[t];
            int pos = a.row_pos[t];
            if (!dcheck(a.chk, pos >= 0 && pos < a.ctx_cap, CHK_POSITION)) pos = 0;
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const size_t idx = rot ? (size_t)pos * half + p0 + p : 0;
                cs[j][p] = a.rope_cos[idx];
                sn[j][p] = a.rope_sin[idx];
            }
        }
    }
};

// Two consecutive activation values (4-byte aligned for bf16, 8 for fp32).
__device__ __forceinline__ void st2(uint16_t* p, size_t o, float x, float y) {
    *(uint32_t*)(p + o) = (uint32_t)f2bf(x) | ((uint32_t)f2bf(y) << 16);
}
__device__ __forceinline__ void st2(float* p, size_t o, float x, float y) { *(float2*)(p + o) = make_float2(x, y); }

// Epilogue of one 16-row weight tile: lane holds y[n = 16*tile + 4g + i][t = 16j + r].
// qp: the tile's preloaded QKV operands (EPI_QKV only).
template <int WT, int NT, int EPI, typename AT>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, const typename WTr<WT>::acc_t (&acc)[NT], int tile,
                                              int last_tile, int lane, const QkvPre<NT>& qp) {
    const int r = lane & 15, g = lane >> 4, T = a.T;
    const int nb = tile * 16 + 4 * g;
    const int nto = col_tiles(T);  // column tiles of a tiled output (NT, or 1 held for a wider layout)
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int t = 16 * j + r;
        if (t >= T) continue;
        float v[4];
        if constexpr (is_int<WT>()) {
            if constexpr (EPI == EPI_RAW) {
                int* o = (int*)a.out + (size_t)t * a.ldo + nb;
#pragma unroll
                for (int i = 0; i < 4; ++i) o[i] = acc[j][i];
                continue;
            } else {
                const float xs = a.xs[t];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float y = (float)acc[j][i] * xs;
                    v[i] = y * a.ws[nb + i];
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = acc[j][i];
        }
        if constexpr (EPI == EPI_STORE) {
            float* o = (float*)a.out + (size_t)t * a.ldo + nb;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = v[i];
        } else if constexpr (EPI == EPI_RESID) {
            float* o = (float*)a.out + (size_t)t * a.ldo + nb;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] += v[i];
        } else if constexpr (EPI == EPI_SWIGLU) {
            constexpr int EO = 16 / sizeof(AT);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const float gt = v[2 * p], up = v[2 * p + 1];
                Act<AT>::st((AT*)a.out, xt_off(t, nb / 2 + p, nto, EO), gt / (1.0f + expf(-gt)) * up);
            }
        } else if constexpr (EPI == EPI_QKV) {
            const int hd = a.hd, qrows = a.H * hd, krows = a.Hkv * hd;
            const int slot = qp.slot[j];
            if (nb < qrows + krows) {
                const bool isq = nb < qrows;
                const int rel = nb - (isq ? 0 : qrows);
                const int head = rel / hd, p0 = (rel % hd) / 2, half = hd / 2;
                float lo[2], hi[2];
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const float cs = qp.cs[j][p], sn = qp.sn[j][p];
                    const float x0 = v[2 * p], x1 = v[2 * p + 1];
                    lo[p] = x0 * cs - x1 * sn;
                    hi[p] = x0 * sn + x1 * cs;
                }
                // the pairs p0, p0 + 1 (p0 even) are adjacent in q and in both K layouts
                if (isq) {
                    AT* o = (AT*)a.out + ((size_t)t * a.H + head) * hd;
                    st2(o, p0, lo[0], lo[1]);
                    st2(o, p0 + half, hi[0], hi[1]);
                } else if (dcheck(a.chk, slot >= 0 && slot < a.ctx_cap, CHK_KV_WRITE)) {
                    constexpr int ET = sizeof(AT) == 2 ? ET_BF16 : ET_F32;
                    AT* o = (AT*)a.kc + (size_t)head * a.ctx_cap * hd;
                    st2(o, kv_k_off(ET, slot, p0, hd, a.ctx_cap), lo[0], lo[1]);
                    st2(o, kv_k_off(ET, slot, p0 + half, hd, a.ctx_cap), hi[0], hi[1]);
                }
            } else if (dcheck(a.chk, slot >= 0 && slot < a.ctx_cap, CHK_KV_WRITE)) {
                constexpr int ET = sizeof(AT) == 2 ? ET_BF16 : ET_F32;
                const int rel = nb - qrows - krows;
                const int head = rel / hd, dd = rel % hd;
                AT* o = (AT*)a.vt + (size_t)head * a.ctx_cap * hd;
#pragma unroll
                for (int i = 0; i < 4; ++i) Act<AT>::st(o, kv_v_off(ET, slot, dd + i, hd, a.ctx_cap), v[i]);
            }
        }
    }
    if constexpr (EPI == EPI_SWIGLU) {
        // the last tile also zeroes the pad columns of the output rows
        constexpr int EO = 16 / sizeof(AT);
        if (tile == last_tile) {
            const int kp = (a.out_k + 16 * EO - 1) / (16 * EO) * (16 * EO);
            const int w = kp - a.out_k;
            for (int idx = lane; idx < T * w; idx += 64)
                Act<AT>::st((AT*)a.out, xt_off(idx / w, a.out_k + idx % w, nto, EO), 0.f);
        }
    }
}

// Weights are streamed with nontemporal loads (read once per forward; the
// hint keeps them from displacing the activation fragments, which every
// workgroup re-reads from L2).
//
// One workgroup = 16 output rows (one weight tile) x all T columns.  Its
// WAVES waves split the tile's chunks into contiguous runs; each wave streams
// its run through a D-stage register ring of UC-step stages (weights and the
// matching activation fragments are issued D stages ahead of use, so the
// oldest-first wait of the vector memory counter never stalls on a fresher
// load).  With the tiled layouts every load instruction of a wave reads 1 KB
// of contiguous memory.  Every load in the ring is unconditional, so the
// outstanding loads at the loop entry equal those at its back edge and each
// wait is exact.  Partial tiles are summed in LDS in wave order
// (deterministic).
template <int WT, int NT, int UC, int D, int WAVES, int EPI, typename AT>
__global__ void __launch_bounds__(64 * WAVES) k_gemm(const GemmArgs a) {
    using Tr = WTr<WT>;
    using ACC = typename Tr::acc_t;
    constexpr int E = Tr::E;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar branches
    const int r = lane & 15, g = lane >> 4;
    const int tile = blockIdx.x;
    const int T = a.T;
    const int C = a.Kp / (16 * E);  // chunks of the tile
    const int c0 = (wave * C) / WAVES, c1 = ((wave + 1) * C) / WAVES;
    const int S0 = c0 * (FRAG_U / UC), S1 = c1 * (FRAG_U / UC);  // stages of UC steps

    static_assert(WT != ET_I4 || UC % 2 == 0, "int4 stages hold whole blocks");
    // 1 KB weight blocks: tile-major, or K-major (wt_kmajor)
    const size_t bstride = a.kmaj ? (size_t)(a.N >> 4) * 1024 : 1024;
    const char* wb = (const char*)a.W + (size_t)lane * 16 + (size_t)tile * (a.kmaj ? 1024 : (size_t)C * wblocks<WT>() * 1024);
    const char* xb = (const char*)a.X + (size_t)lane * 16;
    ACC acc[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[j] = ACC{0, 0, 0, 0};

    i32x4 A[D][UC];
    i32x4 B[D][NT][UC];
    QkvPre<NT> qp;
    if constexpr (EPI == EPI_QKV) qp.load(a, tile, lane);

#define CAS_GEMM_LOAD(st, stage)                                                                 \
    do {                                                                                         \
        const size_t q = (size_t)(stage) * UC;                                                   \
        _Pragma("unroll") for (int u = 0; u < UC; ++u) {                                        \
            if (WT != ET_I4 || (u & 1) == 0)                                                     \
                A[st][u] = __builtin_nontemporal_load(                                           \
                    (const i32x4*)(wb + (WT == ET_I4 ? (q + u) / 2 : q + u) * bstride));         \
            _Pragma("unroll") for (int j = 0; j < NT; ++j) B[st][j][u] =                         \
                *(const i32x4*)(xb + ((q + u) * NT + j) * 1024);                                 \
        }                                                                                        \
    } while (0)
#define CAS_GEMM_MMA(st)                                                                         \
    do {                                                                                         \
        _Pragma("unroll") for (int u = 0; u < UC; ++u) {                                        \
            const i32x4 au = WT == ET_I4 ? i4_step(A[st][u & ~1], u & 1) : A[st][u];             \
            _Pragma("unroll") for (int j = 0; j < NT; ++j) acc[j] =                              \
                mfma_step<WT>(au, B[st][j][u], acc[j]);                                          \
        }                                                                                        \
    } while (0)

    if (S1 > S0) {
#pragma unroll
        for (int s = 0; s < D; ++s) CAS_GEMM_LOAD(s, min(S0 + s, S1 - 1));
        int c = S0;
        for (; c + 2 * D <= S1; c += D) {
#pragma unroll
            for (int s = 0; s < D; ++s) {
                CAS_GEMM_MMA(s);
                // keep each refill behind the MMAs that free its registers
                __builtin_amdgcn_sched_barrier(0);
                CAS_GEMM_LOAD(s, c + s + D);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // drain: fewer than 2D stages left, ring slot s holds stage c + s
#pragma unroll
        for (int s = 0; s < D; ++s) {
            if (c + s < S1) {
                CAS_GEMM_MMA(s);
                mfma_result_pad();
                if (c + s + D < S1) CAS_GEMM_LOAD(s, c + s + D);
            }
        }
#pragma unroll
        for (int s = 0; s < D; ++s)
            if (c + D + s < S1) {
                CAS_GEMM_MMA(s);
                mfma_result_pad();
            }
    }
#undef CAS_GEMM_MMA
#undef CAS_GEMM_LOAD

    if constexpr (WAVES > 1) {
        using S = typename std::conditional<is_int<WT>(), int, float>::type;
        __shared__ S red[WAVES - 1][NT][4][64];
        if (wave > 0) {
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) red[wave - 1][j][i][lane] = acc[j][i];
        }
        __syncthreads();
        if (wave != 0) return;
        for (int w = 1; w < WAVES; ++w)
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[j][i] += red[w - 1][j][i][lane];
    }

    gemm_epilogue<WT, NT, EPI, AT>(a, acc, blockIdx.x, (int)gridDim.x - 1, lane, qp);
}

// Wide variant for tall weight matrices: the WAVES waves of a workgroup own
// WAVES*TPW adjacent 16-row tiles (TPW per wave) over the whole K range, and
// the activation fragments of each stage are loaded once per workgroup (wave
// w loads the stage's 1 KB blocks w, w + WAVES, ...) into a two-slot LDS ring
// that all waves read: WAVES*TPW times less activation traffic than one tile
// per workgroup.  One barrier per stage; register stages as in k_gemm.
// RX (resident activations, calls of at most 16 rows): the workgroup copies
// its T rows of its K range once into LDS (dynamic shared memory, T x K range
// elements) and each MFMA step reads a lane's 16 bytes from there: lanes of
// columns >= T feed zeros.  No stage ring and no per-stage barrier, and the
// activation bytes each workgroup reads drop from 32 padded rows to T rows.
// Every column's MFMA work is the same as in the ringed form, so the sums are
// the same bits.
static constexpr int RX_PIECES = 6;  // 16-byte activation pieces per thread (RX copy)
// QX (with RX, integer weights, a bf16 source): the workgroup first takes
// every row's amax over the row's whole width, then writes the codes of its
// K range to LDS by the row quantiser's rule (scale amax / qx, round to
// nearest even, clamp), and dequantises with those scales: the same codes and
// sums as quantising in a separate pass, without that pass.  Every workgroup
// reads the whole rows for the amax, which pays for one row only: the O and
// down projections of one-node quantised drafts (13B W8A8 2.08 -> 2.00 ms,
// W4A4 1.75 -> 1.63 ms; at four rows the same use was 2% slower, and the
// QKV and gate/up inputs, whose norm already writes codes, were slower too).
static constexpr int QX_MAX_T = 1;
// MX (with RX, bf16 weights, at most one merge item of 4 elements per
// thread): the input rows are merged on load from the attention's split
// partials by the same routine, with the same bf16 rounding, as the merge
// kernel; each workgroup merges only its K range (the heads it covers), and
// the merge kernel is not launched.  Measured one-row verify: 7B 3.10 ->
// 3.02 ms (ctx 1024) and 3.91 -> 3.84 ms (8192), 8B 3.49 -> 3.42 and 3.76 ->
// 3.67 ms (1024, 4096).  With two items per thread (two rows of 7B, or the
// 13B K ranges of 14 heads) the serial merges cost more than the launch at
// longer contexts (7B two rows at 8192: 3.90 -> 4.01 ms; 13B one row at 4096:
// 5.65 -> 5.70 ms).
static constexpr int MX_MAX_T = 2;
// GV (drafts of one row, bf16 or int8 weights): GEMV-style tiles.  Each lane
// takes the activation row's 16 bytes at its own k-group straight from the
// tiled activations (lane 16g of each 1 KB block) and accumulates VALU dot
// products of its weight fragment with them; the four k-group lanes of a
// weight row are summed with two cross-lane exchanges at the end.  No padded
// MFMA columns, no LDS stage ring and no barrier.  Measured alone on the 7B
// shapes at one row: gate/up 28.7 -> 27.9 us, LM head 42.8 -> 39.4 us.  The
// sums are in a different order than the MFMA's, so verify calls (whose rows
// must not depend on the tree size) keep the MFMA form.
// EV: one-tile waves, and the grid splits the N/16 tiles as evenly as it can
// (workgroup i takes tiles floor(i n / G) .. floor((i + 1) n / G), at most
// WAVES of them); a wave past its workgroup's share repeats the share's last
// tile (those loads hit the cache) and stores nothing.
template <int WT, int NT, int UC, int D, int WAVES, int TPW, int EPI, typename AT, bool RX, bool QX = false,
          bool MX = false, bool GV = false, bool KM = false, bool EV = false>
__global__ void __launch_bounds__(64 * WAVES) k_gemm_wide(const GemmArgs a) {
    using Tr = WTr<WT>;
    using ACC = typename Tr::acc_t;
    constexpr int E = Tr::E;
    static_assert(!GV || (!RX && (WT == ET_BF16 || WT == ET_I8)), "GEMV tiles: one streamed row, bf16 or int8");
    static_assert(!RX || NT == 1, "resident activations feed one column tile");
    static_assert(!QX || (RX && is_int<WT>()), "quantise-on-load feeds resident integer codes");
    static_assert(!MX || (RX && WT == ET_BF16), "merge-on-load feeds a resident bf16 row");
    __shared__ float qsc[QX ? QX_MAX_T : 1], qred[QX ? WAVES : 1];
    constexpr int NB = NT * UC;  // 1 KB activation blocks per stage
    constexpr int LPT = (NB + WAVES - 1) / WAVES;  // 1 KB blocks per wave per stage
    static_assert(D % 2 == 0 && FRAG_U % UC == 0, "stage shape");
    static_assert(WT != ET_I4 || UC % 2 == 0, "int4 stages hold whole blocks");
    constexpr int WB = wblocks<WT>();                  // weight blocks per chunk
    constexpr int UB = WT == ET_I4 ? UC / 2 : UC;     // weight blocks per stage
    __shared__ __attribute__((aligned(16))) char lds[2][RX ? 16 : NB * 1024];
    extern __shared__ __attribute__((aligned(16))) char xr[];  // RX: T rows of the K range
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    static_assert(!EV || (TPW == 1 && !RX && !GV), "even split: one-tile waves of the ringed loop");
    int tile0 = (blockIdx.x * WAVES + wave) * TPW;
    bool wact = true;
    if constexpr (EV) {
        const unsigned ntl = (unsigned)a.N >> 4;
        const int wg0 = (int)((blockIdx.x * ntl) / gridDim.x), wg1 = (int)(((blockIdx.x + 1) * ntl) / gridDim.x);
        wact = wg0 + wave < wg1;
        tile0 = min(wg0 + wave, wg1 - 1);
    }
    const int C = a.Kp / (16 * E);
    // stages of this workgroup: the whole K range, or split gridDim.y ways at
    // chunk boundaries, so the K ranges (and every row's summation order) do
    // not depend on the stage width, which changes with the column tiles
    const int c0 = (int)(((long)blockIdx.y * C) / gridDim.y);
    const int c1 = (int)(((long)(blockIdx.y + 1) * C) / gridDim.y);
    const int s0 = c0 * (FRAG_U / UC), NS = (c1 - c0) * (FRAG_U / UC);
    // 1 KB weight blocks: tile-major (tiles tstride apart, a tile's blocks
    // adjacent) or, KM, K-major (wt_kmajor: tiles adjacent, a tile's blocks
    // N/16 KB apart).  A compile-time choice: a runtime block stride costs
    // the tile-major loops their immediate load offsets (13B W4A4 draft
    // 1.63 -> 1.73 ms when both orders shared one kernel).
    const size_t tstride = KM ? 1024 : (size_t)C * WB * 1024;
    const size_t bstride = KM ? (size_t)(a.N >> 4) * 1024 : 1024;
    const char* wb = (const char*)a.W + (size_t)lane * 16 + (size_t)tile0 * tstride + (size_t)s0 * UB * bstride;
    const char* xb = (const char*)a.X + (size_t)lane * 16 + (size_t)s0 * NB * 1024;
    // RX: element k0 of the range, row t, at xr + t * RS + k0 * EB (rows 16 bytes
    // apart in the banks); lane (g, col) of step u in chunk ch reads
    // k0 = ch * 16E + g * 4E + u * E (the tiled order)
    constexpr int EB = 16 / E;
    const int KR = (c1 - c0) * 16 * E, RS = KR * EB + 16;
    const int rxc = min(lane & 15, a.T - 1);
    const bool rxz = (lane & 15) >= a.T;
    const char* xrl = xr + (size_t)rxc * RS + (lane >> 4) * 4 * E * EB;
    ACC acc[TPW][NT];
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[t][j] = ACC{0, 0, 0, 0};
    i32x4 A[D][TPW][UB];
    i32x4 Bv[D][GV ? 1 : LPT];
    // GV: the row's fragments of the stage (lane 16g of each block) and the lane sums
    using GS = typename std::conditional<is_int<WT>(), int, float>::type;
    i32x4 Xv[D][GV ? UC : 1];
    GS gacc[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) gacc[t] = 0;
    const char* xg = (const char*)a.X + (size_t)(lane >> 4) * 256 + (size_t)s0 * NB * 1024;
    QkvPre<NT> qp[TPW];
    if constexpr (EPI == EPI_QKV) {
#pragma unroll
        for (int t = 0; t < TPW; ++t) qp[t].load(a, tile0 + t, lane);
    }

#define CAS_W_LOAD(st, stage)                                                                    \
    do {                                                                                         \
        const size_t q = (size_t)(stage) * UB;                                                   \
        _Pragma("unroll") for (int t = 0; t < TPW; ++t)                                         \
            _Pragma("unroll") for (int u = 0; u < UB; ++u) A[st][t][u] =                        \
                __builtin_nontemporal_load((const i32x4*)(wb + t * tstride + (q + u) * bstride)); \
        /* a block index past the stage (WAVES not dividing NB) reloads the last block, */  \
        /* so every wave issues the same loads; it is not stored */                         \
        if constexpr (GV)                                                                        \
            _Pragma("unroll") for (int u = 0; u < UC; ++u) Xv[st][u] =                           \
                *(const i32x4*)(xg + ((size_t)(stage) * NB + u * NT) * 1024);                   \
        else if constexpr (!RX)                                                                  \
            _Pragma("unroll") for (int p = 0; p < LPT; ++p) Bv[st][p] = *(const i32x4*)(        \
                xb + ((size_t)(stage) * NB + min(p * WAVES + wave, NB - 1)) * 1024);             \
    } while (0)
#define CAS_W_STAGE(st, slot, stage)                                                             \
    do {                                                                                         \
        if constexpr (GV) {                                                                      \
            _Pragma("unroll") for (int u = 0; u < UC; ++u)                                      \
                _Pragma("unroll") for (int t = 0; t < TPW; ++t)                                 \
                    gacc[t] = gv_dot(A[st][t][u], Xv[st][u], gacc[t]);                           \
        } else {                                                                                 \
            if constexpr (!RX) {                                                                 \
                _Pragma("unroll") for (int p = 0; p < LPT; ++p) if (p * WAVES + wave < NB)      \
                    *(i32x4*)(&lds[slot][(p * WAVES + wave) * 1024 + lane * 16]) = Bv[st][p];    \
                __syncthreads();                                                                 \
            }                                                                                    \
            _Pragma("unroll") for (int u = 0; u < UC; ++u) {                                    \
                i32x4 au[TPW];                                                                   \
                _Pragma("unroll") for (int t = 0; t < TPW; ++t)                                 \
                    au[t] = WT == ET_I4 ? i4_step(A[st][t][u >> 1], u & 1) : A[st][t][u];        \
                _Pragma("unroll") for (int j = 0; j < NT; ++j) {                                \
                    i32x4 b;                                                                     \
                    if constexpr (RX) {                                                          \
                        const int v = (stage) * UC + u; /* step of the K range */                \
                        b = *(const i32x4*)(xrl + ((v / FRAG_U) * 16 * E + (v % FRAG_U) * E) * EB); \
                        if (rxz) b = i32x4{0, 0, 0, 0};                                          \
                    } else {                                                                     \
                        b = *(const i32x4*)(&lds[slot][(u * NT + j) * 1024 + lane * 16]);        \
                    }                                                                            \
                    _Pragma("unroll") for (int t = 0; t < TPW; ++t)                             \
                        acc[t][j] = mfma_step<WT>(au[t], b, acc[t][j]);                          \
                }                                                                                \
            }                                                                                    \
        }                                                                                        \
    } while (0)

#pragma unroll
    for (int s = 0; s < D; ++s) CAS_W_LOAD(s, min(s, NS - 1));
    if constexpr (QX) {
        // after the first weight loads are in flight
        const int NTS = col_tiles(a.T), Kpa = (a.xk + 127) / 128 * 128, nth = 64 * WAVES;
        const uint16_t* xh = (const uint16_t*)a.X;
        const float qm = (float)a.qx;
        for (int t = 0; t < a.T; ++t) {
            float m = 0.f;
            for (int p = threadIdx.x; p < Kpa / 8; p += 4 * nth) {
                i32x4 v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    v[i] = *(const i32x4*)(xh + xt_off(t, min(p + i * nth, Kpa / 8 - 1) * 8, NTS, 8));
#pragma unroll
                for (int i = 0; i < 4; ++i) m = fmaxf(m, amax_bf8(v[i]));  // clamped repeats change no max
            }
            m = block_max<WAVES>(m, qred);
            if (threadIdx.x == 0) qsc[t] = m / qm;
        }
        __syncthreads();
        const int ppr = KR / 16, np = a.T * ppr;  // 16 codes per piece
        for (int p = threadIdx.x; p < np; p += nth) {
            const int t = p / ppr, k = (p % ppr) * 16, kg = c0 * 256 + k;
            const float sc = qsc[t];
            i32x4 h[2] = {i32x4{0, 0, 0, 0}, i32x4{0, 0, 0, 0}};
            if (kg < Kpa) {
                h[0] = *(const i32x4*)(xh + xt_off(t, kg, NTS, 8));
                h[1] = *(const i32x4*)(xh + xt_off(t, kg + 8, NTS, 8));
            }
            i32x4 q;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t w0 = (uint32_t)h[j >> 1][(j & 1) * 2], w1 = (uint32_t)h[j >> 1][(j & 1) * 2 + 1];
                const float x[4] = {__uint_as_float(w0 << 16), __uint_as_float(w0 & 0xffff0000u),
                                    __uint_as_float(w1 << 16), __uint_as_float(w1 & 0xffff0000u)};
                uint32_t b = 0;
#pragma unroll
                for (int u = 0; u < 4; ++u) b |= (uint32_t)(uint8_t)(int8_t)qcode(x[u], sc, qm) << (8 * u);
                q[j] = (int)b;
            }
            *(i32x4*)(xr + (size_t)t * RS + k) = q;
        }
        __syncthreads();
    } else if constexpr (MX) {
        // row t, element k0 + k of the K range at xr + t * RS + 2k (bf16)
        AttnArgs m{};
        m.H = a.H;
        m.T = a.T;
        m.part_o = (float*)a.mx_o;
        m.part_ml = (float*)a.mx_ml;
        const int k0 = c0 * 16 * E, kin = a.H * a.hd, ipr = KR / 4;
        for (int i = threadIdx.x; i < a.T * ipr; i += 64 * WAVES) {
            const int t = i / ipr, k = k0 + 4 * (i % ipr);
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (k < kin) v = attn_merge_row_hd(m, a.mx_S, (size_t)(k / a.hd) * a.T + t, k % a.hd, a.hd);
            *(uint2*)(xr + (size_t)t * RS + (size_t)8 * (i % ipr)) =
                make_uint2((uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                           (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
        }
        __syncthreads();
    } else if constexpr (RX) {
        // after the first weight loads are in flight: all pieces' loads issue
        // back to back (at most RX_PIECES per thread), then the LDS stores
        const int NTS = col_tiles(a.T), ppr = KR / E, np = a.T * ppr;  // 16-byte pieces
        i32x4 xp[RX_PIECES];
#pragma unroll
        for (int i = 0; i < RX_PIECES; ++i) {
            const int p = min((int)threadIdx.x + 64 * WAVES * i, np - 1), t = p / ppr, k = (p % ppr) * E;
            xp[i] = *(const i32x4*)((const char*)a.X + xt_off(t, c0 * 16 * E + k, NTS, E) * EB);
        }
#pragma unroll
        for (int i = 0; i < RX_PIECES; ++i) {
            const int p = (int)threadIdx.x + 64 * WAVES * i, t = p / ppr, k = (p % ppr) * E;
            if (p < np) *(i32x4*)(xr + (size_t)t * RS + (size_t)k * EB) = xp[i];
        }
        __syncthreads();
    }
    int c = 0;
    for (; c + 2 * D <= NS; c += D) {
#pragma unroll
        for (int s = 0; s < D; ++s) {
            CAS_W_STAGE(s, s & 1, c + s);
            __builtin_amdgcn_sched_barrier(0);
            CAS_W_LOAD(s, c + s + D);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // drain (c is a multiple of the even D, so stage c + s uses LDS slot s & 1)
#pragma unroll
    for (int s = 0; s < D; ++s) {
        if (c + s < NS) {
            CAS_W_STAGE(s, s & 1, c + s);
            mfma_result_pad();
            if (c + s + D < NS) CAS_W_LOAD(s, c + s + D);
        }
    }
#pragma unroll
    for (int s = 0; s < D; ++s)
        if (c + D + s < NS) {
            CAS_W_STAGE(s, s & 1, c + D + s);
            mfma_result_pad();
        }
#undef CAS_W_STAGE
#undef CAS_W_LOAD
    if constexpr (GV) {
        // sum the four k-group lanes of each weight row, then put row
        // 16 tile + 4g + i of activation row 0 where the MFMA epilogue
        // expects it (element i of lane 16g); other lanes feed columns >= T
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            GS v = gacc[t];
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[t][0][i] = __shfl(v, 4 * (lane >> 4) + i);
        }
    }
    GemmArgs ae = a;
    if constexpr (QX) ae.xs = qsc;  // the scales this workgroup derived
    if constexpr (EV) {
        if (!wact) return;
    }
    if (gridDim.y == 1) {
#pragma unroll
        for (int t = 0; t < TPW; ++t) gemm_epilogue<WT, NT, EPI, AT>(ae, acc[t], tile0 + t, a.N / 16 - 1, lane, qp[t]);
    } else {
        GemmArgs b = ae;
        b.out = (float*)a.out + blockIdx.y * a.part_stride;
#pragma unroll
        for (int t = 0; t < TPW; ++t) gemm_epilogue<WT, NT, EPI, AT>(b, acc[t], tile0 + t, a.N / 16 - 1, lane, qp[t]);
    }
}

// Matrices with at least 8192 rows (in tiles: a multiple of 3 or 4) take the wide variant;
// shorter ones split K across the waves of a 16-row workgroup so that the
// grid still covers every CU.
// Stage shape of the wide kernel: UC steps per stage and D stages in the
// register ring, by column tiles NT and tiles per wave TPW.  The ring keeps
// 8-16 KB of weights in flight per wave; wider activations (larger NT) take
// fewer steps per stage, so the ring gets deeper (measured on the 7B
// shapes: T = 64 gate/up 38.7 -> 35.8 us, T = 128 69.6 -> 50.8 us, T <= 32
// QKV 17.9 -> 17.2 us).
template <int NT, int TPW> struct WideStage {
    static constexpr int UC = TPW == 2 ? (NT == 2 ? 4 : 2) : (NT == 8 ? 1 : 2);
    static constexpr int D = TPW == 2 && NT == 2 ? 2 : 4;
};
// ... with whole int4 blocks per stage
template <int WT, int NT, int TPW> struct WideStageW {
    static constexpr int UC = stage_uc<WT, WideStage<NT, TPW>::UC>();
    static constexpr int D = WideStage<NT, TPW>::D;
};

// Resident activations (RX) serve the int4-weight GEMMs of calls of at most
// 16 rows whose rows of one workgroup's K range are at most RX_PIECES 16-byte
// pieces per thread of a 3-wave workgroup.  Measured against the ringed
// kernel: 13B W4A4 draft of one node 1.85 -> 1.75 ms, of four nodes 1%
// faster; the same change made bf16 and int8 forwards slower (7B one-node
// draft 1.55 -> 1.60 ms, 13B W8A8 2.07 -> 2.11 ms), where the activation
// rows are a smaller share of what each workgroup streams.
static constexpr int RX_MAX_T = 16;
static int rx_lds_bytes(int wtype, int T, int Kp, int ksplit) {
    const int kc = chunk_k(wtype), C = Kp / kc;
    const int kr = (C + ksplit - 1) / ksplit * kc;  // elements of the longest K range
    return T * (kr * (int)frag_elem_bytes(wtype) + 16);
}
bool gemm_mx_ok(int wtype, int N, int Kp, int T, int ksplit) {
    if (wtype != ET_BF16 || T < 1 || T > MX_MAX_T || N % 64 || Kp % chunk_k(wtype) || ksplit < 2) return false;
    // at most one (row, 4 elements) merge item per thread of the 256-thread workgroup
    const int kc = chunk_k(wtype), C = Kp / kc, kr = (C + ksplit - 1) / ksplit * kc;
    return T * kr <= 4 * 256 && rx_lds_bytes(wtype, T, Kp, ksplit) <= 65536;
}
bool gemm_qx_ok(int wtype, int N, int Kp, int T, int ksplit) {
    if ((wtype != ET_I8 && wtype != ET_I4) || T < 1 || T > QX_MAX_T || N % 64 || Kp % chunk_k(wtype)) return false;
    return ksplit >= 2 && rx_lds_bytes(wtype, T, Kp, ksplit) <= 65536;
}
static bool rx_use(int wtype, const GemmArgs& a, int ksplit) {
    const int kc = chunk_k(wtype), C = a.Kp / kc, kr = (C + ksplit - 1) / ksplit * kc;
    const long pieces = (long)a.T * kr * frag_elem_bytes(wtype) / 16;
    return wtype == ET_I4 && a.T <= RX_MAX_T && pieces <= 192L * RX_PIECES;
}

template <int WT, int NT, int EPI, typename AT, bool KM>
static hipError_t gemm_go(const GemmArgs& a, hipStream_t s) {
    if (a.qx || a.mx_o || a.kmaj != (int)KM) return hipErrorInvalidValue;  // quantise / merge on load: the split-K form only
    constexpr int UC = stage_uc<WT, NT == 2 ? 4 : (NT == 4 ? 2 : 1)>();
    if (a.N >= 8192 && ((a.N / 16) % 4 == 0 || (a.N / 16) % 3 == 0)) {
        using S1 = WideStageW<WT, NT, 1>;
        using S2 = WideStageW<WT, NT, 2>;
        // Every workgroup should stay resident on a CU of its own (a CU that
        // holds two workgroups while others hold one sets the pace): take the
        // split of the tiles into equal workgroups of 4x1, 3x1, 4x2 or 3x2
        // tiles (waves x tiles per wave) with the most workgroups up to 256,
        // else 4x2.
        const int tiles = a.N / 16;
        static const int opt[4][2] = {{4, 1}, {3, 1}, {4, 2}, {3, 2}};
        int bw = 0, bt = 0, bg = 0;
        for (const auto& o : opt) {
            const int per = o[0] * o[1];
            if (tiles % per == 0 && tiles / per <= 256 && tiles / per > bg) { bw = o[0]; bt = o[1]; bg = tiles / per; }
        }
        if (!bg) {
            if (tiles % 8 == 0) { bw = 4; bt = 2; bg = tiles / 8; }
            else if (tiles % 4 == 0) { bw = 4; bt = 1; bg = tiles / 4; }
            else { bw = 3; bt = 1; bg = tiles / 3; }
        }
        if constexpr (WT == ET_BF16 || WT == ET_I8) {
            // A tile count with no divisor near the CU count (7B gate/up:
            // 1376 tiles, 172 equal workgroups of eight) leaves CUs without
            // a stream while the others carry eight tiles: split the tiles
            // as evenly as the grid allows over fewer workgroups than CUs,
            // of six one-tile waves (7B gate/up: 230 of 5-6 tiles), else
            // seven (13B gate/up: 247 of 6-7), where that lowers a CU's
            // share below the equal split's.  A CU's share, not the grid,
            // sets the time: the 7B QKV's 256 workgroups of three stay.
            // Interleaved forwards against the equal split: 7B verify T = 32
            // 3.220 -> 3.130 ms (gate/up 31.1 -> 29.5 us), one-node skip-50%
            // draft 1.509 -> 1.474 ms, W8A8 one node 1.205 -> 1.160 ms (eight
            // nodes 1.233 -> 1.247); 13B T = 32 5.575 -> 5.514 ms, skip-50%
            // one node 2.657 -> 2.640 ms.  Above 32 rows it also beats the
            // two-waves-per-SIMD form below (172 workgroups of eight): 7B
            // T = 64 3.739 -> 3.591 ms, T = 128 5.249 -> 5.126 ms (ctx 512),
            // 13B T = 64 6.339 -> 6.272 ms (T = 128 unchanged).  A grid of
            // exactly one workgroup per CU did worse: the 8B gate/up as 256
            // workgroups of seven 0.3-1.3% slower per forward (it keeps the
            // equal split), the 7B one as 256 of 5-6 tiles, alone, 32.5
            // against 31.5-32.0 us for 230-248.  A row's sums do not change.
            constexpr int EUC = NT == 8 ? 2 : S1::UC;  // the stage of the two-waves-per-SIMD form at 8 column tiles
            const int g6 = (tiles + 5) / 6, g7 = (tiles + 6) / 7;
            const bool gv1 = a.gv && a.T == 1;  // the GEMV-style tiles take one-row calls
            const int share = bw * bt;  // tiles per workgroup of the equal split
            if (share > 6 && !gv1 && g6 < 256) {
                hipLaunchKernelGGL((k_gemm_wide<WT, NT, EUC, S1::D, 6, 1, EPI, AT, false, false, false, false, KM, true>),
                                   dim3(g6), dim3(384), 0, s, a);
                return hipGetLastError();
            }
            if (share > 7 && !gv1 && g7 < 256) {
                hipLaunchKernelGGL((k_gemm_wide<WT, NT, EUC, S1::D, 7, 1, EPI, AT, false, false, false, false, KM, true>),
                                   dim3(g7), dim3(448), 0, s, a);
                return hipGetLastError();
            }
        }
        if constexpr (WT == ET_BF16 && NT >= 4) {
            // Trees of more than 32 rows do 2-4x the MFMA and LDS work per
            // weight byte (matrices the even split above does not take):
            // two waves per SIMD (workgroups of 8 one-tile waves, or 6 for 8
            // column tiles where 8 does not divide the
            // tile count into at least 128 workgroups) let one wave's MFMA
            // and LDS reads run under the other's loads.  Measured alone on
            // the 7B shapes: gate/up T = 128 53.3 -> 43.8 us, T = 64 35.1 ->
            // 34.5 us; QKV T = 128 42.9 -> 38.1 us (T = 64 keeps 3x1: 6x1
            // measured 27.6 against 22.3 us).  A row's sums do not change.
            if (tiles % 8 == 0 && tiles / 8 >= 128 && tiles / 8 <= 256) {
                hipLaunchKernelGGL((k_gemm_wide<WT, NT, 2, 4, 8, 1, EPI, AT, false, false, false, false, KM>), dim3(tiles / 8), dim3(512), 0, s,
                                   a);
                return hipGetLastError();
            }
            if (NT == 8 && tiles % 6 == 0 && tiles / 6 >= 96 && tiles / 6 <= 256) {
                hipLaunchKernelGGL((k_gemm_wide<WT, NT, 2, 4, 6, 1, EPI, AT, false, false, false, false, KM>), dim3(tiles / 6), dim3(384), 0, s,
                                   a);
                return hipGetLastError();
            }
        }
        if constexpr (NT == 2 && (WT == ET_BF16 || WT == ET_I8)) {
            if (a.gv && a.T == 1) {
                // GEMV-style tiles, same workgroup split (stage shapes measured
                // best alone at one row: 4x2 UC 2 D 4, 3x1 UC 4 D 4)
                if (bw == 4 && bt == 2)
                    hipLaunchKernelGGL((k_gemm_wide<WT, 2, 2, 4, 4, 2, EPI, AT, false, false, false, true, KM>), dim3(bg),
                                       dim3(256), 0, s, a);
                else if (bw == 3 && bt == 1)
                    hipLaunchKernelGGL((k_gemm_wide<WT, 2, 4, 4, 3, 1, EPI, AT, false, false, false, true, KM>), dim3(bg),
                                       dim3(192), 0, s, a);
                else if (bw == 4 && bt == 1)
                    hipLaunchKernelGGL((k_gemm_wide<WT, 2, 4, 4, 4, 1, EPI, AT, false, false, false, true, KM>), dim3(bg),
                                       dim3(256), 0, s, a);
                else
                    hipLaunchKernelGGL((k_gemm_wide<WT, 2, 2, 4, 3, 2, EPI, AT, false, false, false, true, KM>), dim3(bg),
                                       dim3(192), 0, s, a);
                return hipGetLastError();
            }
        }
        if constexpr (NT == 2 && WT == ET_I4) {
            if (rx_use(WT, a, 1)) {
                const unsigned lb = (unsigned)rx_lds_bytes(WT, a.T, a.Kp, 1);
                if (bw == 4 && bt == 1)
                    hipLaunchKernelGGL((k_gemm_wide<WT, 1, S1::UC, S1::D, 4, 1, EPI, AT, true, false, false, false, KM>), dim3(bg), dim3(256),
                                       lb, s, a);
                else if (bw == 3 && bt == 1)
                    hipLaunchKernelGGL((k_gemm_wide<WT, 1, S1::UC, S1::D, 3, 1, EPI, AT, true, false, false, false, KM>), dim3(bg), dim3(192),
                                       lb, s, a);
                else if (bw == 4)
                    hipLaunchKernelGGL((k_gemm_wide<WT, 1, S2::UC, S2::D, 4, 2, EPI, AT, true, false, false, false, KM>), dim3(bg), dim3(256),
                                       lb, s, a);
                else
                    hipLaunchKernelGGL((k_gemm_wide<WT, 1, S2::UC, S2::D, 3, 2, EPI, AT, true, false, false, false, KM>), dim3(bg), dim3(192),
                                       lb, s, a);
                return hipGetLastError();
            }
        }
        if (bw == 4 && bt == 1)
            hipLaunchKernelGGL((k_gemm_wide<WT, NT, S1::UC, S1::D, 4, 1, EPI, AT, false, false, false, false, KM>), dim3(bg), dim3(256), 0, s, a);
        else if (bw == 3 && bt == 1)
            hipLaunchKernelGGL((k_gemm_wide<WT, NT, S1::UC, S1::D, 3, 1, EPI, AT, false, false, false, false, KM>), dim3(bg), dim3(192), 0, s, a);
        else if (bw == 4)
            hipLaunchKernelGGL((k_gemm_wide<WT, NT, S2::UC, S2::D, 4, 2, EPI, AT, false, false, false, false, KM>), dim3(bg), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((k_gemm_wide<WT, NT, S2::UC, S2::D, 3, 2, EPI, AT, false, false, false, false, KM>), dim3(bg), dim3(192), 0, s, a);
        return hipGetLastError();
    }
    // (int4 at 8 column tiles: two steps per stage, so a shallower ring)
    constexpr int D = NT == 2 || (WT == ET_I4 && NT == 8) ? 2 : 4;
    hipLaunchKernelGGL((k_gemm<WT, NT, UC, D, 4, EPI, AT>), dim3(a.N / 16), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int WT, int EPI, typename AT, bool KM = false>
static hipError_t gemm_nt(const GemmArgs& a, hipStream_t s) {
    switch (col_tiles(a.T)) {
    case 2: return gemm_go<WT, 2, EPI, AT, KM>(a, s);
    case 4: return gemm_go<WT, 4, EPI, AT, KM>(a, s);
    default: return gemm_go<WT, 8, EPI, AT, KM>(a, s);
    }
}

hipError_t launch_gemm(int wtype, int atype, int epi, const GemmArgs& a, hipStream_t s) {
    if (a.N % 16 || a.Kp % chunk_k(wtype) || a.Kp < chunk_k(wtype) || a.T < 1 || a.T > 128)
        return hipErrorInvalidValue;
    const bool bf = atype == ET_BF16;
    switch (wtype) {
    case ET_F32:
        switch (epi) {
        case EPI_STORE:
            return a.kmaj ? gemm_nt<ET_F32, EPI_STORE, float, true>(a, s) : gemm_nt<ET_F32, EPI_STORE, float>(a, s);
        case EPI_RESID: return gemm_nt<ET_F32, EPI_RESID, float>(a, s);
        case EPI_SWIGLU: return gemm_nt<ET_F32, EPI_SWIGLU, float, true>(a, s);
        case EPI_QKV: return gemm_nt<ET_F32, EPI_QKV, float>(a, s);
        }
        break;
    case ET_BF16:
        switch (epi) {
        case EPI_STORE:
            return a.kmaj ? gemm_nt<ET_BF16, EPI_STORE, uint16_t, true>(a, s)
                          : gemm_nt<ET_BF16, EPI_STORE, uint16_t>(a, s);
        case EPI_RESID: return gemm_nt<ET_BF16, EPI_RESID, uint16_t>(a, s);
        case EPI_SWIGLU: return gemm_nt<ET_BF16, EPI_SWIGLU, uint16_t, true>(a, s);
        case EPI_QKV: return gemm_nt<ET_BF16, EPI_QKV, uint16_t>(a, s);
        }
        break;
    case ET_I8:
        switch (epi) {
        case EPI_STORE: return gemm_nt<ET_I8, EPI_STORE, float>(a, s);
        case EPI_RESID: return gemm_nt<ET_I8, EPI_RESID, float>(a, s);
        case EPI_RAW: return gemm_nt<ET_I8, EPI_RAW, float>(a, s);
        case EPI_SWIGLU:
            return bf ? gemm_nt<ET_I8, EPI_SWIGLU, uint16_t, true>(a, s) : gemm_nt<ET_I8, EPI_SWIGLU, float, true>(a, s);
        case EPI_QKV:
            return bf ? gemm_nt<ET_I8, EPI_QKV, uint16_t>(a, s) : gemm_nt<ET_I8, EPI_QKV, float>(a, s);
        }
        break;
    case ET_I4:
        switch (epi) {
        case EPI_STORE: return gemm_nt<ET_I4, EPI_STORE, float>(a, s);
        case EPI_RESID: return gemm_nt<ET_I4, EPI_RESID, float>(a, s);
        case EPI_RAW: return gemm_nt<ET_I4, EPI_RAW, float>(a, s);
        case EPI_SWIGLU:
            return bf ? gemm_nt<ET_I4, EPI_SWIGLU, uint16_t>(a, s) : gemm_nt<ET_I4, EPI_SWIGLU, float>(a, s);
        case EPI_QKV:
            return bf ? gemm_nt<ET_I4, EPI_QKV, uint16_t>(a, s) : gemm_nt<ET_I4, EPI_QKV, float>(a, s);
        }
        break;
    }
    return hipErrorInvalidValue;
}

// The split count depends on the matrix only, never on T, so a row's sums
// are the same for every tree size (greedy speculative output then equals
// greedy decoding bit for bit, not only up to near-ties).
int gemm_parts_count(int wtype, int N, int Kp, int T) {
    if (N % 64 || T < 1 || T > 128) return 1;
    const int groups = N / 64;  // four 16-row tiles per workgroup
    if (groups >= 192) return 1;
    const int C = Kp / chunk_k(wtype);
    int ks = std::min(8, 256 / groups);
    ks = std::min(ks, C / 2);
    return ks >= 2 ? ks : 1;
}

template <int WT, typename AT>
static hipError_t gemm_parts_go(const GemmArgs& a, hipStream_t s) {
    const dim3 grid(a.N / 64, a.ksplit);
    if (a.kmaj) return hipErrorInvalidValue;  // residual projections stay tile-major
    if (a.mx_o) {
        if constexpr (WT == ET_BF16) {
            hipLaunchKernelGGL((k_gemm_wide<WT, 1, 4, 2, 4, 1, EPI_STORE, AT, true, false, true>), grid, dim3(256),
                               (unsigned)rx_lds_bytes(WT, a.T, a.Kp, a.ksplit), s, a);
            return hipGetLastError();
        }
        return hipErrorInvalidValue;
    }
    if (a.qx) {
        if constexpr (is_int<WT>()) {
            hipLaunchKernelGGL((k_gemm_wide<WT, 1, 4, 2, 4, 1, EPI_STORE, AT, true, true>), grid, dim3(256),
                               (unsigned)rx_lds_bytes(WT, a.T, a.Kp, a.ksplit), s, a);
            return hipGetLastError();
        }
        return hipErrorInvalidValue;
    }
    if constexpr (WT == ET_I4) {
        if (rx_use(WT, a, a.ksplit)) {
            hipLaunchKernelGGL((k_gemm_wide<WT, 1, 4, 2, 4, 1, EPI_STORE, AT, true>), grid, dim3(256),
                               (unsigned)rx_lds_bytes(WT, a.T, a.Kp, a.ksplit), s, a);
            return hipGetLastError();
        }
    }
    if constexpr (WT == ET_BF16) {
        // short K ranges (at most 8 chunks per split: the 7B and 8B O
        // projections) at up to 32 rows: workgroups of two one-tile waves,
        // twice as many.  Same K ranges and per-tile sums.  Measured alone
        // with cold weights, 7B O at T = 32: 12.7 -> 11.4 us; the down
        // projection (21.5 chunks per split) was slower this way, 19.2 ->
        // 20.6 us.
        if (col_tiles(a.T) == 2 && a.Kp / chunk_k(WT) <= 8 * a.ksplit) {
            hipLaunchKernelGGL((k_gemm_wide<WT, 2, 4, 2, 2, 1, EPI_STORE, AT, false>), dim3(a.N / 32, a.ksplit),
                               dim3(128), 0, s, a);
            return hipGetLastError();
        }
    }
    switch (col_tiles(a.T)) {
    case 2: hipLaunchKernelGGL((k_gemm_wide<WT, 2, 4, 2, 4, 1, EPI_STORE, AT, false>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_gemm_wide<WT, 4, 2, 4, 4, 1, EPI_STORE, AT, false>), grid, dim3(256), 0, s, a); break;
    default:
        hipLaunchKernelGGL((k_gemm_wide<WT, 8, stage_uc<WT, 1>(), 4, 4, 1, EPI_STORE, AT, false>), grid, dim3(256), 0,
                           s, a);
        break;
    }
    return hipGetLastError();
}

hipError_t launch_gemm_parts(int wtype, const GemmArgs& a, hipStream_t s) {
    if (a.N % 64 || a.Kp % chunk_k(wtype) || a.Kp < chunk_k(wtype) || a.T < 1 || a.T > 128 || a.ksplit < 2 ||
        a.ksplit > 8 || a.part_stride < (size_t)a.T * a.ldo)
        return hipErrorInvalidValue;
    if (wtype == ET_BF16) return gemm_parts_go<ET_BF16, uint16_t>(a, s);
    if (wtype == ET_F32) return gemm_parts_go<ET_F32, float>(a, s);
    // int8: each split dequantises its own int32 sums, (acc * xs[t]) * ws[n]
    if (wtype == ET_I8) return gemm_parts_go<ET_I8, float>(a, s);
    if (wtype == ET_I4) return gemm_parts_go<ET_I4, float>(a, s);
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------- operand tiling

// Row-major weights -> tiled: one thread per 16-byte destination fragment.
template <typename T>
__global__ void k_tile_weight(const T* src, int rows, int K, int Kp, T* dst, int row0, int mode, int hd, int kt) {
    constexpr int E = 16 / sizeof(T);
    const int fpr = Kp / E;
    const size_t total = (size_t)rows * fpr;
    for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        const int i = (int)(idx / fpr), k0 = (int)(idx % fpr) * E;
        int dr;
        if (mode == 1) {
            const int head = i / hd, j = i % hd, half = hd / 2;
            dr = head * hd + (j < half ? 2 * j : 2 * (j - half) + 1);
        } else if (mode == 2) {
            dr = 2 * i;
        } else {
            dr = i;
        }
        size_t off = wt_off(row0 + dr, k0, Kp, E);
        if (kt) off = wt_kmajor(off * sizeof(T), kt, Kp * (int)sizeof(T) / 64) / sizeof(T);
        T* o = dst + off;
#pragma unroll
        for (int e = 0; e < E; ++e) o[e] = (k0 + e < K) ? src[(size_t)i * K + k0 + e] : (T)0;
    }
}

// Row-major activations -> tiled (pad rows and pad columns are zero).
template <typename T>
__global__ void k_tile_act(const T* src, int Tn, int K, int Kp, int NT, T* dst) {
    constexpr int E = 16 / sizeof(T);
    const int fpr = Kp / E;
    const size_t total = (size_t)NT * 16 * fpr;
    for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        const int t = (int)(idx / fpr), k0 = (int)(idx % fpr) * E;
        T* o = dst + xt_off(t, k0, NT, E);
#pragma unroll
        for (int e = 0; e < E; ++e) o[e] = (t < Tn && k0 + e < K) ? src[(size_t)t * K + k0 + e] : (T)0;
    }
}

// Tiled activations -> row-major [Tn][K] (the inverse of k_tile_act; for the
// kernel-level entry points that return a fused kernel's tiled output).
template <typename T>
__global__ void k_untile_act(const T* src, int Tn, int K, int NT, T* dst) {
    constexpr int E = 16 / sizeof(T);
    const int fpr = (K + E - 1) / E;
    const size_t total = (size_t)Tn * fpr;
    for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        const int t = (int)(idx / fpr), k0 = (int)(idx % fpr) * E;
        const T* i = src + xt_off(t, k0, NT, E);
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (k0 + e < K) dst[(size_t)t * K + k0 + e] = i[e];
    }
}

static unsigned grid_for(size_t n) {
    size_t b = (n + 255) / 256;
    if (b > 16384) b = 16384;
    return (unsigned)(b ? b : 1);
}

hipError_t launch_tile_weight(int atype, const void* src, int rows, int K, void* dst, int row0, int mode, int hd,
                              hipStream_t s, int kt) {
    const int Kp = pad_k(K, atype);
    const size_t n = (size_t)rows * (Kp / frag_elems(atype));
    if (kt < 0) return hipErrorInvalidValue;
    if (atype == ET_BF16)
        hipLaunchKernelGGL(k_tile_weight<uint16_t>, dim3(grid_for(n)), dim3(256), 0, s, (const uint16_t*)src, rows, K,
                           Kp, (uint16_t*)dst, row0, mode, hd, kt);
    else if (atype == ET_F32)
        hipLaunchKernelGGL(k_tile_weight<float>, dim3(grid_for(n)), dim3(256), 0, s, (const float*)src, rows, K, Kp,
                           (float*)dst, row0, mode, hd, kt);
    else
        hipLaunchKernelGGL(k_tile_weight<int8_t>, dim3(grid_for(n)), dim3(256), 0, s, (const int8_t*)src, rows, K, Kp,
                           (int8_t*)dst, row0, mode, hd, kt);
    return hipGetLastError();
}

hipError_t launch_tile_act(int atype, const void* src, int Tn, int K, void* dst, hipStream_t s) {
    const int Kp = pad_k(K, atype), NT = col_tiles(Tn);
    const size_t n = (size_t)NT * 16 * (Kp / frag_elems(atype));
    if (atype == ET_BF16)
        hipLaunchKernelGGL(k_tile_act<uint16_t>, dim3(grid_for(n)), dim3(256), 0, s, (const uint16_t*)src, Tn, K, Kp,
                           NT, (uint16_t*)dst);
    else if (atype == ET_F32)
        hipLaunchKernelGGL(k_tile_act<float>, dim3(grid_for(n)), dim3(256), 0, s, (const float*)src, Tn, K, Kp, NT,
                           (float*)dst);
    else
        hipLaunchKernelGGL(k_tile_act<int8_t>, dim3(grid_for(n)), dim3(256), 0, s, (const int8_t*)src, Tn, K, Kp, NT,
                           (int8_t*)dst);
    return hipGetLastError();
}

hipError_t launch_untile_act(int atype, const void* src, int Tn, int K, void* dst, hipStream_t s) {
    const int NT = col_tiles(Tn);
    const size_t n = (size_t)Tn * ((K + frag_elems(atype) - 1) / frag_elems(atype));
    if (atype == ET_BF16)
        hipLaunchKernelGGL(k_untile_act<uint16_t>, dim3(grid_for(n)), dim3(256), 0, s, (const uint16_t*)src, Tn, K, NT,
                           (uint16_t*)dst);
    else if (atype == ET_F32)
        hipLaunchKernelGGL(k_untile_act<float>, dim3(grid_for(n)), dim3(256), 0, s, (const float*)src, Tn, K, NT,
                           (float*)dst);
    else
        hipLaunchKernelGGL(k_untile_act<int8_t>, dim3(grid_for(n)), dim3(256), 0, s, (const int8_t*)src, Tn, K, NT,
                           (int8_t*)dst);
    return hipGetLastError();
}

// ---------------------------------------------------------------- attention

// Store 4 consecutive k (k4 a multiple of 4) of one row into tiled
// activations: they are contiguous inside one fragment.
__device__ __forceinline__ void st4(float* out, size_t o, float a, float b, float c, float d) {
    *(float4*)(out + o) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void st4(uint16_t* out, size_t o, float a, float b, float c, float d) {
    const uint32_t lo = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
    const uint32_t hi = (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16);
    *(uint2*)(out + o) = make_uint2(lo, hi);
}

__device__ __forceinline__ void st4q(int8_t* q, size_t o, float a, float b, float c, float d) {
    const uint32_t v = (uint32_t)(uint8_t)(int8_t)a | ((uint32_t)(uint8_t)(int8_t)b << 8) |
                       ((uint32_t)(uint8_t)(int8_t)c << 16) | ((uint32_t)(uint8_t)(int8_t)d << 24);
    *(uint32_t*)(q + o) = v;
}

// A workgroup covers 4 waves x ATT_TPW key tiles of 32 slots.
static constexpr int ATT_WAVES = 4;
static constexpr int ATT_TPW = 2;
static constexpr int ATT_SPLIT = ATT_WAVES * ATT_TPW * 32;
static constexpr int ATT_MAX_SPLITS = 64;  // contexts up to 16384 slots

int attention_splits(int n_slots) { return (n_slots + ATT_SPLIT - 1) / ATT_SPLIT; }

// Key tiles of a windowed forward: the tiles holding the sink slots, then the
// tiles from the window's first slot to the last tree slot.  Logical tile lt
// is physical tile lt (lt < st) or lt - st + pt0.  Without a window every
// committed slot is visible (csink = wstart = Lc) and the map is the identity.
struct AttnWindow {
    int csink, wstart, st, pt0, n_log;
    __host__ __device__ AttnWindow(int Lc, int n_tree, int win_sink, int win_len) {
        const int n_tiles = (Lc + n_tree + 31) >> 5;
        if (win_len > 0) {
            csink = win_sink < Lc ? win_sink : Lc;
            wstart = Lc - win_len > csink ? Lc - win_len : csink;
            st = (csink + 31) >> 5;
            pt0 = (wstart >> 5) > st ? (wstart >> 5) : st;
            n_log = st + (n_tiles - pt0);
        } else {
            csink = wstart = Lc;
            st = n_tiles;
            pt0 = 0;
            n_log = n_tiles;
        }
    }
    __host__ __device__ int phys(int lt) const { return lt < st ? lt : lt - st + pt0; }
};

int attention_splits_win(int Lc, int n_tree, int win_sink, int win_len) {
    const AttnWindow w(Lc, n_tree, win_sink, win_len);
    return (w.n_log * 32 + ATT_SPLIT - 1) / ATT_SPLIT;
}
size_t attention_work_bytes(int n_slots, int T, int H, int hd) {
    const size_t S = (size_t)attention_splits(n_slots);
    return S * H * T * (size_t)hd * 4 + S * H * T * 2 * 4 + 256;
}

// Butterfly max / sum with the lane 16 and lane 32 apart, through the
// cross-lane swap instructions (no LDS round trip).  Both lanes of a pair get
// the same operands in the same order, so their results are bit-identical.
__device__ __forceinline__ float pair_max16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_max32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair_sum32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ bool anc_bit(uint64_t a0, uint64_t a1, int node) {
    return node < 64 ? ((a0 >> node) & 1ull) : ((a1 >> (node - 64)) & 1ull);
}

// Softmax state of one part (NTL key tiles) for the rows of a 16-row query
// tile, in two steps: attn_part_max gives the scores of visible slots
// scaled to log2 units and their maximum m (at least -1e30, so an empty part
// gives exp2 weights of 0); attn_part_probs gives the probabilities as bf16
// hi + lo pairs in the P-operand order and their sum l.  Both attention
// kernels use these and the merge helpers below with FP contraction off, so
// they round every row the same way.
// Bits e in [lo, hi) of an 8-bit mask.
__device__ __forceinline__ uint32_t bits8(int lo, int hi) {
    lo = max(lo, 0);
    hi = min(hi, 8);
    return lo < hi ? (0xffu >> (8 - (hi - lo))) << lo : 0u;
}
// Visibility of the 8 slots base .. base + 7 for one query row: committed
// slots in [0, csink) or [wstart, Lc), tree slots whose node is an
// ancestor-or-self (bit of the row's 128-bit mask), nothing at or past
// n_slots.  Shifts and range masks instead of a test per slot.
__device__ __forceinline__ uint32_t attn_vis8(int base, int Lc, int n_slots, const AttnWindow& win, uint64_t an0,
                                              uint64_t an1) {
    const uint32_t c = bits8(-base, win.csink - base) | bits8(win.wstart - base, Lc - base);
    const int n0 = base - Lc;  // tree node of bit 0 (negative: bit -n0 holds node 0)
    uint32_t t = 0;
    if (n0 >= 64 && n0 < 128) t = (uint32_t)(an1 >> (n0 - 64));
    else if (n0 > 0 && n0 < 64) t = (uint32_t)((an0 >> n0) | (an1 << (64 - n0)));
    else if (n0 == 0) t = (uint32_t)an0;
    else if (n0 > -8 && n0 < 0) t = (uint32_t)(an0 << (-n0));
    return c | (t & bits8(Lc - base, n_slots - base));
}
template <int NTL>
__device__ __forceinline__ void attn_part_scores(const f32x4 (&S)[NTL][2], const int* ptile, const bool* live, int g,
                                                 int Lc, int n_slots, const AttnWindow& win, uint64_t an0,
                                                 uint64_t an1, float scale_log2, float (&x)[NTL][8]) {
#pragma clang fp contract(off)
#pragma unroll
    for (int tt = 0; tt < NTL; ++tt) {
        const uint32_t vm = live[tt] ? attn_vis8(ptile[tt] * 32 + 8 * g, Lc, n_slots, win, an0, an1) : 0u;
        if (__all(vm == 0xffu)) {  // a tile every lane sees whole (all committed tiles without a window)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                for (int i = 0; i < 4; ++i) x[tt][4 * h2 + i] = S[tt][h2][i] * scale_log2;
        } else {
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    x[tt][4 * h2 + i] = (vm >> (4 * h2 + i)) & 1u ? S[tt][h2][i] * scale_log2 : -INFINITY;
        }
    }
}
template <int NTL>
__device__ __forceinline__ float attn_part_max(const float (&x)[NTL][8]) {
    float mt = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < NTL; ++tt)
#pragma unroll
        for (int e = 0; e < 8; ++e) mt = fmaxf(mt, x[tt][e]);
    return fmaxf(-1e30f, pair_max32(pair_max16(mt)));
}
template <int NTL>
__device__ __forceinline__ float attn_part_probs(const float (&x)[NTL][8], float mn, i32x4 (&Pf)[NTL],
                                                 i32x4 (&Pl)[NTL]) {
#pragma clang fp contract(off)
    float ps = 0.f;
#pragma unroll
    for (int tt = 0; tt < NTL; ++tt) {
        uint16_t pb[8], pl[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float p = __builtin_amdgcn_exp2f(x[tt][e] - mn);
            ps += p;
            pb[e] = f2bf(p);
            pl[e] = f2bf(p - bf2f(pb[e]));  // exact difference, rounded: p = hi + lo to ~2^-17
        }
        Pf[tt] = i32x4{(int)(pb[0] | ((uint32_t)pb[1] << 16)), (int)(pb[2] | ((uint32_t)pb[3] << 16)),
                       (int)(pb[4] | ((uint32_t)pb[5] << 16)), (int)(pb[6] | ((uint32_t)pb[7] << 16))};
        Pl[tt] = i32x4{(int)(pl[0] | ((uint32_t)pl[1] << 16)), (int)(pl[2] | ((uint32_t)pl[3] << 16)),
                       (int)(pl[4] | ((uint32_t)pl[5] << 16)), (int)(pl[6] | ((uint32_t)pl[7] << 16))};
    }
    return pair_sum32(pair_sum16(ps));
}

// The in-order merge of part states under the common maximum M: weight
// exp2(m - M) of a part, then acc = fma(weight, o, acc), L = fma(weight, l, L).
__device__ __forceinline__ float attn_merge_weight(float m, float M) { return exp2f(m - M); }
__device__ __forceinline__ void attn_merge_o(f32x4& acc, const f32x4 o, float f) {
    acc = f32x4{fmaf(o[0], f, acc[0]), fmaf(o[1], f, acc[1]), fmaf(o[2], f, acc[2]), fmaf(o[3], f, acc[3])};
}
__device__ __forceinline__ void attn_merge_l(float& L, float l, float f) { L = fmaf(l, f, L); }

// Query rows of a kv head: its G query heads x T tokens, each head's rows
// padded to Rp and packed into 16-row tiles, row p = 16 tile + r holding
// token p % Rp of head p / Rp of the group.  Up to 16 tokens Rp = T, so the
// heads' rows follow each other (a one-node call of a 4-head group fills one
// tile instead of four, and the group's K/V pass serves every head; a head's
// rows may straddle two tiles); above, Rp rounds T up to 16.  A row's
// arithmetic does not depend on where it sits in its tile.
__host__ __device__ inline int attn_head_rows(int T) { return T <= 16 ? T : (T + 15) & ~15; }
__host__ __device__ inline int attn_query_tiles(int T, int G) { return (G * attn_head_rows(T) + 15) / 16; }

// Workgroup = (split of KV slots, kv head, JT query tiles of 16 rows); each
// of the four waves owns one part (two key tiles) of the split.  The query
// rows of a kv head are its G query heads x T tokens, packed into tiles as
// attn_head_rows describes, so GQA groups share every K/V fragment.  Scores come
// out of the QK^T MFMA with slots along the row index; the cache puts slots
// 8g..8g+7 of a tile in lane group g, which is exactly the k-order of the P
// operand of the PV MFMA, so probabilities never leave registers.  Each wave
// issues its query fragments and then the K and V fragments of its tiles in
// the order they are consumed, before any arithmetic.  The four waves put
// their states in LDS (one barrier) and the workgroup writes the split's
// partial as float4 runs, waves summed in wave order; k_attn_merge then
// merges the splits in split order (deterministic).  (Merging inside this
// kernel by its last-arriving workgroup needs device-scope fences that cost
// more than the separate launch on gfx950.)
template <int HD, int JT, int TPW = ATT_TPW>
__global__ void __launch_bounds__(256) k_attn_bf16(const AttnArgs a, float scale_log2) {
    constexpr int UD = HD / 32;   // k-steps of QK^T over head_dim
    constexpr int DG = HD / 4;    // head_dim span of one lane group
    constexpr int NDT = HD / 16;  // output d tiles
    constexpr int TE = 32 * HD;   // elements per key tile
    constexpr int RS = HD + 4;    // LDS row stride of the wave states (floats; conflict-free float4 rows)
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int split = blockIdx.x, kvh = blockIdx.y, rc = blockIdx.z;
    const int Lc = a.sp->Lc, n_tree = a.sp->n_tree, n_slots = Lc + n_tree;
    if (!dcheck(a.chk, Lc >= 0 && n_slots <= a.sp->cap && a.sp->cap <= a.ctx_cap, CHK_ATTN_SLOTS)) return;
    const int n_tiles = (n_slots + 31) >> 5;
    const AttnWindow win(Lc, n_tree, a.win_sink, a.win_len);
    const int T = a.T, G = a.H / a.Hkv, Rp = attn_head_rows(T);
    const int nct = attn_query_tiles(T, G);
    const uint16_t* q = (const uint16_t*)a.q;

    // query fragments of the JT 16-row tiles; lane row r is row 16 ct + r of
    // the kv head's packed rows (rows past the group's read a valid row and
    // are zeroed below, so every load is unconditional)
    bool rv[JT];
    i32x4 Qf[JT][UD];
    uint64_t an0[JT], an1[JT];
#pragma unroll
    for (int j = 0; j < JT; ++j) {
        const int ct = JT * rc + j, p = ct * 16 + r, hg = p / Rp, tr = p % Rp;
        rv[j] = ct < nct && hg < G && tr < T;
        const int t = min(tr, T - 1), head = kvh * G + min(hg, G - 1);
#pragma unroll
        for (int u = 0; u < UD; ++u) Qf[j][u] = *(const i32x4*)(q + ((size_t)t * a.H + head) * HD + g * DG + u * 8);
        an0[j] = a.anc[2 * t];
        an1[j] = a.anc[2 * t + 1];
    }
    // K and V fragments of this wave's tiles, in the order they are consumed
    const uint16_t* kbase = (const uint16_t*)a.kc + (size_t)kvh * a.ctx_cap * HD + lane * 8;
    const uint16_t* vbase = (const uint16_t*)a.vt + (size_t)kvh * a.ctx_cap * HD + lane * 8;
    const int tile0 = (split * ATT_WAVES + wave) * TPW;  // logical key tiles of this wave
    int ptile[TPW];
    bool live[TPW];
    i32x4 Kf[TPW][2][UD], Vf[TPW][NDT];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
        live[tt] = tile0 + tt < win.n_log;
        ptile[tt] = live[tt] ? win.phys(tile0 + tt) : n_tiles - 1;
        const size_t tb = (size_t)ptile[tt] * TE;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
            for (int u = 0; u < UD; ++u) Kf[tt][h2][u] = *(const i32x4*)(kbase + tb + (h2 * UD + u) * 512);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) Vf[tt][dt] = *(const i32x4*)(vbase + tb + dt * 512);
    }
    const i32x4 zero = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < JT; ++j) {
        if (!rv[j]) {
#pragma unroll
            for (int u = 0; u < UD; ++u) Qf[j][u] = zero;
            an0[j] = an1[j] = 0ull;
        }
    }

    // all of the wave's tiles form one block: scores first, then a single
    // softmax pass (no running rescale), then P V.  Slots past the context
    // and masked slots get probability 0; a wave with no visible slot keeps
    // m = -1e30, l = 0 and contributes nothing to the merge.
    f32x4 S[JT][TPW][2];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
            for (int j = 0; j < JT; ++j) {
                S[j][tt][h2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int u = 0; u < UD; ++u) S[j][tt][h2] = mfma_step<ET_BF16>(Kf[tt][h2][u], Qf[j][u], S[j][tt][h2]);
            }
    float m[JT], l[JT];
    i32x4 Pf[JT][TPW], Pl[JT][TPW];
#pragma unroll
    for (int j = 0; j < JT; ++j) {
        float x[TPW][8];
        attn_part_scores<TPW>(S[j], ptile, live, g, Lc, n_slots, win, an0[j], an1[j], scale_log2, x);
        m[j] = attn_part_max<TPW>(x);
        l[j] = attn_part_probs<TPW>(x, m[j], Pf[j], Pl[j]);
    }
    // P V with the probabilities as a two-term bf16 sum (hi + lo): the
    // product carries them to fp32-level accuracy; V is exact in bf16
    f32x4 O[NDT][JT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int j = 0; j < JT; ++j) {
            O[dt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int tt = 0; tt < TPW; ++tt) {
                O[dt][j] = mfma_step<ET_BF16>(Vf[tt][dt], Pf[j][tt], O[dt][j]);
                O[dt][j] = mfma_step<ET_BF16>(Vf[tt][dt], Pl[j][tt], O[dt][j]);
            }
        }

    // ---- merge the four waves: states to LDS, one barrier, then each
    // (row, 4 d) of the split is the wave-order sum of the rescaled states
    __shared__ float sm_m[ATT_WAVES][JT][16], sm_l[ATT_WAVES][JT][16];
    __shared__ __attribute__((aligned(16))) float sm_o[ATT_WAVES][JT][16][RS];
    if (g == 0) {
#pragma unroll
        for (int j = 0; j < JT; ++j) {
            sm_m[wave][j][r] = m[j];
            sm_l[wave][j][r] = l[j];
        }
    }
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int j = 0; j < JT; ++j) *(f32x4*)(&sm_o[wave][j][r][16 * dt + 4 * g]) = O[dt][j];
    __syncthreads();
    constexpr int D4 = HD / 4;
    for (int idx = threadIdx.x; idx < JT * 16 * D4; idx += 64 * ATT_WAVES) {
        const int j = idx / (16 * D4), rr = (idx / D4) & 15, d4 = (idx % D4) * 4;
        const int ct = JT * rc + j, p = ct * 16 + rr, hg = p / Rp, t = p % Rp;
        if (ct >= nct || hg >= G || t >= T) continue;
        float mw[ATT_WAVES], M = -1e30f;
#pragma unroll
        for (int w = 0; w < ATT_WAVES; ++w) {
            mw[w] = sm_m[w][j][rr];
            M = fmaxf(M, mw[w]);
        }
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < ATT_WAVES; ++w) {
            const float f = attn_merge_weight(mw[w], M);
            attn_merge_o(acc, *(const f32x4*)(&sm_o[w][j][rr][d4]), f);
            attn_merge_l(L, sm_l[w][j][rr], f);
        }
        const size_t o = ((size_t)split * a.H + kvh * G + hg) * T + t;
        *(f32x4*)(a.part_o + o * HD + d4) = acc;
        if (d4 == 0) *(float2*)(a.part_ml + o * 2) = make_float2(M, L);
    }
}

// Workgroup = (split of KV slots, kv head, QT query tiles of 16 rows): each
// wave owns one query tile and the split's K and V pass once through LDS for
// all of them, so a K/V byte leaves L2 once per QT tiles instead of once per
// tile (grouped-query heads and large trees have many tiles per kv head).
// Each wave computes, for its rows, the same four part states (two key tiles
// each) as k_attn_bf16's four waves, with the same helpers, and merges them in
// part order in registers: the partials are the same bits either way, so the
// choice between the two kernels never changes a row's result.  NH = 1:
// the split's K and then its V pass through a 64 KB LDS stage, all loads
// issued up front (two workgroups per CU).  NH = 2: they pass in halves (the
// K of parts 0-1, then of parts 2-3, then their V the same way), so a
// workgroup holds half the LDS and staging registers and three fit on a CU;
// grids of more than one workgroup per CU take it (8B 64 nodes at 4096, 544
// workgroups: 30.6 -> 26.4 us per layer; 7B 48-128 nodes at 8192 2-5%
// faster), smaller grids keep the single stage (7B 128 nodes at 512, 192
// workgroups: 16.4 against 17.4 us).
template <int HD, int QT, int NH>
__global__ void __launch_bounds__(64 * QT, NH == 1 ? 2 : 3) k_attn_rows(const AttnArgs a, float scale_log2) {
    constexpr int UD = HD / 32, DG = HD / 4, NDT = HD / 16, TE = 32 * HD;
    constexpr int NP = ATT_WAVES;        // part states per split
    constexpr int NTS = NP * ATT_TPW;    // key tiles per split
    constexpr int NTH = NTS / NH;        // key tiles per stage
    constexpr int KF = 2 * UD;           // 1 KB fragments per K tile (V: NDT)
    constexpr int FH = NTH * KF;         // fragments per stage, K and V alike
    constexpr int LPH = FH / QT;         // fragments each wave stages per stage
    static_assert(KF == NDT && FH % QT == 0 && NP % NH == 0 && (NH == 1 || NH == 2), "K and V stages must match");
    __shared__ i32x4 kv[FH * 64];        // one stage of the split's K or V (NH 1: 64 KB for head_dim 128)
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int split = blockIdx.x, kvh = blockIdx.y;
    const int Lc = a.sp->Lc, n_tree = a.sp->n_tree, n_slots = Lc + n_tree;
    if (!dcheck(a.chk, Lc >= 0 && n_slots <= a.sp->cap && a.sp->cap <= a.ctx_cap, CHK_ATTN_SLOTS)) return;
    const int n_tiles = (n_slots + 31) >> 5;
    const AttnWindow win(Lc, n_tree, a.win_sink, a.win_len);
    const int T = a.T, Tp = (T + 15) & ~15, G = a.H / a.Hkv;
    const int nct = G * Tp / 16;
    const int ct = QT * blockIdx.z + wave;
    const bool tv = ct < nct;
    const int hg = tv ? (ct * 16) / Tp : 0, t0 = (ct * 16) % Tp, head = kvh * G + hg;
    const uint16_t* q = (const uint16_t*)a.q;

    i32x4 Qf[UD];
    {
        const int t = min(t0 + r, T - 1);
#pragma unroll
        for (int u = 0; u < UD; ++u) Qf[u] = *(const i32x4*)(q + ((size_t)t * a.H + head) * HD + g * DG + u * 8);
    }
    int ptile[NTS];
    bool live[NTS];
#pragma unroll
    for (int tt = 0; tt < NTS; ++tt) {
        live[tt] = split * NTS + tt < win.n_log;
        ptile[tt] = live[tt] ? win.phys(split * NTS + tt) : n_tiles - 1;
    }
    // every wave stages LPH of each stage's 1 KB fragments (one lane-wide
    // load each): fragment f of stage h is fragment h * FH + f of the split
    const uint16_t* kbase = (const uint16_t*)a.kc + (size_t)kvh * a.ctx_cap * HD + lane * 8;
    const uint16_t* vbase = (const uint16_t*)a.vt + (size_t)kvh * a.ctx_cap * HD + lane * 8;
    // (the physical tile of a fragment computed, not looked up: a run-time
    // index into ptile would move that array to LDS)
    auto phys = [&](int tt) { return split * NTS + tt < win.n_log ? win.phys(split * NTS + tt) : n_tiles - 1; };
    auto kfrag = [&](int h, int i) -> const i32x4* {
        const int f = h * FH + wave * LPH + i;
        return (const i32x4*)(kbase + (size_t)phys(f / KF) * TE + (f % KF) * 512);
    };
    auto vfrag = [&](int h, int i) -> const i32x4* {
        const int f = h * FH + wave * LPH + i;
        return (const i32x4*)(vbase + (size_t)phys(f / NDT) * TE + (f % NDT) * 512);
    };
    // NH 2: K halves 0 and 1 (later V halves 0 and 1); NH 1: K and V
    i32x4 St0[LPH], St1[LPH];
#pragma unroll
    for (int i = 0; i < LPH; ++i) St0[i] = *kfrag(0, i);
#pragma unroll
    for (int i = 0; i < LPH; ++i) St1[i] = NH == 2 ? *kfrag(1, i) : *vfrag(0, i);
    uint64_t an0 = a.anc[2 * min(t0 + r, T - 1)], an1 = a.anc[2 * min(t0 + r, T - 1) + 1];
    if (!(tv && t0 + r < T)) {
#pragma unroll
        for (int u = 0; u < UD; ++u) Qf[u] = i32x4{0, 0, 0, 0};
        an0 = an1 = 0ull;
    }

    // scores of the split's tiles, stage by stage
    f32x4 S[NP][ATT_TPW][2];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        if (h) __syncthreads();  // every wave is done with the first half
#pragma unroll
        for (int i = 0; i < LPH; ++i) kv[(wave * LPH + i) * 64 + lane] = h ? St1[i] : St0[i];
        __syncthreads();
#pragma unroll
        for (int th = 0; th < NTH; ++th) {
            const int tt = h * NTH + th;
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int u = 0; u < UD; ++u) acc = mfma_step<ET_BF16>(kv[(th * KF + h2 * UD + u) * 64 + lane], Qf[u], acc);
                S[tt / ATT_TPW][tt % ATT_TPW][h2] = acc;
            }
            // one tile's fragments in registers at a time (three waves per SIMD)
            if constexpr (NH == 2) __builtin_amdgcn_sched_barrier(0);
        }
    }
    if constexpr (NH == 2) {
        // the first half of V, in flight while the scores are scaled and masked
#pragma unroll
        for (int i = 0; i < LPH; ++i) St0[i] = *vfrag(0, i);
    }

    // the parts' scaled, masked scores and maxima first (the merge weights
    // need the maximum over parts), then part by part: probabilities, P V,
    // and the merge step
    float x[NP][ATT_TPW][8], m[NP], M = -1e30f;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        attn_part_scores<ATT_TPW>(S[p], &ptile[p * ATT_TPW], &live[p * ATT_TPW], g, Lc, n_slots, win, an0, an1,
                                  scale_log2, x[p]);
        m[p] = attn_part_max<ATT_TPW>(x[p]);
        M = fmaxf(M, m[p]);
    }
    f32x4 acc[NDT];
    float L = 0.f;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        __syncthreads();  // every wave is done with the LDS stage it read last
#pragma unroll
        for (int i = 0; i < LPH; ++i) kv[(wave * LPH + i) * 64 + lane] = NH == 1 || h ? St1[i] : St0[i];
        __syncthreads();
        if (NH == 2 && h == 0) {
            // the second half of V, in flight during the first half's P V
#pragma unroll
            for (int i = 0; i < LPH; ++i) St1[i] = *vfrag(1, i);
        }
#pragma unroll
        for (int ph = 0; ph < NP / NH; ++ph) {
            const int p = h * (NP / NH) + ph;
            i32x4 Pf[ATT_TPW], Pl[ATT_TPW];
            const float lp = attn_part_probs<ATT_TPW>(x[p], m[p], Pf, Pl);
            const float f = attn_merge_weight(m[p], M);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int tt = 0; tt < ATT_TPW; ++tt) {
                    const i32x4 v = kv[((ph * ATT_TPW + tt) * NDT + dt) * 64 + lane];
                    o = mfma_step<ET_BF16>(v, Pf[tt], o);
                    o = mfma_step<ET_BF16>(v, Pl[tt], o);
                }
                attn_merge_o(acc[dt], o, f);
                if constexpr (NH == 2) __builtin_amdgcn_sched_barrier(0);
            }
            attn_merge_l(L, lp, f);
        }
    }
    const int t = t0 + r;
    if (tv && t < T) {
        const size_t o = ((size_t)split * a.H + head) * T + t;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) *(f32x4*)(a.part_o + o * HD + 16 * dt + 4 * g) = acc[dt];
        if (g == 0) *(float2*)(a.part_ml + o * 2) = make_float2(M, L);
    }
}


// Merge the KV splits of R query rows of one head; each thread owns one
// (row, 4 d) item.
template <int HD, int R = 16>
__global__ void __launch_bounds__(256) k_attn_merge(const AttnArgs a, int S) {
    const int h = blockIdx.y, t0 = blockIdx.x * R, T = a.T;
    const int NTo = col_tiles(T);
    for (int idx = threadIdx.x; idx < R * (HD / 4); idx += blockDim.x) {
        const int rr = idx / (HD / 4), d4 = (idx % (HD / 4)) * 4, t = t0 + rr;
        if (t >= T) continue;
        const f32x4 acc = attn_merge_row<HD>(a, S, (size_t)h * T + t, d4);
        const int kk = h * HD + d4;
        if (a.out_tiled) {
            st4((uint16_t*)a.out, xt_off(t, kk, NTo, 8), acc[0], acc[1], acc[2], acc[3]);
        } else {
            uint16_t* o = (uint16_t*)a.out + (size_t)t * a.H * HD + kk;
            o[0] = f2bf(acc[0]);
            o[1] = f2bf(acc[1]);
            o[2] = f2bf(acc[2]);
            o[3] = f2bf(acc[3]);
        }
    }
}

// Merge and quantise for the quantised-activation drafts: one workgroup per
// query row merges every head of the row (the values k_attn_merge would
// store, rounded to bf16), takes the row's amax and writes the row's codes
// (s = amax / qm, tiled int8 layout, pad zero) and scale, the work of
// k_attn_merge and k_quant_rows_tiled in one launch.  NI (row, 4 d) items
// per thread.
static constexpr int MQ_THREADS = 1024;
template <int HD, int NI>
__global__ void __launch_bounds__(MQ_THREADS) k_attn_merge_q(const AttnArgs a, int S) {
    __shared__ float red[MQ_THREADS / 64];
    const int t = blockIdx.x, T = a.T, NT = col_tiles(T), K = a.H * HD;
    const int kpq = (K + 255) / 256 * 256;
    f32x4 v[NI];
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int k4 = (threadIdx.x + MQ_THREADS * i) * 4;
        v[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (k4 < K) {
            const f32x4 acc = attn_merge_row<HD>(a, S, (size_t)(k4 / HD) * T + t, k4 % HD);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[i][e] = bf2f(f2bf(acc[e]));
            amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[i][0]), fabsf(v[i][1])), fmaxf(fabsf(v[i][2]), fabsf(v[i][3]))));
        }
    }
    amax = block_max<MQ_THREADS / 64>(amax, red);
    const float qm = (float)a.qmax, sc = amax / qm;
    if (threadIdx.x == 0) a.qscale[t] = sc;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int k4 = (threadIdx.x + MQ_THREADS * i) * 4;
        if (k4 < kpq)
            st4q(a.qout, xt_off(t, k4, NT, 16), qcode(v[i][0], sc, qm), qcode(v[i][1], sc, qm), qcode(v[i][2], sc, qm),
                 qcode(v[i][3], sc, qm));
    }
}

// fp32 storage: plain attention, one workgroup per (token, head); scores of
// all visible slots in LDS.
__global__ void __launch_bounds__(256) k_attn_f32(const AttnArgs a, float scale) {
    extern __shared__ float sc[];
    __shared__ float red[4];
    const int t = blockIdx.x, h = blockIdx.y, hd = a.hd;
    const int G = a.H / a.Hkv, kvh = h / G;
    const int Lc = a.sp->Lc, n_slots = Lc + a.sp->n_tree;
    if (!dcheck(a.chk, Lc >= 0 && n_slots <= a.sp->cap && a.sp->cap <= a.ctx_cap, CHK_ATTN_SLOTS)) return;
    const AttnWindow win(Lc, a.sp->n_tree, a.win_sink, a.win_len);
    const uint64_t a0 = a.anc[2 * t], a1 = a.anc[2 * t + 1];
    const float* q = (const float*)a.q + ((size_t)t * a.H + h) * hd;
    const float* kb = (const float*)a.kc + (size_t)kvh * a.ctx_cap * hd;
    const float* vb = (const float*)a.vt + (size_t)kvh * hd * a.ctx_cap;
    float mx = -INFINITY;
    for (int s = threadIdx.x; s < n_slots; s += 256) {
        const bool vis = s < Lc ? (s < win.csink || s >= win.wstart) : anc_bit(a0, a1, s - Lc);
        float v = -INFINITY;
        if (vis) {
            float d = 0.f;
            for (int e = 0; e < hd; ++e) d += q[e] * kb[(size_t)s * hd + e];
            v = d * scale;
        }
        sc[s] = v;
        mx = fmaxf(mx, v);
    }
    mx = block_max256(mx, red);
    float sum = 0.f;
    for (int s = threadIdx.x; s < n_slots; s += 256) {
        const float p = expf(sc[s] - mx);
        sc[s] = p;
        sum += p;
    }
    sum = block_sum256(sum, red);
    __syncthreads();
    for (int d = threadIdx.x; d < hd; d += 256) {
        float o = 0.f;
        for (int s = 0; s < n_slots; ++s) o += sc[s] * vb[(size_t)d * a.ctx_cap + s];
        const size_t oi = a.out_tiled ? xt_off(t, h * hd + d, col_tiles(a.T), 4)
                                      : (size_t)t * a.H * hd + (size_t)h * hd + d;
        ((float*)a.out)[oi] = o / sum;
    }
}

// The merge of the attention's S KV splits (launched by launch_attention
// unless no_merge): bf16 rows, or with qout the rows' codes and scales.
static bool attn_merge_ok(const AttnArgs& a) {
    const int K = a.H * a.hd, kpq = (K + 255) / 256 * 256;
    const int ni = (kpq / 4 + MQ_THREADS - 1) / MQ_THREADS;
    return (a.hd == 64 || a.hd == 128) && (!a.qout || (ni <= 4 && (a.qmax == 127 || a.qmax == 7)));
}

hipError_t launch_attn_merge(const AttnArgs& a, int S, hipStream_t s) {
    if (!attn_merge_ok(a) || S < 1 || S > ATT_MAX_SPLITS || a.T < 1) return hipErrorInvalidValue;
    // plain merge: 4 query rows per workgroup, i.e. many small workgroups
    // (7B layer: attention + merge 12.1 us against 14.2 with 16 rows);
    // quantised output: one merge-and-quantise workgroup per row
    const dim3 mg((a.T + 3) / 4, a.H);
    const int K = a.H * a.hd, kpq = (K + 255) / 256 * 256;
    const int ni = (kpq / 4 + MQ_THREADS - 1) / MQ_THREADS;
    if (a.hd == 128) {
        if (!a.qout) hipLaunchKernelGGL((k_attn_merge<128, 4>), mg, dim3(128), 0, s, a, S);
        else if (ni <= 1) hipLaunchKernelGGL((k_attn_merge_q<128, 1>), dim3(a.T), dim3(MQ_THREADS), 0, s, a, S);
        else if (ni <= 2) hipLaunchKernelGGL((k_attn_merge_q<128, 2>), dim3(a.T), dim3(MQ_THREADS), 0, s, a, S);
        else hipLaunchKernelGGL((k_attn_merge_q<128, 4>), dim3(a.T), dim3(MQ_THREADS), 0, s, a, S);
    } else {
        if (!a.qout) hipLaunchKernelGGL((k_attn_merge<64, 4>), mg, dim3(64), 0, s, a, S);
        else if (ni <= 1) hipLaunchKernelGGL((k_attn_merge_q<64, 1>), dim3(a.T), dim3(MQ_THREADS), 0, s, a, S);
        else if (ni <= 2) hipLaunchKernelGGL((k_attn_merge_q<64, 2>), dim3(a.T), dim3(MQ_THREADS), 0, s, a, S);
        else hipLaunchKernelGGL((k_attn_merge_q<64, 4>), dim3(a.T), dim3(MQ_THREADS), 0, s, a, S);
    }
    return hipGetLastError();
}

hipError_t launch_attention(int atype, const AttnArgs& a, hipStream_t s) {
    if (a.T < 1 || a.T > 128 || a.Hkv < 1 || a.H % a.Hkv) return hipErrorInvalidValue;
    const int n_slots = a.Lc_host + a.n_tree_host;
    if (atype == ET_F32) {
        if (a.ctx_cap > 4096) return hipErrorInvalidValue;
        const float scale = 1.0f / sqrtf((float)a.hd);
        hipLaunchKernelGGL(k_attn_f32, dim3(a.T, a.H), dim3(256), (size_t)a.ctx_cap * 4, s, a, scale);
        return hipGetLastError();
    }
    const int S = attention_splits_win(a.Lc_host, a.n_tree_host, a.win_sink, a.win_len);
    const int G = a.H / a.Hkv, Tp = (a.T + 15) & ~15;
    const int nct = attn_query_tiles(a.T, G);  // 16-row query tiles per kv head
    if (a.ctx_cap % 32 || S > ATT_MAX_SPLITS) return hipErrorInvalidValue;
    const float scale_log2 = (1.0f / sqrtf((float)a.hd)) * 1.4426950408889634f;
    // Several query tiles per kv head, each head with at least 32 rows:
    // four tiles per workgroup share one pass of the split's K/V through LDS
    // (k_attn_rows; per layer, 8B 64 nodes at 4096: 27.7 -> 23.3 us, 7B 128
    // nodes at 8192: 112 -> 65 us).
    // Calls of up to 16 tokens pack the grouped heads' rows into shared tiles
    // (attn_head_rows; 8B one node at 4096: attention 9.6 -> 6.8 us per
    // layer against one tile of one row per head) and take k_attn_bf16.
    // Both kernels give the same bits for a row.  Otherwise the split's
    // key tiles spread over four waves (k_attn_bf16), one 16-row tile per
    // workgroup unless the grid of (split, kv head, tile) units is large; then
    // two tiles share each K/V load (7B 32 nodes at 8192: fewer, longer
    // workgroups halve the per-CU key traffic).
    // With three or four tiles per kv head the shared pass pays only when the
    // per-tile grid is large: from about 1024 tile workgroups (13B 64 nodes at
    // 2048, 1440 of them: 6.33 ms with k_attn_rows, 6.36 without; 7B 64 nodes
    // at 2048, 1152: 4.10 and 4.13 ms; 7B 48 nodes at 8192: 5.22 -> 4.94 ms
    // with the single-stage form); below, the larger grid wins (7B 48 nodes at
    // 2048, 864: 4.00 ms with k_attn_rows, 3.98 without; 7B 64 nodes at 1024,
    // 640: 3.93 and 3.90 ms; at 512: 3.84 and 3.74 ms).
    const bool rows = (nct >= 5 || (nct >= 3 && (long)S * a.Hkv * nct >= 1024)) && Tp >= 32;
    const int JT = (G == 1 && S * a.Hkv * nct >= 1024) ? 2 : 1;
    const dim3 rg(S, a.Hkv, (nct + 3) / 4);
    const bool half = (long)S * a.Hkv * ((nct + 3) / 4) > 256;  // k_attn_rows stages in halves
    const int nrc = (nct + JT - 1) / JT;
    if (a.no_merge && a.qout) return hipErrorInvalidValue;
    if (!a.no_merge && !attn_merge_ok(a)) return hipErrorInvalidValue;
    if (a.hd == 128) {
        if (rows && half) hipLaunchKernelGGL((k_attn_rows<128, 4, 2>), rg, dim3(256), 0, s, a, scale_log2);
        else if (rows) hipLaunchKernelGGL((k_attn_rows<128, 4, 1>), rg, dim3(256), 0, s, a, scale_log2);
        else if (JT == 2) hipLaunchKernelGGL((k_attn_bf16<128, 2>), dim3(S, a.Hkv, nrc), dim3(256), 0, s, a, scale_log2);
        else hipLaunchKernelGGL((k_attn_bf16<128, 1>), dim3(S, a.Hkv, nrc), dim3(256), 0, s, a, scale_log2);
    } else if (a.hd == 64) {
        if (rows && half) hipLaunchKernelGGL((k_attn_rows<64, 4, 2>), rg, dim3(256), 0, s, a, scale_log2);
        else if (rows) hipLaunchKernelGGL((k_attn_rows<64, 4, 1>), rg, dim3(256), 0, s, a, scale_log2);
        else if (JT == 2) hipLaunchKernelGGL((k_attn_bf16<64, 2>), dim3(S, a.Hkv, nrc), dim3(256), 0, s, a, scale_log2);
        else hipLaunchKernelGGL((k_attn_bf16<64, 1>), dim3(S, a.Hkv, nrc), dim3(256), 0, s, a, scale_log2);
    } else {
        return hipErrorInvalidValue;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.no_merge) return e;
    return launch_attn_merge(a, S, s);
}

// Row-major [Hkv][n][hd] <-> cache layout, one thread per (head, slot, d).
template <typename AT>
__global__ void k_kv_convert(AT* kc, AT* vt, const AT* kr, const AT* vr, int Hkv, int n, int hd, int ctx_cap,
                             int to_cache) {
    constexpr int ET = sizeof(AT) == 2 ? ET_BF16 : ET_F32;
    const size_t total = (size_t)Hkv * n * hd;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
        const int d = (int)(i % hd), slot = (int)((i / hd) % n), h = (int)(i / ((size_t)hd * n));
        const size_t base = (size_t)h * ctx_cap * hd;
        const size_t ko = base + kv_k_off(ET, slot, d, hd, ctx_cap), vo = base + kv_v_off(ET, slot, d, hd, ctx_cap);
        if (to_cache) {
            kc[ko] = kr[i];
            vt[vo] = vr[i];
        } else {
            ((AT*)kr)[i] = kc[ko];
            ((AT*)vr)[i] = vt[vo];
        }
    }
}

hipError_t launch_kv_convert(int atype, void* kc, void* vt, const void* k_rows, const void* v_rows, int Hkv, int n,
                             int hd, int ctx_cap, int to_cache, hipStream_t s) {
    size_t total = (size_t)Hkv * n * hd, b = (total + 255) / 256;
    if (b > 16384) b = 16384;
    if (b == 0) return hipSuccess;
    if (atype == ET_BF16)
        hipLaunchKernelGGL(k_kv_convert<uint16_t>, dim3((unsigned)b), dim3(256), 0, s, (uint16_t*)kc, (uint16_t*)vt,
                           (const uint16_t*)k_rows, (const uint16_t*)v_rows, Hkv, n, hd, ctx_cap, to_cache);
    else
        hipLaunchKernelGGL(k_kv_convert<float>, dim3((unsigned)b), dim3(256), 0, s, (float*)kc, (float*)vt,
                           (const float*)k_rows, (const float*)v_rows, Hkv, n, hd, ctx_cap, to_cache);
    return hipGetLastError();
}

// ---------------------------------------------------------------- norms, quantisation

// One workgroup of 16 waves per row: the loads of a row spread over the
// whole CU (measured faster than 4 waves once split-K partials are folded in).
static constexpr int NORM_THREADS = 1024;
static constexpr int NORM_MAXP = 8;  // split-K partial sums a norm folds in (launch_gemm_parts allows 8)
static constexpr int NORM_MAXV = 4;  // float4 per thread: rows up to 16384 elements

// RMSNorm of one row of the residual stream, written as tiled activations
// (pad columns zero) or, with Q, straight to the row's quantisation (codes
// in [-qm, qm], one per byte: int8, or int4 for the W4A4 weights).
// With nparts > 0 the row first takes the pending split-K sums of the last
// projection (summed in split order, then added to the residual, which is
// stored back).  NV float4 per thread; loads are unconditional (clamped into
// the row) so they issue back to back; d is a multiple of 16.
template <typename AT, bool Q, int NV>
__global__ void __launch_bounds__(NORM_THREADS) k_rmsnorm(float* h, const float* gain, int d, float eps, AT* out,
                                                 int8_t* q, float* qs, const float* parts, int nparts,
                                                 size_t pstride, float qm) {
    __shared__ float red[NORM_THREADS / 64];
    const int t = blockIdx.x, NT = col_tiles(gridDim.x), tid = threadIdx.x;
    float* x = h + (size_t)t * d;
    float4 v[NV], gv[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int kc = min((tid + NORM_THREADS * i) * 4, d - 4);
        v[i] = *(const float4*)(x + kc);
        gv[i] = *(const float4*)(gain + kc);
    }
    if (nparts > 0) {
        // rows of up to 8192 elements: every split's loads issue before the
        // first add (a loop over the splits waited for each split's loads in
        // turn), then the sums run in split order; longer rows keep the loop
        // (the registers of all splits would not fit)
        float4 ps[NV];
        const float* pr = parts + (size_t)t * d;
#pragma unroll
        for (int i = 0; i < NV; ++i) ps[i] = *(const float4*)(pr + min((tid + NORM_THREADS * i) * 4, d - 4));
        if constexpr (NV <= 2) {
            float4 pp[NORM_MAXP - 1][NV];
#pragma unroll
            for (int p = 1; p < NORM_MAXP; ++p)
                if (p < nparts)
#pragma unroll
                    for (int i = 0; i < NV; ++i)
                        pp[p - 1][i] = *(const float4*)(pr + p * pstride + min((tid + NORM_THREADS * i) * 4, d - 4));
#pragma unroll
            for (int p = 1; p < NORM_MAXP; ++p)
                if (p < nparts)
#pragma unroll
                    for (int i = 0; i < NV; ++i) {
                        ps[i].x += pp[p - 1][i].x;
                        ps[i].y += pp[p - 1][i].y;
                        ps[i].z += pp[p - 1][i].z;
                        ps[i].w += pp[p - 1][i].w;
                    }
        } else {
            for (int p = 1; p < nparts; ++p) {
                float4 pp[NV];
#pragma unroll
                for (int i = 0; i < NV; ++i)
                    pp[i] = *(const float4*)(pr + p * pstride + min((tid + NORM_THREADS * i) * 4, d - 4));
#pragma unroll
                for (int i = 0; i < NV; ++i) {
                    ps[i].x += pp[i].x;
                    ps[i].y += pp[i].y;
                    ps[i].z += pp[i].z;
                    ps[i].w += pp[i].w;
                }
            }
        }
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            v[i].x += ps[i].x;
            v[i].y += ps[i].y;
            v[i].z += ps[i].z;
            v[i].w += ps[i].w;
            const int k4 = (tid + NORM_THREADS * i) * 4;
            if (k4 < d) *(float4*)(x + k4) = v[i];
        }
    }
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        if ((tid + NORM_THREADS * i) * 4 >= d) v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
    ss = block_sum<NORM_THREADS / 64>(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        v[i].x = Act<AT>::round(v[i].x * inv * gv[i].x);
        v[i].y = Act<AT>::round(v[i].y * inv * gv[i].y);
        v[i].z = Act<AT>::round(v[i].z * inv * gv[i].z);
        v[i].w = Act<AT>::round(v[i].w * inv * gv[i].w);
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[i].x), fabsf(v[i].y)), fmaxf(fabsf(v[i].z), fabsf(v[i].w))));
    }
    if constexpr (!Q) {
        constexpr int EA = 16 / sizeof(AT);
        const int kpa = (d + 16 * EA - 1) / (16 * EA) * (16 * EA);
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int k4 = (tid + NORM_THREADS * i) * 4;
            if (k4 < kpa) st4(out, xt_off(t, k4, NT, EA), v[i].x, v[i].y, v[i].z, v[i].w);  // zero past d
        }
    } else {
        amax = block_max<NORM_THREADS / 64>(amax, red);
        const float sc = amax / qm;
        if (threadIdx.x == 0) qs[t] = sc;
        const int kpq = (d + 255) / 256 * 256;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int k4 = (tid + NORM_THREADS * i) * 4;
            if (k4 < kpq)
                st4q(q, xt_off(t, k4, NT, 16), qcode(v[i].x, sc, qm), qcode(v[i].y, sc, qm), qcode(v[i].z, sc, qm),
                     qcode(v[i].w, sc, qm));
        }
    }
}

template <typename AT, bool Q>
static hipError_t rmsnorm_go(float* h, const float* g, int T, int d, float eps, AT* out, int8_t* q, float* qs,
                             const float* parts, int nparts, size_t pstride, float qm, hipStream_t s) {
    // float4 per thread covering the padded row (int8 output pads to 256, bf16 to 128)
    const int span = (d + 255) / 256 * 256;
    const int nv = (span + 4 * NORM_THREADS - 1) / (4 * NORM_THREADS);
#define CAS_NORM(NV) \
    hipLaunchKernelGGL((k_rmsnorm<AT, Q, NV>), dim3(T), dim3(NORM_THREADS), 0, s, h, g, d, eps, out, q, qs, parts, nparts, \
                       pstride, qm)
    if (nv <= 1) CAS_NORM(1);
    else if (nv <= 2) CAS_NORM(2);
    else CAS_NORM(NORM_MAXV);
#undef CAS_NORM
    return hipGetLastError();
}

hipError_t launch_rmsnorm(int atype, float* h, const float* g, int T, int d, float eps, void* out, int8_t* q,
                          float* qs, const float* parts, int nparts, size_t pstride, int qmax, hipStream_t s) {
    if (d > 4 * NORM_THREADS * NORM_MAXV || d % 16 || nparts < 0 || nparts > NORM_MAXP ||
        (nparts > 0 && (!parts || pstride < (size_t)T * d)) || (q && qmax != 127 && qmax != 7))
        return hipErrorInvalidValue;
    const float qm = (float)qmax;
    if (atype == ET_BF16) {
        if (q) return rmsnorm_go<uint16_t, true>(h, g, T, d, eps, (uint16_t*)out, q, qs, parts, nparts, pstride, qm, s);
        return rmsnorm_go<uint16_t, false>(h, g, T, d, eps, (uint16_t*)out, q, qs, parts, nparts, pstride, qm, s);
    }
    if (q) return rmsnorm_go<float, true>(h, g, T, d, eps, (float*)out, q, qs, parts, nparts, pstride, qm, s);
    return rmsnorm_go<float, false>(h, g, T, d, eps, (float*)out, q, qs, parts, nparts, pstride, qm, s);
}

// Per-row symmetric quantisation of tiled activations: s = amax / qm,
// q = clamp(rne(x / s), -qm, qm) (qm 127 or 7), codes written tiled, one per
// byte (pad zero).  One
// workgroup of 1024 threads per row; a thread takes whole 16-byte fragments
// of the row (EA consecutive k each, which land in one int8 fragment of 16
// k), NF fragments per thread held in registers between the amax and the
// quantisation.
static constexpr int QR_THREADS = 1024;

template <typename AT, int NF>
__global__ void __launch_bounds__(QR_THREADS) k_quant_rows_tiled(const AT* x, int K, int8_t* q, float* qs, float qm) {
    __shared__ float red[QR_THREADS / 64];
    constexpr int EA = 16 / sizeof(AT);
    const int t = blockIdx.x, NT = col_tiles(gridDim.x), tid = threadIdx.x;
    const int nfa = (K + 16 * EA - 1) / (16 * EA) * 16;  // fragments of the padded input row
    const int nfq = (K + 255) / 256 * 256 / EA;           // fragments covering the padded int8 row
    i32x4 v[NF];
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < NF; ++i) {
        const int f = tid + QR_THREADS * i;
        v[i] = *(const i32x4*)(x + xt_off(t, min(f, nfa - 1) * EA, NT, EA));
        const AT* e = (const AT*)&v[i];
#pragma unroll
        for (int j = 0; j < EA; ++j)
            if (f < nfa && f * EA + j < K) amax = fmaxf(amax, fabsf(Act<AT>::ld(e, j)));
    }
    amax = block_max<QR_THREADS / 64>(amax, red);
    const float sc = amax / qm;
    if (tid == 0) qs[t] = sc;
#pragma unroll
    for (int i = 0; i < NF; ++i) {
        const int f = tid + QR_THREADS * i;
        if (f >= nfq) continue;
        const AT* e = (const AT*)&v[i];
        uint32_t w[EA / 4];
#pragma unroll
        for (int j = 0; j < EA / 4; ++j) {
            uint32_t b = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int k = f * EA + 4 * j + u;
                const float c = (f < nfa && k < K) ? qcode(Act<AT>::ld(e, 4 * j + u), sc, qm) : 0.f;
                b |= (uint32_t)(uint8_t)(int8_t)c << (8 * u);
            }
            w[j] = b;
        }
        int8_t* o = q + xt_off(t, f * EA, NT, 16);
        if constexpr (EA == 8) *(uint2*)o = make_uint2(w[0], w[1]);
        else *(uint32_t*)o = w[0];
    }
}

// Row-major form ([T][K] in, [T][K] out), for the kernel-level entry point.
template <typename AT, bool TILED>
__global__ void __launch_bounds__(256) k_quant_rows(const AT* x, int K, int8_t* q, float* qs, float qm) {
    __shared__ float red[4];
    const int t = blockIdx.x, NT = col_tiles(gridDim.x);
    constexpr int EA = 16 / sizeof(AT);
    auto at = [&](int k) -> size_t { return TILED ? xt_off(t, k, NT, EA) : (size_t)t * K + k; };
    float amax = 0.f;
    for (int k = threadIdx.x; k < K; k += 256) amax = fmaxf(amax, fabsf(Act<AT>::ld(x, at(k))));
    amax = block_max256(amax, red);
    const float sc = amax / qm;
    if (threadIdx.x == 0) qs[t] = sc;
    const int kq = TILED ? (K + 255) / 256 * 256 : K;
    for (int k = threadIdx.x; k < kq; k += 256) {
        float rq = 0.f;
        if (k < K) rq = qcode(Act<AT>::ld(x, at(k)), sc, qm);
        q[TILED ? xt_off(t, k, NT, 16) : (size_t)t * K + k] = (int8_t)rq;
    }
}

template <typename AT>
static hipError_t quant_tiled_go(const AT* x, int T, int K, int8_t* q, float* qs, float qm, hipStream_t s) {
    constexpr int EA = 16 / sizeof(AT);
    const int nfq = (K + 255) / 256 * 256 / EA;  // >= fragments of the padded input row
    const int nf = (nfq + QR_THREADS - 1) / QR_THREADS;
#define CAS_QR(NF) hipLaunchKernelGGL((k_quant_rows_tiled<AT, NF>), dim3(T), dim3(QR_THREADS), 0, s, x, K, q, qs, qm)
    if (nf <= 1) CAS_QR(1);
    else if (nf <= 2) CAS_QR(2);
    else if (nf <= 4) CAS_QR(4);
    else if (nf <= 8) CAS_QR(8);
    else CAS_QR(16);
#undef CAS_QR
    return hipGetLastError();
}

hipError_t launch_quant_rows(int atype, const void* x, int T, int K, int8_t* q, float* qs, int tiled, int qmax,
                             hipStream_t s) {
    if (T < 1 || K < 1 || (tiled && (T > 128 || K > 65536)) || (qmax != 127 && qmax != 7)) return hipErrorInvalidValue;
    const float qm = (float)qmax;
    if (atype == ET_BF16) {
        if (tiled) return quant_tiled_go((const uint16_t*)x, T, K, q, qs, qm, s);
        hipLaunchKernelGGL((k_quant_rows<uint16_t, false>), dim3(T), dim3(256), 0, s, (const uint16_t*)x, K, q, qs, qm);
    } else {
        if (tiled) return quant_tiled_go((const float*)x, T, K, q, qs, qm, s);
        hipLaunchKernelGGL((k_quant_rows<float, false>), dim3(T), dim3(256), 0, s, (const float*)x, K, q, qs, qm);
    }
    return hipGetLastError();
}

// Element offset of W[n][k] in a tiled matrix of element size es and padded
// width Kp, tile-major or (kmaj) K-major over ntiles tiles.
__device__ __forceinline__ size_t wt_off_in(int n, int k, int Kp, int E, int es, int kmaj, int ntiles) {
    const size_t off = wt_off(n, k, Kp, E);
    return kmaj ? wt_kmajor(off * es, ntiles, Kp * es / 64) / es : off;
}

// Tiled weights (act type) -> tiled int8 copy with per-row scales, one
// workgroup per 16-row tile: row amax over the whole row, then the codes.
// skm / dkm: the source / the copy in the K-major block order.
template <typename AT>
__global__ void __launch_bounds__(256) k_quant_weight(const AT* w, int K, int8_t* q, float* qs, int skm, int dkm) {
    __shared__ unsigned amax_bits[16];
    __shared__ float scale[16];
    constexpr int EA = 16 / sizeof(AT), ES = sizeof(AT);
    const int tile = blockIdx.x, n0 = tile * 16, nt = gridDim.x;
    const int Kpa = (K + 16 * EA - 1) / (16 * EA) * (16 * EA), Kpq = (K + 255) / 256 * 256;
    if (threadIdx.x < 16) amax_bits[threadIdx.x] = 0u;
    __syncthreads();
    const int r = threadIdx.x & 15;
    float m = 0.f;
    for (int k = threadIdx.x >> 4; k < K; k += 16)
        m = fmaxf(m, fabsf(Act<AT>::ld(w, wt_off_in(n0 + r, k, Kpa, EA, ES, skm, nt))));
    atomicMax(&amax_bits[r], __float_as_uint(m));  // non-negative floats order like their bits
    __syncthreads();
    if (threadIdx.x < 16) {
        const float sc = __uint_as_float(amax_bits[threadIdx.x]) / 127.0f;
        scale[threadIdx.x] = sc;
        qs[n0 + threadIdx.x] = sc;
    }
    __syncthreads();
    const float sc = scale[r];
    for (int k = threadIdx.x >> 4; k < Kpq; k += 16) {
        float rq = 0.f;
        if (k < K && sc != 0.f)
            rq = fminf(fmaxf(rintf(Act<AT>::ld(w, wt_off_in(n0 + r, k, Kpa, EA, ES, skm, nt)) / sc), -127.f), 127.f);
        q[wt_off_in(n0 + r, k, Kpq, 16, 1, dkm, nt)] = (int8_t)rq;
    }
}

hipError_t launch_quant_weight(int wtype, const void* w, int N, int K, int8_t* q, float* qs, hipStream_t s, int skm,
                               int dkm) {
    if (N % 16) return hipErrorInvalidValue;
    if (wtype == ET_BF16)
        hipLaunchKernelGGL(k_quant_weight<uint16_t>, dim3(N / 16), dim3(256), 0, s, (const uint16_t*)w, K, q, qs, skm,
                           dkm);
    else
        hipLaunchKernelGGL(k_quant_weight<float>, dim3(N / 16), dim3(256), 0, s, (const float*)w, K, q, qs, skm, dkm);
    return hipGetLastError();
}

// Tiled int8 weights -> row-major (for checking the copy).
__global__ void k_untile_weight_i8(const int8_t* src, int N, int K, int8_t* dst) {
    const int Kp = (K + 255) / 256 * 256;
    const size_t total = (size_t)N * K;
    for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x)
        dst[idx] = src[wt_off((int)(idx / K), (int)(idx % K), Kp, 16)];
}

hipError_t launch_untile_weight_i8(const int8_t* src, int N, int K, int8_t* dst, hipStream_t s) {
    hipLaunchKernelGGL(k_untile_weight_i8, dim3(grid_for((size_t)N * K)), dim3(256), 0, s, src, N, K, dst);
    return hipGetLastError();
}

// ---- packed int4 weights (wt4_byte layout)

// Tile (n >> 4), chunk c: the byte b of its 2 KB holds rows/k-offsets given
// by wt4_byte; this inverts it: (row in tile, k of the low nibble).
__device__ __forceinline__ void wt4_inv(int b, int c, int& r, int& k) {
    const int blk = b >> 10, lane = (b >> 4) & 63, byte = b & 15;
    const int g = lane >> 4, u = 2 * blk + (byte >> 3), j = byte & 7;
    r = lane & 15;
    k = c * 256 + g * 64 + u * 16 + j;  // the high nibble holds k + 8
}

// Tiled weights (act type) -> packed int4 codes with per-row scales amax / 7,
// one workgroup per 16-row tile: row amax over the whole row, then 4 packed
// bytes per thread and step.
template <typename AT>
__global__ void __launch_bounds__(256) k_quant_weight_i4(const AT* w, int K, uint8_t* q, float* qs, int skm, int dkm) {
    __shared__ unsigned amax_bits[16];
    __shared__ float scale[16];
    constexpr int EA = 16 / sizeof(AT), ES = sizeof(AT);
    const int tile = blockIdx.x, n0 = tile * 16, nt = gridDim.x;
    const int Kpa = (K + 16 * EA - 1) / (16 * EA) * (16 * EA), C = (K + 255) / 256;
    if (threadIdx.x < 16) amax_bits[threadIdx.x] = 0u;
    __syncthreads();
    {
        const int r = threadIdx.x & 15;
        float m = 0.f;
        for (int k = threadIdx.x >> 4; k < K; k += 16)
            m = fmaxf(m, fabsf(Act<AT>::ld(w, wt_off_in(n0 + r, k, Kpa, EA, ES, skm, nt))));
        atomicMax(&amax_bits[r], __float_as_uint(m));  // non-negative floats order like their bits
    }
    __syncthreads();
    if (threadIdx.x < 16) {
        const float sc = __uint_as_float(amax_bits[threadIdx.x]) / 7.0f;
        scale[threadIdx.x] = sc;
        qs[n0 + threadIdx.x] = sc;
    }
    __syncthreads();
    const size_t qt = (size_t)tile * C * 2048;  // the tile's bytes in the tile-major order
    for (int w4 = threadIdx.x; w4 < C * 512; w4 += 256) {
        const int c = w4 >> 9;
        uint32_t word = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int r, k;
            wt4_inv((w4 & 511) * 4 + i, c, r, k);
            const float sc = scale[r];
            const float lo = k < K ? qcode(Act<AT>::ld(w, wt_off_in(n0 + r, k, Kpa, EA, ES, skm, nt)), sc, 7.f) : 0.f;
            const float hi =
                k + 8 < K ? qcode(Act<AT>::ld(w, wt_off_in(n0 + r, k + 8, Kpa, EA, ES, skm, nt)), sc, 7.f) : 0.f;
            word |= (uint32_t)(((int)lo + 8) | (((int)hi + 8) << 4)) << (8 * i);
        }
        const size_t b = qt + (size_t)w4 * 4;
        *(uint32_t*)(q + (dkm ? wt_kmajor(b, nt, C * 2) : b)) = word;
    }
}

hipError_t launch_quant_weight_i4(int wtype, const void* w, int N, int K, uint8_t* q, float* qs, hipStream_t s,
                                  int skm, int dkm) {
    if (N % 16 || K < 1) return hipErrorInvalidValue;
    if (wtype == ET_BF16)
        hipLaunchKernelGGL(k_quant_weight_i4<uint16_t>, dim3(N / 16), dim3(256), 0, s, (const uint16_t*)w, K, q, qs,
                           skm, dkm);
    else
        hipLaunchKernelGGL(k_quant_weight_i4<float>, dim3(N / 16), dim3(256), 0, s, (const float*)w, K, q, qs, skm,
                           dkm);
    return hipGetLastError();
}

// Row-major codes [N][K] in [-7, 7] -> packed int4 (one thread per packed byte).
__global__ void k_pack_weight_i4(const int8_t* src, int N, int K, uint8_t* dst) {
    const int C = (K + 255) / 256;
    const size_t total = (size_t)(N / 16) * C * 2048;
    for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        const int tile = (int)(idx / ((size_t)C * 2048)), rem = (int)(idx % ((size_t)C * 2048));
        int r, k;
        wt4_inv(rem & 2047, rem >> 11, r, k);
        const size_t row = (size_t)(tile * 16 + r) * K;
        const int lo = k < K ? src[row + k] : 0, hi = k + 8 < K ? src[row + k + 8] : 0;
        dst[idx] = (uint8_t)((lo + 8) | ((hi + 8) << 4));
    }
}
hipError_t launch_pack_weight_i4(const int8_t* src, int N, int K, uint8_t* dst, hipStream_t s) {
    if (N % 16 || K < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pack_weight_i4, dim3(grid_for((size_t)(N / 16) * ((K + 255) / 256) * 2048)), dim3(256), 0, s,
                       src, N, K, dst);
    return hipGetLastError();
}

// Packed int4 -> row-major codes (for checking the copy).
__global__ void k_untile_weight_i4(const uint8_t* src, int N, int K, int8_t* dst) {
    const int Kp = (K + 255) / 256 * 256;
    const size_t total = (size_t)N * K;
    for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        int nib;
        const size_t b = wt4_byte((int)(idx / K), (int)(idx % K), Kp, &nib);
        dst[idx] = (int8_t)(((src[b] >> (4 * nib)) & 15) - 8);
    }
}
hipError_t launch_untile_weight_i4(const uint8_t* src, int N, int K, int8_t* dst, hipStream_t s) {
    hipLaunchKernelGGL(k_untile_weight_i4, dim3(grid_for((size_t)N * K)), dim3(256), 0, s, src, N, K, dst);
    return hipGetLastError();
}

// ---------------------------------------------------------------- embedding + tree metadata

// Element e of a 16-byte piece of activations (bf16 bits or fp32), as fp32.
template <typename AT> __device__ __forceinline__ float piece_val(const i32x4 v, int e);
template <> __device__ __forceinline__ float piece_val<uint16_t>(const i32x4 v, int e) {
    const uint32_t w = (uint32_t)v[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
}
template <> __device__ __forceinline__ float piece_val<float>(const i32x4 v, int e) { return __int_as_float(v[e]); }

template <typename AT>
__global__ void __launch_bounds__(256) k_embed(const AT* E, int d, int vocab, const int* rtok, const int* rpar,
                                               const StepParams* sp, float* h, int* row_pos, int* row_slot,
                                               uint64_t* row_anc, int* chk) {
    __shared__ int par[128];
    const int t = blockIdx.x;
    const int node = sp->node_offset + t, Lc = sp->Lc, n_tree = sp->n_tree;
    if (!dcheck(chk, n_tree <= 128 && sp->node_offset >= 0 && node < n_tree, CHK_TREE_SIZE)) {
        if (threadIdx.x == 0) {
            row_pos[t] = 0;
            row_slot[t] = -1;
            row_anc[2 * t] = row_anc[2 * t + 1] = 0;
        }
        return;
    }
    if (threadIdx.x < n_tree) par[threadIdx.x] = rpar[threadIdx.x];
    int tok = rtok[node];
    if (!dcheck(chk, tok >= 0 && tok < vocab, CHK_TOKEN)) tok = 0;
    // the row in 16-byte pieces (d is a multiple of 16), all loads first
    constexpr int EV = 16 / sizeof(AT), MAXP = 4;  // elements per piece; pieces per thread up to d = 8192
    const AT* er = E + (size_t)tok * d;
    float* hr = h + (size_t)t * d;
    i32x4 pc[MAXP];
#pragma unroll
    for (int i = 0; i < MAXP; ++i) {
        const int k = (threadIdx.x + 256 * i) * EV;
        if (k < d) pc[i] = *(const i32x4*)(er + k);
    }
#pragma unroll
    for (int i = 0; i < MAXP; ++i) {
        const int k = (threadIdx.x + 256 * i) * EV;
        if (k >= d) continue;
#pragma unroll
        for (int e = 0; e < EV; e += 4)
            *(float4*)(hr + k + e) = make_float4(piece_val<AT>(pc[i], e), piece_val<AT>(pc[i], e + 1),
                                                 piece_val<AT>(pc[i], e + 2), piece_val<AT>(pc[i], e + 3));
    }
    for (int k = 256 * MAXP * EV + threadIdx.x; k < d; k += 256) hr[k] = Act<AT>::ld(er, k);  // wider rows
    __syncthreads();
    if (threadIdx.x == 0) {
        int depth = 0;
        uint64_t a0 = 0, a1 = 0;
        for (int x = node; x >= 0;) {
            if (x < 64) a0 |= 1ull << x;
            else a1 |= 1ull << (x - 64);
            if (x != node) ++depth;
            const int p = par[x];
            if (!dcheck(chk, x == 0 ? p == -1 : p >= 0 && p < x, CHK_PARENT)) break;
            x = p;
        }
        const bool slots_ok = dcheck(chk, Lc >= 0 && Lc + n_tree <= sp->cap, CHK_SLOTS);
        row_pos[t] = Lc + depth;
        row_slot[t] = slots_ok ? Lc + node : -1;
        row_anc[2 * t] = a0;
        row_anc[2 * t + 1] = a1;
    }
}

hipError_t launch_embed(int atype, const void* embed, int d, int vocab, const int* rtok, const int* rpar,
                        const StepParams* sp, int T, float* h, int* row_pos, int* row_slot, uint64_t* row_anc,
                        int* chk, hipStream_t s) {
    if (atype == ET_BF16)
        hipLaunchKernelGGL(k_embed<uint16_t>, dim3(T), dim3(256), 0, s, (const uint16_t*)embed, d, vocab, rtok, rpar,
                           sp, h, row_pos, row_slot, row_anc, chk);
    else
        hipLaunchKernelGGL(k_embed<float>, dim3(T), dim3(256), 0, s, (const float*)embed, d, vocab, rtok, rpar, sp,
                           h, row_pos, row_slot, row_anc, chk);
    return hipGetLastError();
}

// ---------------------------------------------------------------- draft top-K

// Top-K tokens of one logits row per workgroup with their softmax
// probabilities over the whole vocabulary (the K candidates of a drafted
// position and their normalised probabilities, Alg. 1 and Sec. 4.2
// "Token-Level Information").  Each of the 1024 threads scans a strided
// slice of the row keeping its KL best (value descending, index ascending on
// ties) in a sorted register list, and an online (max, sum of exp) pair.
// The workgroup then pops the best list head K times (workgroup argmax over
// the heads, by value then lower index) and combines the (max, sum) pairs:
// lanes by a fixed butterfly, waves in wave order.  NaN entries are skipped
// and reported in flag.
static constexpr int TOPK_THREADS = 1024;

__device__ __forceinline__ bool tk_better(float a, int ia, float b, int ib) {
    return a > b || (a == b && ia < ib);
}
__device__ __forceinline__ void ms_combine(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    s = (m == -INFINITY ? 0.f : s * __expf(m - M)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - M));
    m = M;
}

template <int KL>
__global__ void __launch_bounds__(TOPK_THREADS) k_topk(const float* logits, int V, int K, int* ids, float* probs,
                                                       int* flag) {
    __shared__ float sh_v[TOPK_THREADS / 64], sh_m[TOPK_THREADS / 64], sh_s[TOPK_THREADS / 64];
    __shared__ int sh_i[TOPK_THREADS / 64];
    const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const float* x = logits + (size_t)row * V;
    float lv[KL];
    int li[KL];
#pragma unroll
    for (int k = 0; k < KL; ++k) { lv[k] = -INFINITY; li[k] = 0x7fffffff; }
    float m = -INFINITY, s = 0.f;
    int nan = 0;
    for (int v = tid; v < V; v += TOPK_THREADS) {
        const float y = x[v];
        if (y != y) { nan = 1; continue; }
        if (y > m) { s = (m == -INFINITY ? 0.f : s * __expf(m - y)) + 1.f; m = y; }
        else s += __expf(y - m);
        if (tk_better(y, v, lv[KL - 1], li[KL - 1])) {
            // insert into the sorted list: shift the worse entries down
            float cv = y;
            int ci = v;
#pragma unroll
            for (int k = 0; k < KL; ++k) {
                if (tk_better(cv, ci, lv[k], li[k])) {
                    const float tv = lv[k];
                    const int ti = li[k];
                    lv[k] = cv; li[k] = ci;
                    cv = tv; ci = ti;
                }
            }
        }
    }
    // softmax normaliser of the row
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float m2 = __shfl_xor(m, o), s2 = __shfl_xor(s, o);
        ms_combine(m, s, m2, s2);
    }
    for (int o = 1; o < 64; o <<= 1) nan |= __shfl_xor(nan, o);
    if (lane == 0) { sh_m[w] = m; sh_s[w] = s; sh_i[w] = nan; }
    __syncthreads();
    float M = sh_m[0], S = sh_s[0];
    nan = sh_i[0];
    for (int k = 1; k < TOPK_THREADS / 64; ++k) {
        ms_combine(M, S, sh_m[k], sh_s[k]);
        nan |= sh_i[k];
    }
    __syncthreads();
    // K rounds of workgroup argmax over the list heads
    for (int r = 0; r < K; ++r) {
        float bv = lv[0];
        int bi = li[0];
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const float ov = __shfl_xor(bv, o);
            const int oi = __shfl_xor(bi, o);
            if (tk_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
        }
        if (lane == 0) { sh_v[w] = bv; sh_i[w] = bi; }
        __syncthreads();
        bv = sh_v[0];
        bi = sh_i[0];
        for (int k = 1; k < TOPK_THREADS / 64; ++k)
            if (tk_better(sh_v[k], sh_i[k], bv, bi)) { bv = sh_v[k]; bi = sh_i[k]; }
        __syncthreads();
        if (tid == 0) {
            const bool ok = bi != 0x7fffffff;  // fewer than K finite entries: id -1, probability 0
            ids[(size_t)row * K + r] = ok ? bi : -1;
            probs[(size_t)row * K + r] = ok && S > 0.f ? __expf(bv - M) / S : 0.f;
        }
        if (li[0] == bi) {  // the owner pops its head (ids are unique within a row)
#pragma unroll
            for (int k = 0; k + 1 < KL; ++k) { lv[k] = lv[k + 1]; li[k] = li[k + 1]; }
            lv[KL - 1] = -INFINITY;
            li[KL - 1] = 0x7fffffff;
        }
    }
    if (tid == 0 && nan) flag[row] = 1;
}

hipError_t launch_topk(const float* logits, int n, int V, int K, int* ids, float* probs, int* flag, hipStream_t s) {
    if (n < 1 || V < 1 || K < 1 || K > 16) return hipErrorInvalidValue;
    if (K <= 1) hipLaunchKernelGGL(k_topk<1>, dim3(n), dim3(TOPK_THREADS), 0, s, logits, V, K, ids, probs, flag);
    else if (K <= 2) hipLaunchKernelGGL(k_topk<2>, dim3(n), dim3(TOPK_THREADS), 0, s, logits, V, K, ids, probs, flag);
    else if (K <= 4) hipLaunchKernelGGL(k_topk<4>, dim3(n), dim3(TOPK_THREADS), 0, s, logits, V, K, ids, probs, flag);
    else if (K <= 8) hipLaunchKernelGGL(k_topk<8>, dim3(n), dim3(TOPK_THREADS), 0, s, logits, V, K, ids, probs, flag);
    else hipLaunchKernelGGL(k_topk<16>, dim3(n), dim3(TOPK_THREADS), 0, s, logits, V, K, ids, probs, flag);
    return hipGetLastError();
}

// ---------------------------------------------------------------- greedy acceptance

// Per-row argmax, lowest index on ties, in ACC_PARTS contiguous parts per
// row (one workgroup each); per-part NaN flag.  The walk merges the parts in
// increasing order, so a tie across parts also keeps the lowest index.
static constexpr int ACC_PARTS = 8;

__global__ void __launch_bounds__(256) k_accept_argmax(const float* logits, int V, int* gbuf) {
    __shared__ float sv[4];
    __shared__ int si[4], sn[4];
    const int t = blockIdx.y, part = blockIdx.x;
    const int len = (V + ACC_PARTS - 1) / ACC_PARTS;
    const int lo = part * len, hi = min(V, lo + len);
    const float* row = logits + (size_t)t * V;
    float best = -INFINITY;
    int bi = 0x7fffffff, nan = 0;
    for (int v = lo + threadIdx.x; v < hi; v += 256) {
        const float x = row[v];
        if (x != x) nan = 1;
        else if (bi == 0x7fffffff || x > best) { best = x; bi = v; }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ob = __shfl_xor(best, o);
        const int oi = __shfl_xor(bi, o);
        nan |= __shfl_xor(nan, o);
        if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) { sv[w] = best; si[w] = bi; sn[w] = nan; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < 4; ++k) {
            if (sv[k] > best || (sv[k] == best && si[k] < bi)) { best = sv[k]; bi = si[k]; }
            nan |= sn[k];
        }
        int* o = gbuf + ((size_t)t * ACC_PARTS + part) * 3;
        o[0] = bi;
        o[1] = __float_as_int(best);
        o[2] = nan;
    }
}

// Merge the parts of every row, then walk from the root: next = lowest-id
// child whose token equals the current node's argmax.
// result: [0] n_accepted, [1] bonus, [2] NaN, [3..] node ids.
__global__ void __launch_bounds__(128) k_accept_walk(const int* gbuf, int T, const int* rtok, const int* rpar, int* result,
                                                     int* chk) {
    __shared__ int fmc[128], gs[128];
    __shared__ int nanf;
    const int i = threadIdx.x;
    if (i == 0) nanf = 0;
    __syncthreads();
    if (i < T) {
        fmc[i] = 0x7fffffff;
        float best = -INFINITY;
        int bi = 0x7fffffff, nan = 0;
        for (int p = 0; p < ACC_PARTS; ++p) {
            const int* g = gbuf + ((size_t)i * ACC_PARTS + p) * 3;
            const float b = __int_as_float(g[1]);
            nan |= g[2];
            if (g[0] != 0x7fffffff && (bi == 0x7fffffff || b > best)) { best = b; bi = g[0]; }
        }
        gs[i] = bi;
        if (nan) atomicOr(&nanf, 1);
    }
    __syncthreads();
    if (i > 0 && i < T) {
        const int p = rpar[i];
        if (dcheck(chk, p >= 0 && p < i, CHK_ACCEPT_PARENT) && rtok[i] == gs[p]) atomicMin(&fmc[p], i);
    }
    __syncthreads();
    if (i == 0) {
        int cur = 0, n = 1;
        result[3] = 0;
        while (fmc[cur] != 0x7fffffff) {
            cur = fmc[cur];
            result[3 + n] = cur;
            ++n;
        }
        result[0] = n;
        result[1] = gs[cur];
        result[2] = nanf;
    }
}

hipError_t launch_accept(const float* logits, int T, int V, const int* rtok, const int* rpar, int* gbuf, int* result,
                         int* chk, hipStream_t s) {
    if (T < 1 || T > 128) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_accept_argmax, dim3(ACC_PARTS, T), dim3(256), 0, s, logits, V, gbuf);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_accept_walk, dim3(1), dim3(128), 0, s, gbuf, T, rtok, rpar, result, chk);
    return hipGetLastError();
}

// ---------------------------------------------------------------- KV compaction

// One workgroup per (layer, kv head): stage the accepted slots' K and V in
// LDS, then write them to slots Lc .. Lc+n_acc-1.  Staging all reads before
// any write makes the move safe when a destination is a later node's source.
template <typename AT>
__global__ void __launch_bounds__(256) k_compact(AT* kc, AT* vt, int hd, int ctx_cap, const StepParams* sp,
                                                 const int* acc, int n_acc, int* chk) {
    constexpr int ET = sizeof(AT) == 2 ? ET_BF16 : ET_F32;
    extern __shared__ unsigned char smem[];
    AT* buf = (AT*)smem;
    const int Lc = sp->Lc;
    if constexpr (kDeviceChecks) {
        // every thread checks the whole path, so all of them leave together
        bool ok = Lc >= 0 && Lc + sp->n_tree <= sp->cap && sp->cap <= ctx_cap && acc[0] == 0;
        for (int j = 1; j < n_acc; ++j) ok = ok && acc[j] > acc[j - 1] && acc[j] < sp->n_tree;
        if (!dcheck(chk, ok, CHK_COMPACT)) return;
    }
    AT* kb = kc + (size_t)blockIdx.x * ctx_cap * hd;
    AT* vb = vt + (size_t)blockIdx.x * ctx_cap * hd;
    const int n = n_acc * hd;
    for (int i = threadIdx.x; i < n; i += 256) buf[i] = kb[kv_k_off(ET, Lc + acc[i / hd], i % hd, hd, ctx_cap)];
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += 256) kb[kv_k_off(ET, Lc + i / hd, i % hd, hd, ctx_cap)] = buf[i];
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += 256) buf[i] = vb[kv_v_off(ET, Lc + acc[i / hd], i % hd, hd, ctx_cap)];
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += 256) vb[kv_v_off(ET, Lc + i / hd, i % hd, hd, ctx_cap)] = buf[i];
}

hipError_t launch_compact(int atype, void* kc, void* vt, int L, int Hkv, int hd, int ctx_cap, const StepParams* sp,
                          const int* accepted, int n_acc, int* chk, hipStream_t s) {
    if (n_acc < 1 || n_acc > 129) return hipErrorInvalidValue;
    if (atype == ET_BF16)
        hipLaunchKernelGGL(k_compact<uint16_t>, dim3(L * Hkv), dim3(256), (size_t)n_acc * hd * 2, s, (uint16_t*)kc,
                           (uint16_t*)vt, hd, ctx_cap, sp, accepted, n_acc, chk);
    else
        hipLaunchKernelGGL(k_compact<float>, dim3(L * Hkv), dim3(256), (size_t)n_acc * hd * 4, s, (float*)kc,
                           (float*)vt, hd, ctx_cap, sp, accepted, n_acc, chk);
    return hipGetLastError();
}

// ---------------------------------------------------------------- copy / fill

__global__ void k_copy16(i32x4* dst, const i32x4* src, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}
__global__ void k_fill0(unsigned char* dst, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        dst[i] = 0;
}

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t s) {
    if (bytes % 16) return hipErrorInvalidValue;
    const size_t n = bytes / 16;
    size_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_copy16, dim3((unsigned)blocks), dim3(256), 0, s, (i32x4*)dst, (const i32x4*)src, n);
    return hipGetLastError();
}

hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s) {
    size_t blocks = (bytes + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill0, dim3((unsigned)blocks), dim3(256), 0, s, (unsigned char*)dst, bytes);
    return hipGetLastError();
}

}  // namespace cas
