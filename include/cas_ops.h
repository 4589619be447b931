/*
 * cas_ops.h - kernel-level entry points of the CAS-Spec tree decoder library,
 * on caller-owned DEVICE buffers.
 *
 * These expose single kernels of the forward of cas.h so that each can be
 * checked against a CPU definition on identical inputs, and timed alone.
 * All pointers are device pointers (except where noted) owned by the caller;
 * `stream` is a hipStream_t (NULL = the null stream).  Every call is
 * asynchronous on that stream and returns CAS_ERR_ARG / CAS_ERR_UNSUPPORTED
 * for shapes it does not handle, CAS_ERR_DEVICE if the launch fails.
 */
#ifndef CAS_OPS_H
#define CAS_OPS_H

#include "cas.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { CAS_W_F32 = 0, CAS_W_BF16 = 1, CAS_W_I8 = 2, CAS_W_I4 = 3 } cas_wtype;
typedef enum {
    CAS_EPI_STORE = 0,   /* out[t*ldo + n] = y (float32) */
    CAS_EPI_RESID = 1,   /* out[t*ldo + n] += y (float32 residual stream) */
    CAS_EPI_RAW_I32 = 2  /* out[t*ldo + n] = integer accumulator (int32; int8 and int4 only) */
} cas_epi;

/*
 * Linear layer y[t][n] = sum_k X[t][k] W[n][k] for t < T, n < N (the weight
 * streaming GEMM of every projection and the LM head).
 *   W: [N][K] row-major, element type wtype (float32, bf16 bits, int8; for
 *      CAS_W_I4 int8 codes in [-7, 7], which the library packs to 4 bits)
 *   X: [T][K] row-major, same element type as W (int8 codes for CAS_W_I4)
 *   xs, ws: for CAS_W_I8 / CAS_W_I4 the per-row activation scales [T] and
 *           per-output channel weight scales [N]; y = (float(acc) * xs[t]) * ws[n]
 *           (ignored for the other types; unused with CAS_EPI_RAW_I32)
 *   work: device scratch of at least cas_op_gemm_work_bytes(...) bytes; the
 *         operands are first rearranged there into the fragment-tiled layout
 *         the kernel streams (the layout the library keeps its weights in)
 * Limits: N multiple of 16, K multiple of 16, 1 <= T <= 128.
 * Accumulation: fp32 (float32, bf16 inputs), exact int32 (int8 and int4
 * inputs; the W4A4 form of activation quantisation, Sec. 4.1 and App. C, runs
 * its int4 codes on the int8 MFMA).  One-row calls (T = 1) with N >= 8192
 * and bf16 or int8 weights run the GEMV-style tiles the library uses for
 * one-node drafts (VALU dot products per lane, the four k-group lanes of a
 * row summed at the end), other calls the MFMA tiles.
 */
size_t cas_op_gemm_work_bytes(int32_t wtype, int32_t N, int32_t K, int32_t T);
cas_status cas_op_gemm(int32_t wtype, const void* W, const void* X, int32_t N, int32_t K, int32_t T,
                       const float* xs, const float* ws, int32_t epi, void* out, int32_t ldo,
                       void* work, size_t work_bytes, void* stream);

/*
 * Per-row symmetric int8 quantisation of activations (App. C, activation
 * quantisation; one row per token): s[t] = max_k |x[t][k]| / 127 (fp32),
 * q[t][k] = clamp(round-half-even(x[t][k] / s[t]), -127, 127); a zero row
 * gives s = 0, q = 0.  x: [T][K] of type atype (CAS_W_F32 or CAS_W_BF16).
 */
cas_status cas_op_quant_rows(int32_t atype, const void* x, int32_t T, int32_t K,
                             int8_t* q, float* s, void* stream);
/* The same rule with codes in [-qmax, qmax]: qmax 127 (int8, as above) or 7
 * (int4 codes of the W4A4 draft, one per int8 byte): s[t] = amax / qmax. */
cas_status cas_op_quant_rows_q(int32_t atype, const void* x, int32_t T, int32_t K, int32_t qmax,
                               int8_t* q, float* s, void* stream);

/* Per-output-channel int8 copy of W [N][K] (same rule, one row per output
 * channel), through the library's tiled weight layout: q [N][K] row-major,
 * s [N].  wtype: CAS_W_F32 or CAS_W_BF16; N and K multiples of 16; work:
 * device scratch of cas_op_quant_weight_work_bytes(...) bytes. */
size_t cas_op_quant_weight_work_bytes(int32_t wtype, int32_t N, int32_t K);
cas_status cas_op_quant_weight(int32_t wtype, const void* W, int32_t N, int32_t K,
                               int8_t* q, float* s, void* work, size_t work_bytes, void* stream);
/* Per-output-channel int4 copy of W (s[n] = amax / 7, codes in [-7, 7]),
 * through the library's tiled weights and its packed 4-bit layout, returned
 * unpacked: q [N][K] row-major int8 codes, s [N].  Same arguments, limits and
 * work size as cas_op_quant_weight. */
cas_status cas_op_quant_weight_i4(int32_t wtype, const void* W, int32_t N, int32_t K,
                                  int8_t* q, float* s, void* work, size_t work_bytes, void* stream);

/*
 * Tree-masked attention of one layer (bf16 storage, fp32 softmax):
 *   q:   [T][n_heads][head_dim] bf16 (after RoPE)
 *   k:   [n_kv_heads][ctx_cap][head_dim] bf16 keys (row-major)
 *   v:   [n_kv_heads][ctx_cap][head_dim] bf16 values (row-major)
 *   anc: [T][2] 64-bit ancestor-or-self masks over the round's nodes
 *        (bit j = node j, whose slot is Lc + j)
 *   out: [T][n_heads*head_dim] bf16
 * Query row t sees slots [0, Lc) and the slots Lc + j of the nodes j set in
 * anc[t]; n_tree nodes exist (Lc + n_tree <= ctx_cap, n_tree <= 128;
 * ctx_cap a multiple of 32).  head_dim 64 or 128; T <= 128.  work: device
 * scratch of cas_op_attention_work_bytes(...) bytes (the keys and values are
 * first copied there into the library's cache layout).
 */
cas_status cas_op_attention(const void* q, const void* k, const void* v, int32_t ctx_cap,
                            int32_t Lc, int32_t n_tree, int32_t T, int32_t n_heads,
                            int32_t n_kv_heads, int32_t head_dim, const uint64_t* anc,
                            void* out, void* work, size_t work_bytes, void* stream);
size_t cas_op_attention_work_bytes(int32_t Lc, int32_t n_tree, int32_t T, int32_t n_heads,
                                   int32_t head_dim, int32_t n_kv_heads, int32_t ctx_cap);

/*
 * cas_op_attention for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, kernels and results, without `work`.  The scratch (the
 * key and value copies in the library's cache layout, the step parameters
 * and the KV-split partials) is a device array of the library of
 * cas_op_attention_noalloc_max_bytes() bytes (64 MiB), one per GPU, held
 * until the process ends.  Calls whose cas_op_attention_work_bytes(...)
 * exceeds it return CAS_ERR_CAPACITY and do nothing.  Nothing is allocated:
 * no hipMalloc, hipFree or allocating library call.  The calling thread's
 * current device must be the device of `stream`.  All calls on one GPU
 * share its array: calls that overlap in time on one GPU (other threads or
 * streams) race; the call returns after its kernels have finished, so calls
 * made one after another from one thread do not.  Every byte of the array a
 * call reads is written by that call first.
 */
size_t cas_op_attention_noalloc_max_bytes(void);
cas_status cas_op_attention_noalloc(const void* q, const void* k, const void* v, int32_t ctx_cap, int32_t Lc,
                                    int32_t n_tree, int32_t T, int32_t n_heads, int32_t n_kv_heads,
                                    int32_t head_dim, const uint64_t* anc, void* out, void* stream);

/*
 * The fused quantisers of the forward, each run alone.  Activation
 * quantisation (Sec. 4.1; App. C) is applied by the forward inside three
 * kernels rather than by a separate pass; these entry points run exactly
 * those kernels, so their codes can be compared bit for bit with the row
 * quantiser's rule (cas_op_quant_rows_q) on identical inputs.
 *
 * RMSNorm of the residual rows, optionally straight to per-token codes (the
 * input of the QKV and gate/up projections of a quantised draft):
 *   h:      [T][d] fp32 residual rows (device).  With nparts > 0 the rows
 *           first take the pending split-K sums: h += parts[0] + ... +
 *           parts[nparts-1], summed in that order, stored back to h
 *   gain:   [d] fp32 gains; eps inside the square root (eps >= 0)
 *   parts:  [nparts][T][d] fp32 (nparts in [0, 8])
 *   qmax:   0: out receives the normalised rows [T][d] in the model type
 *           (atype CAS_W_BF16: bf16 bits rounded to nearest even; CAS_W_F32:
 *           fp32); 127 or 7: q [T][d] receives the codes and qs [T] the
 *           scales of those normalised (rounded) rows, s = amax / qmax,
 *           q = clamp(rne(x / s), -qmax, qmax), zero rows s = 0, q = 0
 *   work:   device scratch of cas_op_rmsnorm_work_bytes(...) bytes (the
 *           kernel's tiled output before it is written back row-major)
 * Limits: 1 <= T <= 128, d a multiple of 16, d <= 16384.
 */
size_t cas_op_rmsnorm_work_bytes(int32_t atype, int32_t T, int32_t d, int32_t qmax);
cas_status cas_op_rmsnorm(int32_t atype, float* h, const float* gain, int32_t T, int32_t d, float eps,
                          const float* parts, int32_t nparts, int32_t qmax, void* out, int8_t* q, float* qs,
                          void* work, size_t work_bytes, void* stream);

/*
 * Merge of the attention's KV-split partial states (the second kernel of
 * the tree attention of a bf16 model), optionally straight to the O
 * projection's per-token codes (the merge-and-quantise kernel of quantised
 * drafts):
 *   part_o:  [S][n_heads][T][head_dim] fp32: split s's unnormalised sum of
 *            2^(x_j - m) v_j over its keys j, where x_j is the score in base-2
 *            units (q.k_j / sqrt(head_dim) * log2(e))
 *   part_ml: [S][n_heads][T][2] fp32: (m, l) = the split's largest x_j and
 *            its sum of 2^(x_j - m)
 *   The merged row is sum_s 2^(m_s - M) part_o_s / sum_s 2^(m_s - M) l_s with
 *   M the running maximum, merged in split order, rounded to bf16.
 *   qmax 0: out [T][n_heads*head_dim] bf16 bits; 127 or 7: q [T][n_heads*
 *   head_dim] codes and qs [T] scales of those bf16 rows (row quantiser rule)
 *   work: device scratch of cas_op_attn_merge_work_bytes(...) bytes
 * Limits: S in [1, 64], 1 <= T <= 128, head_dim 64 or 128,
 * n_heads * head_dim <= 16384.
 */
size_t cas_op_attn_merge_work_bytes(int32_t T, int32_t n_heads, int32_t head_dim, int32_t qmax);
cas_status cas_op_attn_merge(const float* part_o, const float* part_ml, int32_t S, int32_t T, int32_t n_heads,
                             int32_t head_dim, int32_t qmax, uint16_t* out, int8_t* q, float* qs, void* work,
                             size_t work_bytes, void* stream);

/*
 * Split-K residual projection that quantises its bf16 input on load (the O
 * and down projections of one-node quantised drafts on bf16 models): every
 * workgroup takes the row's amax over the whole row, writes the codes of its
 * own K range by the row quantiser's rule (s = amax / qmax) and runs the
 * integer GEMM on them.
 *   wtype:  CAS_W_I8 (W: codes in [-127, 127], qmax 127) or CAS_W_I4 (W:
 *           codes in [-7, 7], packed to 4 bits by the library, qmax 7)
 *   W [N][K] row-major codes, ws [N] per-output-channel weight scales,
 *   x [T][K] bf16 bits (T = 1)
 *   parts:  [splits][T][N] fp32: split k's dequantised sums over its K range,
 *           (fp32(acc_k) * s) * ws[n]; splits = cas_op_gemm_qx_splits(...)
 *           (0: the shape does not take this form)
 *   work:   device scratch of cas_op_gemm_qx_work_bytes(...) bytes
 */
int32_t cas_op_gemm_qx_splits(int32_t wtype, int32_t N, int32_t K, int32_t T);
size_t cas_op_gemm_qx_work_bytes(int32_t wtype, int32_t N, int32_t K, int32_t T);
cas_status cas_op_gemm_qx(int32_t wtype, const int8_t* W, const float* ws, const uint16_t* x, int32_t N, int32_t K,
                          int32_t T, int32_t qmax, float* parts, void* work, size_t work_bytes, void* stream);

/* Plain device copy kernel (16-byte vector loads and stores): the reference
 * traffic for calibrating HBM byte counters.  bytes must be a multiple of 16. */
cas_status cas_op_copy(void* dst, const void* src, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* CAS_OPS_H */
