// Internal interface between the gfx950 kernels (kernels.hip) and the
// runtime behind the C ABI (runtime.hip).  Not installed, not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace cas {

enum ElemType { ET_F32 = 0, ET_BF16 = 1, ET_I8 = 2, ET_I4 = 3 };

// ---------------------------------------------------------------------------
// Fragment-tiled operand layout of the weight-streaming GEMM.
//
// A 16-byte fragment holds E consecutive k of one row (E = 4 fp32, 8 bf16, 16
// int8).  A chunk covers KC = 16E consecutive k as 4 steps u x 4 lane groups
// g: lane (g, r) holds k = c*KC + g*4E + u*E + [0, E) of row r at step u.
// Weights are stored as 16-row tiles, each a run of chunks, each chunk 4
// steps of 64 lane fragments (1 KB per step): a wave's load of one step is
// 1 KB of contiguous memory.  Activations (the GEMM's B operand, T rows padded
// to NT 16-row column tiles) are stored chunk by chunk, step by step, column
// tile by column tile, again 1 KB per (step, column tile).  K is padded with
// zeros to a multiple of KC.
constexpr int FRAG_U = 4;
__host__ __device__ inline int frag_elems(int et) { return et == ET_F32 ? 4 : (et == ET_BF16 ? 8 : 16); }
__host__ __device__ inline int frag_elem_bytes(int et) { return et == ET_F32 ? 4 : (et == ET_BF16 ? 2 : 1); }
__host__ __device__ inline int chunk_k(int et) { return 4 * FRAG_U * frag_elems(et); }
__host__ __device__ inline int pad_k(int K, int et) { return (K + chunk_k(et) - 1) / chunk_k(et) * chunk_k(et); }
// column tiles of the activation layout for T rows (the GEMM's NT)
__host__ __device__ inline int col_tiles(int T) { return T <= 32 ? 2 : (T <= 64 ? 4 : 8); }
// element offset of W[n][k] (padded width Kp) and of X[t][k] (NT column tiles)
__host__ __device__ inline size_t wt_off(int n, int k, int Kp, int E) {
    const int KC = 16 * E, c = k / KC, kk = k % KC;
    const int g = kk / (4 * E), u = (kk / E) & 3, e = kk % E, lane = g * 16 + (n & 15);
    return ((((size_t)(n >> 4) * (Kp / KC) + c) * FRAG_U + u) * 64 + lane) * E + e;
}
// The K-major order of a tiled weight matrix: the same 1 KB blocks, block b of
// tile n at (b * ntiles + n) KB instead of (n * bpt + b) KB (bpt: blocks per
// tile).  byte: offset in the tile-major order.  The GEMM workgroups walking
// K then read adjacent blocks at the same time, which streams the gate/up and
// LM head matrices faster (the runtime's table of block orders gives the
// measurements); the other matrices stay tile-major.
__host__ __device__ inline size_t wt_kmajor(size_t byte, int ntiles, int bpt) {
    const size_t blk = byte >> 10;
    return ((blk % bpt) * ntiles + blk / bpt) * 1024 + (byte & 1023);
}
__host__ __device__ inline size_t xt_off(int t, int k, int NT, int E) {
    const int KC = 16 * E, c = k / KC, kk = k % KC;
    const int g = kk / (4 * E), u = (kk / E) & 3, e = kk % E, lane = g * 16 + (t & 15);
    return ((((size_t)c * FRAG_U + u) * NT + (t >> 4)) * 64 + lane) * E + e;
}

// Packed int4 weights (ET_I4): codes q in [-7, 7] stored as the nibble q + 8,
// chunked like int8 (256 k per chunk, the activations keep the int8 layout).
// A 16-row tile's chunk is two 1 KB blocks: block b holds the int8 steps 2b
// and 2b + 1, lane (g, r) 16 bytes, bytes [8h, 8h + 8) for step 2b + h, byte j
// the step's k-offsets j (low nibble) and j + 8 (high nibble).  One wave load
// of a block feeds two int8 MFMA steps.
__host__ __device__ inline size_t wt4_byte(int n, int k, int Kp, int* nibble) {
    const int c = k >> 8, kk = k & 255, g = kk >> 6, u = (kk >> 4) & 3, e = kk & 15;
    const int lane = g * 16 + (n & 15);
    *nibble = e >> 3;
    return ((((size_t)(n >> 4) * (Kp >> 8) + c) * 2 + (u >> 1)) * 64 + lane) * 16 + (u & 1) * 8 + (e & 7);
}

// ---------------------------------------------------------------------------
// KV cache layout: one block of ctx_cap x hd elements per (layer, kv head).
// fp32 models: K row-major [slot][hd], V slot-contiguous [hd][slot].
// bf16 models: 32-slot tiles of 32*hd elements, each laid out as the MFMA
// fragments the tree attention reads, so every wave load is 1 KB contiguous:
//   K: fragment (h2, u) of 64 lanes x 8 elements; lane (g, r) holds key
//      slot 8*(r/4) + 4*h2 + r%4 of the tile, d = g*hd/4 + u*8 + [0, 8)
//   V: fragment dt of 64 lanes x 8 elements; lane (g, r) holds d = 16*dt + r,
//      slots 8*g + [0, 8) of the tile
__host__ __device__ inline size_t kv_k_tiled(int slot, int d, int hd) {
    const int ti = slot >> 5, sl = slot & 31;
    const int r = 4 * (sl >> 3) + (sl & 3), h2 = (sl >> 2) & 1;
    const int dg = hd / 4, g = d / dg, u = (d % dg) >> 3, e = d & 7;
    return (size_t)ti * 32 * hd + ((size_t)(h2 * (hd / 32) + u) * 64 + g * 16 + r) * 8 + e;
}
__host__ __device__ inline size_t kv_v_tiled(int slot, int d, int hd) {
    const int ti = slot >> 5, sl = slot & 31;
    return (size_t)ti * 32 * hd + ((size_t)(d >> 4) * 64 + (sl >> 3) * 16 + (d & 15)) * 8 + (sl & 7);
}
__host__ __device__ inline size_t kv_k_off(int et, int slot, int d, int hd, int ctx_cap) {
    return et == ET_BF16 ? kv_k_tiled(slot, d, hd) : (size_t)slot * hd + d;
}
__host__ __device__ inline size_t kv_v_off(int et, int slot, int d, int hd, int ctx_cap) {
    return et == ET_BF16 ? kv_v_tiled(slot, d, hd) : (size_t)d * ctx_cap + slot;
}

// GEMM epilogues.  Rows n of the weight matrix produce output column n.
enum Epilogue {
    EPI_STORE = 0,   // out_f32[t*ldo + n] = y
    EPI_RESID = 1,   // out_f32[t*ldo + n] += y
    EPI_RAW = 2,     // out_i32[t*ldo + n] = integer accumulator (int8 weights only)
    EPI_SWIGLU = 3,  // weight rows interleaved (gate m, up m): out_act[t*ldo + m] = silu(gate)*up
    EPI_QKV = 4      // weight rows: q heads, k heads, v heads; q/k rows pair-interleaved for RoPE
};

// Dynamic per-call values that kernels read from device memory, so one
// captured graph serves every call with the same static shape.
struct StepParams {
    int Lc;           // committed slots
    int node_offset;  // id of this call's first node in the round
    int n_tree;       // nodes of the round after this call
    int cap;          // KV slots the device checks allow (the cache's capacity)
};

// Device checks of a CAS_DEBUG build.  Each guards an access whose bounds
// rest on values the kernels read from device memory (step parameters, the
// round's tokens and parents, row slots and positions, accepted ids): the
// host validates all of them before they are copied, so in a correct
// program no check fails.  A failed check stores its code in the context's
// check word (a plain store: when several fail, any one code remains) and
// the guarded access is skipped, so the kernel still ends normally.  Release
// builds compile every check to `true`.
enum DeviceCheck {
    CHK_NONE = 0,
    CHK_TREE_SIZE = 1,      // n_tree > 128, or a row outside the round
    CHK_TOKEN = 2,          // token id outside [0, vocab)
    CHK_PARENT = 3,         // parent not in [0, node) (root: not -1)
    CHK_SLOTS = 4,          // Lc + n_tree beyond the slot capacity
    CHK_POSITION = 5,       // RoPE position outside the table
    CHK_KV_WRITE = 6,       // KV write slot outside the cache
    CHK_ATTN_SLOTS = 7,     // attention over slots beyond the capacity
    CHK_COMPACT = 8,        // accepted ids not increasing from the root within the round
    CHK_ACCEPT_PARENT = 9,  // acceptance walk met a parent not below its child
    CHK_COUNT = 10
};
#ifdef CAS_DEBUG
constexpr bool kDeviceChecks = true;
#else
constexpr bool kDeviceChecks = false;
#endif
// true when ok (always, in release builds); else records code and returns false
__device__ __forceinline__ bool dcheck(int* word, bool ok, int code) {
    if constexpr (kDeviceChecks) {
        if (!ok && word) *word = code;
        return ok;
    } else {
        return true;
    }
}

struct GemmArgs {
    const void* W;      // tiled weights, N rows, padded width Kp (element type wtype)
    const void* X;      // tiled activations, T rows in col_tiles(T) column tiles (same type)
    int N, Kp, T;
    const float* xs;    // int8: per-row activation scales [T]
    const float* ws;    // int8: per-output-channel weight scales [N]
    void* out;          // epilogue output (EPI_SWIGLU: tiled activations of width out_k)
    int ldo;
    int out_k;          // EPI_SWIGLU: width of the output rows (the pad up to pad_k is zeroed)
    // EPI_QKV
    const float* rope_cos;  // [ctx_cap][head_dim/2]
    const float* rope_sin;
    const int* row_pos;     // [T] RoPE position of each row
    const int* row_slot;    // [T] KV slot of each row
    void* kc;               // key cache of the layer (act type, cache layout)
    void* vt;               // value cache of the layer (act type, cache layout)
    int H, Hkv, hd, ctx_cap;
    // split-K partial sums (launch_gemm_parts): split k writes its fp32 sums
    // to out + k * part_stride, [T][ldo]
    int ksplit;
    size_t part_stride;
    // quantise on load (int8 / int4 weights, calls of at most QX_MAX_T rows;
    // gemm_qx_ok says which): X holds bf16 tiled rows of width xk (pad
    // columns zero), and each workgroup derives every row's scale amax / qx
    // and the codes of its own K range itself (xs unused).  0: X holds codes.
    int qx, xk;
    // merge on load (bf16 O projection of a call of one or two rows;
    // gemm_mx_ok says when): the input rows are the attention's mx_S split
    // partials ([split][H][T][hd] sums, [split][H][T][2] max and sum, H heads
    // of hd), merged by each workgroup for its own K range (X unused).
    // nullptr: off.
    const float* mx_o;
    const float* mx_ml;
    int mx_S;
    // GEMV-style tiles (wide GEMMs of one activation row, bf16 or int8
    // weights): the caller allows a summation order of its own (drafts; not
    // verify calls, whose rows must not depend on the tree size).  0: off.
    int gv;
    int* chk;  // device check word (CAS_DEBUG builds; may be nullptr)
    int kmaj;  // W is stored in the K-major block order (wt_kmajor)
};

// wtype: element type of W and X; atype: activation type written by the
// SWIGLU and QKV epilogues (ET_F32 or ET_BF16).
hipError_t launch_gemm(int wtype, int atype, int epi, const GemmArgs& a, hipStream_t s);
// Number of K splits for a residual projection of N rows whose partial sums
// a following RMSNorm adds to the residual stream: 1 = do not split (enough
// workgroups already, int8 weights, or too few stages).
int gemm_parts_count(int wtype, int N, int Kp, int T);
// The split-K form: a.ksplit splits, each writing fp32 sums of its K range to
// a.out + k * a.part_stride ([T][a.ldo]).
hipError_t launch_gemm_parts(int wtype, const GemmArgs& a, hipStream_t s);
// Whether a split-K GEMM of N rows (padded width Kp, T rows of activations,
// ksplit splits) can quantise its bf16 input on load (launch_gemm cannot).
bool gemm_qx_ok(int wtype, int N, int Kp, int T, int ksplit);
// Whether a split-K GEMM can merge its input rows from attention partials.
bool gemm_mx_ok(int wtype, int N, int Kp, int T, int ksplit);

struct AttnArgs {
    const void* q;        // [T][H][hd]
    const void* kc;       // key cache of the layer, Hkv blocks (cache layout)
    const void* vt;       // value cache of the layer, Hkv blocks (cache layout)
    const uint64_t* anc;  // [T][2]
    const StepParams* sp; // Lc, n_tree (device)
    int Lc_host, n_tree_host;  // the same values, known on the host when launching
    void* out;            // T rows of H*hd: tiled activations (out_tiled) or row-major
    int out_tiled;
    float* part_o;        // [splits][H][T][hd]
    float* part_ml;       // [splits][H][T][2]
    int T, H, Hkv, hd, ctx_cap;
    // efficient attention (win_len > 0): of the committed slots only
    // [0, win_sink) and [Lc - win_len, Lc) are visible; the grid covers only
    // the key tiles that hold them
    int win_sink, win_len;
    // bf16 path with qout set: the output is the rows' per-token codes in
    // [-qmax, qmax] (tiled int8 layout) with their scales, in place of out
    int8_t* qout;
    float* qscale;
    int qmax;
    // partials only: the consumer merges the splits itself (the merge is not launched)
    int no_merge;
    int* chk;  // device check word (CAS_DEBUG builds; may be nullptr)
};
size_t attention_work_bytes(int n_slots, int T, int H, int hd);
int attention_splits(int n_slots);
// KV splits of a forward whose committed slots are limited to a sink and a
// window (win_len 0: all of them)
int attention_splits_win(int Lc, int n_tree, int win_sink, int win_len);
// atype: ET_BF16 (MFMA path, then the merge of the KV splits) or ET_F32
// (plain path, ctx_cap <= 4096)
hipError_t launch_attention(int atype, const AttnArgs& a, hipStream_t s);
// Only the merge of S split partials (a.part_o, a.part_ml; a.T rows of a.H
// heads): bf16 rows into a.out, or with a.qout their codes and scales.
hipError_t launch_attn_merge(const AttnArgs& a, int S, hipStream_t s);
// Copy n slots of every kv head between the row-major [Hkv][n][hd] form and
// the cache layout of one layer (to_cache = 1: into the cache).
hipError_t launch_kv_convert(int atype, void* kc, void* vt, const void* k_rows, const void* v_rows, int Hkv,
                             int n, int hd, int ctx_cap, int to_cache, hipStream_t s);

// RMSNorm of rows of the fp32 residual stream h [T][d] with gains g:
// writes the normalised rows as tiled activations of act type (out) or, with
// q != NULL, their int8 quantisation (tiled int8 q, scales qs [T]) instead.
// With nparts > 0 the rows first take the pending split-K sums of the last
// projection: h += parts[0] + ... + parts[nparts-1] (in that order; part p at
// parts + p * pstride, [T][d]), stored back to h.
// qmax (127: int8 codes, 7: int4 codes kept one per byte) sets the range of
// the quantised output.
hipError_t launch_rmsnorm(int atype, float* h, const float* g, int T, int d, float eps, void* out, int8_t* q,
                          float* qs, const float* parts, int nparts, size_t pstride, int qmax, hipStream_t s);
// Per-row quantisation of x [T][K] (act type) to codes in [-qmax, qmax]
// (127 or 7).  tiled = 1: x is tiled activations and q is written tiled;
// tiled = 0: both row-major.
hipError_t launch_quant_rows(int atype, const void* x, int T, int K, int8_t* q, float* qs, int tiled, int qmax,
                             hipStream_t s);
// Tiled int8 copy of a tiled weight matrix (N rows, width K): per-row scales.
// skm / dkm: the source / the copy in the K-major block order.
hipError_t launch_quant_weight(int wtype, const void* w, int N, int K, int8_t* q, float* qs, hipStream_t s,
                               int skm = 0, int dkm = 0);
// Packed int4 copy (wt4_byte layout, width pad_k(K, ET_I8)) of a tiled weight
// matrix: per-row scales amax / 7.
hipError_t launch_quant_weight_i4(int wtype, const void* w, int N, int K, uint8_t* q, float* qs, hipStream_t s,
                                  int skm = 0, int dkm = 0);
hipError_t launch_untile_weight_i4(const uint8_t* src, int N, int K, int8_t* dst, hipStream_t s);
// Row-major int8 codes in [-7, 7] [N][K] -> packed int4 (for the kernel-level entry point).
hipError_t launch_pack_weight_i4(const int8_t* src, int N, int K, uint8_t* dst, hipStream_t s);
// Row-major W [rows][K] (act type) -> tiled weights of width pad_k(K).
// Source row i lands at tiled row row0 + map(i): mode 0 map(i) = i; mode 1
// (q/k heads of hd rows) puts rows i and i + hd/2 of a head next to each
// other; mode 2 map(i) = 2i (interleave with another matrix at 2i + 1).
// kmaj_tiles > 0: dst is stored in the K-major block order of a matrix of
// that many 16-row tiles.
hipError_t launch_tile_weight(int atype, const void* src, int rows, int K, void* dst, int row0, int mode, int hd,
                              hipStream_t s, int kmaj_tiles = 0);
hipError_t launch_untile_weight_i8(const int8_t* src, int N, int K, int8_t* dst, hipStream_t s);
// Row-major X [T][K] -> tiled activations (col_tiles(T) tiles, width pad_k).
hipError_t launch_tile_act(int atype, const void* src, int T, int K, void* dst, hipStream_t s);
// Tiled activations of T rows (col_tiles(T) tiles) -> row-major X [T][K].
hipError_t launch_untile_act(int atype, const void* src, int T, int K, void* dst, hipStream_t s);
// Embedding gather for the call's rows plus tree metadata (depth -> position,
// slot, ancestor masks) from the round's parent array.
hipError_t launch_embed(int atype, const void* embed, int d, int vocab, const int* round_tokens,
                        const int* round_parent, const StepParams* sp, int T, float* h, int* row_pos, int* row_slot,
                        uint64_t* row_anc, int* chk, hipStream_t s);
// Greedy acceptance: per-row argmax of logits [T][V], then the tree walk.
// result: [0] = n_accepted, [1] = bonus token, [2] = NaN flag, [3..] = node ids.
hipError_t launch_accept(const float* logits, int T, int V, const int* round_tokens, const int* round_parent,
                         int* argmax_buf, int* result, int* chk, hipStream_t s);
// Top-K ids (value descending, lower id on ties; -1 past the finite
// entries) and softmax probabilities of each of n logits rows [n][V]; K in
// [1, 16]; flag[row] set to 1 when the row holds a NaN (not cleared here).
hipError_t launch_topk(const float* logits, int n, int V, int K, int* ids, float* probs, int* flag, hipStream_t s);
// Move accepted slots Lc+acc[j] -> Lc+j in every layer (K and V caches).
hipError_t launch_compact(int atype, void* kc, void* vt, int L, int Hkv, int hd, int ctx_cap,
                          const StepParams* sp, const int* accepted, int n_acc, int* chk, hipStream_t s);
hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t s);
hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s);

}  // namespace cas
