// Internal interface between the gfx950 kernels (kernels.hip) and the
// runtime behind the C ABI (runtime.hip).  Not installed, not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace cas {

enum ElemType { ET_F32 = 0, ET_BF16 = 1, ET_I8 = 2 };

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
    int pad;
};

struct GemmArgs {
    const void* W;      // [N][K] weights (element type wtype)
    const void* X;      // [T][K] activations (same element type)
    int N, K, T;
    const float* xs;    // int8: per-row activation scales [T]
    const float* ws;    // int8: per-output-channel weight scales [N]
    void* out;          // epilogue output
    int ldo;
    // EPI_QKV
    const float* rope_cos;  // [ctx_cap][head_dim/2]
    const float* rope_sin;
    const int* row_pos;     // [T] RoPE position of each row
    const int* row_slot;    // [T] KV slot of each row
    void* kc;               // [Hkv][ctx_cap][hd] (act type)
    void* vt;               // [Hkv][hd][ctx_cap] (act type)
    int H, Hkv, hd, ctx_cap;
};

// wtype: element type of W and X; atype: activation type written by the
// SWIGLU and QKV epilogues (ET_F32 or ET_BF16).
hipError_t launch_gemm(int wtype, int atype, int epi, const GemmArgs& a, hipStream_t s);

struct AttnArgs {
    const void* q;        // [T][H][hd]
    const void* kc;       // [Hkv][ctx_cap][hd]
    const void* vt;       // [Hkv][hd][ctx_cap]
    const uint64_t* anc;  // [T][2]
    const StepParams* sp; // Lc, n_tree (device)
    int Lc_host, n_tree_host;  // the same values, known on the host when launching
    void* out;            // [T][H*hd]
    float* part_o;        // [splits][H][T][hd]
    float* part_ml;       // [splits][H][T][2]
    int T, H, Hkv, hd, ctx_cap;
};
size_t attention_work_bytes(int n_slots, int T, int H, int hd);
int attention_splits(int n_slots);
// atype: ET_BF16 (MFMA path, then launch_attention_combine merges the KV
// splits) or ET_F32 (plain path, ctx_cap <= 4096, no combine step)
hipError_t launch_attention(int atype, const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_combine(int atype, const AttnArgs& a, hipStream_t s);

// RMSNorm of rows of the fp32 residual stream h [T][d] with gains g:
// writes the normalised rows in act type (out) or, with q != NULL, their int8
// quantisation (q [T][d], qs [T]) instead.
hipError_t launch_rmsnorm(int atype, const float* h, const float* g, int T, int d, float eps,
                          void* out, int8_t* q, float* qs, hipStream_t s);
// Per-row int8 quantisation of x [T][K] (act type).
hipError_t launch_quant_rows(int atype, const void* x, int T, int K, int8_t* q, float* qs, hipStream_t s);
// Per-row int8 copy of a weight matrix [N][K] (act type).
hipError_t launch_quant_weight(int wtype, const void* w, int N, int K, int8_t* q, float* qs, hipStream_t s);
// Embedding gather for the call's rows plus tree metadata (depth -> position,
// slot, ancestor masks) from the round's parent array.
hipError_t launch_embed(int atype, const void* embed, int d, const int* round_tokens, const int* round_parent,
                        const StepParams* sp, int T, float* h, int* row_pos, int* row_slot,
                        uint64_t* row_anc, hipStream_t s);
// Greedy acceptance: per-row argmax of logits [T][V], then the tree walk.
// result: [0] = n_accepted, [1] = bonus token, [2] = NaN flag, [3..] = node ids.
hipError_t launch_accept(const float* logits, int T, int V, const int* round_tokens, const int* round_parent,
                         int* argmax_buf, int* result, hipStream_t s);
// Move accepted slots Lc+acc[j] -> Lc+j in every layer (K and V caches).
hipError_t launch_compact(int atype, void* kc, void* vt, int L, int Hkv, int hd, int ctx_cap,
                          const StepParams* sp, const int* accepted, int n_acc, hipStream_t s);
hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t s);
hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s);

}  // namespace cas
