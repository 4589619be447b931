/*
 * cas.h - C ABI of the MI355X (gfx950) token-tree decoder step of CAS-Spec
 * (cascade adaptive self-speculative decoding, arXiv 2510.26843).
 *
 * One call, cas_forward, runs a Llama-style decoder over the nodes of a small
 * draft token tree against the KV cache.  The same call serves
 *   - the target model's verification of a whole tree in one pass with tree
 *     attention (Sec. 4.2, "Tree Cascade"; Sec. 2 on speculative decoding), and
 *   - the "virtual" draft models that a DSIA strategy switches on per call
 *     (Def. 4.1; Sec. 4.1 strategy list): layer sparsity (skip_mask) and
 *     activation quantisation (act_quant: per-token int8 activations against a
 *     per-output-channel int8 copy of the weights, or the W4A4 form with int4
 *     codes on both sides, App. C), including the
 *     tree-parallel draft calls over a leaf and its siblings (Sec. 4.2,
 *     "Tree-based Parallel Draft Generation").
 * cas_accept_tree performs greedy verification of the tree (lossless decoding,
 * Sec. 5.1: the output equals greedy autoregressive decoding), and
 * cas_kv_compact commits the accepted path into the cache that drafts and
 * target share (self-speculative decoding keeps no separate draft cache, Sec. 2).
 *
 * Conventions
 *   - Every entry point returns a cas_status; on any error nothing in the
 *     context changes and cas_last_error() describes the problem.  No C++
 *     exception or abort crosses this boundary.
 *   - All pointers passed in are host pointers borrowed for the duration of the
 *     call; the library owns every device buffer (weights, int8 copy, KV cache,
 *     workspaces, logits).
 *   - Work is enqueued on the context's HIP stream.  cas_forward returns before
 *     the GPU finishes unless logits_host is non-NULL; cas_accept_tree is
 *     synchronous; cas_kv_compact is asynchronous.
 *   - Tree nodes of one round are numbered 0..n-1 in an order where every
 *     parent precedes its children; node 0 is the root (the last bonus token,
 *     whose KV is not cached yet) and has parent -1.  Node j of the round lives
 *     in KV slot Lc + j, where Lc is the committed length; its position is
 *     Lc + depth(j).  A node attends to every committed slot and to the slots
 *     of its ancestors and itself.
 */
#ifndef CAS_H
#define CAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct cas_ctx cas_ctx;

typedef enum {
    CAS_OK = 0,
    CAS_ERR_ARG = 1,         /* malformed argument (NULL, size, range) */
    CAS_ERR_TREE = 2,        /* parent list is not a valid append to the round's tree */
    CAS_ERR_CAPACITY = 3,    /* beyond max_tree or max_ctx */
    CAS_ERR_UNSUPPORTED = 4, /* shape or mode this build does not handle */
    CAS_ERR_OOM = 5,         /* device allocation failed */
    CAS_ERR_DEVICE = 6,      /* HIP error, or NaN logits met by acceptance */
    CAS_ERR_STATE = 7        /* call out of order (accept before verify, ...) */
} cas_status;

typedef enum { CAS_F32 = 0, CAS_BF16 = 1 } cas_dtype;

/* Decoder shape.  Llama decoder: RMSNorm with eps inside the square root,
 * rotate-half RoPE (pairs i, i+head_dim/2; inv_freq_i = theta^(-2i/head_dim)),
 * grouped-query attention (query head h uses kv head h/(n_heads/n_kv_heads)),
 * SwiGLU FFN, no biases, untied embedding and LM head.
 * Limits: d_model, ffn_dim multiples of 16; head_dim 64 or 128;
 * n_heads * head_dim a multiple of 128 (bf16) or 64 (fp32); max_tree <= 128;
 * max_ctx <= 16256 (fp32 models: <= 3968). */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
    float rope_theta, rms_eps;
    int32_t dtype;     /* cas_dtype: storage type of weights, activations and KV */
    int32_t max_ctx;   /* KV slots: committed tokens plus the largest tree */
    int32_t max_tree;  /* most nodes in one round */
} cas_config;

/* Weight tensors, row-major [out][in] (embed, lm_head: [vocab][d_model];
 * norms: [d_model] float32 gains).  Element type is bf16 bit patterns
 * (uint16) for CAS_BF16 models and float32 for CAS_F32 models; norm gains are
 * always float32. */
typedef enum {
    CAS_T_EMBED = 0, CAS_T_LM_HEAD = 1, CAS_T_FINAL_NORM = 2,
    CAS_T_ATTN_NORM = 3, CAS_T_FFN_NORM = 4,
    CAS_T_WQ = 5, CAS_T_WK = 6, CAS_T_WV = 7, CAS_T_WO = 8,
    CAS_T_W_GATE = 9, CAS_T_W_UP = 10, CAS_T_W_DOWN = 11
} cas_tensor;

/* Create a context on HIP device `device`.  stream: a hipStream_t to enqueue
 * on, or NULL for a stream the context creates (default priority) and owns.
 * Allocates weights, KV cache (zeroed) and workspaces.  *out is NULL on error. */
cas_status cas_create(const cas_config* cfg, int device, void* stream, cas_ctx** out);
void cas_destroy(cas_ctx* ctx);
/* Message of the last error on this context (empty if none; never NULL). */
const char* cas_last_error(const cas_ctx* ctx);
/* Message of the last cas_create failure in this process. */
const char* cas_create_error(void);

/* Copy one weight tensor from host memory (layer is ignored for global
 * tensors).  bytes must equal the tensor's size.  Synchronous. */
cas_status cas_load_tensor(cas_ctx* ctx, int32_t tensor, int32_t layer, const void* host, size_t bytes);

/* Build the per-output-channel int8 copy of every layer's seven projections:
 * s[n] = max_k |W[n][k]| / 127 (fp32), q = clamp(round-half-even(W/s), +-127).
 * Required before act_quant calls (App. C, activation quantisation). */
cas_status cas_build_int8(cas_ctx* ctx);

/* Build the per-output-channel int4 copy of the same projections (the W4A4
 * form of activation quantisation, Sec. 4.1 and App. C): s[n] = max_k
 * |W[n][k]| / 7 (fp32), q = clamp(round-half-even(W/s), +-7), stored as 4-bit
 * codes (half the bytes of the int8 copy).  Required before act_quant = 2
 * calls.  Loading any tensor invalidates both copies. */
cas_status cas_build_int4(cas_ctx* ctx);

/* Commit n tokens as a causal sequence after the committed prefix (prefill),
 * in chunks of at most max_tree.  Leaves no round open. */
cas_status cas_prefill(cas_ctx* ctx, const int32_t* tokens, int32_t n);

/* Write committed KV of one layer directly (a cache restored from elsewhere):
 * k, v are [n_kv_heads][n][head_dim] in the model's storage type (bf16 bits
 * or float32), placed at slots 0..n-1.  Does not change the committed length. */
cas_status cas_kv_load(cas_ctx* ctx, int32_t layer, const void* k, const void* v, int32_t n);

/* Read KV slots 0..n-1 of one layer back to host memory, in the layout of
 * cas_kv_load ([n_kv_heads][n][head_dim], storage type).  Synchronous. */
cas_status cas_kv_read(cas_ctx* ctx, int32_t layer, void* k, void* v, int32_t n);

/* Set the committed length (e.g. after cas_kv_load, or to drop committed
 * tokens).  Must not exceed max_ctx.  Closes any open round. */
cas_status cas_set_committed(cas_ctx* ctx, int32_t n);
cas_status cas_committed_len(const cas_ctx* ctx, int32_t* n);

/*
 * Forward over n tree nodes, ids node_offset .. node_offset+n-1 of the round.
 *   tokens[n]       token ids in [0, vocab)
 *   tree_parent[n]  parent node id of each node (< its own id); -1 for node 0
 *   node_offset     0 starts a new round (node 0 must be among the nodes);
 *                   otherwise it must equal the round's current node count
 *                   (draft calls append the next tree level or a leaf with its
 *                   siblings)
 *   skip_mask       NULL (full depth) or n_layers bytes, 1 = skip that layer
 *                   (layer sparsity); a skipped layer is the identity on the
 *                   residual stream and writes no KV
 *   act_quant       0; 1 = int8 activations for every linear layer of the
 *                   non-skipped layers (needs cas_build_int8); 2 = int4
 *                   activations against the int4 copy (W4A4, needs
 *                   cas_build_int4).  Codes are per token: s = amax / 127 or
 *                   / 7.  The LM head, attention and KV cache keep the
 *                   model's precision
 *   logits_host     NULL keeps logits on the device; else [n][vocab] float32
 *                   copied out (synchronous)
 * Limits: node_offset + n <= max_tree, Lc + node_offset + n <= max_ctx.
 * A call with node_offset 0, no skipped layer and act_quant 0 is a verify
 * call: cas_accept_tree may follow it.
 */
cas_status cas_forward(cas_ctx* ctx, const int32_t* tokens, const int32_t* tree_parent,
                       int32_t n, int32_t node_offset, const uint8_t* skip_mask,
                       int32_t act_quant, float* logits_host);

/* Device pointer to the logits of the last forward, [n][vocab] float32; valid
 * until the next forward.  *n is the number of rows. */
cas_status cas_logits_device(const cas_ctx* ctx, const float** dptr, int32_t* n);

/*
 * Options of a draft forward.  A DSIA draft model (Def. 4.1) is the target
 * with one or more of these strategies switched on for the call (Sec. 4.1):
 *   skip_mask    layer sparsity: NULL or n_layers bytes, 1 = skip that layer
 *                (a suffix of skipped layers is early exit)
 *   act_quant    activation quantisation: 0; 1 = per-token int8
 *                activations (needs cas_build_int8); 2 = W4A4 (needs
 *                cas_build_int4)
 *   attn_sink,   efficient attention (StreamingLLM-style): attn_window > 0
 *   attn_window  limits the committed slots each row attends to to the first
 *                attn_sink and the last attn_window ones (tree ancestors stay
 *                visible); the kernels then read only those key tiles.
 *                attn_window = 0 keeps every committed slot (attn_sink is
 *                ignored).
 */
typedef struct {
    const uint8_t* skip_mask;
    int32_t act_quant;
    int32_t attn_sink;
    int32_t attn_window;
} cas_draft_opts;

/*
 * cas_forward with draft options (NULL opts: a plain forward, as
 * cas_forward with no skip mask and act_quant 0).  Same arguments, limits,
 * errors and synchronisation as cas_forward; negative attn_sink or
 * attn_window give CAS_ERR_ARG.  A call with attn_window > 0 is never a
 * verify call.
 */
cas_status cas_forward_draft(cas_ctx* ctx, const int32_t* tokens, const int32_t* tree_parent, int32_t n,
                             int32_t node_offset, const cas_draft_opts* opts, float* logits_host);

/*
 * Greedy verification of the tree of the last verify call: g[i] is the
 * argmax of node i's logits (lowest index on ties).  From the root, move to
 * the child (lowest id first) whose token equals g of the current node, while
 * there is one.  accepted[0..*n_accepted) receives the accepted node ids, root
 * first (capacity max_tree); *bonus_token = g of the last accepted node.
 * greedy must be 1.  NaN logits give CAS_ERR_DEVICE.  Synchronous.
 */
cas_status cas_accept_tree(cas_ctx* ctx, int32_t greedy, int32_t* accepted,
                           int32_t* n_accepted, int32_t* bonus_token);

/*
 * Draft candidates of the last forward (verify or draft): for each of its n
 * rows, the K tokens of highest logit (decreasing logit, lower id on ties;
 * id -1 and probability 0 past the row's finite entries) and their softmax
 * probabilities over the whole vocabulary, p = exp(l - max) / sum exp(l_v -
 * max) in fp32 (Alg. 1: the K candidates y[i, :] of a drafted position;
 * Sec. 4.2 "Token-Level Information": the normalised probability of a
 * drafted token).  n must equal the last forward's row count; ids and probs
 * are host arrays of n*K (row-major); K in [1, 16].  Only n*K pairs cross
 * PCIe, not the n x vocab logits.  NaN logits give CAS_ERR_DEVICE.
 * Synchronous.
 */
cas_status cas_topk(cas_ctx* ctx, int32_t n, int32_t K, int32_t* ids, float* probs);

/*
 * Commit an accepted root path of the verified round: accepted[j] must be the
 * root for j = 0 and a child of accepted[j-1] otherwise.  Node accepted[j]
 * moves from slot Lc+accepted[j] to slot Lc+j in every layer; then
 * Lc += n_accepted and the round closes.  Asynchronous.
 */
cas_status cas_kv_compact(cas_ctx* ctx, const int32_t* accepted, int32_t n_accepted);

/* Tree metadata on the host, as the library computes it on the device:
 * depth[i] and the ancestor-or-self bitmask anc[2*i], anc[2*i+1] (bit j of
 * the 128-bit mask = node j).  Validates the parent list (n <= 128).  Either
 * output may be NULL. */
cas_status cas_tree_info(const int32_t* tree_parent, int32_t n, int32_t* depth, uint64_t* anc);

/* Capture the forward's launches in HIP graphs keyed on (n, node_offset,
 * skip mask, act_quant, attention split count) and replay them (1, default),
 * or launch kernel by kernel (0). */
cas_status cas_set_graphs(cas_ctx* ctx, int32_t enable);

/* Draft calls of one row (a skip mask, quantised activations or an attention
 * window) with bf16 or int8 weights run their wide GEMMs (QKV, gate/up, LM
 * head) as GEMV-style tiles (1: VALU dot products per lane, summed across
 * the k-group lanes) or as the MFMA tiles every other call uses (0,
 * default).  The GEMV tiles stream a little faster (7B 16-layer one-row
 * draft 1.50 -> 1.48 ms; 8B no change) but sum in another order than the
 * MFMA tiles: with bf16 weights a one-row draft's logits then differ from
 * the verify's by rounding even where the draft computes the same function
 * (a skipped layer that contributes nothing), and a near-tie can pick
 * another token.  With 0 such a draft gives the verify's bits.  Takes effect
 * at the next forward. */
cas_status cas_set_gemv(cas_ctx* ctx, int32_t enable);

/* Per-kernel timing: when enabled, the forward launches kernel by kernel and
 * brackets every launch with HIP events on the context's stream.
 * cas_profile_read sums, for each kernel class (cas_kclass), the elapsed
 * milliseconds and the launch count since the last reset (synchronises). */
typedef enum {
    CAS_K_EMBED = 0, CAS_K_RMSNORM = 1, CAS_K_GEMM_QKV = 2, CAS_K_ATTN = 3,
    CAS_K_GEMM_O = 4, CAS_K_GEMM_GATEUP = 5, CAS_K_GEMM_DOWN = 6,
    CAS_K_GEMM_HEAD = 7, CAS_K_QUANT = 8, CAS_K_ACCEPT = 9, CAS_K_COMPACT = 10,
    CAS_K_TOPK = 11, CAS_K_COUNT = 12
} cas_kclass;
cas_status cas_profile(cas_ctx* ctx, int32_t enable);
cas_status cas_profile_read(cas_ctx* ctx, double* ms, int32_t* launches, int32_t reset);

/* Synchronise the context's stream.  In a CAS_DEBUG build it also reports a
 * failed device check (below) as CAS_ERR_DEVICE. */
cas_status cas_sync(cas_ctx* ctx);

/*
 * Device checks.  The library is also built with -DCAS_DEBUG
 * (libcas_debug.so, same entry points).  Its kernels check every bound that
 * rests on values they read from device memory rather than on their launch
 * shape: the tree size and each row's place in the round, token ids, parent
 * order in the tree walks (parent < child, root -1), the slot capacity of the
 * round (Lc + n <= max_ctx), RoPE positions, KV write slots, the attention's
 * slot range and the compaction path.  The host validates all of these before
 * it copies them, so in a correct program no check fails.  A failed check
 * records its code in a per-context word and skips the access it guards: the
 * kernel ends normally, and that call's results are invalid.  The
 * synchronising calls (cas_accept_tree, cas_topk, cas_forward with
 * logits_host, cas_sync) then return CAS_ERR_DEVICE with the check's name and
 * clear the word; the work of the call has been done.
 *   cas_debug_build        1 in a CAS_DEBUG build, else 0
 *   cas_debug_check        synchronises; *code = the recorded check code
 *                          (0: none; 1 tree size, 2 token, 3 parent,
 *                          4 slot capacity, 5 RoPE position, 6 KV write slot,
 *                          7 attention slots, 8 compaction path,
 *                          9 acceptance parent) and clears it.  Always 0 in
 *                          a release build
 *   cas_debug_limit_slots  makes the checks allow only slots < cap in later
 *                          calls (0: max_ctx again), so that a test can make
 *                          the slot checks fail while every access stays
 *                          inside the real cache.  CAS_ERR_UNSUPPORTED in a
 *                          release build; cap outside [0, max_ctx]:
 *                          CAS_ERR_ARG
 */
int32_t cas_debug_build(void);
cas_status cas_debug_check(cas_ctx* ctx, int32_t* code);
cas_status cas_debug_limit_slots(cas_ctx* ctx, int32_t cap);

#ifdef __cplusplus
}
#endif
#endif /* CAS_H */
