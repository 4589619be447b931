/*
 * cas_runtime_check: drives every entry point of the C ABI (cas.h,
 * cas_ops.h) through its documented behaviour, valid calls and rejected
 * ones alike.  It is built with the runtime's host code under
 * AddressSanitizer and UndefinedBehaviorSanitizer (the kernels are linked in
 * unchanged), so any invalid host memory access or undefined operation in
 * argument validation, tree bookkeeping, staging, the graph cache or
 * profiling aborts the run.
 *
 * Part 1 needs no GPU: tree metadata, configuration checks, the argument
 * checks of the kernel-level entry points and their workspace sizes.
 * Part 2 (skipped when no device can be opened, or with --host-only) runs
 * small fp32 and bf16 grouped-query decoders with random weights through
 * loads, int8 and int4 copies, prefill, many rounds of drafts (skip masks,
 * int8 and int4 activations, windows, appended levels), verify, top-K,
 * acceptance and compaction with varying tree sizes (more shapes than the
 * graph cache holds), profiling, direct launches, KV load and read, and the
 * error paths that must leave the context unchanged.  It checks statuses and
 * state (committed length, round rules), not numerics.
 * Exit status 0: every check passed.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "cas.h"
#include "cas_ops.h"

static int failures = 0;
#define CHECK(c)                                                                \
    do {                                                                        \
        if (!(c)) {                                                             \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);     \
            failures++;                                                         \
        }                                                                       \
    } while (0)
#define OK(ctx, call)                                                                            \
    do {                                                                                         \
        cas_status _s = (call);                                                                  \
        if (_s != CAS_OK) {                                                                      \
            fprintf(stderr, "line %d: %s -> %d (%s)\n", __LINE__, #call, (int)_s,                \
                    cas_last_error(ctx));                                                        \
            failures++;                                                                          \
        }                                                                                        \
    } while (0)

static uint64_t rng = 0x2545f4914f6cdd1dull;
static uint32_t urand(void) {  /* xorshift64* */
    rng ^= rng >> 12;
    rng ^= rng << 25;
    rng ^= rng >> 27;
    return (uint32_t)((rng * 0x2545f4914f6cdd1dull) >> 32);
}
static float frand(float scale) { return ((float)(urand() & 0xffffff) / 16777216.0f - 0.5f) * 2.0f * scale; }

static uint16_t to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7fff + ((u >> 16) & 1)) >> 16);
}

/* ------------------------------------------------------------ part 1: host only */

static void host_checks(void) {
    /* tree metadata */
    int32_t par[130], depth[130];
    uint64_t anc[260];
    par[0] = -1;
    for (int i = 1; i < 130; i++) par[i] = (i - 1) / 2;
    CHECK(cas_tree_info(par, 128, depth, anc) == CAS_OK);
    CHECK(depth[0] == 0 && depth[127] == 7);
    CHECK((anc[2 * 127 + 1] >> 63) == 1 && (anc[2 * 127] & 1) == 1);
    CHECK(cas_tree_info(par, 129, depth, anc) != CAS_OK);
    CHECK(cas_tree_info(par, 0, depth, anc) != CAS_OK);
    CHECK(cas_tree_info(NULL, 4, depth, anc) != CAS_OK);
    CHECK(cas_tree_info(par, 4, NULL, anc) == CAS_OK);  /* either output may be NULL */
    par[3] = 3;  /* self-parent */
    CHECK(cas_tree_info(par, 8, depth, anc) == CAS_ERR_TREE);
    par[3] = 5;  /* forward reference */
    CHECK(cas_tree_info(par, 8, depth, anc) == CAS_ERR_TREE);
    par[3] = -1; /* second root */
    CHECK(cas_tree_info(par, 8, depth, anc) == CAS_ERR_TREE);
    par[3] = 1;
    par[0] = 0;  /* root with a parent */
    CHECK(cas_tree_info(par, 8, depth, anc) == CAS_ERR_TREE);
    par[0] = -1;

    /* configuration checks (all before any device call) */
    cas_ctx* ctx = (cas_ctx*)&rng;
    cas_config ok = {2, 256, 4, 2, 64, 512, 512, 10000.f, 1e-6f, CAS_BF16, 512, 64};
    CHECK(cas_create(NULL, 0, NULL, &ctx) == CAS_ERR_ARG && ctx == NULL);
    CHECK(cas_create(&ok, 0, NULL, NULL) == CAS_ERR_ARG);
    cas_config bad = ok;
    bad.head_dim = 96;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_UNSUPPORTED && ctx == NULL);
    CHECK(strlen(cas_create_error()) > 0);
    bad = ok; bad.n_kv_heads = 3;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_ARG);
    bad = ok; bad.d_model = 250;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_UNSUPPORTED);
    bad = ok; bad.max_tree = 129;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_UNSUPPORTED);
    bad = ok; bad.max_ctx = 32;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_ARG);
    bad = ok; bad.max_ctx = 20000;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_UNSUPPORTED);
    bad = ok; bad.dtype = 7;
    CHECK(cas_create(&bad, 0, NULL, &ctx) != CAS_OK);
    bad = ok; bad.rms_eps = 0.f;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_ARG);
    bad = ok; bad.n_layers = 0;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_ARG);
    bad = ok; bad.dtype = CAS_F32; bad.max_ctx = 4000;
    CHECK(cas_create(&bad, 0, NULL, &ctx) == CAS_ERR_UNSUPPORTED);

    /* entry points on a NULL context */
    int32_t n = 0;
    CHECK(cas_prefill(NULL, par, 1) == CAS_ERR_ARG);
    CHECK(cas_committed_len(NULL, &n) == CAS_ERR_ARG);
    CHECK(cas_sync(NULL) == CAS_ERR_ARG);
    CHECK(cas_debug_check(NULL, &n) == CAS_ERR_ARG);
    CHECK(cas_set_gemv(NULL, 1) == CAS_ERR_ARG);
    CHECK(cas_last_error(NULL) != NULL);
    cas_destroy(NULL);
    CHECK(cas_debug_build() == 0 || cas_debug_build() == 1);

    /* kernel-level entry points: argument checks and workspace sizes */
    CHECK(cas_op_gemm(0, NULL, NULL, 64, 64, 1, NULL, NULL, 0, NULL, 64, NULL, 0, NULL) != CAS_OK);
    CHECK(cas_op_gemm_work_bytes(1, 4096, 4096, 32) > 0);
    CHECK(cas_op_quant_rows(1, NULL, 1, 64, NULL, NULL, NULL) != CAS_OK);
    CHECK(cas_op_quant_rows_q(1, NULL, 1, 64, 5, NULL, NULL, NULL) != CAS_OK);
    CHECK(cas_op_quant_weight(1, NULL, 16, 64, NULL, NULL, NULL, 0, NULL) != CAS_OK);
    CHECK(cas_op_quant_weight_i4(1, NULL, 16, 64, NULL, NULL, NULL, 0, NULL) != CAS_OK);
    CHECK(cas_op_attention(NULL, NULL, NULL, 256, 10, 4, 4, 4, 2, 128, NULL, NULL, NULL, 0, NULL) == CAS_ERR_ARG);
    CHECK(cas_op_attention_work_bytes(1000, 32, 32, 32, 128, 32, 1056) > 0);
    CHECK(cas_op_attention_noalloc(NULL, NULL, NULL, 256, 10, 4, 4, 4, 2, 128, NULL, NULL, NULL) == CAS_ERR_ARG);
    CHECK(cas_op_attention_noalloc_max_bytes() > 0);
    CHECK(cas_op_rmsnorm(1, NULL, NULL, 1, 64, 1e-6f, NULL, 0, 0, NULL, NULL, NULL, NULL, 0, NULL) != CAS_OK);
    CHECK(cas_op_rmsnorm_work_bytes(1, 4, 4096, 5) == 0);
    CHECK(cas_op_attn_merge(NULL, NULL, 2, 4, 4, 128, 0, NULL, NULL, NULL, NULL, 0, NULL) == CAS_ERR_ARG);
    CHECK(cas_op_attn_merge_work_bytes(4, 32, 128, 9) == 0);
    CHECK(cas_op_gemm_qx(2, NULL, NULL, NULL, 4096, 4096, 1, 127, NULL, NULL, 0, NULL) != CAS_OK);
    CHECK(cas_op_copy(NULL, NULL, 16, NULL) != CAS_OK);
}

/* ------------------------------------------------------------ part 2: on a device */

typedef struct {
    int bf16, L, d, H, Hkv, hd, ffn, V, max_ctx, max_tree;
} shape_t;

static size_t tensor_elems(const shape_t* s, int kind) {
    const size_t q = (size_t)s->H * s->hd, kv = (size_t)s->Hkv * s->hd;
    switch (kind) {
    case CAS_T_EMBED: case CAS_T_LM_HEAD: return (size_t)s->V * s->d;
    case CAS_T_FINAL_NORM: case CAS_T_ATTN_NORM: case CAS_T_FFN_NORM: return (size_t)s->d;
    case CAS_T_WQ: return q * s->d;
    case CAS_T_WK: case CAS_T_WV: return kv * s->d;
    case CAS_T_WO: return (size_t)s->d * q;
    case CAS_T_W_GATE: case CAS_T_W_UP: return (size_t)s->ffn * s->d;
    default: return (size_t)s->d * s->ffn;
    }
}

static void load_all(cas_ctx* c, const shape_t* s) {
    for (int kind = CAS_T_EMBED; kind <= CAS_T_W_DOWN; kind++) {
        const int global = kind <= CAS_T_FINAL_NORM;
        const int norm = kind == CAS_T_FINAL_NORM || kind == CAS_T_ATTN_NORM || kind == CAS_T_FFN_NORM;
        const size_t n = tensor_elems(s, kind);
        const size_t es = norm || !s->bf16 ? 4 : 2;
        void* buf = malloc(n * es);
        for (size_t i = 0; i < n; i++) {
            const float f = norm ? 1.0f + frand(0.1f) : frand(kind == CAS_T_EMBED ? 1.0f : 0.05f);
            if (es == 2) ((uint16_t*)buf)[i] = to_bf16(f);
            else ((float*)buf)[i] = f;
        }
        for (int l = 0; l < (global ? 1 : s->L); l++) OK(c, cas_load_tensor(c, kind, l, buf, n * es));
        if (kind == CAS_T_WQ) {
            CHECK(cas_load_tensor(c, kind, 0, buf, n * es - 2) == CAS_ERR_ARG);
            CHECK(cas_load_tensor(c, kind, s->L, buf, n * es) == CAS_ERR_ARG);
            CHECK(cas_load_tensor(c, 12, 0, buf, n * es) == CAS_ERR_ARG);
            CHECK(cas_load_tensor(c, kind, 0, NULL, n * es) == CAS_ERR_ARG);
        }
        free(buf);
    }
}

static int32_t committed(cas_ctx* c) {
    int32_t n = -1;
    OK(c, cas_committed_len(c, &n));
    return n;
}

/* a random tree of n nodes appended after `have` nodes of the round */
static void random_parents(int32_t* par, int have, int n) {
    for (int i = 0; i < n; i++) {
        const int id = have + i;
        par[i] = id == 0 ? -1 : (int32_t)(urand() % (uint32_t)id);
    }
}

static void error_paths(cas_ctx* c, const shape_t* s) {
    int32_t tok[4] = {1, 2, 3, 4}, par[4] = {-1, 0, 0, 1}, acc[4], na = 0, bonus = 0;
    const int32_t Lc = committed(c);
    /* every rejected call leaves the committed length and the round alone */
    CHECK(cas_forward(c, tok, par, 0, 0, NULL, 0, NULL) == CAS_ERR_ARG);
    CHECK(cas_forward(c, NULL, par, 4, 0, NULL, 0, NULL) == CAS_ERR_ARG);
    CHECK(cas_forward(c, tok, par, 4, 3, NULL, 0, NULL) == CAS_ERR_TREE);
    CHECK(cas_forward(c, tok, par, 4, -1, NULL, 0, NULL) == CAS_ERR_ARG);
    CHECK(cas_forward(c, tok, par, 4, 0, NULL, 3, NULL) == CAS_ERR_ARG);
    tok[2] = s->V;
    CHECK(cas_forward(c, tok, par, 4, 0, NULL, 0, NULL) == CAS_ERR_ARG);
    tok[2] = -1;
    CHECK(cas_forward(c, tok, par, 4, 0, NULL, 0, NULL) == CAS_ERR_ARG);
    tok[2] = 3;
    par[2] = 2;
    CHECK(cas_forward(c, tok, par, 4, 0, NULL, 0, NULL) == CAS_ERR_TREE);
    par[2] = 0;
    uint8_t* skip = (uint8_t*)calloc((size_t)s->L, 1);
    skip[0] = 2;
    CHECK(cas_forward(c, tok, par, 4, 0, skip, 0, NULL) == CAS_ERR_ARG);
    free(skip);
    cas_draft_opts o = {NULL, 0, -1, 4};
    CHECK(cas_forward_draft(c, tok, par, 4, 0, &o, NULL) == CAS_ERR_ARG);
    int32_t* big_tok = (int32_t*)calloc((size_t)s->max_tree + 1, 4);
    int32_t* big_par = (int32_t*)calloc((size_t)s->max_tree + 1, 4);
    random_parents(big_par, 0, s->max_tree + 1);
    CHECK(cas_forward(c, big_tok, big_par, s->max_tree + 1, 0, NULL, 0, NULL) == CAS_ERR_CAPACITY);
    free(big_tok);
    free(big_par);
    CHECK(cas_set_committed(c, s->max_ctx + 1) == CAS_ERR_CAPACITY);
    CHECK(committed(c) == Lc);
    /* acceptance and compaction need a verify call covering the round */
    OK(c, cas_set_committed(c, Lc));
    CHECK(cas_accept_tree(c, 1, acc, &na, &bonus) == CAS_ERR_STATE);
    CHECK(cas_kv_compact(c, acc, 1) == CAS_ERR_STATE);
    OK(c, cas_forward(c, tok, par, 1, 0, NULL, 0, NULL));
    OK(c, cas_forward(c, tok + 1, par + 1, 3, 1, NULL, 0, NULL));  /* an appended call: not a verify */
    CHECK(cas_accept_tree(c, 1, acc, &na, &bonus) == CAS_ERR_STATE);
    OK(c, cas_forward(c, tok, par, 4, 0, NULL, 0, NULL));
    CHECK(cas_accept_tree(c, 0, acc, &na, &bonus) == CAS_ERR_UNSUPPORTED);
    CHECK(cas_accept_tree(c, 1, NULL, &na, &bonus) == CAS_ERR_ARG);
    int32_t badpath[2] = {0, 3};  /* node 3 is a child of node 1 */
    CHECK(cas_kv_compact(c, badpath, 2) == CAS_ERR_TREE);
    badpath[0] = 1;
    CHECK(cas_kv_compact(c, badpath, 1) == CAS_ERR_TREE);
    CHECK(cas_kv_compact(c, acc, 0) == CAS_ERR_ARG);
    CHECK(cas_kv_compact(c, NULL, 1) == CAS_ERR_ARG);
    int32_t ids[64];
    float probs[64];
    CHECK(cas_topk(c, 3, 2, ids, probs) == CAS_ERR_ARG);
    CHECK(cas_topk(c, 4, 0, ids, probs) == CAS_ERR_ARG);
    CHECK(cas_topk(c, 4, 17, ids, probs) == CAS_ERR_ARG);
    CHECK(cas_topk(c, 4, 2, NULL, probs) == CAS_ERR_ARG);
    CHECK(cas_logits_device(c, NULL, &na) == CAS_ERR_ARG);
    CHECK(committed(c) == Lc);
    OK(c, cas_set_committed(c, Lc));
    /* capacity: a round that would pass max_ctx */
    OK(c, cas_set_committed(c, s->max_ctx - 2));
    CHECK(cas_forward(c, tok, par, 4, 0, NULL, 0, NULL) == CAS_ERR_CAPACITY);
    CHECK(cas_prefill(c, tok, 3) == CAS_ERR_CAPACITY);
    OK(c, cas_set_committed(c, Lc));
    if (cas_debug_build()) {
        CHECK(cas_debug_limit_slots(c, s->max_ctx + 1) == CAS_ERR_ARG);
    } else {
        CHECK(cas_debug_limit_slots(c, 8) == CAS_ERR_UNSUPPORTED);
    }
}

static void run_model(const shape_t* s) {
    cas_config cfg = {s->L, s->d, s->H, s->Hkv, s->hd, s->ffn, s->V, 10000.f, 1e-6f,
                      s->bf16 ? CAS_BF16 : CAS_F32, s->max_ctx, s->max_tree};
    cas_ctx* c = NULL;
    cas_status st = cas_create(&cfg, 0, NULL, &c);
    CHECK(st == CAS_OK && c != NULL);
    if (st != CAS_OK) {
        fprintf(stderr, "cas_create: %s\n", cas_create_error());
        return;
    }
    int32_t tok[128], par[128], acc[128], ids[128 * 4], na = 0, bonus = 0, code = -1;
    float probs[128 * 4];
    /* not loaded yet */
    tok[0] = 1;
    par[0] = -1;
    CHECK(cas_forward(c, tok, par, 1, 0, NULL, 0, NULL) == CAS_ERR_STATE);
    CHECK(cas_forward(c, tok, par, 1, 0, NULL, 1, NULL) == CAS_ERR_STATE);
    load_all(c, s);
    CHECK(cas_forward(c, tok, par, 1, 0, NULL, 1, NULL) == CAS_ERR_STATE);  /* no int8 copy yet */
    OK(c, cas_build_int8(c));
    OK(c, cas_build_int4(c));

    /* prefill, then KV read back and reload */
    int32_t* prompt = (int32_t*)malloc(sizeof(int32_t) * 300);
    for (int i = 0; i < 300; i++) prompt[i] = (int32_t)(urand() % (uint32_t)s->V);
    OK(c, cas_prefill(c, prompt, 150));
    CHECK(committed(c) == 150);
    const size_t es = s->bf16 ? 2 : 4, kvb = (size_t)s->Hkv * 150 * s->hd * es;
    void *k = malloc(kvb), *v = malloc(kvb), *k2 = malloc(kvb), *v2 = malloc(kvb);
    OK(c, cas_kv_read(c, 1, k, v, 150));
    OK(c, cas_kv_load(c, 1, k, v, 150));
    OK(c, cas_kv_read(c, 1, k2, v2, 150));
    CHECK(memcmp(k, k2, kvb) == 0 && memcmp(v, v2, kvb) == 0);
    CHECK(cas_kv_read(c, s->L, k, v, 10) != CAS_OK);
    CHECK(cas_kv_read(c, 0, k, v, s->max_ctx + 1) != CAS_OK);
    free(k); free(v); free(k2); free(v2);

    /* rounds: drafts of the root and appended levels, then a verify of the
     * whole tree, top-K, acceptance and compaction; the tree size cycles
     * through more shapes than the graph cache keeps */
    uint8_t* skip = (uint8_t*)calloc((size_t)s->L, 1);
    for (int l = 1; l < s->L; l += 2) skip[l] = 1;
    const int rounds = 90;
    for (int r = 0; r < rounds; r++) {
        if (committed(c) + s->max_tree + 2 > s->max_ctx) OK(c, cas_set_committed(c, 150));
        const int Lc = committed(c);
        const int n = 1 + (r * 7) % s->max_tree;
        random_parents(par, 0, n);
        for (int i = 0; i < n; i++) tok[i] = (int32_t)(urand() % (uint32_t)s->V);
        /* draft of the root (layer skip with int8 / int4 / a window on later rounds) */
        cas_draft_opts o = {skip, r % 3, r % 5 == 0 ? 2 : 0, r % 5 == 0 ? 32 : 0};
        OK(c, cas_forward_draft(c, tok, par, 1, 0, &o, NULL));
        OK(c, cas_topk(c, 1, 4, ids, probs));
        if (n > 1) {
            /* the rest of the tree appended in two draft calls */
            const int m = 1 + (n - 1) / 2;
            OK(c, cas_forward(c, tok + 1, par + 1, m - 1 > 0 ? m - 1 : 1, 1, skip, r % 3, NULL));
            const int have = 1 + (m - 1 > 0 ? m - 1 : 1);
            if (have < n) {
                OK(c, cas_forward(c, tok + have, par + have, n - have, have, NULL, 0, NULL));
                OK(c, cas_topk(c, n - have, 4, ids, probs));
            }
        }
        /* verify, every other round copying the logits out */
        float* lg = (r & 1) ? (float*)malloc(sizeof(float) * (size_t)n * s->V) : NULL;
        OK(c, cas_forward(c, tok, par, n, 0, NULL, 0, lg));
        free(lg);
        const float* dl = NULL;
        int32_t rows = 0;
        OK(c, cas_logits_device(c, &dl, &rows));
        CHECK(dl != NULL && rows == n);
        OK(c, cas_topk(c, n, 3, ids, probs));
        for (int i = 0; i < n * 3; i++) CHECK(ids[i] >= -1 && ids[i] < s->V && probs[i] >= 0.f && probs[i] <= 1.f);
        OK(c, cas_accept_tree(c, 1, acc, &na, &bonus));
        CHECK(na >= 1 && na <= n && acc[0] == 0 && bonus >= 0 && bonus < s->V);
        for (int j = 1; j < na; j++) CHECK(par[acc[j]] == acc[j - 1]);
        /* commit a path: the accepted one, or on some rounds the deepest
         * path to the last node (a non-identity move) */
        if (r % 4 == 3) {
            int path[128], len = 0;
            for (int x = n - 1; x >= 0; x = par[x]) path[len++] = x;
            for (int j = 0; j < len; j++) acc[j] = path[len - 1 - j];
            na = len;
        }
        OK(c, cas_kv_compact(c, acc, na));
        CHECK(committed(c) == Lc + na);
        if (r == 30) {
            /* launch kernel by kernel with per-kernel timing for a while */
            double ms[CAS_K_COUNT];
            int32_t launches[CAS_K_COUNT];
            OK(c, cas_profile(c, 1));
            OK(c, cas_profile_read(c, ms, launches, 1));
        }
        if (r == 45) {
            double ms[CAS_K_COUNT];
            int32_t launches[CAS_K_COUNT];
            OK(c, cas_profile_read(c, ms, launches, 1));
            CHECK(launches[CAS_K_EMBED] > 0 && ms[CAS_K_GEMM_QKV] > 0.0);
            OK(c, cas_profile(c, 0));
            OK(c, cas_set_graphs(c, 0));
        }
        if (r == 60) OK(c, cas_set_graphs(c, 1));
        if (r == 20) OK(c, cas_set_gemv(c, 1));
        if (r == 75) OK(c, cas_set_gemv(c, 0));
    }
    free(skip);
    error_paths(c, s);
    OK(c, cas_sync(c));
    OK(c, cas_debug_check(c, &code));
    CHECK(code == 0);
    free(prompt);
    cas_destroy(c);
}

int main(int argc, char** argv) {
    int host_only = argc > 1 && strcmp(argv[1], "--host-only") == 0;
    host_checks();
    int ran_device = 0;
    if (!host_only) {
        /* a device is there if a small context can be created */
        cas_config probe = {1, 64, 1, 1, 64, 64, 64, 10000.f, 1e-6f, CAS_F32, 128, 8};
        cas_ctx* c = NULL;
        if (cas_create(&probe, 0, NULL, &c) == CAS_OK) {
            cas_destroy(c);
            /* bf16, layers, d_model, heads, kv heads, head_dim, ffn, vocab, max_ctx, max_tree */
            const shape_t tiny = {0, 2, 128, 2, 2, 64, 256, 256, 512, 64};
            run_model(&tiny);
            const shape_t gqa = {1, 3, 256, 4, 2, 64, 512, 512, 1024, 128};
            run_model(&gqa);
            ran_device = 1;
        } else {
            printf("no device: %s\n", cas_create_error());
        }
    }
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("runtime check: all checks passed (%s)\n", ran_device ? "host and device" : "host only");
    return 0;
}
