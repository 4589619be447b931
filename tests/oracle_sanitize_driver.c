/*
 * Driver for a sanitized CPU build of the oracle (tests/test_oracle_sanitized.py
 * compiles it together with oracle/cas_oracle.c under AddressSanitizer and
 * UndefinedBehaviorSanitizer, without OpenMP).  It exercises every entry
 * point of the oracle on small decoders: fp32 and bf16 weights, grouped-query
 * attention, tree rounds built in one call and by appended calls, layer skip,
 * int8 and int4 activations, the sink + window attention, the row subset
 * (`need`), compaction, KV set/get, and the argument checks.  It exits 0 when
 * every call behaved as documented; the sanitizers abort on any invalid
 * memory access or undefined operation.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct om_model om_model;
om_model *om_create(int L, int d, int H, int Hkv, int hd, int ffn, int V, double theta, double eps, int bf16,
                    int max_ctx);
void om_destroy(om_model *m);
void om_set_global(om_model *m, const void *embed, const void *lm_head, const float *final_norm);
void om_set_layer(om_model *m, int l, const void *const *w, const float *attn_norm, const float *ffn_norm);
void om_set_layer_i8(om_model *m, int l, const int8_t *const *q, const float *const *s);
void om_set_layer_i4(om_model *m, int l, const int8_t *const *q, const float *const *s);
int om_set_kv(om_model *m, int l, int n, const float *k, const float *v);
int om_get_kv(om_model *m, int l, int kvh, int slot, double *k, double *v);
int om_set_committed(om_model *m, int Lc);
int om_committed(const om_model *m);
int om_set_window(om_model *m, int sink, int window);
int om_forward(om_model *m, const int32_t *tokens, const int32_t *parents, int node_offset, int n,
               const uint8_t *skip, int act_quant, const uint8_t *need, double *logits);
int om_compact(om_model *m, const int32_t *accepted, int n_acc);
void om_quant_weight_q(const void *w, int bf16, int out, int in, int qmax, int8_t *q, float *scale);
void om_quant_row_q(const float *x, int n, int qmax, int8_t *q, float *scale);
int om_dot_i8(const int8_t *a, const int8_t *b, int n, int32_t *out);
double om_round_bf16(double x);

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static double urand(void) {   /* splitmix64 -> [0, 1) */
    uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    z ^= z >> 31;
    return (double)(z >> 11) * (1.0 / 9007199254740992.0);
}
static float nrand(void) { return (float)((urand() + urand() + urand() - 1.5) * 0.04); }

static int failures = 0;
#define CHECK(c)                                                         \
    do {                                                                 \
        if (!(c)) {                                                      \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            failures++;                                                  \
        }                                                                \
    } while (0)

static void *weights(int rows, int cols, int bf16) {
    size_t n = (size_t)rows * cols;
    if (bf16) {
        uint16_t *w = (uint16_t *)malloc(n * 2);
        for (size_t i = 0; i < n; i++) {
            float f = nrand();
            uint32_t u;
            memcpy(&u, &f, 4);
            w[i] = (uint16_t)(u >> 16);
        }
        return w;
    }
    float *w = (float *)malloc(n * 4);
    for (size_t i = 0; i < n; i++) w[i] = nrand();
    return w;
}

static int all_finite(const double *x, size_t n) {
    for (size_t i = 0; i < n; i++)
        if (!isfinite(x[i])) return 0;
    return 1;
}

static void run_model(int bf16, int H, int Hkv) {
    const int L = 3, d = 64, hd = 16, ffn = 96, V = 50, ctx = 48;
    const int dims[7][2] = {{H * hd, d}, {Hkv * hd, d}, {Hkv * hd, d}, {d, H * hd}, {ffn, d}, {ffn, d}, {d, ffn}};
    om_model *m = om_create(L, d, H, Hkv, hd, ffn, V, 1e4, 1e-6, bf16, ctx);
    CHECK(m != NULL);
    void *embed = weights(V, d, bf16), *head = weights(V, d, bf16);
    float *ones = (float *)malloc(sizeof(float) * ffn);
    for (int i = 0; i < ffn; i++) ones[i] = 1.0f;
    om_set_global(m, embed, head, ones);
    void *w[3][7];
    int8_t *q8[3][7], *q4[3][7];
    float *s8[3][7], *s4[3][7];
    for (int l = 0; l < L; l++) {
        for (int i = 0; i < 7; i++) {
            w[l][i] = weights(dims[i][0], dims[i][1], bf16);
            size_t n = (size_t)dims[i][0] * dims[i][1];
            q8[l][i] = (int8_t *)malloc(n);
            q4[l][i] = (int8_t *)malloc(n);
            s8[l][i] = (float *)malloc(sizeof(float) * dims[i][0]);
            s4[l][i] = (float *)malloc(sizeof(float) * dims[i][0]);
            om_quant_weight_q(w[l][i], bf16, dims[i][0], dims[i][1], 127, q8[l][i], s8[l][i]);
            om_quant_weight_q(w[l][i], bf16, dims[i][0], dims[i][1], 7, q4[l][i], s4[l][i]);
        }
        om_set_layer(m, l, (const void *const *)w[l], ones, ones);
        om_set_layer_i8(m, l, (const int8_t *const *)q8[l], (const float *const *)s8[l]);
        om_set_layer_i4(m, l, (const int8_t *const *)q4[l], (const float *const *)s4[l]);
    }
    /* a committed cache of 10 slots */
    const int n0 = 10;
    float *k = (float *)malloc(sizeof(float) * Hkv * n0 * hd), *v = (float *)malloc(sizeof(float) * Hkv * n0 * hd);
    for (int i = 0; i < Hkv * n0 * hd; i++) { k[i] = nrand() * 30; v[i] = nrand() * 30; }
    for (int l = 0; l < L; l++) CHECK(om_set_kv(m, l, n0, k, v) == 0);
    CHECK(om_set_kv(m, L, n0, k, v) != 0);
    CHECK(om_set_committed(m, n0) == 0);
    CHECK(om_committed(m) == n0);
    /* a 7-node tree in one verify call */
    const int32_t tok[7] = {1, 2, 3, 4, 5, 6, 7}, par[7] = {-1, 0, 0, 1, 1, 2, 3};
    double *lg = (double *)calloc((size_t)7 * V, sizeof(double));
    CHECK(om_forward(m, tok, par, 0, 7, NULL, 0, NULL, lg) == 0);
    CHECK(all_finite(lg, (size_t)7 * V));
    const int32_t acc[3] = {0, 1, 3};
    CHECK(om_compact(m, acc, 3) == 0);
    CHECK(om_committed(m) == n0 + 3);
    double kk[16], vv[16];
    CHECK(om_get_kv(m, 1, Hkv - 1, n0 + 2, kk, vv) == 0);
    CHECK(om_get_kv(m, 1, Hkv, 0, kk, vv) != 0);
    /* drafts: the root, then appended levels, with skip, int8, int4, window, need */
    const uint8_t skip[3] = {0, 1, 0};
    const uint8_t need[3] = {0, 0, 1};
    for (int aq = 0; aq <= 2; aq++) {
        CHECK(om_forward(m, tok, par, 0, 1, skip, aq, NULL, lg) == 0);
        CHECK(om_forward(m, tok + 1, par + 1, 1, 2, skip, aq, NULL, lg) == 0);
        CHECK(om_forward(m, tok + 3, par + 3, 3, 3, NULL, aq, need, lg) == 0);
        CHECK(all_finite(lg + 2 * V, V));
    }
    CHECK(om_set_window(m, 2, 4) == 0);
    CHECK(om_forward(m, tok, par, 0, 7, skip, 1, NULL, lg) == 0);
    CHECK(om_set_window(m, 0, 0) == 0);
    CHECK(om_set_window(m, -1, 2) != 0);
    /* compaction needs a verified round: the last call was a draft */
    CHECK(om_compact(m, acc, 3) != 0);
    /* invalid arguments leave the state unchanged */
    const int32_t badpar[2] = {-1, 5};
    CHECK(om_forward(m, tok, badpar, 0, 2, NULL, 0, NULL, lg) != 0);
    const int32_t badtok[1] = {V};
    CHECK(om_forward(m, badtok, par, 0, 1, NULL, 0, NULL, lg) != 0);
    CHECK(om_forward(m, tok, par, 5, 1, NULL, 0, NULL, lg) != 0);
    CHECK(om_forward(m, tok, par, 0, ctx, NULL, 0, NULL, lg) != 0);
    CHECK(om_forward(m, tok, par, 0, 1, NULL, 3, NULL, lg) != 0);
    CHECK(om_set_committed(m, ctx + 1) != 0);
    /* a full round at the end of the cache */
    CHECK(om_set_committed(m, ctx - 7) == 0);
    CHECK(om_forward(m, tok, par, 0, 7, NULL, 2, NULL, lg) == 0);
    CHECK(om_forward(m, tok, par, 0, 7, NULL, 0, NULL, lg) == 0);
    CHECK(om_compact(m, acc, 3) == 0);
    CHECK(om_committed(m) == ctx - 4);
    free(lg); free(k); free(v);
    for (int l = 0; l < L; l++)
        for (int i = 0; i < 7; i++) { free(w[l][i]); free(q8[l][i]); free(q4[l][i]); free(s8[l][i]); free(s4[l][i]); }
    free(embed); free(head); free(ones);
    om_destroy(m);
}

int main(void) {
    run_model(0, 4, 4);
    run_model(1, 4, 2);
    run_model(1, 2, 1);
    /* op-level helpers */
    float x[33];
    int8_t q[33];
    float s;
    for (int i = 0; i < 33; i++) x[i] = (float)(i - 16) * 0.25f;
    om_quant_row_q(x, 33, 127, q, &s);
    CHECK(q[0] == -127 && q[32] == 127);
    om_quant_row_q(x, 33, 7, q, &s);
    CHECK(s == 4.0f / 7.0f && q[32] == 7);
    memset(x, 0, sizeof x);
    om_quant_row_q(x, 33, 127, q, &s);
    CHECK(s == 0.0f && q[5] == 0);
    int8_t a[4] = {127, -127, 127, -127}, b[4] = {127, -127, 127, -127};
    int32_t r;
    CHECK(om_dot_i8(a, b, 4, &r) == 0 && r == 4 * 127 * 127);
    CHECK(om_round_bf16(1.0 + 1.0 / 512) == 1.0);
    CHECK(om_round_bf16(1.0 + 3.0 / 512) == 1.0 + 4.0 / 512);
    om_destroy(NULL);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle sanitized run: all checks passed\n");
    return 0;
}
