/*
 * CPU oracle of the CAS-Spec token-tree decoder step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load this library; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * What it computes (CAS-Spec, arXiv 2510.26843):
 *   - the target model's forward over the nodes of a draft token tree that is
 *     verified in one pass with tree attention (Sec. 4.2, "Tree Cascade" and
 *     "Tree-based Parallel Draft Generation"; Sec. 2, speculative decoding);
 *   - the same forward as a "virtual" draft model switched on by a DSIA
 *     strategy (Def. 4.1 and the strategy list of Sec. 4.1): layer sparsity
 *     (whole layers skipped per call) and activation quantisation (per-token
 *     int8 activations against an int8 copy of the weights; App. C);
 *   - committing the accepted path of a verified tree into the KV cache that
 *     drafts and target share (self-speculative decoding keeps no separate
 *     draft cache, Sec. 2).
 *
 * Plain definition, in fp64: every row (tree node) is computed on its own,
 * every dot product and every attention sum runs sequentially in increasing
 * index order, so a row's result never depends on which other rows are in the
 * call.  Masked keys are skipped rather than added as exp(-inf).
 *
 * Readings where the paper is silent (listed with reasons in the design notes):
 *   - position of a tree node = committed length + its depth (root depth 0);
 *   - a node attends to every committed slot plus its ancestors and itself;
 *   - Llama decoder: RMSNorm (eps inside the square root), rotate-half RoPE
 *     with inv_freq_i = theta^(-2i/hd), GQA head h -> kv head h/(H/Hkv),
 *     SwiGLU FFN, no biases, untied embedding and LM head;
 *   - bf16 models round to bf16 at storage points only: weights, the inputs of
 *     every linear layer (norm output, attention output, SwiGLU output), and
 *     q/k/v after RoPE (the KV cache is bf16).  fp32 models round nowhere;
 *   - int8 activations: per row s = amax/127 (fp32), q = clamp(rne(x/s),
 *     -127, 127), exact integer dot products, y = (fp32(acc) * s) * s_w[n] in
 *     fp32; weights: per output channel, the same rule.  Zero rows give s = 0
 *     and q = 0.  The LM head, attention and KV cache keep full precision;
 *   - int4 activations against int4 weights (the W4A4 form of activation
 *     quantisation the paper names, Sec. 4.1 and App. C): the same rules with
 *     7 in place of 127, codes in [-7, 7].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { W_Q = 0, W_K, W_V, W_O, W_GATE, W_UP, W_DOWN, W_COUNT };

typedef struct {
    const void *w[W_COUNT];           /* row-major [out][in]; bf16 bits or float */
    const float *attn_norm, *ffn_norm;
    const int8_t *q8[W_COUNT];        /* int8 copy (per output channel) */
    const float *s8[W_COUNT];
    const int8_t *q4[W_COUNT];        /* int4 copy: codes in [-7, 7], one per byte */
    const float *s4[W_COUNT];
} om_layer;

typedef struct {
    int L, d, H, Hkv, hd, ffn, V, bf16, max_ctx;
    double theta, eps;
    const void *embed, *lm_head;
    const float *final_norm;
    om_layer *layers;
    double *K, *Vv;                   /* [L][Hkv][max_ctx][hd] */
    int Lc;                           /* committed slots */
    int n_nodes;                      /* nodes of the current tree round */
    int verified;                     /* the last forward covered the whole round at full depth */
    int *parent, *depth, *token;      /* per node of the round */
    int attn_sink, attn_window;       /* efficient-attention draft (window 0: all committed slots) */
} om_model;

/* ------------------------------------------------------------------ numerics */

static double bf16_bits_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round a double to the nearest bfloat16 value (ties to even), returned as a
 * double.  bf16 keeps 8 significant bits; below 2^-126 the spacing is 2^-133. */
double om_round_bf16(double x) {
    if (x == 0.0 || !isfinite(x)) return x;
    int e;
    (void)frexp(x, &e);               /* |x| in [2^(e-1), 2^e) */
    int qexp = e - 8;
    if (qexp < -133) qexp = -133;
    double r = nearbyint(ldexp(x, -qexp));
    return ldexp(r, qexp);
}

static double weight_at(const om_model *m, const void *w, size_t idx) {
    if (m->bf16) return bf16_bits_to_double(((const uint16_t *)w)[idx]);
    return (double)((const float *)w)[idx];
}

/* y[r][o] = sum_k x[r][k] * W[o][k] for the rows r with run[r] set. */
static void linear_f64(const om_model *m, const void *w, int out, int in,
                       const double *x, int xstride, double *y, int ystride,
                       int nrows, const uint8_t *run) {
    #pragma omp parallel for schedule(static)
    for (int o = 0; o < out; o++) {
        for (int r = 0; r < nrows; r++) {
            if (!run[r]) continue;
            const double *xr = x + (size_t)r * xstride;
            double acc = 0.0;
            size_t base = (size_t)o * in;
            for (int k = 0; k < in; k++) acc += xr[k] * weight_at(m, w, base + k);
            y[(size_t)r * ystride + o] = acc;
        }
    }
}

/* Per-row symmetric quantisation to codes in [-qmax, qmax] (qmax 127: int8,
 * 7: int4), fp32 arithmetic, see header. */
void om_quant_row_q(const float *x, int n, int qmax, int8_t *q, float *scale) {
    const float qm = (float)qmax;
    float amax = 0.0f;
    for (int k = 0; k < n; k++) {
        float a = fabsf(x[k]);
        if (a > amax) amax = a;
    }
    float s = amax / qm;
    *scale = s;
    for (int k = 0; k < n; k++) {
        if (s == 0.0f) { q[k] = 0; continue; }
        float r = rintf(x[k] / s);
        if (r > qm) r = qm;
        if (r < -qm) r = -qm;
        q[k] = (int8_t)r;
    }
}
void om_quant_row(const float *x, int n, int8_t *q, float *scale) { om_quant_row_q(x, n, 127, q, scale); }

/* Per-output-channel copy of a weight matrix [out][in] (bf16 bits or float),
 * codes in [-qmax, qmax]. */
void om_quant_weight_q(const void *w, int bf16, int out, int in, int qmax, int8_t *q, float *scale) {
    #pragma omp parallel
    {
        float *row = (float *)malloc(sizeof(float) * (size_t)in);
        #pragma omp for schedule(static)
        for (int o = 0; o < out; o++) {
            for (int k = 0; k < in; k++) {
                size_t idx = (size_t)o * in + k;
                row[k] = bf16 ? (float)bf16_bits_to_double(((const uint16_t *)w)[idx])
                              : ((const float *)w)[idx];
            }
            om_quant_row_q(row, in, qmax, q + (size_t)o * in, scale + o);
        }
        free(row);
    }
}
void om_quant_weight(const void *w, int bf16, int out, int in, int8_t *q, float *scale) {
    om_quant_weight_q(w, bf16, out, in, 127, q, scale);
}

/* Exact integer dot product (int64), reported as int32 (|acc| < 2^31 is checked). */
int om_dot_i8(const int8_t *a, const int8_t *b, int n, int32_t *out) {
    int64_t acc = 0;
    for (int k = 0; k < n; k++) acc += (int64_t)a[k] * (int64_t)b[k];
    if (acc > INT32_MAX || acc < INT32_MIN) return -1;
    *out = (int32_t)acc;
    return 0;
}

/* Quantised-activation path of one linear layer (codes in [-qmax, qmax]
 * against the matching weight copy) for the rows with run[r] set. */
static int linear_iq(const int8_t *wq, const float *ws, int qmax, int out, int in,
                     const double *x, int xstride, double *y, int ystride,
                     int nrows, const uint8_t *run) {
    int8_t *qx = (int8_t *)malloc((size_t)nrows * in);
    float *sx = (float *)malloc(sizeof(float) * (size_t)nrows);
    float *row = (float *)malloc(sizeof(float) * (size_t)in);
    int bad = 0;
    for (int r = 0; r < nrows; r++) {
        if (!run[r]) continue;
        for (int k = 0; k < in; k++) row[k] = (float)x[(size_t)r * xstride + k];
        om_quant_row_q(row, in, qmax, qx + (size_t)r * in, sx + r);
    }
    free(row);
    #pragma omp parallel for schedule(static) reduction(|:bad)
    for (int o = 0; o < out; o++) {
        for (int r = 0; r < nrows; r++) {
            if (!run[r]) continue;
            int32_t acc;
            if (om_dot_i8(qx + (size_t)r * in, wq + (size_t)o * in, in, &acc)) { bad = 1; continue; }
            float v = (float)acc * sx[r];
            v = v * ws[o];
            y[(size_t)r * ystride + o] = (double)v;
        }
    }
    free(qx);
    free(sx);
    return bad ? -1 : 0;
}

/* RMSNorm of one row: y = x / sqrt(mean(x^2) + eps) * g. */
void om_rmsnorm_row(const double *x, const float *g, int n, double eps, double *y) {
    double ss = 0.0;
    for (int k = 0; k < n; k++) ss += x[k] * x[k];
    double r = 1.0 / sqrt(ss / (double)n + eps);
    for (int k = 0; k < n; k++) y[k] = x[k] * r * (double)g[k];
}

/* Rotate-half RoPE of one head vector at position pos. */
void om_rope(double *v, int hd, int pos, double theta) {
    int half = hd / 2;
    for (int i = 0; i < half; i++) {
        double inv_freq = pow(theta, -2.0 * (double)i / (double)hd);
        double ang = (double)pos * inv_freq;
        double c = cos(ang), s = sin(ang);
        double a = v[i], b = v[i + half];
        v[i] = a * c - b * s;
        v[i + half] = a * s + b * c;
    }
}

/* Attention of one query head over an explicit ordered key list:
 * o = sum_j softmax_j(q.k_j / sqrt(hd)) v_j.  keys/vals point at hd-vectors. */
void om_attend(const double *q, const double *const *keys, const double *const *vals,
               int nk, int hd, double *o) {
    double *sc = (double *)malloc(sizeof(double) * (size_t)(nk > 0 ? nk : 1));
    double scale = 1.0 / sqrt((double)hd);
    double mx = -INFINITY;
    for (int j = 0; j < nk; j++) {
        double s = 0.0;
        for (int e = 0; e < hd; e++) s += q[e] * keys[j][e];
        sc[j] = s * scale;
        if (sc[j] > mx) mx = sc[j];
    }
    double den = 0.0;
    for (int j = 0; j < nk; j++) { sc[j] = exp(sc[j] - mx); den += sc[j]; }
    for (int e = 0; e < hd; e++) o[e] = 0.0;
    for (int j = 0; j < nk; j++)
        for (int e = 0; e < hd; e++) o[e] += sc[j] * vals[j][e];
    for (int e = 0; e < hd; e++) o[e] = nk > 0 ? o[e] / den : 0.0;
    free(sc);
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* ------------------------------------------------------------------ model */

om_model *om_create(int L, int d, int H, int Hkv, int hd, int ffn, int V,
                    double theta, double eps, int bf16, int max_ctx) {
    if (L <= 0 || d <= 0 || H <= 0 || Hkv <= 0 || H % Hkv || hd % 2 || max_ctx <= 0) return NULL;
    om_model *m = (om_model *)calloc(1, sizeof(om_model));
    m->L = L; m->d = d; m->H = H; m->Hkv = Hkv; m->hd = hd; m->ffn = ffn; m->V = V;
    m->theta = theta; m->eps = eps; m->bf16 = bf16; m->max_ctx = max_ctx;
    m->layers = (om_layer *)calloc((size_t)L, sizeof(om_layer));
    size_t kv = (size_t)L * Hkv * max_ctx * hd;
    m->K = (double *)calloc(kv, sizeof(double));
    m->Vv = (double *)calloc(kv, sizeof(double));
    m->parent = (int *)calloc((size_t)max_ctx, sizeof(int));
    m->depth = (int *)calloc((size_t)max_ctx, sizeof(int));
    m->token = (int *)calloc((size_t)max_ctx, sizeof(int));
    if (!m->layers || !m->K || !m->Vv || !m->parent || !m->depth || !m->token) {
        free(m->layers); free(m->K); free(m->Vv); free(m->parent); free(m->depth); free(m->token);
        free(m);
        return NULL;
    }
    return m;
}

void om_destroy(om_model *m) {
    if (!m) return;
    free(m->layers); free(m->K); free(m->Vv); free(m->parent); free(m->depth); free(m->token);
    free(m);
}

void om_set_global(om_model *m, const void *embed, const void *lm_head, const float *final_norm) {
    m->embed = embed; m->lm_head = lm_head; m->final_norm = final_norm;
}

/* w: the 7 projections in the order q, k, v, o, gate, up, down. */
void om_set_layer(om_model *m, int l, const void *const *w, const float *attn_norm, const float *ffn_norm) {
    for (int i = 0; i < W_COUNT; i++) m->layers[l].w[i] = w[i];
    m->layers[l].attn_norm = attn_norm;
    m->layers[l].ffn_norm = ffn_norm;
}

void om_set_layer_i4(om_model *m, int l, const int8_t *const *q, const float *const *s) {
    for (int i = 0; i < W_COUNT; i++) { m->layers[l].q4[i] = q[i]; m->layers[l].s4[i] = s[i]; }
}
void om_set_layer_i8(om_model *m, int l, const int8_t *const *q, const float *const *s) {
    for (int i = 0; i < W_COUNT; i++) { m->layers[l].q8[i] = q[i]; m->layers[l].s8[i] = s[i]; }
}

void om_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int om_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

static double *kslot(om_model *m, int l, int kvh, int slot) {
    return m->K + (((size_t)l * m->Hkv + kvh) * m->max_ctx + slot) * m->hd;
}
static double *vslot(om_model *m, int l, int kvh, int slot) {
    return m->Vv + (((size_t)l * m->Hkv + kvh) * m->max_ctx + slot) * m->hd;
}

/* Write committed KV directly (a cache restored from elsewhere): slots
 * [0, n) of one layer, inputs [Hkv][n][hd] float32. */
int om_set_kv(om_model *m, int l, int n, const float *k, const float *v) {
    if (l < 0 || l >= m->L || n < 0 || n > m->max_ctx) return -1;
    for (int h = 0; h < m->Hkv; h++)
        for (int s = 0; s < n; s++)
            for (int e = 0; e < m->hd; e++) {
                size_t src = ((size_t)h * n + s) * m->hd + e;
                kslot(m, l, h, s)[e] = (double)k[src];
                vslot(m, l, h, s)[e] = (double)v[src];
            }
    return 0;
}

int om_get_kv(om_model *m, int l, int kvh, int slot, double *k, double *v) {
    if (l < 0 || l >= m->L || kvh < 0 || kvh >= m->Hkv || slot < 0 || slot >= m->max_ctx) return -1;
    memcpy(k, kslot(m, l, kvh, slot), sizeof(double) * m->hd);
    memcpy(v, vslot(m, l, kvh, slot), sizeof(double) * m->hd);
    return 0;
}

int om_set_committed(om_model *m, int Lc) {
    if (Lc < 0 || Lc > m->max_ctx) return -1;
    m->Lc = Lc; m->n_nodes = 0; m->verified = 0;
    return 0;
}
int om_committed(const om_model *m) { return m->Lc; }

/* Efficient attention as a DSIA strategy (Sec. 4.1, StreamingLLM-style): the
 * forwards that follow see, of the committed slots, only the first `sink`
 * and the last `window` ones (window 0: all of them).  Such a forward is a
 * draft, never a verify. */
int om_set_window(om_model *m, int sink, int window) {
    if (sink < 0 || window < 0) return -1;
    m->attn_sink = window > 0 ? sink : 0;
    m->attn_window = window;
    return 0;
}

/*
 * Forward over n new tree nodes (ids node_offset .. node_offset+n-1 of the
 * current round).  node_offset 0 starts a new round; otherwise the call
 * appends to the round.  parents are node ids (root: -1, only node 0).
 * skip: per-layer 0/1 (NULL = none).  act_quant: 0, 1 = int8 activations
 * against the int8 copy, 2 = int4 activations against the int4 copy.
 * need: rows whose logits are wanted (NULL = all); their ancestors inside the
 * call are computed too, other rows are left out (their KV is not written).
 * logits: [n][V] doubles (rows not computed are untouched).
 * Returns 0, or -1 on invalid arguments (state unchanged), -2 on int8 overflow.
 */
int om_forward(om_model *m, const int32_t *tokens, const int32_t *parents, int node_offset, int n,
               const uint8_t *skip, int act_quant, const uint8_t *need, double *logits) {
    if (n <= 0 || node_offset < 0 || act_quant < 0 || act_quant > 2) return -1;
    if (node_offset != 0 && node_offset != m->n_nodes) return -1;
    if (m->Lc + node_offset + n > m->max_ctx) return -1;
    for (int i = 0; i < n; i++) {
        int node = node_offset + i;
        if (tokens[i] < 0 || tokens[i] >= m->V) return -1;
        if (node == 0) { if (parents[i] != -1) return -1; }
        else if (parents[i] < 0 || parents[i] >= node) return -1;
    }
    if (act_quant) {
        for (int l = 0; l < m->L; l++) {
            if (skip && skip[l]) continue;
            for (int w = 0; w < W_COUNT; w++)
                if (!(act_quant == 1 ? m->layers[l].q8[w] : m->layers[l].q4[w])) return -1;
        }
    }
    const int d = m->d, H = m->H, Hkv = m->Hkv, hd = m->hd, ffn = m->ffn, G = H / Hkv;
    const int qd = H * hd, kd = Hkv * hd;
    int full = 1;
    for (int l = 0; l < m->L; l++) if (skip && skip[l]) full = 0;

    for (int i = 0; i < n; i++) {
        int node = node_offset + i;
        m->parent[node] = parents[i];
        m->token[node] = tokens[i];
        m->depth[node] = parents[i] < 0 ? 0 : m->depth[parents[i]] + 1;
    }
    m->n_nodes = node_offset + n;
    m->verified = (node_offset == 0 && full && !act_quant && m->attn_window == 0);

    uint8_t *run = (uint8_t *)calloc((size_t)n, 1);
    for (int i = n - 1; i >= 0; i--) {
        if (!need || need[i]) run[i] = 1;
        if (run[i] && parents[i] >= node_offset) run[parents[i] - node_offset] = 1;
    }
    int wmax = ffn > qd ? ffn : qd;
    if (d > wmax) wmax = d;
    double *h = (double *)calloc((size_t)n * d, sizeof(double));
    double *xn = (double *)calloc((size_t)n * wmax, sizeof(double));
    double *q = (double *)calloc((size_t)n * qd, sizeof(double));
    double *k = (double *)calloc((size_t)n * kd, sizeof(double));
    double *v = (double *)calloc((size_t)n * kd, sizeof(double));
    double *ao = (double *)calloc((size_t)n * qd, sizeof(double));
    double *g = (double *)calloc((size_t)n * ffn, sizeof(double));
    double *u = (double *)calloc((size_t)n * ffn, sizeof(double));
    double *y = (double *)calloc((size_t)n * wmax, sizeof(double));
    int *anc = (int *)malloc(sizeof(int) * (size_t)(m->n_nodes + 1));
    int rc = 0;

    for (int i = 0; i < n; i++) {
        if (!run[i]) continue;
        for (int e = 0; e < d; e++) h[(size_t)i * d + e] = weight_at(m, m->embed, (size_t)tokens[i] * d + e);
    }

#define ROUND(val) (m->bf16 ? om_round_bf16(val) : (val))
#define LINEAR(widx, out, in, X, xs, Y, ys)                                                     \
    do {                                                                                        \
        if (act_quant) {                                                                        \
            if (act_quant == 1 ? linear_iq(lay->q8[widx], lay->s8[widx], 127, out, in, X, xs, Y, ys, n, run) \
                               : linear_iq(lay->q4[widx], lay->s4[widx], 7, out, in, X, xs, Y, ys, n, run))   \
                rc = -2;                                                                        \
        } else {                                                                                \
            linear_f64(m, lay->w[widx], out, in, X, xs, Y, ys, n, run);                          \
        }                                                                                       \
    } while (0)

    for (int l = 0; l < m->L && rc == 0; l++) {
        if (skip && skip[l]) continue;
        const om_layer *lay = &m->layers[l];
        /* attention block */
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            om_rmsnorm_row(h + (size_t)i * d, lay->attn_norm, d, m->eps, xn + (size_t)i * wmax);
            for (int e = 0; e < d; e++) xn[(size_t)i * wmax + e] = ROUND(xn[(size_t)i * wmax + e]);
        }
        LINEAR(W_Q, qd, d, xn, wmax, q, qd);
        LINEAR(W_K, kd, d, xn, wmax, k, kd);
        LINEAR(W_V, kd, d, xn, wmax, v, kd);
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            int node = node_offset + i;
            int pos = m->Lc + m->depth[node];
            for (int hh = 0; hh < H; hh++) om_rope(q + (size_t)i * qd + (size_t)hh * hd, hd, pos, m->theta);
            for (int hh = 0; hh < Hkv; hh++) om_rope(k + (size_t)i * kd + (size_t)hh * hd, hd, pos, m->theta);
            for (int e = 0; e < qd; e++) q[(size_t)i * qd + e] = ROUND(q[(size_t)i * qd + e]);
            for (int e = 0; e < kd; e++) {
                k[(size_t)i * kd + e] = ROUND(k[(size_t)i * kd + e]);
                v[(size_t)i * kd + e] = ROUND(v[(size_t)i * kd + e]);
            }
            int slot = m->Lc + node;
            for (int hh = 0; hh < Hkv; hh++) {
                memcpy(kslot(m, l, hh, slot), k + (size_t)i * kd + (size_t)hh * hd, sizeof(double) * hd);
                memcpy(vslot(m, l, hh, slot), v + (size_t)i * kd + (size_t)hh * hd, sizeof(double) * hd);
            }
        }
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            int node = node_offset + i;
            /* visible keys: the committed slots (all, or the sink and the
               recent window), then ancestors-or-self by increasing id */
            int na = 0;
            for (int a = node; a >= 0; a = m->parent[a]) anc[na++] = a;
            int c_lo = m->Lc, c_hi = m->Lc;   /* committed slots [0, c_lo) and [c_hi, Lc) */
            if (m->attn_window > 0) {
                c_lo = m->attn_sink < m->Lc ? m->attn_sink : m->Lc;
                c_hi = m->Lc - m->attn_window;
                if (c_hi < c_lo) c_hi = c_lo;
            }
            int nc = c_lo + (m->Lc - c_hi);
            int nk = nc + na;
            #pragma omp parallel for schedule(static)
            for (int hh = 0; hh < H; hh++) {
                int kvh = hh / G;
                const double **kl = (const double **)malloc(sizeof(double *) * (size_t)nk);
                const double **vl = (const double **)malloc(sizeof(double *) * (size_t)nk);
                int c = 0;
                for (int s = 0; s < c_lo; s++, c++) { kl[c] = kslot(m, l, kvh, s); vl[c] = vslot(m, l, kvh, s); }
                for (int s = c_hi; s < m->Lc; s++, c++) { kl[c] = kslot(m, l, kvh, s); vl[c] = vslot(m, l, kvh, s); }
                for (int j = 0; j < na; j++) {
                    int a = anc[na - 1 - j];
                    kl[nc + j] = kslot(m, l, kvh, m->Lc + a);
                    vl[nc + j] = vslot(m, l, kvh, m->Lc + a);
                }
                om_attend(q + (size_t)i * qd + (size_t)hh * hd, kl, vl, nk, hd, ao + (size_t)i * qd + (size_t)hh * hd);
                free(kl); free(vl);
            }
            for (int e = 0; e < qd; e++) ao[(size_t)i * qd + e] = ROUND(ao[(size_t)i * qd + e]);
        }
        LINEAR(W_O, d, qd, ao, qd, y, wmax);
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            for (int e = 0; e < d; e++) h[(size_t)i * d + e] += y[(size_t)i * wmax + e];
        }
        /* FFN block */
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            om_rmsnorm_row(h + (size_t)i * d, lay->ffn_norm, d, m->eps, xn + (size_t)i * wmax);
            for (int e = 0; e < d; e++) xn[(size_t)i * wmax + e] = ROUND(xn[(size_t)i * wmax + e]);
        }
        LINEAR(W_GATE, ffn, d, xn, wmax, g, ffn);
        LINEAR(W_UP, ffn, d, xn, wmax, u, ffn);
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            for (int e = 0; e < ffn; e++) {
                size_t idx = (size_t)i * ffn + e;
                xn[(size_t)i * wmax + e] = ROUND(silu(g[idx]) * u[idx]);
            }
        }
        LINEAR(W_DOWN, d, ffn, xn, wmax, y, wmax);
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            for (int e = 0; e < d; e++) h[(size_t)i * d + e] += y[(size_t)i * wmax + e];
        }
    }
    if (rc == 0) {
        for (int i = 0; i < n; i++) {
            if (!run[i]) continue;
            om_rmsnorm_row(h + (size_t)i * d, m->final_norm, d, m->eps, xn + (size_t)i * wmax);
            for (int e = 0; e < d; e++) xn[(size_t)i * wmax + e] = ROUND(xn[(size_t)i * wmax + e]);
        }
        if (logits) {
            uint8_t *want = (uint8_t *)calloc((size_t)n, 1);
            for (int i = 0; i < n; i++) want[i] = run[i] && (!need || need[i]);
            linear_f64(m, m->lm_head, m->V, d, xn, wmax, logits, m->V, n, want);
            free(want);
        }
    }
#undef LINEAR
#undef ROUND
    free(run); free(h); free(xn); free(q); free(k); free(v); free(ao); free(g); free(u); free(y); free(anc);
    return rc;
}

/*
 * Commit the accepted root path of the current round: node accepted[j] (at
 * depth j) moves from slot Lc+accepted[j] to slot Lc+j in every layer, in
 * increasing depth, then Lc grows by n_acc.  Requires a verified round.
 */
int om_compact(om_model *m, const int32_t *accepted, int n_acc) {
    if (!m->verified || n_acc <= 0 || n_acc > m->n_nodes) return -1;
    if (accepted[0] != 0) return -1;
    for (int j = 1; j < n_acc; j++) {
        if (accepted[j] <= 0 || accepted[j] >= m->n_nodes) return -1;
        if (m->parent[accepted[j]] != accepted[j - 1]) return -1;
    }
    for (int l = 0; l < m->L; l++)
        for (int h = 0; h < m->Hkv; h++)
            for (int j = 0; j < n_acc; j++) {
                int src = m->Lc + accepted[j], dst = m->Lc + j;
                if (src == dst) continue;
                memmove(kslot(m, l, h, dst), kslot(m, l, h, src), sizeof(double) * m->hd);
                memmove(vslot(m, l, h, dst), vslot(m, l, h, src), sizeof(double) * m->hd);
            }
    m->Lc += n_acc;
    m->n_nodes = 0;
    m->verified = 0;
    return 0;
}
