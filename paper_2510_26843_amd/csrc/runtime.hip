// Runtime behind the C ABI of include/cas.h and include/cas_ops.h: weight
// store (device layouts for the fused epilogues), KV cache with committed and
// tree-scratch regions, round bookkeeping, argument validation, launch
// sequencing, HIP graph cache and per-kernel event timing.
#include "cas.h"
#include "cas_ops.h"
#include "cas_internal.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

using namespace cas;

namespace {

constexpr int kStages = 8;          // pinned upload buffers in flight
constexpr size_t kMaxGraphs = 64;   // captured forwards kept at once
// Block order of each layer's projection (QKV, O, gate/up, down) and of its
// int8 copy: 1 = K-major (wt_kmajor).  The LM head is K-major too; the packed
// int4 copies stay tile-major.  Measured with cold weights and in the
// forwards: K-major gate/up 7B T = 32 34.9 -> 34.0 us, 8B one-row verify
// 1.40 -> 1.19 ms per forward; LM head 7B 50.3 -> 43.6 us.  The O projection
// gained on the 7B shape (12.6 -> 11.6 us) but lost on the 13B one (445 ->
// 482 us per forward), and QKV and down lost 3-4%: they stay tile-major.
constexpr int kProjKMajor[4] = {0, 0, 1, 0};
constexpr size_t kStageBytes = 4096;

struct LayerW {
    void* wqkv = nullptr;   // [qkv_rows][d]: q heads, k heads (rows pair-interleaved), v heads
    void* wo = nullptr;     // [d][H*hd]
    void* wgu = nullptr;    // [2*ffn][d]: rows gate 0, up 0, gate 1, up 1, ...
    void* wd = nullptr;     // [d][ffn]
    float* attn_norm = nullptr;
    float* ffn_norm = nullptr;
    int8_t* q8[4] = {nullptr, nullptr, nullptr, nullptr};  // int8 copies in the same row layouts
    float* s8[4] = {nullptr, nullptr, nullptr, nullptr};
    uint8_t* q4[4] = {nullptr, nullptr, nullptr, nullptr};  // packed int4 copies (same rows, int8 chunking)
    float* s4[4] = {nullptr, nullptr, nullptr, nullptr};
    unsigned loaded = 0;    // bit per tensor kind
};

struct Stage {
    unsigned char* host = nullptr;
    hipEvent_t ev = nullptr;
    bool pending = false;
};

struct ProfRec {
    int cls;
    hipEvent_t a, b;
};

}  // namespace

struct cas_ctx {
    cas_config cfg{};
    int dev = 0;
    hipStream_t stream = nullptr;
    bool own_stream = false;
    int et = ET_BF16;
    size_t es = 2;
    int qrows = 0, krows = 0, qkv_rows = 0, ctx_cap = 0;
    // padded widths of the tiled weights (model type) and of the int8 copies
    int kp_d = 0, kp_q = 0, kp_f = 0, kq_d = 0, kq_q = 0, kq_f = 0;
    void* stage_dev = nullptr;  // device staging of one row-major tensor during loads
    size_t stage_dev_bytes = 0;

    void* embed = nullptr;
    void* lm_head = nullptr;
    float* final_norm = nullptr;
    unsigned global_loaded = 0;
    std::vector<LayerW> layers;
    bool int8_ready = false;
    bool int4_ready = false;

    void* kc = nullptr;  // [L][Hkv][ctx_cap][hd]
    void* vt = nullptr;  // [L][Hkv][hd][ctx_cap]
    float* rope_cos = nullptr;
    float* rope_sin = nullptr;

    int Lc = 0, n_nodes = 0, verified_n = 0, logits_rows = 0;
    std::vector<int> parent, token;

    int* d_rtok = nullptr;
    int* d_rpar = nullptr;
    StepParams* d_sp = nullptr;
    int* d_chk = nullptr;  // device check word (CAS_DEBUG builds)
    int chk_cap = 0;       // slot capacity the device checks allow (0: ctx_cap)
    int* d_row_pos = nullptr;
    int* d_row_slot = nullptr;
    uint64_t* d_row_anc = nullptr;
    float* d_h = nullptr;
    void* d_xn = nullptr;
    int8_t* d_xq = nullptr;
    float* d_xs = nullptr;
    void* d_q = nullptr;
    void* d_ao = nullptr;
    void* d_sw = nullptr;
    float* d_logits = nullptr;
    float* d_part = nullptr;
    float* d_gpart = nullptr;  // split-K partial sums of the O / down projections [8][max_tree][d_model]
    size_t part_bytes = 0;
    int* d_gbuf = nullptr;
    int* d_result = nullptr;
    int* d_acc = nullptr;
    int* h_result = nullptr;  // pinned
    int* d_topk = nullptr;    // [max_tree][16] ids, [max_tree][16] probabilities, [max_tree] NaN flags
    int* h_topk = nullptr;    // pinned copy of the same

    Stage stage[kStages];
    int stage_i = 0;

    bool graphs = true;
    bool gemv = false;  // GEMV-style tiles for one-row drafts (cas_set_gemv)
    std::map<std::string, hipGraphExec_t> gcache;
    int win_sink = 0, win_len = 0;  // attention window of the forward being enqueued (0: none)

    bool prof = false;
    std::vector<ProfRec> prec;
    std::vector<hipEvent_t> ev_pool;
    double pms[CAS_K_COUNT] = {};
    int pn[CAS_K_COUNT] = {};

    std::vector<void*> allocs;
    std::string err;
};

namespace {

std::string g_create_err;

cas_status fail(cas_ctx* c, cas_status st, const std::string& msg) {
    if (c) c->err = msg;
    return st;
}

cas_status hip_fail(cas_ctx* c, hipError_t e, const char* what) {
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    return fail(c, CAS_ERR_DEVICE, m);
}

#define HIPCHK(c, expr)                                        \
    do {                                                       \
        hipError_t _e = (expr);                                \
        if (_e != hipSuccess) return hip_fail((c), _e, #expr); \
    } while (0)

// CAS_DEBUG builds: after a synchronisation, report (and clear) a failed
// device check as CAS_ERR_DEVICE.  Release builds: nothing to read.
cas_status poll_checks(cas_ctx* c) {
    if constexpr (kDeviceChecks) {
        int code = 0;
        HIPCHK(c, hipMemcpy(&code, c->d_chk, sizeof code, hipMemcpyDeviceToHost));
        if (code) {
            HIPCHK(c, hipMemset(c->d_chk, 0, sizeof code));
            static const char* const names[CHK_COUNT] = {
                "none", "tree size", "token id", "parent order", "slot capacity", "RoPE position",
                "KV write slot", "attention slots", "compaction path", "acceptance parent"};
            return fail(c, CAS_ERR_DEVICE, std::string("device check failed: ") +
                                               (code > 0 && code < CHK_COUNT ? names[code] : "unknown") +
                                               " (code " + std::to_string(code) + ")");
        }
    }
    return CAS_OK;
}

template <typename T>
hipError_t dalloc(cas_ctx* c, T** p, size_t bytes) {
    void* q = nullptr;
    hipError_t e = hipMalloc(&q, bytes ? bytes : 16);
    if (e != hipSuccess) return e;
    c->allocs.push_back(q);
    *p = (T*)q;
    return hipSuccess;
}

hipEvent_t take_event(cas_ctx* c) {
    if (!c->ev_pool.empty()) {
        hipEvent_t e = c->ev_pool.back();
        c->ev_pool.pop_back();
        return e;
    }
    // timing-only events: no system-scope fence (cache writeback) at record,
    // so the bracket measures the launch rather than the fence
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

// Launch wrapper: with profiling on, bracket the launch with events.
template <typename F>
hipError_t timed(cas_ctx* c, int cls, F&& f) {
    if (!c->prof) return f();
    hipEvent_t a = take_event(c), b = take_event(c);
    if (!a || !b) return hipErrorOutOfMemory;
    hipError_t e = hipEventRecord(a, c->stream);
    if (e != hipSuccess) return e;
    e = f();
    if (e != hipSuccess) return e;
    e = hipEventRecord(b, c->stream);
    if (e != hipSuccess) return e;
    c->prec.push_back({cls, a, b});
    return hipSuccess;
}

// Pinned upload buffer whose previous copy has completed.
unsigned char* next_stage(cas_ctx* c, hipEvent_t* ev) {
    Stage& s = c->stage[c->stage_i];
    c->stage_i = (c->stage_i + 1) % kStages;
    if (s.pending) {
        if (hipEventSynchronize(s.ev) != hipSuccess) return nullptr;
        s.pending = false;
    }
    *ev = s.ev;
    s.pending = true;
    return s.host;
}

size_t tensor_elems(const cas_ctx* c, int kind) {
    const cas_config& f = c->cfg;
    const size_t d = f.d_model, hd = f.head_dim;
    switch (kind) {
    case CAS_T_EMBED:
    case CAS_T_LM_HEAD: return (size_t)f.vocab * d;
    case CAS_T_FINAL_NORM:
    case CAS_T_ATTN_NORM:
    case CAS_T_FFN_NORM: return d;
    case CAS_T_WQ: return (size_t)f.n_heads * hd * d;
    case CAS_T_WK:
    case CAS_T_WV: return (size_t)f.n_kv_heads * hd * d;
    case CAS_T_WO: return d * f.n_heads * hd;
    case CAS_T_W_GATE:
    case CAS_T_W_UP:
    case CAS_T_W_DOWN: return d * (size_t)f.ffn_dim;
    }
    return 0;
}

bool is_norm(int kind) { return kind == CAS_T_FINAL_NORM || kind == CAS_T_ATTN_NORM || kind == CAS_T_FFN_NORM; }
bool is_global(int kind) { return kind == CAS_T_EMBED || kind == CAS_T_LM_HEAD || kind == CAS_T_FINAL_NORM; }
constexpr unsigned kLayerMask = (1u << CAS_T_ATTN_NORM) | (1u << CAS_T_FFN_NORM) | (1u << CAS_T_WQ) |
                                (1u << CAS_T_WK) | (1u << CAS_T_WV) | (1u << CAS_T_WO) | (1u << CAS_T_W_GATE) |
                                (1u << CAS_T_W_UP) | (1u << CAS_T_W_DOWN);
constexpr unsigned kGlobalMask = (1u << CAS_T_EMBED) | (1u << CAS_T_LM_HEAD) | (1u << CAS_T_FINAL_NORM);

// Host copy of the tree checks shared by cas_tree_info and cas_forward.
bool tree_depths(const int32_t* parent, int first, int n, const std::vector<int>& prior, std::vector<int>* depth,
                 std::string* why) {
    depth->assign(first + n, 0);
    for (int j = 0; j < first; ++j) (*depth)[j] = 0;
    // depths of prior nodes
    for (int j = 0; j < first; ++j) {
        const int p = prior[j];
        (*depth)[j] = p < 0 ? 0 : (*depth)[p] + 1;
    }
    for (int i = 0; i < n; ++i) {
        const int node = first + i, p = parent[i];
        if (node == 0) {
            if (p != -1) {
                *why = "node 0 (the root) must have parent -1";
                return false;
            }
            (*depth)[0] = 0;
        } else {
            if (p < 0 || p >= node) {
                char b[128];
                snprintf(b, sizeof b, "node %d has parent %d; parents must precede their children", node, p);
                *why = b;
                return false;
            }
            (*depth)[node] = (*depth)[p] + 1;
        }
    }
    return true;
}

// The forward's launch sequence (captured into a graph, or launched directly).
hipError_t enqueue_forward(cas_ctx* c, int T, const uint8_t* skip, int aq) {
    const cas_config& f = c->cfg;
    const int d = f.d_model, H = f.n_heads, Hkv = f.n_kv_heads, hd = f.head_dim, ffn = f.ffn_dim;
    const int et = c->et;
    hipStream_t s = c->stream;
    hipError_t e;
#define RUN(cls, call)                                        \
    do {                                                      \
        e = timed(c, (cls), [&]() -> hipError_t { return call; }); \
        if (e != hipSuccess) return e;                        \
    } while (0)

    RUN(CAS_K_EMBED, launch_embed(et, c->embed, d, f.vocab, c->d_rtok, c->d_rpar, c->d_sp, T, c->d_h,
                                  c->d_row_pos, c->d_row_slot, c->d_row_anc, c->d_chk, s));
    const size_t kv_layer = (size_t)Hkv * c->ctx_cap * hd * c->es;
    AttnArgs at{};
    at.q = c->d_q;
    at.anc = c->d_row_anc;
    at.sp = c->d_sp;
    at.chk = c->d_chk;
    at.out = c->d_ao;
    at.out_tiled = 1;
    at.T = T;
    at.H = H;
    at.Hkv = Hkv;
    at.hd = hd;
    at.ctx_cap = c->ctx_cap;
    // splits for the attention grid come from the host copy of the state
    at.Lc_host = c->Lc;
    at.n_tree_host = c->n_nodes;  // already the post-call node count
    at.win_sink = c->win_sink;
    at.win_len = c->win_len;
    const int S = attention_splits_win(at.Lc_host, at.n_tree_host, at.win_sink, at.win_len);
    at.part_o = c->d_part;
    at.part_ml = c->d_part + (size_t)S * H * T * hd;
    // act_quant 1: int8 codes against the int8 copy; 2: int4 codes (one per
    // byte) against the packed int4 copy
    const int wq = aq == 2 ? (int)ET_I4 : aq ? (int)ET_I8 : et;
    const int qmax = aq == 2 ? 7 : 127;
    auto wcopy = [&](const LayerW& w, int i) -> const void* { return aq == 2 ? (const void*)w.q4[i] : (const void*)w.q8[i]; };
    auto scopy = [&](const LayerW& w, int i) -> const float* { return aq == 2 ? w.s4[i] : w.s8[i]; };
    // one-node quantised drafts on bf16 models: the O and down projections
    // quantise their bf16 input on load when they can (no codes from the
    // attention merge, no separate quantiser of the SwiGLU output); the QKV
    // and gate/up inputs keep the codes their RMSNorm writes
    const bool qxs = aq && et == ET_BF16;
    // drafts of one row (a layer skipped, quantised activations or an
    // attention window) take the GEMV-style tiles in the wide GEMMs when the
    // caller asks for them (cas_set_gemv); verify calls always keep the MFMA
    // form, whose row sums do not depend on the tree size
    bool skips = false;
    for (int l = 0; skip && l < f.n_layers; ++l) skips = skips || skip[l];
    const int gv = c->gemv && T == 1 && (skips || aq || c->win_len > 0) ? 1 : 0;
    const int ks_o = gemm_parts_count(wq, d, c->kq_q, T), ks_d = gemm_parts_count(wq, d, c->kq_f, T);
    const bool qx_o = qxs && gemm_qx_ok(wq, d, c->kq_q, T, ks_o);
    const bool qx_d = qxs && gemm_qx_ok(wq, d, c->kq_f, T, ks_d);
    // bf16 forwards of one or two rows: the O projection merges the
    // attention's split partials itself (no merge launch)
    const bool mx_o = !aq && et == ET_BF16 && gemm_mx_ok(et, d, c->kp_q, T, gemm_parts_count(et, d, c->kp_q, T));
    // split-K sums of the last O / down projection that the next RMSNorm
    // adds to the residual stream (0: the projection updated it itself)
    int pend = 0;
    const size_t pstride = (size_t)T * d;
    auto norm = [&](const float* gain, void* out, int8_t* qo, float* qso) -> hipError_t {
        const hipError_t r = launch_rmsnorm(et, c->d_h, gain, T, d, f.rms_eps, out, qo, qso, c->d_gpart, pend,
                                            pstride, qmax, s);
        pend = 0;
        return r;
    };
    // a residual projection: split-K partial sums when that fills the GPU better
    auto resid_proj = [&](GemmArgs& g) -> hipError_t {
        const int ks = gemm_parts_count(wq, g.N, g.Kp, T);
        if (ks <= 1) return launch_gemm(wq, et, EPI_RESID, g, s);
        g.out = c->d_gpart;
        g.ksplit = ks;
        g.part_stride = pstride;
        const hipError_t r = launch_gemm_parts(wq, g, s);
        if (r == hipSuccess) pend = ks;
        return r;
    };

    for (int l = 0; l < f.n_layers; ++l) {
        if (skip && skip[l]) continue;
        LayerW& w = c->layers[l];
        void* kc = (char*)c->kc + kv_layer * l;
        void* vt = (char*)c->vt + kv_layer * l;
        // --- attention block
        RUN(CAS_K_RMSNORM, norm(w.attn_norm, aq ? nullptr : c->d_xn, aq ? c->d_xq : nullptr, c->d_xs));
        GemmArgs g{};
        g.T = T;
        g.N = c->qkv_rows;
        g.Kp = aq ? c->kq_d : c->kp_d;
        g.W = aq ? wcopy(w, 0) : w.wqkv;
        g.X = aq ? (const void*)c->d_xq : c->d_xn;
        g.xs = c->d_xs;
        g.ws = scopy(w, 0);
        g.out = c->d_q;
        g.gv = gv;
        g.chk = c->d_chk;
        g.kmaj = aq == 2 ? 0 : kProjKMajor[0];
        g.rope_cos = c->rope_cos;
        g.rope_sin = c->rope_sin;
        g.row_pos = c->d_row_pos;
        g.row_slot = c->d_row_slot;
        g.kc = kc;
        g.vt = vt;
        g.H = H;
        g.Hkv = Hkv;
        g.hd = hd;
        g.ctx_cap = c->ctx_cap;
        RUN(CAS_K_GEMM_QKV, launch_gemm(wq, et, EPI_QKV, g, s));
        at.kc = kc;
        at.vt = vt;
        // quantised drafts on bf16 models: the attention's merge writes the
        // O projection's input codes itself, unless that projection quantises
        // on load
        const bool fused_q = aq && et == ET_BF16 && !qx_o;
        at.qout = fused_q ? c->d_xq : nullptr;
        at.qscale = fused_q ? c->d_xs : nullptr;
        at.qmax = qmax;
        at.no_merge = mx_o ? 1 : 0;
        RUN(CAS_K_ATTN, launch_attention(et, at, s));
        if (aq && !fused_q && !qx_o)
            RUN(CAS_K_QUANT, launch_quant_rows(et, c->d_ao, T, H * hd, c->d_xq, c->d_xs, 1, qmax, s));
        GemmArgs go{};
        go.T = T;
        go.N = d;
        go.Kp = aq ? c->kq_q : c->kp_q;
        go.W = aq ? wcopy(w, 1) : w.wo;
        go.X = aq && !qx_o ? (const void*)c->d_xq : c->d_ao;
        go.qx = qx_o ? qmax : 0;
        go.xk = H * hd;
        go.mx_o = mx_o ? at.part_o : nullptr;
        go.mx_ml = at.part_ml;
        go.mx_S = S;
        go.H = H;
        go.hd = hd;
        go.xs = c->d_xs;
        go.ws = scopy(w, 1);
        go.out = c->d_h;
        go.ldo = d;
        go.kmaj = aq == 2 ? 0 : kProjKMajor[1];
        RUN(CAS_K_GEMM_O, resid_proj(go));
        // --- FFN block
        RUN(CAS_K_RMSNORM, norm(w.ffn_norm, aq ? nullptr : c->d_xn, aq ? c->d_xq : nullptr, c->d_xs));
        GemmArgs gu{};
        gu.T = T;
        gu.N = 2 * ffn;
        gu.Kp = aq ? c->kq_d : c->kp_d;
        gu.W = aq ? wcopy(w, 2) : w.wgu;
        gu.X = aq ? (const void*)c->d_xq : c->d_xn;
        gu.xs = c->d_xs;
        gu.ws = scopy(w, 2);
        gu.out = c->d_sw;
        gu.ldo = ffn;
        gu.out_k = ffn;
        gu.gv = gv;
        gu.kmaj = aq == 2 ? 0 : kProjKMajor[2];
        RUN(CAS_K_GEMM_GATEUP, launch_gemm(wq, et, EPI_SWIGLU, gu, s));
        if (aq && !qx_d) RUN(CAS_K_QUANT, launch_quant_rows(et, c->d_sw, T, ffn, c->d_xq, c->d_xs, 1, qmax, s));
        GemmArgs gd{};
        gd.T = T;
        gd.N = d;
        gd.Kp = aq ? c->kq_f : c->kp_f;
        gd.W = aq ? wcopy(w, 3) : w.wd;
        gd.X = aq && !qx_d ? (const void*)c->d_xq : c->d_sw;
        gd.qx = qx_d ? qmax : 0;
        gd.xk = ffn;
        gd.xs = c->d_xs;
        gd.ws = scopy(w, 3);
        gd.out = c->d_h;
        gd.ldo = d;
        gd.kmaj = aq == 2 ? 0 : kProjKMajor[3];
        RUN(CAS_K_GEMM_DOWN, resid_proj(gd));
    }
    RUN(CAS_K_RMSNORM, norm(c->final_norm, c->d_xn, nullptr, nullptr));
    GemmArgs gh{};
    gh.T = T;
    gh.N = f.vocab;
    gh.Kp = c->kp_d;
    gh.W = c->lm_head;
    gh.X = c->d_xn;
    gh.out = c->d_logits;
    gh.ldo = f.vocab;
    gh.gv = gv;
    gh.kmaj = 1;
    RUN(CAS_K_GEMM_HEAD, launch_gemm(et, et, EPI_STORE, gh, s));
#undef RUN
    return hipSuccess;
}

std::string graph_key(const cas_ctx* c, int T, const uint8_t* skip, int aq, int S) {
    std::string k = std::to_string(T) + ":" + std::to_string(aq) + ":" + std::to_string(S) + ":" +
                    (c->gemv ? "g:" : "m:") +
                    std::to_string(c->win_sink) + ":" + std::to_string(c->win_len) + ":";
    for (int l = 0; l < c->cfg.n_layers; ++l) k.push_back(skip && skip[l] ? '1' : '0');
    return k;
}

cas_status check_ready(cas_ctx* c, const uint8_t* skip) {
    if ((c->global_loaded & kGlobalMask) != kGlobalMask) return fail(c, CAS_ERR_STATE, "embedding, LM head or final norm not loaded");
    for (int l = 0; l < c->cfg.n_layers; ++l) {
        if (skip && skip[l]) continue;
        if ((c->layers[l].loaded & kLayerMask) != kLayerMask) {
            return fail(c, CAS_ERR_STATE, "layer " + std::to_string(l) + " has tensors not loaded");
        }
    }
    return CAS_OK;
}

cas_status do_forward(cas_ctx* c, const int32_t* tokens, const int32_t* parent, int n, int node_offset,
                      const uint8_t* skip, int aq, float* logits_host, bool allow_graph = true, int win_sink = 0,
                      int win_len = 0) {
    const cas_config& f = c->cfg;
    if (!tokens || !parent) return fail(c, CAS_ERR_ARG, "tokens and tree_parent must not be NULL");
    if (win_sink < 0 || win_len < 0) return fail(c, CAS_ERR_ARG, "attn_sink and attn_window must be >= 0");
    if (win_len == 0) win_sink = 0;
    if (n < 1) return fail(c, CAS_ERR_ARG, "n must be >= 1");
    if (node_offset < 0) return fail(c, CAS_ERR_ARG, "node_offset must be >= 0");
    if (aq < 0 || aq > 2) return fail(c, CAS_ERR_ARG, "act_quant must be 0, 1 or 2");
    if (node_offset != 0 && node_offset != c->n_nodes)
        return fail(c, CAS_ERR_TREE, "node_offset must be 0 (new round) or the round's node count " +
                                         std::to_string(c->n_nodes));
    if (node_offset + n > f.max_tree)
        return fail(c, CAS_ERR_CAPACITY, "round would exceed max_tree = " + std::to_string(f.max_tree));
    if (c->Lc + node_offset + n > f.max_ctx)
        return fail(c, CAS_ERR_CAPACITY, "committed + tree slots would exceed max_ctx = " + std::to_string(f.max_ctx));
    for (int i = 0; i < n; ++i)
        if (tokens[i] < 0 || tokens[i] >= f.vocab)
            return fail(c, CAS_ERR_ARG, "token " + std::to_string(tokens[i]) + " out of range");
    bool any_skip = false;
    if (skip) {
        for (int l = 0; l < f.n_layers; ++l) {
            if (skip[l] > 1) return fail(c, CAS_ERR_ARG, "skip_mask entries must be 0 or 1");
            any_skip |= skip[l] != 0;
        }
    }
    if (aq == 1 && !c->int8_ready) return fail(c, CAS_ERR_STATE, "act_quant 1 needs cas_build_int8 first");
    if (aq == 2 && !c->int4_ready) return fail(c, CAS_ERR_STATE, "act_quant 2 needs cas_build_int4 first");
    std::vector<int> depth;
    std::string why;
    if (!tree_depths(parent, node_offset, n, c->parent, &depth, &why)) return fail(c, CAS_ERR_TREE, why);
    cas_status st = check_ready(c, skip);
    if (st != CAS_OK) return st;

    // upload tokens, parents and the step parameters through a pinned buffer
    hipEvent_t ev = nullptr;
    unsigned char* buf = next_stage(c, &ev);
    if (!buf) return fail(c, CAS_ERR_DEVICE, "staging buffer wait failed");
    StepParams sp{c->Lc, node_offset, node_offset + n, c->chk_cap ? c->chk_cap : c->ctx_cap};
    memcpy(buf, &sp, sizeof sp);
    memcpy(buf + 16, tokens, sizeof(int32_t) * n);
    memcpy(buf + 16 + 4 * 128, parent, sizeof(int32_t) * n);
    HIPCHK(c, hipMemcpyAsync(c->d_sp, buf, sizeof sp, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipMemcpyAsync(c->d_rtok + node_offset, buf + 16, 4 * (size_t)n, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipMemcpyAsync(c->d_rpar + node_offset, buf + 16 + 4 * 128, 4 * (size_t)n, hipMemcpyHostToDevice,
                             c->stream));
    HIPCHK(c, hipEventRecord(ev, c->stream));

    // round state (the launch sequence reads the post-call node count)
    const int old_nodes = c->n_nodes;
    c->n_nodes = node_offset + n;
    c->win_sink = win_sink;
    c->win_len = win_len;
    const int S = attention_splits_win(c->Lc, c->n_nodes, win_sink, win_len);
    hipError_t e;
    if (c->graphs && !c->prof && allow_graph) {
        const std::string key = graph_key(c, n, skip, aq, S);
        auto it = c->gcache.find(key);
        if (it == c->gcache.end()) {
            if (c->gcache.size() >= kMaxGraphs) {
                HIPCHK(c, hipStreamSynchronize(c->stream));
                for (auto& kv : c->gcache) (void)hipGraphExecDestroy(kv.second);
                c->gcache.clear();
            }
            hipGraph_t gr = nullptr;
            e = hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal);
            if (e == hipSuccess) {
                hipError_t e2 = enqueue_forward(c, n, skip, aq);
                e = hipStreamEndCapture(c->stream, &gr);
                if (e2 != hipSuccess) e = e2;
            }
            hipGraphExec_t ex = nullptr;
            if (e == hipSuccess) e = hipGraphInstantiate(&ex, gr, nullptr, nullptr, 0);
            if (gr) (void)hipGraphDestroy(gr);
            if (e != hipSuccess) {
                c->n_nodes = old_nodes;
                return hip_fail(c, e, "graph capture of the forward");
            }
            it = c->gcache.emplace(key, ex).first;
        }
        e = hipGraphLaunch(it->second, c->stream);
    } else {
        e = enqueue_forward(c, n, skip, aq);
    }
    if (e != hipSuccess) {
        c->n_nodes = old_nodes;
        return hip_fail(c, e, "forward launch");
    }
    for (int i = 0; i < n; ++i) {
        c->parent[node_offset + i] = parent[i];
        c->token[node_offset + i] = tokens[i];
    }
    c->verified_n = (node_offset == 0 && !any_skip && !aq && win_len == 0) ? n : 0;
    c->logits_rows = n;
    if (logits_host) {
        HIPCHK(c, hipMemcpyAsync(logits_host, c->d_logits, sizeof(float) * (size_t)n * f.vocab, hipMemcpyDeviceToHost,
                                 c->stream));
        HIPCHK(c, hipStreamSynchronize(c->stream));
        return poll_checks(c);
    }
    return CAS_OK;
}

cas_status do_compact(cas_ctx* c, const int32_t* acc, int n_acc) {
    if (!acc) return fail(c, CAS_ERR_ARG, "accepted must not be NULL");
    if (c->verified_n == 0 || c->verified_n != c->n_nodes)
        return fail(c, CAS_ERR_STATE, "cas_kv_compact needs a verify call covering the whole round");
    if (n_acc < 1 || n_acc > c->n_nodes) return fail(c, CAS_ERR_ARG, "n_accepted out of range");
    if (acc[0] != 0) return fail(c, CAS_ERR_TREE, "accepted path must start at the root (node 0)");
    bool identity = true;
    for (int j = 1; j < n_acc; ++j) {
        if (acc[j] <= 0 || acc[j] >= c->n_nodes || c->parent[acc[j]] != acc[j - 1])
            return fail(c, CAS_ERR_TREE, "accepted[" + std::to_string(j) + "] is not a child of accepted[" +
                                             std::to_string(j - 1) + "]");
        identity &= acc[j] == j;
    }
    if (!identity) {
        hipEvent_t ev = nullptr;
        unsigned char* buf = next_stage(c, &ev);
        if (!buf) return fail(c, CAS_ERR_DEVICE, "staging buffer wait failed");
        memcpy(buf, acc, sizeof(int32_t) * n_acc);
        HIPCHK(c, hipMemcpyAsync(c->d_acc, buf, sizeof(int32_t) * n_acc, hipMemcpyHostToDevice, c->stream));
        HIPCHK(c, hipEventRecord(ev, c->stream));
        const cas_config& f = c->cfg;
        hipError_t e = timed(c, CAS_K_COMPACT, [&]() -> hipError_t {
            return launch_compact(c->et, c->kc, c->vt, f.n_layers, f.n_kv_heads, f.head_dim, c->ctx_cap, c->d_sp,
                                  c->d_acc, n_acc, c->d_chk, c->stream);
        });
        if (e != hipSuccess) return hip_fail(c, e, "kv compaction");
    }
    c->Lc += n_acc;
    c->n_nodes = 0;
    c->verified_n = 0;
    return CAS_OK;
}

void free_ctx(cas_ctx* c) {
    if (!c) return;
    if (c->stream) (void)hipStreamSynchronize(c->stream);
    for (auto& kv : c->gcache) (void)hipGraphExecDestroy(kv.second);
    for (auto& r : c->prec) {
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    for (auto e : c->ev_pool) (void)hipEventDestroy(e);
    for (auto& s : c->stage) {
        if (s.ev) (void)hipEventDestroy(s.ev);
        if (s.host) (void)hipHostFree(s.host);
    }
    if (c->h_result) (void)hipHostFree(c->h_result);
    if (c->h_topk) (void)hipHostFree(c->h_topk);
    for (void* p : c->allocs) (void)hipFree(p);
    if (c->own_stream && c->stream) (void)hipStreamDestroy(c->stream);
    delete c;
}

}  // namespace

extern "C" {

const char* cas_create_error(void) { return g_create_err.c_str(); }

const char* cas_last_error(const cas_ctx* c) { return c ? c->err.c_str() : "null context"; }

cas_status cas_tree_info(const int32_t* parent, int32_t n, int32_t* depth, uint64_t* anc) {
    if (!parent || n < 1 || n > 128) return CAS_ERR_ARG;
    std::vector<int> dep;
    std::string why;
    std::vector<int> none;
    if (!tree_depths(parent, 0, n, none, &dep, &why)) return CAS_ERR_TREE;
    for (int i = 0; i < n; ++i) {
        uint64_t a[2] = {0, 0};
        for (int x = i; x >= 0; x = parent[x]) a[x >> 6] |= 1ull << (x & 63);
        if (depth) depth[i] = dep[i];
        if (anc) {
            anc[2 * i] = a[0];
            anc[2 * i + 1] = a[1];
        }
    }
    return CAS_OK;
}

cas_status cas_create(const cas_config* cfg, int device, void* stream, cas_ctx** out) {
    if (!out) return CAS_ERR_ARG;
    *out = nullptr;
    g_create_err.clear();
    auto bad = [](cas_status s, const std::string& m) {
        g_create_err = m;
        return s;
    };
    if (!cfg) return bad(CAS_ERR_ARG, "cfg is NULL");
    const cas_config f = *cfg;
    if (f.n_layers < 1 || f.d_model < 16 || f.n_heads < 1 || f.n_kv_heads < 1 || f.vocab < 16 || f.ffn_dim < 16)
        return bad(CAS_ERR_ARG, "non-positive dimension");
    if (f.n_heads % f.n_kv_heads) return bad(CAS_ERR_ARG, "n_heads must be a multiple of n_kv_heads");
    if (f.head_dim != 64 && f.head_dim != 128) return bad(CAS_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (f.d_model % 16 || f.ffn_dim % 16 || f.vocab % 16)
        return bad(CAS_ERR_UNSUPPORTED, "d_model, ffn_dim and vocab must be multiples of 16");
    if (f.d_model > 8192 || f.ffn_dim > 65536) return bad(CAS_ERR_UNSUPPORTED, "d_model above 8192");
    if ((f.n_heads * f.head_dim) % (f.dtype == CAS_BF16 ? 128 : 64))
        return bad(CAS_ERR_UNSUPPORTED, "n_heads * head_dim must be a multiple of 128 (bf16) or 64 (fp32)");
    if (f.dtype != CAS_F32 && f.dtype != CAS_BF16) return bad(CAS_ERR_ARG, "dtype");
    if (f.max_tree < 1 || f.max_tree > 128) return bad(CAS_ERR_UNSUPPORTED, "max_tree must be in [1, 128]");
    if (f.max_ctx < f.max_tree) return bad(CAS_ERR_ARG, "max_ctx must be >= max_tree");
    if (f.dtype == CAS_F32 && f.max_ctx > 4096 - 128) return bad(CAS_ERR_UNSUPPORTED, "fp32 models need max_ctx <= 3968");
    if (f.max_ctx > 16384 - 128) return bad(CAS_ERR_UNSUPPORTED, "max_ctx must be <= 16256");
    if (!(f.rms_eps > 0.f) || !(f.rope_theta > 1.f)) return bad(CAS_ERR_ARG, "rms_eps / rope_theta");

    hipError_t e = hipSetDevice(device);
    if (e != hipSuccess) return bad(CAS_ERR_DEVICE, std::string("hipSetDevice: ") + hipGetErrorString(e));
    cas_ctx* c = new cas_ctx();
    c->cfg = f;
    c->dev = device;
    c->et = f.dtype == CAS_BF16 ? ET_BF16 : ET_F32;
    c->es = f.dtype == CAS_BF16 ? 2 : 4;
    c->qrows = f.n_heads * f.head_dim;
    c->krows = f.n_kv_heads * f.head_dim;
    c->qkv_rows = c->qrows + 2 * c->krows;
    c->ctx_cap = ((f.max_ctx + 127) / 128) * 128;
    c->layers.resize(f.n_layers);
    c->parent.assign(f.max_tree, -1);
    c->token.assign(f.max_tree, 0);
    auto cleanup = [&](cas_status s, const std::string& m) {
        free_ctx(c);
        return bad(s, m);
    };
#define ALLOC(p, bytes)                                                              \
    do {                                                                             \
        if (dalloc(c, &(p), (bytes)) != hipSuccess)                                  \
            return cleanup(CAS_ERR_OOM, std::string("hipMalloc failed for ") + #p); \
    } while (0)
    if (stream) {
        c->stream = (hipStream_t)stream;
    } else {
        if (hipStreamCreate(&c->stream) != hipSuccess) return cleanup(CAS_ERR_DEVICE, "hipStreamCreate");
        c->own_stream = true;
    }
    const size_t es = c->es, d = f.d_model, ffn = f.ffn_dim, T = f.max_tree;
    ALLOC(c->embed, (size_t)f.vocab * d * es);
    c->kp_d = pad_k(f.d_model, c->et);
    c->kp_q = pad_k(c->qrows, c->et);
    c->kp_f = pad_k(f.ffn_dim, c->et);
    c->kq_d = pad_k(f.d_model, ET_I8);
    c->kq_q = pad_k(c->qrows, ET_I8);
    c->kq_f = pad_k(f.ffn_dim, ET_I8);
    ALLOC(c->lm_head, (size_t)f.vocab * c->kp_d * es);
    ALLOC(c->final_norm, d * 4);
    for (auto& w : c->layers) {
        ALLOC(w.wqkv, (size_t)c->qkv_rows * c->kp_d * es);
        ALLOC(w.wo, d * c->kp_q * es);
        ALLOC(w.wgu, 2 * ffn * c->kp_d * es);
        ALLOC(w.wd, d * c->kp_f * es);
        ALLOC(w.attn_norm, d * 4);
        ALLOC(w.ffn_norm, d * 4);
    }
    const size_t kv = (size_t)f.n_layers * f.n_kv_heads * c->ctx_cap * f.head_dim * es;
    ALLOC(c->kc, kv);
    ALLOC(c->vt, kv);
    if (hipMemset(c->kc, 0, kv) != hipSuccess || hipMemset(c->vt, 0, kv) != hipSuccess)
        return cleanup(CAS_ERR_DEVICE, "hipMemset of the KV cache");
    const int half = f.head_dim / 2;
    ALLOC(c->rope_cos, (size_t)c->ctx_cap * half * 4);
    ALLOC(c->rope_sin, (size_t)c->ctx_cap * half * 4);
    {
        std::vector<float> cs((size_t)c->ctx_cap * half), sn((size_t)c->ctx_cap * half);
        for (int p = 0; p < c->ctx_cap; ++p)
            for (int i = 0; i < half; ++i) {
                const double inv = std::pow((double)f.rope_theta, -2.0 * i / (double)f.head_dim);
                const double ang = (double)p * inv;
                cs[(size_t)p * half + i] = (float)std::cos(ang);
                sn[(size_t)p * half + i] = (float)std::sin(ang);
            }
        if (hipMemcpy(c->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
            hipMemcpy(c->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
            return cleanup(CAS_ERR_DEVICE, "RoPE table upload");
    }
    ALLOC(c->d_rtok, T * 4);
    ALLOC(c->d_rpar, T * 4);
    ALLOC(c->d_sp, sizeof(StepParams));
    ALLOC(c->d_chk, 16);
    if (hipMemset(c->d_chk, 0, 16) != hipSuccess) return cleanup(CAS_ERR_DEVICE, "hipMemset of the check word");
    ALLOC(c->d_row_pos, T * 4);
    ALLOC(c->d_row_slot, T * 4);
    ALLOC(c->d_row_anc, T * 16);
    ALLOC(c->d_h, T * d * 4);
    // tiled activations hold 128 rows (8 column tiles) of the padded width
    const size_t kpmax = std::max(std::max(c->kp_d, c->kp_q), c->kp_f);
    const size_t kqmax = std::max(std::max(c->kq_d, c->kq_q), c->kq_f);
    ALLOC(c->d_xn, 128 * kpmax * es);
    ALLOC(c->d_xq, 128 * kqmax);
    ALLOC(c->d_xs, T * 4);
    ALLOC(c->d_q, T * c->qrows * es);
    ALLOC(c->d_ao, 128 * (size_t)c->kp_q * es);
    ALLOC(c->d_sw, 128 * (size_t)c->kp_f * es);
    ALLOC(c->d_logits, T * (size_t)f.vocab * 4);
    c->part_bytes = attention_work_bytes(c->ctx_cap, (int)T, f.n_heads, f.head_dim);
    ALLOC(c->d_part, c->part_bytes);
    ALLOC(c->d_gpart, sizeof(float) * 8 * (size_t)f.max_tree * f.d_model);
    ALLOC(c->d_gbuf, T * 8 * 3 * 4);  // per row: 8 argmax parts of (index, value, NaN flag)
    ALLOC(c->d_result, (T + 4) * 4);
    ALLOC(c->d_topk, T * (16 + 16 + 1) * 4);
    ALLOC(c->d_acc, (T + 1) * 4);
    if (hipMemset(c->d_rtok, 0, T * 4) != hipSuccess || hipMemset(c->d_rpar, 0xff, T * 4) != hipSuccess)
        return cleanup(CAS_ERR_DEVICE, "hipMemset of the round arrays");
    if (hipHostMalloc((void**)&c->h_result, (T + 4) * 4, hipHostMallocDefault) != hipSuccess)
        return cleanup(CAS_ERR_OOM, "hipHostMalloc");
    if (hipHostMalloc((void**)&c->h_topk, T * (16 + 16 + 1) * 4, hipHostMallocDefault) != hipSuccess)
        return cleanup(CAS_ERR_OOM, "hipHostMalloc");
    for (auto& s : c->stage) {
        if (hipHostMalloc((void**)&s.host, kStageBytes, hipHostMallocDefault) != hipSuccess)
            return cleanup(CAS_ERR_OOM, "hipHostMalloc");
        if (hipEventCreateWithFlags(&s.ev, hipEventDisableTiming) != hipSuccess)
            return cleanup(CAS_ERR_DEVICE, "hipEventCreate");
    }
#undef ALLOC
    if (hipDeviceSynchronize() != hipSuccess) return cleanup(CAS_ERR_DEVICE, "device sync after create");
    *out = c;
    return CAS_OK;
}

void cas_destroy(cas_ctx* c) { free_ctx(c); }

cas_status cas_load_tensor(cas_ctx* c, int32_t kind, int32_t layer, const void* host, size_t bytes) {
    if (!c) return CAS_ERR_ARG;
    if (!host) return fail(c, CAS_ERR_ARG, "host pointer is NULL");
    if (kind < CAS_T_EMBED || kind > CAS_T_W_DOWN) return fail(c, CAS_ERR_ARG, "unknown tensor kind");
    const cas_config& f = c->cfg;
    if (!is_global(kind) && (layer < 0 || layer >= f.n_layers)) return fail(c, CAS_ERR_ARG, "layer out of range");
    const size_t el = is_norm(kind) ? 4 : c->es;
    const size_t want = tensor_elems(c, kind) * el;
    if (bytes != want)
        return fail(c, CAS_ERR_ARG, "tensor size " + std::to_string(bytes) + " bytes, expected " + std::to_string(want));
    LayerW* w = is_global(kind) ? nullptr : &c->layers[layer];
    hipError_t e = hipSuccess;
    if (is_norm(kind) || kind == CAS_T_EMBED) {
        void* dst = kind == CAS_T_EMBED ? c->embed
                    : kind == CAS_T_FINAL_NORM ? (void*)c->final_norm
                    : kind == CAS_T_ATTN_NORM ? (void*)w->attn_norm : (void*)w->ffn_norm;
        e = hipMemcpy(dst, host, bytes, hipMemcpyHostToDevice);
    } else {
        // projections and the LM head: stage row-major on the device, then tile
        if (c->stage_dev_bytes < bytes) {
            if (c->stage_dev) {
                (void)hipFree(c->stage_dev);
                for (auto& p : c->allocs)
                    if (p == c->stage_dev) p = nullptr;
                c->stage_dev = nullptr;
                c->stage_dev_bytes = 0;
            }
            if (dalloc(c, &c->stage_dev, bytes) != hipSuccess) return fail(c, CAS_ERR_OOM, "hipMalloc of the load staging buffer");
            c->stage_dev_bytes = bytes;
        }
        HIPCHK(c, hipStreamSynchronize(c->stream));
        HIPCHK(c, hipMemcpy(c->stage_dev, host, bytes, hipMemcpyHostToDevice));
        const int d = f.d_model, hd = f.head_dim;
        void* dst = nullptr;
        int rows = 0, K = d, row0 = 0, mode = 0;
        switch (kind) {
        case CAS_T_LM_HEAD: dst = c->lm_head; rows = f.vocab; break;
        case CAS_T_WQ: dst = w->wqkv; rows = c->qrows; mode = 1; break;
        case CAS_T_WK: dst = w->wqkv; rows = c->krows; row0 = c->qrows; mode = 1; break;
        case CAS_T_WV: dst = w->wqkv; rows = c->krows; row0 = c->qrows + c->krows; break;
        case CAS_T_WO: dst = w->wo; rows = d; K = c->qrows; break;
        case CAS_T_W_GATE: dst = w->wgu; rows = f.ffn_dim; mode = 2; break;
        case CAS_T_W_UP: dst = w->wgu; rows = f.ffn_dim; row0 = 1; mode = 2; break;
        case CAS_T_W_DOWN: dst = w->wd; rows = d; K = f.ffn_dim; break;
        }
        // the gate/up and LM head matrices are stored in the K-major block order
        const int kt = (kind == CAS_T_W_GATE || kind == CAS_T_W_UP) && kProjKMajor[2] ? 2 * f.ffn_dim / 16
                       : kind == CAS_T_LM_HEAD ? f.vocab / 16 : 0;
        e = launch_tile_weight(c->et, c->stage_dev, rows, K, dst, row0, mode, hd, c->stream, kt);
        if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    }
    if (e != hipSuccess) return hip_fail(c, e, "weight upload");
    if (w) {
        w->loaded |= 1u << kind;
    } else {
        c->global_loaded |= 1u << kind;
    }
    c->int8_ready = false;
    c->int4_ready = false;
    return CAS_OK;
}

cas_status cas_build_int4(cas_ctx* c) {
    if (!c) return CAS_ERR_ARG;
    cas_status st = check_ready(c, nullptr);
    if (st != CAS_OK) return st;
    const cas_config& f = c->cfg;
    const size_t d = f.d_model, ffn = f.ffn_dim;
    for (auto& w : c->layers) {
        const void* src[4] = {w.wqkv, w.wo, w.wgu, w.wd};
        const size_t N[4] = {(size_t)c->qkv_rows, d, 2 * ffn, d};
        const size_t K[4] = {d, (size_t)c->qrows, d, ffn};
        const size_t KQ[4] = {(size_t)c->kq_d, (size_t)c->kq_q, (size_t)c->kq_d, (size_t)c->kq_f};
        for (int i = 0; i < 4; ++i) {
            if (!w.q4[i]) {
                if (dalloc(c, &w.q4[i], N[i] * KQ[i] / 2) != hipSuccess || dalloc(c, &w.s4[i], N[i] * 4) != hipSuccess)
                    return fail(c, CAS_ERR_OOM, "hipMalloc of the int4 weight copy");
            }
            hipError_t e = launch_quant_weight_i4(c->et, src[i], (int)N[i], (int)K[i], w.q4[i], w.s4[i], c->stream,
                                                  kProjKMajor[i], 0);
            if (e != hipSuccess) return hip_fail(c, e, "int4 weight quantisation");
        }
    }
    HIPCHK(c, hipStreamSynchronize(c->stream));
    c->int4_ready = true;
    return CAS_OK;
}

cas_status cas_build_int8(cas_ctx* c) {
    if (!c) return CAS_ERR_ARG;
    cas_status st = check_ready(c, nullptr);
    if (st != CAS_OK) return st;
    const cas_config& f = c->cfg;
    const size_t d = f.d_model, ffn = f.ffn_dim;
    for (auto& w : c->layers) {
        const void* src[4] = {w.wqkv, w.wo, w.wgu, w.wd};
        const size_t N[4] = {(size_t)c->qkv_rows, d, 2 * ffn, d};
        const size_t K[4] = {d, (size_t)c->qrows, d, ffn};
        const size_t KQ[4] = {(size_t)c->kq_d, (size_t)c->kq_q, (size_t)c->kq_d, (size_t)c->kq_f};
        for (int i = 0; i < 4; ++i) {
            if (!w.q8[i]) {
                if (dalloc(c, &w.q8[i], N[i] * KQ[i]) != hipSuccess || dalloc(c, &w.s8[i], N[i] * 4) != hipSuccess)
                    return fail(c, CAS_ERR_OOM, "hipMalloc of the int8 weight copy");
            }
            hipError_t e = launch_quant_weight(c->et, src[i], (int)N[i], (int)K[i], w.q8[i], w.s8[i], c->stream,
                                               kProjKMajor[i], kProjKMajor[i]);
            if (e != hipSuccess) return hip_fail(c, e, "int8 weight quantisation");
        }
    }
    HIPCHK(c, hipStreamSynchronize(c->stream));
    c->int8_ready = true;
    return CAS_OK;
}

cas_status cas_forward(cas_ctx* c, const int32_t* tokens, const int32_t* parent, int32_t n, int32_t node_offset,
                       const uint8_t* skip, int32_t aq, float* logits_host) {
    if (!c) return CAS_ERR_ARG;
    return do_forward(c, tokens, parent, n, node_offset, skip, aq, logits_host);
}

cas_status cas_forward_draft(cas_ctx* c, const int32_t* tokens, const int32_t* parent, int32_t n,
                             int32_t node_offset, const cas_draft_opts* o, float* logits_host) {
    if (!c) return CAS_ERR_ARG;
    if (!o) return do_forward(c, tokens, parent, n, node_offset, nullptr, 0, logits_host);
    return do_forward(c, tokens, parent, n, node_offset, o->skip_mask, o->act_quant, logits_host, true, o->attn_sink,
                      o->attn_window);
}

cas_status cas_prefill(cas_ctx* c, const int32_t* tokens, int32_t n) {
    if (!c) return CAS_ERR_ARG;
    if (!tokens || n < 1) return fail(c, CAS_ERR_ARG, "prefill needs tokens and n >= 1");
    if (c->Lc + n > c->cfg.max_ctx) return fail(c, CAS_ERR_CAPACITY, "prefill would exceed max_ctx");
    for (int i = 0; i < n; ++i)
        if (tokens[i] < 0 || tokens[i] >= c->cfg.vocab) return fail(c, CAS_ERR_ARG, "token out of range");
    std::vector<int32_t> par(c->cfg.max_tree), acc(c->cfg.max_tree);
    for (int i = 0; i < c->cfg.max_tree; ++i) {
        par[i] = i - 1;
        acc[i] = i;
    }
    int done = 0;
    while (done < n) {
        const int m = std::min(c->cfg.max_tree, n - done);
        // one-off shapes: launched directly rather than captured
        cas_status st = do_forward(c, tokens + done, par.data(), m, 0, nullptr, 0, nullptr, false);
        if (st != CAS_OK) return st;
        st = do_compact(c, acc.data(), m);
        if (st != CAS_OK) return st;
        done += m;
    }
    return CAS_OK;
}

// Row-major [Hkv][n][hd] host data <-> one layer's cache, through a device staging buffer.
static cas_status kv_transfer(cas_ctx* c, int32_t layer, void* k, void* v, int32_t n, bool to_cache) {
    const cas_config& f = c->cfg;
    if (!k || !v) return fail(c, CAS_ERR_ARG, "k and v must not be NULL");
    if (layer < 0 || layer >= f.n_layers) return fail(c, CAS_ERR_ARG, "layer out of range");
    if (n < 0 || n > f.max_ctx) return fail(c, CAS_ERR_CAPACITY, "n exceeds max_ctx");
    if (n == 0) return CAS_OK;
    const size_t bytes = (size_t)f.n_kv_heads * n * f.head_dim * c->es;
    const size_t kv_layer = (size_t)f.n_kv_heads * c->ctx_cap * f.head_dim * c->es;
    void* tmp = nullptr;
    HIPCHK(c, hipStreamSynchronize(c->stream));
    HIPCHK(c, hipMalloc(&tmp, 2 * bytes));
    char* tk = (char*)tmp;
    char* tv = tk + bytes;
    hipError_t e = hipSuccess;
    if (to_cache) {
        e = hipMemcpy(tk, k, bytes, hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(tv, v, bytes, hipMemcpyHostToDevice);
    }
    if (e == hipSuccess)
        e = launch_kv_convert(c->et, (char*)c->kc + kv_layer * layer, (char*)c->vt + kv_layer * layer, tk, tv,
                              f.n_kv_heads, n, f.head_dim, c->ctx_cap, to_cache ? 1 : 0, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess && !to_cache) {
        e = hipMemcpy(k, tk, bytes, hipMemcpyDeviceToHost);
        if (e == hipSuccess) e = hipMemcpy(v, tv, bytes, hipMemcpyDeviceToHost);
    }
    (void)hipFree(tmp);
    if (e != hipSuccess) return hip_fail(c, e, "kv transfer");
    return CAS_OK;
}

cas_status cas_kv_load(cas_ctx* c, int32_t layer, const void* k, const void* v, int32_t n) {
    if (!c) return CAS_ERR_ARG;
    return kv_transfer(c, layer, (void*)k, (void*)v, n, true);
}

cas_status cas_kv_read(cas_ctx* c, int32_t layer, void* k, void* v, int32_t n) {
    if (!c) return CAS_ERR_ARG;
    return kv_transfer(c, layer, k, v, n, false);
}

cas_status cas_set_committed(cas_ctx* c, int32_t n) {
    if (!c) return CAS_ERR_ARG;
    if (n < 0 || n > c->cfg.max_ctx) return fail(c, CAS_ERR_CAPACITY, "committed length out of range");
    c->Lc = n;
    c->n_nodes = 0;
    c->verified_n = 0;
    return CAS_OK;
}

cas_status cas_committed_len(const cas_ctx* c, int32_t* n) {
    if (!c || !n) return CAS_ERR_ARG;
    *n = c->Lc;
    return CAS_OK;
}

cas_status cas_logits_device(const cas_ctx* c, const float** p, int32_t* n) {
    if (!c || !p || !n) return CAS_ERR_ARG;
    *p = c->d_logits;
    *n = c->logits_rows;
    return CAS_OK;
}

cas_status cas_accept_tree(cas_ctx* c, int32_t greedy, int32_t* accepted, int32_t* n_accepted, int32_t* bonus) {
    if (!c) return CAS_ERR_ARG;
    if (greedy != 1) return fail(c, CAS_ERR_UNSUPPORTED, "only greedy acceptance is implemented");
    if (!accepted || !n_accepted || !bonus) return fail(c, CAS_ERR_ARG, "output pointers must not be NULL");
    if (c->verified_n == 0 || c->verified_n != c->n_nodes)
        return fail(c, CAS_ERR_STATE, "cas_accept_tree needs a verify call covering the whole round");
    const int T = c->n_nodes;
    hipError_t e = timed(c, CAS_K_ACCEPT, [&]() -> hipError_t {
        return launch_accept(c->d_logits, T, c->cfg.vocab, c->d_rtok, c->d_rpar, c->d_gbuf, c->d_result, c->d_chk,
                             c->stream);
    });
    if (e != hipSuccess) return hip_fail(c, e, "acceptance launch");
    HIPCHK(c, hipMemcpyAsync(c->h_result, c->d_result, sizeof(int) * (size_t)(T + 3), hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    cas_status cst = poll_checks(c);
    if (cst != CAS_OK) return cst;
    if (c->h_result[2]) return fail(c, CAS_ERR_DEVICE, "NaN in the verify logits");
    const int na = c->h_result[0];
    if (na < 1 || na > T) return fail(c, CAS_ERR_DEVICE, "acceptance returned an invalid path length");
    for (int j = 0; j < na; ++j) accepted[j] = c->h_result[3 + j];
    *n_accepted = na;
    *bonus = c->h_result[1];
    return CAS_OK;
}

cas_status cas_topk(cas_ctx* c, int32_t n, int32_t K, int32_t* ids, float* probs) {
    if (!c) return CAS_ERR_ARG;
    if (K < 1 || K > 16) return fail(c, CAS_ERR_ARG, "K must be in [1, 16]");
    if (!ids || !probs) return fail(c, CAS_ERR_ARG, "output pointers must not be NULL");
    if (c->logits_rows < 1) return fail(c, CAS_ERR_STATE, "cas_topk needs a forward first");
    if (n != c->logits_rows)
        return fail(c, CAS_ERR_ARG, "n must equal the last forward's row count " + std::to_string(c->logits_rows));
    const int cap = c->cfg.max_tree;
    int* d_ids = c->d_topk;
    float* d_p = (float*)(c->d_topk + (size_t)cap * 16);
    int* d_flag = c->d_topk + (size_t)cap * 32;
    HIPCHK(c, hipMemsetAsync(d_flag, 0, sizeof(int) * (size_t)n, c->stream));
    hipError_t e = timed(c, CAS_K_TOPK, [&]() -> hipError_t {
        return launch_topk(c->d_logits, n, c->cfg.vocab, K, d_ids, d_p, d_flag, c->stream);
    });
    if (e != hipSuccess) return hip_fail(c, e, "top-K launch");
    int* h_ids = c->h_topk;
    float* h_p = (float*)(c->h_topk + (size_t)cap * 16);
    int* h_flag = c->h_topk + (size_t)cap * 32;
    HIPCHK(c, hipMemcpyAsync(h_ids, d_ids, sizeof(int) * (size_t)n * K, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipMemcpyAsync(h_p, d_p, sizeof(float) * (size_t)n * K, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipMemcpyAsync(h_flag, d_flag, sizeof(int) * (size_t)n, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    cas_status cst = poll_checks(c);
    if (cst != CAS_OK) return cst;
    for (int i = 0; i < n; ++i)
        if (h_flag[i]) return fail(c, CAS_ERR_DEVICE, "NaN in the logits of row " + std::to_string(i));
    memcpy(ids, h_ids, sizeof(int) * (size_t)n * K);
    memcpy(probs, h_p, sizeof(float) * (size_t)n * K);
    return CAS_OK;
}

cas_status cas_kv_compact(cas_ctx* c, const int32_t* accepted, int32_t n_accepted) {
    if (!c) return CAS_ERR_ARG;
    return do_compact(c, accepted, n_accepted);
}

cas_status cas_set_graphs(cas_ctx* c, int32_t enable) {
    if (!c) return CAS_ERR_ARG;
    c->graphs = enable != 0;
    return CAS_OK;
}

cas_status cas_set_gemv(cas_ctx* c, int32_t enable) {
    if (!c) return CAS_ERR_ARG;
    c->gemv = enable != 0;
    return CAS_OK;
}

cas_status cas_profile(cas_ctx* c, int32_t enable) {
    if (!c) return CAS_ERR_ARG;
    c->prof = enable != 0;
    return CAS_OK;
}

cas_status cas_profile_read(cas_ctx* c, double* ms, int32_t* launches, int32_t reset) {
    if (!c) return CAS_ERR_ARG;
    HIPCHK(c, hipStreamSynchronize(c->stream));
    for (auto& r : c->prec) {
        float t = 0.f;
        HIPCHK(c, hipEventElapsedTime(&t, r.a, r.b));
        c->pms[r.cls] += t;
        c->pn[r.cls] += 1;
        c->ev_pool.push_back(r.a);
        c->ev_pool.push_back(r.b);
    }
    c->prec.clear();
    for (int i = 0; i < CAS_K_COUNT; ++i) {
        if (ms) ms[i] = c->pms[i];
        if (launches) launches[i] = c->pn[i];
    }
    if (reset) {
        for (int i = 0; i < CAS_K_COUNT; ++i) {
            c->pms[i] = 0;
            c->pn[i] = 0;
        }
    }
    return CAS_OK;
}

cas_status cas_sync(cas_ctx* c) {
    if (!c) return CAS_ERR_ARG;
    HIPCHK(c, hipStreamSynchronize(c->stream));
    return poll_checks(c);
}

int32_t cas_debug_build(void) { return kDeviceChecks ? 1 : 0; }

cas_status cas_debug_check(cas_ctx* c, int32_t* code) {
    if (!c || !code) return CAS_ERR_ARG;
    HIPCHK(c, hipStreamSynchronize(c->stream));
    *code = 0;
    if constexpr (kDeviceChecks) {
        HIPCHK(c, hipMemcpy(code, c->d_chk, sizeof(int32_t), hipMemcpyDeviceToHost));
        if (*code) HIPCHK(c, hipMemset(c->d_chk, 0, sizeof(int32_t)));
    }
    return CAS_OK;
}

cas_status cas_debug_limit_slots(cas_ctx* c, int32_t cap) {
    if (!c) return CAS_ERR_ARG;
    if (!kDeviceChecks) return fail(c, CAS_ERR_UNSUPPORTED, "device checks are compiled only into CAS_DEBUG builds");
    if (cap < 0 || cap > c->cfg.max_ctx) return fail(c, CAS_ERR_ARG, "cap must be in [0, max_ctx]");
    c->chk_cap = cap;
    return CAS_OK;
}

// ---------------------------------------------------------------- kernel-level entry points

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

size_t cas_op_gemm_work_bytes(int32_t wtype, int32_t N, int32_t K, int32_t T) {
    if (wtype < CAS_W_F32 || wtype > CAS_W_I4 || N < 1 || K < 1 || T < 1 || T > 128) return 0;
    if (wtype == CAS_W_I4) {  // packed weights, int8 activations
        const size_t Kp = pad_k(K, ET_I8);
        return align256((size_t)N * Kp / 2) + align256((size_t)16 * col_tiles(T) * Kp);
    }
    const size_t Kp = pad_k(K, wtype), eb = frag_elem_bytes(wtype);
    return align256((size_t)N * Kp * eb) + align256((size_t)16 * col_tiles(T) * Kp * eb);
}

cas_status cas_op_gemm(int32_t wtype, const void* W, const void* X, int32_t N, int32_t K, int32_t T, const float* xs,
                       const float* ws, int32_t epi, void* out, int32_t ldo, void* work, size_t work_bytes,
                       void* stream) {
    if (!W || !X || !out || !work) return CAS_ERR_ARG;
    if (wtype < CAS_W_F32 || wtype > CAS_W_I4) return CAS_ERR_ARG;
    if (N < 16 || N % 16 || K < 16 || K % 16 || T < 1 || T > 128 || ldo < N) return CAS_ERR_UNSUPPORTED;
    if (epi != CAS_EPI_STORE && epi != CAS_EPI_RESID && epi != CAS_EPI_RAW_I32) return CAS_ERR_ARG;
    const bool integer = wtype == CAS_W_I8 || wtype == CAS_W_I4;
    if (epi == CAS_EPI_RAW_I32 && !integer) return CAS_ERR_UNSUPPORTED;
    if (integer && epi != CAS_EPI_RAW_I32 && (!xs || !ws)) return CAS_ERR_ARG;
    if (work_bytes < cas_op_gemm_work_bytes(wtype, N, K, T)) return CAS_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    const int at = wtype == CAS_W_I4 ? (int)ET_I8 : wtype;  // int4 weights take int8 activations
    const size_t Kp = pad_k(K, at), eb = frag_elem_bytes(at);
    const size_t wbytes = wtype == CAS_W_I4 ? (size_t)N * Kp / 2 : (size_t)N * Kp * eb;
    void* wt = work;
    void* xt = (char*)work + align256(wbytes);
    GemmArgs a{};
    a.W = wt;
    a.X = xt;
    a.N = N;
    a.Kp = (int)Kp;
    a.T = T;
    a.xs = xs;
    a.ws = ws;
    a.out = out;
    a.ldo = ldo;
    a.gv = T == 1 ? 1 : 0;
    const int ep = epi == CAS_EPI_STORE ? EPI_STORE : epi == CAS_EPI_RESID ? EPI_RESID : EPI_RAW;
    hipError_t e = wtype == CAS_W_I4 ? launch_pack_weight_i4((const int8_t*)W, N, K, (uint8_t*)wt, s)
                                     : launch_tile_weight(wtype, W, N, K, wt, 0, 0, 0, s);
    if (e == hipSuccess) e = launch_tile_act(at, X, T, K, xt, s);
    if (e == hipSuccess) e = launch_gemm(wtype, ET_F32, ep, a, s);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

cas_status cas_op_quant_rows(int32_t atype, const void* x, int32_t T, int32_t K, int8_t* q, float* s, void* stream) {
    if (!x || !q || !s || T < 1 || K < 1) return CAS_ERR_ARG;
    if (atype != CAS_W_F32 && atype != CAS_W_BF16) return CAS_ERR_ARG;
    hipError_t e = launch_quant_rows(atype, x, T, K, q, s, 0, 127, (hipStream_t)stream);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}
cas_status cas_op_quant_rows_q(int32_t atype, const void* x, int32_t T, int32_t K, int32_t qmax, int8_t* q, float* s,
                               void* stream) {
    if (!x || !q || !s || T < 1 || K < 1 || (qmax != 127 && qmax != 7)) return CAS_ERR_ARG;
    if (atype != CAS_W_F32 && atype != CAS_W_BF16) return CAS_ERR_ARG;
    hipError_t e = launch_quant_rows(atype, x, T, K, q, s, 0, qmax, (hipStream_t)stream);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

size_t cas_op_quant_weight_work_bytes(int32_t wtype, int32_t N, int32_t K) {
    if ((wtype != CAS_W_F32 && wtype != CAS_W_BF16) || N < 1 || K < 1) return 0;
    return align256((size_t)N * pad_k(K, wtype) * frag_elem_bytes(wtype)) + align256((size_t)N * pad_k(K, ET_I8));
}

cas_status cas_op_quant_weight(int32_t wtype, const void* W, int32_t N, int32_t K, int8_t* q, float* s, void* work,
                               size_t work_bytes, void* stream) {
    if (!W || !q || !s || !work || N < 16 || N % 16 || K < 16 || K % 16) return CAS_ERR_ARG;
    if (wtype != CAS_W_F32 && wtype != CAS_W_BF16) return CAS_ERR_ARG;
    if (work_bytes < cas_op_quant_weight_work_bytes(wtype, N, K)) return CAS_ERR_ARG;
    hipStream_t st = (hipStream_t)stream;
    void* wt = work;
    int8_t* qt = (int8_t*)((char*)work + align256((size_t)N * pad_k(K, wtype) * frag_elem_bytes(wtype)));
    hipError_t e = launch_tile_weight(wtype, W, N, K, wt, 0, 0, 0, st);
    if (e == hipSuccess) e = launch_quant_weight(wtype, wt, N, K, qt, s, st);
    if (e == hipSuccess) e = launch_untile_weight_i8(qt, N, K, q, st);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}
cas_status cas_op_quant_weight_i4(int32_t wtype, const void* W, int32_t N, int32_t K, int8_t* q, float* s,
                                  void* work, size_t work_bytes, void* stream) {
    if (!W || !q || !s || !work || N < 16 || N % 16 || K < 16 || K % 16) return CAS_ERR_ARG;
    if (wtype != CAS_W_F32 && wtype != CAS_W_BF16) return CAS_ERR_ARG;
    if (work_bytes < cas_op_quant_weight_work_bytes(wtype, N, K)) return CAS_ERR_ARG;
    hipStream_t st = (hipStream_t)stream;
    void* wt = work;
    uint8_t* qt = (uint8_t*)((char*)work + align256((size_t)N * pad_k(K, wtype) * frag_elem_bytes(wtype)));
    hipError_t e = launch_tile_weight(wtype, W, N, K, wt, 0, 0, 0, st);
    if (e == hipSuccess) e = launch_quant_weight_i4(wtype, wt, N, K, qt, s, st);
    if (e == hipSuccess) e = launch_untile_weight_i4(qt, N, K, q, st);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

size_t cas_op_attention_work_bytes(int32_t Lc, int32_t n_tree, int32_t T, int32_t H, int32_t hd, int32_t Hkv,
                                   int32_t ctx_cap) {
    return 256 + 2 * align256((size_t)Hkv * ctx_cap * hd * 2) +
           attention_work_bytes(Lc + n_tree, T, H, hd);
}

// The attention op on a scratch region `work` of at least
// cas_op_attention_work_bytes(...) bytes: step parameters | K cache | V
// cache | split partials, every byte the kernels read written first.
static cas_status attention_op(const void* q, const void* k, const void* v, int32_t ctx_cap, int32_t Lc,
                               int32_t n_tree, int32_t T, int32_t H, int32_t Hkv, int32_t hd, const uint64_t* anc,
                               void* out, void* work, hipStream_t s) {
    StepParams sp{Lc, 0, n_tree, ctx_cap};
    char* w = (char*)work;
    StepParams* dsp = (StepParams*)w;
    char* kcache = w + 256;
    char* vcache = kcache + align256((size_t)Hkv * ctx_cap * hd * 2);
    float* part = (float*)(vcache + align256((size_t)Hkv * ctx_cap * hd * 2));
    if (hipMemcpyAsync(dsp, &sp, sizeof sp, hipMemcpyHostToDevice, s) != hipSuccess) return CAS_ERR_DEVICE;
    hipError_t e = launch_kv_convert(ET_BF16, kcache, vcache, k, v, Hkv, ctx_cap, hd, ctx_cap, 1, s);
    AttnArgs a{};
    a.q = q;
    a.kc = kcache;
    a.vt = vcache;
    a.anc = anc;
    a.sp = dsp;
    a.Lc_host = Lc;
    a.n_tree_host = n_tree;
    a.out = out;
    a.out_tiled = 0;
    const int S = attention_splits(Lc + n_tree);
    a.part_o = part;
    a.part_ml = a.part_o + (size_t)S * H * T * hd;
    a.T = T;
    a.H = H;
    a.Hkv = Hkv;
    a.hd = hd;
    a.ctx_cap = ctx_cap;
    if (e == hipSuccess) e = launch_attention(ET_BF16, a, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // sp lives on the caller's stack
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

static cas_status attention_op_check(const void* q, const void* k, const void* v, int32_t ctx_cap, int32_t Lc,
                                     int32_t n_tree, int32_t T, int32_t H, int32_t Hkv, int32_t hd,
                                     const uint64_t* anc, const void* out) {
    if (!q || !k || !v || !anc || !out) return CAS_ERR_ARG;
    if (hd != 64 && hd != 128) return CAS_ERR_UNSUPPORTED;
    if (T < 1 || T > 128 || n_tree < 1 || n_tree > 128 || Lc < 0 || Hkv < 1 || H < 1 || H % Hkv) return CAS_ERR_ARG;
    if (ctx_cap % 32 || Lc + n_tree > ctx_cap) return CAS_ERR_ARG;
    return CAS_OK;
}

cas_status cas_op_attention(const void* q, const void* k, const void* v, int32_t ctx_cap, int32_t Lc, int32_t n_tree,
                            int32_t T, int32_t H, int32_t Hkv, int32_t hd, const uint64_t* anc, void* out, void* work,
                            size_t work_bytes, void* stream) {
    const cas_status st = attention_op_check(q, k, v, ctx_cap, Lc, n_tree, T, H, Hkv, hd, anc, out);
    if (st != CAS_OK) return st;
    if (!work || work_bytes < cas_op_attention_work_bytes(Lc, n_tree, T, H, hd, Hkv, ctx_cap)) return CAS_ERR_ARG;
    return attention_op(q, k, v, ctx_cap, Lc, n_tree, T, H, Hkv, hd, anc, out, work, (hipStream_t)stream);
}

// ---- the allocation-free attention entry point
//
// Its scratch is this file-scope device array: every GPU the library runs on
// holds its own copy (at its own address) until the process ends, and every
// call on that GPU shares it.  In host code the array's name is only a
// host-side stand-in, so the kernels get the device address from
// hipGetSymbolAddress, taken once per device (with that device current) and
// kept in scratch_dev.
static constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)64 << 20;
static constexpr int NOALLOC_MAX_DEVICES = 64;
static __device__ __attribute__((aligned(256))) unsigned char scratch[NOALLOC_SCRATCH_BYTES];
static std::mutex scratch_mu;
static void* scratch_dev[NOALLOC_MAX_DEVICES];

static cas_status scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= NOALLOC_MAX_DEVICES) return CAS_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_dev[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CAS_ERR_DEVICE;
        scratch_dev[dev] = p;
    }
    *out = scratch_dev[dev];
    return CAS_OK;
}

size_t cas_op_attention_noalloc_max_bytes(void) { return NOALLOC_SCRATCH_BYTES; }

cas_status cas_op_attention_noalloc(const void* q, const void* k, const void* v, int32_t ctx_cap, int32_t Lc,
                                    int32_t n_tree, int32_t T, int32_t H, int32_t Hkv, int32_t hd,
                                    const uint64_t* anc, void* out, void* stream) {
    const cas_status st = attention_op_check(q, k, v, ctx_cap, Lc, n_tree, T, H, Hkv, hd, anc, out);
    if (st != CAS_OK) return st;
    if (cas_op_attention_work_bytes(Lc, n_tree, T, H, hd, Hkv, ctx_cap) > NOALLOC_SCRATCH_BYTES)
        return CAS_ERR_CAPACITY;
    void* work = nullptr;
    const cas_status sa = scratch_address(&work);
    if (sa != CAS_OK) return sa;
    return attention_op(q, k, v, ctx_cap, Lc, n_tree, T, H, Hkv, hd, anc, out, work, (hipStream_t)stream);
}

// ---- the fused quantisers of the forward, one kernel each

static size_t norm_tiled_bytes(int32_t atype, int32_t T, int32_t d, int32_t qmax) {
    const int et = qmax ? (int)ET_I8 : atype;
    return (size_t)16 * col_tiles(T) * pad_k(d, et) * frag_elem_bytes(et);
}

size_t cas_op_rmsnorm_work_bytes(int32_t atype, int32_t T, int32_t d, int32_t qmax) {
    if ((atype != CAS_W_F32 && atype != CAS_W_BF16) || T < 1 || T > 128 || d < 16 || d % 16 ||
        (qmax != 0 && qmax != 127 && qmax != 7))
        return 0;
    return align256(norm_tiled_bytes(atype, T, d, qmax));
}

cas_status cas_op_rmsnorm(int32_t atype, float* h, const float* gain, int32_t T, int32_t d, float eps,
                          const float* parts, int32_t nparts, int32_t qmax, void* out, int8_t* q, float* qs,
                          void* work, size_t work_bytes, void* stream) {
    if (!h || !gain || !work || (nparts > 0 && !parts) || nparts < 0 || nparts > 8) return CAS_ERR_ARG;
    if (atype != CAS_W_F32 && atype != CAS_W_BF16) return CAS_ERR_ARG;
    if (qmax != 0 && qmax != 127 && qmax != 7) return CAS_ERR_ARG;
    if (qmax ? (!q || !qs) : !out) return CAS_ERR_ARG;
    if (T < 1 || T > 128 || d < 16 || d % 16 || d > 16384 || !(eps >= 0.f)) return CAS_ERR_UNSUPPORTED;
    if (work_bytes < cas_op_rmsnorm_work_bytes(atype, T, d, qmax)) return CAS_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = launch_rmsnorm(atype, h, gain, T, d, eps, qmax ? nullptr : work, qmax ? (int8_t*)work : nullptr,
                                  qs, parts, nparts, (size_t)T * d, qmax ? qmax : 127, s);
    if (e == hipSuccess) e = launch_untile_act(qmax ? (int)ET_I8 : atype, work, T, d, qmax ? (void*)q : out, s);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

size_t cas_op_attn_merge_work_bytes(int32_t T, int32_t n_heads, int32_t head_dim, int32_t qmax) {
    if (T < 1 || T > 128 || n_heads < 1 || (head_dim != 64 && head_dim != 128)) return 0;
    if (qmax == 0) return 256;
    if (qmax != 127 && qmax != 7) return 0;
    return align256((size_t)16 * col_tiles(T) * pad_k(n_heads * head_dim, ET_I8));
}

cas_status cas_op_attn_merge(const float* part_o, const float* part_ml, int32_t S, int32_t T, int32_t n_heads,
                             int32_t head_dim, int32_t qmax, uint16_t* out, int8_t* q, float* qs, void* work,
                             size_t work_bytes, void* stream) {
    if (!part_o || !part_ml || !work || S < 1 || S > 64) return CAS_ERR_ARG;
    if (qmax != 0 && qmax != 127 && qmax != 7) return CAS_ERR_ARG;
    if (qmax ? (!q || !qs) : !out) return CAS_ERR_ARG;
    if (T < 1 || T > 128 || n_heads < 1 || (head_dim != 64 && head_dim != 128)) return CAS_ERR_UNSUPPORTED;
    const size_t need = cas_op_attn_merge_work_bytes(T, n_heads, head_dim, qmax);
    if (!need) return CAS_ERR_UNSUPPORTED;
    if (work_bytes < need) return CAS_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    AttnArgs a{};
    a.part_o = (float*)part_o;
    a.part_ml = (float*)part_ml;
    a.T = T;
    a.H = n_heads;
    a.hd = head_dim;
    a.out = out;
    a.out_tiled = 0;
    a.qout = qmax ? (int8_t*)work : nullptr;
    a.qscale = qmax ? qs : nullptr;
    a.qmax = qmax;
    hipError_t e = launch_attn_merge(a, S, s);
    if (e == hipSuccess && qmax) e = launch_untile_act(ET_I8, work, T, n_heads * head_dim, q, s);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

int32_t cas_op_gemm_qx_splits(int32_t wtype, int32_t N, int32_t K, int32_t T) {
    if ((wtype != CAS_W_I8 && wtype != CAS_W_I4) || N < 64 || K < 16 || K % 16 || T < 1) return 0;
    const int Kp = pad_k(K, ET_I8);
    const int ks = gemm_parts_count(wtype, N, Kp, T);
    return gemm_qx_ok(wtype, N, Kp, T, ks) ? ks : 0;
}

size_t cas_op_gemm_qx_work_bytes(int32_t wtype, int32_t N, int32_t K, int32_t T) {
    if (!cas_op_gemm_qx_splits(wtype, N, K, T)) return 0;
    const size_t Kp = pad_k(K, ET_I8);
    const size_t wbytes = wtype == CAS_W_I4 ? (size_t)N * Kp / 2 : (size_t)N * Kp;
    return align256(wbytes) + align256((size_t)16 * col_tiles(T) * pad_k(K, ET_BF16) * 2);
}

cas_status cas_op_gemm_qx(int32_t wtype, const int8_t* W, const float* ws, const uint16_t* x, int32_t N, int32_t K,
                          int32_t T, int32_t qmax, float* parts, void* work, size_t work_bytes, void* stream) {
    if (!W || !ws || !x || !parts || !work) return CAS_ERR_ARG;
    if (wtype != CAS_W_I8 && wtype != CAS_W_I4) return CAS_ERR_ARG;
    if (qmax != (wtype == CAS_W_I8 ? 127 : 7)) return CAS_ERR_ARG;
    const int ks = cas_op_gemm_qx_splits(wtype, N, K, T);
    if (!ks || N % 16) return CAS_ERR_UNSUPPORTED;
    if (work_bytes < cas_op_gemm_qx_work_bytes(wtype, N, K, T)) return CAS_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    const size_t Kp = pad_k(K, ET_I8);
    const size_t wbytes = wtype == CAS_W_I4 ? (size_t)N * Kp / 2 : (size_t)N * Kp;
    void* wt = work;
    void* xt = (char*)work + align256(wbytes);
    GemmArgs a{};
    a.W = wt;
    a.X = xt;
    a.N = N;
    a.Kp = (int)Kp;
    a.T = T;
    a.ws = ws;
    a.out = parts;
    a.ldo = N;
    a.ksplit = ks;
    a.part_stride = (size_t)T * N;
    a.qx = qmax;
    a.xk = K;
    hipError_t e = wtype == CAS_W_I4 ? launch_pack_weight_i4(W, N, K, (uint8_t*)wt, s)
                                     : launch_tile_weight(ET_I8, W, N, K, wt, 0, 0, 0, s);
    if (e == hipSuccess) e = launch_tile_act(ET_BF16, x, T, K, xt, s);
    if (e == hipSuccess) e = launch_gemm_parts(wtype, a, s);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

cas_status cas_op_copy(void* dst, const void* src, size_t bytes, void* stream) {
    if (!dst || !src || bytes % 16) return CAS_ERR_ARG;
    hipError_t e = launch_copy(dst, src, bytes, (hipStream_t)stream);
    return e == hipSuccess ? CAS_OK : CAS_ERR_DEVICE;
}

}  // extern "C"
