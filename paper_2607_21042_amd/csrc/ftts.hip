// C ABI entry points of libftts: argument validation, workspace carving and the
// order of kernel launches for prefill, for one decode step and for one guided
// Euler step of the flow-matching DiT.  Every check happens before the first
// enqueue, so a rejected call has no side effects.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>

#include "decode_entry.hpp"
#include "ftts_internal.hpp"

using namespace ftts;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char* where) {
    return fail(FTTS_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
size_t round256(size_t n) { return (n + 255) & ~size_t(255); }
int act_bytes(const ftts_config& c) { return c.wdtype == FTTS_F32 ? 4 : 2; }

int check_config(const ftts_config* c) {
    if (!c) return fail(FTTS_E_INVALID_ARG, "config is NULL");
    if (c->wdtype < FTTS_F32 || c->wdtype > FTTS_W4A16) return fail(FTTS_E_DTYPE, "unknown wdtype %d", c->wdtype);
    if (c->n_layer < 1) return fail(FTTS_E_SHAPE, "n_layer must be >= 1");
    if (c->d_head != kHeadDim) return fail(FTTS_E_UNSUPPORTED, "d_head must be 64 (got %d)", c->d_head);
    if (c->page_size != kPage) return fail(FTTS_E_UNSUPPORTED, "page_size must be 64 (got %d)", c->page_size);
    if (c->n_head < 1 || c->n_head * kHeadDim != c->d_model)
        return fail(FTTS_E_SHAPE, "n_head * d_head must equal d_model");
    if (c->d_model % 128 || c->d_model > 4096) return fail(FTTS_E_SHAPE, "d_model must be a multiple of 128, <= 4096");
    if (c->d_ff < 128 || c->d_ff % 128 || c->d_ff > 16384)
        return fail(FTTS_E_SHAPE, "d_ff must be a multiple of 128, <= 16384");
    if (c->vocab < 2 || c->vocab > 16384) return fail(FTTS_E_SHAPE, "vocab must be in [2, 16384]");
    if (c->n_pos < 1) return fail(FTTS_E_SHAPE, "n_pos must be >= 1");
    if (c->wdtype == FTTS_W4A16 && c->group_size != 128)
        return fail(FTTS_E_UNSUPPORTED, "W4A16 group_size must be 128 (got %d)", c->group_size);
    if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps)) return fail(FTTS_E_RANGE, "ln_eps must be finite and > 0");
    const int head_wt = c->wdtype == FTTS_F32 ? FTTS_F32 : FTTS_BF16;
    if (!gemv_supported(c->wdtype, c->d_model, true) || !gemv_supported(c->wdtype, c->d_model, false) ||
        !gemv_supported(c->wdtype, c->d_ff, false) || !gemv_supported(head_wt, c->d_model, true))
        return fail(FTTS_E_UNSUPPORTED, "no decode tiling for d_model=%d d_ff=%d in this weight mode", c->d_model,
                    c->d_ff);
    return FTTS_OK;
}

int check_ptr(const void* p, const char* name) {
    if (!p) return fail(FTTS_E_INVALID_ARG, "%s is NULL", name);
    if (!aligned16(p)) return fail(FTTS_E_ALIGN, "%s is not 16-byte aligned", name);
    return FTTS_OK;
}

#define TRY(expr)                       \
    do {                                \
        int rc_ = (expr);               \
        if (rc_ != FTTS_OK) return rc_; \
    } while (0)

int check_linear(const ftts_linear& l, int wdtype, const char* name) {
    char buf[64];
    snprintf(buf, sizeof buf, "%s.w", name);
    TRY(check_ptr(l.w, buf));
    snprintf(buf, sizeof buf, "%s.bias", name);
    TRY(check_ptr(l.bias, buf));
    if (wdtype == FTTS_W8A16 || wdtype == FTTS_W4A16) {
        snprintf(buf, sizeof buf, "%s.scale", name);
        TRY(check_ptr(l.scale, buf));
    }
    if (wdtype == FTTS_W4A16) {
        snprintf(buf, sizeof buf, "%s.zero", name);
        TRY(check_ptr(l.zero, buf));
    }
    return FTTS_OK;
}

int check_weights(const ftts_weights* w) {
    if (!w) return fail(FTTS_E_INVALID_ARG, "weights is NULL");
    TRY(check_config(&w->cfg));
    TRY(check_ptr(w->tok_emb, "tok_emb"));
    TRY(check_ptr(w->pos_emb, "pos_emb"));
    TRY(check_ptr(w->lnf_g, "lnf_g"));
    TRY(check_ptr(w->lnf_b, "lnf_b"));
    TRY(check_ptr(w->head.w, "head.w"));
    TRY(check_ptr(w->head.bias, "head.bias"));
    if (!w->layers) return fail(FTTS_E_INVALID_ARG, "layers is NULL");
    for (int l = 0; l < w->cfg.n_layer; ++l) {
        const ftts_layer& L = w->layers[l];
        TRY(check_ptr(L.ln1_g, "ln1_g"));
        TRY(check_ptr(L.ln1_b, "ln1_b"));
        TRY(check_ptr(L.ln2_g, "ln2_g"));
        TRY(check_ptr(L.ln2_b, "ln2_b"));
        TRY(check_linear(L.qkv, w->cfg.wdtype, "qkv"));
        TRY(check_linear(L.out, w->cfg.wdtype, "out"));
        TRY(check_linear(L.fc1, w->cfg.wdtype, "fc1"));
        TRY(check_linear(L.fc2, w->cfg.wdtype, "fc2"));
    }
    return FTTS_OK;
}

int check_kv(const ftts_page_table* pt, const ftts_kv_pool* kv, bool need_seq_lens) {
    if (!pt) return fail(FTTS_E_INVALID_ARG, "page table is NULL");
    if (!kv) return fail(FTTS_E_INVALID_ARG, "kv pool is NULL");
    TRY(check_ptr(kv->base, "kv.base"));
    if (!pt->block_table) return fail(FTTS_E_INVALID_ARG, "block_table is NULL");
    if (need_seq_lens && !pt->seq_lens) return fail(FTTS_E_INVALID_ARG, "seq_lens is NULL");
    if (pt->max_pages < 1 || pt->max_pages > kMaxPages)
        return fail(FTTS_E_SHAPE, "max_pages must be in [1, %d]", kMaxPages);
    if (kv->n_pages < 1) return fail(FTTS_E_SHAPE, "n_pages must be >= 1");
    return FTTS_OK;
}

int check_sampling(const ftts_sampling* s, int V, const float* uniforms) {
    if (!s) return fail(FTTS_E_INVALID_ARG, "sampling is NULL");
    if (s->top_k < 1 || s->top_k > FTTS_MAX_TOP_K || s->top_k > V)
        return fail(FTTS_E_RANGE, "top_k must be in [1, min(%d, vocab)]", FTTS_MAX_TOP_K);
    if (s->top_k > 1) {
        if (!(s->temperature > 0.f) || !std::isfinite(s->temperature))
            return fail(FTTS_E_RANGE, "temperature must be finite and > 0");
        if (!(s->top_p > 0.f && s->top_p <= 1.f)) return fail(FTTS_E_RANGE, "top_p must be in (0, 1]");
        if (!uniforms) return fail(FTTS_E_INVALID_ARG, "uniforms is NULL but top_k > 1");
    }
    return FTTS_OK;
}

// Workspace regions (all 256-byte aligned).  Decode and prefill never run at the
// same time on one workspace, so their regions overlap.
struct DecodeWs {
    float *x, *qkv, *o, *h;
    int32_t* active;
    float2* stats;              // batched path: residual tile statistics [d/32][B]
    uint16_t *o16, *h16;        // batched path: bf16 inputs of the MFMA linears
    float* part;                // batched path: split-K partials
    uint32_t* count;            // batched path: arrival counters
};
struct PrefillWs {
    float* x;        // [M][d] fp32 residual
    void* a;         // [M][d] LayerNorm output, later the attention output
    void* qkv;       // [M][3d]
    void* h;         // [M][d_ff]
    float* xlast;    // [B][d]
    int32_t* active; // [B] all ones (head GEMV reads no flags; kept for symmetry)
    float* part;     // split-K partial tiles of the GEMMs (16-bit modes, short prefixes)
    uint32_t* count; // their per-tile arrival counters
};

// The persistent decode step's control words and exchange buffers sit at the
// start of every workspace, at a fixed size, so that decode and prefill calls
// with different batch sizes agree on where they are.
struct MegaWs {
    uint32_t* ctl;
    uint64_t *x, *qkv, *o, *h, *arg;
};

size_t mega_bytes(MegaWs* out, char* base) {
    size_t off = 0;
    auto take = [&](size_t n) { size_t o = off; off += round256(n); return base ? base + o : nullptr; };
    using namespace ftts::mega;
    char* ctl = take(256);
    char* x = take((size_t)BM * D * 8);
    char* qkv = take((size_t)BM * 3 * D * 8);
    char* o = take((size_t)BM * (D / 2) * 8);  // bf16 pairs
    char* h = take((size_t)BM * (FF / 2) * 8);
    char* arg = take((size_t)G * BM * 2 * 8);
    if (out)
        *out = MegaWs{(uint32_t*)ctl, (uint64_t*)x, (uint64_t*)qkv, (uint64_t*)o, (uint64_t*)h, (uint64_t*)arg};
    return off;
}

// Arrival counters of the batched path: one per 32-feature tile of the widest linear.
int bgemm_counters(const ftts_config& c) {
    const int nmax = std::max(std::max(3 * c.d_model, c.d_ff), c.vocab);
    return (nmax + 31) / 32;
}

// The batched path's largest split-K partial buffer.  The
// linears after a LayerNorm (QKV, FC1, head) normalise their input themselves.
size_t bgemm_part_floats(const ftts_config& c, int B) {
    const int d = c.d_model, F = c.d_ff, V = c.vocab, rows = B < 32 ? B : 32;
    const int NK[5][4] = {{3 * d, d, c.wdtype, 1}, {d, d, c.wdtype, 0}, {F, d, c.wdtype, 1}, {d, F, c.wdtype, 0},
                          {V, d, FTTS_BF16, 1}};
    size_t m = 0;
    for (const auto& t : NK) {
        if (c.wdtype == FTTS_F32) break;
        const int S = bgemm_splits(t[2], t[0], t[1], t[3] != 0);
        const size_t n = S > 1 ? (size_t)S * rows * t[0] : 0;
        m = n > m ? n : m;
    }
    return m;
}

size_t decode_bytes(const ftts_config& c, int B, DecodeWs* out, char* base) {
    size_t off = mega_bytes(nullptr, nullptr);
    auto take = [&](size_t n) { size_t o = off; off += round256(n); return base ? base + o : nullptr; };
    char* x = take((size_t)B * c.d_model * 4);
    char* qkv = take((size_t)B * 3 * c.d_model * 4);
    char* o = take((size_t)B * c.d_model * 4);
    char* h = take((size_t)B * c.d_ff * 4);
    char* act = take((size_t)B * 4);
    const bool batched = B >= batched_min(c.wdtype) && c.wdtype != FTTS_F32 && c.d_model % 64 == 0 &&
                         bgemm_supported(c.wdtype, c.d_model, true) && bgemm_supported(c.wdtype, c.d_model, false) &&
                         bgemm_supported(c.wdtype, c.d_ff, false) && bgemm_supported(FTTS_BF16, c.d_model, true);
    char *stats = nullptr, *o16 = nullptr, *h16 = nullptr, *part = nullptr, *count = nullptr;
    if (batched) {
        stats = take((size_t)(c.d_model / kStatTile) * B * sizeof(float2));
        o16 = take((size_t)B * c.d_model * 2);
        h16 = take((size_t)B * c.d_ff * 2);
        part = take(bgemm_part_floats(c, B) * 4);
        count = take((size_t)bgemm_counters(c) * 4);
    }
    if (out)
        *out = DecodeWs{(float*)x, (float*)qkv, (float*)o, (float*)h, (int32_t*)act, (float2*)stats, (uint16_t*)o16,
                        (uint16_t*)h16, (float*)part, (uint32_t*)count};
    return off;
}

// Split-K scratch of the prefill GEMMs for any row count up to M: the largest
// S * rows * N partial buffer and the largest tile count (the split depends on
// the row count, and a smaller call may split where a larger one does not).
void gemm_scratch(const ftts_config& c, int M, size_t* part_floats, size_t* counters) {
    size_t pf = 0, cn = 0;
    if (c.wdtype != FTTS_F32 && M > 0) {
        const int d = c.d_model, F = c.d_ff;
        const int NK[4][2] = {{3 * d, d}, {d, d}, {F, d}, {d, F}};
        for (int step = 64;; step += 64) {
            const int rows = std::min(step, M);
            bool split = false;
            for (const auto& t : NK) {
                const GemmPlan p = gemm_plan(rows, t[0], t[1]);
                if (p.splits > 1) {
                    split = true;
                    // partial tiles are whole (64 mt) x 128 tiles, past the matrix edges too
                    pf = std::max(pf, (size_t)p.splits * p.tiles_m * p.tiles_n * (64 * p.mt) * 128);
                    cn = std::max(cn, (size_t)p.tiles_m * p.tiles_n);
                }
            }
            if (rows >= M || !split) break;  // more rows only add tiles
        }
    }
    *part_floats = pf;
    *counters = cn;
}

size_t prefill_bytes(const ftts_config& c, int B, int M, PrefillWs* out, char* base) {
    const size_t e = act_bytes(c);
    size_t off = mega_bytes(nullptr, nullptr);
    auto take = [&](size_t n) { size_t o = off; off += round256(n); return base ? base + o : nullptr; };
    char* x = take((size_t)M * c.d_model * 4);
    char* a = take((size_t)M * c.d_model * e);
    char* qkv = take((size_t)M * 3 * c.d_model * e);
    char* h = take((size_t)M * c.d_ff * e);
    char* xl = take((size_t)B * c.d_model * 4);
    char* act = take((size_t)B * 4);
    size_t pf, cn;
    gemm_scratch(c, M, &pf, &cn);
    char* part = pf ? take(pf * 4) : nullptr;
    char* count = cn ? take(cn * 4) : nullptr;
    if (out) *out = PrefillWs{(float*)x, a, qkv, h, (float*)xl, (int32_t*)act, (float*)part, (uint32_t*)count};
    return off;
}

int g_decode_path = 0;  // 0 automatic, 1 kernel per phase, 2 persistent step

// Per-layer pointers of one kind, if they sit at a fixed stride.
template <typename F>
bool stride_of(const ftts_weights* w, F get, Strided* out) {
    const char* p0 = reinterpret_cast<const char*>(get(w->layers[0]));
    const long long st = w->cfg.n_layer > 1 ? reinterpret_cast<const char*>(get(w->layers[1])) - p0 : 0;
    for (int l = 0; l < w->cfg.n_layer; ++l)
        if (reinterpret_cast<const char*>(get(w->layers[l])) != p0 + (long long)l * st) return false;
    *out = Strided{p0, st};
    return true;
}

int device_cus() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    if (!cache[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cache[dev] = n;
    }
    return cache[dev];
}

// Fills the persistent step's arguments when the model and call qualify.
bool mega_args(const ftts_weights* w, int B, mega::Args* a) {
    const ftts_config& c = w->cfg;
    using namespace ftts::mega;
    if (c.wdtype == FTTS_F32 || c.d_model != D || c.d_ff != FF || c.n_head != NH) return false;
    // LM-head rows per group must fit the two 50 KB LDS weight buffers (40 rows of 1280 bf16).
    if (B < 1 || B > BM || c.n_layer > 50 || c.vocab < G || c.vocab > G * 40) return false;
    if (device_cus() != G) return false;
    // every one of the 256 workgroups must be resident at once (one per CU)
    if (decode_mega_blocks_per_cu(c.wdtype, B) < 1) return false;
    bool ok = true;
    ok &= stride_of(w, [](const ftts_layer& L) { return L.ln1_g; }, &a->ln1_g);
    ok &= stride_of(w, [](const ftts_layer& L) { return L.ln1_b; }, &a->ln1_b);
    ok &= stride_of(w, [](const ftts_layer& L) { return L.ln2_g; }, &a->ln2_g);
    ok &= stride_of(w, [](const ftts_layer& L) { return L.ln2_b; }, &a->ln2_b);
#define FTTS_LIN(NAME)                                                                          \
    ok &= stride_of(w, [](const ftts_layer& L) { return L.NAME.w; }, &a->NAME##_w);             \
    ok &= stride_of(w, [](const ftts_layer& L) { return L.NAME.scale; }, &a->NAME##_s);         \
    ok &= stride_of(w, [](const ftts_layer& L) { return L.NAME.zero; }, &a->NAME##_z);          \
    ok &= stride_of(w, [](const ftts_layer& L) { return L.NAME.bias; }, &a->NAME##_b);
    FTTS_LIN(qkv) FTTS_LIN(out) FTTS_LIN(fc1) FTTS_LIN(fc2)
#undef FTTS_LIN
    if (!ok) return false;
    // Weight shares are copied to LDS 16 bytes at a time; LayerNorm gains are read 16 bytes at a time.
    auto al16 = [](const Strided& t) { return ((uintptr_t)t.p % 16) == 0 && (t.s % 16) == 0; };
    ok &= al16(a->qkv_w) && al16(a->out_w) && al16(a->fc1_w) && al16(a->fc2_w);
    ok &= al16(a->ln1_g) && al16(a->ln1_b) && al16(a->ln2_g) && al16(a->ln2_b);
    ok &= (uintptr_t)w->head.w % 16 == 0 && (uintptr_t)w->lnf_g % 16 == 0 && (uintptr_t)w->lnf_b % 16 == 0;
    if (!ok) return false;
    a->n_layer = c.n_layer;
    a->V = c.vocab;
    a->n_pos = c.n_pos;
    a->B = B;
    a->eps = c.ln_eps;
    a->tok_emb = w->tok_emb;
    a->pos_emb = w->pos_emb;
    a->lnf_g = w->lnf_g;
    a->lnf_b = w->lnf_b;
    a->head_w = w->head.w;
    a->head_b = w->head.bias;
    return true;
}

GemvArgs gemv_args(const ftts_linear& L, int N, int K, int B, const float* act, float* out, int out_stride) {
    GemvArgs a{};
    a.w = L.w;
    a.scale = reinterpret_cast<const uint16_t*>(L.scale);
    a.zero = reinterpret_cast<const uint16_t*>(L.zero);
    a.bias = L.bias;
    a.N = N;
    a.K = K;
    a.B = B;
    a.act = act;
    a.out = out;
    a.out_stride = out_stride;
    return a;
}

}  // namespace

// Decode step for batches of batched_min() or more (16-bit and quantised weights):
// the MFMA linears, with each LayerNorm folded into the linear that reads it (the
// residual updates leave per-tile row statistics behind).  Attention writes bf16
// for the out-projection and FC1's GELU output is bf16 for FC2.
int decode_batched(const ftts_weights* w, int B, const DecodeWs& W, const KvAppend& kva, AttnDecodeArgs at,
                   float* logits_out, float* hidden_out, int32_t* sampled_out, const float* uniforms,
                   const ftts_sampling* samp, hipStream_t st) {
    const ftts_config& c = w->cfg;
    const int d = c.d_model, F = c.d_ff, V = c.vocab;
    hipError_t e;
    auto lin = [&](const ftts_linear& L, int N, int K, const void* act, float* out, void* out16, int stride) {
        BgemmArgs g{};
        g.w = L.w;
        g.scale = reinterpret_cast<const uint16_t*>(L.scale);
        g.zero = reinterpret_cast<const uint16_t*>(L.zero);
        g.bias = L.bias;
        g.N = N;
        g.K = K;
        g.B = B;
        g.act = act;
        g.out = out;
        g.out_bf16 = out16;
        g.out_stride = stride;
        g.part = W.part;
        g.count = W.count;
        g.stats_ld = B;
        return g;
    };
    auto normed = [&](BgemmArgs g, const void* ln_g, const void* ln_b) {
        g.ln_x = W.x;
        g.ln_g = ln_g;
        g.ln_b = ln_b;
        g.ln_eps = c.ln_eps;
        g.ln_stats = W.stats;
        return g;
    };
    at.o_bf16 = W.o16;
    for (int l = 0; l < c.n_layer; ++l) {
        const ftts_layer& L = w->layers[l];
        BgemmArgs g = normed(lin(L.qkv, 3 * d, d, nullptr, W.qkv, nullptr, 3 * d), L.ln1_g, L.ln1_b);
        g.kv = kva;
        g.kv.layer = l;
        if ((e = launch_bgemm(c.wdtype, EPI_QKV, g, st)) != hipSuccess) return hip_fail(e, "ln1 + qkv");
        at.layer = l;
        if ((e = launch_attn_decode(c.wdtype, at, B, st)) != hipSuccess) return hip_fail(e, "attention");
        g = lin(L.out, d, d, W.o16, W.x, nullptr, d);
        g.stats_out = W.stats;
        if ((e = launch_bgemm(c.wdtype, EPI_RESID, g, st)) != hipSuccess) return hip_fail(e, "out-proj");
        g = normed(lin(L.fc1, F, d, nullptr, nullptr, W.h16, F), L.ln2_g, L.ln2_b);
        if ((e = launch_bgemm(c.wdtype, EPI_GELU, g, st)) != hipSuccess) return hip_fail(e, "ln2 + fc1");
        g = lin(L.fc2, d, F, W.h16, W.x, nullptr, d);
        g.stats_out = W.stats;
        if ((e = launch_bgemm(c.wdtype, EPI_RESID, g, st)) != hipSuccess) return hip_fail(e, "fc2");
    }
    BgemmArgs g = normed(lin(w->head, V, d, nullptr, logits_out, nullptr, V), w->lnf_g, w->lnf_b);
    g.hidden = hidden_out;
    if ((e = launch_bgemm(c.wdtype, EPI_STORE, g, st)) != hipSuccess) return hip_fail(e, "ln_f + lm head");
    if ((e = launch_sample(logits_out, B, V, *samp, uniforms, W.active, sampled_out, st)) != hipSuccess)
        return hip_fail(e, "sampler");
    return FTTS_OK;
}

extern "C" {

const char* ftts_last_error(void) { return g_err; }

int ftts_set_decode_path(int32_t path) {
    if (path < 0 || path > 2) return fail(FTTS_E_RANGE, "decode path must be 0, 1 or 2");
    g_decode_path = path;
    return FTTS_OK;
}

int ftts_decode_path(const ftts_weights* w, int32_t batch) {
    if (!w) return fail(FTTS_E_INVALID_ARG, "weights is NULL");
    int e = check_config(&w->cfg);
    if (e != FTTS_OK) return e;
    if (batch < 1 || batch > FTTS_MAX_BATCH) return fail(FTTS_E_RANGE, "batch must be in [1, %d]", FTTS_MAX_BATCH);
    if (g_decode_path == 1) return 1;
    mega::Args ma{};
    const bool ok = mega_args(w, batch, &ma);
    if (g_decode_path == 2 && !ok)
        return fail(FTTS_E_UNSUPPORTED, "the persistent decode step does not take this model/batch/device");
    return ok ? 2 : 1;
}

int ftts_check_workspace(const void* ws, size_t ws_bytes, void* stream) {
    if (!ws) return fail(FTTS_E_INVALID_ARG, "workspace is NULL");
    if (ws_bytes < mega_bytes(nullptr, nullptr)) return fail(FTTS_E_WORKSPACE, "workspace too small");
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "check_workspace sync");
    uint32_t ctl[2] = {0, 0};
    e = hipMemcpy(ctl, ws, sizeof ctl, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "check_workspace copy");
    if (ctl[1]) return fail(FTTS_E_HIP, "a persistent decode step timed out waiting for its input (abort word set)");
    return FTTS_OK;
}

const char* ftts_version(void) { return "ftts 0.1.0 gfx950"; }

size_t ftts_workspace_bytes(const ftts_config* cfg, int32_t max_batch, int32_t max_rows) {
    if (check_config(cfg) != FTTS_OK) return 0;
    if (max_batch < 1 || max_batch > FTTS_MAX_BATCH || max_rows < 0) {
        fail(FTTS_E_RANGE, "max_batch must be in [1, %d] and max_rows >= 0", FTTS_MAX_BATCH);
        return 0;
    }
    const size_t d = decode_bytes(*cfg, max_batch, nullptr, nullptr);
    const size_t p = prefill_bytes(*cfg, max_batch, max_rows, nullptr, nullptr);
    return d > p ? d : p;
}

int ftts_quantize_weights(int32_t wdtype, const float* w, int64_t N, int64_t K, int32_t group_size, void* codes,
                          uint16_t* scales, uint16_t* zeros, void* stream) {
    if (wdtype != FTTS_W8A16 && wdtype != FTTS_W4A16)
        return fail(FTTS_E_DTYPE, "quantize: wdtype must be FTTS_W8A16 or FTTS_W4A16");
    if (!w || !codes || !scales) return fail(FTTS_E_INVALID_ARG, "quantize: NULL pointer");
    if (N < 1 || K < 1 || N > 65535LL * 32768LL) return fail(FTTS_E_SHAPE, "quantize: bad N or K");
    if (wdtype == FTTS_W8A16) {
        if (K % 16) return fail(FTTS_E_SHAPE, "quantize: K must be a multiple of 16 for W8A16");
        if (N > 0x7FFFFFFF) return fail(FTTS_E_SHAPE, "quantize: N too large");
    } else {
        if (group_size != 128) return fail(FTTS_E_UNSUPPORTED, "quantize: group_size must be 128");
        if (K % group_size) return fail(FTTS_E_SHAPE, "quantize: K must be a multiple of group_size");
        if (!zeros) return fail(FTTS_E_INVALID_ARG, "quantize: zeros is NULL for W4A16");
        if (N > 65535) return fail(FTTS_E_SHAPE, "quantize: N must be <= 65535 for W4A16");
        if (reinterpret_cast<uintptr_t>(codes) & 3u) return fail(FTTS_E_ALIGN, "quantize: codes not 4-byte aligned");
    }
    if (reinterpret_cast<uintptr_t>(w) & 3u) return fail(FTTS_E_ALIGN, "quantize: w not 4-byte aligned");
    (void)hipGetLastError();
    hipError_t e = launch_quantize(wdtype, w, N, K, group_size, codes, scales, zeros, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "quantize launch");
    return FTTS_OK;
}

int ftts_sample(const float* logits, int32_t B, int32_t V, const ftts_sampling* samp, const float* uniforms,
                int32_t* sampled_out, void* stream) {
    if (!logits || !sampled_out) return fail(FTTS_E_INVALID_ARG, "sample: NULL pointer");
    if (B < 1 || B > 65535) return fail(FTTS_E_SHAPE, "sample: B must be in [1, 65535]");
    if (V < 1 || V > 16384) return fail(FTTS_E_SHAPE, "sample: V must be in [1, 16384]");
    TRY(check_sampling(samp, V, uniforms));
    (void)hipGetLastError();
    hipError_t e = launch_sample(logits, B, V, *samp, uniforms, nullptr, sampled_out, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "sample launch");
    return FTTS_OK;
}

int ftts_advance(int32_t* tokens, int32_t* positions, int32_t* seq_lens, int32_t* sampled, int32_t* remaining,
                 int32_t stop_token, int32_t retire_on_stop, int32_t* history, int32_t* step_counter,
                 int32_t max_steps, int32_t B, void* stream) {
    if (!tokens || !positions || !seq_lens || !sampled) return fail(FTTS_E_INVALID_ARG, "advance: NULL pointer");
    if (B < 1 || B > 1024) return fail(FTTS_E_SHAPE, "advance: B must be in [1, 1024]");
    if (history && (max_steps < 1 || !step_counter))
        return fail(FTTS_E_INVALID_ARG, "advance: history needs step_counter and max_steps >= 1");
    (void)hipGetLastError();
    hipError_t e = launch_advance(tokens, positions, seq_lens, sampled, remaining, stop_token, retire_on_stop != 0,
                                  history, step_counter, max_steps, B, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "advance launch");
    return FTTS_OK;
}

}  // extern "C"

namespace ftts {

size_t decode_control_bytes() { return mega_bytes(nullptr, nullptr); }

int set_error(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int decode_step(const ftts_weights* w, const int32_t* tokens, const int32_t* positions, const ftts_page_table* pt,
                const ftts_kv_pool* kv, float* logits_out, float* hidden_out, int32_t* sampled_out,
                const float* uniforms, const ftts_sampling* samp, int32_t B, void* ws, size_t ws_bytes, void* stream,
                int (*prepare)(void* ws, hipStream_t st)) {
    TRY(check_weights(w));
    if (reinterpret_cast<uintptr_t>(hidden_out) % 16) return fail(FTTS_E_ALIGN, "hidden_out must be 16-byte aligned");
    const ftts_config& c = w->cfg;
    if (B < 1 || B > FTTS_MAX_BATCH) return fail(FTTS_E_SHAPE, "B must be in [1, %d]", FTTS_MAX_BATCH);
    if (!tokens || !positions) return fail(FTTS_E_INVALID_ARG, "tokens/positions is NULL");
    if (!logits_out || !sampled_out) return fail(FTTS_E_INVALID_ARG, "logits_out/sampled_out is NULL");
    TRY(check_kv(pt, kv, true));
    TRY(check_sampling(samp, c.vocab, uniforms));
    TRY(check_ptr(ws, "workspace"));
    const size_t need = decode_bytes(c, B, nullptr, nullptr);
    if (ws_bytes < need) return fail(FTTS_E_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);

    hipStream_t st = (hipStream_t)stream;
    if (prepare) TRY(prepare(ws, st));
    DecodeWs W;
    decode_bytes(c, B, &W, reinterpret_cast<char*>(ws));
    const int d = c.d_model, H = c.n_head, F = c.d_ff, V = c.vocab;

    mega::Args ma{};
    const bool mega_ok = g_decode_path != 1 && mega_args(w, B, &ma);
    if (g_decode_path == 2 && !mega_ok)
        return fail(FTTS_E_UNSUPPORTED, "the persistent decode step does not take this model/batch/device");
    if (mega_ok) {
        MegaWs M;
        mega_bytes(&M, reinterpret_cast<char*>(ws));
        ma.max_pages = pt->max_pages;
        ma.n_pages = kv->n_pages;
        ma.greedy = samp->top_k == 1;
        ma.tokens = tokens;
        ma.positions = positions;
        ma.seq_lens = pt->seq_lens;
        ma.block_table = pt->block_table;
        ma.kv = kv->base;
        ma.logits = logits_out;
        ma.hidden = hidden_out;
        ma.sampled = sampled_out;
        ma.active_out = W.active;
        ma.ex_x = M.x;
        ma.ex_qkv = M.qkv;
        ma.ex_o = M.o;
        ma.ex_h = M.h;
        ma.ex_arg = M.arg;
        ma.ctl = M.ctl;
        (void)hipGetLastError();
        hipError_t e = launch_decode_mega(c.wdtype, ma, st);
        if (e != hipSuccess) return hip_fail(e, "persistent decode step");
        if (samp->top_k != 1) {
            e = launch_sample(logits_out, B, V, *samp, uniforms, W.active, sampled_out, st);
            if (e != hipSuccess) return hip_fail(e, "sampler");
        }
        return FTTS_OK;
    }

    (void)hipGetLastError();
    // the batched path also takes the first LayerNorm's statistics and zeroes its counters here
    hipError_t e = launch_embed(c.wdtype, w->tok_emb, w->pos_emb, V, c.n_pos, d, tokens, positions, pt->seq_lens,
                                pt->block_table, pt->max_pages, kv->n_pages, B, W.x, W.active, W.stats, W.count,
                                W.stats ? bgemm_counters(c) : 0, st);
    if (e != hipSuccess) return hip_fail(e, "embed");

    KvAppend kva{};
    kva.base = kv->base;
    kva.n_pages = kv->n_pages;
    kva.n_head = H;
    kva.d_model = d;
    kva.max_pages = pt->max_pages;
    kva.block_table = pt->block_table;
    kva.seq_lens = pt->seq_lens;
    kva.active = W.active;

    AttnDecodeArgs at{};
    at.qkv = W.qkv;
    at.qkv_stride = 3 * d;
    at.kv_base = kv->base;
    at.n_pages = kv->n_pages;
    at.n_head = H;
    at.max_pages = pt->max_pages;
    at.block_table = pt->block_table;
    at.seq_lens = pt->seq_lens;
    at.active = W.active;
    at.o = W.o;
    at.o_stride = d;
    if (W.stats) return decode_batched(w, B, W, kva, at, logits_out, hidden_out, sampled_out, uniforms, samp, st);

    for (int l = 0; l < c.n_layer; ++l) {
        const ftts_layer& L = w->layers[l];
        GemvArgs g = gemv_args(L.qkv, 3 * d, d, B, W.x, W.qkv, 3 * d);
        g.ln_g = L.ln1_g;
        g.ln_b = L.ln1_b;
        g.eps = c.ln_eps;
        g.kv = kva;
        g.kv.layer = l;
        if ((e = launch_gemv(c.wdtype, EPI_QKV, true, g, st)) != hipSuccess) return hip_fail(e, "qkv");
        at.layer = l;
        if ((e = launch_attn_decode(c.wdtype, at, B, st)) != hipSuccess) return hip_fail(e, "attention");
        g = gemv_args(L.out, d, d, B, W.o, W.x, d);
        if ((e = launch_gemv(c.wdtype, EPI_RESID, false, g, st)) != hipSuccess) return hip_fail(e, "out-proj");
        g = gemv_args(L.fc1, F, d, B, W.x, W.h, F);
        g.ln_g = L.ln2_g;
        g.ln_b = L.ln2_b;
        g.eps = c.ln_eps;
        if ((e = launch_gemv(c.wdtype, EPI_GELU, true, g, st)) != hipSuccess) return hip_fail(e, "fc1");
        g = gemv_args(L.fc2, d, F, B, W.h, W.x, d);
        if ((e = launch_gemv(c.wdtype, EPI_RESID, false, g, st)) != hipSuccess) return hip_fail(e, "fc2");
    }
    GemvArgs g = gemv_args(w->head, V, d, B, W.x, logits_out, V);
    g.ln_g = w->lnf_g;
    g.ln_b = w->lnf_b;
    g.eps = c.ln_eps;
    g.hidden = hidden_out;
    if ((e = launch_gemv(c.wdtype, EPI_STORE, true, g, st)) != hipSuccess) return hip_fail(e, "lm head");
    if ((e = launch_sample(logits_out, B, V, *samp, uniforms, W.active, sampled_out, st)) != hipSuccess)
        return hip_fail(e, "sampler");
    return FTTS_OK;
}

}  // namespace ftts

extern "C" {

int ftts_decode_step(const ftts_weights* w, const int32_t* tokens, const int32_t* positions,
                     const ftts_page_table* pt, const ftts_kv_pool* kv, float* logits_out, int32_t* sampled_out,
                     const float* uniforms, const ftts_sampling* samp, int32_t B, void* ws, size_t ws_bytes,
                     void* stream) {
    return decode_step(w, tokens, positions, pt, kv, logits_out, nullptr, sampled_out, uniforms, samp, B, ws,
                       ws_bytes, stream, nullptr);
}

int ftts_decode_step_hidden(const ftts_weights* w, const int32_t* tokens, const int32_t* positions,
                            const ftts_page_table* pt, const ftts_kv_pool* kv, float* logits_out, float* hidden_out,
                            int32_t* sampled_out, const float* uniforms, const ftts_sampling* samp, int32_t B,
                            void* ws, size_t ws_bytes, void* stream) {
    return decode_step(w, tokens, positions, pt, kv, logits_out, hidden_out, sampled_out, uniforms, samp, B, ws,
                       ws_bytes, stream, nullptr);
}

// Where the prefill's input rows come from: ready embeddings, or the model's
// own input assembly (conditioning rows, then text ids through the merged table).
struct PrefixSource {
    const void* emb;             // [sum lens][d] activation dtype, or null
    const void* cond;            // [sum cond_lens][d] activation dtype
    const int32_t* cond_lens;    // [host][B]
    const int32_t* text_ids;     // [sum text_lens] device
    int text_vocab, text_pos0;
};

static int prefill(const ftts_weights* w, const PrefixSource& src, const int32_t* lens, int32_t B,
                   const ftts_page_table* pt, const ftts_kv_pool* kv, float* last_logits, void* ws, size_t ws_bytes,
                   void* stream) {
    const ftts_config& c = w->cfg;
    TRY(check_kv(pt, kv, false));
    TRY(check_ptr(ws, "workspace"));
    SeqTable seqs{};
    AttnPrefillArgs ap{};
    seqs.n = B;
    seqs.cu[0] = 0;
    ap.tiles_cu[0] = 0;
    int64_t M = 0;
    for (int b = 0; b < B; ++b) {
        if (lens[b] < 1) return fail(FTTS_E_RANGE, "lens[%d] = %d must be >= 1", b, lens[b]);
        if ((int64_t)lens[b] > (int64_t)pt->max_pages * kPage)
            return fail(FTTS_E_RANGE, "lens[%d] = %d exceeds max_pages * 64", b, lens[b]);
        M += lens[b];
        if (M > (1 << 24)) return fail(FTTS_E_RANGE, "total prefix rows too large");
        seqs.cu[b + 1] = (int)M;
        ap.tiles_cu[b + 1] = ap.tiles_cu[b] + (lens[b] + prefill_tile_rows(c.wdtype) - 1) / prefill_tile_rows(c.wdtype);
    }
    const size_t need = prefill_bytes(c, B, (int)M, nullptr, nullptr);
    if (ws_bytes < need) return fail(FTTS_E_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);

    hipStream_t st = (hipStream_t)stream;
    PrefillWs P;
    prefill_bytes(c, B, (int)M, &P, reinterpret_cast<char*>(ws));
    const int d = c.d_model, F = c.d_ff, V = c.vocab, Mi = (int)M;

    (void)hipGetLastError();
    hipError_t e;
    if (src.emb) {
        if ((e = launch_act_to_f32(c.wdtype, src.emb, Mi, d, P.x, st)) != hipSuccess) return hip_fail(e, "prefix copy");
    } else {
        AssembleArgs as{};
        as.seqs = seqs;
        as.cond_cu[0] = 0;
        for (int b = 0; b < B; ++b) as.cond_cu[b + 1] = as.cond_cu[b] + src.cond_lens[b];
        as.cond = src.cond;
        as.text_ids = src.text_ids;
        as.tok_emb = w->tok_emb;
        as.pos_emb = w->pos_emb;
        as.d = d;
        as.vocab = V;
        as.text_vocab = src.text_vocab;
        as.text_pos0 = src.text_pos0;
        as.x = P.x;
        if ((e = launch_assemble_prefix(c.wdtype, as, Mi, st)) != hipSuccess) return hip_fail(e, "input assembly");
    }
    if (P.count) {
        size_t pf, cn;
        gemm_scratch(c, Mi, &pf, &cn);
        if ((e = launch_fill_u32(P.count, cn, 0u, st)) != hipSuccess) return hip_fail(e, "gemm counters");
    }

    KvAppend kva{};
    kva.base = kv->base;
    kva.n_pages = kv->n_pages;
    kva.n_head = c.n_head;
    kva.d_model = d;
    kva.max_pages = pt->max_pages;
    kva.block_table = pt->block_table;

    ap.qkv = P.qkv;
    ap.o = P.a;
    ap.d_model = d;
    ap.n_head = c.n_head;
    ap.seqs = seqs;

    for (int l = 0; l < c.n_layer; ++l) {
        const ftts_layer& L = w->layers[l];
        if ((e = launch_ln_rows(c.wdtype, P.x, L.ln1_g, L.ln1_b, c.ln_eps, Mi, d, P.a, st)) != hipSuccess)
            return hip_fail(e, "ln1");
        GemmArgs g{};
        g.part = P.part;
        g.count = P.count;
        g.a = P.a;
        g.w = L.qkv.w;
        g.scale = (const uint16_t*)L.qkv.scale;
        g.zero = (const uint16_t*)L.qkv.zero;
        g.bias = L.qkv.bias;
        g.M = Mi;
        g.N = 3 * d;
        g.K = d;
        g.out = P.qkv;
        g.kv = kva;
        g.kv.layer = l;
        g.seqs = seqs;
        if ((e = launch_gemm(c.wdtype, EPI_QKV, g, st)) != hipSuccess) return hip_fail(e, "qkv gemm");
        if ((e = launch_attn_prefill(c.wdtype, ap, ap.tiles_cu[B], st)) != hipSuccess)
            return hip_fail(e, "prefill attention");
        g.w = L.out.w;
        g.scale = (const uint16_t*)L.out.scale;
        g.zero = (const uint16_t*)L.out.zero;
        g.bias = L.out.bias;
        g.N = d;
        g.K = d;
        g.out = P.x;
        if ((e = launch_gemm(c.wdtype, EPI_RESID, g, st)) != hipSuccess) return hip_fail(e, "out gemm");
        if ((e = launch_ln_rows(c.wdtype, P.x, L.ln2_g, L.ln2_b, c.ln_eps, Mi, d, P.a, st)) != hipSuccess)
            return hip_fail(e, "ln2");
        g.w = L.fc1.w;
        g.scale = (const uint16_t*)L.fc1.scale;
        g.zero = (const uint16_t*)L.fc1.zero;
        g.bias = L.fc1.bias;
        g.N = F;
        g.K = d;
        g.out = P.h;
        if ((e = launch_gemm(c.wdtype, EPI_GELU, g, st)) != hipSuccess) return hip_fail(e, "fc1 gemm");
        g.a = P.h;
        g.w = L.fc2.w;
        g.scale = (const uint16_t*)L.fc2.scale;
        g.zero = (const uint16_t*)L.fc2.zero;
        g.bias = L.fc2.bias;
        g.N = d;
        g.K = F;
        g.out = P.x;
        if ((e = launch_gemm(c.wdtype, EPI_RESID, g, st)) != hipSuccess) return hip_fail(e, "fc2 gemm");
    }
    // A new generation starts: clear the persistent step's control words and
    // exchange buffers (epoch 0 never matches a live epoch).
    if ((e = launch_fill_u32(reinterpret_cast<uint32_t*>(ws), mega_bytes(nullptr, nullptr) / 4, 0u, st)) !=
        hipSuccess)
        return hip_fail(e, "workspace reset");
    if (last_logits) {
        if ((e = launch_gather_rows(P.x, d, seqs, P.xlast, st)) != hipSuccess) return hip_fail(e, "gather");
        GemvArgs g = gemv_args(w->head, V, d, B, P.xlast, last_logits, V);
        g.ln_g = w->lnf_g;
        g.ln_b = w->lnf_b;
        g.eps = c.ln_eps;
        if ((e = launch_gemv(c.wdtype, EPI_STORE, true, g, st)) != hipSuccess) return hip_fail(e, "lm head");
    }
    return FTTS_OK;
}

int ftts_prefill(const ftts_weights* w, const void* prefix_emb, const int32_t* lens, int32_t B,
                 const ftts_page_table* pt, const ftts_kv_pool* kv, float* last_logits, void* ws, size_t ws_bytes,
                 void* stream) {
    TRY(check_weights(w));
    if (B < 1 || B > FTTS_MAX_BATCH) return fail(FTTS_E_SHAPE, "B must be in [1, %d]", FTTS_MAX_BATCH);
    TRY(check_ptr(prefix_emb, "prefix_emb"));
    if (!lens) return fail(FTTS_E_INVALID_ARG, "lens is NULL");
    PrefixSource src{};
    src.emb = prefix_emb;
    return prefill(w, src, lens, B, pt, kv, last_logits, ws, ws_bytes, stream);
}

int ftts_prefill_ids(const ftts_weights* w, const void* cond_emb, const int32_t* cond_lens, const int32_t* text_ids,
                     const int32_t* text_lens, int32_t text_vocab, int32_t text_pos0, int32_t B,
                     const ftts_page_table* pt, const ftts_kv_pool* kv, float* last_logits, void* ws,
                     size_t ws_bytes, void* stream) {
    TRY(check_weights(w));
    const ftts_config& c = w->cfg;
    if (B < 1 || B > FTTS_MAX_BATCH) return fail(FTTS_E_SHAPE, "B must be in [1, %d]", FTTS_MAX_BATCH);
    if (!cond_lens || !text_lens) return fail(FTTS_E_INVALID_ARG, "cond_lens/text_lens is NULL");
    if (text_pos0 < 0) return fail(FTTS_E_RANGE, "text_pos0 must be >= 0");
    int32_t lens[FTTS_MAX_BATCH];
    int64_t n_cond = 0, n_text = 0;
    for (int b = 0; b < B; ++b) {
        if (cond_lens[b] < 0 || text_lens[b] < 0)
            return fail(FTTS_E_RANGE, "cond_lens[%d] / text_lens[%d] must be >= 0", b, b);
        if ((int64_t)text_pos0 + text_lens[b] > c.n_pos)
            return fail(FTTS_E_RANGE, "text positions of sequence %d run past n_pos", b);
        if ((int64_t)cond_lens[b] + text_lens[b] > (1 << 24)) return fail(FTTS_E_RANGE, "prefix too long");
        lens[b] = cond_lens[b] + text_lens[b];
        n_cond += cond_lens[b];
        n_text += text_lens[b];
    }
    if (n_cond > 0) TRY(check_ptr(cond_emb, "cond_emb"));
    if (n_text > 0) {
        if (!text_ids) return fail(FTTS_E_INVALID_ARG, "text_ids is NULL");
        if (text_vocab < 1) return fail(FTTS_E_RANGE, "text_vocab must be >= 1");
    }
    PrefixSource src{};
    src.cond = cond_emb;
    src.cond_lens = cond_lens;
    src.text_ids = text_ids;
    src.text_vocab = text_vocab;
    src.text_pos0 = text_pos0;
    return prefill(w, src, lens, B, pt, kv, last_logits, ws, ws_bytes, stream);
}

}  // extern "C"

// ---- flow-matching DiT step -------------------------------------------------------------

static_assert(2 * FTTS_DIT_MAX_BATCH <= kMaxPrefillSeqs, "both guidance branches of every utterance need a sequence");

namespace {

struct DitWs {
    float* h;        // [M][D] fp32 residual stream
    void* a;         // [M][max(D, Kin)] bf16: input rows, LayerNorm outputs, attention outputs
    void* qkv;       // [M][3D] bf16
    void* f;         // [M][F] bf16 GELU activations
    float* vel;      // [M][n_mel] fp32 velocities of both branches
    float* u;        // [D] time MLP hidden
    float* e;        // [D] time embedding
    float* part;     // split-K partial tiles
    uint32_t* count; // split-K arrival counters
    size_t n_count;
};

int check_dit_config(const ftts_dit_config* c) {
    if (!c) return fail(FTTS_E_INVALID_ARG, "config is NULL");
    if (c->n_layer < 1) return fail(FTTS_E_SHAPE, "n_layer must be >= 1");
    if (c->d_head != kHeadDim) return fail(FTTS_E_UNSUPPORTED, "d_head must be 64 (got %d)", c->d_head);
    if (c->n_head < 1 || c->n_head * kHeadDim != c->d_model)
        return fail(FTTS_E_SHAPE, "n_head * d_head must equal d_model");
    if (c->d_model % 64 || c->d_model > 2048) return fail(FTTS_E_SHAPE, "d_model must be a multiple of 64, <= 2048");
    if (c->d_ff < 64 || c->d_ff % 64 || c->d_ff > 16384) return fail(FTTS_E_SHAPE, "d_ff must be a multiple of 64");
    if (c->n_mel < 64 || c->n_mel % 64) return fail(FTTS_E_SHAPE, "n_mel must be a positive multiple of 64");
    if (c->d_cond < 0 || (c->n_mel + c->d_cond) % 64)
        return fail(FTTS_E_SHAPE, "n_mel + d_cond must be a multiple of 64");
    if (c->t_dim < 2 || c->t_dim > 1024 || c->t_dim % 2) return fail(FTTS_E_SHAPE, "t_dim must be even, <= 1024");
    if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps)) return fail(FTTS_E_RANGE, "ln_eps must be finite and > 0");
    return FTTS_OK;
}

// Split-K scratch of the step's six GEMM shapes at M = 2T rows, maximised over every
// row count up to M (a smaller call may split where a larger one does not).
void dit_gemm_scratch(const ftts_dit_config& c, int M, size_t* part_floats, size_t* counters) {
    const int d = c.d_model, F = c.d_ff, Kin = c.n_mel + c.d_cond;
    const int NK[6][2] = {{d, Kin}, {3 * d, d}, {d, d}, {F, d}, {d, F}, {c.n_mel, d}};
    size_t pf = 0, cn = 0;
    for (int r = 64;; r += 64) {
        const int rows = std::min(r, M);
        for (const auto& t : NK) {
            const GemmPlan p = gemm_plan(rows, t[0], t[1]);
            if (p.splits > 1) {
                // partial tiles are whole (64 mt) x 128 tiles, past the matrix edges too
                pf = std::max(pf, (size_t)p.splits * p.tiles_m * p.tiles_n * (64 * p.mt) * 128);
                cn = std::max(cn, (size_t)p.tiles_m * p.tiles_n);
            }
        }
        if (rows >= M) break;
    }
    *part_floats = pf;
    *counters = cn;
}

size_t dit_bytes(const ftts_dit_config& c, int T, DitWs* out, char* base) {
    const size_t M = 2 * (size_t)T, d = c.d_model, Kin = (size_t)c.n_mel + c.d_cond;
    size_t off = 0;
    auto take = [&](size_t n) { size_t o = off; off += round256(n); return base ? base + o : nullptr; };
    char* h = take(M * d * 4);
    char* a = take(M * std::max(d, Kin) * 2);
    char* qkv = take(M * 3 * d * 2);
    char* f = take(M * (size_t)c.d_ff * 2);
    char* vel = take(M * (size_t)c.n_mel * 4);
    char* u = take(d * 4);
    char* e = take(d * 4);
    size_t pf, cn;
    dit_gemm_scratch(c, (int)M, &pf, &cn);
    char* part = pf ? take(pf * 4) : nullptr;
    char* count = cn ? take(cn * 4) : nullptr;
    if (out) *out = DitWs{(float*)h, a, qkv, f, (float*)vel, (float*)u, (float*)e, (float*)part, (uint32_t*)count, cn};
    return off;
}

int check_bf16_linear(const ftts_linear& l, const char* name) {
    char buf[64];
    snprintf(buf, sizeof(buf), "%s.w", name);
    TRY(check_ptr(l.w, buf));
    snprintf(buf, sizeof(buf), "%s.bias", name);
    TRY(check_ptr(l.bias, buf));
    return FTTS_OK;
}

int check_dit_weights(const ftts_dit_weights* w) {
    if (!w) return fail(FTTS_E_INVALID_ARG, "weights is NULL");
    TRY(check_dit_config(&w->cfg));
    TRY(check_bf16_linear(w->in, "in"));
    TRY(check_bf16_linear(w->t1, "t1"));
    TRY(check_bf16_linear(w->t2, "t2"));
    TRY(check_bf16_linear(w->mel, "mel"));
    TRY(check_ptr(w->lnf_g, "lnf_g"));
    TRY(check_ptr(w->lnf_b, "lnf_b"));
    if (!w->layers) return fail(FTTS_E_INVALID_ARG, "layers is NULL");
    for (int l = 0; l < w->cfg.n_layer; ++l) {
        const ftts_layer& L = w->layers[l];
        TRY(check_ptr(L.ln1_g, "ln1_g"));
        TRY(check_ptr(L.ln1_b, "ln1_b"));
        TRY(check_ptr(L.ln2_g, "ln2_g"));
        TRY(check_ptr(L.ln2_b, "ln2_b"));
        TRY(check_bf16_linear(L.qkv, "qkv"));
        TRY(check_bf16_linear(L.out, "out"));
        TRY(check_bf16_linear(L.fc1, "fc1"));
        TRY(check_bf16_linear(L.fc2, "fc2"));
    }
    return FTTS_OK;
}

GemmArgs dit_gemm(const ftts_linear& l, const void* a, int M, int N, int K, void* out, const DitWs& W) {
    GemmArgs g{};
    g.a = a;
    g.w = l.w;
    g.bias = l.bias;
    g.M = M;
    g.N = N;
    g.K = K;
    g.out = out;
    g.part = W.part;
    g.count = W.count;
    return g;
}

}  // namespace

extern "C" {

size_t ftts_dit_workspace_bytes(const ftts_dit_config* cfg, int32_t max_frames) {
    if (check_dit_config(cfg) != FTTS_OK || max_frames < 1 || max_frames > (1 << 20)) return 0;
    return dit_bytes(*cfg, max_frames, nullptr, nullptr);
}

int ftts_dit_step(const ftts_dit_weights* w, const float* x, const void* cond, const int32_t* lens, int32_t B,
                  float t, float dt, float cfg_w, float* x_out, float* v_out, void* ws, size_t ws_bytes,
                  void* stream) {
    TRY(check_dit_weights(w));
    const ftts_dit_config& c = w->cfg;
    if (B < 1 || B > FTTS_DIT_MAX_BATCH) return fail(FTTS_E_SHAPE, "B must be in [1, %d]", FTTS_DIT_MAX_BATCH);
    if (!lens) return fail(FTTS_E_INVALID_ARG, "lens is NULL");
    int64_t total = 0;
    for (int b = 0; b < B; ++b) {
        if (lens[b] < 1) return fail(FTTS_E_SHAPE, "lens[%d] = %d must be >= 1", b, lens[b]);
        total += lens[b];
        if (total > (1 << 20)) return fail(FTTS_E_SHAPE, "more than 2^20 frames in one step");
    }
    const int T = (int)total;  // frames of the whole batch
    if (!std::isfinite(t) || !std::isfinite(dt) || !std::isfinite(cfg_w))
        return fail(FTTS_E_RANGE, "t, dt and cfg_w must be finite");
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(x_out, "x_out"));
    if (c.d_cond > 0) TRY(check_ptr(cond, "cond"));
    if (v_out) TRY(check_ptr(v_out, "v_out"));
    TRY(check_ptr(ws, "workspace"));
    const size_t need = dit_bytes(c, T, nullptr, nullptr);
    if (ws_bytes < need) return fail(FTTS_E_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);

    hipStream_t st = (hipStream_t)stream;
    DitWs W;
    dit_bytes(c, T, &W, reinterpret_cast<char*>(ws));
    const int d = c.d_model, F = c.d_ff, M = 2 * T, Kin = c.n_mel + c.d_cond;

    (void)hipGetLastError();
    hipError_t e;
    if ((e = launch_dit_time(t, w->t1.w, w->t1.bias, w->t2.w, w->t2.bias, d, c.t_dim, W.u, W.e, st)) != hipSuccess)
        return hip_fail(e, "time embedding");
    DitPrepareArgs pa{};
    pa.T = T;
    pa.n_mel = c.n_mel;
    pa.d_cond = c.d_cond;
    pa.d_model = d;
    pa.x = x;
    pa.cond = cond;
    pa.e = W.e;
    pa.inp = W.a;
    pa.h = W.h;
    pa.vel = W.vel;
    pa.count = W.count;
    pa.n_count = W.n_count;
    if ((e = launch_dit_prepare(pa, st)) != hipSuccess) return hip_fail(e, "step inputs");
    // h = [x | c] W_in^T + b_in + e(t)
    if ((e = launch_gemm(FTTS_BF16, EPI_RESID, dit_gemm(w->in, W.a, M, d, Kin, W.h, W), st)) != hipSuccess)
        return hip_fail(e, "input projection");

    AttnPrefillArgs ap{};
    ap.qkv = W.qkv;
    ap.o = W.a;
    ap.d_model = d;
    ap.n_head = c.n_head;
    // 2B sequences: the conditional rows of every utterance, then the unconditional ones
    ap.seqs.n = 2 * B;
    ap.seqs.cu[0] = 0;
    for (int b = 0; b < B; ++b) {
        ap.seqs.cu[b + 1] = ap.seqs.cu[b] + lens[b];
        ap.seqs.cu[B + b + 1] = T + ap.seqs.cu[b + 1];
    }

    for (int l = 0; l < c.n_layer; ++l) {
        const ftts_layer& L = w->layers[l];
        if ((e = launch_ln_rows(FTTS_BF16, W.h, L.ln1_g, L.ln1_b, c.ln_eps, M, d, W.a, st)) != hipSuccess)
            return hip_fail(e, "ln1");
        if ((e = launch_gemm(FTTS_BF16, EPI_STORE, dit_gemm(L.qkv, W.a, M, 3 * d, d, W.qkv, W), st)) != hipSuccess)
            return hip_fail(e, "qkv gemm");
        if ((e = launch_attn_full_bf16(ap, st)) != hipSuccess) return hip_fail(e, "attention");
        if ((e = launch_gemm(FTTS_BF16, EPI_RESID, dit_gemm(L.out, W.a, M, d, d, W.h, W), st)) != hipSuccess)
            return hip_fail(e, "out gemm");
        if ((e = launch_ln_rows(FTTS_BF16, W.h, L.ln2_g, L.ln2_b, c.ln_eps, M, d, W.a, st)) != hipSuccess)
            return hip_fail(e, "ln2");
        if ((e = launch_gemm(FTTS_BF16, EPI_GELU, dit_gemm(L.fc1, W.a, M, F, d, W.f, W), st)) != hipSuccess)
            return hip_fail(e, "fc1 gemm");
        if ((e = launch_gemm(FTTS_BF16, EPI_RESID, dit_gemm(L.fc2, W.f, M, d, F, W.h, W), st)) != hipSuccess)
            return hip_fail(e, "fc2 gemm");
    }
    if ((e = launch_ln_rows(FTTS_BF16, W.h, w->lnf_g, w->lnf_b, c.ln_eps, M, d, W.a, st)) != hipSuccess)
        return hip_fail(e, "final layer norm");
    if ((e = launch_gemm(FTTS_BF16, EPI_RESID, dit_gemm(w->mel, W.a, M, c.n_mel, d, W.vel, W), st)) != hipSuccess)
        return hip_fail(e, "mel projection");
    if ((e = launch_dit_guide(W.vel, T, c.n_mel, cfg_w, dt, x, x_out, v_out, st)) != hipSuccess)
        return hip_fail(e, "guidance");
    return FTTS_OK;
}

}  // extern "C"
