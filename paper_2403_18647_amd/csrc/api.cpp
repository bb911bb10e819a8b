// Host runtime of the SDSAT block-decode library: context, workspace layout,
// weight packing, block forward, verification, KV commit and the draft/verify
// generation loop (Section 2.1).  Declared in include/sdsat.h.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/sdsat.h"
#include "kernels.h"

using namespace sdsat;

namespace {

thread_local std::string g_init_error = "no error";

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Bump allocator over the caller's workspace; with base == 0 it only measures.
struct Carver {
    char* base;
    size_t off = 0;
    explicit Carver(void* b) : base(static_cast<char*>(b)) {}
    void* take(size_t bytes) {
        off = align_up(off, 256);
        void* p = base ? base + off : nullptr;
        off += bytes;
        return p;
    }
};

struct Dims {
    int L, d, H, Dh, F, V, A, esz, dtype;
    int S;           // KV slots per sequence (max_ctx rounded up to 32)
    int maxB, maxQ, maxM;
    int ks_d, ks_f;  // k-steps for K = d and K = F
    int nt_qkv, nt_o, nt_gu, nt_down, nt_lm;
    int n_ssq;       // d / 16
    int d_pad, F_pad;  // activation row strides (contraction lengths padded to 32)
};

constexpr int kMaxBlock = 4096;   // rows per sequence per block
constexpr int kSkinnyRows = 64;   // blocks of at most this many rows (B*q) run the skinny GEMM kernels
constexpr int kRecLoops = 64;     // generation loops enqueued between two host synchronisations, at most
constexpr int kPreRoundRows = 1;  // blocks of more rows round normalised GEMM inputs once (rms_rows)
constexpr int kQkvFloatRows = 8;  // except the QKV GEMM, which reads the float rows up to this many

int make_dims(const sdsat_config* c, Dims* D, std::string* why) {
    if (!c) { *why = "config is NULL"; return SDSAT_EINVAL; }
    if (c->n_layers < 1 || c->d_model < 16 || c->n_heads < 1 || c->d_ffn < 8 || c->vocab < 2 ||
        c->n_adaptive < 0 || c->max_batch < 1 || c->max_ctx < 1 || c->max_block < 1) {
        *why = "config has a non-positive dimension";
        return SDSAT_EINVAL;
    }
    if (c->head_dim != 64 && c->head_dim != 128) { *why = "head_dim must be 64 or 128"; return SDSAT_EUNSUPPORTED; }
    if (c->n_heads * c->head_dim != c->d_model) { *why = "d_model must equal n_heads * head_dim"; return SDSAT_EINVAL; }
    if (c->d_model % 16) { *why = "d_model must be a multiple of 16"; return SDSAT_EUNSUPPORTED; }
    if (c->dtype != SDSAT_DTYPE_FP32 && c->dtype != SDSAT_DTYPE_BF16) { *why = "dtype must be 0 or 1"; return SDSAT_EINVAL; }
    if (c->max_block > kMaxBlock) { *why = "max_block must be <= 4096"; return SDSAT_EUNSUPPORTED; }
    if ((long)c->max_batch * c->max_block > kSkinnyRows && c->d_ffn % 8) {
        *why = "blocks of more than 64 rows need d_ffn to be a multiple of 8";
        return SDSAT_EUNSUPPORTED;
    }
    if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f)) { *why = "rms_eps must be >= 0 and rope_base > 0"; return SDSAT_EINVAL; }
    D->L = c->n_layers; D->d = c->d_model; D->H = c->n_heads; D->Dh = c->head_dim; D->F = c->d_ffn;
    D->V = c->vocab; D->A = c->n_adaptive; D->dtype = c->dtype; D->esz = c->dtype == SDSAT_DTYPE_BF16 ? 2 : 4;
    D->S = (int)align_up((size_t)c->max_ctx, 32);
    D->maxB = c->max_batch; D->maxQ = c->max_block;
    D->maxM = c->max_batch * c->max_block;
    D->ks_d = (D->d + 31) / 32; D->ks_f = (D->F + 31) / 32;
    D->nt_qkv = 3 * D->d / 16; D->nt_o = D->d / 16; D->nt_gu = (D->F + 7) / 8; D->nt_down = D->d / 16;
    D->nt_lm = (D->V + 15) / 16;
    D->n_ssq = D->d / 16;
    D->d_pad = D->ks_d * 32; D->F_pad = D->ks_f * 32;
    return SDSAT_OK;
}

enum ProfKind {
    PK_OFF = 0, PK_GATEUP = 1, PK_QKV = 2, PK_ATTN = 3, PK_DOWN = 4, PK_O = 5, PK_LM = 6,
    PK_BLOCK = 7,     // block forwards that produce logits (draft and verify blocks)
    PK_PREFILL = 8,   // block forwards without logits (prefill)
};

}  // namespace

struct sdsat_ctx {
    sdsat_config cfg;
    Dims D;
    hipStream_t stream = nullptr;
    std::string err = "no error";
    int device = 0;
    // caller weights
    const void* embed = nullptr;
    std::vector<const float*> attn_norm, ffn_norm;
    const float* final_norm = nullptr;
    // the caller's row-major weights (embed, {attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down} x L,
    // final_norm, lm_head): the prefill GEMMs of large blocks read them
    std::vector<const void*> w_src;
    // packed weights
    std::vector<void*> w_qkv, w_o, w_gu, w_down;
    void* w_lm = nullptr;
    // cache
    void* kc = nullptr; void* vc = nullptr;
    size_t layer_elems = 0;   // elements per layer of K (and of V)
    double* inv_freq = nullptr;   // rotary inverse frequencies [Dh/2]
    float* rope = nullptr;        // rotary cos / sin per cache slot [S][Dh/2][2]
    // activations
    float* x = nullptr; float* ssq = nullptr;
    float* xg = nullptr;  // x o (next RMSNorm gain), float, row stride d_pad (zero pad)
    void* qbuf = nullptr; void* obuf = nullptr; void* ubuf = nullptr;
    // scratch
    float* attn_part = nullptr;
    size_t attn_part_floats = 0;
    int* attn_ctr = nullptr;      // attention split arrival counters (zero between launches)
    float* gemm_part = nullptr;   // partial tiles of split residual GEMMs
    int* cache_len = nullptr; int* err_flag = nullptr; int* verify_cnt = nullptr;
    // generation buffers
    int *tok1 = nullptr, *out1 = nullptr, *out2 = nullptr, *n_accept = nullptr, *pending = nullptr;
    int *active = nullptr, *n_commit = nullptr, *pos0 = nullptr, *adaptive = nullptr, *ptok = nullptr;
    // draft tree (draft step 2 of the tree loop): tokens, ancestor masks, depths, targets, branch rows
    int *tree_tok = nullptr, *tree_depth = nullptr, *tree_target = nullptr, *tree_rows = nullptr;
    uint64_t* tree_mask = nullptr;
    float* logits = nullptr;
    // large blocks (more than kSkinnyRows rows): normalised rows (element type) and float GEMM outputs
    void* hbuf = nullptr; float* c_y = nullptr;
    int* h_pin = nullptr;   // pinned host staging
    size_t h_pin_ints = 0;
    int* h_rec = nullptr;      // pinned host copy of the loop records
    int* loop_rec = nullptr;   // device loop records [kRecLoops][maxB][kLoopRecCols]
    int* produced = nullptr;   // tokens each sequence has emitted in the current generation (device)
    // upper bounds of cache_len, tracked on the host for launch planning
    std::vector<int> len_hint;
    // profiling
    int prof_kind = PK_OFF;
    int prof_period = 1;
    int64_t prof_seen = 0;
    std::vector<hipEvent_t> events;
    size_t ev_used = 0;

    ~sdsat_ctx() {
        for (hipEvent_t e : events) (void)hipEventDestroy(e);
        if (h_pin) (void)hipHostFree(h_pin);
        if (h_rec) (void)hipHostFree(h_rec);
    }
};

namespace {

int fail(sdsat_ctx* c, int code, const std::string& msg) {
    if (c) c->err = msg; else g_init_error = msg;
    return code;
}

#define HIPCHK(ctx, expr)                                                                   \
    do {                                                                                    \
        hipError_t e_ = (expr);                                                             \
        if (e_ != hipSuccess)                                                               \
            return fail((ctx), SDSAT_EDEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

// Carve every device buffer of a context (ctx may be a measuring dummy).
void carve(sdsat_ctx* c, Carver& cv) {
    const Dims& D = c->D;
    const size_t e = D.esz;
    c->w_qkv.resize(D.L); c->w_o.resize(D.L); c->w_gu.resize(D.L); c->w_down.resize(D.L);
    for (int l = 0; l < D.L; ++l) {
        c->w_qkv[l] = cv.take(packed_elems(D.nt_qkv, D.ks_d) * e);
        c->w_o[l] = cv.take(packed_elems(D.nt_o, D.ks_d) * e);
        c->w_gu[l] = cv.take(packed_elems(D.nt_gu, D.ks_d) * e);
        c->w_down[l] = cv.take(packed_elems(D.nt_down, D.ks_f) * e);
    }
    c->w_lm = cv.take(packed_elems(D.nt_lm, D.ks_d) * e);
    c->layer_elems = (size_t)D.maxB * D.H * D.S * D.Dh;
    c->kc = cv.take(c->layer_elems * D.L * e);
    c->vc = cv.take(c->layer_elems * D.L * e);
    c->inv_freq = (double*)cv.take((size_t)(D.Dh / 2) * 8);
    c->rope = (float*)cv.take((size_t)D.S * (D.Dh / 2) * 8);
    c->x = (float*)cv.take((size_t)D.maxM * D.d * 4);
    c->ssq = (float*)cv.take((size_t)D.maxM * D.n_ssq * 4);
    c->xg = (float*)cv.take((size_t)D.maxM * D.d_pad * 4);
    c->qbuf = cv.take((size_t)D.maxB * D.maxQ * D.d * 4);
    c->obuf = cv.take((size_t)D.maxM * D.d_pad * e);
    c->ubuf = cv.take((size_t)D.maxM * D.F_pad * e);
    c->attn_part_floats = std::max<size_t>(1, attention_partial_floats(D.maxB, D.H, D.maxQ, D.Dh, D.S));
    c->attn_part = (float*)cv.take(c->attn_part_floats * 4);
    c->attn_ctr = (int*)cv.take(attention_counter_ints(D.maxB, D.H, D.maxQ) * 4);
    {
        const int rows = std::min(D.maxM, kSkinnyRows);
        const size_t part = std::max(gemm_resid_part_bytes(D.nt_o, D.ks_d, rows),
                                     gemm_resid_part_bytes(D.nt_down, D.ks_f, rows));
        c->gemm_part = part ? (float*)cv.take(part) : nullptr;
    }
    c->cache_len = (int*)cv.take((size_t)D.maxB * 4);
    c->err_flag = (int*)cv.take(4);
    c->verify_cnt = (int*)cv.take((size_t)D.maxB * 4);
    c->produced = (int*)cv.take((size_t)D.maxB * 4);
    c->loop_rec = (int*)cv.take((size_t)kRecLoops * D.maxB * kLoopRecCols * 4);
    const size_t bq = (size_t)D.maxB * D.maxQ;
    c->tok1 = (int*)cv.take(bq * 4);
    c->out1 = (int*)cv.take(bq * 4);
    c->out2 = (int*)cv.take(bq * 4);
    c->ptok = (int*)cv.take(bq * 4);
    c->n_accept = (int*)cv.take((size_t)D.maxB * 4);
    c->pending = (int*)cv.take((size_t)D.maxB * 4);
    c->active = (int*)cv.take((size_t)D.maxB * 4);
    c->n_commit = (int*)cv.take((size_t)D.maxB * 4);
    c->pos0 = (int*)cv.take((size_t)D.maxB * 4);
    c->adaptive = (int*)cv.take(64 * 4);
    c->tree_tok = (int*)cv.take(bq * 4);
    c->tree_depth = (int*)cv.take(bq * 4);
    c->tree_target = (int*)cv.take(bq * 4);
    c->tree_rows = (int*)cv.take(bq * 4);
    c->tree_mask = (uint64_t*)cv.take(bq * 8);
    c->logits = (float*)cv.take(bq * D.V * 4);
    c->hbuf = cv.take((size_t)D.maxM * D.d_pad * e);
    if (D.maxM > kSkinnyRows) c->c_y = (float*)cv.take((size_t)D.maxM * D.d * 4 * kPrefillMaxSplit);   // split-K parts
}

void* layer_k(sdsat_ctx* c, int l) { return (char*)c->kc + (size_t)l * c->layer_elems * c->D.esz; }
void* layer_v(sdsat_ctx* c, int l) { return (char*)c->vc + (size_t)l * c->layer_elems * c->D.esz; }

// ---------------------------------------------------------------- profiling
// Takes the next event pair of the pool for a sampled launch of `kind` (null
// when this launch is not sampled).
void prof_take(sdsat_ctx* c, int kind, hipEvent_t* out) {
    *out = nullptr;
    if (c->prof_kind != kind) return;
    if (c->prof_seen++ % c->prof_period != 0) return;
    if (c->ev_used + 2 > c->events.size()) {
        for (int i = 0; i < 64; ++i) {
            // no system-scope fence on record: the interval then covers the kernel, not a cache flush
            hipEvent_t ev;
            if (hipEventCreateWithFlags(&ev, hipEventDisableSystemFence) != hipSuccess) return;
            c->events.push_back(ev);
        }
    }
    *out = c->events[c->ev_used];
    c->ev_used += 2;
}

void prof_begin(sdsat_ctx* c, int kind, hipEvent_t* out) {
    prof_take(c, kind, out);
    if (*out) (void)hipEventRecord(*out, c->stream);
}

// Event pair for one launch of a profiled kind, taken at the kernel's own start
// and end (hipExtLaunchKernel) rather than recorded around it.
void prof_pair(sdsat_ctx* c, int kind, hipEvent_t* e0, hipEvent_t* e1) {
    *e0 = *e1 = nullptr;
    hipEvent_t s;
    prof_take(c, kind, &s);
    if (!s) return;
    *e0 = s;
    *e1 = c->events[c->ev_used - 1];
}

void prof_end(sdsat_ctx* c, hipEvent_t start) {
    if (!start) return;
    // the stop event follows its start in the pool
    for (size_t i = 0; i + 1 < c->ev_used; i += 2)
        if (c->events[i] == start) { (void)hipEventRecord(c->events[i + 1], c->stream); return; }
}

// ---------------------------------------------------------------- GEMM helpers
int run_gemm(sdsat_ctx* c, int kind, int ep, int M, int n_tiles, int k_steps, int N, int K, const void* W,
             GemmArgs a) {
    const GemmPlan p = ep == EP_RESID ? plan_gemm_resid(M, n_tiles, k_steps) : plan_gemm(M, n_tiles, k_steps);
    a.M = M; a.N = N; a.K = K; a.n_tiles = n_tiles; a.k_steps = k_steps; a.W = W; a.err = c->err_flag;
    a.ksplit = p.ksplit; a.part = c->gemm_part;
    hipEvent_t e0, e1;
    prof_pair(c, kind, &e0, &e1);
    HIPCHK(c, launch_gemm(c->D.dtype, ep, p, a, c->stream, e0, e1));
    return SDSAT_OK;
}

int check_block_args(sdsat_ctx* c, int B, int q) {
    if (B < 1 || q < 1) return fail(c, SDSAT_EINVAL, "batch and q must be >= 1");
    if (B > c->D.maxB) return fail(c, SDSAT_ECAPACITY, "batch exceeds max_batch");
    if (q > c->D.maxQ) return fail(c, SDSAT_ECAPACITY, "q exceeds max_block");
    return SDSAT_OK;
}

int max_hint(sdsat_ctx* c, int B) {
    int m = 0;
    for (int b = 0; b < B; ++b) m = c->len_hint[b] > m ? c->len_hint[b] : m;
    return m;
}

// The host keeps upper bounds of cache_len (commit amounts live on the device).
// When a bound says a block would not fit, read the true lengths once.
int fits(sdsat_ctx* c, int B, int q, bool* ok) {
    *ok = max_hint(c, B) + q <= c->D.S;
    if (*ok) return SDSAT_OK;
    std::vector<int> len(B);
    HIPCHK(c, hipMemcpyAsync(len.data(), c->cache_len, (size_t)B * 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    for (int b = 0; b < B; ++b) c->len_hint[b] = len[b];
    *ok = max_hint(c, B) + q <= c->D.S;
    return SDSAT_OK;
}

int attention_layer(sdsat_ctx* c, int layer, int B, int q, const uint64_t* mask, const float* qbuf, void* out,
                    int out_f32, int ldo) {
    const Dims& D = c->D;
    if (!mask && q > kAttnSplitRows && attention_rows_supported(D.dtype, D.Dh)) {   // prefill: 64-row tiles
        AttnArgs a{};
        a.qbuf = qbuf; a.kc = layer_k(c, layer); a.vc = layer_v(c, layer); a.cache_len = c->cache_len;
        a.B = B; a.q = q; a.H = D.H; a.S_max = D.S; a.scale = (float)(1.0 / std::sqrt((double)D.Dh));
        a.out = out; a.out_f32 = out_f32; a.ldo = ldo; a.err = c->err_flag;
        hipEvent_t e0, e1;
        prof_pair(c, PK_ATTN, &e0, &e1);
        HIPCHK(c, launch_attention_rows(D.dtype, D.Dh, a, c->stream, e0, e1));
        return SDSAT_OK;
    }
    const AttnPlan p = plan_attention(B, D.H, q, D.Dh, max_hint(c, B), D.S);
    if (attention_plan_partial_floats(p, B, D.H, D.Dh) > c->attn_part_floats)   // sized at init for every plan
        return fail(c, SDSAT_EDEVICE, "attention plan needs more split partials than the workspace holds");
    AttnArgs a{};
    a.qbuf = qbuf; a.kc = layer_k(c, layer); a.vc = layer_v(c, layer);
    a.cache_len = c->cache_len; a.per_split = p.per_split; a.mask = mask;
    a.B = B; a.q = q; a.H = D.H; a.S_max = D.S;
    a.scale = (float)(1.0 / std::sqrt((double)D.Dh));
    a.splits = p.splits; a.cols = p.cols; a.part = c->attn_part; a.counter = c->attn_ctr;
    a.out = out; a.out_f32 = out_f32; a.ldo = ldo; a.err = c->err_flag;
    hipEvent_t e0, e1;
    prof_pair(c, PK_ATTN, &e0, &e1);
    HIPCHK(c, launch_attention(D.dtype, D.Dh, p, a, c->stream, e0, e1));
    return SDSAT_OK;
}

// C[M][N] (row stride ldc, float) = A[M][K] (row stride lda) . W[N][K]^T, A and W in the model's element
// type, W the caller's row-major [out, in] weights (up to three of n_per rows each, stacked along N): the
// matrix-core GEMM of large blocks.
// With c_part > 0 (the offset between partial outputs, room for kPrefillMaxSplit of them) a GEMM with
// fewer than 256 tiles and a long contraction is split (prefill_gemm_ksplit); *parts tells the caller how
// many partials to add.
int big_gemm(sdsat_ctx* c, int M, int N, int K, const void* A, int lda, const void* W0, const void* W1,
             const void* W2, int n_per, float* C, int ldc, size_t c_part = 0, int* parts = nullptr) {
    PrefillGemmArgs p{};
    p.M = M; p.N = N; p.K = K; p.A = A; p.lda = lda; p.W0 = W0; p.W1 = W1; p.W2 = W2; p.n_per = n_per;
    p.C = C; p.ldc = ldc;
    p.ksplit = c_part ? prefill_gemm_ksplit(M, N, K) : 1;
    p.c_part = c_part;
    if (parts) *parts = p.ksplit;
    HIPCHK(c, launch_prefill_gemm(c->D.dtype, p, c->stream));
    return SDSAT_OK;
}

// The QKV GEMM of a large block with RoPE, the Q output and the K / V cache writes in its epilogue.
int big_gemm_qkv(sdsat_ctx* c, int B, int q, const void* A, const void* const* w, int l) {
    const Dims& D = c->D;
    PrefillGemmArgs p{};
    p.M = B * q; p.N = 3 * D.d; p.K = D.d; p.A = A; p.lda = D.d_pad;
    p.W0 = w[1]; p.W1 = w[2]; p.W2 = w[3]; p.n_per = D.d; p.ksplit = 1;
    p.ep = PG_QKV; p.q = q; p.H = D.H; p.Dh = D.Dh; p.S_max = D.S; p.cache_len = c->cache_len; p.rope = c->rope;
    p.qbuf = (float*)c->qbuf; p.kc = layer_k(c, l); p.vc = layer_v(c, l); p.err = c->err_flag;
    HIPCHK(c, launch_prefill_gemm(D.dtype, p, c->stream));
    return SDSAT_OK;
}

// The gate | up GEMM of a large block with SwiGLU in its epilogue: u = silu(gate) * up in the element type.
int big_gemm_swiglu(sdsat_ctx* c, int M, const void* A, const void* w_gate, const void* w_up) {
    const Dims& D = c->D;
    PrefillGemmArgs p{};
    p.M = M; p.N = 2 * D.F; p.K = D.d; p.A = A; p.lda = D.d_pad;
    p.W0 = w_gate; p.W1 = w_up; p.n_per = D.F; p.ksplit = 1;
    p.ep = PG_SWIGLU; p.u = c->ubuf; p.ldu = D.F_pad;
    HIPCHK(c, launch_prefill_gemm(D.dtype, p, c->stream));
    return SDSAT_OK;
}

// Block forward of a large block (B*q > kSkinnyRows rows, chain mask): linear layers as matrix-core GEMMs
// on the caller's weights (QKV and gate | up with their RoPE / cache and SwiGLU epilogues), the rest in
// row-wise kernels that round where the skinny path rounds.
int large_block_impl(sdsat_ctx* c, int B, int q, const int32_t* tokens, float* logits) {
    const Dims& D = c->D;
    const int M = B * q;
    const float eps = c->cfg.rms_eps;
    hipEvent_t evb;
    prof_begin(c, logits ? PK_BLOCK : PK_PREFILL, &evb);
    HIPCHK(c, launch_embed(D.dtype, c->embed, D.V + D.A, D.d, tokens, M, c->x, c->xg, c->attn_norm[0], D.d_pad,
                           c->ssq, D.n_ssq, c->err_flag, c->stream));
    // layer 0's normalised input; later layers get theirs from the residual kernel before them
    HIPCHK(c, launch_rms_rows(D.dtype, c->xg, D.d_pad, c->ssq, D.n_ssq, D.d, eps, M, c->hbuf, D.d_pad, c->stream));
    for (int l = 0; l < D.L; ++l) {
        const void* const* w = c->w_src.data() + 1 + 9 * l;   // attn_norm, wq, wk, wv, wo, ffn_norm, wg, wu, wd
        int rc = big_gemm_qkv(c, B, q, c->hbuf, w, l);
        if (rc) return rc;
        rc = attention_layer(c, l, B, q, nullptr, (const float*)c->qbuf, c->obuf, 0, D.d_pad);
        if (rc) return rc;
        const size_t y_part = (size_t)D.maxM * D.d;   // offset between split-K partials in c_y
        int parts = 1;
        rc = big_gemm(c, M, D.d, D.d, c->obuf, D.d_pad, w[4], nullptr, nullptr, D.d, c->c_y, D.d, y_part, &parts);
        if (rc) return rc;
        HIPCHK(c, launch_resid_norm_rows(D.dtype, c->c_y, parts, y_part, D.d, M, D.d, c->x, D.d, c->ffn_norm[l], eps,
                                         c->hbuf, D.d_pad, c->stream));
        rc = big_gemm_swiglu(c, M, c->hbuf, w[6], w[7]);
        if (rc) return rc;
        rc = big_gemm(c, M, D.d, D.F, c->ubuf, D.F_pad, w[8], nullptr, nullptr, D.d, c->c_y, D.d, y_part, &parts);
        if (rc) return rc;
        HIPCHK(c, launch_resid_norm_rows(D.dtype, c->c_y, parts, y_part, D.d, M, D.d, c->x, D.d,
                                         l + 1 < D.L ? c->attn_norm[l + 1] : c->final_norm, eps, c->hbuf, D.d_pad,
                                         c->stream));
    }
    if (logits) {
        int rc = big_gemm(c, M, D.V, D.d, c->hbuf, D.d_pad, c->w_src[2 + 9 * D.L], nullptr, nullptr, D.V, logits, D.V);
        if (rc) return rc;
    }
    prof_end(c, evb);
    return SDSAT_OK;
}

int forward_block_impl(sdsat_ctx* c, int B, int q, const int32_t* tokens, const uint64_t* mask, float* logits) {
    const Dims& D = c->D;
    const int M = B * q;
    if (M > kSkinnyRows) return large_block_impl(c, B, q, tokens, logits);
    // The GEMMs behind an RMSNorm read X either as the float rows x o g, scaled
    // and rounded at the matrix-core input (one-row blocks; QKV up to 8 rows),
    // or as those rows rounded once by rms_rows: every workgroup re-reads X.
    // Both give the same element-type values (same partial-sum order, same
    // rounding).  Measured on the 7B shape at 6 rows: the QKV GEMM's 768
    // workgroups re-reading float rows cost less than an rms_rows launch (block
    // 3.154 -> 3.148 ms), gate/up's 1376 more (3.154 -> 3.194 ms); at 13B's 11
    // rows QKV also loses (6.86 -> 7.14 ms).
    auto norm_input = [&](GemmArgs& g, int float_rows) -> int {
        g.ldx = D.d_pad;
        if (M <= float_rows) {
            g.xf = c->xg; g.ssq = c->ssq; g.n_ssq = D.n_ssq; g.eps = c->cfg.rms_eps;
            return SDSAT_OK;
        }
        HIPCHK(c, launch_rms_rows(D.dtype, c->xg, D.d_pad, c->ssq, D.n_ssq, D.d, c->cfg.rms_eps, M, c->hbuf, D.d_pad,
                                  c->stream));
        g.xa = c->hbuf;
        return SDSAT_OK;
    };
    hipEvent_t evb;
    prof_begin(c, logits ? PK_BLOCK : PK_PREFILL, &evb);
    HIPCHK(c, launch_embed(D.dtype, c->embed, D.V + D.A, D.d, tokens, M, c->x, c->xg, c->attn_norm[0], D.d_pad,
                           c->ssq, D.n_ssq, c->err_flag, c->stream));
    for (int l = 0; l < D.L; ++l) {
        // attention sub-block: RMSNorm -> QKV (+RoPE, KV write) -> attention -> O (+residual);
        // xg holds x o (the gain of the RMSNorm the next GEMM applies)
        GemmArgs a{};
        int rc = norm_input(a, kQkvFloatRows);
        if (rc) return rc;
        a.qbuf = c->qbuf; a.kc = layer_k(c, l); a.vc = layer_v(c, l);
        a.cache_len = c->cache_len; a.q = q; a.H = D.H; a.Dh = D.Dh; a.S_max = D.S; a.mask = mask;
        a.rope = c->rope;
        rc = run_gemm(c, PK_QKV, EP_QKV, M, D.nt_qkv, D.ks_d, 3 * D.d, D.d, c->w_qkv[l], a);
        if (rc) return rc;
        rc = attention_layer(c, l, B, q, mask, (const float*)c->qbuf, c->obuf, 0, D.d_pad);
        if (rc) return rc;
        GemmArgs o{};
        o.xa = c->obuf; o.ldx = D.d_pad; o.resid = c->x; o.ldy = D.d; o.xg_out = c->xg; o.ldxg = D.d_pad;
        o.gnext = c->ffn_norm[l]; o.ssq_out = c->ssq;
        rc = run_gemm(c, PK_O, EP_RESID, M, D.nt_o, D.ks_d, D.d, D.d, c->w_o[l], o);
        if (rc) return rc;
        // feed-forward sub-block: RMSNorm -> gate/up (+SwiGLU) -> down (+residual)
        GemmArgs f{};
        rc = norm_input(f, kPreRoundRows);
        if (rc) return rc;
        f.uout = c->ubuf; f.F = D.F; f.ldu = D.F_pad;
        rc = run_gemm(c, PK_GATEUP, EP_SWIGLU, M, D.nt_gu, D.ks_d, 2 * D.F, D.d, c->w_gu[l], f);
        if (rc) return rc;
        GemmArgs dn{};
        dn.xa = c->ubuf; dn.ldx = D.F_pad; dn.resid = c->x; dn.ldy = D.d; dn.xg_out = c->xg; dn.ldxg = D.d_pad;
        dn.gnext = l + 1 < D.L ? c->attn_norm[l + 1] : c->final_norm; dn.ssq_out = c->ssq;
        rc = run_gemm(c, PK_DOWN, EP_RESID, M, D.nt_down, D.ks_f, D.d, D.F, c->w_down[l], dn);
        if (rc) return rc;
    }
    if (logits) {
        GemmArgs h{};
        int rc = norm_input(h, kPreRoundRows);
        if (rc) return rc;
        h.y = logits; h.ldy = D.V;
        rc = run_gemm(c, PK_LM, EP_STORE, M, D.nt_lm, D.ks_d, D.V, D.d, c->w_lm, h);
        if (rc) return rc;
    }
    prof_end(c, evb);
    return SDSAT_OK;
}

int read_err_flag(sdsat_ctx* c) {
    int h = 0;
    HIPCHK(c, hipMemcpyAsync(&h, c->err_flag, 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    if (h) {
        HIPCHK(c, launch_fill_i32(c->err_flag, 1, 0, c->stream));
        return fail(c, SDSAT_EDATA, (h & 1)   ? "token id out of range in a block"
                                    : (h & 2) ? "invalid commit rows"
                                    : (h & 4) ? "cache capacity exceeded"
                                              : "attention launched for a shorter cache than committed");
    }
    return SDSAT_OK;
}

}  // namespace

int sdsat::report_error(int code, const std::string& msg) { return fail(nullptr, code, msg); }

// ================================================================= C-ABI
extern "C" {

int sdsat_query_sizes(const sdsat_config* cfg, size_t* workspace_bytes) {
    if (!workspace_bytes) return fail(nullptr, SDSAT_EINVAL, "workspace_bytes is NULL");
    sdsat_ctx tmp;
    std::string why;
    int rc = make_dims(cfg, &tmp.D, &why);
    if (rc) return fail(nullptr, rc, why);
    tmp.cfg = *cfg;
    Carver cv(nullptr);
    carve(&tmp, cv);
    *workspace_bytes = align_up(cv.off, 256);
    return SDSAT_OK;
}

int sdsat_init(const sdsat_config* cfg, const void* const* weights, int32_t n_weights, void* workspace,
               size_t workspace_bytes, void* hip_stream, sdsat_ctx** out) {
    if (!out) return fail(nullptr, SDSAT_EINVAL, "out is NULL");
    *out = nullptr;
    sdsat_ctx* c = new (std::nothrow) sdsat_ctx();
    if (!c) return fail(nullptr, SDSAT_ENOMEM, "host allocation failed");
    std::string why;
    int rc = make_dims(cfg, &c->D, &why);
    if (rc) { delete c; return fail(nullptr, rc, why); }
    c->cfg = *cfg;
    const Dims& D = c->D;
    if (!weights || n_weights != 1 + 9 * D.L + 2) {
        delete c;
        return fail(nullptr, SDSAT_EINVAL, "weights must hold 1 + 9*n_layers + 2 pointers");
    }
    for (int i = 0; i < n_weights; ++i)
        if (!weights[i]) { delete c; return fail(nullptr, SDSAT_EINVAL, "a weight pointer is NULL"); }
    if (!workspace || ((uintptr_t)workspace & 255)) {
        delete c;
        return fail(nullptr, SDSAT_EINVAL, "workspace must be non-NULL and 256-byte aligned");
    }
    size_t need = 0;
    sdsat_query_sizes(cfg, &need);
    if (workspace_bytes < need) {
        delete c;
        return fail(nullptr, SDSAT_ENOMEM, "workspace smaller than sdsat_query_sizes()");
    }
    c->stream = (hipStream_t)hip_stream;
    Carver cv(workspace);
    carve(c, cv);
    c->len_hint.assign(D.maxB, 0);
    (void)hipGetDevice(&c->device);

    c->embed = weights[0];
    c->w_src.assign(weights, weights + n_weights);
    c->attn_norm.resize(D.L); c->ffn_norm.resize(D.L);
    for (int l = 0; l < D.L; ++l) {
        const void* const* w = weights + 1 + 9 * l;
        c->attn_norm[l] = (const float*)w[0];
        c->ffn_norm[l] = (const float*)w[5];
        PackArgs p{};
        p.dtype = D.dtype; p.K = D.d; p.k_steps = D.ks_d; p.head_dim = D.Dh; p.F = D.F;
        // Wq, Wk, Wv stacked, rows grouped for RoPE pairs
        p.perm = PACK_ROPE; p.N = 3 * D.d; p.n_tiles = D.nt_qkv; p.src0 = w[1]; p.src1 = w[2]; p.src2 = w[3];
        p.N0 = D.d; p.N1 = D.d; p.dst = c->w_qkv[l];
        launch_pack(p, c->stream);
        p.perm = PACK_PLAIN; p.N = D.d; p.n_tiles = D.nt_o; p.src0 = w[4]; p.src1 = p.src2 = nullptr;
        p.N0 = D.d; p.N1 = 0; p.dst = c->w_o[l];
        launch_pack(p, c->stream);
        // gate and up interleaved per tile
        p.perm = PACK_GATEUP; p.N = 2 * D.F; p.n_tiles = D.nt_gu; p.src0 = w[6]; p.src1 = w[7];
        p.N0 = D.F; p.N1 = D.F; p.dst = c->w_gu[l];
        launch_pack(p, c->stream);
        p.perm = PACK_PLAIN; p.N = D.d; p.K = D.F; p.k_steps = D.ks_f; p.n_tiles = D.nt_down; p.src0 = w[8];
        p.src1 = nullptr; p.N0 = D.d; p.N1 = 0; p.dst = c->w_down[l];
        launch_pack(p, c->stream);
    }
    c->final_norm = (const float*)weights[1 + 9 * D.L];
    {
        PackArgs p{};
        p.dtype = D.dtype; p.K = D.d; p.k_steps = D.ks_d; p.perm = PACK_PLAIN; p.N = D.V; p.n_tiles = D.nt_lm;
        p.src0 = weights[2 + 9 * D.L]; p.N0 = D.V; p.dst = c->w_lm;
        launch_pack(p, c->stream);
    }
    auto init_fail = [&](int code) { std::string m = c->err; delete c; return fail(nullptr, code, m); };
    if (hipGetLastError() != hipSuccess) { c->err = "weight packing launch failed"; return init_fail(SDSAT_EDEVICE); }
    // rotary inverse frequencies base^(-2i/Dh) in double, and the table of cos / sin
    // of pos * inv_freq (formed in double, rounded to float) the QKV epilogue reads
    {
        const int half = D.Dh / 2;
        std::vector<double> inv(half);
        for (int i = 0; i < half; ++i) inv[i] = std::pow((double)cfg->rope_base, -2.0 * i / D.Dh);
        if (hipMemcpyAsync(c->inv_freq, inv.data(), inv.size() * 8, hipMemcpyHostToDevice, c->stream) != hipSuccess) {
            c->err = "rotary table upload failed";
            return init_fail(SDSAT_EDEVICE);
        }
        if (launch_rope_table(c->inv_freq, D.S, half, c->rope, c->stream) != hipSuccess) {
            c->err = "rotary table launch failed";
            return init_fail(SDSAT_EDEVICE);
        }
        if (hipStreamSynchronize(c->stream) != hipSuccess) {   // the host vector goes out of scope
            c->err = "rotary table upload failed";
            return init_fail(SDSAT_EDEVICE);
        }
        // KV cache starts zero-filled: slots past a sequence's keys are read (and masked) inside
        // 32-key blocks, so they must hold finite values
        const size_t kv_words = c->layer_elems * D.L * D.esz / 4;
        if (launch_fill_i32((int*)c->kc, kv_words, 0, c->stream) != hipSuccess ||
            launch_fill_i32((int*)c->vc, kv_words, 0, c->stream) != hipSuccess) {
            c->err = "cache fill failed";
            return init_fail(SDSAT_EDEVICE);
        }
        // activation pads must read as zero
        (void)launch_fill_i32((int*)c->xg, (size_t)D.maxM * D.d_pad, 0, c->stream);
        (void)launch_fill_i32((int*)c->obuf, (size_t)D.maxM * D.d_pad * D.esz / 4, 0, c->stream);
        (void)launch_fill_i32((int*)c->ubuf, (size_t)D.maxM * D.F_pad * D.esz / 4, 0, c->stream);
        (void)launch_fill_i32((int*)c->hbuf, (size_t)D.maxM * D.d_pad * D.esz / 4, 0, c->stream);
        (void)launch_fill_i32(c->verify_cnt, D.maxB, 0, c->stream);
        (void)launch_fill_i32(c->attn_ctr, attention_counter_ints(D.maxB, D.H, D.maxQ), 0, c->stream);
        (void)launch_fill_i32(c->cache_len, D.maxB, 0, c->stream);
        (void)launch_fill_i32(c->err_flag, 1, 0, c->stream);
        if (hipStreamSynchronize(c->stream) != hipSuccess) {
            c->err = std::string("init failed: ") + hipGetErrorString(hipGetLastError());
            return init_fail(SDSAT_EDEVICE);
        }
    }
    c->h_pin_ints = (size_t)D.maxB * D.maxQ * 4 + 64;
    if (hipHostMalloc((void**)&c->h_pin, c->h_pin_ints * 4, hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc((void**)&c->h_rec, (size_t)kRecLoops * D.maxB * kLoopRecCols * 4, hipHostMallocDefault) !=
            hipSuccess) {
        c->err = "pinned host allocation failed";
        return init_fail(SDSAT_ENOMEM);
    }
    *out = c;
    return SDSAT_OK;
}

int sdsat_reset(sdsat_ctx* c, int32_t batch) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    if (batch < 1 || batch > c->D.maxB) return fail(c, SDSAT_EINVAL, "batch out of range");
    HIPCHK(c, launch_set_len(c->cache_len, batch, nullptr, 0, c->stream));
    for (int b = 0; b < batch; ++b) c->len_hint[b] = 0;
    return SDSAT_OK;
}

int sdsat_set_cache_len(sdsat_ctx* c, int32_t batch, const int32_t* h_len) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    if (batch < 1 || batch > c->D.maxB || !h_len) return fail(c, SDSAT_EINVAL, "bad batch or h_len");
    for (int b = 0; b < batch; ++b)
        if (h_len[b] < 0 || h_len[b] > c->D.S) return fail(c, SDSAT_ECAPACITY, "length exceeds max_ctx");
    // stage through the pinned buffer; wait so the staging can be reused
    HIPCHK(c, hipStreamSynchronize(c->stream));
    std::memcpy(c->h_pin, h_len, (size_t)batch * 4);
    HIPCHK(c, hipMemcpyAsync(c->n_commit, c->h_pin, (size_t)batch * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, launch_set_len(c->cache_len, batch, c->n_commit, 0, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    for (int b = 0; b < batch; ++b) c->len_hint[b] = h_len[b];
    return SDSAT_OK;
}

const int32_t* sdsat_cache_len_ptr(const sdsat_ctx* c) { return c ? c->cache_len : nullptr; }

int sdsat_forward_block(sdsat_ctx* c, int32_t batch, int32_t q, const int32_t* d_tokens,
                        const uint64_t* d_ancestor_mask, float* d_logits) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    int rc = check_block_args(c, batch, q);
    if (rc) return rc;
    if (!d_tokens) return fail(c, SDSAT_EINVAL, "d_tokens is NULL");
    if (batch * q > kSkinnyRows && d_ancestor_mask)
        return fail(c, SDSAT_EUNSUPPORTED, "ancestor masks need batch * q <= 64");
    bool ok = false;
    rc = fits(c, batch, q, &ok);
    if (rc) return rc;
    if (!ok) return fail(c, SDSAT_ECAPACITY, "cache_len + q exceeds max_ctx");
    return forward_block_impl(c, batch, q, d_tokens, d_ancestor_mask, d_logits);
}

int sdsat_verify_greedy(sdsat_ctx* c, int32_t batch, int32_t q, const float* d_logits, const int32_t* d_drafts,
                        int32_t* d_tokens_out, int32_t* d_n_accept) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    int rc = check_block_args(c, batch, q);
    if (rc) return rc;
    if (!d_logits || !d_tokens_out || (d_drafts && !d_n_accept))
        return fail(c, SDSAT_EINVAL, "NULL logits, tokens_out, or n_accept with drafts");
    HIPCHK(c, launch_verify_greedy(d_logits, batch, q, c->D.V, d_drafts, q - 1, d_tokens_out, d_n_accept,
                                   c->verify_cnt, c->stream));
    return SDSAT_OK;
}

int sdsat_verify_nucleus(sdsat_ctx* c, int32_t batch, int32_t q, const float* d_logits, const int32_t* d_drafts,
                         float temperature, float top_p, int32_t top_k, uint64_t seed, const int32_t* d_pos0,
                         int32_t* d_tokens_out, int32_t* d_n_accept) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    int rc = check_block_args(c, batch, q);
    if (rc) return rc;
    if (!d_logits || !d_tokens_out || !d_pos0 || (d_drafts && !d_n_accept))
        return fail(c, SDSAT_EINVAL, "NULL logits, tokens_out, pos0, or n_accept with drafts");
    if (c->D.V > 131072) return fail(c, SDSAT_EUNSUPPORTED, "nucleus verification needs vocab <= 131072");
    if (!(top_p > 0.f) || std::isnan(temperature)) return fail(c, SDSAT_EINVAL, "top_p must be > 0");
    HIPCHK(c, launch_verify_nucleus(d_logits, batch, q, c->D.V, d_drafts, q - 1, temperature, top_p, top_k, seed,
                                    d_pos0, d_tokens_out, d_n_accept, c->verify_cnt, c->stream));
    return SDSAT_OK;
}

int sdsat_commit_kv(sdsat_ctx* c, int32_t batch, int32_t q, const int32_t* d_n_commit, const int32_t* d_rows) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    int rc = check_block_args(c, batch, q);
    if (rc) return rc;
    if (!d_n_commit) return fail(c, SDSAT_EINVAL, "d_n_commit is NULL");
    const Dims& D = c->D;
    if (d_rows)
        HIPCHK(c, launch_commit_gather(D.dtype, c->kc, c->vc, c->layer_elems, D.L, batch, D.H, D.Dh, D.S,
                                       c->cache_len, d_n_commit, d_rows, q, c->err_flag, c->stream));
    HIPCHK(c, launch_commit(c->cache_len, batch, d_n_commit, D.S, c->err_flag, c->stream));
    for (int b = 0; b < batch; ++b) c->len_hint[b] = std::min(c->len_hint[b] + q, D.S);
    return SDSAT_OK;
}

}  // extern "C"

namespace {

// The generation loop of sdsat_generate; with h_ref, draft step 2 takes its drafts d_1..d_k of
// sequence b from h_ref[b][n+1..n+k] (n = tokens emitted so far) instead of draft step 1's rows.
int generate_impl(sdsat_ctx* c, int32_t batch, const int32_t* h_prompts, int32_t P, int32_t max_new, int32_t k,
                  int32_t width, const int32_t* h_adaptive_ids, int32_t mode, float temperature, float top_p,
                  int32_t top_k, uint64_t seed, const int32_t* h_ref, int32_t ref_len, int32_t* h_out,
                  sdsat_stats* h_stats) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    const Dims& D = c->D;
    if (batch < 1 || batch > D.maxB) return fail(c, SDSAT_ECAPACITY, "batch exceeds max_batch");
    if (!h_prompts || !h_out || P < 1 || max_new < 0 || k < 0) return fail(c, SDSAT_EINVAL, "bad prompts/out/P/k");
    if (k > 0 && !h_adaptive_ids) return fail(c, SDSAT_EINVAL, "h_adaptive_ids is NULL");
    const int q = k + 1;
    if (width < 1 || width > kMaxTreeWidth) return fail(c, SDSAT_EINVAL, "tree width must be 1..8");
    const bool tree = width > 1 && k > 0;
    const int q2 = tree ? 1 + k * width : q;   // rows of draft step 2 (the tree block)
    if (q2 > D.maxQ) return fail(c, SDSAT_ECAPACITY, "k + 1 (tree: 1 + k * width) exceeds max_block");
    if (batch * q2 > 64) return fail(c, SDSAT_ECAPACITY, "batch * (k + 1) (tree: 1 + k * width) must be <= 64");
    if (mode != SDSAT_MODE_GREEDY && mode != SDSAT_MODE_NUCLEUS) return fail(c, SDSAT_EINVAL, "bad mode");
    const bool nucleus = mode == SDSAT_MODE_NUCLEUS && temperature > 0.f;
    if (nucleus && D.V > 131072) return fail(c, SDSAT_EUNSUPPORTED, "nucleus verification needs vocab <= 131072");
    for (int j = 0; j < k; ++j)
        if (h_adaptive_ids[j] < 0 || h_adaptive_ids[j] >= D.V + D.A)
            return fail(c, SDSAT_EINVAL, "adaptive id out of range");
    // A sequence's last loop starts below max_new tokens and may overshoot to max_new + k + 1, i.e.
    // cache_len P + max_new + k.  With batch > 1 a finished sequence keeps riding along (commit 0), its
    // blocks written at that cache_len, so its rows reach slot P + max_new + k + q2 - 1.
    const long need = (long)P + max_new + q2 + (batch > 1 ? k : 0);
    if (need > D.S) return fail(c, SDSAT_ECAPACITY, "prompt + max_new (+ k + 1 rows for batch > 1) exceeds max_ctx");
    for (long i = 0; i < (long)batch * P; ++i)
        if (h_prompts[i] < 0 || h_prompts[i] >= D.V + D.A) return fail(c, SDSAT_EINVAL, "prompt id out of range");

    sdsat_stats st;
    std::memset(&st, 0, sizeof(st));
    using clk = std::chrono::steady_clock;
    HIPCHK(c, hipStreamSynchronize(c->stream));
    const auto t0 = clk::now();
    int rc = sdsat_reset(c, batch);
    if (rc) return rc;
    // prefill: prompt tokens 0..P-2 in blocks of up to max_block rows per sequence
    const int qc = D.maxQ;
    for (int lo = 0; lo < P - 1; lo += qc) {
        const int n = std::min(qc, P - 1 - lo);
        for (int b = 0; b < batch; ++b)
            for (int r = 0; r < n; ++r) c->h_pin[b * n + r] = h_prompts[(size_t)b * P + lo + r];
        HIPCHK(c, hipMemcpyAsync(c->ptok, c->h_pin, (size_t)batch * n * 4, hipMemcpyHostToDevice, c->stream));
        rc = forward_block_impl(c, batch, n, c->ptok, nullptr, nullptr);
        if (rc) return rc;
        HIPCHK(c, launch_fill_i32(c->n_commit, batch, n, c->stream));
        HIPCHK(c, launch_commit(c->cache_len, batch, c->n_commit, D.S, c->err_flag, c->stream));
        for (int b = 0; b < batch; ++b) c->len_hint[b] += n;
        HIPCHK(c, hipStreamSynchronize(c->stream));   // the pinned staging buffer is reused
        st.prefill_blocks++;
    }
    for (int b = 0; b < batch; ++b) c->h_pin[b] = h_prompts[(size_t)b * P + P - 1];
    for (int j = 0; j < k; ++j) c->h_pin[batch + j] = h_adaptive_ids[j];
    HIPCHK(c, hipMemcpyAsync(c->pending, c->h_pin, (size_t)batch * 4, hipMemcpyHostToDevice, c->stream));
    if (k) HIPCHK(c, hipMemcpyAsync(c->adaptive, c->h_pin + batch, (size_t)k * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    rc = read_err_flag(c);
    if (rc) return rc;
    const auto t1 = clk::now();

    std::vector<int> produced(batch, 0);
    std::vector<int> len_exact(c->len_hint.begin(), c->len_hint.begin() + batch);
    // the device tracks each sequence's progress (produced, active) so that loops run back to back;
    // every sequence starts active
    for (int b = 0; b < batch; ++b) c->h_pin[b] = max_new > 0 ? 1 : 0;
    HIPCHK(c, hipMemcpyAsync(c->active, c->h_pin, (size_t)batch * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, launch_fill_i32(c->produced, batch, 0, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));   // the pinned staging buffer is reused
    int* h_err = c->h_pin;
    const size_t rec_stride = (size_t)D.maxB * kLoopRecCols;
    for (;;) {
        // Loops of this batch: as many as the least advanced active sequence needs at the least
        // (k + 2 tokens per loop), so every loop of the batch has an active sequence.  Drafts taken
        // from a reference depend on the host's counts: one loop per batch then.
        int minp = -1;
        for (int b = 0; b < batch; ++b)
            if (produced[b] < max_new && (minp < 0 || produced[b] < minp)) minp = produced[b];
        if (minp < 0) break;
        const int n_b = h_ref ? 1 : std::min(kRecLoops, std::max(1, (max_new - minp + k + 1) / (k + 2)));
        for (int i = 0; i < n_b; ++i) {
            // upper bounds of the cache lengths for the attention plans (an over-estimate only adds
            // empty key splits); the exact lengths are restored after the batch
            if (i > 0)
                for (int b = 0; b < batch; ++b)
                    if (produced[b] < max_new) c->len_hint[b] = std::min(D.S, c->len_hint[b] + k + 1);
            // draft step 1 (Eq. 1): [pending, a_1..a_k]
            HIPCHK(c, launch_build_draft1(c->pending, c->adaptive, batch, k, c->tok1, c->stream));
            rc = forward_block_impl(c, batch, q, c->tok1, nullptr, c->logits);
            if (rc) return rc;
            if (nucleus) {
                HIPCHK(c, launch_pos0(c->cache_len, batch, 1, c->pos0, c->stream));
                HIPCHK(c, launch_verify_nucleus(c->logits, batch, q, D.V, nullptr, q - 1, temperature, top_p, top_k,
                                                seed, c->pos0, c->out1, nullptr, c->verify_cnt, c->stream));
            } else {
                HIPCHK(c, launch_verify_greedy(c->logits, batch, q, D.V, nullptr, q - 1, c->out1, nullptr,
                                               c->verify_cnt, c->stream));
            }
            HIPCHK(c, launch_commit(c->cache_len, batch, c->active, D.S, c->err_flag, c->stream));   // keep row 0
            for (int b = 0; b < batch; ++b)
                if (produced[b] < max_new) c->len_hint[b] = std::min(D.S, c->len_hint[b] + 1);
            if (h_ref && k > 0) {   // drafts from the reference continuation (pinned staging after h_err)
                int* dr = h_err + 1;
                for (int b = 0; b < batch; ++b)
                    for (int j = 0; j < k; ++j) {
                        const long idx = (long)produced[b] + 1 + j;
                        dr[b * k + j] = idx < ref_len ? h_ref[(size_t)b * ref_len + idx] : 0;
                    }
                HIPCHK(c, hipMemcpy2DAsync(c->out1 + 1, (size_t)q * 4, dr, (size_t)k * 4, (size_t)k * 4, batch,
                                           hipMemcpyHostToDevice, c->stream));
            }
            if (tree) {
                // draft step 2 over the tree (Section 2.1.2): candidates of draft step 1's adaptive rows, rows
                // at position L + depth seeing their ancestors; the target's token at every node; the longest
                // confirmed branch; its rows gathered to slots L.. and committed, pending = the last token
                HIPCHK(c, launch_tree_build(c->logits, batch, q, D.V, c->out1, k, width, q2, c->tree_tok,
                                            c->tree_mask, c->tree_depth, c->stream));
                rc = forward_block_impl(c, batch, q2, c->tree_tok, c->tree_mask, c->logits);
                if (rc) return rc;
                if (nucleus) {
                    HIPCHK(c, launch_pos0(c->cache_len, batch, 1, c->pos0, c->stream));
                    HIPCHK(c, launch_verify_nucleus(c->logits, batch, q2, D.V, nullptr, 0, temperature, top_p, top_k,
                                                    seed, c->pos0, c->tree_target, nullptr, c->verify_cnt, c->stream,
                                                    c->tree_depth));
                } else {
                    HIPCHK(c, launch_verify_greedy(c->logits, batch, q2, D.V, nullptr, 0, c->tree_target, nullptr,
                                                   c->verify_cnt, c->stream));
                }
                HIPCHK(c, launch_tree_walk(batch, q2, k, width, c->tree_tok, c->tree_target, c->active, c->out2,
                                           c->n_accept, c->tree_rows, c->pending, c->n_commit, c->stream));
                HIPCHK(c, launch_commit_gather(D.dtype, c->kc, c->vc, c->layer_elems, D.L, batch, D.H, D.Dh, D.S,
                                               c->cache_len, c->n_commit, c->tree_rows, q2, c->err_flag, c->stream));
                HIPCHK(c, launch_commit(c->cache_len, batch, c->n_commit, D.S, c->err_flag, c->stream));
            } else {
                // draft step 2 (Eq. 2): [t1, d_1..d_k] = out1
                rc = forward_block_impl(c, batch, q, c->out1, nullptr, c->logits);
                if (rc) return rc;
                if (nucleus) {
                    HIPCHK(c, launch_pos0(c->cache_len, batch, 1, c->pos0, c->stream));
                    HIPCHK(c, launch_verify_nucleus(c->logits, batch, q, D.V, c->out1 + 1, q, temperature, top_p,
                                                    top_k, seed, c->pos0, c->out2, c->n_accept, c->verify_cnt,
                                                    c->stream));
                } else {
                    HIPCHK(c, launch_verify_greedy(c->logits, batch, q, D.V, c->out1 + 1, q, c->out2, c->n_accept,
                                                   c->verify_cnt, c->stream));
                }
                // verification (Eq. 3): commit rows 0..m, pending = o_m
                HIPCHK(c, launch_loop_commit(c->cache_len, batch, q, c->active, c->n_accept, c->out2, c->pending,
                                             c->n_commit, c->stream));
            }
            HIPCHK(c, launch_loop_record(c->loop_rec + i * rec_stride, batch, q, q2, k, max_new, c->out1, c->out2,
                                         c->n_accept, c->active, c->produced, c->stream));
        }
        HIPCHK(c, hipMemcpyAsync(c->h_rec, c->loop_rec, (size_t)n_b * rec_stride * 4, hipMemcpyDeviceToHost,
                                 c->stream));
        HIPCHK(c, hipMemcpyAsync(h_err, c->err_flag, 4, hipMemcpyDeviceToHost, c->stream));
        HIPCHK(c, hipStreamSynchronize(c->stream));
        if (*h_err) {
            rc = read_err_flag(c);
            return rc ? rc : fail(c, SDSAT_EDATA, "device error flag set");
        }
        // replay the batch's records with the same rule the device used for activity
        for (int i = 0; i < n_b; ++i) {
            const int* rec = c->h_rec + i * rec_stride;
            st.loops++;
            st.blocks += 2;
            for (int b = 0; b < batch; ++b) {
                if (produced[b] >= max_new) continue;
                const int* r = rec + (size_t)b * kLoopRecCols;
                const int m = r[0];
                if (m < 0 || m > k) return fail(c, SDSAT_EDEVICE, "verification returned an invalid prefix length");
                st.accepted += m;
                st.accept_hist[m]++;
                st.tokens += m + 2;
                int* row = h_out + (size_t)b * max_new;
                row[produced[b]++] = r[1];
                for (int j = 0; j <= m && produced[b] < max_new; ++j) row[produced[b]++] = r[2 + j];
                len_exact[b] += m + 2;
            }
        }
        for (int b = 0; b < batch; ++b) c->len_hint[b] = len_exact[b];
    }
    const auto t2 = clk::now();
    st.prefill_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
    st.decode_ms = std::chrono::duration<double, std::milli>(t2 - t1).count();
    if (h_stats) *h_stats = st;
    return SDSAT_OK;
}

}  // namespace

extern "C" {

int sdsat_generate(sdsat_ctx* c, int32_t batch, const int32_t* h_prompts, int32_t P, int32_t max_new, int32_t k,
                   const int32_t* h_adaptive_ids, int32_t mode, float temperature, float top_p, int32_t top_k,
                   uint64_t seed, int32_t* h_out, sdsat_stats* h_stats) {
    return generate_impl(c, batch, h_prompts, P, max_new, k, 1, h_adaptive_ids, mode, temperature, top_p, top_k,
                         seed, nullptr, 0, h_out, h_stats);
}

int sdsat_generate_tree(sdsat_ctx* c, int32_t batch, const int32_t* h_prompts, int32_t P, int32_t max_new,
                        int32_t k, int32_t width, const int32_t* h_adaptive_ids, int32_t mode, float temperature,
                        float top_p, int32_t top_k, uint64_t seed, int32_t* h_out, sdsat_stats* h_stats) {
    return generate_impl(c, batch, h_prompts, P, max_new, k, width, h_adaptive_ids, mode, temperature, top_p, top_k,
                         seed, nullptr, 0, h_out, h_stats);
}

int sdsat_generate_forced(sdsat_ctx* c, int32_t batch, const int32_t* h_prompts, int32_t P, int32_t max_new,
                          int32_t k, const int32_t* h_adaptive_ids, int32_t mode, float temperature, float top_p,
                          int32_t top_k, uint64_t seed, const int32_t* h_ref, int32_t ref_len, int32_t* h_out,
                          sdsat_stats* h_stats) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    if (!h_ref || ref_len < 1) return fail(c, SDSAT_EINVAL, "h_ref is NULL or ref_len < 1");
    for (long i = 0; i < (long)batch * ref_len; ++i)
        if (h_ref[i] < 0 || h_ref[i] >= c->D.V + c->D.A) return fail(c, SDSAT_EINVAL, "reference id out of range");
    return generate_impl(c, batch, h_prompts, P, max_new, k, 1, h_adaptive_ids, mode, temperature, top_p, top_k,
                         seed, h_ref, ref_len, h_out, h_stats);
}

int sdsat_kv_write(sdsat_ctx* c, int32_t layer, int32_t batch, int32_t n, const float* d_k, const float* d_v,
                   const int32_t* d_pos) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    const Dims& D = c->D;
    if (layer < 0 || layer >= D.L || batch < 1 || batch > D.maxB || n < 0 || !d_k || !d_v || !d_pos)
        return fail(c, SDSAT_EINVAL, "bad kv_write arguments");
    HIPCHK(c, launch_kv_write(D.dtype, layer_k(c, layer), layer_v(c, layer), batch, n, D.H, D.Dh, D.S, d_k, d_v,
                              d_pos, c->stream));
    return SDSAT_OK;
}

int sdsat_attention(sdsat_ctx* c, int32_t layer, int32_t batch, int32_t q, const float* d_q,
                    const uint64_t* d_ancestor_mask, float* d_out) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    int rc = check_block_args(c, batch, q);
    if (rc) return rc;
    const Dims& D = c->D;
    if (layer < 0 || layer >= D.L || !d_q || !d_out) return fail(c, SDSAT_EINVAL, "bad attention arguments");
    bool ok = false;
    rc = fits(c, batch, q, &ok);
    if (rc) return rc;
    if (!ok) return fail(c, SDSAT_ECAPACITY, "cache_len + q exceeds max_ctx");
    HIPCHK(c, hipMemcpyAsync(c->qbuf, d_q, (size_t)batch * q * D.d * 4, hipMemcpyDeviceToDevice, c->stream));
    return attention_layer(c, layer, batch, q, d_ancestor_mask, (const float*)c->qbuf, d_out, 1, D.d);
}

size_t sdsat_linear_packed_bytes(int32_t dtype, int32_t N, int32_t K) {
    if (N < 1 || K < 1) return 0;
    return packed_elems((N + 15) / 16, (K + 31) / 32) * (dtype == SDSAT_DTYPE_BF16 ? 2 : 4);
}

int sdsat_linear_pack(int32_t dtype, int32_t N, int32_t K, const void* d_w, void* d_packed, void* hip_stream) {
    if ((dtype != 0 && dtype != 1) || N < 1 || K < 1 || !d_w || !d_packed)
        return fail(nullptr, SDSAT_EINVAL, "bad linear_pack arguments");
    PackArgs p{};
    p.dtype = dtype; p.N = N; p.K = K; p.n_tiles = (N + 15) / 16; p.k_steps = (K + 31) / 32; p.perm = PACK_PLAIN;
    p.src0 = d_w; p.N0 = N; p.dst = d_packed;
    launch_pack(p, (hipStream_t)hip_stream);
    if (hipGetLastError() != hipSuccess) return fail(nullptr, SDSAT_EDEVICE, "pack launch failed");
    return SDSAT_OK;
}

size_t sdsat_linear_scratch_bytes(int32_t M, int32_t N, int32_t K) {
    if (M < 1 || M > 64 || N < 1 || K < 1) return 0;
    return align_up((size_t)M * align_up((size_t)K, 32) * 4, 256);   // x converted to the matrix type
}

int sdsat_linear(int32_t dtype, int32_t M, int32_t N, int32_t K, const float* d_x, const void* d_packed, float* d_y,
                 void* d_scratch, void* hip_stream) {
    if ((dtype != 0 && dtype != 1) || M < 1 || M > 64 || N < 1 || K < 1 || !d_x || !d_packed || !d_y || !d_scratch)
        return fail(nullptr, SDSAT_EINVAL, "bad linear arguments");
    const int nt = (N + 15) / 16, ks = (K + 31) / 32;
    hipStream_t st = (hipStream_t)hip_stream;
    hipError_t e = launch_to_elem_rows(dtype, d_x, M, K, d_scratch, ks * 32, st);
    if (e != hipSuccess) return fail(nullptr, SDSAT_EDEVICE, std::string("linear input: ") + hipGetErrorString(e));
    const GemmPlan p = plan_gemm(M, nt, ks);
    GemmArgs a{};
    a.M = M; a.N = N; a.K = K; a.n_tiles = nt; a.k_steps = ks; a.W = d_packed;
    a.xa = d_scratch; a.ldx = ks * 32; a.y = d_y; a.ldy = N;
    e = launch_gemm(dtype, EP_STORE, p, a, st);
    if (e != hipSuccess) return fail(nullptr, SDSAT_EDEVICE, std::string("linear launch: ") + hipGetErrorString(e));
    return SDSAT_OK;
}

int sdsat_profile_kernel(sdsat_ctx* c, int32_t kind, int32_t period) {
    if (!c) return fail(nullptr, SDSAT_EINVAL, "ctx is NULL");
    if (kind < 0 || kind > 8) return fail(c, SDSAT_EINVAL, "bad kernel kind");
    if (period < 1) return fail(c, SDSAT_EINVAL, "period must be >= 1");
    HIPCHK(c, hipStreamSynchronize(c->stream));
    c->prof_kind = kind;
    c->prof_period = period;
    c->prof_seen = 0;
    c->ev_used = 0;
    return SDSAT_OK;
}

int sdsat_kernel_time(sdsat_ctx* c, double* total_ms, int64_t* launches) {
    if (!c || !total_ms || !launches) return fail(c, SDSAT_EINVAL, "NULL argument");
    HIPCHK(c, hipStreamSynchronize(c->stream));
    double tot = 0.0;
    for (size_t i = 0; i + 1 < c->ev_used; i += 2) {
        float ms = 0.f;
        HIPCHK(c, hipEventElapsedTime(&ms, c->events[i], c->events[i + 1]));
        tot += ms;
    }
    *total_ms = tot;
    *launches = (int64_t)(c->ev_used / 2);
    c->ev_used = 0;
    return SDSAT_OK;
}

int sdsat_kernel_samples(sdsat_ctx* c, float* h_ms, int64_t cap, int64_t* launches) {
    if (!c || !launches || (cap > 0 && !h_ms) || cap < 0) return fail(c, SDSAT_EINVAL, "bad argument");
    HIPCHK(c, hipStreamSynchronize(c->stream));
    int64_t n = 0;
    for (size_t i = 0; i + 1 < c->ev_used; i += 2, ++n) {
        float ms = 0.f;
        HIPCHK(c, hipEventElapsedTime(&ms, c->events[i], c->events[i + 1]));
        if (n < cap) h_ms[n] = ms;
    }
    *launches = n;
    c->ev_used = 0;
    return SDSAT_OK;
}

int sdsat_stream_read(const void* d_src, size_t bytes, void* hip_stream) {
    if (!d_src && bytes) return fail(nullptr, SDSAT_EINVAL, "d_src is NULL");
    if (bytes % 16) return fail(nullptr, SDSAT_EINVAL, "bytes must be a multiple of 16");
    const hipError_t e = launch_stream_read(d_src, bytes, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(nullptr, SDSAT_EDEVICE, std::string("stream read: ") + hipGetErrorString(e));
    return SDSAT_OK;
}

int sdsat_destroy(sdsat_ctx* c) {
    if (!c) return SDSAT_OK;
    (void)hipStreamSynchronize(c->stream);
    delete c;
    return SDSAT_OK;
}

const char* sdsat_last_error(const sdsat_ctx* c) { return c ? c->err.c_str() : g_init_error.c_str(); }

}  // extern "C"
