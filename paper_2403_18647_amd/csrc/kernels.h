// Internal launcher interface between the host runtime (api.cpp) and the HIP
// kernels.  Not part of the public C-ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

namespace sdsat {

// ---------------------------------------------------------------- packed weights
// A matrix W [N, K] is stored as 16-column tiles x 32-wide contraction steps:
// packed[tile][kstep][lane][8] with lane l holding row perm(tile, l % 16) and
// k = 32*kstep + 8*(l/16) + 0..7 (zero past K or past N).  The row permutation
// groups rows so that an epilogue finds partner rows in the same tile:
enum PackPerm {
    PACK_PLAIN = 0,   // tile t, column c -> row 16t + c
    PACK_ROPE = 1,    // rows in heads of Dh: tile j of a head holds pair indices 8j..8j+7,
                      // column c<8 -> row 8j+c, c>=8 -> row Dh/2 + 8j + c-8
    PACK_GATEUP = 2,  // two stacked [F, K] matrices (gate then up): tile t, c<8 -> gate row 8t+c,
                      // c>=8 -> up row 8t+c-8
};

struct PackArgs {
    int dtype;          // 0 fp32, 1 bf16
    int N, K;           // rows / columns of the (stacked) source
    int n_tiles, k_steps;
    int perm, head_dim, F;
    const void* src0;   // rows [0, N0)
    const void* src1;   // rows [N0, N0+N1) (stacked second matrix) or null
    const void* src2;
    int N0, N1;         // row counts of src0, src1 (src2 takes the rest)
    void* dst;
};
void launch_pack(const PackArgs& a, hipStream_t s);
size_t packed_elems(int n_tiles, int k_steps);

// ---------------------------------------------------------------- skinny GEMM
// One workgroup per 16-column tile (or 4 tiles for prefill chunks); its waves
// split the contraction and reduce through LDS.  X rows are read straight from
// global memory as matrix-core fragments, either
//  * stored in the matrix element type with a row stride that covers the
//    32-padded contraction length, zero past K (xa), or
//  * as the float rows x o g of an RMSNorm input (xf, gain already applied):
//    each element is scaled by its row's 1/sqrt(mean(x^2) + eps) and rounded
//    to the element type at the matrix-core input, the value a bf16 model
//    stores as the normalised activation.
enum Epilogue { EP_STORE = 0, EP_QKV = 1, EP_RESID = 2, EP_SWIGLU = 3 };

struct GemmArgs {
    int M, N, K;             // rows of X; real output columns; real contraction length
    int n_tiles, k_steps;    // packed tile counts
    const void* W;           // packed weights
    const void* xa;          // T [M][ldx], or null when xf is given
    const float* xf;         // float [M][ldx]: x o gain of the RMSNorm this GEMM consumes
    int ldx;
    // RMSNorm row scales: 1/sqrt(sum_t ssq[m][t] / K + eps) (with xf)
    const float* ssq; int n_ssq; float eps;
    // epilogues
    float* y; int ldy;                   // EP_STORE: float [M][ldy]
    float* resid;                        // EP_RESID: float [M][ldy] (+=)
    float* xg_out; int ldxg;             // EP_RESID: updated rows times gnext (the next RMSNorm's gain)
    const float* gnext;
    float* ssq_out;                      // EP_RESID: per-tile sums of squares [M][n_tiles]
    void* qbuf; void* kc; void* vc;      // EP_QKV: Q float [M][H][Dh]; layer base of K and V caches
    const int* cache_len; int q, H, Dh, S_max;
    const uint64_t* mask;                // [M] ancestor masks or null (chain)
    const float* rope;                   // [S_max][Dh/2][2] rotary cos, sin of position x base^(-2i/Dh)
    void* uout; int F; int ldu;          // EP_SWIGLU: T [M][ldu]
    int* err;                            // device error flags (bit 4: write past the cache)
    // EP_RESID split over ksplit workgroups per tile (ksplit > 1): every wave's raw partial tile goes to
    // part [n_tiles][waves * ksplit][MT][64] (f32x4), folded in wave order by a second kernel
    int ksplit; float* part;
};

struct GemmPlan {
    int waves, mt, ntw, grid, lds_bytes;   // ntw: 16-column tiles per workgroup; waves per workgroup
    int ksplit;                            // workgroups per column tile (EP_RESID only), 1 = one
};
GemmPlan plan_gemm(int M, int n_tiles, int k_steps);
// The residual GEMMs' plan with each tile's waves spread over ksplit workgroups where that balances
// the compute units (same wave slices, same fold order: the same values).
GemmPlan plan_gemm_resid(int M, int n_tiles, int k_steps);
// bytes of the partial-tile buffer the residual GEMMs of this shape need (0: never split)
size_t gemm_resid_part_bytes(int n_tiles, int k_steps, int max_rows);
// ev0 / ev1 (optional): events taken at the kernel's own start and end (its
// dispatch packet's timestamps), for timing one launch
hipError_t launch_gemm(int dtype, int ep, const GemmPlan& p, const GemmArgs& a, hipStream_t s,
                       hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

// ---------------------------------------------------------------- attention
struct AttnArgs {
    const float* qbuf;       // float [B*q][H][Dh]
    const void* kc;          // T K cache of one layer: [B][H][S_max][Dh]
    const void* vc;          // T V cache of one layer: [B][H][S_max/32][Dh][32] (keys permuted, vperm)
    const int* cache_len;
    int per_split;           // 32-key blocks per split (split sp owns blocks [sp * per_split, ...))
    const uint64_t* mask;    // [B*q] or null
    int B, q, H, S_max;
    float scale;
    int splits;              // workgroups per (b, h); > 1: partials to `part`, merged by the last split
    int cols;                // column slices (splits == 1 only): workgroups per (b, h) that each write
                             // Dh / cols columns of O
    float* part;             // [B*H][splits][16*MT rows][Dh + 4]: unnormalised O, row max, row sum
    int* counter;            // [B*H][row tiles] arrival counts of the splits (zero between launches)
    void* out;               // T (or float if out_f32) [B*q][ldo], head h at columns h*Dh..
    int out_f32, ldo;
    int* err;                // device error flags (bit 4: read past the cache)
};
// `splits` x `cols` workgroups of `waves` waves per (sequence, head, 16-row tile); max_len: the
// host's upper bound of the cache lengths; S_max: key slots per sequence
struct AttnPlan { int waves, splits, per_split, row_tiles, grid, lds_bytes, cols; };
// Blocks of up to this many rows per sequence (every decode block: M <= 64) keep the decode key
// partition, so a row's logits do not depend on the block size; longer blocks (prefill chunks) take
// one split, and with the chain mask the row kernel below.
constexpr int kAttnSplitRows = 64;
AttnPlan plan_attention(int B, int H, int q, int head_dim, int max_len, int S_max);
// partial buffer and arrival counters a context needs for its largest blocks; what one plan needs
size_t attention_partial_floats(int B_max, int H, int q_max, int head_dim, int S_max);
size_t attention_plan_partial_floats(const AttnPlan& p, int B, int H, int head_dim);
size_t attention_counter_ints(int B_max, int H, int q_max);
// ev0 / ev1 (optional): start and end of the attention kernel
hipError_t launch_attention(int dtype, int head_dim, const AttnPlan& p, const AttnArgs& a, hipStream_t s,
                            hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// Blocks of more than kAttnSplitRows rows with the chain mask (mask NULL): 64-row tiles, the key blocks staged in LDS;
// plan, splits, per_split, cols, part and counter are not used.  bf16 with heads of 64 or 128 columns,
// float with 64 (attention_rows_supported)
inline bool attention_rows_supported(int dtype, int head_dim) { return head_dim == 64 || (dtype == 1 && head_dim == 128); }
hipError_t launch_attention_rows(int dtype, int head_dim, const AttnArgs& a, hipStream_t s,
                                 hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

// ---------------------------------------------------------------- misc kernels
hipError_t launch_embed(int dtype, const void* embed, int n_rows_emb, int d, const int* tokens, int M,
                        float* x, float* xg, const float* gain, int ldxg, float* ssq, int n_ssq, int* err,
                        hipStream_t s);
hipError_t launch_to_elem_rows(int dtype, const float* src, int rows, int cols, void* dst, int ld, hipStream_t s);
hipError_t launch_kv_write(int dtype, void* kc, void* vc, int B, int n, int H, int Dh, int S_max,
                           const float* k, const float* v, const int* pos, hipStream_t s);
hipError_t launch_to_elem(int dtype, const float* src, void* dst, size_t n, hipStream_t s);
hipError_t launch_commit(int* cache_len, int B, const int* n_commit, int S_max, int* err, hipStream_t s);
hipError_t launch_commit_gather(int dtype, void* kc, void* vc, size_t layer_stride_elems, int n_layers,
                                int B, int H, int Dh, int S_max, const int* cache_len, const int* n_commit,
                                const int* rows, int q, int* err, hipStream_t s);
hipError_t launch_set_len(int* cache_len, int B, const int* vals_or_null, int value, hipStream_t s);
hipError_t launch_fill_i32(int* p, size_t n, int value, hipStream_t s);
// reads `bytes` (a multiple of 16) from src and writes nothing: the device's achievable read rate
hipError_t launch_stream_read(const void* src, size_t bytes, hipStream_t s);
// rotary table [S][half][2]: cos and sin of the angle pos * inv_freq[i], formed in double, rounded to float
hipError_t launch_rope_table(const double* inv_freq, int S, int half, float* rope, hipStream_t s);

// ---------------------------------------------------------------- large blocks (prefill)
// C[M][ldc] (float) = A[M][lda] (element type) . W[N][K]^T on the matrix cores, W = up to three
// row-major [n_per, K] matrices stacked along N (W0 rows 0..n_per-1, W1 the next n_per, ...).
// K must be a multiple of 8 (16-byte loads); rows of A past K read as zero only up to K.
// With ksplit > 1 (prefill_gemm_ksplit, at most kPrefillMaxSplit) the contraction is split into parts of
// whole stages whose partial products go to C + part * c_part; the consumer adds them in part order.
// Epilogues of the prefill GEMM: PG_STORE writes C (float); PG_QKV takes N = 3 n_per columns Q | K | V
// (heads of Dh columns), applies RoPE at cache_len[b] + row and writes Q (float) to qbuf [M][H][Dh],
// K and V in the element type into the cache (K [B][H][S_max][Dh], V key-permuted [B][H][S_max/32][Dh][32]);
// PG_SWIGLU takes N = 2 n_per columns gate | up and writes u = silu(gate) * up in the element type to
// u [M][ldu].  The fused epilogues need ksplit 1.
enum { PG_STORE = 0, PG_QKV = 1, PG_SWIGLU = 2 };
struct PrefillGemmArgs {
    int M, N, K;
    const void* A; int lda;
    const void* W0; const void* W1; const void* W2; int n_per;
    float* C; int ldc;
    int ksplit; size_t c_part;
    int ep;
    // PG_QKV
    int q, H, Dh, S_max; const int* cache_len; const float* rope; float* qbuf; void* kc; void* vc; int* err;
    // PG_SWIGLU
    void* u; int ldu;
};
constexpr int kPrefillMaxSplit = 4;
int prefill_gemm_ksplit(int M, int N, int K);
hipError_t launch_prefill_gemm(int dtype, const PrefillGemmArgs& p, hipStream_t s);
// Row-wise steps around the prefill GEMMs of blocks of more than 64 rows.
// h = elem(xg / rms) with rms from the row's per-16-column sums of squares
hipError_t launch_rms_rows(int dtype, const float* xg, int ldxg, const float* ssq, int n_ssq, int K, float eps, int M,
                           void* h, int ldh, hipStream_t s);
// x += y with y = ((y_0 + y_1) + y_2) + ..., the parts of a split contraction (parts >= 1, part p at
// y + p * part_stride); h = elem((x o g) / rms(x)), bitwise what the residual epilogue's per-16-column
// sums of squares and rms_rows give (rows of up to 8192 columns)
hipError_t launch_resid_norm_rows(int dtype, const float* y, int parts, size_t part_stride, int ldy, int M, int N,
                                  float* x, int ldx, const float* g, float eps, void* h, int ldh, hipStream_t s);

// ---------------------------------------------------------------- verify
hipError_t launch_verify_greedy(const float* logits, int B, int q, int V, const int* drafts, int drafts_ld,
                                int* tokens_out, int* n_accept, int* counter, hipStream_t s);
// row_depth (optional, a draft tree; drafts must be NULL): every row is sampled with the uniform of
// position pos0[b] + row_depth[b*q + row]
hipError_t launch_verify_nucleus(const float* logits, int B, int q, int V, const int* drafts, int drafts_ld,
                                 float temperature, float top_p, int top_k, uint64_t seed, const int* pos0,
                                 int* tokens_out, int* n_accept, int* counter, hipStream_t s,
                                 const int* row_depth = nullptr);

// draft tree of width w over draft step 1's rows (k adaptive rows): q2 = 1 + k*w block rows
constexpr int kMaxTreeWidth = 8;
hipError_t launch_tree_build(const float* logits1, int B, int q1, int V, const int* out1, int k, int w, int q2,
                             int* tok2, uint64_t* mask2, int* depth2, hipStream_t s);
hipError_t launch_tree_walk(int B, int q2, int k, int w, const int* tok2, const int* targets, const int* active,
                            int* emitted, int* n_accept, int* rows, int* pending, int* n_commit, hipStream_t s);

// ---------------------------------------------------------------- decode-loop helpers
hipError_t launch_build_draft1(const int* pending, const int* adaptive, int B, int k, int* tokens, hipStream_t s);
hipError_t launch_loop_commit(int* cache_len, int B, int q, const int* active, const int* n_accept,
                              const int* tokens2, int* pending, int* n_commit_out, hipStream_t s);
hipError_t launch_pos0(const int* cache_len, int B, int offset, int* pos0, hipStream_t s);
// per-loop record for the host, [B][kLoopRecCols] ints: m, draft step 1's token, emitted rows 0..k; advances
// the device's produced counts and active flags
constexpr int kLoopRecCols = 66;   // k <= 63 (a block holds at most 64 rows)
hipError_t launch_loop_record(int* rec, int B, int q1, int q2, int k, int max_new, const int* out1, const int* out2,
                              const int* n_accept, int* active, int* produced, hipStream_t s);

// ---------------------------------------------------------------- host runtime
// Records msg as the text sdsat_last_error(NULL) returns and passes code through.
int report_error(int code, const std::string& msg);
// Size of the static device array behind sdsat_linear_noalloc.
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;

}  // namespace sdsat
