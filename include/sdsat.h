/*
 * sdsat.h - C-ABI of the SDSAT block-decode library for MI355X (gfx950).
 *
 * SDSAT (Speculative Decoding with Semantic Adaptive Tokens, arXiv 2403.18647)
 * decodes with a loop of two forward passes of the unmodified target model over
 * a short block of k+1 rows (Section 2.1):
 *   draft step 1 (Eq. 1)  block [pending, a_1..a_k]: row 0 gives the next exact
 *                         token, rows 1..k give drafts;
 *   draft step 2 (Eq. 2)  block [t1, d_1..d_k]: row j gives the target's token
 *                         after the first j drafts;
 *   verification (Eq. 3)  the longest prefix of drafts that the step-2 outputs
 *                         confirm is accepted; a loop emits m+2 tokens, m <= k.
 * The nucleus variant (Section 2.1.2) replaces arg-max by sampling.
 *
 * Conventions (every function):
 *   - returns an int status: SDSAT_OK (0) or a negative SDSAT_E* code; nothing
 *     is thrown across the ABI.  On error the outputs are unspecified and the
 *     context stays usable unless the code is SDSAT_EDEVICE.
 *     sdsat_last_error() describes the most recent failure.
 *   - "d_" pointers are device pointers, "h_" pointers host pointers.  All
 *     buffers are owned by the caller and must stay alive for the duration of
 *     the call (weights and workspace: for the context's lifetime).
 *   - calls marked "stream-ordered" only enqueue work on the context's HIP
 *     stream and return without waiting; their device outputs are valid once
 *     the stream reaches them.  A device-side data error (a token id out of
 *     range) sets a flag that the next synchronous call reports as SDSAT_EDATA.
 *   - one context per stream and per host thread; calls on one context are not
 *     thread-safe.
 *   - layouts are row-major; int32 token ids; float32 logits.
 */
#ifndef SDSAT_H
#define SDSAT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SDSAT_OK 0
#define SDSAT_EINVAL (-1)       /* bad argument, shape or pointer */
#define SDSAT_ENOMEM (-2)       /* host allocation failed or workspace too small */
#define SDSAT_EDEVICE (-3)      /* HIP runtime error */
#define SDSAT_ECAPACITY (-4)    /* cache_len+q > max_ctx, q > max_block, batch > max_batch */
#define SDSAT_EUNSUPPORTED (-5) /* configuration the kernels do not implement */
#define SDSAT_EDATA (-6)        /* device-side data error (token id out of range) */

#define SDSAT_DTYPE_FP32 0
#define SDSAT_DTYPE_BF16 1

#define SDSAT_MODE_GREEDY 0
#define SDSAT_MODE_NUCLEUS 1

/* Opaque, library-owned context. */
typedef struct sdsat_ctx sdsat_ctx;

/* Target-model shape.  The paper keeps the target model unmodified (Section 2,
 * Section 2.2); its targets are CodeLlama-7B/13B (Section 3), i.e. Llama
 * decoders: RMSNorm, rotate-half RoPE, multi-head attention (n_kv_heads ==
 * n_heads), SwiGLU, no biases, untied LM head. */
typedef struct sdsat_config {
    int32_t n_layers, d_model, n_heads, head_dim, d_ffn;
    int32_t vocab;       /* V: LM-head width; generated ids are < V */
    int32_t n_adaptive;  /* A: embedding rows V..V+A-1 are the adaptive tokens */
    float rms_eps, rope_base;
    int32_t dtype;       /* SDSAT_DTYPE_FP32 or SDSAT_DTYPE_BF16: weights, KV cache, GEMM inputs */
    int32_t max_batch;   /* B_max */
    int32_t max_ctx;     /* KV slots per sequence (committed + one block) */
    int32_t max_block;   /* largest q (rows per sequence per block), <= 4096; also the
                            prefill block of sdsat_generate.  Blocks of more than 64 rows
                            in total (batch * q) run their linear layers as matrix-core
                            GEMMs on the caller's weights (d_ffn must then be a multiple
                            of 8) and take no ancestor mask; decode blocks need
                            batch * (k + 1) <= 64 */
} sdsat_config;

/* Statistics of sdsat_generate (Section 3.4 reports tokens/s and accept rate). */
typedef struct sdsat_stats {
    int64_t loops;             /* draft-draft-verify loops run */
    int64_t blocks;            /* block forwards run, prefill excluded */
    int64_t prefill_blocks;
    int64_t tokens;            /* new tokens emitted (before truncation to max_new), all sequences */
    int64_t accepted;          /* sum over loops and sequences of m (accepted drafts) */
    int64_t accept_hist[65];   /* histogram of m over (loop, active sequence) */
    double prefill_ms, decode_ms;
} sdsat_stats;

/* Required workspace size for a configuration.  Host-only; no device work. */
int sdsat_query_sizes(const sdsat_config* cfg, size_t* workspace_bytes);

/* Create a context.
 * weights: n_weights device pointers in the fixed order
 *   embed [V+A, d],
 *   per layer: attn_norm [d], wq [d, d], wk [d, d], wv [d, d], wo [d, d],
 *              ffn_norm [d], w_gate [F, d], w_up [F, d], w_down [d, F],
 *   final_norm [d], lm_head [V, d];
 *   matrices are [out, in] row-major, element type per cfg->dtype (norm gains
 *   are always float32).  n_weights must be 1 + 9*n_layers + 2.
 * workspace: device buffer of at least sdsat_query_sizes() bytes, 256-byte
 *   aligned, caller-owned.  The context packs the weight matrices into it
 *   (so the caller's matrices are only read during init), and keeps there the
 *   KV cache, activations and scratch.
 * hip_stream: the hipStream_t all work is enqueued on (NULL: default stream).
 * Synchronous.  Cache lengths start at 0. */
int sdsat_init(const sdsat_config* cfg, const void* const* weights, int32_t n_weights,
               void* workspace, size_t workspace_bytes, void* hip_stream, sdsat_ctx** out);

/* Set cache_len[b] = 0 for b < batch.  Stream-ordered. */
int sdsat_reset(sdsat_ctx* ctx, int32_t batch);

/* Set cache_len[b] = h_len[b] for b < batch (slots must hold valid K/V, e.g.
 * written by sdsat_kv_write).  Stream-ordered. */
int sdsat_set_cache_len(sdsat_ctx* ctx, int32_t batch, const int32_t* h_len);

/* Device pointer to cache_len[max_batch] (int32), read-only for the caller. */
const int32_t* sdsat_cache_len_ptr(const sdsat_ctx* ctx);

/* One forward pass of the target model over a block (Eq. 1 and Eq. 2 each run
 * one): row r of sequence b holds d_tokens[b*q + r] at absolute position
 * cache_len[b] + r and attends to cache slots 0..cache_len[b]-1 plus the block
 * rows its mask allows.  d_ancestor_mask: [batch*q] uint64, bit j of row r set
 * if row r may attend to block row j (tree attention, Section 2.1.2); NULL
 * means block-causal (rows 0..r).  The block's K and V are written
 * tentatively to slots cache_len[b]..cache_len[b]+q-1; cache_len is NOT
 * advanced (see sdsat_commit_kv).  d_logits: [batch*q, V] float32, or NULL to
 * skip the LM head (prefill).  Stream-ordered. */
int sdsat_forward_block(sdsat_ctx* ctx, int32_t batch, int32_t q, const int32_t* d_tokens,
                        const uint64_t* d_ancestor_mask, float* d_logits);

/* Greedy verification, Eq. 3.  d_tokens_out[b*q + j] = arg-max of logits row
 * (b, j) (lowest id among ties).  With d_drafts ([batch, q-1]: the tokens the
 * block fed at rows 1..q-1), d_n_accept[b] = the number m of leading j >= 1
 * with drafts[b][j-1] == tokens_out[b][j-1]; the loop emits tokens_out[b][0..m].
 * d_drafts NULL (draft step 1): only the arg-maxes, n_accept = 0 (may be NULL).
 * Stream-ordered. */
int sdsat_verify_greedy(sdsat_ctx* ctx, int32_t batch, int32_t q, const float* d_logits,
                        const int32_t* d_drafts, int32_t* d_tokens_out, int32_t* d_n_accept);

/* Nucleus verification (Section 2.1.2, chain form).  Each sampled row uses
 * z = logits / temperature (temperature <= 0: arg-max), keeps the top_k largest
 * (top_k <= 0: all; ties keep lower ids), and samples from the smallest
 * value-threshold set whose softmax mass reaches top_p (every id tied at the
 * threshold kept), by ascending-id inverse CDF with u = U(seed, b, pos): the
 * (c+1)-th SplitMix64 output from state `seed`, c = b*2^32 + pos, top 53 bits.
 * Arithmetic in float64.  pos of row j is d_pos0[b] + j.
 * With d_drafts: every row is sampled and n_accept counts leading matches as in
 * sdsat_verify_greedy.  Without (draft step 1): row 0 is sampled, rows 1..q-1
 * are arg-maxed (the chain of most probable drafts), n_accept = 0.
 * Requires V <= 131072 (SDSAT_EUNSUPPORTED otherwise).  Stream-ordered. */
int sdsat_verify_nucleus(sdsat_ctx* ctx, int32_t batch, int32_t q, const float* d_logits,
                         const int32_t* d_drafts, float temperature, float top_p, int32_t top_k,
                         uint64_t seed, const int32_t* d_pos0, int32_t* d_tokens_out,
                         int32_t* d_n_accept);

/* Commit block rows to the KV cache (the step after Eq. 1 keeps row 0, the
 * step after Eq. 3 keeps rows 0..m).  d_n_commit[b] rows of sequence b become
 * committed: cache_len[b] += n.  d_rows NULL: the committed rows are block rows
 * 0..n-1, already in place (chain case: a length bump; rejected rows are
 * overwritten by the next block).  d_rows [batch, q]: rows d_rows[b][0..n-1],
 * strictly ascending, are gathered to slots cache_len[b]..+n-1 first (tree
 * case).  q is the row stride of d_rows.  Stream-ordered. */
int sdsat_commit_kv(sdsat_ctx* ctx, int32_t batch, int32_t q, const int32_t* d_n_commit,
                    const int32_t* d_rows);

/* Full SDSAT generation (Section 2.1): prefill of h_prompts[b][0..P-2]
 * (blocks of max_block rows, LM head skipped), then loops of draft step 1,
 * draft step 2 and verification until every sequence has max_new tokens
 * (overshoot truncated; finished sequences ride along with commit 0).
 * k adaptive ids h_adaptive_ids[k] (k+1 <= max_block); k = 0 gives plain
 * decoding at two blocks per loop.  mode SDSAT_MODE_GREEDY or _NUCLEUS
 * (temperature, top_p, top_k, seed as in sdsat_verify_nucleus).
 * h_out: [batch, max_new] int32.  h_stats may be NULL.  Synchronous.
 * Capacity: max_ctx (rounded up to 32) must be at least P + max_new + k + 1,
 * plus k more slots when batch > 1 (a finished sequence stops at up to
 * P + max_new + k committed tokens and still receives blocks); otherwise
 * SDSAT_ECAPACITY. */
int sdsat_generate(sdsat_ctx* ctx, int32_t batch, const int32_t* h_prompts, int32_t P,
                   int32_t max_new, int32_t k, const int32_t* h_adaptive_ids, int32_t mode,
                   float temperature, float top_p, int32_t top_k, uint64_t seed,
                   int32_t* h_out, sdsat_stats* h_stats);

/* sdsat_generate with draft step 2 run over a draft tree (Section 2.1.2):
 * depth j = 1..k holds the `width` most probable tokens of draft step 1's
 * adaptive row j (ties to the lower id); the first of each depth forms the
 * main chain, the others are leaves under the chain node one level up.  The
 * tree's 1 + k*width rows run as one block with ancestor masks (each row at
 * position cache_len + depth, seeing its ancestors); the target's token at
 * every node (greedy arg-max, or the nucleus sample keyed by the position it
 * is for) is computed, the longest branch whose tokens the targets confirm
 * is accepted (m of its nodes), its rows are gathered into the cache and
 * m + 1 tokens are emitted after t1.  width = 1 is sdsat_generate.  Needs
 * width in 1..8, 1 + k*width <= max_block and batch * (1 + k*width) <= 64.
 * Other arguments and the output as sdsat_generate.  Synchronous. */
int sdsat_generate_tree(sdsat_ctx* ctx, int32_t batch, const int32_t* h_prompts, int32_t P,
                        int32_t max_new, int32_t k, int32_t width, const int32_t* h_adaptive_ids,
                        int32_t mode, float temperature, float top_p, int32_t top_k, uint64_t seed,
                        int32_t* h_out, sdsat_stats* h_stats);

/* sdsat_generate with the drafts of every draft step 2 taken from a known
 * continuation instead of draft step 1's adaptive rows: d_j of sequence b
 * = h_ref[b][n + j] (n = tokens sequence b has emitted so far, j = 1..k; ids
 * past ref_len read as 0).  With h_ref = the autoregressive output of the
 * same prompts (ref_len >= max_new + k + 1), verification (Eq. 3) accepts
 * every draft, so each loop emits k + 2 tokens: the loop at full acceptance,
 * for measurement on weights whose adaptive rows do not predict the target.
 * h_ref: [batch, ref_len] int32 (host).  Other arguments and the output as
 * sdsat_generate.  Synchronous. */
int sdsat_generate_forced(sdsat_ctx* ctx, int32_t batch, const int32_t* h_prompts, int32_t P,
                          int32_t max_new, int32_t k, const int32_t* h_adaptive_ids, int32_t mode,
                          float temperature, float top_p, int32_t top_k, uint64_t seed,
                          const int32_t* h_ref, int32_t ref_len, int32_t* h_out, sdsat_stats* h_stats);

/* ---- op-level entry points (kernel tests and micro-benchmarks) ---- */

/* Write K and V rows (float32, [batch, n, H, Dh]) of `layer` into cache slots
 * d_pos[b*n + i] of sequence b, converted to the cache dtype.  Stream-ordered. */
int sdsat_kv_write(sdsat_ctx* ctx, int32_t layer, int32_t batch, int32_t n, const float* d_k,
                   const float* d_v, const int32_t* d_pos);

/* Block attention of `layer` alone: queries d_q ([batch*q, H*Dh] float32, RoPE
 * already applied) against cache slots 0..cache_len[b]+q-1 of sequence b (the
 * block's own rows must already be in the cache), mask as in
 * sdsat_forward_block.  d_out: [batch*q, H*Dh] float32.  Stream-ordered. */
int sdsat_attention(sdsat_ctx* ctx, int32_t layer, int32_t batch, int32_t q, const float* d_q,
                    const uint64_t* d_ancestor_mask, float* d_out);

/* Bytes of the packed form of an [N, K] weight matrix. */
size_t sdsat_linear_packed_bytes(int32_t dtype, int32_t N, int32_t K);

/* Pack a row-major [N, K] weight matrix (dtype elements) for sdsat_linear.
 * Stream-ordered on hip_stream. */
int sdsat_linear_pack(int32_t dtype, int32_t N, int32_t K, const void* d_w, void* d_packed,
                      void* hip_stream);

/* Skinny GEMM y[M, N] = x[M, K] . W[N, K]^T with x float32 (rounded to dtype
 * as the matrix-core input), float32 accumulation and output; M <= 64.
 * d_scratch: sdsat_linear_scratch_bytes() bytes of device memory (caller-owned;
 * every call rewrites the part it reads, so it needs no initial contents).
 * Stream-ordered on hip_stream. */
size_t sdsat_linear_scratch_bytes(int32_t M, int32_t N, int32_t K);
int sdsat_linear(int32_t dtype, int32_t M, int32_t N, int32_t K, const float* d_x,
                 const void* d_packed, float* d_y, void* d_scratch, void* hip_stream);

/* sdsat_linear for callers that cannot allocate device memory (code under
 * stream capture, serving loops that forbid allocation): the same kernels and
 * results, with the scratch taken from a 4 MiB array the library holds in
 * static device memory (one copy per GPU, kept until the process ends).  It
 * allocates nothing; the caller still owns d_x, d_packed and d_y.
 * M * (K rounded up to 32) * (4 bytes fp32, 2 bf16) must be <= 4 MiB, else
 * SDSAT_EINVAL.  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (other streams, other threads) race and must be
 * serialised by the caller.  The device is the current one.  Stream-ordered on
 * hip_stream; the first call on a device also looks up its array's address. */
int sdsat_linear_noalloc(int32_t dtype, int32_t M, int32_t N, int32_t K, const float* d_x,
                         const void* d_packed, float* d_y, void* hip_stream);

/* Per-kernel timing with HIP events on the context's stream.  kind: 0 off,
 * 1 gate/up GEMM, 2 QKV GEMM, 3 attention, 4 down GEMM, 5 O GEMM, 6 LM head,
 * 7 whole block forward with logits (draft / verify blocks), 8 whole block
 * forward without logits (prefill).  period >= 1: one launch of that kind in
 * every `period` is timed.  Kinds 1-6 take their events from the kernel's own
 * dispatch (start and end of the kernel, or of the first and last kernel of a
 * pair: attention and its split combine, a split GEMM and its fold), the
 * interval a kernel trace reports; kinds 7 and 8 record a
 * pair of events around the block (each pair costs a few microseconds of
 * queue time, so a period > 1 keeps timed runs undisturbed).
 * sdsat_kernel_time synchronizes the stream and returns the summed
 * milliseconds and the number of timed launches since the last call. */
int sdsat_profile_kernel(sdsat_ctx* ctx, int32_t kind, int32_t period);
int sdsat_kernel_time(sdsat_ctx* ctx, double* total_ms, int64_t* launches);

/* As sdsat_kernel_time, but returns each timed launch's milliseconds: the
 * first min(cap, *launches) of them, in launch order, into the caller's host
 * array h_ms (cap >= 0; h_ms may be NULL when cap is 0).  *launches = the
 * number of timed launches since the last call; the samples are consumed. */
int sdsat_kernel_samples(sdsat_ctx* ctx, float* h_ms, int64_t cap, int64_t* launches);

/* Measurement helper, outside the decoding method: streams `bytes` (a
 * multiple of 16; EINVAL otherwise) from the device buffer d_src through the
 * read pattern that measured fastest on MI355X (16 KiB contiguous per
 * workgroup, 16-byte nontemporal loads) and writes nothing, on hip_stream
 * (NULL = the default stream).  Time it with events on that stream to get
 * the achievable HBM read rate that the block forward's bandwidth can be set
 * against.  The buffer stays the caller's; no context is needed. */
int sdsat_stream_read(const void* d_src, size_t bytes, void* hip_stream);

/* Release the context (not the caller's buffers).  NULL is accepted. */
int sdsat_destroy(sdsat_ctx* ctx);

/* Text of the most recent error on ctx (or of the last failed sdsat_init when
 * ctx is NULL).  Never NULL. */
const char* sdsat_last_error(const sdsat_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* SDSAT_H */
