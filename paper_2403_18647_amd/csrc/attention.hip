// Block-causal decode attention over the KV cache (the target model's attention,
// run on the q rows of one SDSAT block; tree masks for Section 2.1.2).
//
// For sequence b, head h and block row r (query at position L_b + r):
//   O_r = softmax(Q_r K^T / sqrt(Dh)) V over keys 0..L_b-1 (committed) plus
//   the block rows r may see (0..r, or the rows set in its ancestor mask).
// The block's own K/V rows were written into slots L_b.. by the QKV epilogue.
//
// Workgroups per (b, h, 16-row tile of the block): one per key split (the
// splits are fixed 32-key block ranges, see plan_attention).  Each split
// writes its partial result (unnormalised O, row maximum, row sum) with
// device-coherent stores and counts itself done on a per-tile counter; the
// split that arrives last merges all partials of the tile in split order and
// writes O, so no second kernel runs and every key is read once.  Where only
// one split is planned, a one-tile block may instead spread each head over
// column slices: every slice's workgroup forms all of the head's scores but
// only its share of the columns of O.  Waves take the workgroup's 32-key
// blocks round-robin.
// Q arrives in float and the probabilities are formed in float; on bf16
// models each enters the matrix cores as a pair of bf16 fragments (value and
// rounding remainder, about 16 significant bits), so neither is rounded to
// bf16 on its way: the scores and the weighted sum of V keep float accuracy
// (K and V are bf16 as stored).
// Query rows are handled 16 at a time (one matrix-core tile); the row tiles
// of a longer block (a prefill chunk) are separate workgroups that read the
// same keys (the later readers from L2), each only up to its last row.  Per
// block a wave computes the 32 x 16 score tile
// S^T = K Q^T on the matrix cores (A = K rows straight from the cache, B = Q^T
// from registers), runs an online softmax per query row (query rows live in
// lanes, keys in registers and lane groups), and accumulates O^T = V^T P^T
// with A = V^T read from the cache's key-permuted 32-key blocks (vperm) and
// B = P^T taken from the score registers as they are.  The next block's K and
// V are in flight while the current one is computed; the first two are
// requested from the host's upper bound of the cache length before the true
// length has arrived.  The waves' partial results are merged in LDS with a
// log-sum-exp combine in wave order (deterministic).
#include <hip/hip_ext.h>

#include "device.h"
#include "kernels.h"

namespace sdsat {

static constexpr int kMaxWaves = 8;
static constexpr int kMaxSplits = 16;
static constexpr int kMaxCols = 8;
// workgroups a full cache is cut into per row tile (key splits x sequences x heads), at most
static constexpr int kAttnWorkgroups = 256;

// Keys are partitioned by absolute 32-key block index only: split sp owns
// blocks [sp * P, (sp + 1) * P) with P fixed by the cache capacity (at full
// capacity, as many splits as fit one round of 256 workgroups per row tile),
// and within a split block i goes to wave i mod waves.  Each 16-row tile of
// the block has its own workgroups and reads only the key blocks its last row
// can see.  A query row of a block of up to kAttnSplitRows rows (every decode
// block) therefore sees the same keys in the same order of accumulation
// whatever the block size q and the cache length: blocks it cannot see (later
// rows of its own block) add exact zeros, and so do the partials of splits
// that hold none of its keys.  So a token's logits do not depend on how many
// draft rows share its block, and greedy SDSAT reproduces autoregressive
// decoding bit for bit.  Longer blocks (prefill chunks) take one split (with
// the chain mask, the row kernel below), whose order of accumulation differs.
// Waves per workgroup:
// one per block of the split, at most 8.  Column slices change which
// workgroup writes a column of O, not how it is computed: each slice's values
// are those of the single workgroup, bit for bit, so the slice count may
// follow the block size.
AttnPlan plan_attention(int B, int H, int q, int head_dim, int max_len, int S_max) {
    AttnPlan p;
    const int cap = std::max(1, S_max / 32);
    const int nblk = std::max(1, std::min(cap, (max_len + q + 31) / 32));
    const int pairs = B * H;
    // a full cache gives about kAttnWorkgroups workgroups per row tile; where that allows only two
    // splits, one split is planned (measured at batch 4 x 32 heads with a combine kernel: 26.4 ->
    // 23.6 us per layer)
    // A prefill chunk (more than kAttnSplitRows rows) has workgroups enough across its row tiles and
    // takes one split: the key partition only has to be the same for every decode block size.
    p.row_tiles = (q + 15) / 16;
    int target = std::max(1, std::min(kMaxSplits, kAttnWorkgroups / pairs));
    if (target <= 2 || q > kAttnSplitRows) target = 1;
    p.per_split = (cap + target - 1) / target;
    p.splits = (nblk + p.per_split - 1) / p.per_split;
    p.waves = std::max(1, std::min(p.per_split, kMaxWaves));
    // column slices (one split, one row tile): as many as keep one round of 256 workgroups
    p.cols = 1;
    if (p.splits == 1 && p.row_tiles == 1)
        while (p.cols * 2 <= std::min(kMaxCols, head_dim / 16) && pairs * p.cols * 2 <= 256) p.cols *= 2;
    p.grid = pairs * p.row_tiles * p.splits * p.cols;
    p.lds_bytes = p.waves * (head_dim / 16) * 64 * 16;
    return p;
}

size_t attention_plan_partial_floats(const AttnPlan& p, int B, int H, int head_dim) {
    return p.splits > 1 ? (size_t)B * H * p.splits * p.row_tiles * 16 * (head_dim + 4) : 0;
}

// The most any block of up to q_max rows and up to B_max sequences needs: a one-row-tile (decode) block
// may take more key splits than a longer one, so both sizes are planned, at full cache length.
size_t attention_partial_floats(int B_max, int H, int q_max, int head_dim, int S_max) {
    size_t most = 0;
    for (int b = 1; b <= B_max; ++b)
        for (int q : {std::min(q_max, 16), std::min(q_max, kAttnSplitRows), q_max})
            most = std::max(most, attention_plan_partial_floats(plan_attention(b, H, q, head_dim, S_max, S_max), b, H,
                                                                head_dim));
    return most;
}

size_t attention_counter_ints(int B_max, int H, int q_max) { return (size_t)B_max * H * ((q_max + 15) / 16); }

// K and V of one 32-key block through buffer resources over this (sequence,
// head)'s cache rows: one 32-bit lane offset per 16-key half of K and one for
// V, fragment offsets as wave-uniform constants (keeps the addresses out of
// the register budget).
template <typename T, int NDS, int NDT>
__device__ __forceinline__ void load_kv(Frag<T> (&kf)[2][NDS], Frag<T> (&vf)[NDT], __amdgpu_buffer_rsrc_t kr,
                                        __amdgpu_buffer_rsrc_t vr, int blk, int c, int g, uint32_t vsoff) {
    constexpr int DH = NDS * 32;
    constexpr uint32_t E = sizeof(T);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        const uint32_t ko = ((uint32_t)(blk * 32 + 16 * kt + c) * DH + 8 * g) * E;
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds) kf[kt][ds] = buf_frag<T>(kr, ko, ds * 32 * E);
    }
    const uint32_t vo = ((uint32_t)blk * DH * 32 + c * 32 + 8 * g) * E;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) vf[dt] = buf_frag<T>(vr, vo, vsoff + dt * 16 * 32 * E);
}

// x as the matrix-core operand pair hi + lo (lo = the bf16 rounding remainder;
// float models use x itself and no second fragment).
template <typename T>
__device__ __forceinline__ void split_frag(const float (&x)[8], Frag<T>& hi, Frag<T>& lo) {
    hi = Frag<T>::from_f32(x);
    if constexpr (sizeof(T) == 2) {
        float r[8];
        const uint32_t w[4] = {hi.v.x, hi.v.y, hi.v.z, hi.v.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) r[i] = x[i] - bf16_to_f32((uint16_t)(w[i / 2] >> (16 * (i % 2))));
        lo = Frag<T>::from_f32(r);
    }
}

// One 32-key block for the 16 query rows of this lane group (lane column c is
// block row m = m0 + c).
// Q fragments of the current row tile, in LDS: [hi / lo][ds][lane].  They are
// read where they are used, which keeps them out of the register budget: the
// index passes through an empty asm statement, so the compiler cannot hoist
// the reads out of the block loop (a volatile read would do the same but also
// makes it wait for every outstanding global load, the next blocks' K and V).
template <typename T>
__device__ __forceinline__ Frag<T> lds_frag(const Frag<T>* qs, int idx) {
    asm volatile("" : "+v"(idx));
    return qs[idx];
}

template <typename T, int NDS, int NDT>
__device__ __forceinline__ void attend_block(const Frag<T> (&kf)[2][NDS], const Frag<T> (&vf)[NDT],
                                             const Frag<T>* qs, int lane, uint64_t mrow,
                                             int blk, int m, int L, int Tb, int q, bool tree, float scale, int g,
                                             float& rmax, float& rsum, f32x4_t (&o)[NDT]) {
    constexpr bool two = sizeof(T) == 2;
    const int kb0 = blk * 32;
    f32x4_t s0 = f32x4_t{0.f, 0.f, 0.f, 0.f}, s1 = s0;
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) {
        const Frag<T> qh = lds_frag<T>(qs, ds * 64 + lane);
        mma(s0, kf[0][ds], qh);
        mma(s1, kf[1][ds], qh);
        if constexpr (two) {
            const Frag<T> ql = lds_frag<T>(qs, (NDS + ds) * 64 + lane);
            mma(s0, kf[0][ds], ql);
            mma(s1, kf[1][ds], ql);
        }
    }
    // s0[r], s1[r] = S^T[key = kb0 + 16kt + 4g + r][row m]
    float sv[8];
    bool vis[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int key = kb0 + (i < 4 ? 4 * g + i : 16 + 4 * g + (i - 4));
        bool v = key < Tb && m < q;
        if (tree) v = v && (key < L || ((mrow >> (key - L)) & 1ull));
        else v = v && key <= L + m;
        vis[i] = v;
        sv[i] = (i < 4 ? s0[i] : s1[i - 4]) * scale;
    }
    float bm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) if (vis[i]) bm = fmaxf(bm, sv[i]);
    bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
    bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
    const float nmax = fmaxf(rmax, bm);
    const float alpha = rmax == -INFINITY ? 0.f : expf(rmax - nmax);
    float p[8];
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        p[i] = vis[i] ? expf(sv[i] - nmax) : 0.f;
        ps += p[i];
    }
    rsum = rsum * alpha + ps;
    rmax = nmax;
    Frag<T> ph, pl;
    split_frag<T>(p, ph, pl);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
        o[dt] *= alpha;
        mma(o[dt], vf[dt], ph);
        if constexpr (two) mma(o[dt], vf[dt], pl);
    }
}

// Merge the split partials of one (sequence, head, 16-row tile): each thread
// takes 4 head dimensions of a row, log-sum-exp over the splits in split
// order.  The partials are read with device-coherent (agent-scope) loads.
// (Rows of a sequence whose cache overflowed were flagged; their output is
// then unspecified.)
template <typename T, int DH>
__device__ __forceinline__ void combine_tile(const AttnArgs& a, int bh, int rt, int n_rt) {
    constexpr int D4 = DH / 4;
    const int b = bh / a.H, h = bh % a.H;
    const int rows = n_rt * 16;
    const size_t sstride = (size_t)rows * (DH + 4);
    for (int e = threadIdx.x; e < 16 * D4; e += blockDim.x) {
        const int m = 16 * rt + e / D4, d = 4 * (e % D4);
        if (m >= a.q) continue;
        const float* base = a.part + ((size_t)bh * a.splits * rows + m) * (DH + 4);
        float mx[kMaxSplits], sm[kMaxSplits];
        f32x4_t ov[kMaxSplits];
#pragma unroll
        for (int sp = 0; sp < kMaxSplits; ++sp) {
            if (sp < a.splits) {
                const float* pr = base + sp * sstride;
                mx[sp] = __hip_atomic_load(pr + DH, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                sm[sp] = __hip_atomic_load(pr + DH + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    ov[sp][r] = __hip_atomic_load(pr + d + r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        float gmax = -INFINITY;
#pragma unroll
        for (int sp = 0; sp < kMaxSplits; ++sp) if (sp < a.splits) gmax = fmaxf(gmax, mx[sp]);
        float den = 0.f;
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int sp = 0; sp < kMaxSplits; ++sp) {
            if (sp < a.splits) {
                const float w = mx[sp] == -INFINITY ? 0.f : expf(mx[sp] - gmax);
                den += w * sm[sp];
                acc += w * ov[sp];
            }
        }
        const float inv = 1.0f / den;
        const size_t row = ((size_t)b * a.q + m) * a.ldo + (size_t)h * DH + d;
        if (a.out_f32) {
            float* po = reinterpret_cast<float*>(a.out) + row;
#pragma unroll
            for (int r = 0; r < 4; ++r) po[r] = acc[r] * inv;
        } else {
            T* po = reinterpret_cast<T*>(a.out) + row;
#pragma unroll
            for (int r = 0; r < 4; ++r) po[r] = to_elem<T>(acc[r] * inv);
        }
    }
}

// One workgroup per (sequence, head, 16-row tile, key split, column slice).
template <typename T, int DH, int CS>
__global__ void __launch_bounds__(512) attn_kernel(AttnArgs a) {
    constexpr int NDS = DH / 32;        // 32-wide steps over the head dimension
    constexpr int NDT = DH / 16 / CS;   // 16-row output tiles of this column slice
    constexpr int RGN = DH / 16;        // f32x4 rows (of 64 lanes) in a wave's LDS region
    // Per wave DH * 64 bytes of LDS: its Q fragments of the row tile
    // ([hi / lo][ds][lane], read back in every block), then its partial O
    // ([dt][lane]) for the merge.
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ float s_max[kMaxWaves][16], s_sum[kMaxWaves][16];

    const int nw = blockDim.x >> 6;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63, c = lane & 15, g = lane >> 4;
    Frag<T>* s_q = reinterpret_cast<Frag<T>*>(smem_raw + (size_t)wave * DH * 64);
    const f32x4_t* opart = reinterpret_cast<const f32x4_t*>(smem_raw);   // [waves][RGN][64]
    const int q = a.q;
    const int n_rt = (q + 15) / 16;
    // the column slice is the slowest index: the slices of one head sit on the same XCD (workgroups
    // go to XCDs round-robin, and B * H * n_rt * splits is a multiple of 8 at the model shapes), so
    // all but the first read its keys from that XCD's L2
    const int n_in = a.B * a.H * n_rt * a.splits;
    const int cx = CS == 1 ? 0 : (int)blockIdx.x / n_in;
    const int bid = (int)blockIdx.x - cx * n_in;
    const int sp = bid % a.splits, rt = (bid / a.splits) % n_rt;
    const int bh = bid / (a.splits * n_rt);
    const uint32_t vsoff = (uint32_t)(cx * NDT * 16 * 32 * sizeof(T));   // the slice's V columns
    const int b = bh / a.H, h = bh % a.H;
    const uint32_t slice_bytes = (uint32_t)a.S_max * DH * sizeof(T);
    const __amdgpu_buffer_rsrc_t kr =
        buf_rsrc(reinterpret_cast<const T*>(a.kc) + ((size_t)b * a.H + h) * a.S_max * DH, slice_bytes);
    const __amdgpu_buffer_rsrc_t vr =
        buf_rsrc(reinterpret_cast<const T*>(a.vc) + ((size_t)b * a.H + h) * a.S_max * DH, slice_bytes);
    const float* qb = a.qbuf;
    const bool tree = a.mask != nullptr;

    // Split sp owns blocks [wlo, wlo + per_split) (the last split runs on to
    // the true end, so a stale host bound costs time, never keys).  The
    // wave's blocks are first + i * nw; the first two are requested before the
    // true length is known (indices clamped into the cache; a block past the
    // length is loaded, not used), the second only if the wave can own it.
    const int wlo = sp * a.per_split;
    const int first = wlo + wave;
    const int last_blk = a.S_max / 32 - 1;
    // The cache length is the first request, as a vector load (a scalar one
    // would be scheduled after the K/V requests, and the first block waits
    // for it).
    int bv = b;
    asm volatile("" : "+v"(bv));
    const int Lv = a.cache_len[bv];
    {
        // Issue order: the ancestor mask, the wave's Q fragments, its first two
        // K/V blocks; Q is split and parked in the wave's LDS while the keys
        // are in flight (no barrier: each wave reads only its own copy).
        // Query rows past q read row q-1 (their scores are masked out).  The
        // loads ahead of the block loop are unconditional or wave-uniform, so
        // the compiler's wait counts stay exact.
        const int m = 16 * rt + c;
        const int mr = min(m, q - 1);
        const uint64_t mrow = tree ? a.mask[(size_t)b * q + mr] : 0ull;
        const f32x4_t* qsrc = reinterpret_cast<const f32x4_t*>(qb + (((size_t)b * q + mr) * a.H + h) * DH + 8 * g);
        f32x4_t qv[NDS][2];
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds) {
            qv[ds][0] = qsrc[ds * 8];
            qv[ds][1] = qsrc[ds * 8 + 1];
        }
        Frag<T> kA[2][NDS], kB[2][NDS], vA[NDT], vB[NDT];
        load_kv<T, NDS, NDT>(kA, vA, kr, vr, min(first, last_blk), c, g, vsoff);
        // a wave of a split other than the last owns at most ceil(per_split / nw)
        // blocks: when that is one (decode at short contexts), its second block
        // is never used and is not requested (measured: 13.7 -> 13.0 us per
        // layer, 7B decode at context ~600)
        const bool second = sp == a.splits - 1 || a.per_split > nw;
        if (second) load_kv<T, NDS, NDT>(kB, vB, kr, vr, min(first + nw, last_blk), c, g, vsoff);
        __builtin_amdgcn_sched_barrier(0);   // keep the K/V requests ahead of the wait for Q
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds) {   // Q columns 32ds.. of the tile's rows as hi / lo
            const float x8[8] = {qv[ds][0].x, qv[ds][0].y, qv[ds][0].z, qv[ds][0].w,
                                 qv[ds][1].x, qv[ds][1].y, qv[ds][1].z, qv[ds][1].w};
            Frag<T> fh, fl;
            split_frag<T>(x8, fh, fl);
            s_q[ds * 64 + lane] = fh;
            if constexpr (sizeof(T) == 2) s_q[(NDS + ds) * 64 + lane] = fl;
        }
        const int L = __builtin_amdgcn_readfirstlane(Lv);
        // the host checks capacity; never read past this sequence's cache (a workgroup of a split
        // tile still takes part in the arrival count, with no keys, so the count stays whole)
        const bool over = L + q > a.S_max;
        if (over && threadIdx.x == 0) atomicOr(a.err, 4);
        // key blocks the tile's last row can see (keys up to L + that row)
        const int nblk = over ? 0 : (L + min(16 * rt + 15, q - 1) + 32) / 32;
        const int whi = sp == a.splits - 1 ? nblk : min(nblk, wlo + a.per_split);
        const int Tb = L + q;

        float rmax = -INFINITY, rsum = 0.f;
        f32x4_t o[NDT];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

        // this wave's blocks: first + i * nw for i < cnt; buffers A and B alternate
        const int cnt = first < whi ? (whi - first + nw - 1) / nw : 0;
        // the loop below expects blocks 0 and 1 loaded; without the second request cnt <= 1, so this
        // only guards that invariant
        if (!second && cnt >= 2) load_kv<T, NDS, NDT>(kB, vB, kr, vr, first + nw, c, g, vsoff);
        int i = 0;
        // steady state (unconditional loads): blocks i and i + 1 are loaded
        for (; i + 4 <= cnt; i += 2) {
            attend_block<T, NDS, NDT>(kA, vA, s_q, lane, mrow, first + i * nw, m, L, Tb, q, tree, a.scale, g, rmax, rsum, o);
            load_kv<T, NDS, NDT>(kA, vA, kr, vr, first + (i + 2) * nw, c, g, vsoff);
            attend_block<T, NDS, NDT>(kB, vB, s_q, lane, mrow, first + (i + 1) * nw, m, L, Tb, q, tree, a.scale, g, rmax,
                                      rsum, o);
            load_kv<T, NDS, NDT>(kB, vB, kr, vr, first + (i + 3) * nw, c, g, vsoff);
        }
        // 0 .. 3 blocks left, blocks i and i + 1 loaded.  Three left is its own
        // straight-line path, so its one load does not make the compiler wait
        // for it before block i + 1.
        const int rem = cnt - i;
        if (rem == 3) {
            attend_block<T, NDS, NDT>(kA, vA, s_q, lane, mrow, first + i * nw, m, L, Tb, q, tree, a.scale, g, rmax, rsum, o);
            load_kv<T, NDS, NDT>(kA, vA, kr, vr, first + (i + 2) * nw, c, g, vsoff);
            attend_block<T, NDS, NDT>(kB, vB, s_q, lane, mrow, first + (i + 1) * nw, m, L, Tb, q, tree, a.scale, g, rmax,
                                      rsum, o);
            attend_block<T, NDS, NDT>(kA, vA, s_q, lane, mrow, first + (i + 2) * nw, m, L, Tb, q, tree, a.scale, g, rmax,
                                      rsum, o);
        } else {
            if (rem >= 1)
                attend_block<T, NDS, NDT>(kA, vA, s_q, lane, mrow, first + i * nw, m, L, Tb, q, tree, a.scale, g, rmax,
                                          rsum, o);
            if (rem == 2)
                attend_block<T, NDS, NDT>(kB, vB, s_q, lane, mrow, first + (i + 1) * nw, m, L, Tb, q, tree, a.scale, g,
                                          rmax, rsum, o);
        }

        rsum += __shfl_xor(rsum, 16, 64);
        rsum += __shfl_xor(rsum, 32, 64);
        // the wave's partial (to its own maximum) goes to its LDS region, in
        // place of its Q
        {
            f32x4_t* own = reinterpret_cast<f32x4_t*>(s_q);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) own[dt * 64 + lane] = o[dt];
        }
        if (g == 0) {
            s_max[wave][c] = rmax;
            s_sum[wave][c] = rsum;
        }
        __syncthreads();
        // log-sum-exp merge of the waves' partials in wave order; output tiles
        // are spread over the waves
        float alpha[kMaxWaves];
        float gmax = -INFINITY;
#pragma unroll
        for (int w = 0; w < kMaxWaves; ++w) {
            alpha[w] = w < nw ? s_max[w][c] : -INFINITY;
            gmax = fmaxf(gmax, alpha[w]);
        }
        float den = 0.f;
#pragma unroll
        for (int w = 0; w < kMaxWaves; ++w) {
            alpha[w] = alpha[w] == -INFINITY ? 0.f : expf(alpha[w] - gmax);
            if (w < nw) den += alpha[w] * s_sum[w][c];
        }
        for (int dt = wave; dt < NDT; dt += nw) {
            f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int w = 0; w < kMaxWaves; ++w)
                if (w < nw) acc += opart[(w * RGN + dt) * 64 + lane] * alpha[w];
            if (m >= q) continue;
            const int d = 16 * (cx * NDT + dt) + 4 * g;
            if (a.splits > 1) {
                // partial of this workgroup: O scaled to its row maximum, the maximum, the sum; stored
                // device-coherent (agent scope), since the tile's last split may run on another XCD
                float* pr = a.part + (((size_t)bh * a.splits + sp) * (n_rt * 16) + m) * (DH + 4);
#pragma unroll
                for (int r = 0; r < 4; ++r) __hip_atomic_store(pr + d + r, acc[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (dt == 0 && g == 0) {
                    __hip_atomic_store(pr + DH, gmax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(pr + DH + 1, den, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                continue;
            }
            const float inv = 1.0f / den;
            const size_t row = ((size_t)b * q + m) * a.ldo + (size_t)h * DH;
            if (a.out_f32) {
                float* po = reinterpret_cast<float*>(a.out) + row + d;
#pragma unroll
                for (int r = 0; r < 4; ++r) po[r] = acc[r] * inv;
            } else if constexpr (sizeof(T) == 2) {   // 4 bf16 in one 8-byte store
                const uint2 pk = {f32x2_to_bf16x2(acc[0] * inv, acc[1] * inv), f32x2_to_bf16x2(acc[2] * inv, acc[3] * inv)};
                *reinterpret_cast<uint2*>(reinterpret_cast<T*>(a.out) + row + d) = pk;
            } else {
                T* po = reinterpret_cast<T*>(a.out) + row + d;
#pragma unroll
                for (int r = 0; r < 4; ++r) po[r] = to_elem<T>(acc[r] * inv);
            }
        }
    }
    if (a.splits > 1) {
        // Arrival: every thread's partial stores have completed at device scope before the count is
        // raised (the wait covers them; agent-scope stores write through to the coherence point), so
        // the split that brings the count to `splits` sees every partial of the tile.  It resets the
        // count for the next launch and merges.
        __shared__ int s_last;
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0) {
            int* ctr = a.counter + (size_t)bh * n_rt + rt;
            const int old = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = old == a.splits - 1;
            if (s_last) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();
        if (s_last) combine_tile<T, DH>(a, bh, rt, n_rt);
    }
}

// Blocks of many rows with the chain mask (prefill chunks): one workgroup of
// 8 waves per (sequence, head, 64-row tile).  The waves come in pairs per 16
// rows: wave (r, kp) owns rows 16r .. 16r + 15 of the tile and the key blocks
// of parity kp, and runs the per-block step above over those its rows can see;
// at the end each pair merges its two partial results by log-sum-exp through
// LDS (parity 0 first).  A 32-key block's K rows and V's key-permuted columns
// are contiguous runs of the cache; the workgroup stages two blocks per step in
// LDS (rows padded by 32 bytes, two buffers, two register sets of loads so the
// blocks of step i + 2 are requested while step i's are used), so a block is
// read from L2 once per tile rather than once per wave.
static constexpr int kRowSub = 4;                 // 16-row subtiles per workgroup
static constexpr int kRowWaves = 2 * kRowSub;     // two key parities per subtile
template <typename T, int DH>
__global__ void __launch_bounds__(64 * kRowWaves) attn_rows_kernel(AttnArgs a) {
    constexpr int NDS = DH / 32, NDT = DH / 16, E = (int)sizeof(T);
    constexpr int KLD = DH + 32 / E, VLD = 32 + 32 / E;   // staged row strides (elements)
    constexpr int CH = 16 / E;                              // elements per 16-byte chunk
    constexpr int NCH = 32 * DH / CH;                       // chunks per staged operand of one block
    constexpr int NT = 64 * kRowWaves, PER = 2 * NCH / NT;  // two blocks per step
    static_assert(PER * NT == 2 * NCH, "whole chunks per thread");
    constexpr int NQF = (E == 2 ? 2 : 1) * NDS;              // Q fragments per lane (hi, and lo for bf16)
    constexpr int KBLK = 32 * KLD, VBLK = DH * VLD;
    // [buffer][block of the step] K and V tiles; after the last step, the parity-1 partials for the merge
    constexpr int STAGE_BYTES = 2 * 2 * (KBLK + VBLK) * E;
    constexpr int MERGE_BYTES = kRowSub * (NDT * 64 * 16 + 2 * 64 * 4);
    static_assert(MERGE_BYTES <= STAGE_BYTES, "merge buffer fits the stage buffers");
    __shared__ __align__(16) unsigned char smem[STAGE_BYTES];
    __shared__ Frag<T> s_qf[kRowSub][NQF * 64];
    T* s_stage = reinterpret_cast<T*>(smem);
    auto s_k = [&](int buf, int j) { return s_stage + (buf * 2 + j) * (KBLK + VBLK); };
    auto s_v = [&](int buf, int j) { return s_stage + (buf * 2 + j) * (KBLK + VBLK) + KBLK; };

    const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int rs = wave % kRowSub, kp = wave / kRowSub;
    const int c = lane & 15, g = lane >> 4;
    const int q = a.q, n_rt = (q + 63) / 64;
    const int rt = (int)blockIdx.x % n_rt, bh = (int)blockIdx.x / n_rt;
    const int b = bh / a.H, h = bh % a.H;
    const int L = a.cache_len[b];
    if (L + q > a.S_max) {   // the host checks capacity; never read past this sequence's cache
        if (tid == 0) atomicOr(a.err, 4);
        return;
    }
    const T* kbase = reinterpret_cast<const T*>(a.kc) + ((size_t)b * a.H + h) * a.S_max * DH;
    const T* vbase = reinterpret_cast<const T*>(a.vc) + ((size_t)b * a.H + h) * a.S_max * DH;
    const int r0 = 64 * rt, w0 = r0 + 16 * rs, m = w0 + c;
    const int nblk = (L + min(r0 + 63, q - 1) + 32) / 32;                 // the tile's last row
    const int wblk = w0 < q ? (L + min(w0 + 15, q - 1) + 32) / 32 : 0;     // this subtile's last row
    const int nstep = (nblk + 1) / 2;

    // the subtile's Q rows as matrix-core fragments (hi / lo) in LDS, written by its parity-0 wave;
    // rows past q read row q - 1
    if (kp == 0) {
        const f32x4_t* qsrc =
            reinterpret_cast<const f32x4_t*>(a.qbuf + (((size_t)b * q + min(m, q - 1)) * a.H + h) * DH + 8 * g);
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds) {
            const f32x4_t q0 = qsrc[ds * 8], q1 = qsrc[ds * 8 + 1];
            const float x8[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
            Frag<T> fh, fl;
            split_frag<T>(x8, fh, fl);
            s_qf[rs][ds * 64 + lane] = fh;
            if constexpr (E == 2) s_qf[rs][(NDS + ds) * 64 + lane] = fl;
        }
    }
    // Two register sets: while step i's blocks are used from LDS, step i + 1's (requested one step
    // earlier) go to the other buffer and step i + 2's are requested.  Block indices are clamped (a
    // repeated last block is staged, never used), and the steps run in unconditional pairs, so the
    // wait before each LDS write counts only the older set's loads.
    struct Stage { u32x4_t k[PER], v[PER]; };
    Stage st0, st1;
    auto gload = [&](Stage& r, int step) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int ch = tid + NT * i, j = ch / NCH, cc = ch % NCH;
            const size_t off = (size_t)min(2 * step + j, nblk - 1) * 32 * DH;
            r.k[i] = reinterpret_cast<const u32x4_t*>(kbase + off)[cc];
            r.v[i] = reinterpret_cast<const u32x4_t*>(vbase + off)[cc];
        }
    };
    auto lstore = [&](const Stage& r, int buf) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int ch = tid + NT * i, j = ch / NCH, cc = ch % NCH;
            *reinterpret_cast<u32x4_t*>(s_k(buf, j) + (cc / (DH / CH)) * KLD + (cc % (DH / CH)) * CH) = r.k[i];
            *reinterpret_cast<u32x4_t*>(s_v(buf, j) + (cc / (32 / CH)) * VLD + (cc % (32 / CH)) * CH) = r.v[i];
        }
    };
    gload(st0, 0);
    gload(st1, 1);
    lstore(st0, 0);
    __syncthreads();

    float rmax = -INFINITY, rsum = 0.f;
    f32x4_t o[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int Tb = L + q;
    // step i from LDS buffer i & 1 (this wave: block 2i + kp); `next` holds step i + 1, `free` takes i + 2
    auto step = [&](int i, const Stage& next, Stage& free) {
        const int buf = i & 1, blk = 2 * i + kp;
        gload(free, i + 2);
        if (blk < wblk) {
            const T* sk = s_k(buf, kp);
            const T* sv = s_v(buf, kp);
            Frag<T> kf[2][NDS], vf[NDT];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds) kf[kt][ds] = Frag<T>::load(sk + (16 * kt + c) * KLD + ds * 32 + 8 * g);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) vf[dt] = Frag<T>::load(sv + (16 * dt + c) * VLD + 8 * g);
            attend_block<T, NDS, NDT>(kf, vf, s_qf[rs], lane, 0ull, blk, m, L, Tb, q, false, a.scale, g, rmax, rsum, o);
        }
        __builtin_amdgcn_sched_barrier(0);
        // the other buffer was last read in step i - 1, before the barrier that ended it
        lstore(next, buf ^ 1);
        __syncthreads();
    };
    int i = 0;
    for (; i + 1 < nstep; i += 2) {
        step(i, st1, st0);
        step(i + 1, st0, st1);
    }
    if (i < nstep) step(i, st1, st0);

    // merge the two key parities of each subtile: parity 1 leaves its partial in LDS (the stage
    // buffers are free after the last step's barrier), parity 0 combines and writes
    rsum += __shfl_xor(rsum, 16, 64);
    rsum += __shfl_xor(rsum, 32, 64);
    f32x4_t* m_o = reinterpret_cast<f32x4_t*>(smem) + rs * NDT * 64;
    float* m_s = reinterpret_cast<float*>(smem + kRowSub * NDT * 64 * 16) + rs * 128;
    if (kp == 1) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) m_o[dt * 64 + lane] = o[dt];
        m_s[lane] = rmax;
        m_s[64 + lane] = rsum;
    }
    __syncthreads();
    if (kp == 1 || m >= q || wblk == 0) return;
    const float m1 = m_s[lane], s1 = m_s[64 + lane];
    const float gmax = fmaxf(rmax, m1);
    const float a0 = rmax == -INFINITY ? 0.f : expf(rmax - gmax), a1 = m1 == -INFINITY ? 0.f : expf(m1 - gmax);
    const float inv = 1.0f / (a0 * rsum + a1 * s1);
    const size_t row = ((size_t)b * q + m) * a.ldo + (size_t)h * DH;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
        const int d = 16 * dt + 4 * g;
        const f32x4_t acc = o[dt] * a0 + m_o[dt * 64 + lane] * a1;
        if (a.out_f32) {
            float* po = reinterpret_cast<float*>(a.out) + row + d;
#pragma unroll
            for (int r = 0; r < 4; ++r) po[r] = acc[r] * inv;
        } else if constexpr (E == 2) {   // 4 bf16 in one 8-byte store
            const uint2 pk = {f32x2_to_bf16x2(acc[0] * inv, acc[1] * inv), f32x2_to_bf16x2(acc[2] * inv, acc[3] * inv)};
            *reinterpret_cast<uint2*>(reinterpret_cast<T*>(a.out) + row + d) = pk;
        } else {
            T* po = reinterpret_cast<T*>(a.out) + row + d;
#pragma unroll
            for (int r = 0; r < 4; ++r) po[r] = to_elem<T>(acc[r] * inv);
        }
    }
}

hipError_t launch_attention_rows(int dtype, int head_dim, const AttnArgs& a, hipStream_t s, hipEvent_t ev0,
                                 hipEvent_t ev1) {
    if (a.q < 1 || a.q > 4096 || a.mask || a.B < 1 || a.H < 1 || a.S_max < 32 || a.S_max % 32 || a.ldo % 4 ||
        !a.qbuf || !a.kc || !a.vc || !a.cache_len || !a.out || !a.err)
        return hipErrorInvalidValue;
    void (*kern)(AttnArgs) = nullptr;
    // float models with 128-wide heads would need more LDS than a workgroup has: attn_kernel serves them
    if (dtype == 1) kern = head_dim == 128 ? attn_rows_kernel<uint16_t, 128> : head_dim == 64 ? attn_rows_kernel<uint16_t, 64> : nullptr;
    else kern = head_dim == 64 ? attn_rows_kernel<float, 64> : nullptr;
    if (!kern) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(a.B * a.H * ((a.q + 63) / 64)));
    if (ev0)
        hipExtLaunchKernelGGL(kern, grid, dim3(64 * kRowWaves), 0, s, ev0, ev1, 0, a);
    else
        hipLaunchKernelGGL(kern, grid, dim3(64 * kRowWaves), 0, s, a);
    return hipGetLastError();
}

template <typename T, int DH>
static hipError_t launch_dh(const AttnPlan& p, const AttnArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    void (*kern)(AttnArgs) = attn_kernel<T, DH, 1>;
    if (p.cols == 2) kern = attn_kernel<T, DH, 2>;
    else if (p.cols == 4) kern = attn_kernel<T, DH, 4>;
    else if constexpr (DH / 16 >= 8) { if (p.cols == 8) kern = attn_kernel<T, DH, 8>; }
    if (ev0)
        hipExtLaunchKernelGGL(kern, dim3(p.grid), dim3(64 * p.waves), p.lds_bytes, s, ev0, ev1, 0, a);
    else
        hipLaunchKernelGGL(kern, dim3(p.grid), dim3(64 * p.waves), p.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_attention(int dtype, int head_dim, const AttnPlan& p, const AttnArgs& a, hipStream_t s,
                            hipEvent_t ev0, hipEvent_t ev1) {
    if (a.q < 1 || a.q > 4096 || (a.mask && a.q > 64) || p.waves < 1 || p.waves > kMaxWaves || a.splits < 1 || a.splits > kMaxSplits ||
        a.splits != p.splits || (a.splits > 1 && (!a.part || !a.counter)) || p.row_tiles != (a.q + 15) / 16 ||
        p.grid != a.B * a.H * a.splits * p.row_tiles * p.cols || a.ldo % 4 != 0 ||
        a.per_split != p.per_split || a.per_split < 1 || a.cols != p.cols || p.cols < 1 || p.cols > kMaxCols ||
        (p.cols & (p.cols - 1)) != 0 || p.cols > head_dim / 16 || (p.cols > 1 && a.splits != 1))
        return hipErrorInvalidValue;
    if (dtype == 1) {
        if (head_dim == 128) return launch_dh<uint16_t, 128>(p, a, s, ev0, ev1);
        if (head_dim == 64) return launch_dh<uint16_t, 64>(p, a, s, ev0, ev1);
    } else {
        if (head_dim == 128) return launch_dh<float, 128>(p, a, s, ev0, ev1);
        if (head_dim == 64) return launch_dh<float, 64>(p, a, s, ev0, ev1);
    }
    return hipErrorInvalidValue;
}

}  // namespace sdsat
