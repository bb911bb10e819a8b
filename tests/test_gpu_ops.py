"""GPU parity of the individual kernels through the C-ABI: skinny GEMM,
block attention, verification and KV commit.  Sizes span several tiles
and ragged tails; verification and commit must be bit-exact."""
import math

import numpy as np
import pytest

from oracle import decode as D
from oracle import model as M
from oracle import sampling as S
from paper_2403_18647_amd import binding as B
from paper_2403_18647_amd import synth

import helpers

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


# ---------------------------------------------------------------- skinny GEMM
@pytest.mark.parametrize("dtype", [0, 1])
@pytest.mark.parametrize("M_,N,K", [(1, 16, 32), (6, 100, 200), (11, 4096, 11008), (24, 1000, 4096),
                                    (64, 530, 777), (3, 33, 1000), (17, 2001 * 16, 256)])
def test_linear_matches_fp64_reference(dtype, M_, N, K):
    print(f"linear dtype={dtype} M={M_} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M_ * 1000 + N + K)
    x = rng.standard_normal((M_, K)).astype(np.float32)
    w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    if dtype == 1:
        w = helpers.bf16_round_f32(w)
        wdev = torch.from_numpy((w.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).view(torch.bfloat16).cuda()
        xr = helpers.bf16_round_f32(x)
    else:
        wdev = torch.from_numpy(w).cuda()
        xr = x
    packed = torch.empty(B.sdsat_linear_packed_bytes(dtype, N, K), dtype=torch.uint8, device="cuda")
    B.sdsat_linear_pack(dtype, N, K, wdev, packed)
    scratch = torch.zeros(B.sdsat_linear_scratch_bytes(M_, N, K), dtype=torch.uint8, device="cuda")
    y = torch.empty((M_, N), dtype=torch.float32, device="cuda")
    xd = torch.from_numpy(x).cuda()
    for _ in range(2):   # second call checks the split-K counters were left at zero
        y.fill_(float("nan"))
        B.sdsat_linear(dtype, M_, N, K, xd, packed, y, scratch)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        ref = xr.astype(np.float64) @ w.astype(np.float64).T
        bound = 1e-5 * (np.abs(xr).astype(np.float64) @ np.abs(w).astype(np.float64).T) + 1e-7
        assert np.all(np.abs(got - ref) <= bound), float(np.max(np.abs(got - ref) / bound))


# ---------------------------------------------------------------- attention
def _attn_case(wl, lens, q, mask=None, seed=0):
    sh = wl.shape
    Bn = len(lens)
    H, Dh = sh.n_heads, sh.head_dim
    ctx = helpers.make_ctx(wl, max_batch=Bn, max_ctx=max(lens) + q + 40, max_block=q)
    rng = np.random.default_rng(seed)
    n = max(lens) + q
    K = rng.standard_normal((Bn, n, H, Dh)).astype(np.float32)
    V = rng.standard_normal((Bn, n, H, Dh)).astype(np.float32)
    Q = rng.standard_normal((Bn, q, H, Dh)).astype(np.float32)
    # block rows of sequence b sit at slots lens[b]..lens[b]+q-1
    pos = np.stack([np.arange(n) for _ in range(Bn)]).astype(np.int32)
    Kw = np.stack([np.concatenate([K[b, :lens[b]], K[b, n - q:], K[b, lens[b]:n - q]]) for b in range(Bn)])
    Vw = np.stack([np.concatenate([V[b, :lens[b]], V[b, n - q:], V[b, lens[b]:n - q]]) for b in range(Bn)])
    B.sdsat_kv_write(ctx.handle, 0, Bn, n, torch.from_numpy(Kw).cuda(), torch.from_numpy(Vw).cuda(),
                     torch.from_numpy(pos).cuda())
    B.sdsat_set_cache_len(ctx.handle, np.array(lens, np.int32))
    out = torch.empty((Bn * q, H * Dh), dtype=torch.float32, device="cuda")
    md = None if mask is None else torch.from_numpy(np.asarray(mask, np.uint64).view(np.int64)).cuda()
    B.sdsat_attention(ctx.handle, 0, Bn, q, torch.from_numpy(Q.reshape(Bn * q, H * Dh)).cuda(), md, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(Bn, q, H, Dh)
    rnd = helpers.bf16_round_f32 if sh.dtype == "bf16" else (lambda a: a)
    for b in range(Bn):
        L = lens[b]
        if mask is None:
            vis = M.chain_visibility(q)
        else:
            mb = np.asarray(mask, np.uint64).reshape(Bn, q)[b]
            vis = np.array([[(int(mb[r]) >> j) & 1 for j in range(q)] for r in range(q)], bool)
        ref = M.attention(rnd(Q[b]).astype(np.float64), rnd(K[b, n - q:]).astype(np.float64),
                          rnd(V[b, n - q:]).astype(np.float64), rnd(K[b, :L]).astype(np.float64),
                          rnd(V[b, :L]).astype(np.float64), vis, 1.0 / math.sqrt(Dh))
        tol = 2e-2 if sh.dtype == "bf16" else 2e-5
        err = np.abs(got[b] - ref).max()
        assert err <= tol, (b, L, err)
    ctx.close()


@pytest.mark.parametrize("lens,q", [([0], 1), ([5], 6), ([31, 32, 33], 6), ([127], 11), ([300, 7], 17),
                                    ([1000], 6), ([64, 2], 40)])
def test_attention_fp32_head64(lens, q):
    print(f"attention fp32 lens={lens} q={q}", flush=True)
    _attn_case(synth.workload("tiny"), lens, q)


@pytest.mark.parametrize("lens,q", [([0], 1), ([45], 6), ([300, 31, 0], 11), ([2000], 6), ([96, 64], 33)])
def test_attention_bf16_head128(lens, q):
    print(f"attention bf16 lens={lens} q={q}", flush=True)
    _attn_case(helpers.small_bf16(), lens, q)


@pytest.mark.parametrize("dtype,lens,q", [("bf16", [0, 37], 200), ("bf16", [129], 511), ("bf16", [1000, 0, 64], 70),
                                          ("fp32", [0], 130), ("fp32", [70, 3], 97)])
def test_attention_prefill_rows(dtype, lens, q):
    """Blocks of more than 16 rows (the prefill attention: 64-row tiles, two waves per 16 rows on
    alternate key blocks, merged at the end): several tiles, a ragged last tile, cache prefixes of
    0 to 1000 keys, a batch with different lengths; every element against the oracle's attention."""
    print(f"attention prefill rows {dtype} lens={lens} q={q}", flush=True)
    _attn_case(helpers.small_bf16() if dtype == "bf16" else synth.workload("tiny"), lens, q)


def test_attention_tree_mask():
    # row 0 root, rows 1,2 children of 0, row 3 child of 2, row 4 child of 1
    par = [-1, 0, 0, 2, 1]
    masks = []
    for r in range(5):
        m, a = 0, r
        while a >= 0:
            m |= 1 << a
            a = par[a]
        masks.append(m)
    _attn_case(helpers.small_bf16(), [20, 70], 5, mask=masks * 2)


# ---------------------------------------------------------------- verification
def _logits(Bn, q, V, std, seed):
    return (np.random.default_rng(seed).standard_normal((Bn, q, V)) * std).astype(np.float32)


def _tiny_ctx(Bn=8, q=11, V=32016):
    sh = synth.small_shape(n_layers=1, d_model=64, n_heads=1, head_dim=64, d_ffn=64, vocab=V,
                           n_adaptive=5, dtype="fp32")
    wl = synth.Workload("verify", sh, seed=4, batch=Bn, k=q - 1, prompt_len=1, max_new=1)
    return helpers.make_ctx(wl, max_batch=Bn, max_ctx=64, max_block=q)


@pytest.mark.parametrize("std", [4.0, 2.0])
def test_verify_greedy_bit_exact(std):
    Bn, q, V = 8, 11, 32016
    lg = _logits(Bn, q, V, std, 4)
    lg[3, 2, [17, 30000]] = lg[3, 2].max() + 1.0          # exact tie: lowest id must win
    o = lg.argmax(-1)
    drafts = np.zeros((Bn, q - 1), np.int32)
    for b in range(Bn):
        mb = b % q
        drafts[b] = (o[b, : q - 1] + 1) % V
        drafts[b, :mb] = o[b, :mb]
    ctx = _tiny_ctx(Bn, q, V)
    tok = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    m = torch.empty(Bn, dtype=torch.int32, device="cuda")
    B.sdsat_verify_greedy(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), torch.from_numpy(drafts).cuda(), tok, m)
    torch.cuda.synchronize()
    tok, m = tok.cpu().numpy().reshape(Bn, q), m.cpu().numpy()
    for b in range(Bn):
        ro, rm = D.verify_greedy(lg[b], drafts[b])
        assert list(tok[b]) == list(ro) and m[b] == rm == b % q
    assert tok[3, 2] == 17
    # draft step 1 form: no drafts, arg-max only
    B.sdsat_verify_greedy(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), None,
                          tok2 := torch.empty(Bn * q, dtype=torch.int32, device="cuda"), None)
    torch.cuda.synchronize()
    assert np.array_equal(tok2.cpu().numpy().reshape(Bn, q), o)
    ctx.close()


@pytest.mark.parametrize("std,T,p,top_k", [(4.0, 0.8, 0.95, 0), (2.0, 0.8, 0.95, 0), (1.3, 1.0, 0.9, 0),
                                           (2.0, 1.0, 0.95, 10), (2.0, 0.2, 0.95, 10), (4.0, 0.0, 0.95, 0)])
def test_verify_nucleus_bit_exact(std, T, p, top_k):
    print(f"nucleus std={std} T={T} p={p} top_k={top_k}", flush=True)
    Bn, q, V = 8, 11, 32016
    lg = _logits(Bn, q, V, std, 5)
    seed = 12345
    pos0 = (100 + 7 * np.arange(Bn)).astype(np.int32)
    # oracle samples first, then drafts that accept exactly b % q of them
    ref = [D.verify_nucleus(lg[b], np.zeros(q - 1), T, p, top_k, seed, b, int(pos0[b])) for b in range(Bn)]
    drafts = np.zeros((Bn, q - 1), np.int32)
    for b in range(Bn):
        s = ref[b][0]
        mb = b % q
        drafts[b] = (s[: q - 1] + 1) % V
        drafts[b, :mb] = s[:mb]
    ctx = _tiny_ctx(Bn, q, V)
    tok = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    m = torch.empty(Bn, dtype=torch.int32, device="cuda")
    B.sdsat_verify_nucleus(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), torch.from_numpy(drafts).cuda(), T, p,
                           top_k, seed, torch.from_numpy(pos0).cuda(), tok, m)
    torch.cuda.synchronize()
    tok, m = tok.cpu().numpy().reshape(Bn, q), m.cpu().numpy()
    for b in range(Bn):
        s, rm, margin = D.verify_nucleus(lg[b], drafts[b], T, p, top_k, seed, b, int(pos0[b]))
        assert margin > 1e-9, "a draw sits at rounding distance from a boundary; pick another seed"
        assert list(tok[b]) == list(s), b
        assert m[b] == rm == b % q
    # draft step 1 form: row 0 sampled, rows 1.. arg-max
    tok1 = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    B.sdsat_verify_nucleus(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), None, T, p, top_k, seed,
                           torch.from_numpy(pos0).cuda(), tok1, None)
    torch.cuda.synchronize()
    tok1 = tok1.cpu().numpy().reshape(Bn, q)
    for b in range(Bn):
        s, _, _ = D.verify_nucleus(lg[b], None, T, p, top_k, seed, b, int(pos0[b]))
        assert list(tok1[b]) == list(s)
    ctx.close()


def test_verify_nucleus_exact_top_p_boundary():
    """The top-p set is the smallest top set whose probability reaches p, inclusive of exact equality.
    At temperature 1e30 every id of a row with distinct logits weighs exactly 1.0 in float64, so at
    p = 0.5 the nucleus is exactly the top half (16008 of 32016 ids), where the mass equals p * E
    exactly; the sampled ids and the accepted lengths must equal the oracle's."""
    Bn, q, V = 2, 4, 32016
    row = -np.arange(V, dtype=np.float32) * np.float32(1e-3)   # distinct, descending: id 0 largest
    lg = np.ascontiguousarray(np.broadcast_to(row, (Bn, q, V)))
    T, p, seed = 1e30, 0.5, 777
    pos0 = np.array([5, 9000], np.int32)
    ids, _, _ = S.nucleus_set(row, T, p)
    assert len(ids) == V // 2
    ref = [D.verify_nucleus(lg[b], np.zeros(q - 1), T, p, 0, seed, b, int(pos0[b])) for b in range(Bn)]
    drafts = np.stack([ref[b][0][: q - 1] for b in range(Bn)]).astype(np.int32)   # accept every draft
    ctx = _tiny_ctx(Bn, q, V)
    tok = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    m = torch.empty(Bn, dtype=torch.int32, device="cuda")
    B.sdsat_verify_nucleus(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), torch.from_numpy(drafts).cuda(), T, p,
                           0, seed, torch.from_numpy(pos0).cuda(), tok, m)
    torch.cuda.synchronize()
    tok, m = tok.cpu().numpy().reshape(Bn, q), m.cpu().numpy()
    for b in range(Bn):
        s_, rm, _ = D.verify_nucleus(lg[b], drafts[b], T, p, 0, seed, b, int(pos0[b]))
        assert list(tok[b]) == list(s_) and m[b] == rm == q - 1, b
        assert all(0 <= t < V // 2 for t in tok[b])
    ctx.close()


@pytest.mark.parametrize("top_k", [10, 60, 20000])
def test_verify_nucleus_top_k_ties_keep_lower_ids(top_k):
    """Top-k with ties at the cut keeps exactly k ids, the lower ids first.  Logits from {0, 1, 2}
    put about 10700 ids in the top tie group: top_k 10 (the small top-k path) and 60 (the radix path)
    cut inside it, 20000 keeps the whole group and cuts inside the next.  Samples and accepted
    lengths must equal the oracle's."""
    Bn, q, V = 4, 3, 32016
    rng = np.random.default_rng(21)
    lg = rng.integers(0, 3, (Bn, q, V)).astype(np.float32)
    T, p, seed = 1.0, 0.9, 4242
    pos0 = (50 + 13 * np.arange(Bn)).astype(np.int32)
    ref = [D.verify_nucleus(lg[b], np.zeros(q - 1), T, p, top_k, seed, b, int(pos0[b])) for b in range(Bn)]
    drafts = np.zeros((Bn, q - 1), np.int32)
    for b in range(Bn):
        s_ = ref[b][0]
        mb = b % q
        drafts[b] = (s_[: q - 1] + 1) % V
        drafts[b, :mb] = s_[:mb]
    ctx = _tiny_ctx(Bn, q, V)
    tok = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    m = torch.empty(Bn, dtype=torch.int32, device="cuda")
    B.sdsat_verify_nucleus(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), torch.from_numpy(drafts).cuda(), T, p,
                           top_k, seed, torch.from_numpy(pos0).cuda(), tok, m)
    torch.cuda.synchronize()
    tok, m = tok.cpu().numpy().reshape(Bn, q), m.cpu().numpy()
    for b in range(Bn):
        s_, rm, margin = D.verify_nucleus(lg[b], drafts[b], T, p, top_k, seed, b, int(pos0[b]))
        assert margin > 1e-9
        assert list(tok[b]) == list(s_) and m[b] == rm == b % q, b
        for j in range(q):   # every sample lies among the k kept ids
            top = np.lexsort((np.arange(V), -lg[b, j]))[:top_k]
            assert tok[b, j] in set(top.tolist())
    ctx.close()


@pytest.mark.parametrize("V,T,p,top_k", [(50000, 0.8, 0.95, 0), (50000, 1.0, 0.9, 100), (131072, 0.8, 0.95, 0),
                                         (131072, 1.0, 0.95, 10), (128256, 1.5, 0.98, 0)])
def test_verify_nucleus_long_vocab_bit_exact(V, T, p, top_k):
    """Vocabularies past 32768 ids (sampled chunk by chunk): samples, accepted lengths and the
    draft-step-1 form equal the oracle's, as for the 32016-id rows.  Ties at a top-k cut and the
    ascending-id inverse CDF cross chunk boundaries here: a tie group spans ids in several chunks."""
    print(f"nucleus V={V} T={T} p={p} top_k={top_k}", flush=True)
    Bn, q = 3, 4
    lg = _logits(Bn, q, V, 2.0, 6)
    lg[1, 1, [5, 40000, V - 1]] = lg[1, 1].max() + 0.5   # a three-way tie for the top across chunks
    seed = 2024
    pos0 = (17 + 5 * np.arange(Bn)).astype(np.int32)
    ref = [D.verify_nucleus(lg[b], np.zeros(q - 1), T, p, top_k, seed, b, int(pos0[b])) for b in range(Bn)]
    drafts = np.zeros((Bn, q - 1), np.int32)
    for b in range(Bn):
        s_ = ref[b][0]
        mb = b % q
        drafts[b] = (s_[: q - 1] + 1) % V
        drafts[b, :mb] = s_[:mb]
    ctx = _tiny_ctx(Bn, q, V)
    tok = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    m = torch.empty(Bn, dtype=torch.int32, device="cuda")
    B.sdsat_verify_nucleus(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), torch.from_numpy(drafts).cuda(), T, p,
                           top_k, seed, torch.from_numpy(pos0).cuda(), tok, m)
    torch.cuda.synchronize()
    tok, m = tok.cpu().numpy().reshape(Bn, q), m.cpu().numpy()
    for b in range(Bn):
        s_, rm, margin = D.verify_nucleus(lg[b], drafts[b], T, p, top_k, seed, b, int(pos0[b]))
        assert margin > 1e-9
        assert list(tok[b]) == list(s_) and m[b] == rm == b % q, b
    tok1 = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    B.sdsat_verify_nucleus(ctx.handle, Bn, q, torch.from_numpy(lg).cuda(), None, T, p, top_k, seed,
                           torch.from_numpy(pos0).cuda(), tok1, None)
    torch.cuda.synchronize()
    tok1 = tok1.cpu().numpy().reshape(Bn, q)
    for b in range(Bn):
        assert list(tok1[b]) == list(D.verify_nucleus(lg[b], None, T, p, top_k, seed, b, int(pos0[b]))[0])
    assert tok1[1, 1] == 5   # row 1 of draft step 1 is the arg-max: the lowest of the tied ids
    ctx.close()


def test_verify_nucleus_vocab_limit():
    """Past 131072 ids nucleus verification reports SDSAT_EUNSUPPORTED; greedy has no limit."""
    Bn, q, V = 1, 2, 131073
    ctx = _tiny_ctx(Bn, q, V)
    lg = torch.zeros((Bn * q, V), dtype=torch.float32, device="cuda")
    tok = torch.empty(Bn * q, dtype=torch.int32, device="cuda")
    pos0 = torch.zeros(Bn, dtype=torch.int32, device="cuda")
    with pytest.raises(B.SdsatError, match="131072"):
        B.sdsat_verify_nucleus(ctx.handle, Bn, q, lg, None, 1.0, 0.9, 0, 1, pos0, tok, None)
    B.sdsat_verify_greedy(ctx.handle, Bn, q, lg, None, tok, None)
    torch.cuda.synchronize()
    assert tok.cpu().numpy().tolist() == [0, 0]
    ctx.close()


# ---------------------------------------------------------------- commit
def test_commit_chain_and_tree_gather():
    wl = helpers.small_bf16()
    sh = wl.shape
    H, Dh = sh.n_heads, sh.head_dim
    ctx = helpers.make_ctx(wl, max_batch=2, max_ctx=128, max_block=6)
    rng = np.random.default_rng(9)
    L = [10, 37]
    n = 50
    K = rng.standard_normal((2, n, H, Dh)).astype(np.float32)
    V = rng.standard_normal((2, n, H, Dh)).astype(np.float32)
    pos = np.stack([np.arange(n)] * 2).astype(np.int32)
    for layer in range(sh.n_layers):
        B.sdsat_kv_write(ctx.handle, layer, 2, n, torch.from_numpy(K).cuda(), torch.from_numpy(V).cuda(),
                         torch.from_numpy(pos).cuda())
    B.sdsat_set_cache_len(ctx.handle, np.array(L, np.int32))
    # chain commit: lengths bump
    B.sdsat_commit_kv(ctx.handle, 2, 6, torch.tensor([3, 0], dtype=torch.int32, device="cuda"))
    assert list(ctx.cache_len()[:2]) == [13, 37]
    B.sdsat_set_cache_len(ctx.handle, np.array(L, np.int32))
    # tree commit: block rows [0, 2, 5] of seq 0 and [1, 4] of seq 1 (rows index slots L..L+5)
    rows = np.array([[0, 2, 5, 0, 0, 0], [1, 4, 0, 0, 0, 0]], np.int32)
    B.sdsat_commit_kv(ctx.handle, 2, 6, torch.tensor([3, 2], dtype=torch.int32, device="cuda"),
                      torch.from_numpy(rows).cuda())
    assert list(ctx.cache_len()[:2]) == [13, 39]
    # the gathered cache, seen by a single query at the new end
    q = 1
    Q = rng.standard_normal((2, q, H, Dh)).astype(np.float32)
    newlen = [13, 39]
    Kq = np.zeros((2, n, H, Dh), np.float32)
    Vq = np.zeros((2, n, H, Dh), np.float32)
    Kn = rng.standard_normal((2, H, Dh)).astype(np.float32)
    Vn = rng.standard_normal((2, H, Dh)).astype(np.float32)
    for layer in range(sh.n_layers):
        B.sdsat_kv_write(ctx.handle, layer, 2, 1, torch.from_numpy(Kn[:, None]).cuda(),
                         torch.from_numpy(Vn[:, None]).cuda(),
                         torch.tensor(newlen, dtype=torch.int32, device="cuda"))
    out = torch.empty((2, H * Dh), dtype=torch.float32, device="cuda")
    B.sdsat_attention(ctx.handle, 1, 2, 1, torch.from_numpy(Q.reshape(2, H * Dh)).cuda(), None, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(2, 1, H, Dh)
    r = helpers.bf16_round_f32
    for b in range(2):
        keep = list(range(L[b])) + [L[b] + int(j) for j in rows[b][: (3 if b == 0 else 2)]]
        ref = M.attention(r(Q[b]).astype(np.float64), r(Kn[b][None]).astype(np.float64),
                          r(Vn[b][None]).astype(np.float64), r(K[b, keep]).astype(np.float64),
                          r(V[b, keep]).astype(np.float64), M.chain_visibility(1), 1.0 / math.sqrt(Dh))
        assert np.abs(got[b] - ref).max() < 2e-2
    ctx.close()


def test_attention_column_slices_do_not_change_values():
    """One key split per head: the sequence replicated 4 times (2 column slices per head) and 8 times
    (one workgroup per head) gives bitwise equal outputs.  Batch 1 (key splits merged by the last
    split to arrive) run three times in a row gives bitwise the same output each time, so the arrival
    counters are back at zero after every launch."""
    shape = synth.small_shape(n_layers=1, d_model=4096, n_heads=32, head_dim=128, d_ffn=64, vocab=64,
                              n_adaptive=2, rope_base=1e6, dtype="bf16")
    H, Dh, L, q = 32, 128, 200, 6
    n = L + q
    rng = np.random.default_rng(11)
    K = rng.standard_normal((n, H, Dh)).astype(np.float32)
    V = rng.standard_normal((n, H, Dh)).astype(np.float32)
    Q = rng.standard_normal((q, H, Dh)).astype(np.float32)
    outs = []
    for Bn in (1, 4, 8):
        wl = synth.Workload("heads32", shape, seed=5, batch=Bn, k=5, prompt_len=1, max_new=1)
        ctx = helpers.make_ctx(wl, max_batch=Bn, max_ctx=n + 40, max_block=q)
        pos = np.tile(np.arange(n, dtype=np.int32), (Bn, 1))
        B.sdsat_kv_write(ctx.handle, 0, Bn, n, torch.from_numpy(np.stack([K] * Bn)).cuda(),
                         torch.from_numpy(np.stack([V] * Bn)).cuda(), torch.from_numpy(pos).cuda())
        B.sdsat_set_cache_len(ctx.handle, np.full(Bn, L, np.int32))
        for _ in range(3 if Bn == 1 else 1):
            out = torch.empty((Bn * q, H * Dh), dtype=torch.float32, device="cuda")
            B.sdsat_attention(ctx.handle, 0, Bn, q,
                              torch.from_numpy(np.concatenate([Q.reshape(q, H * Dh)] * Bn)).cuda(), None, out)
            torch.cuda.synchronize()
            outs.append(out.cpu().numpy().reshape(Bn, q, H * Dh))
        ctx.close()
    one, again, third, four, eight = outs
    assert np.array_equal(one.view(np.uint32), again.view(np.uint32))
    assert np.array_equal(one.view(np.uint32), third.view(np.uint32))
    for b in range(8):
        assert np.array_equal(four[b % 4].view(np.uint32), eight[b].view(np.uint32)), b
    # key splits and one split agree to float rounding
    assert np.abs(one[0] - eight[0]).max() < 1e-5


@pytest.mark.parametrize("lens", [[300], [300, 0], [300, 0, 31, 64], [300, 0, 31, 64, 129, 5, 250, 77]])
def test_attention_32_heads_column_slices(lens):
    """32 heads of 128 over a short cache: batch 1 and 2 split each head's keys over workgroups (the
    last to arrive merges), batch 4 and 8 take one split with 2 and 1 column slices of the output;
    every plan matches the reference."""
    print(f"attention 32 heads, batch {len(lens)}", flush=True)
    shape = synth.small_shape(n_layers=1, d_model=4096, n_heads=32, head_dim=128, d_ffn=64, vocab=64,
                              n_adaptive=2, rope_base=1e6, dtype="bf16")
    wl = synth.Workload("heads32", shape, seed=5, batch=len(lens), k=5, prompt_len=1, max_new=1)
    _attn_case(wl, lens, 6)


@pytest.mark.parametrize("q", [6, 11])
def test_attention_16384_keys_batch8(q):
    """The attention micro-benchmark's shape: batch 8, 32 heads of 128, 16384 committed keys plus the
    block's q rows (Q, K, V ~ N(0, 1)), every output element against the oracle's attention."""
    print(f"attention B8 H32 keys 16384 q={q}", flush=True)
    shape = synth.small_shape(n_layers=1, d_model=4096, n_heads=32, head_dim=128, d_ffn=64, vocab=64,
                              n_adaptive=2, rope_base=1e6, dtype="bf16")
    wl = synth.Workload("attn16k", shape, seed=4, batch=8, k=q - 1, prompt_len=1, max_new=1)
    _attn_case(wl, [16384] * 8, q, seed=4)


def test_stream_read_and_kernel_samples():
    print("stream read (ragged length) and per-launch samples", flush=True)
    # three whole 16 KiB workgroups plus 48 bytes; the kernel only reads
    buf = torch.arange(3 * 4096 + 12, dtype=torch.int32, device="cuda")
    before = buf.clone()
    B.sdsat_stream_read(buf)
    B.sdsat_stream_read(buf, 0)
    torch.cuda.synchronize()
    assert torch.equal(buf, before)
    ctx = _tiny_ctx(1, 2, 1024)
    tok = torch.tensor([3, 7], dtype=torch.int32, device="cuda")
    lg = torch.empty((2, 1024), dtype=torch.float32, device="cuda")
    B.sdsat_reset(ctx.handle, 1)
    B.sdsat_profile_kernel(ctx.handle, "block")
    for _ in range(3):
        B.sdsat_forward_block(ctx.handle, 1, 2, tok, None, lg)
    s = B.sdsat_kernel_samples(ctx.handle)
    assert len(s) == 3 and all(x > 0 for x in s)
    B.sdsat_forward_block(ctx.handle, 1, 2, tok, None, lg)
    ms, n = B.sdsat_kernel_time(ctx.handle)
    assert n == 1 and ms > 0
    B.sdsat_profile_kernel(ctx.handle, "off")
    ctx.close()
