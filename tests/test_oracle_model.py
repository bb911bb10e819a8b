"""Pins for the oracle's decoder forward (CPU only).

Each test fixes the oracle against something other than its own code:
closed forms at hand-built weights, bit-level definitions, and invariants
that a wrong sign, index, pairing or transposition would break.
"""
import math
from types import SimpleNamespace

import numpy as np
import pytest

from oracle import model as M
from paper_2403_18647_amd import synth


def _shape(**kw):
    base = dict(n_layers=1, d_model=4, n_heads=1, head_dim=4, d_ffn=2, vocab=6,
                n_adaptive=2, rms_eps=1e-6, rope_base=10000.0, dtype="fp32")
    base.update(kw)
    return SimpleNamespace(**base)


def _zero_weights(sh):
    d, f = sh.d_model, sh.d_ffn
    W = {"embed": np.zeros((sh.vocab + sh.n_adaptive, d), np.float32),
         "final_norm": np.ones(d, np.float32), "lm_head": np.zeros((sh.vocab, d), np.float32)}
    for i in range(sh.n_layers):
        p = f"l{i}."
        W.update({p + "attn_norm": np.ones(d, np.float32), p + "ffn_norm": np.ones(d, np.float32),
                  p + "wq": np.zeros((d, d), np.float32), p + "wk": np.zeros((d, d), np.float32),
                  p + "wv": np.zeros((d, d), np.float32), p + "wo": np.zeros((d, d), np.float32),
                  p + "w_gate": np.zeros((f, d), np.float32), p + "w_up": np.zeros((f, d), np.float32),
                  p + "w_down": np.zeros((d, f), np.float32)})
    return W


# ---------------------------------------------------------------- bf16 rounding
def test_bf16_round_matches_bit_level_rne():
    """frexp-based rounding == the IEEE bit-level definition on float32 inputs."""
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * s for s in (1e-3, 1.0, 300.0)])
    # exact halfway cases: low 16 bits == 0x8000, with even and odd kept parts
    hw = (rng.integers(0x3F000000, 0x40800000, 2000, dtype=np.uint32) & ~np.uint32(0xFFFF)) | np.uint32(0x8000)
    x = np.concatenate([x, hw.view(np.float32)])
    bits = x.view(np.uint32).astype(np.uint64)
    low = bits & 0xFFFF
    keep = bits >> 16
    up = (low > 0x8000) | ((low == 0x8000) & ((keep & 1) == 1))
    ref = ((keep + up.astype(np.uint64)) << 16).astype(np.uint32).view(np.float32)
    got = M.bf16_round(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref.astype(np.float64))


def test_bf16_round_values():
    vals = M.bf16_round(np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(2 ** -130), 0.0]))
    np.testing.assert_array_equal(vals, [1.0, 1.0, 1.0 + 2 ** -6, -(2 ** -130), 0.0])


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_constant_vector_closed_form():
    c, eps, d = -3.0, 1e-5, 16
    g = np.linspace(0.5, 2.0, d)
    out = M.rms_norm(np.full((1, d), c), g, eps)
    np.testing.assert_allclose(out[0], c / math.sqrt(c * c + eps) * g, rtol=1e-15)


def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64))
    y = M.rms_norm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1) / math.sqrt(64), 1.0, rtol=1e-14)
    np.testing.assert_allclose(M.rms_norm(7.5 * x, np.ones(64), 0.0), y, rtol=1e-13)


# ---------------------------------------------------------------- RoPE
def test_rope_closed_form_head_dim_4():
    """Dh=4: pairs (0,2) at frequency 1 and (1,3) at base^-1/2."""
    base, pos = 100.0, 3
    cos, sin = M.rope_cos_sin([pos], 4, base)
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    y = M.apply_rope(x, cos, sin)[0, 0]
    a0, a1 = pos * 1.0, pos * base ** -0.5
    c0, s0 = float(np.float32(math.cos(a0))), float(np.float32(math.sin(a0)))
    c1, s1 = float(np.float32(math.cos(a1))), float(np.float32(math.sin(a1)))
    expect = [1 * c0 - 3 * s0, 2 * c1 - 4 * s1, 1 * s0 + 3 * c0, 2 * s1 + 4 * c1]
    np.testing.assert_allclose(y, expect, rtol=1e-15, atol=1e-15)


def test_rope_identity_at_zero_norm_and_relative_position():
    rng = np.random.default_rng(1)
    Dh = 64
    q = rng.standard_normal((1, 1, Dh))
    k = rng.standard_normal((1, 1, Dh))
    c0, s0 = M.rope_cos_sin([0], Dh, 1e4)
    np.testing.assert_array_equal(M.apply_rope(q, c0, s0), q)
    for m, n, s in [(5, 2, 11), (100, 37, 1000), (0, 9, 3)]:
        cm, sm = M.rope_cos_sin([m], Dh, 1e4)
        cn, sn = M.rope_cos_sin([n], Dh, 1e4)
        cms, sms = M.rope_cos_sin([m + s], Dh, 1e4)
        cns, sns = M.rope_cos_sin([n + s], Dh, 1e4)
        qm = M.apply_rope(q, cm, sm)
        np.testing.assert_allclose(np.linalg.norm(qm), np.linalg.norm(q), rtol=1e-6)
        a = np.sum(qm * M.apply_rope(k, cn, sn))
        b = np.sum(M.apply_rope(q, cms, sms) * M.apply_rope(k, cns, sns))
        np.testing.assert_allclose(a, b, rtol=1e-5, atol=1e-5)   # float32 tables


# ---------------------------------------------------------------- forward, hand-built models
def test_zero_layers_contribution_gives_normalised_embedding_logits():
    """Wo = Wd = 0: the residual stream is the embedding, logits = RMSNorm(E[t]) W_lm^T."""
    sh = _shape(n_layers=2, d_model=8, head_dim=8, vocab=5)
    W = _zero_weights(sh)
    rng = np.random.default_rng(2)
    W["embed"][:] = rng.standard_normal(W["embed"].shape)
    W["lm_head"][:] = rng.standard_normal(W["lm_head"].shape)
    W["final_norm"][:] = rng.uniform(0.5, 1.5, 8)
    for i in range(2):          # attention and FFN are live but their outputs are projected to zero
        for n in ("wq", "wk", "wv", "w_gate", "w_up"):
            W[f"l{i}.{n}"][:] = rng.standard_normal(W[f"l{i}.{n}"].shape)
    w = M.Weights(sh, W)
    cache = M.KVCache(2, 1, 8)
    toks = [3, 0, 6, 1]
    logits, _ = M.forward_block(sh, w, cache, toks, np.arange(4))
    for r, t in enumerate(toks):
        e = W["embed"][t].astype(np.float64)
        rms = np.linalg.norm(e) / math.sqrt(8)
        expect = W["lm_head"].astype(np.float64) @ (e / math.sqrt(rms * rms + sh.rms_eps) * W["final_norm"])
        np.testing.assert_allclose(logits[r], expect, rtol=1e-12)


def test_uniform_attention_takes_prefix_mean_of_permuted_values():
    """Wq = Wk = 0 gives equal scores: each row averages V over its visible prefix.

    Wv is a cyclic shift and Wo is triangular, so a transposed Wv (the inverse
    shift), a transposed Wo or a causal off-by-one changes the result."""
    d = 4
    sh = _shape(d_model=d, head_dim=d, vocab=6)
    W = _zero_weights(sh)
    rng = np.random.default_rng(3)
    W["embed"][:] = rng.standard_normal(W["embed"].shape)
    P = np.roll(np.eye(d), 1, axis=0)            # (P h)_i = h_{i-1}
    W["l0.wv"][:] = P
    Wo = np.triu(np.ones((d, d))) * 0.5 + np.eye(d) * 0.5
    W["l0.wo"][:] = Wo
    W["lm_head"][: d] = np.eye(d)                 # logits[:d] = final normalised x
    w = M.Weights(sh, W)
    toks = [1, 4, 2, 5, 0]
    logits, _ = M.forward_block(sh, w, M.KVCache(1, 1, d), toks, np.arange(5))
    E = W["embed"].astype(np.float64)
    hs = [E[t] / math.sqrt(np.mean(E[t] ** 2) + sh.rms_eps) for t in toks]
    for r in range(5):
        vmean = np.mean([np.roll(hs[j], 1) for j in range(r + 1)], axis=0)
        x = E[toks[r]] + Wo @ vmean
        xf = x / math.sqrt(np.mean(x ** 2) + sh.rms_eps)
        np.testing.assert_allclose(logits[r][:d], xf, rtol=1e-12, atol=1e-12)


def test_two_key_softmax_uses_inverse_sqrt_head_dim():
    """Two visible keys with scores a and b weigh their values by the logistic
    of (a - b) / sqrt(Dh).  Wq and Wk are not symmetric, so a transposed
    projection changes the scores."""
    d = 4
    sh = _shape(d_model=d, head_dim=d, vocab=6, rms_eps=0.0)
    W = _zero_weights(sh)
    W["embed"][0] = [2.0, 0.0, 0.0, 0.0]          # unit RMS: RMSNorm leaves it unchanged
    W["embed"][1] = [0.0, 2.0, 0.0, 0.0]
    Wq = np.array([[0.3, 1.5, 0, 0], [0, 0, 0, 0], [0, 0.2, 0, 0], [0, 0, 0, 0]])
    Wk = np.array([[1.0, 0, 0, 0], [0.4, 0.7, 0, 0], [0, 0, 0, 0], [0, 0, 0, 0]])
    W["l0.wq"][:] = Wq
    W["l0.wk"][:] = Wk
    W["l0.wv"][:] = np.eye(d)
    W["l0.wo"][:] = np.eye(d)
    W["lm_head"][:d] = np.eye(d)
    w = M.Weights(sh, W)
    cache = M.KVCache(1, 1, d)
    _, kv = M.forward_block(sh, w, cache, [0], [0])     # position 0: RoPE is the identity
    cache.commit(kv, [0])
    logits, _ = M.forward_block(sh, w, cache, [1], [0])
    e0, e1 = W["embed"][0].astype(np.float64), W["embed"][1].astype(np.float64)
    q = Wq @ e1
    s_cached, s_self = float(q @ (Wk @ e0)), float(q @ (Wk @ e1))
    assert abs(s_cached - s_self) > 1.0
    wt_self = 1.0 / (1.0 + math.exp(-(s_self - s_cached) / math.sqrt(d)))
    x = e1 + wt_self * e1 + (1 - wt_self) * e0
    xf = x / math.sqrt(np.mean(x ** 2))
    np.testing.assert_allclose(logits[0][:d], xf, rtol=1e-12, atol=1e-12)


def test_swiglu_gates_with_the_gate_projection():
    """d=2, F=1: FFN adds silu(h_0) * h_1 to dimension 0 (gate reads h_0, up reads h_1)."""
    sh = _shape(d_model=2, head_dim=2, d_ffn=1, vocab=3, rms_eps=0.0)
    W = _zero_weights(sh)
    W["embed"][0] = [1.2, -0.4]
    W["l0.w_gate"][:] = [[1.0, 0.0]]
    W["l0.w_up"][:] = [[0.0, 1.0]]
    W["l0.w_down"][:] = [[1.0], [0.0]]
    W["lm_head"][:2] = np.eye(2)
    w = M.Weights(sh, W)
    logits, _ = M.forward_block(sh, w, M.KVCache(1, 1, 2), [0], [0])
    e = W["embed"][0].astype(np.float64)
    h = e / math.sqrt(np.mean(e ** 2))
    silu_h0 = h[0] * (1.0 / (1.0 + math.exp(-h[0])))
    x = e + np.array([silu_h0 * h[1], 0.0])
    np.testing.assert_allclose(logits[0][:2], x / math.sqrt(np.mean(x ** 2)), rtol=1e-12)


# ---------------------------------------------------------------- forward, invariants
def _tiny(gain_std=0.1, **kw):
    wl = synth.workload("tiny", gain_std=gain_std, **kw)
    W = {n: synth.tensor(wl, n) for n in synth.tensor_names(wl.shape)}
    return wl, M.Weights(wl.shape, W)


def test_causality_row_ignores_later_rows():
    wl, w = _tiny()
    sh = wl.shape
    cache = M.prefill(sh, w, synth.prompts(wl)[0][:10])
    a, _ = M.forward_block(sh, w, cache, [5, 6, 7, 8], np.arange(10, 14))
    b, _ = M.forward_block(sh, w, cache, [5, 6, 900, 901], np.arange(10, 14))
    np.testing.assert_array_equal(a[:2], b[:2])
    assert np.abs(a[2:] - b[2:]).max() > 1e-6


def test_position_shift_invariance():
    """RoPE makes scores depend on relative positions only: shifting every
    position (cache and block) by s leaves the logits unchanged up to the
    float32 rounding of the rotary tables."""
    wl, w = _tiny(weight_std=0.2)
    sh = wl.shape
    toks = synth.prompts(wl)[0][:12]
    outs = []
    for shift in (0, 777):
        cache = M.KVCache(sh.n_layers, sh.n_heads, sh.head_dim)
        _, kv = M.forward_block(sh, w, cache, toks[:8], np.arange(8) + shift, want_logits=True)
        cache.commit(kv, range(8))
        lg, _ = M.forward_block(sh, w, cache, toks[8:], np.arange(8, 12) + shift)
        outs.append(lg)
    np.testing.assert_allclose(outs[0], outs[1], atol=2e-5 * np.abs(outs[0]).max())
    assert np.abs(outs[0]).max() > 1.0


def test_block_equals_rows_one_at_a_time_bitwise():
    """Block-causal attention over q rows == q single-row blocks, committed one by one
    (per-row arithmetic; the property the greedy-equivalence claim rests on)."""
    wl, w = _tiny()
    sh = wl.shape
    pr = synth.prompts(wl)[0]
    cache = M.prefill(sh, w, pr[:20], per_row=True)
    blk = [int(t) for t in pr[20:26]]
    lg_blk, _ = M.forward_block(sh, w, cache, blk, np.arange(20, 26), per_row=True)
    c2 = cache.copy()
    for r, t in enumerate(blk):
        lg1, kv = M.forward_block(sh, w, c2, [t], [20 + r], per_row=True)
        np.testing.assert_array_equal(lg1[0], lg_blk[r])
        c2.commit(kv, [0])


def test_tree_visibility_matches_chain_on_each_branch():
    """A row that sees only its ancestors equals the same row in a chain block
    built from those ancestors (tree-attention mask, Section 2.1.2)."""
    wl, w = _tiny()
    sh = wl.shape
    pr = synth.prompts(wl)[0]
    cache = M.prefill(sh, w, pr[:16], per_row=True)
    # tree: row0 root; rows 1,2 children of 0; row 3 child of 2
    toks = [10, 11, 12, 13]
    vis = np.array([[1, 0, 0, 0], [1, 1, 0, 0], [1, 0, 1, 0], [1, 0, 1, 1]], bool)
    depth = [0, 1, 1, 2]
    lg_tree, _ = M.forward_block(sh, w, cache, toks, [16 + d for d in depth], visible=vis, per_row=True)
    lg_chain, _ = M.forward_block(sh, w, cache, [10, 12, 13], [16, 17, 18], per_row=True)
    np.testing.assert_array_equal(lg_tree[3], lg_chain[2])
    np.testing.assert_array_equal(lg_tree[2], lg_chain[1])


def test_bf16_mode_rounds_kv_cache():
    wl, w = _tiny()
    sh = wl.shape
    _, kv = M.forward_block(sh, w, M.KVCache(sh.n_layers, sh.n_heads, sh.head_dim), [1, 2, 3],
                            np.arange(3), bf16=True)
    for k, v in kv:
        np.testing.assert_array_equal(M.bf16_round(k), k)
        np.testing.assert_array_equal(M.bf16_round(v), v)


def test_out_of_range_token_rejected():
    wl, w = _tiny()
    sh = wl.shape
    with pytest.raises(ValueError):
        M.forward_block(sh, w, M.KVCache(sh.n_layers, sh.n_heads, sh.head_dim),
                        [sh.vocab + sh.n_adaptive], [0])


def test_bf16_round_of_strided_and_transposed_arrays():
    """Rounding is elementwise whatever the memory layout: a transposed or strided
    view rounds to the same values as a C-contiguous copy of it."""
    rng = np.random.default_rng(9)
    a = rng.standard_normal((6, 4)) * 37.0
    for view in (a.T, a[::2, ::-1], np.asfortranarray(a)):
        ref = M.bf16_round(np.ascontiguousarray(view))
        got = M.bf16_round(view)
        np.testing.assert_array_equal(got, ref)
        assert np.abs(got - view).max() <= np.abs(view).max() * 2.0 ** -8


# ---------------------------------------------------------------- bf16 rounding points, hand-built models
# Each model below uses embedding rows of +-1 entries (RMS 1, so RMSNorm leaves
# them unchanged), eps 0, every token at position 0 (rotary embedding is the
# identity), and float32 weights that are exact binary fractions.  One storage
# rounding of the bf16 model turns a value that is not a bf16 number into one
# that is, and a cancellation right after it makes the difference decide a
# logit exactly.  bf16 keeps 8 significant bits: near 1 its spacing is 2**-7,
# so 1 + e rounds to 1 for |e| < 2**-8.
def _bf16_shape(**kw):
    base = dict(n_layers=1, d_model=4, n_heads=1, head_dim=4, d_ffn=2, vocab=4, n_adaptive=0,
                rms_eps=0.0, rope_base=10000.0, dtype="bf16")
    base.update(kw)
    return SimpleNamespace(**base)


def _run_at_position_zero(sh, W, cached, query, bf16):
    """Commit the tokens ``cached`` one at a time, then run ``query`` as a one-row
    block; every row at position 0."""
    w = M.Weights(sh, W)
    cache = M.KVCache(sh.n_layers, sh.n_heads, sh.head_dim)
    for t in cached:
        _, kv = M.forward_block(sh, w, cache, [t], [0], bf16=bf16)
        cache.commit(kv, [0])
    logits, _ = M.forward_block(sh, w, cache, [query], [0], bf16=bf16)
    return logits[0]


def test_bf16_attention_norm_output_is_rounded():
    """The first RMSNorm's output is stored in bf16.  Gain 1 + 2**-9 on dimension 0
    rounds to 1, so Q_0 = h_0 - h_1 is exactly 0: the two keys (K_0 = -512 and
    +512) get equal weight, the values -1 and +1 average to 0, and the residual
    stream keeps the embedding [1, 1, 1, 1]; logit 0 reads h_0 - h_1 of the final
    norm = 0.  Unrounded, Q_0 = 2**-9 makes the self weight sigmoid(1)."""
    sh = _bf16_shape()
    W = _zero_weights(sh)
    W["embed"][0] = [1, 1, 1, 1]         # the query token
    W["embed"][1] = [1, 1, -1, 1]        # the cached key
    W["l0.attn_norm"][:] = [1 + 2.0 ** -9, 1, 1, 1]
    W["l0.wq"][0] = [1, -1, 0, 0]
    W["l0.wk"][0] = [0, 0, 512, 0]
    W["l0.wv"][0] = [0, 0, 1, 0]
    W["l0.wo"][0] = [1, 0, 0, 0]
    W["lm_head"][0] = [1, -1, 0, 0]
    W["lm_head"][1] = [0, 1, 0, 0]
    lg = _run_at_position_zero(sh, W, [1], 0, bf16=True)
    assert lg[0] == 0.0 and lg[1] == 1.0
    # without the storage roundings the same model moves logit 0: the construction sees the rounding
    assert abs(_run_at_position_zero(sh, W, [1], 0, bf16=False)[0]) > 0.1


def test_bf16_attention_output_is_rounded():
    """The attention output is stored in bf16.  Uniform weights over three keys
    with V_0 = 1 + 2**-7, 1, 1 average to 1 + 2**-7/3, which rounds to 1; the
    output projection adds it to x_0 = -1, leaving exactly 0 there, which logit 0
    reads through the final norm (bf16(0) = 0)."""
    sh = _bf16_shape()
    W = _zero_weights(sh)
    W["embed"][0] = [-1, 1, 1, 1]        # query, V_0 = -a + b = 1
    W["embed"][1] = [1, 1, 1, 1]         # V_0 = a + b = 1 + 2**-7
    W["embed"][2] = [-1, 1, -1, -1]      # V_0 = 1
    W["l0.wv"][0] = [2.0 ** -8, 1 + 2.0 ** -8, 0, 0]
    W["l0.wo"][0] = [1, 0, 0, 0]
    W["lm_head"][0] = [1, 0, 0, 0]
    lg = _run_at_position_zero(sh, W, [1, 2], 0, bf16=True)
    assert lg[0] == 0.0
    assert _run_at_position_zero(sh, W, [1, 2], 0, bf16=False)[0] != 0.0


def test_bf16_swiglu_product_is_rounded():
    """The SwiGLU product is stored in bf16: silu(16) * 2**-4 = 1 - 1.1e-7 rounds to
    1, the down projection adds it to x_0 = -1, and logit 0 reads exactly 0."""
    sh = _bf16_shape()
    W = _zero_weights(sh)
    W["embed"][0] = [-1, 1, 1, 1]
    W["l0.w_gate"][0] = [0, 16, 0, 0]
    W["l0.w_up"][0] = [0, 2.0 ** -4, 0, 0]
    W["l0.w_down"][0] = [1, 0]
    W["lm_head"][0] = [1, 0, 0, 0]
    assert _run_at_position_zero(sh, W, [], 0, bf16=True)[0] == 0.0
    assert _run_at_position_zero(sh, W, [], 0, bf16=False)[0] != 0.0


def test_bf16_ffn_norm_output_is_rounded():
    """The second RMSNorm's output is stored in bf16: gain 1 + 2**-9 rounds to 1,
    so the gate input h_0 - h_1 is exactly 0, silu(0) = 0 and the feed-forward
    adds nothing (unrounded it adds silu(2**-9) * 64 to x_0)."""
    sh = _bf16_shape()
    W = _zero_weights(sh)
    W["embed"][0] = [1, 1, 1, 1]
    W["l0.ffn_norm"][:] = [1 + 2.0 ** -9, 1, 1, 1]
    W["l0.w_gate"][0] = [1, -1, 0, 0]
    W["l0.w_up"][0] = [0, 0, 64, 0]
    W["l0.w_down"][0] = [1, 0]
    W["lm_head"][0] = [1, -1, 0, 0]
    assert _run_at_position_zero(sh, W, [], 0, bf16=True)[0] == 0.0
    assert _run_at_position_zero(sh, W, [], 0, bf16=False)[0] != 0.0


def test_bf16_final_norm_output_is_rounded():
    """The final RMSNorm's output is stored in bf16 before the LM head: gain
    1 + 2**-9 rounds to 1, so the logit h_0 - h_1 is exactly 0 (unrounded 2**-9)."""
    sh = _bf16_shape()
    W = _zero_weights(sh)
    W["embed"][0] = [1, 1, 1, 1]
    W["final_norm"][:] = [1 + 2.0 ** -9, 1, 1, 1]
    W["lm_head"][0] = [1, -1, 0, 0]
    assert _run_at_position_zero(sh, W, [], 0, bf16=True)[0] == 0.0
    assert _run_at_position_zero(sh, W, [], 0, bf16=False)[0] == 2.0 ** -9


# ---------------------------------------------------------------- multi-head split
def test_two_heads_split_projections_head_major():
    """Two heads of 2: head h owns projection rows (and output columns) 2h, 2h+1.
    Head 0 weighs the cached key and itself by the logistic of its score
    difference; head 1 has zero queries and averages its values.  Each head's
    output lands in its own two columns of the output projection's input.  A
    dim-major split (head h on rows h, h+2) mixes the heads and changes the logits."""
    sh = _shape(d_model=4, n_heads=2, head_dim=2, vocab=4, rms_eps=0.0)
    W = _zero_weights(sh)
    W["embed"][0] = [1, 1, -1, 1]        # query
    W["embed"][1] = [1, -1, 1, -1]       # cached key
    # head 0: q = 1.5 * h_0, k = h_1 (dimension 0 of the head); v = (h_2, h_3)
    W["l0.wq"][0] = [1.5, 0, 0, 0]
    W["l0.wk"][0] = [0, 1, 0, 0]
    W["l0.wv"][0] = [0, 0, 1, 0]
    W["l0.wv"][1] = [0, 0, 0, 1]
    # head 1: q = 0, v = (h_0 + h_1, h_2 - h_3) / 2
    W["l0.wv"][2] = [0.5, 0.5, 0, 0]
    W["l0.wv"][3] = [0, 0, 0.5, -0.5]
    W["l0.wo"][:] = np.array([[1, 0, 0, 0], [0, 2, 0, 0], [0, 0, 3, 0], [0, 0, 0, 4]], np.float32)
    W["lm_head"][:] = np.eye(4)
    lg = _run_at_position_zero(sh, W, [1], 0, bf16=False)
    eq, ek = W["embed"][0].astype(np.float64), W["embed"][1].astype(np.float64)
    # head 0 scores (scale 1/sqrt(2)): q = 1.5, keys k = ek_1 = -1 (cached), eq_1 = 1 (self)
    s_c, s_s = 1.5 * ek[1] / math.sqrt(2), 1.5 * eq[1] / math.sqrt(2)
    w_s = 1.0 / (1.0 + math.exp(-(s_s - s_c)))
    o0 = w_s * eq[2:4] + (1 - w_s) * ek[2:4]
    v1 = lambda e: np.array([(e[0] + e[1]) / 2, (e[2] - e[3]) / 2])
    o1 = 0.5 * (v1(eq) + v1(ek))
    o = np.concatenate([o0, o1])
    x = eq + np.array([1, 2, 3, 4]) * o
    np.testing.assert_allclose(lg, x / math.sqrt(np.mean(x ** 2)), rtol=1e-12, atol=1e-12)


def test_float32_blas_mode_matches_float64_within_float32_rounding():
    """Float32 weights switch the linear layers and attention to float32 products (the mode used
    for the 7B / 13B shapes): the logits equal the float64 oracle's up to float32 rounding, and
    differ from them (so the float32 path is really taken).  Float32 tensors are used in place."""
    wl, w64 = _tiny()
    W = {n: synth.tensor(wl, n) for n in synth.tensor_names(wl.shape)}
    w32 = M.Weights(wl.shape, W, dtype=np.float32)
    assert np.shares_memory(w32["l0.wq"], W["l0.wq"])
    sh = wl.shape
    pr = synth.prompts(wl)[0]
    outs = []
    for w in (w64, w32):
        cache = M.prefill(sh, w, pr[:20], chunk=8)
        lg, _ = M.forward_block(sh, w, cache, pr[20:26], np.arange(20, 26))
        outs.append(lg)
    d = np.abs(outs[0] - outs[1]).max()
    assert 0 < d <= 1e-5 * np.abs(outs[0]).max()
