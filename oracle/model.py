"""Oracle forward pass of the (unmodified) Llama-style target decoder.

The paper adds adaptive tokens without changing the model's structure
(Section 2 and Section 2.2); its target models are CodeLlama-7B/13B
(Section 3).  The paper does not restate the architecture, so this file
takes the Llama reading: RMSNorm, rotate-half rotary embeddings, multi-head
attention without GQA, SwiGLU feed-forward, no biases, untied LM head.

One call runs one *block* of rows of one sequence against that sequence's
committed KV cache.  Row r of the block sits at absolute position
``positions[r]`` and attends to every committed cache slot plus the block
rows that ``visible[r]`` marks (the chain case is block-causal: rows 0..r).
The block's K/V rows are returned, not stored: the caller commits the ones
it accepts (``KVCache.commit``), which is what draft step 1 and the
verification step do.

Arithmetic is float64 throughout, except that weights held as float32
(``Weights(..., dtype=np.float32)``, the float32-BLAS mode for the 7B / 13B
shapes) make the linear layers float32 matrix products: their inputs are
bf16 values on bf16 models (exact in float32), so that mode differs from the
float64 one only by float32 accumulation in the library's summation order.
With ``bf16=True`` the oracle also rounds
to bf16 (round to nearest even) exactly where a bf16 model stores values:
RMSNorm outputs, K and V (after RoPE, as stored in the cache), the attention
output, and the SwiGLU product.  The residual stream and logits keep full
precision.  With ``per_row=True`` every row is computed by its own
matrix-vector products, so a row's result does not depend on which other
rows share its block (used for the bitwise greedy-equivalence pin).
"""
from __future__ import annotations

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), returned as float64.

    A bf16 value is a float32 whose low 16 bits are zero; rounding goes
    float64 -> bf16 directly (no double rounding through float32).
    """
    # C-contiguous copies, so that the flat views below alias ``out`` (a view of
    # a transposed or strided array would be a copy, never written back)
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.float64)
    flat, res = x.reshape(-1), out.reshape(-1)
    m, e = np.frexp(flat)                       # flat = m * 2**e, 0.5 <= |m| < 1
    # bf16 keeps 8 significant bits: scale so that the kept bits are integral
    scaled = np.ldexp(m, 8)
    r = np.round(scaled)                        # numpy rounds half to even
    res[:] = np.ldexp(r, e - 8)
    res[flat == 0] = 0.0
    return out


def weight_f64(shape, w, dtype=np.float64) -> np.ndarray:
    """Widen a stored weight (float32 values, or uint16 bf16 bit patterns) to
    float64 (or to ``dtype``; no copy when it already has it)."""
    w = np.asarray(w)
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << 16).view(np.float32).astype(dtype)
    return np.asarray(w, dtype)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope_cos_sin(positions, head_dim: int, base: float):
    """Rotary tables for rotate-half RoPE.

    Frequency i (0 <= i < head_dim/2) is base**(-2i/head_dim); the angle is
    position * frequency, both in float64.  cos and sin are then rounded to
    float32 (the table a bf16 or fp32 kernel reads) and returned as float64.
    """
    half = head_dim // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = np.power(float(base), -2.0 * i / head_dim)
    ang = np.asarray(positions, np.float64)[:, None] * inv_freq[None, :]
    return (np.cos(ang).astype(np.float32).astype(np.float64),
            np.sin(ang).astype(np.float32).astype(np.float64))


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE on x [rows, heads, head_dim].

    The pair (x_i, x_{i+D/2}) is rotated by the row's angle i:
    (x_i cos - x_{i+D/2} sin, x_i sin + x_{i+D/2} cos).
    """
    half = x.shape[-1] // 2
    a, b = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


class KVCache:
    """Committed K/V rows of one sequence: per layer, arrays [n, heads, head_dim]."""

    def __init__(self, n_layers: int, n_heads: int, head_dim: int):
        self._k = [np.zeros((16, n_heads, head_dim)) for _ in range(n_layers)]
        self._v = [np.zeros((16, n_heads, head_dim)) for _ in range(n_layers)]
        self._n = 0

    @property
    def length(self) -> int:
        return self._n

    @property
    def k(self):
        return [a[: self._n] for a in self._k]

    @property
    def v(self):
        return [a[: self._n] for a in self._v]

    def commit(self, block_kv, rows) -> None:
        """Append the block rows ``rows`` (in that order) to the committed cache."""
        rows = list(rows)
        n_new = self._n + len(rows)
        for layer, (bk, bv) in enumerate(block_kv):
            if n_new > self._k[layer].shape[0]:
                cap = max(n_new, 2 * self._k[layer].shape[0])
                for store in (self._k, self._v):
                    grown = np.zeros((cap,) + store[layer].shape[1:])
                    grown[: self._n] = store[layer][: self._n]
                    store[layer] = grown
            self._k[layer][self._n:n_new] = bk[rows]
            self._v[layer][self._n:n_new] = bv[rows]
        self._n = n_new

    def copy(self) -> "KVCache":
        c = KVCache.__new__(KVCache)
        c._k = [a.copy() for a in self._k]
        c._v = [a.copy() for a in self._v]
        c._n = self._n
        return c


class Weights:
    """Float64 (or float32: the float32-BLAS mode) view of a weight mapping,
    converted lazily and cached per tensor."""

    def __init__(self, shape, tensors, cache: bool = True, dtype=np.float64):
        self.shape = shape
        self.tensors = tensors
        self.dtype = np.dtype(dtype)
        self._cache = {} if cache else None

    def __getitem__(self, name: str) -> np.ndarray:
        if self._cache is not None and name in self._cache:
            return self._cache[name]
        w = weight_f64(self.shape, self.tensors[name], self.dtype)
        if self._cache is not None:
            self._cache[name] = w
        return w


def _linear(x: np.ndarray, w: np.ndarray, per_row: bool) -> np.ndarray:
    """y = x @ w.T for x [rows, in], w [out, in]; a float32 weight makes it a
    float32 product (x converted to float32), returned as float64."""
    if w.dtype == np.float32:
        x32 = np.ascontiguousarray(x, np.float32)
        if per_row:
            return np.stack([w @ x32[r] for r in range(x.shape[0])]).astype(np.float64) \
                if x.shape[0] else np.zeros((0, w.shape[0]))
        return (x32 @ w.T).astype(np.float64)
    if per_row:
        return np.stack([w @ np.ascontiguousarray(x[r]) for r in range(x.shape[0])]) \
            if x.shape[0] else np.zeros((0, w.shape[0]))
    return x @ w.T


def attention(qh, kh, vh, ck, cv, vis, scale, per_row=False, dtype=np.float64):
    """softmax(q k^T * scale) v over the committed cache plus the visible block rows.

    qh, kh, vh: [q, H, Dh] block rows; ck, cv: [L, H, Dh] committed rows.
    Scores are max-subtracted before exponentiation.  ``dtype`` float32 (the
    float32-BLAS mode) forms scores, softmax and the weighted sum in float32.
    """
    q, H, Dh = qh.shape
    o = np.empty((q, H, Dh))
    if per_row:
        # each row gathers exactly its visible keys, so a row's arithmetic does
        # not depend on how many other rows share its block
        for r in range(q):
            keys = np.concatenate([ck, kh[vis[r]]], axis=0)
            vals = np.concatenate([cv, vh[vis[r]]], axis=0)
            for hd in range(H):
                s = (keys[:, hd, :] @ qh[r, hd]) * scale
                e = np.exp(s - s.max())
                o[r, hd] = (e / e.sum()) @ vals[:, hd, :]
        return o
    L = ck.shape[0]
    keys = np.concatenate([ck, kh], axis=0).transpose(1, 0, 2).astype(dtype)      # [H, L+q, Dh]
    vals = np.concatenate([cv, vh], axis=0).transpose(1, 0, 2).astype(dtype)
    allowed = np.concatenate([np.ones((q, L), bool), vis], axis=1)  # [q, L+q]
    s = np.matmul(qh.transpose(1, 0, 2).astype(dtype), keys.transpose(0, 2, 1)) * dtype(scale)  # [H, q, L+q]
    s = np.where(allowed[None], s, -np.inf)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    p = e / e.sum(axis=-1, keepdims=True)
    return np.matmul(p, vals).transpose(1, 0, 2).astype(np.float64)  # [q, H, Dh]


def chain_visibility(q: int) -> np.ndarray:
    """Block-causal visibility: row r sees block rows 0..r."""
    return np.tril(np.ones((q, q), dtype=bool))


def forward_block(shape, weights: Weights, cache: KVCache, tokens, positions,
                  visible=None, bf16: bool = False, per_row: bool = False,
                  want_logits: bool = True):
    """Run one block of rows through the decoder.

    Returns (logits [q, V] float64 or None, block_kv) where block_kv is a list
    over layers of (K [q, H, Dh], V [q, H, Dh]) for the block rows, ready to be
    committed.  ``visible`` is a [q, q] boolean matrix (row r may attend to
    block row j); None means block-causal.
    """
    tokens = np.asarray(tokens, np.int64)
    positions = np.asarray(positions, np.int64)
    q = tokens.shape[0]
    H, Dh, d = shape.n_heads, shape.head_dim, shape.d_model
    n_emb = shape.vocab + shape.n_adaptive
    if np.any(tokens < 0) or np.any(tokens >= n_emb):
        raise ValueError("token id out of range")
    vis = chain_visibility(q) if visible is None else np.asarray(visible, bool)
    rnd = bf16_round if bf16 else (lambda a: a)
    eps = shape.rms_eps

    x = weights["embed"][tokens].astype(np.float64)           # [q, d]
    cos, sin = rope_cos_sin(positions, Dh, shape.rope_base)
    scale = 1.0 / np.sqrt(Dh)
    block_kv = []
    for layer in range(shape.n_layers):
        p = f"l{layer}."
        h = rnd(rms_norm(x, weights[p + "attn_norm"], eps))
        qh = _linear(h, weights[p + "wq"], per_row).reshape(q, H, Dh)
        kh = _linear(h, weights[p + "wk"], per_row).reshape(q, H, Dh)
        vh = _linear(h, weights[p + "wv"], per_row).reshape(q, H, Dh)
        qh = apply_rope(qh, cos, sin)
        kh = rnd(apply_rope(kh, cos, sin))
        vh = rnd(vh)
        block_kv.append((kh, vh))
        o = attention(qh, kh, vh, cache.k[layer], cache.v[layer], vis, scale, per_row,
                      getattr(weights, "dtype", np.dtype(np.float64)).type)
        o = rnd(o.reshape(q, d))
        x = x + _linear(o, weights[p + "wo"], per_row)
        h2 = rnd(rms_norm(x, weights[p + "ffn_norm"], eps))
        g = _linear(h2, weights[p + "w_gate"], per_row)
        u = _linear(h2, weights[p + "w_up"], per_row)
        a = rnd(silu(g) * u)
        x = x + _linear(a, weights[p + "w_down"], per_row)
    if not want_logits:
        return None, block_kv
    hf = rnd(rms_norm(x, weights["final_norm"], eps))
    logits = _linear(hf, weights["lm_head"], per_row)
    return logits, block_kv


def prefill(shape, weights: Weights, tokens, bf16=False, per_row=False, chunk: int = 0,
            on_chunk=None) -> KVCache:
    """Commit the given tokens at positions 0..n-1 (in chunks of ``chunk`` rows; 0 = one block).
    ``on_chunk(rows_done)``, if given, is called after each chunk (progress reporting)."""
    cache = KVCache(shape.n_layers, shape.n_heads, shape.head_dim)
    tokens = np.asarray(tokens, np.int64)
    n = tokens.shape[0]
    step = n if chunk <= 0 else chunk
    for lo in range(0, n, max(step, 1)):
        t = tokens[lo:lo + step]
        _, kv = forward_block(shape, weights, cache, t, np.arange(lo, lo + len(t)),
                              bf16=bf16, per_row=per_row, want_logits=False)
        cache.commit(kv, range(len(t)))
        if on_chunk is not None:
            on_chunk(lo + len(t))
    return cache
