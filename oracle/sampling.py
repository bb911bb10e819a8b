"""Oracle sampler for the nucleus variant (Section 2.1.2; settings in Section 3.4.2).

The paper names nucleus (top-p) sampling with temperature and top-k but does
not fix the order of the three steps, tie handling, or the random numbers.
This oracle takes the following reading, in float64 from float32 logits:

1. z = logits / T.
2. If top_k > 0, keep the top_k largest z; ties at the cut keep the lower ids.
3. e_i = exp(z_i - max z) over the kept ids, E = sum of e_i.
4. The threshold tau* is the largest kept z-value tau with
   S(tau) = sum_{z_i >= tau} e_i >= p * E.  The nucleus is N = {i : z_i >= tau*}
   (every id tied at tau* is in it).
5. With M = S(tau*), return the smallest id i in N whose ascending-id
   cumulative sum of e over N exceeds u * M.

T <= 0 means greedy: the arg-max (lowest id among ties), as the paper treats
greedy search as the special case of nucleus sampling (Figure 1, Table 4).

The uniform u of the token at absolute position ``pos`` of sequence ``b`` is
U(seed, b, pos): output number ``c + 1`` of a SplitMix64 generator
(Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014) started from state ``seed``, with counter c = b * 2**32 + pos,
mapped to [0, 1) by its top 53 bits.
"""
from __future__ import annotations

import numpy as np

_MASK = (1 << 64) - 1
_GOLDEN_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(state: int, n: int) -> int:
    """Output number n (n >= 1) of SplitMix64 started from ``state``."""
    z = (state + n * _GOLDEN_GAMMA) & _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def uniform(seed: int, b: int, pos: int) -> float:
    """U(seed, b, pos) in [0, 1) with 53 random bits."""
    assert 0 <= b < (1 << 31) and 0 <= pos < (1 << 32)
    c = (b << 32) | pos
    return (splitmix64(seed & _MASK, c + 1) >> 11) * (1.0 / (1 << 53))


def argmax_lowest(row: np.ndarray) -> int:
    """Index of the largest value; ties go to the lowest index."""
    return int(np.argmax(row))


def nucleus_set(logits: np.ndarray, temperature: float, top_p: float, top_k: int = 0):
    """Return (ids in N ascending, e over those ids, margin).

    ``margin`` is |S(tau*) - p E| / E, the distance of the top-p decision
    from flipping; a kernel computing the same sums in another order can only
    disagree when it is at rounding level.
    """
    z = np.asarray(logits, np.float32).astype(np.float64) / float(np.float32(temperature))
    V = z.shape[0]
    kept = np.ones(V, bool)
    if top_k and top_k < V:
        order = np.lexsort((np.arange(V), -z))          # by z descending, then id ascending
        kept[:] = False
        kept[order[:top_k]] = True
    zk = np.where(kept, z, -np.inf)
    zmax = zk.max()
    e = np.where(kept, np.exp(zk - zmax), 0.0)
    p = float(np.float32(top_p))
    # S(tau) at every distinct kept value tau, largest first: sort the kept
    # values in descending order and take running sums up to the last copy of tau
    vals = np.unique(zk[kept])[::-1]
    srt = np.sort(zk[kept])[::-1]
    cum = np.cumsum(np.exp(srt - zmax))
    last = np.searchsorted(-srt, -vals, side="right") - 1
    S = cum[last]
    E = S[-1]                                           # S at the smallest kept value
    ok = np.nonzero(S >= p * E)[0]
    j = ok[0] if ok.size else len(vals) - 1
    tau = vals[j]
    ids = np.nonzero(zk >= tau)[0]
    margin = abs(S[j] - p * E) / E
    if j > 0:
        margin = min(margin, abs(S[j - 1] - p * E) / E)
    return ids, e[ids], margin


def sample(logits: np.ndarray, temperature: float, top_p: float, top_k: int, u: float):
    """Sample one id per the module docstring.  Returns (id, margin).

    ``margin`` is the smaller of the top-p margin and |C_i - u M| / M at the
    chosen id's cumulative boundaries.
    """
    if temperature <= 0.0:
        return argmax_lowest(np.asarray(logits, np.float32)), np.inf
    ids, e, m1 = nucleus_set(logits, temperature, top_p, top_k)
    M = e.sum()
    target = u * M
    cum = np.cumsum(e)
    hit = np.nonzero(cum > target)[0]
    i = hit[0] if hit.size else len(ids) - 1
    lo = cum[i - 1] if i > 0 else 0.0
    m2 = min(abs(cum[i] - target), abs(target - lo)) / M
    return int(ids[i]), min(m1, m2)
