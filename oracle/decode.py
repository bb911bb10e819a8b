"""Oracle for the two-step-draft-then-verify loop (Section 2.1, Eq. 1-3).

State of one sequence: a committed KV cache holding tokens t_0..t_{L-1} and
a *pending* token t_L that is known but not yet cached.

One loop (greedy, Section 2.1.1):

* Draft step 1 (Eq. 1): run the block [t_L, a_1, ..., a_k] at positions
  L..L+k.  Row 0 gives the exact next token t_{L+1}; row j (j >= 1, an
  adaptive token) gives the draft d_j for position L+1+j.  Only row 0 is
  committed (the adaptive rows' K/V are discarded).
* Draft step 2 (Eq. 2): with L advanced by one, run [t_L, d_1, ..., d_k] at
  positions L..L+k.  Row j gives o_j, the target's token after the first j
  drafts.
* Verification (Eq. 3): draft d_j is accepted while every earlier draft was
  accepted and d_j equals o_{j-1} (the "stop cur loop" branch ends the
  loop at the first mismatch, so acceptance is a prefix).  With m accepted
  drafts the loop emits o_0..o_m and commits block rows 0..m; the pending
  token becomes o_m.

So a loop costs two block forwards and emits m + 2 tokens, 2 <= m + 2 <= k + 2
(the bound stated after Eq. 3), and the emitted sequence equals plain greedy
decoding (stated at the end of Section 2.1.1).

Nucleus variant (Section 2.1.2), chain form: the exact tokens are sampled
instead of arg-maxed, each with the uniform keyed by its own absolute
position, and drafts are the arg-max of the adaptive rows (one branch of the
paper's draft tree).  Verification keeps the longest prefix of drafts that
the sampled outputs confirm, as in the greedy rule.  Because the token at
position i is always Sample(p(. | t_<i), U(seed, b, i)), the output equals
plain autoregressive nucleus sampling with the same uniforms.

Start-up (the paper leaves it open): the prompt's first P-1 tokens are
committed by a prefill and the last prompt token is the first pending token.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import model as M
from . import sampling as S


def verify_greedy(logits: np.ndarray, drafts=None):
    """Eq. 3 on one block.  Returns (o [q] int, m).

    o_j is the arg-max of row j (lowest id among ties).  With drafts
    d_1..d_{q-1} (the block's rows 1..q-1), m is the number of leading j with
    d_j == o_{j-1}.  Without drafts (draft step 1) m is 0.
    """
    o = np.array([S.argmax_lowest(r) for r in np.asarray(logits, np.float32)], np.int64)
    if drafts is None:
        return o, 0
    m = 0
    for j in range(1, o.shape[0]):
        if int(drafts[j - 1]) != int(o[j - 1]):
            break
        m = j
    return o, m


def verify_nucleus(logits: np.ndarray, drafts, temperature, top_p, top_k, seed, b, pos0):
    """Nucleus counterpart of ``verify_greedy``.  Returns (tokens [q], m, margin).

    With drafts: s_j = Sample(row j, U(seed, b, pos0 + j)) for every row and m
    counts leading matches d_j == s_{j-1}.  Without drafts (draft step 1):
    row 0 is sampled with U(seed, b, pos0), rows 1.. are arg-maxed (the chain
    of most probable drafts), and m is 0.  ``pos0`` is the absolute position
    of the token sampled from row 0.  ``margin`` is the smallest rounding
    margin of any sample taken.
    """
    lg = np.asarray(logits, np.float32)
    q = lg.shape[0]
    out = np.zeros(q, np.int64)
    margin = np.inf
    for j in range(q):
        if drafts is None and j > 0:
            out[j] = S.argmax_lowest(lg[j])
            continue
        tok, mg = S.sample(lg[j], temperature, top_p, top_k, S.uniform(seed, b, pos0 + j))
        out[j] = tok
        margin = min(margin, mg)
    if drafts is None:
        return out, 0, margin
    m = 0
    for j in range(1, q):
        if int(drafts[j - 1]) != int(out[j - 1]):
            break
        m = j
    return out, m, margin


@dataclass
class Trace:
    """Every block the loop ran: tokens, positions, cache length, logits."""
    blocks: list = field(default_factory=list)
    loop_m: list = field(default_factory=list)
    margins: list = field(default_factory=list)
    paths: list = field(default_factory=list)     # draft tree: the accepted branch's block rows per loop


def _block(shape, weights, cache, tokens, bf16, per_row, trace):
    L = cache.length
    pos = np.arange(L, L + len(tokens))
    logits, kv = M.forward_block(shape, weights, cache, tokens, pos, bf16=bf16, per_row=per_row)
    if trace is not None:
        trace.blocks.append({"tokens": np.asarray(tokens, np.int64), "cache_len": L,
                             "logits": logits.astype(np.float32) if bf16 else logits})
    return logits, kv


def generate_sdsat(shape, weights, prompt, k, max_new, adaptive, mode="greedy",
                   temperature=1.0, top_p=1.0, top_k=0, seed=0, b=0,
                   bf16=False, per_row=False, force_drafts=None, trace=None, prefill_chunk=0,
                   on_prefill_chunk=None):
    """SDSAT generation of ``max_new`` tokens for one sequence.

    ``force_drafts(n, k)``, if given, replaces the drafts of draft step 1 by
    the tokens it returns for output positions n..n+k-1 (used to force the
    all-accept and all-reject bounds).  ``prefill_chunk`` > 0 prefills the
    prompt in blocks of that many rows (the same values up to summation
    order).  Returns (tokens, per-loop m list).
    """
    prompt = np.asarray(prompt, np.int64)
    adaptive = [int(a) for a in adaptive[:k]]
    cache = M.prefill(shape, weights, prompt[:-1], bf16=bf16, per_row=per_row, chunk=prefill_chunk,
                      on_chunk=on_prefill_chunk)
    pending = int(prompt[-1])
    out: list[int] = []
    ms: list[int] = []
    greedy = mode == "greedy" or temperature <= 0.0
    while len(out) < max_new:
        # draft step 1: [pending, a_1..a_k]
        L = cache.length
        logits, kv = _block(shape, weights, cache, [pending] + adaptive, bf16, per_row, trace)
        if greedy:
            d1, _ = verify_greedy(logits, None)
        else:
            d1, _, mg = verify_nucleus(logits, None, temperature, top_p, top_k, seed, b, L + 1)
            if trace is not None:
                trace.margins.append(mg)
        t1 = int(d1[0])
        drafts = [int(x) for x in d1[1:]]
        cache.commit(kv, [0])
        out.append(t1)
        if force_drafts is not None:
            drafts = [int(x) for x in force_drafts(len(out), k)]
        # draft step 2: [t1, d_1..d_k]
        L = cache.length
        logits, kv = _block(shape, weights, cache, [t1] + drafts, bf16, per_row, trace)
        if greedy:
            o, m = verify_greedy(logits, drafts)
        else:
            o, m, mg = verify_nucleus(logits, drafts, temperature, top_p, top_k, seed, b, L + 1)
            if trace is not None:
                trace.margins.append(mg)
        cache.commit(kv, range(m + 1))
        out.extend(int(x) for x in o[: m + 1])
        pending = int(o[m])
        ms.append(m)
    if trace is not None:
        trace.loop_m = ms
    return out[:max_new], ms


# ---------------------------------------------------------------- draft tree (Section 2.1.2)
#
# Draft step 1 offers, at each adaptive row j, several possible draft tokens.
# Draft step 2 arranges them as a tree run in one block with tree attention,
# and verification keeps the longest branch the target confirms.  The paper
# leaves the tree shape to a manual design; the reading here is a chain plus
# siblings of width w: depth j holds the w most probable tokens of adaptive
# row j (ties to the lower id); the first forms the main chain, the other
# w - 1 are leaves under the chain node one level up.  w = 1 is the chain.


def top_candidates(row: np.ndarray, w: int) -> list[int]:
    """The w largest values of a logit row, ties to the lower id."""
    r = np.asarray(row, np.float32).astype(np.float64)
    order = np.lexsort((np.arange(r.shape[0]), -r))
    return [int(i) for i in order[:w]]


def draft_tree(t1: int, cand: list[list[int]]):
    """Draft step 2's block for the candidates cand[j-1] of depths j = 1..k.

    Rows: 0 the root t1; 1..k the chain (depth j, parent j-1); then, depth by
    depth, each depth's other candidates (parent: the chain node one level
    up).  Returns (tokens, parent, depth) lists over the rows.
    """
    tokens, parent, depth = [int(t1)], [-1], [0]
    k = len(cand)
    for j in range(1, k + 1):
        tokens.append(int(cand[j - 1][0]))
        parent.append(j - 1)
        depth.append(j)
    for j in range(1, k + 1):
        for t in cand[j - 1][1:]:
            tokens.append(int(t))
            parent.append(j - 1)
            depth.append(j)
    return tokens, parent, depth


def tree_visibility(parent) -> np.ndarray:
    """[q, q] boolean: row r may attend to block row a iff a is r or one of its ancestors."""
    q = len(parent)
    vis = np.zeros((q, q), bool)
    for r in range(q):
        a = r
        while a >= 0:
            vis[r, a] = True
            a = parent[a]
    return vis


def verify_tree(targets, tokens, parent):
    """Longest confirmed branch (the verification of Section 2.1.2, in the
    form of Eq. 3).  From the root, the target's token at the current node
    (targets[node]) is emitted; if a child of the node carries that token (the
    lowest such row) the walk descends into it, otherwise it stops.  Returns
    (path rows from the root, emitted tokens); m = len(path) - 1 drafts were
    accepted and len(path) tokens emitted."""
    children: dict[int, list[int]] = {}
    for r in range(1, len(parent)):
        children.setdefault(parent[r], []).append(r)
    path, emitted, node = [0], [], 0
    while True:
        t = int(targets[node])
        emitted.append(t)
        nxt = next((r for r in children.get(node, []) if int(tokens[r]) == t), None)
        if nxt is None:
            return path, emitted
        path.append(nxt)
        node = nxt


def generate_sdsat_tree(shape, weights, prompt, k, width, max_new, adaptive, mode="nucleus",
                        temperature=1.0, top_p=1.0, top_k=0, seed=0, b=0, bf16=False, per_row=False,
                        force_cand=None, trace=None):
    """SDSAT with a draft tree of the given width (Section 2.1.2).  Returns (tokens, per-loop m).

    ``force_cand(n, k, width)``, if given, replaces draft step 1's candidates
    (a list of k lists of width tokens) for a loop whose first token is output
    number n (to place known continuations at chosen tree nodes)."""
    prompt = np.asarray(prompt, np.int64)
    adaptive = [int(a) for a in adaptive[:k]]
    cache = M.prefill(shape, weights, prompt[:-1], bf16=bf16, per_row=per_row)
    pending = int(prompt[-1])
    out: list[int] = []
    ms: list[int] = []
    greedy = mode == "greedy" or temperature <= 0.0
    while len(out) < max_new:
        # draft step 1: [pending, a_1..a_k]; t1 from row 0, candidates from the adaptive rows
        L = cache.length
        logits, kv = _block(shape, weights, cache, [pending] + adaptive, bf16, per_row, trace)
        lg = np.asarray(logits, np.float32)
        if greedy:
            t1 = S.argmax_lowest(lg[0])
        else:
            t1, mg = S.sample(lg[0], temperature, top_p, top_k, S.uniform(seed, b, L + 1))
            if trace is not None:
                trace.margins.append(mg)
        cand = [top_candidates(lg[j], width) for j in range(1, k + 1)]
        cache.commit(kv, [0])
        out.append(int(t1))
        if force_cand is not None:
            cand = [[int(t) for t in c] for c in force_cand(len(out), k, width)]
        # draft step 2: the tree, rows at positions L + depth, each seeing its ancestors
        tokens, parent, depth = draft_tree(t1, cand)
        L = cache.length
        vis = tree_visibility(parent)
        logits, kv = M.forward_block(shape, weights, cache, tokens, L + np.asarray(depth), visible=vis,
                                     bf16=bf16, per_row=per_row)
        if trace is not None:
            trace.blocks.append({"tokens": np.asarray(tokens, np.int64), "cache_len": L, "parent": list(parent),
                                 "logits": logits.astype(np.float32) if bf16 else logits})
        lg = np.asarray(logits, np.float32)
        targets = []
        for r in range(len(tokens)):
            if greedy:
                targets.append(S.argmax_lowest(lg[r]))
            else:
                t, mg = S.sample(lg[r], temperature, top_p, top_k, S.uniform(seed, b, L + 1 + depth[r]))
                targets.append(t)
                if trace is not None:
                    trace.margins.append(mg)
        path, emitted = verify_tree(targets, tokens, parent)
        if trace is not None:
            trace.paths.append(list(path))
        cache.commit(kv, path)
        out.extend(emitted)
        pending = emitted[-1]
        ms.append(len(path) - 1)
    if trace is not None:
        trace.loop_m = ms
    return out[:max_new], ms


def generate_ar(shape, weights, prompt, max_new, mode="greedy", temperature=1.0, top_p=1.0,
                top_k=0, seed=0, b=0, bf16=False, per_row=False, trace=None):
    """Plain autoregressive decoding, one token per block forward."""
    prompt = np.asarray(prompt, np.int64)
    cache = M.prefill(shape, weights, prompt[:-1], bf16=bf16, per_row=per_row)
    pending = int(prompt[-1])
    out: list[int] = []
    greedy = mode == "greedy" or temperature <= 0.0
    while len(out) < max_new:
        L = cache.length
        logits, kv = _block(shape, weights, cache, [pending], bf16, per_row, trace)
        if greedy:
            t = S.argmax_lowest(logits[0].astype(np.float32))
        else:
            t, mg = S.sample(logits[0].astype(np.float32), temperature, top_p, top_k,
                             S.uniform(seed, b, L + 1))
            if trace is not None:
                trace.margins.append(mg)
        cache.commit(kv, [0])
        out.append(int(t))
        pending = int(t)
    return out
