"""fp64 CPU oracle for the output layer of one beam-search decode step.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline of the benchmark may import this module.  It shares no code with
the HIP path: it does not load the native library and reads nothing it
produces.

What it computes (Hoang et al., "Fast Neural Machine Translation
Implementation", WNMT 2018):

* Section 2.2, the four output-layer steps: projection ``p = w x``, bias
  ``p = p + b``, softmax, and k-best search over the output classes.
* Algorithm 3 (AddBias, three-pass Softmax, Find-Best), written out as the
  plain definition.  The fused kernel (Algorithm 4) reaches the same result
  up to rounding order, so the definition is the reference.
* Beam k-best across each sentence's beam: the k best (hypothesis, word)
  continuations of every sentence, scored as the previous cumulative
  log-probability plus the new log-probability.  The paper calls the k-best
  search a simple extension of the 1-best scan and leaves it unspecified;
  ties keep the lowest flat index, matching the strict ``>`` of every scan
  in Algorithms 3-6 (the first index wins).
* Section 2.1, Algorithm 2: finished hypotheses are removed from the batch
  in order (stable compaction).

Also here, for pinning the readings of the paper: Algorithm 4 (fused
softmax and best, with the corrected sum update), Algorithm 5 (argmax only)
and Algorithm 6 (sharded argmax with reduction), as sequential loops for
small inputs.

Every function works in float64.  bf16 / float32 inputs are widened exactly.
Parity is pinned for every function here (see the ``not gpu`` tests);
orderings of candidates whose scores lie within the comparison tolerance
are not unique and are checked for validity instead of identity.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


# --------------------------------------------------------------------------
# exact widening of the storage formats
# --------------------------------------------------------------------------
def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """float64 copy of a float32 array, or of bf16 bit patterns (uint16)."""
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        u = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# Section 2.2 steps 1-2 / Algorithm 3 AddBias
# --------------------------------------------------------------------------
def logits(h64: np.ndarray, W64: np.ndarray, b64: np.ndarray) -> np.ndarray:
    """x[n, j] = sum_i h[n, i] W[i, j] + b[j]   (projection, then bias)."""
    return h64 @ W64 + b64[None, :]


# --------------------------------------------------------------------------
# Algorithm 3 Softmax (three passes: max, denominator, normalise)
# --------------------------------------------------------------------------
def softmax_three_pass(x: np.ndarray):
    """Row-wise softmax in the three passes of Algorithm 3.

    Returns ``(p, m, s)``: probabilities, row max and row denominator
    ``s = sum_j exp(x_j - m)``.
    """
    m = x.max(axis=1)                                  # pass 1: max for stability
    e = np.exp(x - m[:, None])
    s = e.sum(axis=1)                                  # pass 2: denominator
    p = e / s[:, None]                                 # pass 3: normalise
    return p, m, s


def log_softmax(x: np.ndarray):
    """log p = x - m - ln s; also returns LSE = m + ln s per row."""
    _, m, s = softmax_three_pass(x)
    lse = m + np.log(s)
    return x - lse[:, None], lse


# --------------------------------------------------------------------------
# beam k-best over each sentence's hypotheses (the full definition)
# --------------------------------------------------------------------------
@dataclass
class KBestResult:
    token: np.ndarray      # S x k int64, word index in [0, V)
    parent: np.ndarray     # S x k int64, global row index of the parent hypothesis
    score: np.ndarray      # S x k float64, prev + log p, sorted descending
    next_score: np.ndarray  # S float64, the (k+1)-th best score (-inf if none)
    lse: np.ndarray        # N float64, log-sum-exp of each row


def _check_offsets(off: np.ndarray, N: int):
    off = np.asarray(off, dtype=np.int64)
    if off[0] != 0 or off[-1] != N or np.any(np.diff(off) < 1):
        raise ValueError("offsets must start at 0, end at N and give every sentence >= 1 row")
    return off


def kbest_step(h, W, b, prev, off, k: int, dtype: str = "f32") -> KBestResult:
    """One decode step of the output layer, by definition.

    For every sentence s with rows ``off[s]..off[s+1]-1``: score every
    (row, word) continuation as ``prev[row] + log_softmax(x[row])[word]``,
    flatten parent-major / word-minor, and fully sort by descending score
    with a stable sort (equal scores keep the lower flat index).  The first
    k entries are the result; the (k+1)-th score is kept for the boundary
    rule of the comparison.
    """
    h64, W64 = widen(h, dtype), widen(W, dtype)
    b64 = np.asarray(b, dtype=np.float32).astype(np.float64)
    p64 = np.asarray(prev, dtype=np.float32).astype(np.float64)
    N, V = h64.shape[0], W64.shape[1]
    off = _check_offsets(off, N)
    x = logits(h64, W64, b64)
    logp, lse = log_softmax(x)
    cand = p64[:, None] + logp
    S = off.shape[0] - 1
    tok = np.zeros((S, k), dtype=np.int64)
    par = np.zeros((S, k), dtype=np.int64)
    sc = np.zeros((S, k), dtype=np.float64)
    nxt = np.full(S, -np.inf)
    for s in range(S):
        r0, r1 = off[s], off[s + 1]
        f = cand[r0:r1].reshape(-1)
        order = np.argsort(-f, kind="stable")
        top = order[:k]
        tok[s] = top % V
        par[s] = r0 + top // V
        sc[s] = f[top]
        if f.size > k:
            nxt[s] = f[order[k]]
    return KBestResult(tok, par, sc, nxt, lse)


def kbest_step_threshold(h, W, b, prev, off, k: int, dtype: str = "f32",
                         sentences=None, row_block: int = 256) -> KBestResult:
    """Same result as :func:`kbest_step`, with an exact shortcut for large inputs.

    Per sentence: tau = the (k+1)-th largest score (``np.partition``); every
    flat index with score >= tau is taken in flat order and stably sorted.
    All entries that a full stable sort ranks among the first k+1 have
    score >= tau, and the stable sort of that subset keeps their relative
    order, so the first k+1 entries are identical.

    ``sentences`` restricts the work (and the returned rows of token /
    parent / score / next_score) to the listed sentences; ``lse`` is then
    filled only on their rows (NaN elsewhere).  ``row_block`` bounds the rows
    whose logits are held at once (whole sentences; memory only).
    """
    W64 = widen(W, dtype)
    b64 = np.asarray(b, dtype=np.float32).astype(np.float64)
    prev32 = np.asarray(prev, dtype=np.float32)
    N, V = h.shape[0], W64.shape[1]
    off = _check_offsets(off, N)
    S = off.shape[0] - 1
    sel = list(range(S)) if sentences is None else [int(s) for s in sentences]
    tok = np.zeros((len(sel), k), dtype=np.int64)
    par = np.zeros((len(sel), k), dtype=np.int64)
    sc = np.zeros((len(sel), k), dtype=np.float64)
    nxt = np.full(len(sel), -np.inf)
    lse_all = np.full(N, np.nan)
    # the logits of several sentences' rows come from one product (each row's
    # value is the same sum h[n] . W[:, j] + b[j]); then each sentence is
    # ranked on its own
    i = 0
    while i < len(sel):
        j, nrows = i, 0
        while j < len(sel) and (j == i or nrows + off[sel[j] + 1] - off[sel[j]] <= row_block):
            nrows += off[sel[j] + 1] - off[sel[j]]
            j += 1
        rows = np.concatenate([np.arange(off[s], off[s + 1]) for s in sel[i:j]]).astype(np.int64)
        xb = logits(widen(h[rows], dtype), W64, b64)
        pos = 0
        for q in range(i, j):
            s = sel[q]
            r0, r1 = off[s], off[s + 1]
            x = xb[pos:pos + (r1 - r0)]
            pos += r1 - r0
            logp, lse = log_softmax(x)
            lse_all[r0:r1] = lse
            f = (prev32[r0:r1].astype(np.float64)[:, None] + logp).reshape(-1)
            if f.size > k:
                tau = np.partition(f, f.size - (k + 1))[f.size - (k + 1)]
                idx = np.flatnonzero(f >= tau)
            else:
                idx = np.arange(f.size)
            order = idx[np.argsort(-f[idx], kind="stable")]
            top = order[:k]
            tok[q] = top % V
            par[q] = r0 + top // V
            sc[q] = f[top]
            if order.size > k:
                nxt[q] = f[order[k]]
        i = j
    return KBestResult(tok, par, sc, nxt, lse_all)


# --------------------------------------------------------------------------
# Algorithm 3 Find-Best, Algorithm 4 (fused), Algorithm 5, Algorithm 6
# sequential loops over one vector, for small inputs and for pinning.
# --------------------------------------------------------------------------
def find_best(p) -> tuple:
    """Algorithm 3 Find-Best: scan with strict '>' so the first maximum wins."""
    mx, best = -math.inf, -1
    for i, v in enumerate(p):
        if v > mx:
            mx, best = v, i
    return mx, best


def fused_softmax_best(p, b) -> tuple:
    """Algorithm 4 with the sum update read as ``sum <- exp(delta) * sum + 1``.

    The printed update multiplies by delta; the derivation that follows the
    algorithm rescales the running sum by ``e^delta`` with
    ``delta = max_old - max_new``, which is what is used here.  Returns
    ``(1/sum, best, max, sum)``: the probability of the best class, its
    index, the row max and the denominator relative to that max.
    """
    mx, s, best = -math.inf, 0.0, -1
    for i in range(len(p)):
        q = float(p[i]) + float(b[i])
        if q > mx:
            delta = mx - q
            s = math.exp(delta) * s + 1.0
            mx, best = q, i
        else:
            s = s + math.exp(q - mx)
    return 1.0 / s, best, mx, s


def fused_softmax_best_literal(p, b) -> tuple:
    """Algorithm 4 exactly as printed (``sum <- delta * sum + 1``).

    Kept only so that a test can show the printed update disagreeing with the
    derivation: at the first element delta is -inf and the running sum 0, so
    the literal product is NaN in IEEE arithmetic."""
    mx, s, best = -math.inf, 0.0, -1
    for i in range(len(p)):
        q = float(p[i]) + float(b[i])
        if q > mx:
            delta = mx - q
            s = delta * s + 1.0
            mx, best = q, i
        else:
            s = s + math.exp(q - mx)
    return 1.0 / s, best, mx, s


def argmax_only(p, b) -> int:
    """Algorithm 5: best class of p + b without any softmax (beam 1)."""
    mx, best = -math.inf, -1
    for i in range(len(p)):
        q = float(p[i]) + float(b[i])
        if q > mx:
            mx, best = q, i
    return best


def argmax_sharded(p, b, n_shards: int) -> int:
    """Algorithm 6: per-shard (max, best) in parallel, then a strict '>' reduction.

    Readings: each shard compares against its own running max, indices are
    global, and shards are contiguous and reduced in ascending order, so the
    lowest index wins among equal maxima.
    """
    V = len(p)
    bounds = np.linspace(0, V, n_shards + 1).round().astype(int)
    part = []
    for j in range(n_shards):
        mj, bj = -math.inf, -1
        for i in range(bounds[j], bounds[j + 1]):
            q = float(p[i]) + float(b[i])
            if q > mj:
                mj, bj = q, i
        part.append((mj, bj))
    mx, best = -math.inf, -1
    for mj, bj in part:
        if mj > mx:
            mx, best = mj, bj
    return best


@dataclass
class ArgmaxResult:
    token: np.ndarray     # N int64: argmax_j x[n, j], the lowest j among equal maxima
    value: np.ndarray     # N float64: x[n, token[n]]
    second: np.ndarray    # N float64: the largest x[n, j] over j != token[n] (-inf if V == 1)


def argmax_rows(h, W, b, dtype: str = "f32", rows=None) -> ArgmaxResult:
    """Greedy (beam 1) output layer, Algorithm 5 for every row: the best class
    of p = W h + b, no softmax (the softmax is monotone, so the class is the
    same as the most probable one).  The definition written out: fp64 scores
    and numpy's argmax, which returns the first maximum (the strict '>' scan).
    ``rows`` restricts the work to a subset of rows (results in that order).
    """
    h64 = widen(h, dtype)
    if rows is not None:
        h64 = h64[np.asarray(rows)]
    x = logits(h64, widen(W, dtype), np.asarray(b, dtype=np.float64))
    tok = np.argmax(x, axis=1)
    r = np.arange(x.shape[0])
    val = x[r, tok]
    if x.shape[1] > 1:
        y = x.copy()
        y[r, tok] = -np.inf
        second = y.max(axis=1)
    else:
        second = np.full(x.shape[0], -np.inf)
    return ArgmaxResult(tok, val, second)


def merge_softmax_stats(parts) -> tuple:
    """Combine per-shard (max, sum-of-exp relative to that max) pairs.

    The rescaling identity that follows Algorithm 4, applied between shards:
    ``M = max(m1, m2)``, ``S = s1 e^(m1-M) + s2 e^(m2-M)``.
    """
    M = -math.inf
    for m, _ in parts:
        M = max(M, m)
    S = 0.0
    for m, s in parts:
        if s > 0.0:
            S += s * math.exp(m - M)
    return M, S


# --------------------------------------------------------------------------
# Section 2.1, Algorithm 2: remove finished hypotheses from the batch
# --------------------------------------------------------------------------
@dataclass
class CompactResult:
    keep_idx: np.ndarray        # kept entries, ascending (stable)
    kept_count: int
    new_offsets: np.ndarray     # new_S + 1 offsets of the surviving sentences
    kept_sentence: np.ndarray   # new_S old sentence index of each surviving sentence
    new_S: int


def compact(alive, S: int, k: int) -> CompactResult:
    """Stable removal of finished entries from an S x k batch (sentence-major).

    ``keep_idx`` lists the surviving entries in their original order; a
    sentence survives if any of its entries does, and the new offsets count
    its surviving entries.
    """
    a = np.asarray(alive).reshape(S * k).astype(bool)
    keep = np.flatnonzero(a)
    per_sent = a.reshape(S, k).sum(axis=1)
    ks = np.flatnonzero(per_sent > 0)
    new_off = np.concatenate([[0], np.cumsum(per_sent[ks])]).astype(np.int64)
    return CompactResult(keep, int(keep.size), new_off, ks, int(ks.size))


def compact_entries(alive, entry_sentence=None) -> CompactResult:
    """Section 2.1, Algorithm 2 on a batch given as a flat list of M entries.

    Every entry whose ``alive`` flag is 0 (its hypothesis produced EOS) leaves
    the batch; the rest keep their order (``keep_idx``).  With the sentence id
    of every entry (non-decreasing along the list), a sentence stays in the
    batch if any of its entries does; its new offset counts the surviving
    entries of the sentences before it.  ``kept_sentence`` holds the ids of the
    surviving sentences.
    """
    a = np.asarray(alive).reshape(-1).astype(bool)
    keep = np.flatnonzero(a)
    if entry_sentence is None:
        return CompactResult(keep, int(keep.size), np.zeros(0, np.int64), np.zeros(0, np.int64), 0)
    es = np.asarray(entry_sentence).reshape(-1).astype(np.int64)
    ks, per_sent = np.unique(es[keep], return_counts=True)   # sorted ids with a surviving entry
    new_off = np.concatenate([[0], np.cumsum(per_sent)]).astype(np.int64)
    return CompactResult(keep, int(keep.size), new_off, ks.astype(np.int64), int(ks.size))
