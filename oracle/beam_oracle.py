"""fp64 CPU oracle of beam search with per-hypothesis end of sentence.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline of the benchmark may import this module.  It shares no code with
the HIP path and reads nothing the native library produces, except the
device results the tests hand it to check.

What it computes (Hoang et al., "Fast Neural Machine Translation
Implementation", WNMT 2018, Section 2.1, Algorithm 2): after every decode
step each sentence keeps the best continuations of its hypotheses, as many
as its beam holds; a continuation ending in EOS leaves the batch as a
finished hypothesis and the sentence's beam shrinks by one; a sentence is
done when its beam is empty (the decode stops when the batch is).  The
paper leaves the rest to the engine; the readings used:

* the step scores are the cumulative log-probabilities of the k-best step
  (``kbest_oracle.kbest_step``), taken in that order;
* at the last step T - 1 every taken continuation finishes, EOS or not;
* a sentence's translation is its finished hypothesis with the best
  ``score / length**alpha`` (length counts the tokens, EOS included; alpha = 0
  compares raw scores), the first finished one among equals;
* the tokens are read back through the parent links of every step.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import kbest_oracle as ko


@dataclass
class FinishResult:
    alive: np.ndarray          # S*k uint8: taken continuations that did not finish
    beam: np.ndarray           # S int: beam sizes after the step
    finished: list             # (original sentence, score, length, history id) in order of finishing
    hist_token: np.ndarray     # S*k tokens of the step
    hist_parent: np.ndarray    # S*k history ids of their parents


def finish_step(token, parent, score, beam, sent_id, row_hist, t: int, T: int, eos: int, k: int,
                hist_base: int) -> FinishResult:
    """The bookkeeping of one step.  ``token``, ``parent`` (global row), ``score``
    are the S x k step outputs, ``beam`` the S beam sizes (the first
    min(beam, k) continuations are taken), ``row_hist`` the history id of each
    row's hypothesis (-1: a root)."""
    token = np.asarray(token).reshape(-1, k)
    parent = np.asarray(parent).reshape(-1, k)
    score = np.asarray(score).reshape(-1, k)
    S = token.shape[0]
    alive = np.zeros(S * k, dtype=np.uint8)
    nb = np.array(beam, dtype=np.int64).copy()
    fins = []
    for s in range(S):
        for r in range(min(int(beam[s]), k)):
            e = s * k + r
            if int(token[s, r]) == eos or t + 1 >= T:
                fins.append((int(sent_id[s]), float(score[s, r]), t + 1, hist_base + e))
                nb[s] -= 1
            else:
                alive[e] = 1
    htok = token.reshape(-1).astype(np.int64)
    hpar = np.asarray(row_hist, dtype=np.int64)[parent.reshape(-1)]
    return FinishResult(alive, nb, fins, htok, hpar)


def best_finished(fins: list, alpha: float) -> int:
    """Index of the best of (score, length, ...) entries by score / length**alpha; first among equals."""
    best, bv = -1, -np.inf
    for i, f in enumerate(fins):
        v = f[1] / (float(f[2]) ** alpha)
        if best < 0 or v > bv:
            best, bv = i, v
    return best


def backtrace(hist_token, hist_parent, h_last: int, length: int) -> list:
    out = [0] * length
    h = h_last
    for pos in range(length - 1, -1, -1):
        out[pos] = int(hist_token[h])
        h = int(hist_parent[h])
    assert h == -1, "history does not end at a root"
    return out


@dataclass
class BeamResult:
    tokens: list = field(default_factory=list)   # per sentence: the tokens, EOS included
    score: list = field(default_factory=list)    # raw cumulative log-probability
    norm: list = field(default_factory=list)     # score / length**alpha
    steps: int = 0


def beam_search(h_of, W, b, S0: int, k: int, T: int, eos: int, alpha: float = 0.0, dtype: str = "f32",
                prev0=None) -> BeamResult:
    """Beam search over S0 sentences, each starting from one hypothesis (score
    prev0[s], default 0) with a beam of k.  ``h_of(s, t, r, prefix)`` gives the
    state of the hypothesis in slot r of sentence s at step t whose tokens so
    far are ``prefix`` (a tuple)."""
    sid = np.arange(S0)
    beam = np.full(S0, k)
    rows = [((), -1, 0.0 if prev0 is None else float(prev0[s])) for s in range(S0)]   # (prefix, hist, score)
    rows_per = np.ones(S0, dtype=np.int64)
    hist_tok, hist_par = [], []
    fin = {s: [] for s in range(S0)}
    t = 0
    while len(sid) > 0 and t < T:
        off = np.concatenate([[0], np.cumsum(rows_per)]).astype(np.int64)
        slot = np.concatenate([np.arange(n) for n in rows_per])
        owner = np.repeat(np.arange(len(sid)), rows_per)
        h = np.stack([h_of(int(sid[owner[i]]), t, int(slot[i]), rows[i][0]) for i in range(len(rows))])
        prev = np.array([r[2] for r in rows])
        # (k continuations per sentence, or all of them where fewer exist: only
        # the exhaustive check asks for more than a sentence has)
        ks = int(min(k, rows_per.min() * np.asarray(W).shape[1]))
        res = ko.kbest_step(h, W, b, prev, off, ks, dtype=dtype)
        base = len(hist_tok)
        fr = finish_step(res.token, res.parent, res.score, beam, sid, [r[1] for r in rows], t, T, eos, ks, base)
        hist_tok.extend(fr.hist_token.tolist())
        hist_par.extend(fr.hist_parent.tolist())
        for f in fr.finished:
            fin[f[0]].append(f)
        keep = np.flatnonzero(fr.alive)
        new_rows = []
        for e in keep:
            s, r = divmod(int(e), ks)
            p = int(res.parent[s, r])
            new_rows.append((rows[p][0] + (int(res.token[s, r]),), base + int(e), float(res.score[s, r])))
        kept_s = sorted(set(int(e) // ks for e in keep))
        rows_per = np.array([int(fr.alive[s * ks:(s + 1) * ks].sum()) for s in kept_s], dtype=np.int64)
        beam = fr.beam[kept_s]
        sid = sid[kept_s]
        rows = new_rows
        t += 1
    out = BeamResult(steps=t)
    for s in range(S0):
        i = best_finished(fin[s], alpha)
        if i < 0:
            out.tokens.append([]), out.score.append(-np.inf), out.norm.append(-np.inf)
            continue
        f = fin[s][i]
        out.tokens.append(backtrace(hist_tok, hist_par, f[3], f[2]))
        out.score.append(f[1])
        out.norm.append(f[1] / float(f[2]) ** alpha)
    return out


def exhaustive_best(h_of, W, b, T: int, eos: int, alpha: float = 0.0, dtype: str = "f32", s: int = 0):
    """Every sequence of at most T tokens that ends in EOS or has length T, scored
    by its summed log-probabilities; the best by score / length**alpha (first in
    lexicographic order among equals).  Exponential: tiny V and T only."""
    V = np.asarray(W).shape[1]
    W64, b64 = ko.widen(W, dtype), np.asarray(b, dtype=np.float64)
    best = (None, -np.inf, -np.inf)

    def rec(prefix, sc):
        nonlocal best
        t = len(prefix)
        x = ko.widen(np.asarray(h_of(s, t, 0, prefix))[None, :], dtype) @ W64 + b64[None, :]
        lp = ko.log_softmax(x)[0][0]
        for j in range(V):
            seq, tot = prefix + (j,), sc + lp[j]
            if j == eos or t + 1 == T:
                v = tot / float(len(seq)) ** alpha
                if v > best[2]:
                    best = (seq, tot, v)
            else:
                rec(seq, tot)

    rec((), 0.0)
    return list(best[0]), best[1], best[2]
