"""Comparison rule between a device result and the fp64 oracle.

TEST INFRASTRUCTURE ONLY (imported by the tests, the smoke check and the
benchmark's CPU baseline).

For each sentence, with oracle scores ``o_0 >= ... >= o_k`` (``o_k`` is the
(k+1)-th candidate) and device results ``g_0 .. g_{k-1}``:

(i)   the device list is sorted by descending score and
      ``|g_r.score - o_r| <= tol`` at every rank;
(ii)  where the ranking is clear -- (r == 0 or o_{r-1} - o_r > tol) and
      o_r - o_{r+1} > tol -- token and parent equal the oracle's at rank r;
(iii) every device choice is legal: (parent, token) pairs are unique, the
      parent lies in the sentence's rows, the token in [0, V), and the
      oracle's fp64 re-score of that pair is within tol of the device score.

Near-ties inside the tolerance have several correct orderings; rule (iii)
checks that the device picked one of them.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class Report:
    ok: bool = True
    max_score_err: float = 0.0
    max_rescore_err: float = 0.0
    n_checked_idx: int = 0
    errors: list = field(default_factory=list)

    def fail(self, msg: str):
        self.ok = False
        if len(self.errors) < 20:
            self.errors.append(msg)


def compare_step(dev_token, dev_parent, dev_score, oracle, off, V: int, tol: float,
                 rescore=None, sentences=None) -> Report:
    """Apply rules (i)-(iii).

    ``oracle`` is a ``KBestResult`` (rows aligned with ``sentences`` if
    given).  ``rescore(parent, token) -> float64`` gives the oracle's exact
    score of one candidate; if omitted, rule (iii)'s re-score is skipped.
    """
    rep = Report()
    dev_token = np.asarray(dev_token)
    dev_parent = np.asarray(dev_parent)
    dev_score = np.asarray(dev_score, dtype=np.float64)
    off = np.asarray(off, dtype=np.int64)
    sel = range(dev_token.shape[0]) if sentences is None else sentences
    for i, s in enumerate(sel):
        oi = i if sentences is not None else s
        o = oracle.score[oi]
        k = o.shape[0]
        on = np.append(o, oracle.next_score[oi])
        g = dev_score[s]
        # (i) sorted and scored
        if np.any(np.diff(g) > 0):
            rep.fail(f"sentence {s}: device scores not sorted: {g}")
        err = np.abs(g - o)
        rep.max_score_err = max(rep.max_score_err, float(err.max()))
        if np.any(err > tol):
            r = int(np.argmax(err))
            rep.fail(f"sentence {s} rank {r}: score {g[r]!r} vs oracle {o[r]!r} (tol {tol})")
        # (ii) indices where the ranking is clear
        for r in range(k):
            clear_above = (r == 0) or (on[r - 1] - on[r] > tol)
            clear_below = on[r] - on[r + 1] > tol
            if clear_above and clear_below:
                rep.n_checked_idx += 1
                if dev_token[s, r] != oracle.token[oi, r] or dev_parent[s, r] != oracle.parent[oi, r]:
                    rep.fail(f"sentence {s} rank {r}: (parent, token) = "
                             f"({dev_parent[s, r]}, {dev_token[s, r]}) vs oracle "
                             f"({oracle.parent[oi, r]}, {oracle.token[oi, r]})")
        # (iii) legality
        pairs = set()
        for r in range(k):
            p, t = int(dev_parent[s, r]), int(dev_token[s, r])
            if not (off[s] <= p < off[s + 1]) or not (0 <= t < V):
                rep.fail(f"sentence {s} rank {r}: illegal (parent, token) = ({p}, {t})")
                continue
            if (p, t) in pairs:
                rep.fail(f"sentence {s} rank {r}: duplicate (parent, token) = ({p}, {t})")
            pairs.add((p, t))
            if rescore is not None:
                e = abs(rescore(p, t) - g[r])
                rep.max_rescore_err = max(rep.max_rescore_err, e)
                if e > tol:
                    rep.fail(f"sentence {s} rank {r}: re-score error {e} > {tol}")
    return rep


def make_rescorer(h, W, b, prev, dtype: str, lse):
    """fp64 score of a single (parent row, token) pair, from the oracle's LSE."""
    from .kbest_oracle import widen

    b64 = np.asarray(b, dtype=np.float32).astype(np.float64)
    prev64 = np.asarray(prev, dtype=np.float32).astype(np.float64)

    def rescore(p: int, t: int) -> float:
        x = float(widen(h[p], dtype) @ widen(W[:, t], dtype)) + b64[t]
        return prev64[p] + x - float(lse[p])

    return rescore
