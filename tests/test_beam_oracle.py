"""Pins of the beam-search oracle with per-hypothesis end of sentence
(Section 2.1, Algorithm 2), against what fixes it independently: exhaustive
search over every sequence (a beam wide enough to keep every hypothesis
must find the best one), greedy argmax decoding at beam 1, and hand-worked
bookkeeping cases.
"""
import hashlib

import numpy as np
import pytest

from oracle import beam_oracle as bo
from oracle import kbest_oracle as ko


def _prefix_model(H, seed):
    """A decoder whose state depends on the sentence and the tokens so far."""
    def h_of(s, t, r, prefix):
        key = hashlib.sha256(repr((seed, s, tuple(int(x) for x in prefix))).encode()).digest()
        g = np.random.default_rng(np.frombuffer(key[:8], dtype=np.uint64)[0])
        return g.normal(0, 1.5, H).astype(np.float32)
    return h_of


@pytest.mark.parametrize("seed", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("alpha", [0.0, 0.7, 1.0])
def test_wide_beam_equals_exhaustive_search(seed, alpha):
    H, V, T, eos = 4, 3, 3, 0
    g = np.random.default_rng(seed)
    W = g.normal(0, 1, (H, V)).astype(np.float32)
    b = g.normal(0, 0.3, V).astype(np.float32)
    h_of = _prefix_model(H, seed)
    res = bo.beam_search(h_of, W, b, 1, 64, T, eos, alpha)     # 64 >= 3^2 hypotheses: nothing is pruned
    tok, sc, nv = bo.exhaustive_best(h_of, W, b, T, eos, alpha)
    assert res.tokens[0] == tok
    assert abs(res.score[0] - sc) < 1e-5 and abs(res.norm[0] - nv) < 1e-5


def test_beam1_without_eos_is_greedy_argmax():
    H, V, T, eos = 8, 50, 6, 7
    g = np.random.default_rng(9)
    W = g.normal(0, 1, (H, V)).astype(np.float32)
    b = g.normal(0, 0.3, V).astype(np.float32)
    b[eos] = -1e4                                    # never chosen
    h_of = _prefix_model(H, 9)
    res = bo.beam_search(h_of, W, b, 2, 1, T, eos)
    for s in range(2):
        prefix, total = (), 0.0
        for t in range(T):
            x = h_of(s, t, 0, prefix).astype(np.float64) @ W.astype(np.float64) + b
            lp = x - np.log(np.exp(x - x.max()).sum()) - x.max()
            j = int(np.argmax(x))
            prefix, total = prefix + (j,), total + lp[j]
        assert res.tokens[s] == list(prefix)
        assert abs(res.score[s] - total) < 1e-4
    assert res.steps == T


def test_finish_step_hand_worked():
    # two sentences, k = 3; sentence 0 has beam 3, sentence 1 beam 2 (its third
    # continuation is not taken); EOS = 5
    tok = np.array([[4, 5, 1], [5, 2, 9]])
    par = np.array([[0, 1, 0], [2, 2, 3]])
    sc = np.array([[-1.0, -1.5, -2.0], [-0.5, -0.7, -0.9]])
    row_hist = np.array([10, 11, 12, 13])
    fr = bo.finish_step(tok, par, sc, [3, 2], [7, 4], row_hist, t=3, T=10, eos=5, k=3, hist_base=100)
    assert fr.alive.tolist() == [1, 0, 1, 0, 1, 0]
    assert fr.beam.tolist() == [2, 1]
    assert fr.finished == [(7, -1.5, 4, 101), (4, -0.5, 4, 103)]
    assert fr.hist_token.tolist() == [4, 5, 1, 5, 2, 9]
    assert fr.hist_parent.tolist() == [10, 11, 10, 12, 12, 13]
    # the last step finishes every taken continuation, EOS or not
    fr = bo.finish_step(tok, par, sc, [3, 2], [7, 4], row_hist, t=9, T=10, eos=5, k=3, hist_base=0)
    assert fr.alive.sum() == 0 and fr.beam.tolist() == [0, 0]
    assert [f[2] for f in fr.finished] == [10] * 5


def test_backtrace_and_best_finished():
    hist_tok = [3, 4, 8, 1, 2, 6]
    hist_par = [-1, -1, 0, 2, 1, 4]
    assert bo.backtrace(hist_tok, hist_par, 3, 3) == [3, 8, 1]
    assert bo.backtrace(hist_tok, hist_par, 5, 3) == [4, 2, 6]
    fins = [(0, -3.0, 3, 3), (0, -2.0, 1, 0), (0, -3.0, 3, 5)]
    assert bo.best_finished(fins, 0.0) == 1
    assert bo.best_finished(fins, 1.0) == 0             # -1.0 per token beats -2.0; first among equals
    assert bo.best_finished([], 0.5) == -1
