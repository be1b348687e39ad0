"""The comparison rule itself: mistakes planted in oracle output must be caught.

Mistakes are planted on the CPU, in copies of the oracle's own result.
"""
import numpy as np

from oracle import compare as cmp
from oracle import kbest_oracle as ko
from synth import workloads as wl


def _case(seed=21, k=5):
    inp = wl.make_step(H=16, V=300, k=k, S=6, beam=4, seed=seed)
    res = ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, k)
    rescore = cmp.make_rescorer(inp.h, inp.W, inp.b, inp.prev, "f32", res.lse)
    return inp, res, rescore


def _run(inp, res, tok, par, sc, rescore, tol=1e-4):
    return cmp.compare_step(tok, par, sc, res, inp.off, inp.V, tol, rescore=rescore)


def test_oracle_against_itself_passes():
    inp, res, rs = _case()
    rep = _run(inp, res, res.token, res.parent, res.score, rs)
    assert rep.ok, rep.errors
    assert rep.n_checked_idx > 0


def test_swapped_clear_ranks_fail():
    inp, res, rs = _case()
    tok, par = res.token.copy(), res.parent.copy()
    tok[2, [0, 1]] = tok[2, [1, 0]]
    par[2, [0, 1]] = par[2, [1, 0]]
    assert not _run(inp, res, tok, par, res.score, rs).ok


def test_score_offset_fails():
    inp, res, rs = _case()
    sc = res.score.copy()
    sc[3] += 2e-4
    assert not _run(inp, res, res.token, res.parent, sc, rs).ok


def test_unsorted_fails():
    inp, res, rs = _case()
    sc = res.score.copy()
    sc[1, [2, 3]] = sc[1, [3, 2]]
    assert not _run(inp, res, res.token, res.parent, sc, rs).ok


def test_duplicate_pair_fails():
    inp, res, rs = _case()
    tok, par = res.token.copy(), res.parent.copy()
    tok[0, 4], par[0, 4] = tok[0, 3], par[0, 3]
    assert not _run(inp, res, tok, par, res.score, rs).ok


def test_parent_outside_sentence_fails():
    inp, res, rs = _case()
    par = res.parent.copy()
    par[1, 0] = inp.off[2]
    assert not _run(inp, res, res.token, par, res.score, rs).ok


def test_wrong_token_with_right_score_fails_rescore():
    inp, res, rs = _case()
    tok = res.token.copy()
    tok[4, 4] = (tok[4, 4] + 1) % inp.V
    assert not _run(inp, res, tok, res.parent, res.score, rs).ok


def test_near_tie_swap_is_accepted():
    # Two candidates whose scores differ by less than tol may come in either order.
    inp, res, rs = _case()
    s = 0
    res.score[s, 1] = res.score[s, 2] = 0.5 * (res.score[s, 1] + res.score[s, 2])
    tok, par = res.token.copy(), res.parent.copy()
    tok[s, [1, 2]] = tok[s, [2, 1]]
    par[s, [1, 2]] = par[s, [2, 1]]
    rep = cmp.compare_step(tok, par, res.score, res, inp.off, inp.V, 1e-4, rescore=None)
    assert rep.ok, rep.errors
