"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Each test ties one part of the oracle to a closed form, an invariant the
paper states, a special case that reduces to a library routine, or brute
force on tiny inputs, so that a dropped term, a wrong sign or index, or a
transposed operand in the oracle fails at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import kbest_oracle as ko
from synth import workloads as wl

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ---------------------------------------------------------------- softmax
def test_softmax_sums_to_one():
    g = np.random.default_rng(1)
    x = g.normal(0, 3, size=(50, 777))
    p, _, _ = ko.softmax_three_pass(x)
    assert np.all(np.abs(p.sum(axis=1) - 1.0) < 1e-12)
    assert np.all(p > 0)


def test_softmax_closed_form_rational():
    # exp(ln j) = j, so p_j = j / 10 exactly and LSE = ln 10.
    x = np.log(np.array([[1.0, 2.0, 3.0, 4.0]]))
    p, _, _ = ko.softmax_three_pass(x)
    assert np.allclose(p[0], [0.1, 0.2, 0.3, 0.4], rtol=0, atol=1e-15)
    logp, lse = ko.log_softmax(x)
    assert abs(lse[0] - math.log(10.0)) < 1e-15
    assert np.allclose(logp[0], np.log([0.1, 0.2, 0.3, 0.4]), rtol=0, atol=1e-15)


def test_all_equal_row():
    V = 1234
    x = np.full((1, V), 0.75)
    p, _, _ = ko.softmax_three_pass(x)
    assert np.allclose(p, 1.0 / V, rtol=1e-14, atol=0)
    _, lse = ko.log_softmax(x)
    assert abs(lse[0] - (0.75 + math.log(V))) < 1e-13


def test_single_dominant_logit():
    x = np.zeros((1, 100))
    x[0, 37] = 1000.0
    p, _, _ = ko.softmax_three_pass(x)
    assert p[0, 37] == 1.0
    assert np.all(p[0, np.arange(100) != 37] < 1e-300)


def test_shift_invariance():
    g = np.random.default_rng(2)
    x = g.normal(size=(7, 300))
    c = 12.375
    lp1, lse1 = ko.log_softmax(x)
    lp2, lse2 = ko.log_softmax(x + c)
    assert np.allclose(lp1, lp2, rtol=0, atol=1e-12)
    assert np.allclose(lse2 - lse1, c, rtol=0, atol=1e-12)


def test_shift_of_bias_keeps_selection():
    inp = wl.make_step(H=8, V=200, k=4, S=3, beam=2, seed=5)
    b = _dyadic(np.random.default_rng(5), (200,), -1, 1)   # b + 3 stays exact in float32
    r1 = ko.kbest_step(inp.h, inp.W, b, inp.prev, inp.off, inp.k)
    r2 = ko.kbest_step(inp.h, inp.W, b + np.float32(3.0), inp.prev, inp.off, inp.k)
    assert np.array_equal(r1.token, r2.token) and np.array_equal(r1.parent, r2.parent)
    assert np.allclose(r1.score, r2.score, rtol=0, atol=1e-9)
    assert np.allclose(r2.lse - r1.lse, 3.0, rtol=0, atol=1e-9)


def test_topk_of_logits_equals_topk_of_softmax():
    # Section 2.2: softmax and exp are monotonic, so the best classes can be
    # found before normalising.
    g = np.random.default_rng(3)
    x = g.normal(size=(20, 5000))
    p, _, _ = ko.softmax_three_pass(x)
    logp, _ = ko.log_softmax(x)
    for r in range(x.shape[0]):
        a = np.argsort(-x[r], kind="stable")[:12]
        assert np.array_equal(a, np.argsort(-p[r], kind="stable")[:12])
        assert np.array_equal(a, np.argsort(-logp[r], kind="stable")[:12])


# ---------------------------------------------------------------- brute force
def _brute(h, W, b, prev, off, k):
    """Enumerate every (row, word) candidate with Python floats and math.fsum."""
    N, H = len(h), len(h[0])
    V = len(W[0])
    x = [[math.fsum(h[n][i] * W[i][j] for i in range(H)) + b[j] for j in range(V)] for n in range(N)]
    lse = []
    for n in range(N):
        m = max(x[n])
        lse.append(m + math.log(math.fsum(math.exp(v - m) for v in x[n])))
    out = []
    for s in range(len(off) - 1):
        cands = []
        for r in range(off[s], off[s + 1]):
            for j in range(V):
                flat = (r - off[s]) * V + j
                cands.append((-(prev[r] + x[r][j] - lse[r]), flat, r, j))
        cands.sort()
        out.append(cands)
    return out, lse


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_brute_force_tiny(dtype):
    g = np.random.default_rng(11)
    for trial in range(60):
        rps = [int(g.integers(1, 4)) for _ in range(2)]
        H = int(g.integers(1, 5))
        V = int(g.integers(2, 14))
        k = int(g.integers(1, min(5, min(rps) * V) + 1))
        inp = wl.make_step(H=H, V=V, k=k, rows_per_sentence=rps, dtype=dtype, seed=1000 + trial)
        res = ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, k, dtype=dtype)
        h = ko.widen(inp.h, dtype).tolist()
        W = ko.widen(inp.W, dtype).tolist()
        b = inp.b.astype(np.float64).tolist()
        prev = inp.prev.astype(np.float64).tolist()
        brute, lse = _brute(h, W, b, prev, inp.off.tolist(), k)
        assert np.allclose(res.lse, lse, rtol=0, atol=1e-12)
        for s in range(2):
            for r in range(k):
                negsc, _, row, j = brute[s][r]
                assert res.token[s, r] == j and res.parent[s, r] == row
                assert abs(res.score[s, r] + negsc) < 1e-12
            if len(brute[s]) > k:
                assert abs(res.next_score[s] + brute[s][k][0]) < 1e-12


def test_worked_example_golden(repo_root):
    with open(os.path.join(repo_root, "tests", "golden", "worked_example.json")) as f:
        ex = json.load(f)
    env = {"log": math.log, "e": math.e}
    h = np.array(ex["h"], dtype=np.float32)
    W = np.array(ex["W"], dtype=np.float32)
    b = np.array(ex["b"], dtype=np.float32)
    prev = np.array(ex["prev"], dtype=np.float32)
    res = ko.kbest_step(h, W, b, prev, np.array(ex["off"]), ex["k"])
    assert res.token.tolist() == ex["token"]
    assert res.parent.tolist() == ex["parent"]
    want = np.array([[eval(e, env) for e in row] for row in ex["score"]])  # noqa: S307
    assert np.allclose(res.score, want, rtol=0, atol=1e-14)
    assert np.allclose(res.next_score, [eval(e, env) for e in ex["next_score"]], rtol=0, atol=1e-14)  # noqa: S307
    assert np.allclose(res.lse, [eval(e, env) for e in ex["row_lse"]], rtol=0, atol=1e-14)  # noqa: S307


# ---------------------------------------------------------------- tie breaking
def _dyadic(g, shape, lo=-4, hi=4):
    """Small multiples of 1/8: every product and sum below is exact in fp64."""
    return (g.integers(lo * 8, hi * 8 + 1, size=shape) / 8.0).astype(np.float32)


def test_duplicate_rows_prefer_lower_parent():
    g = np.random.default_rng(4)
    H, V, k = 3, 9, 6
    h = _dyadic(g, (4, H))
    h[2] = h[1]                       # rows 1 and 2 of sentence 0 are identical
    W = _dyadic(g, (H, V))
    b = _dyadic(g, (V,), -1, 1)
    prev = np.array([-1.0, -0.5, -0.5, -2.0], dtype=np.float32)
    off = np.array([0, 3, 4])
    res = ko.kbest_step(h, W, b, prev, off, k)
    # every candidate of row 2 ties one of row 1; row 1's copy must come first
    seen = {}
    for r in range(k):
        p, t = int(res.parent[0, r]), int(res.token[0, r])
        if p == 2:
            assert (1, t) in seen, "a row-2 tie appeared before its row-1 twin"
        seen[(p, t)] = r
    assert any(p == 2 for p, _ in seen), "the tie case was not exercised"


def test_duplicate_columns_prefer_lower_token():
    g = np.random.default_rng(5)
    H, V, k = 4, 12, 5
    h = _dyadic(g, (2, H))
    W = _dyadic(g, (H, V))
    b = _dyadic(g, (V,), -1, 1)
    x = h.astype(np.float64) @ W.astype(np.float64) + b
    j_best = int(np.argmax(x[0]))
    twin = V - 1 if j_best != V - 1 else 0
    W[:, twin] = W[:, j_best]
    b[twin] = b[j_best]
    res = ko.kbest_step(h, W, b, np.zeros(2, np.float32), np.array([0, 1, 2]), k)
    lo, hi = min(j_best, twin), max(j_best, twin)
    assert res.token[0, 0] == lo and res.token[0, 1] == hi
    assert res.score[0, 0] == res.score[0, 1]


def test_beam1_k1_is_numpy_argmax():
    # Algorithm 5 special case: one row per sentence, k = 1 -> first argmax.
    inp = wl.make_step(H=16, V=500, k=1, S=6, beam=1, seed=9)
    res = ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, 1)
    x = inp.h.astype(np.float64) @ inp.W.astype(np.float64) + inp.b
    assert np.array_equal(res.token[:, 0], np.argmax(x, axis=1))
    assert np.array_equal(res.parent[:, 0], np.arange(6))
    m = x.max(axis=1)
    lse = np.array([math.log(math.fsum(np.exp(r - r.max()))) for r in x]) + m
    assert np.allclose(res.score[:, 0], inp.prev + m - lse, rtol=0, atol=1e-12)


# ------------------------------------------------- Algorithms 4, 5, 6 (loops)
@pytest.mark.parametrize("kind", ["random", "increasing", "decreasing", "constant", "ties"])
def test_fused_alg4_matches_three_pass(kind):
    g = np.random.default_rng(6)
    n = 400
    if kind == "random":
        p = g.normal(0, 2, n)
    elif kind == "increasing":
        p = np.linspace(-3, 5, n)            # the max changes at every element
    elif kind == "decreasing":
        p = np.linspace(5, -3, n)
    elif kind == "constant":
        p = np.full(n, 0.3)
    else:
        p = np.round(g.normal(0, 1, n) * 2) / 2
    b = g.uniform(-0.1, 0.1, n) if kind != "constant" else np.zeros(n)
    inv, best, mx, s = ko.fused_softmax_best(p, b)
    q = (p + b)[None, :]
    pr, m3, s3 = ko.softmax_three_pass(q)
    assert best == int(np.argmax(q[0]))
    assert mx == m3[0]
    assert abs(s - s3[0]) <= 1e-12 * s3[0]
    assert abs(inv - pr[0, best]) <= 1e-12


def test_alg4_printed_update_disagrees():
    # Reading of Algorithm 4: the printed 'delta x sum' cannot be meant; the
    # derivation rescales by e^delta.  The literal form is NaN from the start.
    p = np.array([0.0, 1.0, 2.0, 0.5])
    b = np.zeros(4)
    lit = ko.fused_softmax_best_literal(p, b)
    assert math.isnan(lit[3])
    cor = ko.fused_softmax_best(p, b)
    assert abs(cor[3] - sum(math.exp(v - 2.0) for v in p)) < 1e-15


def test_argmax_only_and_sharded():
    g = np.random.default_rng(7)
    for trial in range(30):
        n = int(g.integers(1, 60))
        p = np.round(g.normal(0, 1, n) * 2) / 2    # many exact ties
        b = np.zeros(n)
        want = int(np.argmax(p))                   # numpy: first occurrence
        assert ko.argmax_only(p, b) == want
        assert ko.find_best(p)[1] == want
        for shards in range(1, n + 1):
            assert ko.argmax_sharded(p, b, shards) == want


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_argmax_rows_is_alg5_per_row(dtype):
    # The vectorised greedy oracle against the Algorithm 5 loop (strict '>')
    # and the Algorithm 6 sharded reduction, row by row, on the exact widened
    # scores; duplicated columns force exact ties, which the lower word wins.
    inp = wl.make_step(H=24, V=300, k=1, S=20, beam=1, dtype=dtype, seed=31)
    W = inp.W.copy()
    W[:, 150:180] = W[:, 10:40]                 # twins of 30 columns (b differs: copy it too)
    b = inp.b.copy()
    b[150:180] = b[10:40]
    res = ko.argmax_rows(inp.h, W, b, dtype)
    x = ko.widen(inp.h, dtype) @ ko.widen(W, dtype) + b.astype(np.float64)[None, :]
    for n in range(inp.N):
        want = ko.argmax_only(x[n], np.zeros(inp.V))
        assert res.token[n] == want
        assert ko.argmax_sharded(x[n], np.zeros(inp.V), 7) == want
        assert res.value[n] == x[n, want]
        assert res.second[n] == np.max(np.delete(x[n], want))
        assert want < 150 or want >= 180          # a twin never beats its original


def test_argmax_rows_brute_force_and_subset():
    # Tiny inputs in plain Python floats (math.fsum dot products); a subset of
    # rows gives the same answers as the full call.
    g = np.random.default_rng(12)
    h = np.round(g.normal(0, 1, (7, 3)) * 4) / 4
    W = np.round(g.normal(0, 1, (3, 11)) * 4) / 4
    b = np.round(g.normal(0, 1, 11) * 4) / 4
    res = ko.argmax_rows(h.astype(np.float32), W.astype(np.float32), b.astype(np.float32))
    for n in range(7):
        sc = [math.fsum([float(h[n, i]) * float(W[i, j]) for i in range(3)] + [float(b[j])]) for j in range(11)]
        best = max(range(11), key=lambda j: (sc[j], -j))
        assert res.token[n] == best and res.value[n] == sc[best]
    sub = ko.argmax_rows(h.astype(np.float32), W.astype(np.float32), b.astype(np.float32), rows=[5, 1])
    assert list(sub.token) == [res.token[5], res.token[1]]


def test_merge_softmax_stats_any_sharding():
    g = np.random.default_rng(8)
    x = g.normal(0, 3, 3000)
    _, m_all, s_all = ko.softmax_three_pass(x[None, :])
    for trial in range(20):
        cuts = np.sort(g.choice(np.arange(1, x.size), size=int(g.integers(1, 40)), replace=False))
        parts = []
        for a, c in zip(np.concatenate([[0], cuts]), np.concatenate([cuts, [x.size]])):
            _, m, s = ko.softmax_three_pass(x[None, a:c])
            parts.append((m[0], s[0]))
        g.shuffle(parts)
        M, S = ko.merge_softmax_stats(parts)
        assert M == m_all[0]
        assert abs(S - s_all[0]) <= 1e-12 * s_all[0]


# ---------------------------------------------- exact shortcut and the lemma
def test_threshold_shortcut_equals_full_sort_random_and_ties():
    g = np.random.default_rng(12)
    for trial in range(25):
        rps = [int(r) for r in g.integers(1, 6, size=int(g.integers(1, 6)))]
        H, V = int(g.integers(1, 6)), int(g.integers(2, 40))
        k = int(g.integers(1, min(8, min(rps) * V) + 1))
        N = sum(rps)
        h = _dyadic(g, (N, H), -2, 2)
        W = _dyadic(g, (H, V), -2, 2)
        b = _dyadic(g, (V,), -1, 1)
        prev = _dyadic(g, (N,), -2, 0)
        off = np.concatenate([[0], np.cumsum(rps)])
        a = ko.kbest_step(h, W, b, prev, off, k)
        c = ko.kbest_step_threshold(h, W, b, prev, off, k)
        assert np.array_equal(a.token, c.token) and np.array_equal(a.parent, c.parent)
        assert np.array_equal(a.score, c.score) and np.array_equal(a.next_score, c.next_score)


@pytest.mark.parametrize("name", [wl.SMALL, wl.NEARTIE])
def test_threshold_shortcut_equals_full_sort_configs(name):
    inp = wl.make_workload(name)
    if name == wl.NEARTIE:        # a sample of sentences keeps the CPU suite short
        inp = _slice_sentences(inp, range(0, 64, 8))
    a = ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, inp.k, inp.dtype)
    c = ko.kbest_step_threshold(inp.h, inp.W, inp.b, inp.prev, inp.off, inp.k, inp.dtype)
    assert np.array_equal(a.token, c.token) and np.array_equal(a.parent, c.parent)
    assert np.array_equal(a.score, c.score) and np.array_equal(a.next_score, c.next_score)


def _slice_sentences(inp, sents):
    sents = list(sents)
    rows = np.concatenate([np.arange(inp.off[s], inp.off[s + 1]) for s in sents])
    rps = [int(inp.off[s + 1] - inp.off[s]) for s in sents]
    off = np.concatenate([[0], np.cumsum(rps)]).astype(np.int32)
    return wl.StepInputs(inp.dtype, inp.h[rows], inp.W, inp.b, inp.prev[rows], off, inp.k,
                         name=inp.name, seed=inp.seed)


def test_sentence_topk_within_union_of_row_topk():
    # Score = x + (prev - LSE) adds a row constant, so each sentence's k best
    # lie inside the union of its rows' k best logits.
    g = np.random.default_rng(13)
    for trial in range(20):
        inp = wl.make_step(H=6, V=80, k=int(g.integers(1, 9)),
                           rows_per_sentence=list(g.integers(1, 7, size=4)), seed=300 + trial)
        res = ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, inp.k)
        x = inp.h.astype(np.float64) @ inp.W.astype(np.float64) + inp.b
        for s in range(inp.S):
            union = set()
            for r in range(inp.off[s], inp.off[s + 1]):
                for j in np.argsort(-x[r], kind="stable")[:inp.k]:
                    union.add((r, int(j)))
            for r in range(inp.k):
                assert (int(res.parent[s, r]), int(res.token[s, r])) in union


# ---------------------------------------------------------------- compaction
def _compact_loop(alive, S, k):
    keep, off, ks = [], [0], []
    for s in range(S):
        c = 0
        for j in range(k):
            if alive[s * k + j]:
                keep.append(s * k + j)
                c += 1
        if c:
            ks.append(s)
            off.append(off[-1] + c)
    return keep, off, ks


@pytest.mark.parametrize("pattern", ["random", "all", "none", "alternating", "single", "sentences"])
def test_compact_matches_loop(pattern):
    g = np.random.default_rng(14)
    S, k = 37, 5
    M = S * k
    if pattern == "random":
        a = g.random(M) < 0.5
    elif pattern == "all":
        a = np.ones(M, bool)
    elif pattern == "none":
        a = np.zeros(M, bool)
    elif pattern == "alternating":
        a = (np.arange(M) % 2) == 0
    elif pattern == "single":
        a = np.zeros(M, bool)
        a[101] = True
    else:
        a = np.repeat(g.random(S) < 0.6, k)
    res = ko.compact(a.astype(np.uint8), S, k)
    keep, off, ks = _compact_loop(a.tolist(), S, k)
    assert res.keep_idx.tolist() == keep
    assert res.kept_count == len(keep)
    assert res.new_offsets.tolist() == off
    assert res.kept_sentence.tolist() == ks
    assert res.new_S == len(ks)


def test_exhaustive_compaction_small():
    for S, k in [(1, 1), (2, 2), (3, 2), (1, 4)]:
        for bits in itertools.product([0, 1], repeat=S * k):
            res = ko.compact(np.array(bits, np.uint8), S, k)
            keep, off, ks = _compact_loop(list(bits), S, k)
            assert res.keep_idx.tolist() == keep and res.new_offsets.tolist() == off
            assert res.kept_sentence.tolist() == ks


def _compact_entries_loop(alive, es):
    # the batch walked entry by entry: a sentence opens when its first
    # surviving entry is met
    keep, off, ks = [], [], []
    for i, a in enumerate(alive):
        if a:
            if not ks or ks[-1] != es[i]:
                ks.append(es[i])
                off.append(len(keep))
            keep.append(i)
    off.append(len(keep))
    return keep, off, ks


@pytest.mark.parametrize("seed", range(6))
def test_compact_entries_matches_loop(seed):
    g = np.random.default_rng(300 + seed)
    sizes = g.integers(0, 7, g.integers(1, 40))          # empty sentences included
    es = np.repeat(np.arange(sizes.size), sizes)
    a = (g.random(es.size) < [0.0, 0.3, 0.5, 0.9, 1.0, 0.5][seed]).astype(np.uint8)
    res = ko.compact_entries(a, es)
    keep, off, ks = _compact_entries_loop(a.tolist(), es.tolist())
    assert res.keep_idx.tolist() == keep and res.kept_count == len(keep)
    assert res.new_offsets.tolist() == off and res.kept_sentence.tolist() == ks and res.new_S == len(ks)
    bare = ko.compact_entries(a)
    assert bare.keep_idx.tolist() == keep and bare.kept_count == len(keep)


def test_compact_entries_exhaustive_small():
    for es in ([0, 0, 1], [0, 1, 1, 3], [2, 2, 2], [0, 1, 2, 3]):
        for bits in itertools.product([0, 1], repeat=len(es)):
            res = ko.compact_entries(np.array(bits, np.uint8), np.array(es))
            keep, off, ks = _compact_entries_loop(list(bits), es)
            assert res.keep_idx.tolist() == keep and res.new_offsets.tolist() == off
            assert res.kept_sentence.tolist() == ks
