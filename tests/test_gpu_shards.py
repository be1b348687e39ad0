"""Vocabulary shards through the C ABI (one device's part of a vocabulary-split
step, Section 2.2 Algorithm 6 across devices): each shard's fused projection
writes its splits into its slice of the combined partials, then one reduction
over all splits merges the beam.  Checked against the fp64 oracle of the whole
vocabulary with the rule of the single step (scores within 1e-4 / 2e-2, ranks
exact where clear, every choice legal), row log-sum-exp included.
"""
import numpy as np
import pytest
import torch

from synth import workloads as wl
from tests.gpu_util import check, say, to_dev
from tests.parity_cases import SHARDS, tile_env

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


def run_sharded(kb, inp, cuts):
    """Shards W[:, cuts[i]:cuts[i+1]] (contiguous copies, as each device would
    hold them), partials into one poisoned buffer, then the merge."""
    h, W, b, prev, off = to_dev(inp)
    shards = [(a, W[:, a:z].contiguous(), b[a:z].contiguous()) for a, z in zip(cuts, cuts[1:])]
    Ps = [kb.shard_splits(h, Wg, bg, inp.k) for _, Wg, bg in shards]
    P, N, k = sum(Ps), inp.N, inp.k
    stats = torch.full((P, N, 2), float("nan"), dtype=torch.float32, device="cuda")
    lists = torch.full((P, N, k, 2), -7, dtype=torch.int32, device="cuda")
    p0 = 0
    for (a, Wg, bg), Pg in zip(shards, Ps):
        assert kb.shard_partials(h, Wg, bg, k, a, stats[p0:p0 + Pg], lists[p0:p0 + Pg]) == Pg
        p0 += Pg
    lse = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    tok, par, sc = kb.merge_partials(stats, lists, P, inp.V, k, prev, off, row_lse=lse)
    torch.cuda.synchronize()
    return (tok.cpu().numpy(), par.cpu().numpy(), sc.cpu().numpy(), lse.cpu().numpy()), Ps




@pytest.mark.parametrize("case", range(len(SHARDS)))
def test_shards_match_the_whole_vocabulary(kb, case, monkeypatch):
    rps, H, V, k, dt, cuts, plans = SHARDS[case]
    tile_env(monkeypatch, plans)
    inp = wl.make_step(H=H, V=V, k=k, rows_per_sentence=rps, dtype=dt, seed=1700 + case, name=f"shards{case}")
    out, Ps = run_sharded(kb, inp, cuts)
    say(f"shards case {case}: N={inp.N} V={V} k={k} {dt}, {len(cuts) - 1} shards, splits {Ps}")
    rep, _ = check(inp, out)
    say(f"  max score err {rep.max_score_err:.2e}, {rep.n_checked_idx} exact ranks")


def test_v90k_over_eight_shards_sampled(kb):
    # the V=90k workload cut on multiples of 8 into 7 x 11,256 + 11,208 words
    inp = wl.make_workload(wl.V90K)
    cuts = [11256 * i for i in range(8)] + [inp.V]
    out, Ps = run_sharded(kb, inp, cuts)
    say(f"workload {inp.name} over 8 shards, splits {Ps}, oracle on sampled sentences")
    sents = sorted(set(np.random.default_rng(5).choice(inp.S, 10, replace=False).tolist()) | {0, inp.S - 1})
    rep, _ = check(inp, out, sentences=sents)
    say(f"  max score err {rep.max_score_err:.2e}, {rep.n_checked_idx} exact ranks")
