"""Mini-batching decode loop (Algorithm 2) against the naive batch (Algorithm 1)
and the oracle, step by step.

At every step of the compacted loop the same state is also decoded inside the
full constant-size batch (finished sentences' rows kept, as Algorithm 1
does); the live sentences' results must agree.  The oracle checks sampled
sentences of every step, fed the step's own inputs (teacher forcing).
"""
import numpy as np
import pytest
import torch

from oracle import compare as cmp
from oracle import kbest_oracle as ko
from synth import workloads as wl
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


def _upload(work):
    tab = work.h_table().reshape(-1, work.H)
    h_table = torch.from_numpy(tab.view(np.int16)).view(torch.bfloat16).cuda()
    W = torch.from_numpy(work.W.view(np.int16)).view(torch.bfloat16).cuda()
    b = torch.from_numpy(work.b).cuda()
    L = torch.from_numpy(work.lengths).cuda()
    p0 = torch.from_numpy(work.prev0).cuda()
    return h_table, W, b, L, p0


def _run(kb, work, sample_per_step):
    from paper_1805_09863_amd.decode import decode_loop
    h_table, W, b, L, p0 = _upload(work)
    k = work.k
    S0 = work.S
    g = np.random.default_rng(9)
    checked = {"oracle": 0, "naive": 0, "steps": 0, "padded": 0}

    def on_step(t, st):
        S, N = st["S"], st["N"]
        checked["steps"] += 1
        # launched for the previous step's counts: the sentences past this
        # step's batch came out empty
        assert st["S_launch"] >= S and st["N_launch"] >= N
        assert (st["token_launch"][S:] == -1).all()
        assert torch.isneginf(st["score_launch"][S:]).all()
        checked["padded"] += st["S_launch"] - S
        tok, par, sc = (x.cpu().numpy() for x in (st["token"], st["parent"], st["score"]))
        off = st["off"].cpu().numpy()
        sid = st["sid"].cpu().numpy()
        # (1) oracle on sampled sentences, fed this step's inputs
        h = st["h"].view(torch.int16).cpu().numpy().view(np.uint16)
        prev = st["prev"].cpu().numpy()
        # every sentence on every tenth step, a sample on the others
        n_s = S if t % 10 == 0 else min(S, sample_per_step)
        sents = sorted(set(g.choice(S, n_s, replace=False).tolist()))
        ref = ko.kbest_step_threshold(h, work.W, work.b, prev, off, k, dtype="bf16", sentences=sents)
        rs = cmp.make_rescorer(h, work.W, work.b, prev, "bf16", ref.lse)
        rep = cmp.compare_step(tok, par, sc, ref, off, work.V, 2e-2, rescore=rs, sentences=sents)
        assert rep.ok, f"step {t}: " + "; ".join(rep.errors)
        checked["oracle"] += len(sents)
        # (2) the same state inside the naive constant batch
        hn = torch.zeros((S0 * k, work.H), dtype=torch.bfloat16, device="cuda")
        pn = torch.full((S0 * k,), -3.0, dtype=torch.float32, device="cuda")
        rows = (torch.from_numpy(sid).long().cuda()[:, None] * k + torch.arange(k, device="cuda")).reshape(-1)
        hn[rows] = st["h"]
        pn[rows] = st["prev"]
        offn = (torch.arange(S0 + 1, dtype=torch.int32, device="cuda") * k)
        tn, pa, sn = kb.kbest_step(hn, W, b, pn, offn, k)
        tn, pa, sn = (x.cpu().numpy() for x in (tn, pa, sn))
        # Scores agree to float32 rounding: the batch size changes how the
        # vocabulary is split, hence the summation order of the softmax
        # statistics, by a few ulps of |score| (which grows with the step).
        for i, s0 in enumerate(sid):
            tol = 1e-6 * np.abs(sc[i]) + 1e-6
            assert np.all(np.abs(sn[s0] - sc[i]) <= tol), f"step {t} sentence {s0}: scores"
            gaps = np.abs(np.diff(sc[i]))
            for r in range(k):
                clear = (r == 0 or gaps[r - 1] > 2 * tol[r]) and (r == k - 1 or gaps[r] > 2 * tol[r])
                if clear:
                    assert tn[s0, r] == tok[i, r], f"step {t} sentence {s0} rank {r}: token"
                    assert pa[s0, r] - s0 * k == par[i, r] - off[i], f"step {t} sentence {s0} rank {r}: parent"
        checked["naive"] += S

    p0_in = p0.clone()
    stats = decode_loop(h_table, W, b, L, p0, k, work.T, compact=True, on_step=on_step)
    assert torch.equal(p0, p0_in), "the loop must not write into the caller's step-0 scores"
    want_rows = [k * int((work.lengths > t).sum()) for t in range(int(work.lengths.max()))]
    assert stats.rows == want_rows
    # step t is launched sized by step t - 1's batch; a last, empty launch
    # follows when the longest sentence ends before T
    assert stats.launch_rows[:len(want_rows)] == want_rows[:1] + want_rows[:-1]
    assert stats.launch_rows[len(want_rows):] == ([want_rows[-1]] if len(want_rows) < work.T else [])
    naive = decode_loop(h_table, W, b, L, p0, k, work.T, compact=False)
    assert torch.equal(p0, p0_in)
    assert naive.steps == stats.steps == int(work.lengths.max())
    assert naive.total_rows == stats.total_rows
    say(f"decode: {stats.steps} steps, {stats.total_rows} live rows, checked {checked}")


def test_decode_loop_small(kb):
    work = wl.make_loop_workload(S=48, V=5003, H=256, T=12, Lmin=1, Lmax=12, seed=123)
    _run(kb, work, sample_per_step=6)


def test_decode_loop_config4(kb):
    work = wl.make_loop_workload()
    say(f"decode-loop workload: S={work.S} V={work.V} H={work.H} T={work.T}")
    _run(kb, work, sample_per_step=32)


def test_decode_loop_on_its_own_stream(kb):
    # the loop's kernels, count read-back and events all follow the stream it
    # is given, while torch's current stream stays the default one
    from paper_1805_09863_amd.decode import decode_loop
    work = wl.make_loop_workload(S=40, V=3001, H=128, T=10, Lmin=1, Lmax=10, seed=77)
    h_table, W, b, L, p0 = _upload(work)
    want = [work.k * int((work.lengths > t).sum()) for t in range(int(work.lengths.max()))]
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    for compact in (True, False):
        got = []

        def on_step(t, st):
            with torch.cuda.stream(s):
                got.append((st["token"].clone(), st["score"].clone()))
        stats = decode_loop(h_table, W, b, L, p0, work.k, work.T, compact=compact, on_step=on_step, stream=s)
        s.synchronize()
        assert stats.rows == want
        ref = []
        decode_loop(h_table, W, b, L, p0, work.k, work.T, compact=compact,
                    on_step=lambda t, st: ref.append((st["token"].clone(), st["score"].clone())))
        torch.cuda.synchronize()
        assert len(got) == len(ref)
        for (ta, sa), (tb, sb) in zip(got, ref):
            assert torch.equal(ta.cpu(), tb.cpu()) and torch.equal(sa.cpu(), sb.cpu())
    say(f"decode loop on a side stream: {len(want)} steps, rows {want[:4]}...")
