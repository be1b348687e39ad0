"""Beam search with per-hypothesis end of sentence (Section 2.1, Algorithm 2)
on the GPU, step by step against the oracle (teacher forcing: each step's
oracle is fed the device state of that step):

* the output layer's k-best, with the comparison rules of the fused step;
* kb_beam_finish: the alive mask, the shrunk beams, the step's history and
  every entry of the finished store, bit for bit;
* kb_beam_backtrace: each sentence's chosen hypothesis (by score /
  length**alpha) and its tokens read back through the device history.
"""
import numpy as np
import pytest
import torch

from oracle import beam_oracle as bo
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


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def _run(work, alpha, sample):
    from paper_1805_09863_amd.decode import beam_search
    k, T, eos, S0 = work.k, work.T, work.eos, work.S
    tab = work.h_table().reshape(-1, work.H)
    h_table, W, b = _bf16(tab), _bf16(work.W), torch.from_numpy(work.b).cuda()
    g = np.random.default_rng(17)
    mirror = {o: [] for o in range(S0)}
    seen = {"steps": 0, "finished": 0}

    def on_step(t, st):
        S, N = st["S"], st["N"]
        seen["steps"] += 1
        tok, par, sc = (x.cpu().numpy() for x in (st["token"], st["parent"], st["score"]))
        h = st["h"].view(torch.int16).cpu().numpy().view(np.uint16)
        prev, off, sid = (st[x].cpu().numpy() for x in ("prev", "off", "sid"))
        # (1) the output layer on sampled sentences
        sents = sorted(set(g.choice(S, min(S, sample), replace=False).tolist()))
        ref = ko.kbest_step_threshold(h, work.W, work.b, prev, off, k, dtype="bf16", sentences=sents)
        rs = cmp.make_rescorer(h, work.W, work.b, prev, "bf16", ref.lse)
        rep = cmp.compare_step(tok, par, sc, ref, off, work.V, 2e-2, rescore=rs, sentences=sents)
        assert rep.ok, f"step {t}: " + "; ".join(rep.errors)
        # (2) the end-of-sentence bookkeeping, exactly
        row_hist = (np.full(N, -1) if st["prev_keep"] is None
                    else st["prev_base"] + st["prev_keep"].cpu().numpy().astype(np.int64))
        fr = bo.finish_step(tok, par, sc, st["beam_before"].cpu().numpy(), sid, row_hist, t, T, eos, k, st["base"])
        assert np.array_equal(st["alive"].cpu().numpy(), fr.alive), f"step {t}: alive"
        assert np.array_equal(st["beam_after"].cpu().numpy(), fr.beam), f"step {t}: beams"
        base = st["base"]
        ht = st["hist_token"][base:base + S * k].cpu().numpy()
        hp = st["hist_parent"][base:base + S * k].cpu().numpy()
        assert np.array_equal(ht, fr.hist_token) and np.array_equal(hp, fr.hist_parent), f"step {t}: history"
        for f in fr.finished:
            mirror[f[0]].append(f)
        seen["finished"] += len(fr.finished)
        fc, fs, fl, fh = (x.cpu().numpy() for x in st["fin"])
        for o in range(S0):
            assert fc[o] == len(mirror[o]), f"step {t}: finished count of sentence {o}"
            for i, f in enumerate(mirror[o]):
                assert np.float32(fs[o * k + i]) == np.float32(f[1]), f"step {t}: finished score"
                assert fl[o * k + i] == f[2] and fh[o * k + i] == f[3], f"step {t}: finished entry"

    res = beam_search(h_table, W, b, k, T, eos, alpha=alpha, on_step=on_step)
    torch.cuda.synchronize()
    # (3) the translations: best finished hypothesis and its tokens
    toks, ln, sc, nm = (x.cpu().numpy() for x in (res.tokens, res.length, res.score, res.norm))
    ht, hp = (x.cpu().numpy() for x in res.hist)
    for o in range(S0):
        fins = mirror[o]
        assert fins, f"sentence {o} never finished"
        vals = [np.float32(f[1]) / np.float32(f[2]) ** np.float32(alpha) for f in fins]
        i = bo.best_finished(fins, alpha)
        best = max(vals)
        j = next(m for m, f in enumerate(fins) if f[2] == ln[o] and np.float32(f[1]) == sc[o]
                 and abs(vals[m] - nm[o]) <= 1e-6 * max(1.0, abs(nm[o])))
        assert vals[j] >= best - 1e-5 * max(1.0, abs(best)), f"sentence {o}: not the best finished"
        if all(abs(v - vals[i]) > 1e-4 for m, v in enumerate(vals) if m != i):
            assert j == i, f"sentence {o}: chose {j}, the oracle {i}"
        want = bo.backtrace(ht, hp, fins[j][3], fins[j][2])
        assert list(toks[o, :ln[o]]) == want and np.all(toks[o, ln[o]:] == -1), f"sentence {o}: tokens"
        assert want[-1] == eos or ln[o] == T
    say(f"beam search: {res.steps} steps, {seen['finished']} finished hypotheses, checked {seen['steps']} steps")
    return res


@pytest.mark.parametrize("alpha", [0.0, 1.0])
def test_beam_search_small(kb, alpha):
    work = wl.make_eos_workload(S=24, k=4, H=128, V=500, T=14, Lmin=2, Lmax=9, seed=601)
    res = _run(work, alpha, sample=8)
    assert res.steps < work.T            # every sentence ended on EOS before the cap


def test_beam_search_cap_and_beam1(kb):
    # beam 1 and a cap shorter than some sentences: the last step finishes the rest
    work = wl.make_eos_workload(S=30, k=1, H=128, V=800, T=6, Lmin=2, Lmax=12, seed=602)
    res = _run(work, 0.5, sample=10)
    assert res.steps == work.T


def test_beam_search_larger(kb):
    work = wl.make_eos_workload(S=64, k=5, H=256, V=5000, T=20, Lmin=3, Lmax=14, seed=603)
    _run(work, 1.0, sample=4)
