"""GPU parity of the few-row projection (at most 8 live rows, 16-byte operands)
against the fp64 oracle, through the C ABI.

These steps stream W once through vector FMAs (float32) or two-state bf16 dot
products, fold every chunk of words into the row's statistics and k best, and
hand the same partials to the merge kernel as the matrix-core paths.
"""
import dataclasses

import numpy as np
import pytest
import torch

from synth import workloads as wl
from tests.gpu_util import check, run_step, say, to_dev
from tests.parity_cases import FEW

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb




@pytest.mark.parametrize("case", range(len(FEW)))
def test_few_rows(kb, case):
    rps, H, V, k, dt, _plan = FEW[case]
    inp = wl.make_step(H=H, V=V, k=k, rows_per_sentence=rps, dtype=dt, seed=1700 + case, name=f"few{case}")
    say(f"few-row case {case}: N={inp.N} H={H} V={V} k={k} {dt}")
    out = run_step(kb, inp, row_lse=True)
    rep, _ = check(inp, out)
    say(f"  max score err {rep.max_score_err:.2e}, {rep.n_checked_idx} exact ranks")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_few_rows_twin_columns_and_rows(kb, dt):
    # Every row's best column duplicated (bitwise-equal logits: the lower word
    # first), and rows 1 and 2 of each sentence identical (the lower parent first).
    inp = wl.make_step(H=64, V=6000, k=6, S=2, beam=3, dtype=dt, seed=1790, name=f"few_twins_{dt}")
    from oracle import kbest_oracle as ko
    x = ko.widen(inp.h, dt) @ ko.widen(inp.W, dt) + inp.b
    W, b, h, prev = inp.W.copy(), inp.b.copy(), inp.h.copy(), inp.prev.copy()
    for r in range(inp.N):
        j = int(np.argmax(x[r]))
        t = (j + 3001) % inp.V
        W[:, t] = W[:, j]
        b[t] = b[j]
    for s in range(inp.S):
        h[inp.off[s] + 2] = h[inp.off[s] + 1]
        prev[inp.off[s] + 2] = prev[inp.off[s] + 1]
    inp = dataclasses.replace(inp, W=W, b=b, h=h, prev=prev)
    tok, par, sc = run_step(kb, inp)
    check(inp, (tok, par, sc))
    for s in range(inp.S):
        row = [(int(par[s, i]) - int(inp.off[s]), int(tok[s, i]), float(sc[s, i])) for i in range(inp.k)]
        for i in range(1, len(row)):
            assert row[i - 1][2] >= row[i][2]
            if row[i - 1][2] == row[i][2]:     # equal scores: lower flat index first
                assert (row[i - 1][0], row[i - 1][1]) < (row[i][0], row[i][1]), f"sentence {s}: {row}"


def test_few_rows_deterministic_with_poisoned_buffers(kb):
    inp = wl.make_step(H=1024, V=12000, k=5, S=1, beam=5, dtype="bf16", seed=1795, name="few_det")
    h, W, b, prev, off = to_dev(inp)
    res = []
    for ws_byte, fill in ((0xFF, float("nan")), (0x7F, float("-inf"))):
        need = kb.kbest_workspace_bytes(kb.KB_BF16, inp.N, inp.H, inp.V, inp.k, inp.S)
        ws = torch.full((need,), ws_byte, dtype=torch.uint8, device="cuda")
        tok = torch.full((1, inp.k), -7, dtype=torch.int32, device="cuda")
        par = torch.full((1, inp.k), -7, dtype=torch.int32, device="cuda")
        sc = torch.full((1, inp.k), fill, dtype=torch.float32, device="cuda")
        lse = torch.full((inp.N,), fill, dtype=torch.float32, device="cuda")
        kb.kbest_step(h, W, b, prev, off, inp.k, out=(tok, par, sc), ws=ws, row_lse=lse)
        torch.cuda.synchronize()
        res.append([x.cpu().numpy() for x in (tok, par, sc, lse)])
    for x, y in zip(*res):
        assert np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                              y.view(np.uint32) if y.dtype == np.float32 else y)
    check(inp, tuple(res[0]))


def test_few_rows_past_the_batch(kb):
    # launched for more sentences and rows than the batch holds (the decode
    # loop's lagged sizing): empty sentences and rows past off[S]
    inp = wl.make_step(H=256, V=9000, k=4, rows_per_sentence=[2, 3], dtype="bf16", seed=1797, name="few_holes")
    h, W, b, prev, _ = to_dev(inp)
    extra = 3
    h = torch.cat([h, torch.randn((extra, inp.H), device="cuda").to(h.dtype) * 4]).contiguous()
    prev = torch.cat([prev, torch.zeros(extra, device="cuda")]).contiguous()
    layout = [2, 0, 3, 0]
    off = torch.tensor(np.concatenate([[0], np.cumsum(layout)]).astype(np.int32), device="cuda")
    tok, par, sc = kb.kbest_step(h, W, b, prev, off, inp.k, S=len(layout))
    torch.cuda.synchronize()
    tok, par, sc = tok.cpu().numpy(), par.cpu().numpy(), sc.cpu().numpy()
    assert (tok[[1, 3]] == -1).all() and (par[[1, 3]] == -1).all() and np.isneginf(sc[[1, 3]]).all()
    check(inp, (tok[[0, 2]], par[[0, 2]], sc[[0, 2]]))
