"""GPU parity of the unfused baseline (kb_kbest_step_unfused): Algorithm 3
(mode 0: separate projection, AddBias, three-pass Softmax, k-best
extraction, beam merge) and Algorithm 4 over stored scores (mode 1), against
the fp64 oracle with the same rules as the fused step, and against the fused
step itself.
"""
import numpy as np
import pytest
import torch

from synth import workloads as wl
from tests.gpu_util import TOL, check, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


CASES = [
    # (rows per sentence, H, V, k)
    ([5] * 4, 128, 1000, 5),            # 20 rows, one row tile, ragged word tile
    ([1] * 300, 256, 2056, 1),          # beam 1; last word tile of 8 words
    ([3] * 100, 128, 9000, 3),          # beam 3
    ([9] * 70, 384, 6216, 9),           # beam 9, 630 rows: three row tiles
    ([12] * 50, 256, 5000, 12),
    ([16] * 20, 128, 3000, 16),
]


def _run(kb, inp, mode):
    h, W, b, prev, off = to_dev(inp)
    lse = torch.full((inp.N,), float("nan"), dtype=torch.float32, device="cuda")
    tok, par, sc = kb.kbest_step_unfused(h, W, b, prev, off, inp.k, mode=mode, row_lse=lse)
    torch.cuda.synchronize()
    return tok.cpu().numpy(), par.cpu().numpy(), sc.cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_unfused_shapes(kb, case, mode):
    rps, H, V, k = CASES[case]
    inp = wl.make_step(H=H, V=V, k=k, rows_per_sentence=rps, dtype="bf16", seed=1200 + case,
                       name=f"unfused{case}")
    say(f"unfused case {case} mode {mode}: N={inp.N} H={H} V={V} k={k}")
    out = _run(kb, inp, mode)
    rep, _ = check(inp, out)
    say(f"  max score err {rep.max_score_err:.2e}, {rep.n_checked_idx} exact ranks")


@pytest.mark.parametrize("mode", [0, 1])
def test_unfused_matches_fused_v90k_sampled(kb, mode):
    # the V=90k shape: oracle on sampled sentences, and the fused step's
    # scores within float32 rounding of the baseline's
    inp = wl.make_workload(wl.V90K)
    h, W, b, prev, off = to_dev(inp)
    t1, p1, s1 = kb.kbest_step_unfused(h, W, b, prev, off, inp.k, mode=mode)
    t2, p2, s2 = kb.kbest_step(h, W, b, prev, off, inp.k)
    torch.cuda.synchronize()
    out = (t1.cpu().numpy(), p1.cpu().numpy(), s1.cpu().numpy())
    sents = sorted(set(np.random.default_rng(11).choice(inp.S, 8, replace=False).tolist()) | {0, inp.S - 1})
    check(inp, out, sentences=sents)
    d = np.abs(out[2] - s2.cpu().numpy()).max()
    assert d <= TOL["bf16"], f"unfused vs fused scores differ by {d}"
    say(f"unfused mode {mode} V=90k: max |unfused - fused| = {d:.2e}")
