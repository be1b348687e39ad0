"""Seeded random step shapes against the fp64 oracle: dtype, state size,
vocabulary (multiples of the vector width and ragged), k from 1 to 16 and
sentences of mixed beam widths, so that the planner's choices (few-row
kernel, 256 x 256 tiles, the other DMA tiles, register-staged tiles) meet
combinations no hand-picked case covers.  The plan of each case is printed
with it."""
import numpy as np
import pytest
import torch

from synth import workloads as wl
from tests.gpu_util import check, run_step, say

pytestmark = pytest.mark.gpu

N_CASES = 40
MAX_WORK = 6e8  # N * H * V of a case, which bounds the oracle's time


def _cases():
    g = np.random.default_rng(20260)
    out = []
    while len(out) < N_CASES:
        dt = "bf16" if g.random() < 0.7 else "f32"
        # half of them DMA-able (H a multiple of 128, V of 8), the rest not
        dma = g.random() < 0.5
        H = int(g.choice([128, 256, 384, 512])) if dma else int(g.choice([32, 64, 96, 200, 256]))
        V = int(g.integers(17, 40000))
        if dma or g.random() < 0.3:
            V -= V % 8                      # 16-byte loadable rows
        V = max(V, 17)
        k = int(min(g.integers(1, 17), V))
        rps = []
        n_rows = int(g.integers(1, 700))
        while sum(rps) < n_rows:
            rps.append(int(g.integers(1, 17)))
        if sum(rps) * H * V > MAX_WORK:
            continue
        out.append((rps, H, V, k, dt))
    return out


CASES = _cases()


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_shape(kb, case):
    rps, H, V, k, dt = CASES[case]
    inp = wl.make_step(H=H, V=V, k=k, rows_per_sentence=rps, dtype=dt, seed=3000 + case, name=f"rand{case}")
    p = kb.kbest_plan(kb.KB_BF16 if dt == "bf16" else kb.KB_F32, inp.N, H, V, k)
    say(f"random case {case}: N={inp.N} S={inp.S} H={H} V={V} k={k} {dt}: {p['kernel']} "
        f"{p['tile_rows']}x{p['tile_words']}, {p['splits']} splits of {p['tiles_per_split']}")
    rep, _ = check(inp, run_step(kb, inp, row_lse=True))
    say(f"  max score err {rep.max_score_err:.2e}")
