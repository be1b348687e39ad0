"""Every projection tile on the same ragged steps, forced with KB_TILE, against
the fp64 oracle: the tiles the cost model picks for other shapes are checked
here on shapes it would not give them (many row tiles of 32 rows, a 256 x 256
tile over few rows, ...)."""
import pytest
import torch

from synth import workloads as wl
from tests.gpu_util import check, run_step, say

pytestmark = pytest.mark.gpu

DMA_TILES = ("256x256", "128x256", "256x128", "32x512", "32x256", "32x128", "64x128")
REG_TILES = ("128x256", "256x128", "32x512", "32x256", "32x128")
F32_DMA_TILES = REG_TILES + ("64x128",)            # the 256 x 256 tile is bf16 only
STEPS = [
    # (rows per sentence, H, V, k, dtype, tiles): bf16 DMA pipeline, register-staged, float32 DMA
    ([7] * 43, 128, 5000, 7, "bf16", DMA_TILES),     # 301 rows, ragged words (5000 = 19 x 256 + 136)
    ([3] * 15, 256, 9000, 3, "bf16", DMA_TILES),     # 45 rows: a 256-row tile mostly padding
    ([7] * 43, 96, 5003, 7, "bf16", REG_TILES),      # H not a multiple of 128, V odd
    ([5] * 61, 96, 4100, 5, "f32", REG_TILES),       # 305 rows, H not a multiple of 64
    ([5] * 61, 64, 4100, 5, "f32", F32_DMA_TILES),   # float32 DMA pipeline
    ([3] * 15, 192, 9004, 3, "f32", F32_DMA_TILES),  # 45 rows, words 9004 = 35 x 256 + 44
]


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


@pytest.mark.parametrize("case", range(len(STEPS)))
def test_every_tile_matches_the_oracle(kb, case, monkeypatch):
    rps, H, V, k, dt, tiles = STEPS[case]
    inp = wl.make_step(H=H, V=V, k=k, rows_per_sentence=rps, dtype=dt, seed=2100 + case, name=f"tiles{case}")
    code = kb.KB_BF16 if dt == "bf16" else kb.KB_F32
    for tile in tiles:
        monkeypatch.setenv("KB_TILE", tile)
        plan = kb.kbest_plan(code, inp.N, H, V, k)
        assert f"{plan['tile_rows']}x{plan['tile_words']}" == tile
        say(f"tiles case {case}: N={inp.N} H={H} V={V} k={k} {dt}, tile {tile} ({plan['kernel']})")
        rep, _ = check(inp, run_step(kb, inp, row_lse=True))
        say(f"  max score err {rep.max_score_err:.2e}")
