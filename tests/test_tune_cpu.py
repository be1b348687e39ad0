"""The tile override (KB_TILE) and the planner-tuning script's fit, on the CPU."""
import numpy as np
import pytest

import paper_1805_09863_amd as kb
from paper_1805_09863_amd import tune_planner as tp


@pytest.fixture
def tile_env(monkeypatch):
    def set_tile(v):
        if v is None:
            monkeypatch.delenv("KB_TILE", raising=False)
        else:
            monkeypatch.setenv("KB_TILE", v)
    return set_tile


def _p(dt, N, H, V, aligned=True):
    p = kb.kbest_plan(dt, N, H, V, 5, aligned=aligned)
    return f"{p['kernel']} {p['tile_rows']}x{p['tile_words']}"


def test_tile_override_follows_the_path(tile_env):
    tile_env(None)
    assert _p(kb.KB_BF16, 640, 1024, 60000) == "wide 256x256"
    tile_env("32x512")
    assert _p(kb.KB_BF16, 640, 1024, 60000) == "dma 32x512"
    assert _p(kb.KB_F32, 640, 1024, 60000) == "dma 32x512"
    assert _p(kb.KB_F32, 640, 1000, 60000) == "reg 32x512"
    tile_env("256x256")
    assert _p(kb.KB_BF16, 40, 1024, 50000) == "wide 256x256"
    assert _p(kb.KB_F32, 320, 512, 30000) == "dma 64x128"             # no 256 x 256 tile there: ignored
    assert _p(kb.KB_F32, 320, 520, 30000) == "reg 32x256"
    assert _p(kb.KB_BF16, 640, 1024, 60000, aligned=False) == "reg 256x128"
    assert _p(kb.KB_BF16, 300, 128, 200) == "dma 32x128"              # V < 256: ignored
    tile_env("64x128")
    assert _p(kb.KB_BF16, 640, 1024, 60000) == "dma 64x128"
    assert _p(kb.KB_F32, 640, 1024, 60000) == "dma 64x128"
    assert _p(kb.KB_BF16, 640, 1000, 60000) == "reg 256x128"            # the register-staged path has no 64-row tile: ignored
    tile_env("128x256")
    assert _p(kb.KB_F32, 5, 256, 8000) == "few 8x64"                  # the few-row kernel keeps its steps
    for bad in ("64x64", "32x256x", "x", "", "256"):
        tile_env(bad)
        assert _p(kb.KB_BF16, 640, 1024, 60000) == "wide 256x256"


def test_workspace_follows_the_override(tile_env):
    tile_env(None)
    a = kb.kbest_workspace_bytes(kb.KB_BF16, 3072, 1024, 90000, 12, 256)
    tile_env("32x128")
    b = kb.kbest_workspace_bytes(kb.KB_BF16, 3072, 1024, 90000, 12, 256)
    assert b != a   # 32-row tiles give other splits, hence other partials


def test_fit_recovers_the_model_and_evaluation_picks_it():
    rng = np.random.default_rng(0)
    truth = {"32x128": (8e-6, 3e-4, 25.0), "32x512": (7e-6, 3.3e-4, 20.0), "128x256": (5e-6, 4e-4, 15.0)}
    rows = []
    for H in (256, 512, 1024, 2048):
        for V in (8000, 30000, 60000):
            for N in (40, 100, 320, 1280):
                us = {}
                for t, (a, e, f) in truth.items():
                    r, w = tp.TILES[t]
                    us[t] = ((a * H + e) * tp.workgroup_words(N, V, r, w) + f) * (1 + 0.01 * rng.standard_normal())
                rows.append({"H": H, "V": V, "N": N, "us": us})
    model = tp.fit(rows, truth)
    for t, (a, e, f) in truth.items():
        assert model[t]["a"] == pytest.approx(a, rel=0.05) and model[t]["f"] == pytest.approx(f, rel=0.1)
        assert model[t]["mean_rel_err"] < 0.02
    ev = tp.evaluate(rows, model)
    assert ev["worst_ratio"] < 1.05 and ev["sum_us_model_choice"] <= 1.02 * ev["sum_us_best"]


def test_workgroup_words_matches_the_plan(tile_env):
    # the script's split rule, two 32 x 128 workgroups per CU on the DMA pipeline included
    for dt, path, N, H, V in ((kb.KB_F32, "f32", 320, 512, 30000), (kb.KB_F32, "f32reg", 320, 520, 30000),
                              (kb.KB_BF16, "bf16", 3072, 1024, 90000), (kb.KB_BF16, "bf16", 100, 256, 8000)):
        for tile in (None, "32x128", "32x256", "128x256"):
            tile_env(tile)
            p = kb.kbest_plan(dt, N, H, V, 5)
            t = f"{p['tile_rows']}x{p['tile_words']}"
            assert tp.workgroup_words(N, V, p["tile_rows"], p["tile_words"], tp.per_cu(path, t)) == \
                p["tile_rows"] * p["tile_words"] * p["tiles_per_split"]
