"""The projection plan (kb_kbest_plan, no device needed): every GPU parity
case, its tile pinned as the GPU tests pin it, runs on the kernel and tile it
was written for, and the workloads' plans (the cost models' own choices) are
the ones the design describes."""
import pytest

import paper_1805_09863_amd as kb
from paper_1805_09863_amd.binding import KBestError
from tests.parity_cases import ARGMAX, FEW, SHARDS, SMALL, WIDE, tile_env


def _code(dt: str) -> int:
    return kb.KB_BF16 if dt == "bf16" else kb.KB_F32


def _plan_str(p: dict) -> str:
    return f"{p['kernel']} {p['tile_rows']}x{p['tile_words']}"


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_case_plans(case, monkeypatch):
    rps, H, V, k, dt, want = SMALL[case]
    tile_env(monkeypatch, want)
    assert _plan_str(kb.kbest_plan(_code(dt), sum(rps), H, V, k)) == want


@pytest.mark.parametrize("case", range(len(WIDE)))
def test_wide_case_plans(case, monkeypatch):
    rps, H, V, k, want = WIDE[case]
    tile_env(monkeypatch, want)
    assert _plan_str(kb.kbest_plan(kb.KB_BF16, sum(rps), H, V, k)) == want


@pytest.mark.parametrize("case", range(len(FEW)))
def test_few_case_plans(case, monkeypatch):
    rps, H, V, k, dt, want = FEW[case]
    tile_env(monkeypatch, want)
    assert _plan_str(kb.kbest_plan(_code(dt), sum(rps), H, V, k)) == want


@pytest.mark.parametrize("case", range(len(ARGMAX)))
def test_argmax_case_plans(case, monkeypatch):
    N, H, V, dt, want = ARGMAX[case]
    tile_env(monkeypatch, want)
    assert _plan_str(kb.kbest_plan(_code(dt), N, H, V, 1)) == want


@pytest.mark.parametrize("case", range(len(SHARDS)))
def test_shard_case_plans(case, monkeypatch):
    rps, H, V, k, dt, cuts, want = SHARDS[case]
    tile_env(monkeypatch, want)
    got = {_plan_str(kb.kbest_plan(_code(dt), sum(rps), H, b - a, k)) for a, b in zip(cuts, cuts[1:])}
    assert got == want


def test_wide_cases_keep_their_edges(monkeypatch):
    # the features the 256 x 256 cases are listed for
    monkeypatch.setenv("KB_TILE", "256x256")

    def plan(i):
        rps, H, V, k, _ = WIDE[i]
        return kb.kbest_plan(kb.KB_BF16, sum(rps), H, V, k), sum(rps), V
    p, N, V = plan(0)
    assert p["row_tiles"] == 1 and N == 129
    p, N, V = plan(2)
    assert p["row_tiles"] == 2 and N % 256
    for i, tail in ((4, 8), (5, 136)):
        p, N, V = plan(i)
        nt = -(-V // 256)
        assert V % 256 == tail and p["tiles_per_split"] >= 2
        assert nt - (p["splits"] - 1) * p["tiles_per_split"] == 1   # the ragged tile alone in the last split
    p, N, V = plan(8)
    assert p["row_tiles"] == 4 and p["tiles_per_split"] >= 2
    p, N, V = plan(10)
    assert p["tiles_per_split"] == 1


@pytest.mark.parametrize("dt,N,H,V,k,want", [
    ("f32", 5, 256, 8000, 5, ("few", 8, 64, 1, 125, 1)),              # one sentence, beam 5
    ("f32", 320, 512, 30000, 5, ("dma", 64, 128, 5, 79, 3)),         # 64 sentences, beam 5: two workgroups a CU
    ("bf16", 640, 1024, 60000, 5, ("wide", 256, 256, 3, 79, 3)),     # 128 sentences, beam 5
    ("bf16", 3072, 1024, 90000, 12, ("wide", 256, 256, 12, 21, 17)),  # 256 sentences, beam 12
    ("bf16", 2560, 1024, 50000, 5, ("wide", 256, 256, 10, 25, 8)),   # the decode loop's first step
])
def test_workload_plans(dt, N, H, V, k, want):
    p = kb.kbest_plan(_code(dt), N, H, V, k)
    assert (p["kernel"], p["tile_rows"], p["tile_words"], p["row_tiles"], p["splits"], p["tiles_per_split"]) == want


def test_plan_follows_alignment():
    # bf16 at unaligned addresses cannot use the DMA pipeline
    assert kb.kbest_plan(kb.KB_BF16, 640, 1024, 60000, 5)["kernel"] == "wide"
    assert kb.kbest_plan(kb.KB_BF16, 640, 1024, 60000, 5, aligned=False)["kernel"] == "reg"
    # nor can H that is not a multiple of 128
    assert kb.kbest_plan(kb.KB_BF16, 640, 1000, 60000, 5)["kernel"] == "reg"
    # float32: H a multiple of 64 and V of 4, 16-byte aligned
    assert kb.kbest_plan(kb.KB_F32, 320, 512, 30000, 5)["kernel"] == "dma"
    assert kb.kbest_plan(kb.KB_F32, 320, 512, 30000, 5, aligned=False)["kernel"] == "reg"
    assert kb.kbest_plan(kb.KB_F32, 320, 544, 30000, 5)["kernel"] == "reg"
    assert kb.kbest_plan(kb.KB_F32, 320, 512, 30002, 5)["kernel"] == "reg"


def test_plan_split_invariants():
    for dt in ("f32", "bf16"):
        for N in (9, 33, 100, 257, 1000, 5000):
            for V in (200, 3001, 50000, 131072):
                p = kb.kbest_plan(_code(dt), N, 256, V, 5)
                nt = -(-V // p["tile_words"])
                assert p["row_tiles"] == -(-N // p["tile_rows"])
                # one workgroup per CU, two of the DMA pipeline's 32 x 128 and (k <= 8) 64 x 128 tiles
                per = 2 if (p["kernel"] == "dma" and p["tile_words"] == 128 and p["tile_rows"] in (32, 64)) else 1
                assert 1 <= p["splits"] <= 256 and p["row_tiles"] * p["splits"] <= max(per * 256, p["row_tiles"])
                assert (p["splits"] - 1) * p["tiles_per_split"] < nt <= p["splits"] * p["tiles_per_split"]


def test_plan_errors():
    assert kb.kbest_plan(kb.KB_BF16, 0, 1024, 50000, 5)["kernel"] is None
    with pytest.raises(KBestError):
        kb.kbest_plan(kb.KB_BF16, 10, 1024, 50000, 0)
    with pytest.raises(KBestError):
        kb.kbest_plan(7, 10, 1024, 50000, 5)
    L = kb.lib()
    assert L.kb_kbest_plan(kb.KB_BF16, 10, 1024, 50000, 5, 1 << 20, 1 << 20, 1 << 20, None) == 1
    out = (__import__("ctypes").c_int32 * 6)()
    assert L.kb_kbest_plan(kb.KB_BF16, 10, 1024, 50000, 5, (1 << 20) + 1, 1 << 20, 1 << 20, out) == 1
