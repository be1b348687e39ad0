"""Measure every projection tile over a grid of step shapes and fit the
planner's cost model.

For each shape and each tile its path offers (forced with KB_TILE), the
projection kernel of kbest_step is timed with HIP events on its own stream
(median of the timed launches after warm-up).  Then, per tile, the model

    t = (a H + e) w + f        w = rows x words one workgroup covers
                                 = tile rows x tile words x tiles per split,
                                 doubled for a tile at two workgroups per CU
                                 whose grid exceeds 256 workgroups

is fitted by least squares on relative error, and the choice the model
makes on each shape is compared with the fastest tile measured there.  The
constants of kF32DmaCosts, kF32Costs and kBf16DmaCosts in csrc/kbest_abi.hip
come from this script's fit, one per path: --dtype f32 (H 256-2048, multiples
of 64: the DMA pipeline), f32reg (H 264-2056: the register-staged kernel;
kF32Costs was fitted at H 256-2048 while those shapes took it) and bf16 (the
DMA pipeline, H 512-2048 x V 8k-90k x 40-2,560 rows); float32 over V 8k-60k x
40-1,280 rows; k = 5.

    python -m paper_1805_09863_amd.tune_planner --dtype bf16 --out gpurun_out/tune_bf16.json

Operands are drawn on the device (normal h, W scaled by 1/sqrt(H), small
uniform bias); times do not depend on their values beyond the candidate
work a flat prior gives.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np
import torch

from paper_1805_09863_amd import binding
from paper_1805_09863_amd.hipevents import HipEvents

TILES = {  # KB_TILE value -> (rows, words) per tile
    "256x256": (256, 256), "128x256": (128, 256), "256x128": (256, 128),
    "32x512": (32, 512), "32x256": (32, 256), "32x128": (32, 128), "64x128": (64, 128),
}
GRIDS = {
    "f32": dict(H=(256, 512, 1024, 2048), V=(8000, 30000, 60000),
                N=(40, 64, 100, 160, 240, 320, 480, 640, 960, 1280),
                tiles=("128x256", "256x128", "32x512", "32x256", "32x128", "64x128")),
    "f32reg": dict(H=(264, 520, 1032, 2056), V=(8000, 30000, 60000),
                   N=(40, 64, 100, 160, 240, 320, 480, 640, 960, 1280),
                   tiles=("128x256", "256x128", "32x512", "32x256", "32x128")),
    "bf16": dict(H=(512, 1024, 2048), V=(8000, 30000, 50000, 90000),
                 N=(40, 64, 100, 160, 240, 320, 480, 640, 960, 1280, 2560),
                 tiles=tuple(TILES)),
}


def per_cu(dtype, tile: str) -> int:
    """Workgroups one CU holds at once, as the planner counts them at k <= 8:
    two of the DMA pipeline's 32 x 128 and 64 x 128 tiles, one of every other."""
    return 2 if dtype in ("f32", "bf16") and tile in ("32x128", "64x128") else 1


def workgroup_words(N: int, V: int, rows: int, words: int, per: int = 1) -> int:
    """rows x words one workgroup covers, with the planner's split rule."""
    rt, nt = -(-N // rows), -(-V // words)
    P = max(1, min(per * 256 // rt, nt, 256))
    return rows * words * -(-nt // P)


def model_words(N: int, V: int, rows: int, words: int, per: int = 1) -> int:
    """The model's w: a workgroup's rows x words, doubled for a tile planned at
    two workgroups per CU once its grid (row tiles x splits) exceeds 256."""
    w = workgroup_words(N, V, rows, words, per)
    rt, nt = -(-N // rows), -(-V // words)
    tps = w // (rows * words)
    return w * (2 if per == 2 and rt * -(-nt // tps) > 256 else 1)


def measure(dtype: str, grid: dict, reps: int, log) -> list:
    ev = HipEvents()
    code = binding.KB_BF16 if dtype == "bf16" else binding.KB_F32
    want = {"bf16": ("wide", "dma"), "f32": ("dma",), "f32reg": ("reg",)}[dtype]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device="cuda").manual_seed(7)
    rows = []
    for H in grid["H"]:
        for V in grid["V"]:
            W = (torch.randn((H, V), generator=g, device="cuda") / H ** 0.5).to(tdt)
            b = (torch.rand(V, generator=g, device="cuda") - 0.5) * 0.2
            for N in grid["N"]:
                S = (N + 4) // 5
                h = torch.randn((N, H), generator=g, device="cuda").to(tdt)
                prev = torch.zeros(N, device="cuda")
                off = torch.tensor([min(i * 5, N) for i in range(S + 1)], dtype=torch.int32, device="cuda")
                out = tuple(torch.empty((S, 5), dtype=t, device="cuda")
                            for t in (torch.int32, torch.int32, torch.float32))
                rec = {"H": H, "V": V, "N": N, "us": {}}
                for tile in grid["tiles"]:
                    os.environ["KB_TILE"] = tile
                    plan = binding.kbest_plan(code, N, H, V, 5)
                    if f"{plan['tile_rows']}x{plan['tile_words']}" != tile or plan["kernel"] not in want:
                        continue  # not on this path
                    ws = binding.workspace(binding.kbest_workspace_bytes(code, N, H, V, 5, S))
                    for _ in range(3):
                        binding.kbest_step(h, W, b, prev, off, 5, out=out, ws=ws)
                    torch.cuda.synchronize()
                    pairs = [(ev.create(), ev.create()) for _ in range(reps)]
                    for a, c in pairs:
                        binding.kbest_step(h, W, b, prev, off, 5, out=out, ws=ws, events=(a, c))
                    torch.cuda.synchronize()
                    t = sorted(ev.elapsed_ms(a, c) * 1e3 for a, c in pairs)
                    for a, c in pairs:
                        ev.destroy(a)
                        ev.destroy(c)
                    rec["us"][tile] = t[reps // 2]
                    del ws
                os.environ.pop("KB_TILE", None)
                rows.append(rec)
                log(json.dumps(rec))
            del W, b
            torch.cuda.empty_cache()
    return rows


def fit(rows: list, tiles, dtype=None) -> dict:
    """(a, e, f) per tile: least squares on relative error."""
    out = {}
    for tile in tiles:
        r, w = TILES[tile]
        pts = [x for x in rows if tile in x["us"]]
        if len(pts) < 3:
            continue
        pc = per_cu(dtype, tile)
        X = np.array([[x["H"] * model_words(x["N"], x["V"], r, w, pc), model_words(x["N"], x["V"], r, w, pc), 1.0]
                      for x in pts])
        y = np.array([x["us"][tile] for x in pts])
        c, *_ = np.linalg.lstsq(X / y[:, None], np.ones_like(y), rcond=None)
        err = np.abs(X @ c - y) / y
        out[tile] = {"a": float(c[0]), "e": float(c[1]), "f": float(c[2]),
                     "mean_rel_err": float(err.mean()), "max_rel_err": float(err.max())}
    return out


def planner_skips(N: int, V: int, tile: str, dtype) -> bool:
    """The planner leaves out a two-per-CU tile that would run alone on its CU
    with more than one tile in turn (its grid at most 256 workgroups)."""
    rows, words = TILES[tile]
    per = per_cu(dtype, tile)
    tps = workgroup_words(N, V, rows, words, per) // (rows * words)
    rt, nt = -(-N // rows), -(-V // words)
    return per == 2 and tps > 1 and rt * -(-nt // tps) <= 256


def evaluate(rows: list, model: dict, dtype=None) -> dict:
    """The model's choice on each shape against the fastest tile measured."""
    worst, tot_choice, tot_best = 1.0, 0.0, 0.0
    for x in rows:
        cands = [t for t in model if t in x["us"] and not planner_skips(x["N"], x["V"], t, dtype)]
        if not cands:
            continue

        def pred(t):
            r, w = TILES[t]
            wg = model_words(x["N"], x["V"], r, w, per_cu(dtype, t))
            m = model[t]
            return (m["a"] * x["H"] + m["e"]) * wg + m["f"]
        choice = min(cands, key=pred)
        best = min(x["us"].values())
        tot_choice += x["us"][choice]
        tot_best += best
        worst = max(worst, x["us"][choice] / best)
    return {"sum_us_model_choice": tot_choice, "sum_us_best": tot_best, "worst_ratio": worst}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--dtype", choices=tuple(GRIDS), required=True)
    ap.add_argument("--reps", type=int, default=15)
    ap.add_argument("--out", required=True, help="JSON: measured times, fitted constants, evaluation")
    ap.add_argument("--rows", help="comma-separated row counts in place of the grid's (e.g. 9,16,24,32)")
    ap.add_argument("--check", action="store_true",
                    help="no fit: compare the library's own choice (kb_kbest_plan) with the fastest tile")
    args = ap.parse_args()

    def log(msg):
        print(msg, file=sys.stderr, flush=True)
    grid = dict(GRIDS[args.dtype])
    if args.rows:
        grid["N"] = tuple(int(x) for x in args.rows.split(","))
    rows = measure(args.dtype, grid, args.reps, log)
    if args.check:
        code = binding.KB_BF16 if args.dtype == "bf16" else binding.KB_F32
        for x in rows:
            p = binding.kbest_plan(code, x["N"], x["H"], x["V"], 5)
            x["planner"] = f"{p['tile_rows']}x{p['tile_words']}"
        res = {"dtype": args.dtype, "grid": {k: list(v) for k, v in grid.items()}, "rows": rows,
               "sum_us_planner": sum(x["us"][x["planner"]] for x in rows),
               "sum_us_best": sum(min(x["us"].values()) for x in rows),
               "worst_ratio": max(x["us"][x["planner"]] / min(x["us"].values()) for x in rows)}
        with open(args.out, "w") as f:
            json.dump(res, f)
        log(json.dumps({k: v for k, v in res.items() if k.startswith(("sum", "worst"))}))
        return
    model = fit(rows, grid["tiles"], args.dtype)
    # the register-staged float32 planner leaves out the 256-row tile (it fits the model poorly)
    used = {t: m for t, m in model.items() if not (args.dtype == "f32reg" and t == "256x128")}
    res = {"dtype": args.dtype, "grid": {k: list(v) for k, v in grid.items()}, "rows": rows,
           "fit": model, "evaluation_of_the_planner_set": evaluate(rows, used, args.dtype)}
    with open(args.out, "w") as f:
        json.dump(res, f)
    for t, m in model.items():
        log(f"{t:8s} a={m['a']:.3e} e={m['e']:.3e} f={m['f']:.2f}  rel err mean {m['mean_rel_err']:.3f} "
            f"max {m['max_rel_err']:.3f}")
    log(json.dumps(res["evaluation_of_the_planner_set"]))


if __name__ == "__main__":
    main()
