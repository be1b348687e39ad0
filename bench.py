#!/usr/bin/env python3
"""Throughput of the fused output-layer step on MI355X.

Headline workload: one decode step of 256 sentences x beam 12 (N = 3072
hypotheses), state size H = 1024, vocabulary V = 90,000, k = 12, bf16 h and W
with float32 accumulation, Zipf-shaped bias.  A timed step is one full
``kbest_step`` (fused projection + softmax statistics + per-split k-best,
then the split/beam merge) with every input already resident in HBM.

Prints ONE JSON line on stdout.  Besides the throughput it carries
  * ``roofline``: the fused projection kernel's achieved MFMA rate (2*N*H*V
    flops per launch / its mean duration from HIP events recorded around
    each launch on the launch stream) against the bf16 dense peak, and the
    HBM bytes per launch measured by rocprofv3 counters when a matching
    counter summary is present;
  * ``cpu_baseline``: the fp64 oracle on a bounded sample of the same
    workload, on this host's cores;
  * ``decode_loop``: the 512-sentence multi-step loop with removal of
    finished hypotheses against the constant-size batch.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
K1_SOURCES = [os.path.join(ROOT, "paper_1805_09863_amd", "csrc", f)
              for f in ("kb_common.hpp", "k1_common.hpp", "k1_wide.hpp")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k1_wide_N3072_H1024_V90000_k12_hbm_traffic.txt")


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


class HipEvents:
    """Raw hipEvent_t handles from the HIP runtime torch already loaded."""

    def __init__(self):
        self.rt = ctypes.CDLL("libamdhip64.so.7")
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self) -> int:
        ev = ctypes.c_void_p()
        if self.rt.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        if self.rt.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def destroy(self, ev: int):
        self.rt.hipEventDestroy(ctypes.c_void_p(ev))


def k1_source_hash() -> str:
    """Hash of the projection kernel's code (line comments and blank lines
    dropped): counter summaries apply only to this code."""
    h = hashlib.sha256()
    for p in K1_SOURCES:
        with open(p) as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def read_traffic():
    """HBM bytes per fused-projection launch from the committed counter summary,
    if it was taken on the current kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    with open(TRAFFIC_FILE) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                key, val = line.split("=", 1)
                kv[key.strip()] = val.strip()
    if kv.get("k1_source_sha256_16") != k1_source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def to_dev(inp, torch, np):
    h = torch.from_numpy(inp.h.view(np.int16)).view(torch.bfloat16).cuda()
    W = torch.from_numpy(inp.W.view(np.int16)).view(torch.bfloat16).cuda()
    b = torch.from_numpy(inp.b).cuda()
    prev = torch.from_numpy(inp.prev).cuda()
    off = torch.from_numpy(inp.off).cuda()
    return h, W, b, prev, off


def cpu_baseline(inp, n_sent: int):
    """The fp64 oracle (full definition, stable sort) on the first n_sent sentences."""
    import numpy as np
    from oracle import kbest_oracle as ko
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"] or [1])
    except Exception:  # threadpoolctl missing or no BLAS info
        threads = os.cpu_count() or 1
    rows = int(inp.off[n_sent])
    t0 = time.perf_counter()
    ko.kbest_step(inp.h[:rows], inp.W, inp.b, inp.prev[:rows], inp.off[:n_sent + 1], inp.k, dtype=inp.dtype)
    dt = time.perf_counter() - t0
    return {"value": rows / dt, "unit": "hyps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {n_sent} of {inp.S} sentences ({rows} of {inp.N} rows), full V={inp.V}, "
                      f"fp64 logits + 3-pass softmax + full stable sort per sentence; {dt:.1f} s",
            "seconds": dt, "host_cpus": os.cpu_count()}


def decode_loop_bench(torch, np, reps: int = 2):
    from paper_1805_09863_amd.decode import decode_loop
    from synth import workloads as wl
    work = wl.make_loop_workload()
    tab = work.h_table().reshape(-1, work.H)
    h_table = torch.from_numpy(tab.view(np.int16)).view(torch.bfloat16).cuda()
    W = torch.from_numpy(work.W.view(np.int16)).view(torch.bfloat16).cuda()
    b = torch.from_numpy(work.b).cuda()
    L = torch.from_numpy(work.lengths).cuda()
    p0 = torch.from_numpy(work.prev0).cuda()
    out = {}
    for name, compact in (("compacted", True), ("naive", False)):
        decode_loop(h_table, W, b, L, p0, work.k, work.T, compact=compact)     # warm-up
        best = None
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            st = decode_loop(h_table, W, b, L, p0, work.k, work.T, compact=compact)
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            best = dt if best is None else min(best, dt)
        out[name] = {"seconds": best, "steps": st.steps, "live_rows": st.total_rows,
                     "live_hyps_per_s": st.total_rows / best}
        log(f"decode loop {name}: {best * 1e3:.2f} ms, {st.steps} steps, {st.total_rows} live rows")
    out["speedup_from_compaction"] = out["naive"]["seconds"] / out["compacted"]["seconds"]
    out["workload"] = f"S={work.S} beam={work.k} H={work.H} V={work.V} k={work.k} bf16, L~U[5,60]"
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-sample-sentences", type=int, default=160)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode-loop", action="store_true")
    ap.add_argument("--print-k1-hash", action="store_true", help="print the projection-kernel source hash and exit")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB three times (to scale HBM "
                         "byte counters against a kernel of known traffic), then exit")
    args = ap.parse_args()
    if args.print_k1_hash:
        print(k1_source_hash())
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the output layer shards by sentence or vocabulary; no multi-GPU path is built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_1805_09863_amd as kb
    from synth import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration_mib:
        nbytes = args.copy_calibration_mib << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "launches": 3}))
        return
    kb.lib()
    log("generating the V=90k workload ...")
    inp = wl.make_workload(wl.V90K)
    N, H, V, k, S = inp.N, inp.H, inp.V, inp.k, inp.S
    h, W, b, prev, off = to_dev(inp, torch, np)
    tok = torch.empty((S, k), dtype=torch.int32, device="cuda")
    par = torch.empty((S, k), dtype=torch.int32, device="cuda")
    sc = torch.empty((S, k), dtype=torch.float32, device="cuda")
    ws = kb.workspace(kb.kbest_workspace_bytes(kb.KB_BF16, N, H, V, k, S))
    ev = HipEvents()
    pairs = [(ev.create(), ev.create()) for _ in range(args.steps)]

    for _ in range(args.warmup):
        kb.kbest_step(h, W, b, prev, off, k, out=(tok, par, sc), ws=ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        kb.kbest_step(h, W, b, prev, off, k, out=(tok, par, sc), ws=ws, events=pairs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    k1_ms = [ev.elapsed_ms(a, c) for a, c in pairs]
    k1_mean = sum(k1_ms) / len(k1_ms)
    for a, c in pairs:
        ev.destroy(a)
        ev.destroy(c)
    flops = 2.0 * N * H * V
    achieved = flops / (k1_mean * 1e-3) / 1e12
    log(f"step {ms_per_step:.3f} ms, fused projection {k1_mean:.3f} ms (min {min(k1_ms):.3f}), "
        f"{achieved:.1f} TFLOP/s")

    result = {
        "metric": "hypotheses/sec through fused kbest_step (V=90k); MFMA % and HBM GB/s of peak",
        "value": N / (ms_per_step * 1e-3),
        "unit": "hyps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; h~N(0,1), W~N(0,1/sqrt(H)), Zipf bias -0.5*ln(j+1), prev~U(-5,0))",
        "config": {"workload": inp.name, "sentences": S, "beam": inp.N // S, "N": N, "H": H, "V": V, "k": k,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": read_traffic(),
                     "kernel": "k1_wide (projection + bias + softmax statistics + per-split k-best)",
                     "kernel_ms": k1_mean, "flops_per_launch": flops},
    }
    tr = result["roofline"]["traffic"]
    if tr is not None:
        result["roofline"]["hbm_gbs"] = tr / (k1_mean * 1e-3) / 1e9
        result["roofline"]["hbm_frac"] = result["roofline"]["hbm_gbs"] / PEAK_HBM_GBS
    if not args.no_decode_loop:
        result["decode_loop"] = decode_loop_bench(torch, np)
    if not args.no_cpu_baseline:
        log(f"timing the oracle on {args.cpu_sample_sentences} sentences ...")
        result["cpu_baseline"] = cpu_baseline(inp, args.cpu_sample_sentences)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
