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


def HipEvents():
    """Raw hipEvent_t handles (paper_1805_09863_amd/hipevents.py), imported
    when first needed so that argument errors come before torch loads."""
    from paper_1805_09863_amd.hipevents import HipEvents as _HipEvents
    return _HipEvents()


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
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": rows / dt, "unit": "hyps/s", "cores": int(threads), "kind": "oracle", "cpu_model": model,
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


def _mean_stage_ms(ev, sets):
    """Mean over repetitions of the gaps between consecutive events of each set."""
    n = len(sets[0]) - 1
    return [sum(ev.elapsed_ms(es[i], es[i + 1]) for es in sets) / len(sets) for i in range(n)]


def ablation_bench(torch, np, kb, reps: int = 10):
    """Time per stage of one step, fused against the unfused baselines (the
    paper's breakdown into multiplication, add bias, softmax and k-best),
    256 sentences at V=90k (H=1024, bf16, Zipf bias) with beam = k = 1, 3, 9."""
    from synth import workloads as wl
    ev = HipEvents()
    S, H, V = 256, 1024, 90000
    big = wl.make_step(H=H, V=V, k=9, S=S, beam=9, dtype="bf16", seed=wl.SEED_BASE + 77, bias="zipf")
    W = torch.from_numpy(big.W.view(np.int16)).view(torch.bfloat16).cuda()
    b = torch.from_numpy(big.b).cuda()
    rows = []
    for beam in (1, 3, 9):
        N, k = S * beam, beam
        h = torch.from_numpy(np.ascontiguousarray(big.h[:N]).view(np.int16)).view(torch.bfloat16).cuda()
        prev = torch.from_numpy(np.ascontiguousarray(big.prev[:N])).cuda()
        off = torch.from_numpy(wl.uniform_offsets(S, beam)).cuda()
        out = tuple(torch.empty((S, k), dtype=t, device="cuda") for t in (torch.int32, torch.int32, torch.float32))
        ws_f = kb.workspace(kb.kbest_workspace_bytes(kb.KB_BF16, N, H, V, k, S))
        ws_u = kb.workspace(kb.unfused_workspace_bytes(kb.KB_BF16, N, H, V, k, S))
        res = {"beam": beam, "k": k, "N": N}
        # fused: reset kernel, [event] K1 [event] K2 [event]  (the 12 KB threshold reset before
        # the first event, a few microseconds, is left out: the event before it would also
        # time the host's launch work on an idle GPU)
        sets = [[ev.create() for _ in range(3)] for _ in range(reps)]
        for i in range(2 + reps):
            es = sets[i - 2] if i >= 2 else sets[0]
            kb.kbest_step(h, W, b, prev, off, k, out=out, ws=ws_f, events=(es[0], es[1]))
            ev.rt.hipEventRecord(ctypes.c_void_p(es[2]), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            torch.cuda.synchronize()
        g = _mean_stage_ms(ev, sets)
        res["fused_ms"] = {"projection_bias_softmax_kbest": g[0], "merge": g[1], "total": sum(g)}
        for mode, names in ((0, ["multiplication", "add_bias", "softmax", "kbest", "merge"]),
                            (1, ["multiplication", "fused_pass", "merge"])):
            sets = [[ev.create() for _ in range(len(names) + 1)] for _ in range(reps)]
            for i in range(2 + reps):
                es = sets[i - 2] if i >= 2 else sets[0]
                kb.kbest_step_unfused(h, W, b, prev, off, k, mode=mode, out=out, ws=ws_u, events=es)
                torch.cuda.synchronize()
            g = _mean_stage_ms(ev, sets)
            d = dict(zip(names, g))
            d["total"] = sum(g)
            res["alg3_unfused_ms" if mode == 0 else "alg4_over_stored_ms"] = d
        rows.append(res)
        log(f"ablation beam {beam}: fused {res['fused_ms']['total']:.3f} ms, "
            f"Alg.4 over stored {res['alg4_over_stored_ms']['total']:.3f} ms, "
            f"Alg.3 {res['alg3_unfused_ms']['total']:.3f} ms")
        del ws_u
    # greedy decoding (Algorithm 5, no softmax) against the k = 1 step, beam 1,
    # back-to-back launches (mean per call)
    greedy = []
    for N in (256, 1280, 2304):
        h = torch.from_numpy(np.ascontiguousarray(big.h[:N]).view(np.int16)).view(torch.bfloat16).cuda()
        prev = torch.from_numpy(np.ascontiguousarray(big.prev[:N])).cuda()
        off = torch.from_numpy(wl.uniform_offsets(N, 1)).cuda()
        out = tuple(torch.empty((N, 1), dtype=t, device="cuda") for t in (torch.int32, torch.int32, torch.float32))
        tv = (torch.empty(N, dtype=torch.int32, device="cuda"), torch.empty(N, dtype=torch.float32, device="cuda"))
        ws_f = kb.workspace(kb.kbest_workspace_bytes(kb.KB_BF16, N, H, V, 1, N))
        ws_a = kb.workspace(kb.argmax_workspace_bytes(kb.KB_BF16, N, H, V))
        g = {"N": N}
        for name, fn in (("kbest_k1", lambda: kb.kbest_step(h, W, b, prev, off, 1, out=out, ws=ws_f)),
                         ("greedy_argmax", lambda: kb.argmax_step(h, W, b, out=tv, ws=ws_a))):
            for _ in range(3):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps * 2):
                fn()
            e1.record()
            torch.cuda.synchronize()
            g[name + "_ms"] = e0.elapsed_time(e1) / (reps * 2)
        log(f"greedy N={N}: k=1 step {g['kbest_k1_ms']:.3f} ms, argmax {g['greedy_argmax_ms']:.3f} ms")
        greedy.append(g)
    # the half-precision comparison (the paper's tensor-core table): the same step
    # with float32 h and W (fp32 MFMA) against bf16 storage (bf16 MFMA), beams 1 and 9
    prec = []
    W32 = torch.from_numpy(wl.bf16_bits_to_f32(big.W)).cuda()
    for beam in (1, 9):
        N, k = S * beam, beam
        hb = torch.from_numpy(np.ascontiguousarray(big.h[:N]).view(np.int16)).view(torch.bfloat16).cuda()
        h32 = hb.float()
        prev = torch.from_numpy(np.ascontiguousarray(big.prev[:N])).cuda()
        off = torch.from_numpy(wl.uniform_offsets(S, beam)).cuda()
        out = tuple(torch.empty((S, k), dtype=t, device="cuda") for t in (torch.int32, torch.int32, torch.float32))
        g = {"beam": beam, "N": N}
        for name, hh, WW, dt in (("float32", h32, W32, kb.KB_F32), ("bf16", hb, W, kb.KB_BF16)):
            ws = kb.workspace(kb.kbest_workspace_bytes(dt, N, H, V, k, S))
            for _ in range(2):
                kb.kbest_step(hh, WW, b, prev, off, k, out=out, ws=ws)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps):
                kb.kbest_step(hh, WW, b, prev, off, k, out=out, ws=ws)
            e1.record()
            torch.cuda.synchronize()
            g[name + "_ms"] = e0.elapsed_time(e1) / reps
        log(f"precision beam {beam}: float32 {g['float32_ms']:.3f} ms, bf16 {g['bf16_ms']:.3f} ms")
        prec.append(g)
    del W32
    return {"workload": f"S={S} sentences x beam 1/3/9 (k = beam), H={H}, V={V}, bf16, Zipf bias",
            "reps": reps, "rows": rows, "greedy_beam1": greedy, "precision": prec}


PEAK_F32_TFLOPS = 157.3


def configs_bench(torch, np, kb, reps: int = 50):
    """Every single-step workload (the decode-loop one is timed by the loop):
    warm steps back to back (HIP events around all of them: the time per
    step), each step alone between its own events (latency: median and min;
    an event record costs the device a few microseconds), cold steps
    after a 512 MB write, the projection kernel alone, its roofline, and the
    fp64 oracle on the whole workload beside it (on the host's cores)."""
    from oracle import kbest_oracle as ko
    from synth import workloads as wl
    res = []
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    ev = HipEvents()
    stream = torch.cuda.current_stream().cuda_stream
    for c in wl.WORKLOADS[:4]:
        inp = wl.make_workload(c["name"])
        N, H, V, k, S = inp.N, inp.H, inp.V, inp.k, inp.S
        if inp.dtype == "bf16":
            h, W, b, prev, off = to_dev(inp, torch, np)
        else:
            h, W = torch.from_numpy(inp.h).cuda(), torch.from_numpy(inp.W).cuda()
            b, prev, off = (torch.from_numpy(x).cuda() for x in (inp.b, inp.prev, inp.off))
        dt = kb.KB_BF16 if inp.dtype == "bf16" else kb.KB_F32
        out = tuple(torch.empty((S, k), dtype=t, device="cuda") for t in (torch.int32, torch.int32, torch.float32))
        ws = kb.workspace(kb.kbest_workspace_bytes(dt, N, H, V, k, S))
        step = lambda events=None: kb.kbest_step(h, W, b, prev, off, k, out=out, ws=ws, events=events)
        for _ in range(50):                # the clock settles over the first ~40 launches of a heavy step
            step()
        torch.cuda.synchronize()
        pairs = [(ev.create(), ev.create()) for _ in range(reps)]
        ev.record(pairs[0][0], stream)     # warm, back to back: one pair of events around all the steps
        for i in range(reps):
            step()
        ev.record(pairs[0][1], stream)
        torch.cuda.synchronize()
        b2b = ev.elapsed_ms(*pairs[0]) / reps
        for i in range(reps):              # warm latency: each step alone between its own events
            ev.record(pairs[i][0], stream)
            step()
            ev.record(pairs[i][1], stream)
        torch.cuda.synchronize()
        warm = sorted(ev.elapsed_ms(x, y) for x, y in pairs)
        for i in range(reps):              # the projection kernel alone
            step(events=pairs[i])
        torch.cuda.synchronize()
        kern = sorted(ev.elapsed_ms(x, y) for x, y in pairs)
        cold = []
        for i in range(10):
            flush.fill_(1)
            ev.record(pairs[i][0], stream)
            step()
            ev.record(pairs[i][1], stream)
            torch.cuda.synchronize()
            cold.append(ev.elapsed_ms(*pairs[i]))
        cold.sort()
        for x, y in pairs:
            ev.destroy(x)
            ev.destroy(y)
        esz = 2 if inp.dtype == "bf16" else 4
        nbytes = H * V * esz + N * H * esz + V * 4 + N * 4 + S * k * 12
        flops = 2.0 * N * H * V
        km = kern[len(kern) // 2]
        if flops / nbytes < (PEAK_BF16_TFLOPS if inp.dtype == "bf16" else PEAK_F32_TFLOPS) * 1e12 / (PEAK_HBM_GBS * 1e9):
            roof = {"bound": "hbm", "achieved": nbytes / (km * 1e-3) / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
        else:
            pk = PEAK_BF16_TFLOPS if inp.dtype == "bf16" else PEAK_F32_TFLOPS
            roof = {"bound": "mfma", "achieved": flops / (km * 1e-3) / 1e12, "peak": pk, "unit": "TFLOP/s"}
        roof["frac"] = roof["achieved"] / roof["peak"]
        t0 = time.perf_counter()
        orc_runs = 10 if N * V < 1e6 else 1
        whole = N * V < 1e8               # the V=90k workload's oracle is timed on a sample by the main bench
        for _ in range(orc_runs if whole else 0):
            ko.kbest_step(inp.h, inp.W, inp.b, inp.prev, inp.off, k, dtype=inp.dtype)
        orc = (time.perf_counter() - t0) / orc_runs if whole else None
        res.append({"workload": inp.name, "N": N, "H": H, "V": V, "k": k, "dtype": inp.dtype,
                    "step_ms": b2b, "step_latency_ms_median": warm[len(warm) // 2],
                    "step_latency_ms_min": warm[0],
                    "cold_step_ms_median": cold[len(cold) // 2], "kernel_ms_median": km,
                    "hyps_per_s": N / (b2b * 1e-3), "roofline": roof,
                    "oracle_s": orc, "oracle_hyps_per_s": (N / orc) if orc else None})
        log(f"{inp.name}: step {b2b:.4f} ms back to back, {warm[len(warm) // 2]:.4f} ms alone, kernel {km:.4f} ms, "
            f"{roof['bound']} {roof['frac'] * 100:.1f}%, oracle {orc}")
    del flush
    return res


def shard_bench(torch, np, kb, reps: int = 20):
    """One device's part of a vocabulary-split step (Algorithm 6 across devices):
    the V=90k workload cut into 8 shards on multiples of 8 words; each shard's
    fused projection and the merge of all shards' partials, timed with events
    on the stream, next to the whole step on one device.  The all-gather of the
    partials between devices is not built; its size is reported."""
    from synth import workloads as wl
    inp = wl.make_workload(wl.V90K)
    h, W, b, prev, off = to_dev(inp, torch, np)
    N, k, V = inp.N, inp.k, inp.V
    cuts = [11256 * i for i in range(8)] + [V]
    shards = [(a, W[:, a:z].contiguous(), b[a:z].contiguous()) for a, z in zip(cuts, cuts[1:])]
    Ps = [kb.shard_splits(h, Wg, bg, k) for _, Wg, bg in shards]
    P = sum(Ps)
    stats = torch.empty((P, N, 2), dtype=torch.float32, device="cuda")
    lists = torch.empty((P, N, k, 2), dtype=torch.int32, device="cuda")
    wss = [kb.workspace(kb.binding.lib().kb_shard_workspace_bytes(kb.KB_BF16, N, inp.H, Wg.shape[1], k))
           for _, Wg, _ in shards]
    offs = np.concatenate([[0], np.cumsum(Ps)]).tolist()
    out = tuple(torch.empty((inp.S, k), dtype=t, device="cuda") for t in (torch.int32, torch.int32, torch.float32))
    ws_full = kb.workspace(kb.kbest_workspace_bytes(kb.KB_BF16, N, inp.H, V, k, inp.S))

    def timed(fn):
        for _ in range(5):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    shard_ms = []
    for i, (a, Wg, bg) in enumerate(shards):
        sl = slice(offs[i], offs[i + 1])
        shard_ms.append(timed(lambda: kb.shard_partials(h, Wg, bg, k, a, stats[sl], lists[sl], ws=wss[i])))
    merge_ms = timed(lambda: kb.merge_partials(stats, lists, P, V, k, prev, off, out=out))
    whole_ms = timed(lambda: kb.kbest_step(h, W, b, prev, off, k, out=out, ws=ws_full))
    flops = 2.0 * N * inp.H * 11256
    return {"workload": f"{inp.name} over 8 vocabulary shards (7 x 11256 + {V - 7 * 11256} words)",
            "splits_per_shard": Ps, "shard_ms": shard_ms, "shard_tflops": flops / (max(shard_ms) * 1e-3) / 1e12,
            "merge_ms": merge_ms, "one_device_share_ms": max(shard_ms) + merge_ms, "whole_step_one_device_ms": whole_ms,
            "exchange_bytes_per_device": Ps[0] * N * (8 + 8 * k),
            "note": "the all-gather of the partials between devices is not built (one GPU); its size is given"}


def sweep_bench(torch, np, kb):
    """Step time against the number of rows, the per-step time of a 1280-sentence
    decode (compacted and naive), and decode throughput against the number of
    sentences (beam 5, H=1024, V=50k, bf16)."""
    from paper_1805_09863_amd.decode import decode_loop
    from synth import workloads as wl
    S0, T, beam, H = 1280, 60, 5, 1024
    work = wl.make_loop_workload(S=S0)
    V = work.V
    W = torch.from_numpy(work.W.view(np.int16)).view(torch.bfloat16).cuda()
    b = torch.from_numpy(work.b).cuda()
    gen = torch.Generator(device="cuda").manual_seed(wl.SEED_BASE + 5)
    h_table = torch.empty((S0 * T * beam, H), dtype=torch.bfloat16, device="cuda")
    for i in range(0, h_table.shape[0], 65536):   # the decoder stand-in's states, drawn on the device
        h_table[i:i + 65536] = torch.randn((min(65536, h_table.shape[0] - i), H), generator=gen, device="cuda")
    L = torch.from_numpy(work.lengths).cuda()
    p0 = torch.from_numpy(work.prev0).cuda()
    out = {"workload": f"beam {beam}, H={H}, V={V}, bf16, uniform bias, lengths ~U{{5..60}}"}
    # (1) one step against the number of rows
    step = []
    for N in (5, 10, 25, 50, 100, 200, 320, 500, 640, 1000, 1280, 2000, 2560, 3200, 4096):
        Sx = (N + beam - 1) // beam
        h = h_table[:N].contiguous()
        prev = torch.zeros(N, device="cuda")
        off = torch.tensor([min(i * beam, N) for i in range(Sx + 1)], dtype=torch.int32, device="cuda")
        ws = kb.workspace(kb.kbest_workspace_bytes(kb.KB_BF16, N, H, V, beam, Sx))
        for _ in range(3):
            kb.kbest_step(h, W, b, prev, off, beam, ws=ws)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(20):
            kb.kbest_step(h, W, b, prev, off, beam, ws=ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 20
        step.append({"N": N, "ms": ms, "hyps_per_s": N / (ms * 1e-3)})
        log(f"sweep step N={N}: {ms * 1e3:.1f} us")
    out["step_vs_rows"] = step
    # (2) per-step time of the 1280-sentence decode: three timed runs after a
    # warm-up, each step's median over them (a host that stalls between two
    # steps of one run leaves the device idle, and that gap would count)
    curves = {}
    for compact in (True, False):
        decode_loop(h_table, W, b, L, p0, beam, T, compact=compact)          # warm-up
        torch.cuda.synchronize()
        runs = []
        for _ in range(3):
            marks = []

            def on_step(t, st, marks=marks):
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks.append((st["N"], e))
            start = torch.cuda.Event(enable_timing=True)
            start.record()
            decode_loop(h_table, W, b, L, p0, beam, T, compact=compact, on_step=on_step)
            torch.cuda.synchronize()
            prev_e, per = start, []
            for n, e in marks:
                per.append((n, prev_e.elapsed_time(e)))
                prev_e = e
            runs.append(per)
        curves["compacted" if compact else "naive"] = [
            {"rows": runs[0][t][0], "ms": float(np.median([r[t][1] for r in runs])),
             "ms_runs": [r[t][1] for r in runs]} for t in range(len(runs[0]))]
    out["per_step_1280"] = curves
    # (3) decode throughput against the number of sentences
    by_s = []
    for Sx in (1, 2, 5, 10, 20, 50, 100, 200, 500, 1000, 1280):
        r = {"S": Sx}
        for compact in (True, False):
            tab = h_table[:Sx * T * beam]
            decode_loop(tab, W, b, L[:Sx], p0[:Sx * beam], beam, T, compact=compact)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            st = decode_loop(tab, W, b, L[:Sx], p0[:Sx * beam], beam, T, compact=compact)
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            r["compacted" if compact else "naive"] = {"seconds": dt, "live_rows": st.total_rows,
                                                      "live_hyps_per_s": st.total_rows / dt,
                                                      "sentences_per_s": Sx / dt}
        log(f"sweep S={Sx}: compacted {r['compacted']['seconds'] * 1e3:.2f} ms, "
            f"naive {r['naive']['seconds'] * 1e3:.2f} ms")
        by_s.append(r)
    out["decode_vs_sentences"] = by_s
    # (4) beam search with natural end of sentence (per-hypothesis EOS, beam shrink,
    # length-normalised choice, backtrace), 1280 sentences at beam 5
    from paper_1805_09863_amd.decode import beam_search
    eos, T2 = 3, 80
    gen = torch.Generator(device="cuda").manual_seed(wl.SEED_BASE + 6)
    Ls = torch.randint(5, 61, (S0,), generator=gen, device="cuda").float()
    w = W[:, eos].float()
    u = (w / (w @ w)).to(torch.bfloat16)
    tab = torch.empty((S0 * T2 * beam, H), dtype=torch.bfloat16, device="cuda")
    step_of_row = (torch.arange(T2, device="cuda").repeat_interleave(beam)).float()   # t of rows (s, t, r)
    for s0 in range(0, S0, 64):                       # the stand-in's states, drawn on the device
        n = min(64, S0 - s0)
        x = torch.randn((n, T2 * beam, H), generator=gen, device="cuda")
        ramp = 3.0 * (step_of_row[None, :] - Ls[s0:s0 + n, None])
        tab[s0 * T2 * beam:(s0 + n) * T2 * beam] = (x + ramp[:, :, None] * u.float()[None, None, :]).reshape(
            -1, H).to(torch.bfloat16)
    beam_search(tab, W, b, beam, T2, eos, alpha=1.0)   # warm-up
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = beam_search(tab, W, b, beam, T2, eos, alpha=1.0)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ln = r.length.float()
    out["beam_search_natural_eos_1280"] = {
        "seconds": dt, "steps": r.steps, "live_rows": sum(r.rows), "live_hyps_per_s": sum(r.rows) / dt,
        "sentences_per_s": S0 / dt, "mean_length": float(ln.mean()), "max_length": int(ln.max()),
        "setup": f"{S0} sentences, beam {beam}, EOS score rising 3 per step past a length ~U{{5..60}}, "
                 f"cap T={T2}, alpha=1"}
    log(f"beam search, natural EOS: {dt * 1e3:.2f} ms, {r.steps} steps, {sum(r.rows)} live rows")
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--cpu-sample-sentences", type=int, default=160)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode-loop", action="store_true")
    ap.add_argument("--print-k1-hash", action="store_true", help="print the projection-kernel source hash and exit")
    ap.add_argument("--ablation", action="store_true",
                    help="only time the fused step against the unfused baselines, stage by stage "
                         "(beams 1/3/9 at V=90k), print that as the JSON line and exit")
    ap.add_argument("--sweep", action="store_true",
                    help="only run the row-count and batch-size sweeps and the per-step curves of a "
                         "1280-sentence decode, print them as the JSON line and exit")
    ap.add_argument("--configs", action="store_true",
                    help="only time every single-step workload (warm, cold, kernel, roofline, oracle beside it), "
                         "print that as the JSON line and exit")
    ap.add_argument("--shards", action="store_true",
                    help="only time one device's part of a step split over 8 vocabulary shards (each shard's "
                         "projection and the merge of all partials) at V=90k, print it as the JSON line and exit")
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
    if args.configs:
        kb.lib()
        res = {"metric": "step time per workload", "unit": "ms", "data": "synthetic (seeded)", "n_gpus": 1,
               "configs": configs_bench(torch, np, kb)}
        print(json.dumps(res), flush=True)
        return
    if args.shards:
        kb.lib()
        res = {"metric": "vocabulary-split step, one device's part", "unit": "ms", "data": "synthetic (seeded)",
               "n_gpus": 1, "shards": shard_bench(torch, np, kb)}
        print(json.dumps(res), flush=True)
        return
    if args.ablation or args.sweep:
        kb.lib()
        res = {"metric": "fused vs unfused step time by stage" if args.ablation else "sweeps",
               "unit": "ms", "data": "synthetic (seeded)", "n_gpus": 1}
        res["ablation" if args.ablation else "sweep"] = (ablation_bench if args.ablation else sweep_bench)(
            torch, np, kb)
        print(json.dumps(res), flush=True)
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

    for _ in range(args.warmup):
        kb.kbest_step(h, W, b, prev, off, k, out=(tok, par, sc), ws=ws)

    def kernel_pass(n):
        """n steps with HIP events recorded on the step's stream right before
        and after the projection kernel; returns the kernel's durations (ms)
        and the pass's wall time per step."""
        ps = [(ev.create(), ev.create()) for _ in range(n)]
        torch.cuda.synchronize()
        ta = time.perf_counter()
        for i in range(n):
            kb.kbest_step(h, W, b, prev, off, k, out=(tok, par, sc), ws=ws, events=ps[i])
        torch.cuda.synchronize()
        tb = time.perf_counter()
        d = [ev.elapsed_ms(a, c) for a, c in ps]
        for a, c in ps:
            ev.destroy(a)
            ev.destroy(c)
        return d, (tb - ta) * 1e3 / n

    # the kernel pass runs first as well (at least 40 launches): the clock
    # under this load settles over the first few dozen launches, and the
    # timed passes below should both see the settled clock
    settle_ms, _ = kernel_pass(max(args.steps, 40))
    # timed step pass: K steps back to back, nothing else on the stream (an
    # event marker between two kernels costs the GPU ~5 us)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        kb.kbest_step(h, W, b, prev, off, k, out=(tok, par, sc), ws=ws)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    # timed kernel pass: the same K steps with events around the projection
    k1_ms, ms_with_events = kernel_pass(args.steps)
    k1_mean = sum(k1_ms) / len(k1_ms)
    k1_sorted = sorted(k1_ms)
    k1_median = k1_sorted[len(k1_sorted) // 2]
    # cold steps: a 512 MB write between steps evicts W (184 MB) from the
    # 256 MB last-level cache, so each timed step streams W from HBM; the
    # step and its projection kernel are timed with events
    cold_ms, cold_k1 = [], []
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    c0, c1, e0, e1 = ev.create(), ev.create(), ev.create(), ev.create()
    stream = torch.cuda.current_stream().cuda_stream
    for _ in range(10):
        flush.fill_(1)
        ev.record(c0, stream)
        kb.kbest_step(h, W, b, prev, off, k, out=(tok, par, sc), ws=ws, events=(e0, e1))
        ev.record(c1, stream)
        torch.cuda.synchronize()
        cold_ms.append(ev.elapsed_ms(c0, c1))
        cold_k1.append(ev.elapsed_ms(e0, e1))
    for e in (c0, c1, e0, e1):
        ev.destroy(e)
    del flush
    cold_ms.sort()
    cold_k1.sort()
    flops = 2.0 * N * H * V
    achieved = flops / (k1_mean * 1e-3) / 1e12
    cold_step, cold_kernel = cold_ms[len(cold_ms) // 2], cold_k1[len(cold_k1) // 2]
    log(f"step {ms_per_step:.3f} ms, fused projection {k1_mean:.3f} ms (min {min(k1_ms):.3f}), "
        f"{achieved:.1f} TFLOP/s; cold step {cold_step:.3f} ms, kernel {cold_kernel:.3f} ms")

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
                     "kernel_ms": k1_mean, "kernel_ms_median": k1_median, "kernel_ms_min": k1_sorted[0],
                     "flops_per_launch": flops,
                     "cold": {"hyps_per_s": N / (cold_step * 1e-3), "kernel_ms": cold_kernel,
                              "achieved": flops / (cold_kernel * 1e-3) / 1e12,
                              "frac": flops / (cold_kernel * 1e-3) / 1e12 / PEAK_BF16_TFLOPS},
                     "timing": "after the W warm-up steps, a kernel-event pass of max(K, 40) steps lets the "
                               "clock settle (untimed); then ms_per_step: K steps back to back, wall clock "
                               "synchronised on both sides; then kernel_ms: the same K steps with HIP events "
                               "on the kernel's stream around each projection launch; cold: 10 steps each "
                               "after a 512 MB write that evicts W from the last-level cache (medians)"},
        "ms_per_step_with_kernel_events": ms_with_events,
        "kernel_ms_settling_pass": sum(settle_ms) / len(settle_ms),
        "cold": {"ms_per_step_median": cold_step, "ms_per_step_min": cold_ms[0], "kernel_ms_median": cold_kernel,
                 "kernel_ms_min": cold_k1[0], "reps": 10,
                 "note": "512 MB written between steps; each step timed alone with HIP events"},
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
