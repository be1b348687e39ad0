"""Decode loops over a fixed synthetic schedule: mini-batching with removal of
finished hypotheses (Section 2.1, Algorithm 2) and the naive constant batch
(Algorithm 1).

The decoder RNN is not part of this library: each row's state h for step t
comes from a device table indexed by (sentence, step, beam slot), standing in
for the decoder.  Every output-layer step (projection, fused softmax/k-best,
beam merge) and every compaction and state gather runs in libkbest's kernels;
the decoder stand-in's bookkeeping (EOS mask of the schedule, next states)
runs in its own small kernels (include/kbest_standin.h).
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Callable, Optional

import torch

from . import binding as kbb


def _poll_tag(cn, tag: int):
    """Wait until the kernel has written ``tag`` to cn[2] (pinned host memory,
    after the counts it guards): no event is recorded or waited on per step
    (an event cost the device about 6 us a step).  A tag that does not come
    within a second leads to a device synchronisation, which raises if the
    device has failed, and then to an error."""
    n = 0
    while cn[2] != tag:
        n += 1
        if n & 0xFFFF == 0:
            if n == 0x10000:
                t0 = time.perf_counter()
            elif time.perf_counter() - t0 > 1.0:
                torch.cuda.synchronize()
                if cn[2] != tag:
                    raise RuntimeError(f"step tag {tag} never arrived (found {int(cn[2])})")


def _wait(ev: torch.cuda.Event):
    """Wait for ev by polling.  The wait covers most of a step, and a blocking
    wait of that length woke the host tens of microseconds after the event, by
    which time the device had drained the one step queued behind it."""
    while not ev.query():
        pass


@dataclass
class LoopStats:
    steps: int = 0
    rows: list = field(default_factory=list)         # live rows decoded at each step
    total_rows: int = 0
    launch_rows: list = field(default_factory=list)  # rows each launch was sized for (compacted loop)


def decode_loop(h_table: torch.Tensor, W: torch.Tensor, b: torch.Tensor, lengths: torch.Tensor,
                prev0: torch.Tensor, k: int, T: int, *, compact: bool = True,
                on_step: Optional[Callable] = None, stream=None) -> LoopStats:
    """Run the beam-search output layer over the whole schedule.

    ``h_table`` is (S0*T*beam) x H on the device (row (s*T + t)*beam + r is the
    state of slot r of sentence s at step t), ``lengths`` S0 int32: sentence s
    emits EOS on all its continuations at step L_s - 1 (1 <= L_s <= T).
    ``prev0`` holds the S0*k scores of the step-0 hypotheses (beam = k rows
    per sentence).

    ``compact=True``: after each step the finished entries are removed
    (Algorithm 2) and the loop ends when the batch is empty.
    ``compact=False``: the batch keeps all S0 sentences until the longest is
    done (Algorithm 1); finished sentences' rows are decoded and ignored.

    A compacted step enqueues the output layer and the stand-in's step (EOS
    mask, compaction, gathers of the surviving scores, sentence ids and next
    states: one launch).  The batch only shrinks, so step
    t + 1 is launched sized by the exact counts of step t (rows, sentences), read from the
    device while step t is still queued: the host never waits for the step it
    has just launched, and the device never waits for the host.  Every kernel
    of a step takes the exact counts of its own batch from the device (the
    compaction's outputs); rows and sentences past them are launched but
    empty, since the compaction pads the sentence offsets past its last kept
    sentence.  The price is a few rows of the sentences that ended at the step
    before, and one launch at the end whose batch turns out to be empty.

    ``on_step(t, state)`` is called once step t's work is queued, with a dict
    of the device tensors of that step cut to its exact counts; work that
    on_step queues on ``stream`` sees them complete, and they stay intact
    until on_step returns.  In the compacted loop ``S_launch`` and
    ``N_launch`` give the sizes the step was launched with, ``token_launch``
    and ``score_launch`` its whole outputs.
    """
    dev = W.device
    beam = k
    S0 = lengths.numel()
    H, V = W.shape
    stats = LoopStats()
    if S0 == 0:
        return stats
    len_host = lengths.cpu().tolist()
    Lmax = max(len_host)
    if Lmax > T or min(len_host) < 1:
        raise ValueError("lengths must lie in [1, T]")
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    M0 = S0 * k
    lengths = lengths.to(device=dev, dtype=torch.int32).contiguous()
    # the plan (and so the workspace) depends on the row count, which shrinks
    dt = kbb._dtype_code(W)
    ws = kbb.workspace(max(kbb.kbest_workspace_bytes(dt, s * beam, H, V, k, s) for s in range(1, S0 + 1)), dev)
    i32 = dict(dtype=torch.int32, device=dev)
    tok = torch.empty(M0, **i32)
    par = torch.empty(M0, **i32)
    sc = torch.empty(M0, dtype=torch.float32, device=dev)
    h_cur = torch.empty((M0, H), dtype=h_table.dtype, device=dev)
    ident = torch.arange(M0, **i32)                      # entry e of an S0 x k batch is row e
    sid = torch.arange(S0, **i32)                        # original id of each live sentence
    off = (torch.arange(S0 + 1, **i32) * beam).contiguous()
    prev = prev0.to(device=dev, dtype=torch.float32, copy=True).contiguous()   # the loop writes its own
    kbb.standin_next_h(h_table, ident, sid, k, T, 0, M0, out=h_cur, stream=stream)
    S, N, t = S0, M0, 0
    if compact:
        keep = torch.empty(M0, **i32)
        noff = torch.empty(S0 + 1, **i32)
        # rows past a step's exact count are projected: keep them finite
        h_nx = torch.zeros((M0, H), dtype=h_table.dtype, device=dev)
        prev_nx = torch.zeros(M0, dtype=torch.float32, device=dev)
        sid_nx = torch.empty(S0, **i32)
        # counts (kept rows, kept sentences) of each step, double-buffered on
        # both sides: step t writes slot t % 2, read back one step later; the
        # host copy carries the step's tag t + 1 after the counts (0: none yet)
        cnt = [torch.empty(2, **i32) for _ in range(2)]
        cnt_host = [torch.zeros(3, dtype=torch.int32, pin_memory=True) for _ in range(2)]
        # A step's host work bounds small batches (its device work is a few
        # tens of us), so the buffers are checked once here, at the largest
        # batch, as the binding checks them, and the steps call the library
        # with their cached addresses (no per-step tensor views or checks).
        f32, i32t = torch.float32, torch.int32
        for name, x, d, n in (("h", h_cur, h_table.dtype, M0 * H), ("h_next", h_nx, h_table.dtype, M0 * H),
                              ("W", W, h_table.dtype, H * V), ("b", b, f32, V), ("prev", prev, f32, M0),
                              ("prev_next", prev_nx, f32, M0), ("sent_offsets", off, i32t, S0 + 1),
                              ("new_sent_offsets", noff, i32t, S0 + 1), ("token", tok, i32t, M0),
                              ("parent", par, i32t, M0), ("score", sc, f32, M0), ("keep", keep, i32t, M0),
                              ("sid", sid, i32t, S0), ("sid_next", sid_nx, i32t, S0), ("lengths", lengths, i32t, S0),
                              ("table", h_table, h_table.dtype, S0 * T * k * H), ("counts", cnt[0], i32t, 2),
                              ("counts", cnt[1], i32t, 2), ("ws", ws, None, None)):
            kbb._need(x, name, dtype=d, numel=n)
        if h_table.dim() != 2 or h_table.shape[1] != H:
            raise ValueError("h_table must be rows x H")
        L = kbb.lib()
        st_h = kbb._stream(stream, dev)
        Wp, bp, tokp, parp, scp, keepp = (x.data_ptr() for x in (W, b, tok, par, sc, keep))
        lenp, tabp, wsp, ws_bytes = lengths.data_ptr(), h_table.data_ptr(), ws.data_ptr(), ws.numel()
        row_bytes = H * h_table.element_size()
        cnt_p = [c.data_ptr() for c in cnt]
        cnt_hp = [c.data_ptr() for c in cnt_host]
        cnt_np = [c.numpy() for c in cnt_host]          # views of the pinned counts
        hp, hnp = h_cur.data_ptr(), h_nx.data_ptr()
        pp, pnp = prev.data_ptr(), prev_nx.data_ptr()
        sidp, sidnp = sid.data_ptr(), sid_nx.data_ptr()
        offp, noffp = off.data_ptr(), noff.data_ptr()
        S_exp = None                                    # the device's count of the current batch's sentences
        while t < T:
            kbb._check(L.kb_kbest_step(dt, N, H, V, k, S, hp, Wp, bp, pp, offp, tokp, parp, scp, None, wsp,
                                       ws_bytes, st_h))
            # EOS mask, compaction, surviving scores, sentence ids and next states:
            # one launch (the counts also land in pinned host memory, read once
            # the step is done)
            nxt = t + 1 < T
            kbb._check(L.kb_standin_step(S, S_exp, k, t, sidp, lenp, scp, keepp, cnt_p[t % 2], noffp, pnp, sidnp,
                                         None, cnt_hp[t % 2], tabp if nxt else None, T, hnp if nxt else None,
                                         row_bytes, st_h))
            stats.launch_rows.append(N)
            # the exact counts of this step's batch: the previous step's output
            if t == 0:
                N_ex, S_now = M0, S0
            else:
                cn = cnt_np[(t - 1) % 2]
                _poll_tag(cn, t)
                N_ex, S_now = int(cn[0]), int(cn[1])
            if N_ex == 0:
                break                                    # every sentence had ended: this launch was empty
            stats.rows.append(N_ex)
            if on_step is not None:
                on_step(t, dict(h=h_cur[:N_ex], prev=prev[:N_ex], off=off[:S_now + 1], sid=sid[:S_now],
                                token=tok[:S_now * k].view(S_now, k), parent=par[:S_now * k].view(S_now, k),
                                score=sc[:S_now * k].view(S_now, k), S=S_now, N=N_ex, S_launch=S, N_launch=N,
                                token_launch=tok[:S * k].view(S, k), score_launch=sc[:S * k].view(S, k)))
            N, S = N_ex, S_now                           # bounds of the next step's batch
            S_exp = cnt_p[t % 2] + 4                     # counts[1] of this step
            prev, prev_nx, pp, pnp = prev_nx, prev, pnp, pp
            sid, sid_nx, sidp, sidnp = sid_nx, sid, sidnp, sidp
            off, noff, offp, noffp = noff, off, noffp, offp
            h_cur, h_nx, hp, hnp = h_nx, h_cur, hnp, hp
            t += 1
    else:
        while t < Lmax:
            kbb.kbest_step(h_cur, W, b, prev, off, k, S=S0,
                           out=(tok.view(S0, k), par.view(S0, k), sc.view(S0, k)), ws=ws, stream=stream)
            stats.rows.append(sum(1 for L in len_host if L > t) * beam)
            if on_step is not None:
                on_step(t, dict(h=h_cur, prev=prev, off=off, sid=sid, token=tok.view(S0, k),
                                parent=par.view(S0, k), score=sc.view(S0, k), S=S0, N=M0))
            prev, sc = sc, prev                            # this step's scores feed the next
            if t + 1 < T:
                kbb.standin_next_h(h_table, ident, sid, k, T, t + 1, M0, out=h_cur, stream=stream)
            t += 1
    stats.steps = t
    stats.total_rows = sum(stats.rows)
    return stats


@dataclass
class BeamSearchResult:
    tokens: torch.Tensor      # S0 x T int32: each sentence's translation, EOS included, then -1
    length: torch.Tensor      # S0 int32
    score: torch.Tensor       # S0 float32, cumulative log-probability
    norm: torch.Tensor        # S0 float32, score / length**alpha
    steps: int = 0
    rows: list = field(default_factory=list)   # live rows decoded at each step


def beam_search(h_table: torch.Tensor, W: torch.Tensor, b: torch.Tensor, k: int, T: int, eos: int, *,
                alpha: float = 0.0, on_step: Optional[Callable] = None, stream=None) -> BeamSearchResult:
    """Beam search with per-hypothesis end of sentence (Section 2.1, Algorithm 2).

    ``h_table`` is (S0*T*k) x H on the device: row (s*T + t)*k + r is the state
    of the hypothesis in slot r (its rank in the sentence's beam) of sentence s
    at step t, the decoder stand-in.  Every sentence starts from one hypothesis
    (slot 0, score 0) with a beam of k.  Each step: the output layer
    (kb_kbest_step), kb_beam_finish (history, finished store, beam shrink),
    kb_compact_beams, the gathers of the surviving scores, sentence ids and
    beam sizes, and the stand-in's next states; then one wait for the two
    counts.  A sentence ends when its beam is empty; step T - 1 finishes every
    hypothesis left.  kb_beam_backtrace then picks each sentence's translation
    by score / length**alpha.

    ``on_step(t, state)`` is called after each step's kb_beam_finish with a
    dict of the step's device tensors (before the batch is compacted).
    """
    dev = W.device
    H, V = W.shape
    S0 = h_table.shape[0] // (T * k)
    if h_table.shape[0] != S0 * T * k or S0 == 0:
        raise ValueError("h_table must hold S0 * T * k rows")
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    M0 = S0 * k
    i32 = dict(dtype=torch.int32, device=dev)
    dt = kbb._dtype_code(W)
    # the plan (and so the workspace) depends on the row count, anything from 1 to S0*k
    ws = kbb.workspace(max(kbb.kbest_workspace_bytes(dt, n, H, V, k, 1) for n in range(1, M0 + 1)), dev)
    tok = torch.empty(M0, **i32)
    par = torch.empty(M0, **i32)
    sc = torch.empty(M0, dtype=torch.float32, device=dev)
    h_cur = torch.empty((M0, H), dtype=h_table.dtype, device=dev)
    alive = torch.empty(M0, dtype=torch.uint8, device=dev)
    keep = [torch.empty(M0, **i32), torch.empty(M0, **i32)]
    cnt = torch.empty(2, **i32)
    noff = torch.empty(S0 + 1, **i32)
    ksent = torch.empty(S0, **i32)
    hist_tok = torch.empty(T * M0, **i32)
    hist_par = torch.empty(T * M0, **i32)
    fin = (torch.zeros(S0, **i32), torch.empty(M0, dtype=torch.float32, device=dev), torch.empty(M0, **i32),
           torch.empty(M0, **i32))
    sid, sid_nx = torch.arange(S0, **i32), torch.empty(S0, **i32)
    beam, beam_nx = torch.full((S0,), k, **i32), torch.empty(S0, **i32)
    prev, prev_nx = torch.zeros(M0, dtype=torch.float32, device=dev), torch.empty(M0, dtype=torch.float32, device=dev)
    off = torch.arange(S0 + 1, **i32)                  # one row per sentence at the start
    cnt_host = torch.empty(2, dtype=torch.int32, pin_memory=True)
    ready = torch.cuda.Event()
    # step 0's states: slot 0 of every sentence
    kbb.standin_next_h(h_table, torch.arange(S0, **i32) * k, torch.arange(S0, **i32), k, T, 0, S0, out=h_cur,
                       stream=stream)
    out = BeamSearchResult(None, None, None, None)
    S, N, t, cur, prev_base = S0, S0, 0, 0, 0
    while S > 0 and t < T:
        kbb.kbest_step(h_cur[:N], W, b, prev[:N], off[:S + 1], k, S=S,
                       out=(tok[:S * k].view(S, k), par[:S * k].view(S, k), sc[:S * k].view(S, k)),
                       ws=ws, stream=stream)
        out.rows.append(N)
        beam_before = beam[:S].clone() if on_step is not None else None
        base = t * M0
        kbb.beam_finish(S, k, t, T, eos, tok, par, sc, sid, beam, keep[1 - cur] if t > 0 else None, prev_base,
                        base, hist_tok, hist_par, fin, alive, stream=stream)
        if on_step is not None:
            on_step(t, dict(h=h_cur[:N], prev=prev[:N], off=off[:S + 1], sid=sid[:S], beam_before=beam_before,
                            beam_after=beam[:S], token=tok[:S * k].view(S, k), parent=par[:S * k].view(S, k),
                            score=sc[:S * k].view(S, k), alive=alive[:S * k],
                            prev_keep=keep[1 - cur][:N] if t > 0 else None, prev_base=prev_base, base=base,
                            hist_token=hist_tok, hist_parent=hist_par, fin=fin, S=S, N=N))
        kbb.compact_beams(alive[:S * k], S, k, out=(keep[cur], cnt[0:1], noff, ksent, cnt[1:2]), stream=stream)
        with torch.cuda.stream(stream):                # the copy runs on the loop's stream
            cnt_host.copy_(cnt, non_blocking=True)
        ready.record(stream)
        kbb.gather_rows(sc[:S * k].view(S * k, 1), keep[cur], n_dev=cnt[0:1], n_max=S * k,
                        out=prev_nx.view(M0, 1), stream=stream)
        kbb.gather_rows(sid[:S].view(S, 1), ksent, n_dev=cnt[1:2], n_max=S, out=sid_nx.view(S0, 1), stream=stream)
        kbb.gather_rows(beam[:S].view(S, 1), ksent, n_dev=cnt[1:2], n_max=S, out=beam_nx.view(S0, 1),
                        stream=stream)
        if t + 1 < T:
            kbb.standin_next_h(h_table, keep[cur], sid, k, T, t + 1, S * k, n_dev=cnt[0:1], out=h_cur, stream=stream)
        _wait(ready)                                   # the step's one host sync
        N, S = (int(x) for x in cnt_host.tolist())
        prev, prev_nx = prev_nx, prev
        sid, sid_nx = sid_nx, sid
        beam, beam_nx = beam_nx, beam
        off, noff = noff, off
        prev_base = base
        cur = 1 - cur
        t += 1
    out.tokens, out.length, out.score, out.norm = kbb.beam_backtrace(S0, k, T, alpha, fin, hist_tok, hist_par,
                                                                     stream=stream)
    out.steps = t
    out.fin = fin
    out.hist = (hist_tok, hist_par)
    return out
