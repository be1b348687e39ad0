"""Decode loops over a fixed synthetic schedule: mini-batching with removal of
finished hypotheses (Section 2.1, Algorithm 2) and the naive constant batch
(Algorithm 1).

The decoder RNN is not part of this library: each row's state h for step t
comes from a device table indexed by (sentence, step, beam slot), standing in
for the decoder.  Every output-layer step (projection, fused softmax/k-best,
beam merge) and every compaction and state gather runs in libkbest's kernels;
the few small torch ops here only form the decoder stand-in's row indices and
the EOS mask of the schedule.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Optional

import torch

from . import binding as kbb


@dataclass
class LoopStats:
    steps: int = 0
    rows: list = field(default_factory=list)     # live rows decoded at each step
    total_rows: int = 0


def _hrow_index(sid_rows: torch.Tensor, slot_rows: torch.Tensor, t: int, T: int, beam: int) -> torch.Tensor:
    return ((sid_rows.long() * T + t) * beam + slot_rows.long()).to(torch.int32)


def decode_loop(h_table: torch.Tensor, W: torch.Tensor, b: torch.Tensor, lengths: torch.Tensor,
                prev0: torch.Tensor, k: int, T: int, *, compact: bool = True,
                on_step: Optional[Callable] = None, stream=None) -> LoopStats:
    """Run the beam-search output layer over the whole schedule.

    ``h_table`` is (S0*T*beam) x H on the device (row (s*T + t)*beam + r is the
    state of slot r of sentence s at step t), ``lengths`` S0 int32: sentence s
    emits EOS on all its continuations at step L_s - 1.  ``prev0`` holds the
    S0*k scores of the step-0 hypotheses (beam = k rows per sentence).

    ``compact=True``: after each step the finished entries are removed
    (Algorithm 2) and the loop ends when the batch is empty.
    ``compact=False``: the batch keeps all S0 sentences until the longest is
    done (Algorithm 1); finished sentences' rows are decoded and ignored.

    ``on_step(t, state)`` is called after each output-layer step with a dict
    of the device tensors of that step.
    """
    dev = W.device
    beam = k
    S0 = lengths.numel()
    Lmax = int(lengths.max().item()) if S0 > 0 else 0
    sid = torch.arange(S0, dtype=torch.int32, device=dev)            # original id of each live sentence
    row_sid = sid.repeat_interleave(beam)
    row_slot = torch.arange(beam, dtype=torch.int32, device=dev).repeat(S0)
    prev = prev0.to(torch.float32).contiguous()
    off = (torch.arange(S0 + 1, dtype=torch.int32, device=dev) * beam).contiguous()
    S, N = S0, S0 * beam
    H, V = W.shape
    # the plan (and so the workspace) depends on the row count, which shrinks
    dt = kbb._dtype_code(W)
    ws = kbb.workspace(max(kbb.kbest_workspace_bytes(dt, s * beam, H, V, k, s) for s in range(1, S0 + 1))
                       if S0 > 0 else 1, dev)
    h_cur = torch.empty((N, H), dtype=h_table.dtype, device=dev)
    stats = LoopStats()
    len_host = lengths.cpu().tolist()
    lengths = lengths.to(device=dev, dtype=torch.int32)
    t = 0
    while (S > 0) if compact else (t < Lmax):
        hidx = _hrow_index(row_sid, row_slot, t, T, beam)
        kbb.gather_rows(h_table, hidx, out=h_cur[:N], stream=stream)
        tok, par, sc = kbb.kbest_step(h_cur[:N], W, b, prev, off, k, S=S, ws=ws, stream=stream)
        stats.rows.append(N if compact else sum(1 for L in len_host if L > t) * beam)
        if on_step is not None:
            on_step(t, dict(h=h_cur[:N], prev=prev, off=off, sid=sid, token=tok, parent=par, score=sc, S=S, N=N))
        if compact:
            alive = (t < lengths[sid.long()] - 1).to(torch.uint8).repeat_interleave(k)
            keep, kept, noff, ksent, nS = kbb.compact_batch(alive, S, k, stream=stream)
            n_new, s_new = (int(x) for x in torch.cat([kept, nS]).cpu())   # the step's one host sync
            prev = kbb.gather_rows(sc.view(S * k, 1), keep, n_max=n_new, stream=stream).view(n_new)
            new_sid = kbb.gather_rows(sid.view(S, 1), ksent, n_max=s_new, stream=stream).view(s_new)
            kk = keep[:n_new].long()
            row_sid = sid[kk // k] if n_new else sid[:0]
            row_slot = (kk % k).to(torch.int32)
            sid, S, N = new_sid, s_new, n_new
            off = noff[:s_new + 1].contiguous()
        else:
            prev = sc.view(S * k)
            row_slot = torch.arange(beam, dtype=torch.int32, device=dev).repeat(S0)
        t += 1
    stats.steps = t
    stats.total_rows = sum(stats.rows)
    return stats
