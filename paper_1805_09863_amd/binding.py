"""ctypes binding of libkbest (the C ABI in include/kbest.h).

Argument marshalling only: every step of the output layer runs in the HIP
kernels of libkbest.  PyTorch supplies device memory and the current stream.
There is no fallback: if the library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkbest.so")

KB_OK, KB_ERR_INVALID_ARG, KB_ERR_UNSUPPORTED, KB_ERR_WORKSPACE, KB_ERR_HIP = range(5)
KB_F32, KB_BF16 = 0, 1
KB_MAX_K = 16

_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t

# name -> (restype, argtypes), mirroring include/kbest.h and include/kbest_standin.h
SIGNATURES = {
    "kb_abi_version": (_I, []),
    "kb_status_string": (ctypes.c_char_p, [_I]),
    "kb_last_error": (ctypes.c_char_p, []),
    "kb_kbest_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I, _I]),
    "kb_kbest_plan": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _P]),
    "kb_kbest_step": (_I, [_I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "kb_kbest_step_events": (_I, [_I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P,
                                  _P, _P]),
    "kb_kbest_step_scratch_max": (_SZ, []),
    "kb_kbest_step_noalloc": (_I, [_I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kb_argmax_workspace_bytes": (_SZ, [_I, _I, _I, _I]),
    "kb_argmax_step": (_I, [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "kb_unfused_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I, _I]),
    "kb_kbest_step_unfused": (_I, [_I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                   _P, _I, _P]),
    "kb_beam_finish": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kb_beam_backtrace": (_I, [_I, _I, _I, ctypes.c_float, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kb_compact_workspace_bytes": (_SZ, [_I]),
    "kb_compact_batch": (_I, [_I, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "kb_compact_beams": (_I, [_I, _I, _P, _P, _P, _P, _P, _P, _P]),
    "kb_gather_rows": (_I, [_I, _P, _P, _P, _P, _SZ, _P]),
    "kb_shard_splits": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _P]),
    "kb_shard_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I]),
    "kb_shard_partials": (_I, [_I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "kb_merge_partials": (_I, [_I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    # decoder stand-in of the synthetic decode loop (include/kbest_standin.h)
    "kb_standin_alive": (_I, [_I, _P, _I, _I, _P, _P, _P, _P]),
    "kb_standin_next_h": (_I, [_I, _P, _I, _I, _I, _P, _P, _P, _P, _SZ, _P]),
    "kb_standin_step": (_I, [_I, _P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _P, _SZ, _P]),
}


class KBestError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"libkbest status {status}: {detail}")


def lib() -> ctypes.CDLL:
    """Load libkbest.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "or python -m paper_1805_09863_amd._build")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != KB_OK:
        raise KBestError(status, lib().kb_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    # a plain int: the declared argtypes (c_void_p) convert it, at a fraction
    # of the cost of building a c_void_p per pointer
    return None if t is None else t.data_ptr()


def _ptr_host(t: Optional[torch.Tensor]):
    """Address of a pinned host tensor (checked by the caller) that kernels write."""
    return None if t is None else t.data_ptr()


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(stream, device: Optional[torch.device] = None) -> int:
    """The hipStream_t to launch on: ``stream``'s, else the current stream of
    ``device`` (by default the current device), read as a raw handle without
    building a torch.cuda.Stream object."""
    if stream is None:
        if _raw_stream is not None:
            idx = device.index if device is not None and device.index is not None else torch.cuda.current_device()
            return _raw_stream(idx)
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return KB_F32
    if t.dtype == torch.bfloat16:
        return KB_BF16
    raise TypeError(f"h and W must be float32 or bfloat16, got {t.dtype}")


def _need(t: torch.Tensor, name: str, dtype=None, dim=None, numel=None):
    """Every tensor handed to the library as a pointer: on the GPU, contiguous,
    of the given type and rank, and (numel) at least that many elements."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a tensor on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if dim is not None and t.dim() != dim:
        raise ValueError(f"{name} must have {dim} dimensions")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, {numel} needed")


def _need_ws(ws: torch.Tensor, nbytes: int, name: str = "ws"):
    _need(ws, name)
    if ws.numel() * ws.element_size() < nbytes:
        raise ValueError(f"{name} has {ws.numel() * ws.element_size()} bytes, {nbytes} needed")


def _need_outs(out, names, dtypes, numel):
    if len(out) != len(names):
        raise ValueError(f"out must hold {len(names)} tensors ({', '.join(names)})")
    for t, n, d in zip(out, names, dtypes):
        _need(t, n, dtype=d, numel=numel)


def abi_version() -> int:
    return lib().kb_abi_version()


_ws_bytes_cache: dict = {}


def kbest_workspace_bytes(dtype: int, N: int, H: int, V: int, k: int, S: int) -> int:
    # a pure function of the shape (for one loaded library and tile override):
    # asked once per shape
    L = lib()
    key = (id(L), os.environ.get("KB_TILE"), dtype, N, H, V, k, S)
    n = _ws_bytes_cache.get(key)
    if n is None:
        n = _ws_bytes_cache[key] = int(L.kb_kbest_workspace_bytes(dtype, N, H, V, k, S))
    return n


KB_KERNEL_NAMES = ("few", "wide", "dma", "reg")
_PLAN_FIELDS = ("kernel", "tile_rows", "tile_words", "row_tiles", "splits", "tiles_per_split")


def kbest_plan(dtype: int, N: int, H: int, V: int, k: int, aligned: bool = True) -> dict:
    """The projection plan kbest_step chooses for this shape (kb_kbest_plan):
    kernel ("few", "wide", "dma" or "reg"), tile rows and words, row tiles,
    vocabulary splits and tiles per split.  ``aligned``: whether h, W and b
    sit at 16-byte aligned addresses (torch allocations do)."""
    esz = 2 if dtype == KB_BF16 else 4
    base = 1 << 20 if aligned else (1 << 20) + esz
    out = (ctypes.c_int32 * 6)()
    _check(lib().kb_kbest_plan(dtype, N, H, V, k, base, base, (1 << 20) if aligned else (1 << 20) + 4, out))
    plan = dict(zip(_PLAN_FIELDS, list(out)))
    plan["kernel"] = KB_KERNEL_NAMES[plan["kernel"]] if N > 0 else None
    return plan


def workspace(nbytes: int, device=None) -> torch.Tensor:
    """A device byte buffer usable as a workspace (torch allocations are 256-B aligned)."""
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device or "cuda")


def kbest_step(h: torch.Tensor, W: torch.Tensor, b: torch.Tensor, prev_score: torch.Tensor,
               sent_offsets: torch.Tensor, k: int, *, S: Optional[int] = None,
               out: Optional[tuple] = None, ws: Optional[torch.Tensor] = None,
               row_lse: Optional[torch.Tensor] = None, stream=None, events: Optional[tuple] = None):
    """One decode step of the output layer: returns (token, parent, score), each S x k.

    ``h`` is N x H, ``W`` is H x V (float32 or bfloat16, same type), ``b`` V
    float32, ``prev_score`` N float32, ``sent_offsets`` S+1 int32, all on the
    GPU.  ``out`` may supply preallocated (token, parent, score), ``ws`` a
    workspace of at least ``kbest_workspace_bytes`` bytes, ``row_lse`` an N
    float32 tensor to receive each row's log-sum-exp, ``events`` a pair of
    raw hipEvent_t handles recorded around the projection kernel.
    """
    _need(h, "h", dim=2)
    _need(W, "W", dtype=h.dtype, dim=2)
    _need(b, "b", dtype=torch.float32, dim=1)
    _need(prev_score, "prev_score", dtype=torch.float32, dim=1)
    _need(sent_offsets, "sent_offsets", dtype=torch.int32, dim=1)
    dt = _dtype_code(h)
    N, H = h.shape
    H2, V = W.shape
    if H2 != H or b.shape[0] != V or prev_score.shape[0] != N:
        raise ValueError("shape mismatch among h, W, b, prev_score")
    S = sent_offsets.shape[0] - 1 if S is None else S
    if sent_offsets.shape[0] != S + 1:
        raise ValueError("sent_offsets must have S+1 entries")
    dev = h.device
    if out is None:
        tok = torch.empty((S, k), dtype=torch.int32, device=dev)
        par = torch.empty((S, k), dtype=torch.int32, device=dev)
        sc = torch.empty((S, k), dtype=torch.float32, device=dev)
    else:
        _need_outs(out, ("token", "parent", "score"), (torch.int32, torch.int32, torch.float32), S * k)
        tok, par, sc = out
    need = kbest_workspace_bytes(dt, N, H, V, k, S)
    if ws is None:
        ws = workspace(need, dev)
    _need_ws(ws, need)
    if row_lse is not None:
        _need(row_lse, "row_lse", dtype=torch.float32, numel=N)
    L = lib()
    args = [dt, N, H, V, k, S, _ptr(h), _ptr(W), _ptr(b), _ptr(prev_score), _ptr(sent_offsets),
            _ptr(tok), _ptr(par), _ptr(sc), _ptr(row_lse), _ptr(ws), ws.numel() * ws.element_size(),
            _stream(stream, dev)]
    if events is None:
        _check(L.kb_kbest_step(*args))
    else:
        _check(L.kb_kbest_step_events(*args, ctypes.c_void_p(events[0]), ctypes.c_void_p(events[1])))
    return tok, par, sc


def kbest_step_noalloc(h: torch.Tensor, W: torch.Tensor, b: torch.Tensor, prev_score: torch.Tensor,
                       sent_offsets: torch.Tensor, k: int, *, out: tuple, S: Optional[int] = None,
                       row_lse: Optional[torch.Tensor] = None, stream=None):
    """kbest_step without a workspace (include/kbest.h, kb_kbest_step_noalloc): the
    library's fixed per-device scratch array takes the partials, so nothing is
    allocated, here or in the library; ``out`` = (token, parent, score) must be given."""
    _need(h, "h", dim=2)
    _need(W, "W", dtype=h.dtype, dim=2)
    _need(b, "b", dtype=torch.float32, dim=1)
    _need(prev_score, "prev_score", dtype=torch.float32, dim=1)
    _need(sent_offsets, "sent_offsets", dtype=torch.int32, dim=1)
    dt = _dtype_code(h)
    N, H = h.shape
    H2, V = W.shape
    if H2 != H or b.shape[0] != V or prev_score.shape[0] != N:
        raise ValueError("shape mismatch among h, W, b, prev_score")
    S = sent_offsets.shape[0] - 1 if S is None else S
    if sent_offsets.shape[0] != S + 1:
        raise ValueError("sent_offsets must have S+1 entries")
    _need_outs(out, ("token", "parent", "score"), (torch.int32, torch.int32, torch.float32), S * k)
    if row_lse is not None:
        _need(row_lse, "row_lse", dtype=torch.float32, numel=N)
    tok, par, sc = out
    _check(lib().kb_kbest_step_noalloc(dt, N, H, V, k, S, _ptr(h), _ptr(W), _ptr(b), _ptr(prev_score),
                                       _ptr(sent_offsets), _ptr(tok), _ptr(par), _ptr(sc), _ptr(row_lse),
                                       _stream(stream)))
    return tok, par, sc


def argmax_workspace_bytes(dtype: int, N: int, H: int, V: int) -> int:
    return int(lib().kb_argmax_workspace_bytes(dtype, N, H, V))


def argmax_step(h: torch.Tensor, W: torch.Tensor, b: torch.Tensor, *, out: Optional[tuple] = None,
                ws: Optional[torch.Tensor] = None, stream=None):
    """Greedy (beam 1) step (Algorithms 5 and 6): returns (token[N] int32, logit[N] float32),
    the best word of every row of h @ W + b and its raw score, without a softmax."""
    _need(h, "h", dim=2)
    _need(W, "W", dtype=h.dtype, dim=2)
    _need(b, "b", dtype=torch.float32, dim=1)
    dt = _dtype_code(h)
    N, H = h.shape
    H2, V = W.shape
    if H2 != H or b.shape[0] != V:
        raise ValueError("shape mismatch among h, W, b")
    if out is None:
        tok = torch.empty(N, dtype=torch.int32, device=h.device)
        val = torch.empty(N, dtype=torch.float32, device=h.device)
    else:
        _need_outs(out, ("token", "logit"), (torch.int32, torch.float32), N)
        tok, val = out
    need = argmax_workspace_bytes(dt, N, H, V)
    if ws is None:
        ws = workspace(need, h.device)
    _need_ws(ws, need)
    _check(lib().kb_argmax_step(dt, N, H, V, _ptr(h), _ptr(W), _ptr(b), _ptr(tok), _ptr(val), _ptr(ws),
                                ws.numel() * ws.element_size(), _stream(stream)))
    return tok, val


def unfused_workspace_bytes(dtype: int, N: int, H: int, V: int, k: int, S: int) -> int:
    return int(lib().kb_unfused_workspace_bytes(dtype, N, H, V, k, S))


def kbest_step_unfused(h: torch.Tensor, W: torch.Tensor, b: torch.Tensor, prev_score: torch.Tensor,
                       sent_offsets: torch.Tensor, k: int, *, mode: int = 0, out: Optional[tuple] = None,
                       ws: Optional[torch.Tensor] = None, row_lse: Optional[torch.Tensor] = None,
                       events: Optional[list] = None, stream=None):
    """The unfused baseline of kbest_step (mode 0: Algorithm 3; mode 1: Algorithm 4
    over stored scores); ``events`` is a list of raw hipEvent_t handles recorded
    at the stage boundaries (see include/kbest.h)."""
    _need(h, "h", dim=2)
    _need(W, "W", dtype=h.dtype, dim=2)
    _need(b, "b", dtype=torch.float32, dim=1)
    _need(prev_score, "prev_score", dtype=torch.float32, dim=1)
    _need(sent_offsets, "sent_offsets", dtype=torch.int32, dim=1)
    dt = _dtype_code(h)
    N, H = h.shape
    V = W.shape[1]
    S = sent_offsets.shape[0] - 1
    if out is None:
        out = tuple(torch.empty((S, k), dtype=t, device=h.device)
                    for t in (torch.int32, torch.int32, torch.float32))
    _need_outs(out, ("token", "parent", "score"), (torch.int32, torch.int32, torch.float32), S * k)
    tok, par, sc = out
    need = unfused_workspace_bytes(dt, N, H, V, k, S)
    if ws is None:
        ws = workspace(need, h.device)
    _need_ws(ws, need)
    if row_lse is not None:
        _need(row_lse, "row_lse", dtype=torch.float32, numel=N)
    ev = None
    if events:
        ev = (ctypes.c_void_p * len(events))(*[ctypes.c_void_p(e) for e in events])
    _check(lib().kb_kbest_step_unfused(mode, dt, N, H, V, k, S, _ptr(h), _ptr(W), _ptr(b), _ptr(prev_score),
                                       _ptr(sent_offsets), _ptr(tok), _ptr(par), _ptr(sc), _ptr(row_lse),
                                       _ptr(ws), ws.numel() * ws.element_size(), ev,
                                       len(events) if events else 0, _stream(stream)))
    return tok, par, sc


def compact_workspace_bytes(M: int) -> int:
    return int(lib().kb_compact_workspace_bytes(M))


def compact_batch(alive: torch.Tensor, entry_sentence: Optional[torch.Tensor] = None, *,
                  out: Optional[tuple] = None, ws: Optional[torch.Tensor] = None, stream=None):
    """Stable removal of finished entries from a batch of M entries (Algorithm 2).

    ``alive`` is M uint8 on the GPU; ``entry_sentence`` (optional) M int32,
    the non-decreasing sentence id of every entry.  Returns device tensors
    (keep_idx[M], kept_count[1], new_sent_offsets, new_S[1]); only the first
    kept_count / new_S + 1 entries are meaningful.  Without entry_sentence the
    last two are None.  ``out`` may supply (keep_idx, kept_count,
    new_sent_offsets, new_S); new_sent_offsets needs one more entry than
    entry_sentence has distinct ids (M + 1 always suffices).
    """
    _need(alive, "alive", dtype=torch.uint8, dim=1)
    M = alive.numel()
    dev = alive.device
    if entry_sentence is not None:
        _need(entry_sentence, "entry_sentence", dtype=torch.int32, dim=1, numel=M)
    if out is None:
        keep = torch.empty(max(M, 1), dtype=torch.int32, device=dev)
        kept = torch.empty(1, dtype=torch.int32, device=dev)
        noff = torch.empty(M + 1, dtype=torch.int32, device=dev) if entry_sentence is not None else None
        nS = torch.empty(1, dtype=torch.int32, device=dev) if entry_sentence is not None else None
    else:
        keep, kept, noff, nS = out
        _need(keep, "keep_idx", dtype=torch.int32, numel=M)
        _need(kept, "kept_count", dtype=torch.int32, numel=1)
        if noff is not None:
            _need(noff, "new_sent_offsets", dtype=torch.int32, numel=1)
        if nS is not None:
            _need(nS, "new_S", dtype=torch.int32, numel=1)
    need = compact_workspace_bytes(M)
    if ws is None and need > 0:
        ws = workspace(need, dev)
    if ws is not None:
        _need_ws(ws, need)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().kb_compact_batch(M, _ptr(alive), _ptr(keep), _ptr(kept), _ptr(entry_sentence), _ptr(noff),
                                  _ptr(nS), _ptr(ws), nbytes, _stream(stream)))
    return keep, kept, noff, nS


def compact_beams(alive: torch.Tensor, S: int, k: int, *, out: Optional[tuple] = None, stream=None):
    """Stable removal of finished entries from the S x k output of a step (Algorithm 2).

    ``alive`` is S*k uint8 on the GPU.  Returns device tensors
    (keep_idx[S*k], kept_count[1], new_sent_offsets[S+1], kept_sentence[S], new_S[1]);
    only the first kept_count / new_S (+1) entries are meaningful.
    """
    _need(alive, "alive", dtype=torch.uint8)
    if alive.numel() != S * k:
        raise ValueError("alive must have S*k entries")
    dev = alive.device
    if out is None:
        keep = torch.empty(max(S * k, 1), dtype=torch.int32, device=dev)
        kept = torch.empty(1, dtype=torch.int32, device=dev)
        noff = torch.empty(S + 1, dtype=torch.int32, device=dev)
        ksent = torch.empty(max(S, 1), dtype=torch.int32, device=dev)
        nS = torch.empty(1, dtype=torch.int32, device=dev)
    else:
        keep, kept, noff, ksent, nS = out
        _need(keep, "keep_idx", dtype=torch.int32, numel=S * k)
        _need(kept, "kept_count", dtype=torch.int32, numel=1)
        if noff is not None:
            _need(noff, "new_sent_offsets", dtype=torch.int32, numel=S + 1)
        if ksent is not None:
            _need(ksent, "kept_sentence", dtype=torch.int32, numel=S)
        if nS is not None:
            _need(nS, "new_S", dtype=torch.int32, numel=1)
    _check(lib().kb_compact_beams(S, k, _ptr(alive), _ptr(keep), _ptr(kept), _ptr(noff), _ptr(ksent),
                                  _ptr(nS), _stream(stream)))
    return keep, kept, noff, ksent, nS


def gather_rows(src: torch.Tensor, idx: torch.Tensor, *, n_dev: Optional[torch.Tensor] = None,
                n_max: Optional[int] = None, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """out[i] = src[idx[i]] for i < min(n_max, n_dev[0]) (rows of src along dim 0)."""
    _need(src, "src")
    n_max = idx.shape[0] if n_max is None else n_max
    _need(idx, "idx", dtype=torch.int32, dim=1, numel=n_max)
    if n_dev is not None:
        _need(n_dev, "n_dev", dtype=torch.int32, numel=1)
    row_bytes = src[0].numel() * src.element_size() if src.shape[0] > 0 else 0
    if out is None:
        out = torch.empty((n_max,) + tuple(src.shape[1:]), dtype=src.dtype, device=src.device)
    _need(out, "out", dtype=src.dtype, numel=n_max * (src[0].numel() if src.shape[0] > 0 else 0))
    if n_max == 0:
        return out
    _check(lib().kb_gather_rows(n_max, _ptr(n_dev), _ptr(idx), _ptr(src), _ptr(out), row_bytes,
                                _stream(stream)))
    return out


# ---------------------------------------------------------------- decoder stand-in
def shard_splits(h: torch.Tensor, W_shard: torch.Tensor, b_shard: torch.Tensor, k: int) -> int:
    """Number of vocabulary splits shard_partials writes for these operands."""
    N, H = h.shape
    out = ctypes.c_int(0)
    _check(lib().kb_shard_splits(_dtype_code(h), N, H, W_shard.shape[1], k, _ptr(h), _ptr(W_shard), _ptr(b_shard),
                                 ctypes.byref(out)))
    return int(out.value)


def shard_partials(h: torch.Tensor, W_shard: torch.Tensor, b_shard: torch.Tensor, k: int, word_base: int,
                   stats: torch.Tensor, lists: torch.Tensor, *, ws: Optional[torch.Tensor] = None, stream=None):
    """One vocabulary shard's fused projection (see include/kbest.h): its splits'
    statistics into ``stats`` (splits x N x 2 float32) and k-best lists into
    ``lists`` (splits x N x k x 2 int32, global words), normally slices of the
    combined arrays that merge_partials reduces."""
    _need(h, "h", dim=2)
    _need(W_shard, "W_shard", dtype=h.dtype, dim=2)
    _need(b_shard, "b_shard", dtype=torch.float32, dim=1)
    _need(stats, "stats", dtype=torch.float32)
    _need(lists, "lists", dtype=torch.int32)
    N, H = h.shape
    if W_shard.shape[0] != H or b_shard.shape[0] != W_shard.shape[1]:
        raise ValueError("shape mismatch among h, W_shard, b_shard")
    V_shard = W_shard.shape[1]
    P = shard_splits(h, W_shard, b_shard, k)
    if stats.numel() < P * N * 2 or lists.numel() < P * N * k * 2:
        raise ValueError(f"stats / lists too small for {P} splits")
    dt = _dtype_code(h)
    need = int(lib().kb_shard_workspace_bytes(dt, N, H, V_shard, k))
    if ws is None:
        ws = workspace(need, h.device)
    _need_ws(ws, need)
    _check(lib().kb_shard_partials(dt, N, H, V_shard, word_base, k, _ptr(h), _ptr(W_shard), _ptr(b_shard),
                                   _ptr(stats), _ptr(lists), _ptr(ws), ws.numel() * ws.element_size(),
                                   _stream(stream)))
    return P


def merge_partials(stats: torch.Tensor, lists: torch.Tensor, P: int, V: int, k: int, prev_score: torch.Tensor,
                   sent_offsets: torch.Tensor, *, out: Optional[tuple] = None,
                   row_lse: Optional[torch.Tensor] = None, stream=None):
    """Reduce the combined partials of all shards (P splits in total) and merge the
    beam: returns (token, parent, score), each S x k, as kbest_step does."""
    _need(stats, "stats", dtype=torch.float32)
    _need(lists, "lists", dtype=torch.int32)
    _need(prev_score, "prev_score", dtype=torch.float32, dim=1)
    _need(sent_offsets, "sent_offsets", dtype=torch.int32, dim=1)
    N = prev_score.shape[0]
    S = sent_offsets.shape[0] - 1
    if stats.numel() < P * N * 2 or lists.numel() < P * N * k * 2:
        raise ValueError(f"stats / lists too small for {P} splits")
    if out is None:
        out = tuple(torch.empty((S, k), dtype=t, device=prev_score.device)
                    for t in (torch.int32, torch.int32, torch.float32))
    _need_outs(out, ("token", "parent", "score"), (torch.int32, torch.int32, torch.float32), S * k)
    tok, par, sc = out
    if row_lse is not None:
        _need(row_lse, "row_lse", dtype=torch.float32, numel=N)
    _check(lib().kb_merge_partials(N, V, k, S, P, _ptr(stats), _ptr(lists), _ptr(prev_score), _ptr(sent_offsets),
                                   _ptr(tok), _ptr(par), _ptr(sc), _ptr(row_lse), _stream(stream)))
    return tok, par, sc


def standin_alive(sid: torch.Tensor, lengths: torch.Tensor, S: int, k: int, t: int, *, out: torch.Tensor,
                  S_dev: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """out[s*k + r] = (s < min(S, S_dev[0]) and t < lengths[sid[s]] - 1) for s < S
    (include/kbest_standin.h)."""
    _need(sid, "sid", dtype=torch.int32, numel=S)
    _need(lengths, "lengths", dtype=torch.int32)
    _need(out, "out", dtype=torch.uint8, numel=S * k)
    if S_dev is not None:
        _need(S_dev, "S_dev", dtype=torch.int32, numel=1)
    _check(lib().kb_standin_alive(S, _ptr(S_dev), k, t, _ptr(sid), _ptr(lengths), _ptr(out), _stream(stream)))
    return out


def standin_step(sid: torch.Tensor, lengths: torch.Tensor, score: torch.Tensor, S: int, k: int, t: int, *,
                 out: tuple, S_dev: Optional[torch.Tensor] = None, alive: Optional[torch.Tensor] = None,
                 counts_host: Optional[torch.Tensor] = None, next_state: Optional[tuple] = None, stream=None):
    """The loop step's bookkeeping in one launch (include/kbest_standin.h): the
    EOS mask, its compaction and the gathers of the surviving scores and sentence
    ids.  ``out`` = (keep_idx[S*k], counts[2], new_sent_offsets[S+1],
    prev_next[S*k] float32, sid_next[S]); returns it.  ``counts_host``, a pinned
    int32 host tensor of 3, receives the counts too, then the tag t + 1 (a host
    that polls [2] may read [0] and [1] once the tag is there).  ``next_state`` = (table, T, next_h): the surviving
    entries' states of step t + 1 gathered into next_h (rows x H, like table)
    in the same launch."""
    keep, counts, noff, prev_next, sid_next = out
    _need(sid, "sid", dtype=torch.int32, numel=S)
    _need(lengths, "lengths", dtype=torch.int32)
    _need(score, "score", dtype=torch.float32, numel=S * k)
    _need(keep, "keep_idx", dtype=torch.int32, numel=S * k)
    _need(counts, "counts", dtype=torch.int32, numel=2)
    _need(noff, "new_sent_offsets", dtype=torch.int32, numel=S + 1)
    _need(prev_next, "prev_next", dtype=torch.float32, numel=S * k)
    _need(sid_next, "sid_next", dtype=torch.int32, numel=S)
    if S_dev is not None:
        _need(S_dev, "S_dev", dtype=torch.int32, numel=1)
    if alive is not None:
        _need(alive, "alive", dtype=torch.uint8, numel=S * k)
    if counts_host is not None:
        if not isinstance(counts_host, torch.Tensor) or counts_host.is_cuda or not counts_host.is_pinned():
            raise TypeError("counts_host must be a pinned host tensor")
        if counts_host.dtype != torch.int32 or counts_host.numel() < 3 or not counts_host.is_contiguous():
            raise ValueError("counts_host must be 3 contiguous int32")
    table = next_h = None
    T, row_bytes = 0, 0
    if next_state is not None:
        table, T, next_h = next_state
        _need(table, "table", dim=2)
        _need(next_h, "next_h", dtype=table.dtype, numel=S * k * table.shape[1])
        row_bytes = table.shape[1] * table.element_size()
    _check(lib().kb_standin_step(S, _ptr(S_dev), k, t, _ptr(sid), _ptr(lengths), _ptr(score), _ptr(keep),
                                 _ptr(counts), _ptr(noff), _ptr(prev_next), _ptr(sid_next), _ptr(alive),
                                 _ptr_host(counts_host), _ptr(table), T, _ptr(next_h), row_bytes,
                                 _stream(stream)))
    return out


def standin_next_h(table: torch.Tensor, keep: torch.Tensor, sid: torch.Tensor, k: int, T: int, t: int,
                   n_max: int, *, n_dev: Optional[torch.Tensor] = None, out: torch.Tensor, stream=None):
    """out[i] = table[(sid[keep[i] // k] * T + t) * k + keep[i] % k] for i < min(n_max, n_dev[0])."""
    _need(table, "table")
    _need(keep, "keep", dtype=torch.int32, numel=n_max)
    _need(sid, "sid", dtype=torch.int32)
    _need(out, "out", dtype=table.dtype, numel=n_max * table[0].numel())
    if n_dev is not None:
        _need(n_dev, "n_dev", dtype=torch.int32, numel=1)
    row_bytes = table[0].numel() * table.element_size()
    _check(lib().kb_standin_next_h(n_max, _ptr(n_dev), k, T, t, _ptr(keep), _ptr(sid), _ptr(table), _ptr(out),
                                   row_bytes, _stream(stream)))
    return out


# ---------------------------------------------------------------- per-hypothesis EOS
def beam_finish(S: int, k: int, t: int, T: int, eos: int, token, parent, score, sent_id, beam, prev_keep,
                prev_hist_base: int, hist_base: int, hist_token, hist_parent, fin: tuple, alive, stream=None):
    """After a step: take each sentence's first beam[s] continuations, record the step's
    history, move EOS (or last-step) continuations to the finished store ``fin`` =
    (count, score, len, hist), shrink the beams and fill ``alive`` (include/kbest.h)."""
    fc, fs, fl, fh = fin
    n = S * k
    for x, nm, d, m in ((token, "token", torch.int32, n), (parent, "parent", torch.int32, n),
                        (score, "score", torch.float32, n), (sent_id, "sent_id", torch.int32, S),
                        (beam, "beam", torch.int32, S), (hist_token, "hist_token", torch.int32, hist_base + n),
                        (hist_parent, "hist_parent", torch.int32, hist_base + n),
                        (fc, "fin_count", torch.int32, S), (alive, "alive", torch.uint8, n)):
        _need(x, nm, dtype=d, numel=m)
    S0 = fc.numel()             # the finished store holds k slots per original sentence
    for x, nm, d in ((fs, "fin_score", torch.float32), (fl, "fin_len", torch.int32), (fh, "fin_hist", torch.int32)):
        _need(x, nm, dtype=d, numel=S0 * k)
    if prev_keep is not None:
        _need(prev_keep, "prev_keep", dtype=torch.int32, numel=S)
    _check(lib().kb_beam_finish(S, k, t, T, eos, _ptr(token), _ptr(parent), _ptr(score), _ptr(sent_id), _ptr(beam),
                                _ptr(prev_keep), prev_hist_base, hist_base, _ptr(hist_token), _ptr(hist_parent),
                                _ptr(fc), _ptr(fs), _ptr(fl), _ptr(fh), _ptr(alive), _stream(stream)))


def beam_backtrace(S0: int, k: int, T: int, alpha: float, fin: tuple, hist_token, hist_parent, *, out=None,
                   stream=None):
    """Best finished hypothesis of every sentence by score / len**alpha, and its tokens:
    returns (tokens[S0, T], len[S0], score[S0], normalised score[S0])."""
    fc, fs, fl, fh = fin
    dev = fc.device
    if out is None:
        out = (torch.empty((S0, T), dtype=torch.int32, device=dev), torch.empty(S0, dtype=torch.int32, device=dev),
               torch.empty(S0, dtype=torch.float32, device=dev), torch.empty(S0, dtype=torch.float32, device=dev))
    for x, nm_, d in ((fc, "fin_count", torch.int32), (fs, "fin_score", torch.float32),
                      (fl, "fin_len", torch.int32), (fh, "fin_hist", torch.int32)):
        _need(x, nm_, dtype=d, numel=S0 * (1 if nm_ == "fin_count" else k))
    _need(hist_token, "hist_token", dtype=torch.int32)
    _need(hist_parent, "hist_parent", dtype=torch.int32)
    _need_outs(out[:1], ("tokens",), (torch.int32,), S0 * T)
    _need_outs(out[1:], ("len", "score", "norm"), (torch.int32, torch.float32, torch.float32), S0)
    toks, ln, sc, nm = out
    _check(lib().kb_beam_backtrace(S0, k, T, float(alpha), _ptr(fc), _ptr(fs), _ptr(fl), _ptr(fh), _ptr(hist_token),
                                   _ptr(hist_parent), _ptr(toks), _ptr(ln), _ptr(sc), _ptr(nm), _stream(stream)))
    return toks, ln, sc, nm
