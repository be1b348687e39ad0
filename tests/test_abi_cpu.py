"""The C ABI on the host: loading, exported symbols and argument validation.

Every call here returns before any HIP work is enqueued, so no GPU is needed.
"""
import ctypes
import glob
import os
import re

import pytest

kb = pytest.importorskip("paper_1805_09863_amd")
from paper_1805_09863_amd import binding  # noqa: E402

KB_OK, KB_ERR_INVALID_ARG, KB_ERR_UNSUPPORTED, KB_ERR_WORKSPACE = 0, 1, 2, 3
FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first


def _header_functions(repo_root):
    names = set()
    for h in sorted(glob.glob(os.path.join(repo_root, "include", "*.h"))):
        with open(h) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(kb_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function(repo_root):
    L = binding.lib()
    names = _header_functions(repo_root)
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/*.h but not exported"
    assert set(names) == set(binding.SIGNATURES), "binding signatures out of sync with include/*.h"


def test_standin_argument_checks():
    L = binding.lib()
    assert L.kb_standin_alive(0, None, 5, 0, None, None, None, None) == KB_OK            # empty batch: no-op
    assert L.kb_standin_alive(-1, None, 5, 0, FAKE, FAKE, FAKE, None) == KB_ERR_INVALID_ARG
    assert L.kb_standin_alive(3, None, 0, 0, FAKE, FAKE, FAKE, None) == KB_ERR_INVALID_ARG
    assert L.kb_standin_alive(3, None, 5, 0, None, FAKE, FAKE, None) == KB_ERR_INVALID_ARG
    assert L.kb_standin_alive(1 << 30, None, 4, 0, FAKE, FAKE, FAKE, None) == KB_ERR_UNSUPPORTED
    nh = L.kb_standin_next_h
    assert nh(0, None, 5, 60, 1, FAKE, FAKE, FAKE, FAKE, 2048, None) == KB_OK        # nothing to gather
    assert nh(4, None, 5, 60, 60, FAKE, FAKE, FAKE, FAKE, 2048, None) == KB_ERR_INVALID_ARG   # t >= T
    assert nh(4, None, 5, 60, -1, FAKE, FAKE, FAKE, FAKE, 2048, None) == KB_ERR_INVALID_ARG
    assert nh(4, None, 5, 60, 1, FAKE, FAKE, FAKE, FAKE, 6, None) == KB_ERR_INVALID_ARG       # row bytes % 4
    assert nh(4, None, 5, 60, 1, None, FAKE, FAKE, FAKE, 2048, None) == KB_ERR_INVALID_ARG
    assert nh(4, None, 5, 60, 1, FAKE, FAKE, ctypes.c_void_p(0x1002), FAKE, 2048, None) == KB_ERR_INVALID_ARG


def test_standin_step_argument_checks():
    L = binding.lib()
    # no host copy of the counts, no state gather
    st = lambda *a: L.kb_standin_step(*a[:13], None, None, 0, None, 0, a[13])   # noqa: E731
    F = FAKE
    assert st(-1, None, 5, 0, F, F, F, F, F, F, F, F, None, None) == KB_ERR_INVALID_ARG
    assert st(3, None, 0, 0, F, F, F, F, F, F, F, F, None, None) == KB_ERR_INVALID_ARG
    assert st(3, None, 1024, 0, F, F, F, F, F, F, F, F, None, None) == KB_ERR_UNSUPPORTED      # k >= 1024
    assert st(1 << 30, None, 4, 0, F, F, F, F, F, F, F, F, None, None) == KB_ERR_UNSUPPORTED
    for i in range(4, 12):                      # each required pointer in turn
        args = [3, None, 5, 0] + [F] * 8 + [None, None]
        args[i] = None
        assert st(*args) == KB_ERR_INVALID_ARG, f"argument {i} may not be null"
    # with the next states: (table, T, next_h, row_bytes)
    nx = lambda t, table, T, nh, rb: L.kb_standin_step(3, None, 5, t, F, F, F, F, F, F, F, F, None, None,  # noqa: E731
                                                       table, T, nh, rb, None)
    assert nx(0, None, 60, F, 2048) == KB_ERR_INVALID_ARG                      # no table
    assert nx(59, F, 60, F, 2048) == KB_ERR_INVALID_ARG                        # t + 1 == T: no next step
    assert nx(-1, F, 60, F, 2048) == KB_ERR_INVALID_ARG
    assert nx(0, F, 60, F, 6) == KB_ERR_INVALID_ARG                            # row bytes % 4
    assert nx(0, F, 60, F, 0) == KB_ERR_INVALID_ARG
    assert nx(0, F, 60, ctypes.c_void_p(0x1002), 2048) == KB_ERR_INVALID_ARG   # misaligned next_h


def test_abi_version_and_status_strings():
    L = binding.lib()
    assert L.kb_abi_version() == 2
    for s in range(5):
        assert L.kb_status_string(s)
    assert L.kb_status_string(99) == b"unknown status"


def test_workspace_bytes():
    L = binding.lib()
    big = L.kb_kbest_workspace_bytes(1, 3072, 1024, 90000, 12, 256)
    # partials are far smaller than the N x V float32 scores they replace
    assert 0 < big < 3072 * 90000 * 4 // 50
    assert big % 256 == 0
    assert L.kb_kbest_workspace_bytes(1, 3072, 1024, 90000, 12, 256) == big   # deterministic
    assert L.kb_kbest_workspace_bytes(0, 0, 16, 100, 5, 0) == 0
    assert L.kb_kbest_workspace_bytes(0, 5, 16, 100, 0, 1) == 0                # invalid k


def _step(L, dtype=0, N=10, H=16, V=100, k=5, S=2, ptr=FAKE, ws=FAKE, ws_bytes=1 << 30, null_out=False):
    out = None if null_out else ptr
    return L.kb_kbest_step(dtype, N, H, V, k, S, ptr, ptr, ptr, ptr, ptr, out, out, out, None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), KB_ERR_INVALID_ARG),
    (dict(k=0), KB_ERR_INVALID_ARG),
    (dict(k=17), KB_ERR_INVALID_ARG),
    (dict(V=4, k=5), KB_ERR_INVALID_ARG),
    (dict(N=1, S=2), KB_ERR_INVALID_ARG),
    (dict(N=-1), KB_ERR_INVALID_ARG),
    (dict(N=0, S=1), KB_ERR_INVALID_ARG),
    (dict(H=0), KB_ERR_INVALID_ARG),
    (dict(ptr=None), KB_ERR_INVALID_ARG),
    (dict(null_out=True), KB_ERR_INVALID_ARG),
    (dict(ws=None), KB_ERR_WORKSPACE),
    (dict(ws_bytes=16), KB_ERR_WORKSPACE),
    (dict(ws=ctypes.c_void_p(0x1010)), KB_ERR_WORKSPACE),
    (dict(dtype=1, ptr=ctypes.c_void_p(0x1001)), KB_ERR_INVALID_ARG),
])
def test_kbest_step_validation(kw, status):
    L = binding.lib()
    assert _step(L, **kw) == status
    assert L.kb_last_error()


def test_empty_batch_is_noop():
    L = binding.lib()
    assert _step(L, N=0, S=0, ptr=None, ws=None, ws_bytes=0) == KB_OK
    assert L.kb_last_error() == b""


def test_compact_beams_validation():
    L = binding.lib()
    assert L.kb_compact_beams(-1, 5, FAKE, FAKE, FAKE, None, None, None, None) == KB_ERR_INVALID_ARG
    assert L.kb_compact_beams(4, 0, FAKE, FAKE, FAKE, None, None, None, None) == KB_ERR_INVALID_ARG
    assert L.kb_compact_beams(4, 5, None, FAKE, FAKE, None, None, None, None) == KB_ERR_INVALID_ARG
    assert L.kb_compact_beams(4, 5, FAKE, FAKE, None, None, None, None, None) == KB_ERR_INVALID_ARG
    assert L.kb_compact_beams(1 << 30, 8, FAKE, FAKE, FAKE, None, None, None, None) == KB_ERR_UNSUPPORTED


def test_compact_batch_validation_and_workspace():
    L = binding.lib()
    # one workgroup up to 16,384 entries: no workspace; beyond, two counts per
    # 4,096 entries and two totals, rounded to 256 bytes
    assert L.kb_compact_workspace_bytes(0) == 0
    assert L.kb_compact_workspace_bytes(16384) == 0
    assert L.kb_compact_workspace_bytes(16385) == 256
    assert L.kb_compact_workspace_bytes(1 << 24) == ((2 * 4096 + 2) * 4 + 255) // 256 * 256
    cb = L.kb_compact_batch   # (M, alive, keep, kept, es, new_off, new_S, ws, ws_bytes, stream)
    assert cb(-1, FAKE, FAKE, FAKE, None, None, None, None, 0, None) == KB_ERR_INVALID_ARG
    assert cb(10, None, FAKE, FAKE, None, None, None, None, 0, None) == KB_ERR_INVALID_ARG
    assert cb(10, FAKE, None, FAKE, None, None, None, None, 0, None) == KB_ERR_INVALID_ARG
    assert cb(10, FAKE, FAKE, None, None, None, None, None, 0, None) == KB_ERR_INVALID_ARG
    # sentence outputs need the entries' sentence ids
    assert cb(10, FAKE, FAKE, FAKE, None, FAKE, None, None, 0, None) == KB_ERR_INVALID_ARG
    assert cb(10, FAKE, FAKE, FAKE, None, None, FAKE, None, 0, None) == KB_ERR_INVALID_ARG
    # past one workgroup the workspace is required and checked
    assert cb(20000, FAKE, FAKE, FAKE, None, None, None, None, 0, None) == KB_ERR_WORKSPACE
    assert cb(20000, FAKE, FAKE, FAKE, None, None, None, FAKE, 16, None) == KB_ERR_WORKSPACE
    assert cb(20000, FAKE, FAKE, FAKE, None, None, None, ctypes.c_void_p(0x1002), 1 << 20, None) == KB_ERR_WORKSPACE
    assert L.kb_last_error()


def test_size_limits_are_reported_unsupported():
    L = binding.lib()
    # a sentence's flat index (row * V + word) must be an int32
    assert _step(L, dtype=1, N=23861, H=128, V=90000, k=5, S=1) == KB_ERR_UNSUPPORTED
    assert b"INT_MAX" in L.kb_last_error()
    assert L.kb_kbest_workspace_bytes(1, 23861, 128, 90000, 5, 1) == 0
    # h of 4 GiB or more (32-bit byte offsets)
    assert _step(L, dtype=1, N=1 << 20, H=2048, V=16, k=5, S=1) == KB_ERR_UNSUPPORTED
    assert _step(L, dtype=0, N=1 << 20, H=1024, V=16, k=5, S=1) == KB_ERR_UNSUPPORTED
    mp = L.kb_merge_partials
    assert mp(23861, 90000, 5, 1, 4, *([FAKE] * 7), None, None) == KB_ERR_UNSUPPORTED


def test_gather_validation():
    L = binding.lib()
    assert L.kb_gather_rows(-1, None, FAKE, FAKE, FAKE, 16, None) == KB_ERR_INVALID_ARG
    assert L.kb_gather_rows(4, None, FAKE, FAKE, FAKE, 6, None) == KB_ERR_INVALID_ARG
    assert L.kb_gather_rows(4, None, None, FAKE, FAKE, 16, None) == KB_ERR_INVALID_ARG
    assert L.kb_gather_rows(4, None, FAKE, ctypes.c_void_p(0x1002), FAKE, 16, None) == KB_ERR_INVALID_ARG
    assert L.kb_gather_rows(0, None, None, None, None, 16, None) == KB_OK


def test_argmax_and_unfused_argument_checks():
    L = binding.lib()
    # greedy step
    assert L.kb_argmax_workspace_bytes(1, 0, 16, 100) == 0
    assert L.kb_argmax_workspace_bytes(1, 10, 128, 1000) > 0
    assert L.kb_argmax_step(7, 10, 128, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == KB_ERR_INVALID_ARG
    assert L.kb_argmax_step(1, 0, 128, 1000, None, None, None, None, None, None, 0, None) == KB_OK
    assert L.kb_argmax_step(1, 10, 128, 1000, FAKE, FAKE, FAKE, None, FAKE, FAKE, 1 << 30, None) == KB_ERR_INVALID_ARG
    assert L.kb_argmax_step(1, 10, 128, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == KB_ERR_WORKSPACE
    # unfused baseline
    assert L.kb_unfused_workspace_bytes(1, 3072, 1024, 90000, 12, 256) >= 3072 * 90000 * 4
    assert L.kb_unfused_workspace_bytes(0, 64, 128, 1000, 5, 8) == 0          # float32: not supported
    args = [FAKE] * 10 + [1 << 40, None, 0, None]
    assert L.kb_kbest_step_unfused(2, 1, 10, 128, 1000, 5, 2, *args) == KB_ERR_INVALID_ARG   # mode
    assert L.kb_kbest_step_unfused(0, 1, 10, 100, 1000, 5, 2, *args) == KB_ERR_UNSUPPORTED   # H % 128
    assert L.kb_kbest_step_unfused(0, 1, 10, 128, 200, 5, 2, *args) == KB_ERR_UNSUPPORTED    # V < 256
    small = [FAKE] * 10 + [64, None, 0, None]
    assert L.kb_kbest_step_unfused(1, 1, 10, 128, 1000, 5, 2, *small) == KB_ERR_WORKSPACE
    assert L.kb_kbest_step_unfused(0, 1, 0, 128, 1000, 5, 0, *args) == KB_OK                 # empty batch


def test_beam_argument_checks():
    L = binding.lib()
    P = [FAKE] * 3
    # kb_beam_finish(S, k, t, T, eos, token, parent, score, sid, beam, prev_keep, prev_base, base, ...)
    fin = [FAKE] * 4
    ok_tail = [FAKE, FAKE, None, 0, 0, FAKE, FAKE] + fin + [FAKE, None]   # sid, beam, prev_keep, bases, ...
    assert L.kb_beam_finish(0, 4, 0, 10, 3, *P, *ok_tail) == KB_OK                            # empty batch
    assert L.kb_beam_finish(5, 0, 0, 10, 3, *P, *ok_tail) == KB_ERR_INVALID_ARG               # k
    assert L.kb_beam_finish(5, 17, 0, 10, 3, *P, *ok_tail) == KB_ERR_INVALID_ARG              # k > 16
    assert L.kb_beam_finish(5, 4, 10, 10, 3, *P, *ok_tail) == KB_ERR_INVALID_ARG              # t >= T
    bad = [FAKE, FAKE, None, 0, 0, None, FAKE] + fin + [FAKE, None]
    assert L.kb_beam_finish(5, 4, 0, 10, 3, *P, *bad) == KB_ERR_INVALID_ARG                   # null history
    neg = [FAKE, FAKE, None, 0, -1, FAKE, FAKE] + fin + [FAKE, None]
    assert L.kb_beam_finish(5, 4, 0, 10, 3, *P, *neg) == KB_ERR_INVALID_ARG                   # base < 0
    out = [FAKE] * 4
    assert L.kb_beam_backtrace(0, 4, 10, 1.0, *fin, FAKE, FAKE, *out, None) == KB_OK
    assert L.kb_beam_backtrace(5, 4, 0, 1.0, *fin, FAKE, FAKE, *out, None) == KB_ERR_INVALID_ARG
    assert L.kb_beam_backtrace(5, 4, 10, 1.0, *fin, None, FAKE, *out, None) == KB_ERR_INVALID_ARG


def test_shard_argument_checks():
    L = binding.lib()
    n = ctypes.c_int(-1)
    # splits follow the projection's plan: 3072 rows x 11,256 words (V=90k over 8 devices, cut on
    # multiples of 8), 16-byte aligned bf16 operands -> 12 row tiles x 15 splits of 3 word tiles
    assert L.kb_shard_splits(1, 3072, 1024, 11256, 12, FAKE, FAKE, FAKE, ctypes.byref(n)) == KB_OK
    assert n.value == 15
    # 11,250 words (V % 8 != 0) take the register-staged kernel's 128-word tiles: 18 splits of 5
    assert L.kb_shard_splits(1, 3072, 1024, 11250, 12, FAKE, FAKE, FAKE, ctypes.byref(n)) == KB_OK
    assert n.value == 18
    assert L.kb_shard_splits(1, 0, 1024, 11250, 12, None, None, None, ctypes.byref(n)) == KB_OK and n.value == 0
    assert L.kb_shard_splits(1, 3072, 1024, 11250, 12, FAKE, FAKE, FAKE, None) == KB_ERR_INVALID_ARG
    assert L.kb_shard_splits(1, 64, 1024, 8, 12, FAKE, FAKE, FAKE, ctypes.byref(n)) == KB_ERR_INVALID_ARG   # k > V
    assert L.kb_shard_workspace_bytes(1, 3072, 1024, 11250, 12) > 0
    assert L.kb_shard_workspace_bytes(1, 0, 1024, 11250, 12) == 0
    # kb_shard_partials(dtype, N, H, V_shard, word_base, k, h, W, b, stats, lists, ws, ws_bytes, stream)
    sp = L.kb_shard_partials
    assert sp(1, 0, 128, 1000, 0, 5, None, None, None, None, None, None, 0, None) == KB_OK   # empty batch
    assert sp(1, 10, 128, 1000, -1, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == KB_ERR_INVALID_ARG
    assert sp(1, 10, 128, 1000, (1 << 31) - 100, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30,
              None) == KB_ERR_INVALID_ARG                                                        # base + V overflows
    assert sp(1, 10, 128, 1000, 0, 5, FAKE, FAKE, FAKE, None, FAKE, FAKE, 1 << 30, None) == KB_ERR_INVALID_ARG
    assert sp(1, 10, 128, 1000, 0, 5, FAKE, FAKE, FAKE, ctypes.c_void_p(0x1004), FAKE, FAKE, 1 << 30,
              None) == KB_ERR_INVALID_ARG                                                        # stats alignment
    assert sp(1, 10, 128, 1000, 0, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == KB_ERR_WORKSPACE
    # kb_merge_partials(N, V, k, S, P, stats, lists, prev, off, tok, par, score, lse, stream)
    mp = L.kb_merge_partials
    out = [FAKE] * 7
    assert mp(0, 1000, 5, 0, 4, *out, None, None) == KB_OK                                       # empty batch
    assert mp(10, 1000, 5, 2, 0, *out, None, None) == KB_ERR_UNSUPPORTED                         # P < 1
    assert mp(10, 1000, 5, 2, 257, *out, None, None) == KB_ERR_UNSUPPORTED                       # P > 256
    assert mp(10, 1000, 17, 2, 4, *out, None, None) == KB_ERR_INVALID_ARG                        # k > 16
    assert mp(10, 4, 5, 2, 4, *out, None, None) == KB_ERR_INVALID_ARG                            # k > V
    assert mp(2, 1000, 5, 3, 4, *out, None, None) == KB_ERR_INVALID_ARG                          # N < S
    assert mp(10, 1000, 5, 2, 4, None, *out[1:], None, None) == KB_ERR_INVALID_ARG


def test_host_tensors_are_refused_not_computed():
    # the product path has no host fallback: tensors off the GPU are an error
    import torch
    h = torch.zeros((5, 64), dtype=torch.float32)
    W = torch.zeros((64, 100), dtype=torch.float32)
    b = torch.zeros(100, dtype=torch.float32)
    prev = torch.zeros(5, dtype=torch.float32)
    off = torch.tensor([0, 5], dtype=torch.int32)
    with pytest.raises(TypeError, match="on the GPU"):
        kb.kbest_step(h, W, b, prev, off, 3)
    with pytest.raises(TypeError, match="on the GPU"):
        kb.compact_beams(torch.ones(10, dtype=torch.uint8), 2, 5)
    with pytest.raises(TypeError, match="on the GPU"):
        kb.compact_batch(torch.ones(10, dtype=torch.uint8))
    with pytest.raises(TypeError, match="on the GPU"):
        kb.binding.standin_step(torch.zeros(2, dtype=torch.int32), torch.zeros(4, dtype=torch.int32),
                                torch.zeros(6), 2, 3, 0,
                                out=(torch.zeros(6, dtype=torch.int32), torch.zeros(2, dtype=torch.int32),
                                     torch.zeros(3, dtype=torch.int32), torch.zeros(6),
                                     torch.zeros(2, dtype=torch.int32)))


class _FakeLib:
    """Stands in for libkbest: every entry point succeeds without touching memory,
    after checking the arguments against the declared signature (count, and
    that each integer, size, float and pointer slot gets a value of that kind)."""

    def __getattr__(self, name):
        res, argtypes = binding.SIGNATURES[name]

        def call(*a):
            assert len(a) == len(argtypes), f"{name}: {len(a)} arguments, {len(argtypes)} declared"
            for i, (v, t) in enumerate(zip(a, argtypes)):
                if t in (ctypes.c_int, ctypes.c_size_t):
                    assert isinstance(v, int) and not isinstance(v, bool), f"{name} argument {i}: {v!r}"
                elif t is ctypes.c_float:
                    assert isinstance(v, (int, float)), f"{name} argument {i}: {v!r}"
                else:
                    assert v is None or isinstance(v, (ctypes.c_void_p, int)) or hasattr(v, "_obj"), \
                        f"{name} argument {i}: {v!r}"
            if name.endswith("_workspace_bytes"):
                return 4096
            if name == "kb_shard_splits":
                a[-1]._obj.value = 2
            if name == "kb_last_error":
                return b""
            return 0
        return call


def _fake_stream():
    class S:
        cuda_stream = 0
    return S()


def test_every_pointer_the_binding_passes_was_checked(monkeypatch):
    # each tensor whose address reaches the library has been through the
    # binding's check (device, layout, type and size) first: output tensors,
    # workspaces and optional arrays included, not only the inputs
    import torch
    checked, passed = set(), []
    monkeypatch.setattr(binding, "_lib", _FakeLib())
    monkeypatch.setattr(binding, "_need", lambda t, *a, **k: checked.add(id(t)))
    real_ptr = binding._ptr

    def ptr(t):
        if t is not None:
            passed.append(t)
        return real_ptr(t)
    monkeypatch.setattr(binding, "_ptr", ptr)
    st = _fake_stream()
    f32, i32, u8, bf = torch.float32, torch.int32, torch.uint8, torch.bfloat16
    z = lambda *shape, d=f32: torch.zeros(shape, dtype=d)     # noqa: E731
    N, H, V, k, S = 6, 16, 40, 3, 2
    h, W, b, prev, off = z(N, H, d=bf), z(H, V, d=bf), z(V), z(N), torch.tensor([0, 3, 6], dtype=i32)
    out3 = (z(S, k, d=i32), z(S, k, d=i32), z(S, k))
    binding.kbest_step(h, W, b, prev, off, k, out=out3, ws=z(4096, d=u8), row_lse=z(N), stream=st)
    binding.argmax_step(h, W, b, out=(z(N, d=i32), z(N)), ws=z(4096, d=u8), stream=st)
    binding.kbest_step_unfused(h, W, b, prev, off, k, out=out3, ws=z(4096, d=u8), row_lse=z(N), stream=st)
    binding.compact_batch(z(10, d=u8), torch.arange(10, dtype=i32) // 3,
                          out=(z(10, d=i32), z(1, d=i32), z(11, d=i32), z(1, d=i32)), ws=z(4096, d=u8), stream=st)
    binding.compact_beams(z(S * k, d=u8), S, k, out=(z(S * k, d=i32), z(1, d=i32), z(S + 1, d=i32), z(S, d=i32),
                                                    z(1, d=i32)), stream=st)
    binding.gather_rows(z(10, 4), torch.arange(5, dtype=i32), n_dev=z(1, d=i32), out=z(5, 4), stream=st)
    stats, lists = z(2 * N * 2), z(2 * N * k * 2, d=i32)
    binding.shard_partials(h, W, b, k, 0, stats, lists, ws=z(4096, d=u8), stream=st)
    binding.merge_partials(stats, lists, 2, V, k, prev, off, out=out3, row_lse=z(N), stream=st)
    binding.standin_alive(z(S, d=i32), z(4, d=i32), S, k, 0, out=z(S * k, d=u8), S_dev=z(1, d=i32), stream=st)
    binding.standin_next_h(z(40, H, d=bf), z(S * k, d=i32), z(S, d=i32), k, 4, 1, S * k, n_dev=z(1, d=i32),
                           out=z(S * k, H, d=bf), stream=st)
    binding.standin_step(z(S, d=i32), z(4, d=i32), z(S * k), S, k, 0,
                         out=(z(S * k, d=i32), z(2, d=i32), z(S + 1, d=i32), z(S * k), z(S, d=i32)),
                         S_dev=z(1, d=i32), alive=z(S * k, d=u8), next_state=(z(40, H, d=bf), 4, z(S * k, H, d=bf)),
                         stream=st)
    fin = (z(4, d=i32), z(4 * k), z(4 * k, d=i32), z(4 * k, d=i32))
    binding.beam_finish(S, k, 0, 4, 1, out3[0], out3[1], out3[2], z(S, d=i32), z(S, d=i32), z(S, d=i32), 0, 0,
                        z(4 * S * k, d=i32), z(4 * S * k, d=i32), fin, z(S * k, d=u8), stream=st)
    binding.beam_backtrace(4, k, 4, 1.0, fin, z(4 * S * k, d=i32), z(4 * S * k, d=i32),
                           out=(z(4, 4, d=i32), z(4, d=i32), z(4), z(4)), stream=st)
    unchecked = [tuple(t.shape) for t in passed if id(t) not in checked]
    assert passed and not unchecked, f"pointers passed without a check: {unchecked}"


def test_output_and_workspace_checks_raise():
    import torch
    # the checks themselves: host tensors, short outputs, small workspaces
    with pytest.raises(TypeError, match="on the GPU"):
        binding._need_outs((torch.zeros(4, dtype=torch.int32),), ("token",), (torch.int32,), 4)
    with pytest.raises(TypeError, match="on the GPU"):
        binding._need_ws(torch.zeros(64, dtype=torch.uint8), 16)

