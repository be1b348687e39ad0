"""kb_kbest_step_noalloc, the step for callers that cannot allocate, through the C ABI.

Its results must equal kb_kbest_step's with a caller workspace (the same
kernels run; only where their partials live differs) and meet the oracle's
bar, on two calls in a row, the second on a smaller batch, so that stale
contents of the shared scratch array from the first call cannot leak in.
"""
import numpy as np
import pytest
import torch

from synth import workloads as wl
from tests.gpu_util import check, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


def _both(kb, inp):
    h, W, b, prev, off = to_dev(inp)
    S, k, N = inp.S, inp.k, inp.N
    mk = lambda fill, dt: torch.full((S, k), fill, dtype=dt, device="cuda")  # noqa: E731
    ref = (mk(-7, torch.int32), mk(-7, torch.int32), mk(float("nan"), torch.float32))
    got = (mk(9, torch.int32), mk(9, torch.int32), mk(float("-inf"), torch.float32))
    lse_ref = torch.full((N,), float("nan"), device="cuda")
    lse_got = torch.full((N,), 3.0, device="cuda")
    kb.kbest_step(h, W, b, prev, off, k, out=ref, row_lse=lse_ref)
    kb.kbest_step_noalloc(h, W, b, prev, off, k, out=got, row_lse=lse_got)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in ref + (lse_ref,)], [x.cpu().numpy() for x in got + (lse_got,)]


def test_noalloc_matches_workspace_step_twice_then_smaller(kb):
    first = wl.make_step(H=512, V=30000, k=12, S=64, beam=12, dtype="bf16", seed=811, bias="zipf",
                         name="noalloc_768rows")
    second = wl.make_step(H=128, V=3001, k=4, rows_per_sentence=[3, 1, 4, 2, 5], dtype="f32", seed=812,
                          name="noalloc_15rows")
    for inp in (first, second):
        say(f"no-alloc step: {inp.name} N={inp.N} H={inp.H} V={inp.V} k={inp.k} {inp.dtype}")
        ref, got = _both(kb, inp)
        for x, y, name in zip(ref, got, ("token", "parent", "score", "row_lse")):
            assert np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                                  y.view(np.uint32) if y.dtype == np.float32 else y), f"{inp.name}: {name}"
        rep, _ = check(inp, tuple(got))
        say(f"  equal to the workspace step; max score err {rep.max_score_err:.2e}")


def test_noalloc_refuses_shapes_beyond_its_array(kb):
    # 200,000 rows at V = 8,000, k = 16: the partials need about 41 MB; the
    # call is refused on the host before anything is enqueued
    L = kb.lib()
    need = L.kb_kbest_workspace_bytes(1, 200000, 128, 8000, 16, 100)
    assert need > L.kb_kbest_step_scratch_max()
    h = torch.zeros((200000, 128), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((128, 8000), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(8000, device="cuda")
    prev = torch.zeros(200000, device="cuda")
    off = torch.arange(101, dtype=torch.int32, device="cuda") * 2000
    out = tuple(torch.empty((100, 16), dtype=t, device="cuda") for t in (torch.int32, torch.int32, torch.float32))
    with pytest.raises(kb.KBestError) as e:
        kb.kbest_step_noalloc(h, W, b, prev, off, 16, out=out)
    assert e.value.status == 2 and "scratch" in str(e.value)
