"""GPU compaction (Algorithm 2's removal of finished hypotheses) and row gather.

Integer work: results must be bit-exact against the oracle.
"""
import numpy as np
import pytest
import torch

from oracle import kbest_oracle as ko
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1805_09863_amd as kb
    kb.lib()
    return kb


def _mask(pattern, S, k, g):
    M = S * k
    if pattern == "random":
        return (g.random(M) < 0.5).astype(np.uint8)
    if pattern == "all":
        return np.ones(M, np.uint8)
    if pattern == "none":
        return np.zeros(M, np.uint8)
    if pattern == "alternating":
        return (np.arange(M) % 2 == 0).astype(np.uint8)
    if pattern == "single":
        a = np.zeros(M, np.uint8)
        a[g.integers(M)] = 1
        return a
    if pattern == "sentences":
        return np.repeat(g.random(S) < 0.6, k).astype(np.uint8)
    if pattern == "values":              # nonzero values other than 1 mean alive
        return (g.integers(0, 4, M) * 37).astype(np.uint8)
    raise ValueError(pattern)


@pytest.mark.parametrize("pattern", ["random", "all", "none", "alternating", "single", "sentences", "values"])
@pytest.mark.parametrize("S,k", [(1, 1), (1, 5), (37, 5), (512, 5), (1638, 5), (700, 12), (3000, 3)])
def test_compact_bit_exact(kb, pattern, S, k):
    g = np.random.default_rng(S * 31 + k)
    a = _mask(pattern, S, k, g)
    say(f"compact S={S} k={k} {pattern}")
    keep, kept, noff, ksent, nS = kb.compact_batch(torch.from_numpy(a).cuda(), S, k)
    torch.cuda.synchronize()
    ref = ko.compact(a != 0, S, k)
    n = int(kept.item())
    assert n == ref.kept_count
    assert np.array_equal(keep.cpu().numpy()[:n], ref.keep_idx)
    ns = int(nS.item())
    assert ns == ref.new_S
    assert np.array_equal(noff.cpu().numpy()[:ns + 1], ref.new_offsets)
    # past the kept sentences the offsets repeat the kept count (empty sentences)
    assert (noff.cpu().numpy()[ns + 1:S + 1] == n).all()
    assert np.array_equal(ksent.cpu().numpy()[:ns], ref.kept_sentence)


def test_compact_empty_batch(kb):
    keep = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    kept = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    noff = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    ksent = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    nS = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    kb.compact_batch(torch.zeros(0, dtype=torch.uint8, device="cuda"), 0, 5, out=(keep, kept, noff, ksent, nS))
    torch.cuda.synchronize()
    assert kept.item() == 0 and nS.item() == 0 and noff.item() == 0 and keep.item() == -7


@pytest.mark.parametrize("row_elems,dtype", [(1024, torch.bfloat16), (1, torch.float32), (3, torch.int32),
                                             (40, torch.float32)])
def test_gather_rows(kb, row_elems, dtype):
    g = np.random.default_rng(row_elems)
    src = torch.from_numpy(g.standard_normal((300, row_elems)).astype(np.float32)).to(dtype).cuda()
    idx = torch.from_numpy(g.integers(0, 300, 200).astype(np.int32)).cuda()
    n_dev = torch.tensor([150], dtype=torch.int32, device="cuda")
    out = torch.zeros((200, row_elems), dtype=dtype, device="cuda")
    kb.gather_rows(src, idx, n_dev=n_dev, out=out)
    torch.cuda.synchronize()
    want = src[idx[:150].long()]
    assert torch.equal(out[:150], want)
    assert torch.count_nonzero(out[150:]) == 0


@pytest.mark.parametrize("S_live", [None, 0, 1, 9, 20, 25])
def test_standin_alive_device_count(kb, S_live):
    # EOS mask of the decoder stand-in: entries of sentences at or past the
    # device count are 0 and their (stale) sentence ids are never read
    S, k, t = 20, 3, 4
    g = np.random.default_rng(77)
    lengths = g.integers(1, 9, 50).astype(np.int32)
    lengths[49] = 8                               # alive at step t
    sid = g.permutation(49)[:S].astype(np.int32)
    live = S if S_live is None else min(S, S_live)
    sid_dev = torch.from_numpy(sid).cuda()
    sid_dev[live:] = 49                           # stale ids: would read as alive
    alive = torch.full((S * k,), 7, dtype=torch.uint8, device="cuda")
    s_dev = None if S_live is None else torch.tensor([S_live], dtype=torch.int32, device="cuda")
    from paper_1805_09863_amd import binding as kbb
    kbb.standin_alive(sid_dev, torch.from_numpy(lengths).cuda(), S, k, t, out=alive, S_dev=s_dev)
    torch.cuda.synchronize()
    want = np.repeat((np.arange(S) < live) & (t < lengths[sid] - 1), k).astype(np.uint8)
    assert np.array_equal(alive.cpu().numpy(), want)
