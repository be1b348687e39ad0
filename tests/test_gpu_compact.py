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
    keep, kept, noff, ksent, nS = kb.compact_beams(torch.from_numpy(a).cuda(), S, k)
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
    kb.compact_beams(torch.zeros(0, dtype=torch.uint8, device="cuda"), 0, 5, out=(keep, kept, noff, ksent, nS))
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


@pytest.mark.parametrize("S,k,S_live,H", [(0, 5, None, 8), (20, 3, None, 5), (20, 3, 0, 8), (20, 3, 9, 8),
                                           (1, 5, None, 5), (512, 5, 300, 8), (1500, 4, 1400, 5),
                                           (2048, 12, None, 8)])
@pytest.mark.parametrize("gather", [False, True])
def test_standin_step_matches_its_definition(kb, S, k, S_live, H, gather):
    # the fused step = the stand-in's EOS mask, the stable compaction of that
    # mask (np.flatnonzero), the sentence offsets and the gathers (scores,
    # sentence ids and, with gather, the next states: 16-byte rows at H = 8,
    # 4-byte words at H = 5; one launch while entries and ids fit in 64 KB, two past it at
    # 2048 x 12); sentences past the device count are dropped without reading
    # their (stale) ids
    from paper_1805_09863_amd import binding as kbb
    g = np.random.default_rng(S * 7 + k)
    t, T = 6, 8
    n_orig = S + 40
    lengths = g.integers(1, 14, n_orig).astype(np.int32)
    lengths[n_orig - 1] = 13                      # the stale id below: would read as alive
    sid = g.permutation(n_orig - 1)[:S].astype(np.int32)
    live = S if S_live is None else min(S, S_live)
    score = g.standard_normal(S * k).astype(np.float32)
    mask = np.repeat((np.arange(S) < live) & (t < lengths[np.where(np.arange(S) < live, sid, 0)] - 1), k)
    keep_want = np.flatnonzero(mask).astype(np.int32)
    sent_alive = mask.reshape(S, k).any(axis=1)
    ks = np.flatnonzero(sent_alive)
    per_sent = mask.reshape(S, k).sum(axis=1)[ks]
    off_want = np.concatenate([[0], np.cumsum(per_sent)]).astype(np.int32)
    sid_dev = torch.from_numpy(sid).cuda()
    sid_dev[live:] = n_orig - 1                   # stale ids past the device count
    keep = torch.full((S * k,), -9, dtype=torch.int32, device="cuda")
    counts = torch.full((2,), -9, dtype=torch.int32, device="cuda")
    noff = torch.full((S + 1,), -9, dtype=torch.int32, device="cuda")
    prev_next = torch.full((S * k,), float("nan"), dtype=torch.float32, device="cuda")
    sid_next = torch.full((S,), -9, dtype=torch.int32, device="cuda")
    alive = torch.full((S * k,), 7, dtype=torch.uint8, device="cuda")
    s_dev = None if S_live is None else torch.tensor([S_live], dtype=torch.int32, device="cuda")
    counts_host = torch.full((3,), -9, dtype=torch.int32, pin_memory=True)
    table = torch.from_numpy(g.standard_normal((n_orig * T * k, H)).astype(np.float32)).cuda()
    nh = torch.full((S * k, H), float("nan"), dtype=torch.float32, device="cuda")
    kbb.standin_step(sid_dev, torch.from_numpy(lengths).cuda(), torch.from_numpy(score).cuda(), S, k, t,
                     out=(keep, counts, noff, prev_next, sid_next), S_dev=s_dev, alive=alive,
                     counts_host=counts_host, next_state=(table, T, nh) if gather else None)
    torch.cuda.synchronize()
    n, ns = (int(x) for x in counts.cpu())
    assert counts_host.tolist() == [n, ns, t + 1]  # the copy the kernel writes to pinned host memory, and the tag
    assert (n, ns) == (keep_want.size, ks.size)
    assert np.array_equal(keep.cpu().numpy()[:n], keep_want)
    assert np.array_equal(alive.cpu().numpy(), mask.astype(np.uint8))
    noff_h = noff.cpu().numpy()
    assert np.array_equal(noff_h[:ns + 1], off_want)
    assert (noff_h[ns:] == n).all()               # empty sentences past the survivors
    assert np.array_equal(prev_next.cpu().numpy()[:n].view(np.uint32), score[keep_want].view(np.uint32))
    assert np.array_equal(sid_next.cpu().numpy()[:ns], sid[ks])
    nh_h = nh.cpu().numpy()
    if gather:
        src = (sid[keep_want // k].astype(np.int64) * T + t + 1) * k + keep_want % k
        assert np.array_equal(nh_h[:n].view(np.uint32), table.cpu().numpy()[src].view(np.uint32))
    assert np.isnan(nh_h[n:]).all()               # rows past the survivors are not written


# ---------------------------------------------------------------- the M-entry form (kb_compact_batch)
def _entries(M, g, max_sent=6):
    sizes = g.integers(0, max_sent + 1, M + 1)                # empty sentences included
    es = np.repeat(np.arange(sizes.size), sizes)[:M]          # sum(sizes) >= M unless all draws are 0
    if es.size < M:
        es = np.concatenate([es, np.full(M - es.size, sizes.size)])
    return (es + 3).astype(np.int32)                          # ids need not start at 0


@pytest.mark.parametrize("M", [0, 1, 7, 4096, 4097, 16384, 16385, 100_003, 1_000_000])
@pytest.mark.parametrize("pattern", ["random", "none", "all", "sparse"])
def test_compact_batch_entries_bit_exact(kb, M, pattern):
    # one workgroup up to 16,384 entries, the three-kernel form past that
    # (ragged last workgroup, several workgroups in the count scan)
    g = np.random.default_rng(M + len(pattern))
    a = {"random": g.random(M) < 0.5, "none": np.zeros(M, bool), "all": np.ones(M, bool),
         "sparse": g.random(M) < 0.002}[pattern].astype(np.uint8) * np.uint8(g.integers(1, 200))
    es = _entries(M, g)
    say(f"compact_batch M={M} {pattern}: {int((a != 0).sum())} alive")
    alive = torch.from_numpy(a).cuda()
    es_d = torch.from_numpy(es).cuda()
    keep = torch.full((max(M, 1),), -5, dtype=torch.int32, device="cuda")
    kept = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    noff = torch.full((M + 1,), -5, dtype=torch.int32, device="cuda")
    nS = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    kb.compact_batch(alive, es_d, out=(keep, kept, noff, nS))
    torch.cuda.synchronize()
    ref = ko.compact_entries(a, es)
    n, ns = int(kept.item()), int(nS.item())
    assert n == ref.kept_count and ns == ref.new_S
    assert np.array_equal(keep.cpu().numpy()[:n], ref.keep_idx)
    assert np.array_equal(noff.cpu().numpy()[:ns + 1], ref.new_offsets)
    assert (noff.cpu().numpy()[ns + 1:] == -5).all()          # nothing written past new_S
    # without sentence ids: the kept list only
    keep2, kept2, noff2, nS2 = kb.compact_batch(alive)
    torch.cuda.synchronize()
    assert noff2 is None and nS2 is None
    assert int(kept2.item()) == n and np.array_equal(keep2.cpu().numpy()[:n], ref.keep_idx)


def test_compact_batch_matches_beam_form(kb):
    # an S x k batch with entry_sentence = i // k gives the S x k form's results
    g = np.random.default_rng(12)
    S, k = 900, 5
    a = (g.random(S * k) < 0.4).astype(np.uint8)
    alive = torch.from_numpy(a).cuda()
    es = torch.arange(S * k, dtype=torch.int32, device="cuda") // k
    keep, kept, noff, nS = kb.compact_batch(alive, es)
    keep_b, kept_b, noff_b, ksent_b, nS_b = kb.compact_beams(alive, S, k)
    torch.cuda.synchronize()
    n, ns = int(kept.item()), int(nS.item())
    assert n == int(kept_b.item()) and ns == int(nS_b.item())
    assert torch.equal(keep[:n], keep_b[:n]) and torch.equal(noff[:ns + 1], noff_b[:ns + 1])


# ---------------------------------------------------------------- KB_DEBUG validation
def _small_step_inputs(S=4, beam=3, V=900, H=64):
    from synth import workloads as wl
    from tests.gpu_util import to_dev
    inp = wl.make_step(H=H, V=V, k=4, S=S, beam=beam, dtype="f32", seed=3, name="dbg")
    return inp, to_dev(inp)


@pytest.mark.parametrize("bad", ["first", "decreasing", "past_N"])
def test_debug_rejects_bad_sentence_offsets(kb, monkeypatch, bad):
    inp, (h, W, b, prev, off) = _small_step_inputs()
    o = inp.off.copy()
    if bad == "first":
        o[0] = 1
    elif bad == "decreasing":
        o[2], o[3] = o[3], o[2]
    else:
        o[-1] = inp.N + 1
    off_bad = torch.from_numpy(o).cuda()
    tok = torch.full((inp.S, inp.k), 123, dtype=torch.int32, device="cuda")
    par = torch.full((inp.S, inp.k), 123, dtype=torch.int32, device="cuda")
    sc = torch.full((inp.S, inp.k), 1.5, dtype=torch.float32, device="cuda")
    monkeypatch.setenv("KB_DEBUG", "1")
    with pytest.raises(kb.KBestError) as e:
        kb.kbest_step(h, W, b, prev, off_bad, inp.k, out=(tok, par, sc))
    assert e.value.status == 1 and "KB_DEBUG" in str(e.value)
    torch.cuda.synchronize()
    # nothing but the verdict word was written: no merge ran
    assert (par == 123).all() and (sc == 1.5).all() and (tok.view(-1)[1:] == 123).all()
    # the same offsets through the vocabulary-shard merge
    stats = torch.zeros((1, inp.N, 2), dtype=torch.float32, device="cuda")
    lists = torch.zeros((1, inp.N, inp.k, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(kb.KBestError) as e:
        kb.merge_partials(stats, lists, 1, inp.V, inp.k, prev, off_bad)
    assert e.value.status == 1
    # valid offsets pass under KB_DEBUG and give the usual result
    t1, p1, s1 = kb.kbest_step(h, W, b, prev, off, inp.k)
    monkeypatch.delenv("KB_DEBUG")
    t0, p0, s0 = kb.kbest_step(h, W, b, prev, off, inp.k)
    torch.cuda.synchronize()
    assert torch.equal(t0, t1) and torch.equal(p0, p1) and torch.equal(s0, s1)


def test_debug_rejects_unsorted_entry_sentences(kb, monkeypatch):
    alive = torch.ones(10, dtype=torch.uint8, device="cuda")
    es = torch.tensor([0, 0, 1, 1, 2, 1, 3, 3, 4, 4], dtype=torch.int32, device="cuda")
    monkeypatch.setenv("KB_DEBUG", "1")
    with pytest.raises(kb.KBestError) as e:
        kb.compact_batch(alive, es)
    assert e.value.status == 1
    with pytest.raises(kb.KBestError):
        kb.compact_batch(alive, torch.full((10,), -1, dtype=torch.int32, device="cuda"))
    keep, kept, noff, nS = kb.compact_batch(alive, torch.sort(es).values.contiguous())
    torch.cuda.synchronize()
    assert int(kept.item()) == 10 and int(nS.item()) == 5
