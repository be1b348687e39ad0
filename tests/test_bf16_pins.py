"""Independent pins of the bf16 storage format on both sides of the oracle.

The oracle widens bf16 bit patterns to float64 (``oracle.widen``) and the
seeded generators round float32 to bf16 (``synth.f32_to_bf16_bits``).  Neither
may be checked against itself: here they are fixed by a hand table of bit
patterns whose values follow from the format's definition (1 sign bit, 8
exponent bits with bias 127, 7 fraction bits; the top half of an IEEE float32)
and by torch's own bfloat16 conversions, which share no code with either.
"""
import numpy as np
import pytest
import torch

from oracle import kbest_oracle as ko
from synth import workloads as wl

# (bits, value): each value worked out from sign, exponent and fraction
HAND = [
    (0x3F80, 1.0),                            # exponent 127, fraction 0
    (0xC000, -2.0),                           # sign 1, exponent 128
    (0x3F81, 1.0 + 2.0 ** -7),                # lowest fraction bit of 1.0
    (0x4049, 3.140625),                       # 1.5703125 * 2: fraction 0b1001001
    (0x3E80, 0.25),                           # exponent 125
    (0x0001, 2.0 ** -133),                    # smallest subnormal: 2^-126 * 2^-7
    (0x0080, 2.0 ** -126),                    # smallest normal
    (0x8000, -0.0),
    (0x0000, 0.0),
    (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127),  # largest finite
    (0xFF7F, -(2.0 - 2.0 ** -7) * 2.0 ** 127),
    (0x4780, 65536.0),                        # exponent 143
    (0xBF00, -0.5),
]


def _hand_table_errors(widen_fn):
    bits = np.array([b for b, _ in HAND], dtype=np.uint16)
    got = widen_fn(bits, "bf16")
    errs = []
    for (b, v), g in zip(HAND, got):
        if not (g == v and np.signbit(g) == np.signbit(v)):
            errs.append(f"0x{b:04X}: {g!r} != {v!r}")
    return errs


def test_widen_bf16_hand_table():
    assert ko.widen(np.array([0x3F80], dtype=np.uint16), "bf16").dtype == np.float64
    errs = _hand_table_errors(ko.widen)
    assert not errs, "; ".join(errs)


def test_widen_f32_is_exact():
    vals = np.array([1.0, -2.5, 2.0 ** -149, 3.4028234663852886e38, 0.1], dtype=np.float32)
    got = ko.widen(vals, "f32")
    assert got.dtype == np.float64
    assert [float(x) for x in got] == [float(x) for x in vals.tolist()]


def _torch_widen(bits: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(bits.astype(np.uint16).view(np.int16)).view(torch.bfloat16)
    return t.to(torch.float64).numpy()


def test_widen_bf16_matches_torch_on_random_patterns():
    g = np.random.default_rng(20180509)
    bits = g.integers(0, 1 << 16, size=100_000, dtype=np.uint32).astype(np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]          # finite patterns only
    ours = ko.widen(bits, "bf16")
    ref = _torch_widen(bits)
    assert np.array_equal(ours.view(np.uint64), ref.view(np.uint64))


def test_generator_rounding_matches_torch_cast():
    # round-to-nearest-even from float32, the storage conversion of the bf16
    # workloads: ordinary draws, values on the rounding midpoints (ties go to
    # the even pattern), just above and below them, and subnormals
    g = np.random.default_rng(7)
    normal = (g.standard_normal(200_000) * np.exp(g.uniform(-30, 30, 200_000))).astype(np.float32)
    base = g.integers(0, 1 << 16, size=50_000, dtype=np.uint32)
    base = base[((base << 16) & 0x7F800000) != 0x7F800000]
    mid = ((base << 16) | 0x8000).astype(np.uint32)          # exactly halfway
    near = np.concatenate([mid, mid + 1, mid - 1]).view(np.float32)
    near = near[np.isfinite(near)]
    sub = (g.integers(1, 1 << 23, size=10_000, dtype=np.uint32)).view(np.float32)
    for a in (normal, near, sub, np.array([0.0, -0.0, 1.0, -1.0], dtype=np.float32)):
        ours = wl.f32_to_bf16_bits(a)
        ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        bad = np.flatnonzero(ours != ref)
        assert bad.size == 0, f"{bad.size} mismatches, e.g. {a[bad[:3]]}: {ours[bad[:3]]} vs {ref[bad[:3]]}"


def test_generator_widening_matches_oracle_widening():
    # the generator's own float32 view of bf16 bits (used to build inputs)
    # and the oracle's float64 view agree exactly
    g = np.random.default_rng(11)
    bits = g.integers(0, 1 << 16, size=20_000, dtype=np.uint32).astype(np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]
    assert np.array_equal(wl.bf16_bits_to_f32(bits).astype(np.float64), _torch_widen(bits))


def _widen_slipped(shift, swap_bytes=False):
    # the oracle's widening with one plausible slip planted
    def f(a, dtype):
        u = np.asarray(a, dtype=np.uint16)
        if swap_bytes:
            u = u.byteswap()
        u = u.astype(np.uint64) << np.uint64(shift)
        return (u & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32).astype(np.float64)
    return f


@pytest.mark.parametrize("shift,swap", [(15, False), (17, False), (16, True)])
def test_hand_table_catches_planted_slips(shift, swap):
    with np.errstate(all="ignore"):
        assert _hand_table_errors(_widen_slipped(shift, swap))
    assert not _hand_table_errors(_widen_slipped(16))
