"""Pins of the oracle's fp32 -> bf16 cast (O2) against things other than itself.

* a hand-derived IEEE 754 roundTiesToEven table (tests/golden/bf16_rne_pins.txt);
* exact rational rounding from the definition (Fractions, nearest / ties-to-even
  / overflow threshold), on a structured sample of every exponent;
* a library routine: torch's CPU float32 -> bfloat16 conversion, for every
  non-NaN input on a sweep of all 2^16 upper halves x the rounding-critical
  lower halves, plus random patterns;
* NaN: every NaN stays NaN with its sign and the quiet bit set.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import rne_bf16


def _load_pins(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "bf16_rne_pins.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b = line.split()[:2]
            rows.append((int(a, 16), int(b, 16)))
    return rows


def test_hand_derived_table(golden_dir):
    rows = _load_pins(golden_dir)
    assert len(rows) >= 30
    inp = np.array([a for a, _ in rows], dtype=np.uint32)
    exp = np.array([b for _, b in rows], dtype=np.uint16)
    got = rne_bf16(inp)
    bad = [(hex(a), hex(b), hex(int(g))) for (a, b), g in zip(rows, got) if b != g]
    assert not bad, bad


# ------------------------------------------------------------------ exact rational definition
def _f32_value(u):
    s = -1 if u >> 31 else 1
    e = (u >> 23) & 0xFF
    m = u & 0x7FFFFF
    if e == 0:
        return s * Fraction(m, 1 << 149)
    return s * Fraction((1 << 23) | m, 1 << 23) * (Fraction(2) ** (e - 127))


def _bf16_magnitude(b):
    """Value of a non-negative bf16 pattern; 0x7F80 stands for 2^128 (the unbounded next step)."""
    e = (b >> 7) & 0xFF
    m = b & 0x7F
    if e == 0:
        return Fraction(m, 1 << 133)
    return Fraction(128 + m, 128) * (Fraction(2) ** (e - 127))


def _rne_by_definition(u):
    """Nearest bf16 to the exact value; ties to even significand; >= max+half ulp -> Inf."""
    x = _f32_value(u)
    sign = 0x8000 if u >> 31 else 0
    ax = abs(x)
    if u & 0x7FFFFFFF == 0x7F800000:
        return sign | 0x7F80
    # largest bf16 magnitude not above |x| (search over the ordered encodings)
    lo, hi = 0, 0x7F7F
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if _bf16_magnitude(mid) <= ax:
            lo = mid
        else:
            hi = mid - 1
    below = lo
    above = below + 1  # 0x7F80 -> treated as 2^128 for the overflow rule
    if _bf16_magnitude(below) == ax:
        return sign | below
    d_lo = ax - _bf16_magnitude(below)
    d_hi = _bf16_magnitude(above) - ax
    if d_lo < d_hi:
        pick = below
    elif d_hi < d_lo:
        pick = above
    else:
        pick = below if below % 2 == 0 else above
    return sign | pick


def _structured_sample(rng, per_exp=12):
    vals = []
    for e in range(0, 255):
        for low in (0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF):
            top = int(rng.integers(0, 128))
            s = int(rng.integers(0, 2))
            vals.append((s << 31) | (e << 23) | (top << 16) | low)
        for _ in range(per_exp):
            vals.append(int(rng.integers(0, 1 << 31)) & 0x807FFFFF | (e << 23))
    return vals


def test_exact_rational_rounding():
    rng = np.random.default_rng(1234)
    vals = _structured_sample(rng) + [0x7F7F8000, 0x7F7F7FFF, 0x7F7FFFFF, 0x007FFFFF, 0x00000001, 0x7F800000]
    got = rne_bf16(np.array(vals, dtype=np.uint32))
    for u, g in zip(vals, got):
        assert int(g) == _rne_by_definition(u), hex(u)


# ------------------------------------------------------------------ library routine
def _torch_bf16_bits(u32):
    f = torch.from_numpy(u32.view(np.float32))
    return f.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _non_nan(u):
    return (u & np.uint32(0x7FFFFFFF)) <= np.uint32(0x7F800000)


def test_against_torch_all_upper_halves():
    hi = np.arange(1 << 16, dtype=np.uint32) << np.uint32(16)
    for low in (0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF):
        u = hi | np.uint32(low)
        keep = _non_nan(u)
        u = u[keep]
        np.testing.assert_array_equal(rne_bf16(u), _torch_bf16_bits(u))


def test_against_torch_random_patterns():
    rng = np.random.default_rng(99)
    u = rng.integers(0, 1 << 32, size=1 << 22, dtype=np.uint64).astype(np.uint32)
    u = u[_non_nan(u)]
    np.testing.assert_array_equal(rne_bf16(u), _torch_bf16_bits(u))


@pytest.mark.skipif(os.environ.get("DR_EXHAUSTIVE_CAST") != "1", reason="set DR_EXHAUSTIVE_CAST=1 for the 2^32 sweep")
def test_against_torch_exhaustive():
    step = 1 << 26
    for start in range(0, 1 << 32, step):
        u = np.arange(start, start + step, dtype=np.uint64).astype(np.uint32)
        u = u[_non_nan(u)]
        np.testing.assert_array_equal(rne_bf16(u), _torch_bf16_bits(u))


# ------------------------------------------------------------------ NaN
def test_nan_stays_nan_with_sign_and_quiet_bit():
    rng = np.random.default_rng(5)
    payload = rng.integers(1, 1 << 23, size=1 << 16, dtype=np.uint32)
    sign = rng.integers(0, 2, size=payload.size, dtype=np.uint32) << np.uint32(31)
    u = sign | np.uint32(0x7F800000) | payload
    out = rne_bf16(u).astype(np.uint32)
    assert np.all((out & 0x7F80) == 0x7F80)          # exponent all ones
    assert np.all((out & 0x007F) != 0)               # significand nonzero: NaN, not Inf
    assert np.all((out & 0x0040) != 0)               # quiet
    assert np.all((out >> 15) == (u >> 31))          # sign kept
    # payload bits above the quiet bit survive
    assert np.all((out & 0x003F) == ((u >> 16) & 0x3F))


# ------------------------------------------------------------------ bf16 -> fp32 widening
# The round-trip pin widens the rebuilt bf16 tensors back to fp32, so the widening
# is pinned on its own: closed forms of the encoding, the exact value of every bf16
# pattern, torch's CPU bfloat16 -> float32 conversion, and the cast as its left inverse.
import oracle  # noqa: E402  (module attribute: the mutation tests patch it)


def test_widen_closed_forms():
    rows = [(0x0000, 0x00000000), (0x8000, 0x80000000), (0x3F80, 0x3F800000), (0xBF80, 0xBF800000),
            (0x0001, 0x00010000), (0x8001, 0x80010000), (0x007F, 0x007F0000), (0x0080, 0x00800000),
            (0x7F7F, 0x7F7F0000), (0x7F80, 0x7F800000), (0xFF80, 0xFF800000), (0x7FC0, 0x7FC00000),
            (0xFFC0, 0xFFC00000), (0x7FFF, 0x7FFF0000), (0x4049, 0x40490000)]
    got = oracle.widen_bf16(np.array([a for a, _ in rows], dtype=np.uint16))
    assert got.dtype == np.uint32
    assert [hex(int(g)) for g in got] == [hex(b) for _, b in rows]


def test_widen_is_exact_on_every_pattern():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    w = oracle.widen_bf16(b)
    for bb, ww in zip(b.tolist(), w.tolist()):
        if (bb & 0x7F80) == 0x7F80:   # Inf / NaN: same class, sign and payload prefix
            assert (ww >> 23) & 0xFF == 0xFF and (ww >> 31) == (bb >> 15) and ((ww >> 16) & 0x7F) == (bb & 0x7F)
            continue
        sign = -1 if bb >> 15 else 1
        assert _f32_value(ww) == sign * _bf16_magnitude(bb & 0x7FFF), hex(bb)


def test_widen_against_torch():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    keep = (b & np.uint16(0x7FFF)) <= np.uint16(0x7F80)  # torch may canonicalise NaN bits
    b = b[keep]
    ref = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(torch.float32).view(torch.int32).numpy()
    np.testing.assert_array_equal(oracle.widen_bf16(b), ref.view(np.uint32))


def test_cast_undoes_widen():
    # rne(widen(b)) == b for every bf16 pattern except signalling NaNs, which come back quiet
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    back = rne_bf16(oracle.widen_bf16(b))
    snan = ((b & np.uint16(0x7F80)) == 0x7F80) & ((b & np.uint16(0x7F)) != 0) & ((b & np.uint16(0x40)) == 0)
    np.testing.assert_array_equal(back[~snan], b[~snan])
    np.testing.assert_array_equal(back[snan], b[snan] | np.uint16(0x40))
