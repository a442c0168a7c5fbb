"""Pins of the oracle's chunk checksum (O5) and moment stream (O6).

Closed forms (all-zero, constant word, single word), byte order, the
concatenation law s(A||B) = (s1A + s1B, s2A + s2B + |A| s1B) that follows from
the definition, and an arbitrary-precision Python evaluation reduced mod 2^64
at the end (exercises the wrap-around of the uint64 sums).
"""
import numpy as np
import pytest

import oracle

M64 = 1 << 64


def _words(ws):
    return np.array(ws, dtype="<u4").view(np.uint8)


def test_zero_chunk():
    assert oracle.checksum(np.zeros(4096, dtype=np.uint8)) == (0, 0)


@pytest.mark.parametrize("c,n", [(1, 10), (0xFFFFFFFF, 1 << 20), (0x3F803F80, 12345)])
def test_constant_word(c, n):
    s1, s2 = oracle.checksum(_words([c] * n))
    assert s1 == (n * c) % M64
    assert s2 == (c * n * (n + 1) // 2) % M64


def test_single_word_position():
    for j in (0, 1, 7, 1000):
        ws = [0] * 1001
        ws[j] = 0xDEADBEEF
        assert oracle.checksum(_words(ws)) == (0xDEADBEEF, (j + 1) * 0xDEADBEEF)


def test_little_endian_words_from_bf16_pairs():
    # word j = bf16[2j] | bf16[2j+1] << 16
    b = np.array([0x1234, 0xABCD, 0x0001, 0x8000], dtype=np.uint16)
    s1, s2 = oracle.checksum(b)
    w0, w1 = 0xABCD1234, 0x80000001
    assert (s1, s2) == (w0 + w1, w0 + 2 * w1)


def test_concatenation_law():
    rng = np.random.default_rng(3)
    a = rng.integers(0, 1 << 32, size=5000, dtype=np.uint64).astype("<u4")
    b = rng.integers(0, 1 << 32, size=777, dtype=np.uint64).astype("<u4")
    s1a, s2a = oracle.checksum(a.view(np.uint8))
    s1b, s2b = oracle.checksum(b.view(np.uint8))
    s1, s2 = oracle.checksum(np.concatenate([a, b]).view(np.uint8))
    assert s1 == (s1a + s1b) % M64
    assert s2 == (s2a + s2b + a.size * s1b) % M64


def test_big_int_reference_with_wraparound():
    rng = np.random.default_rng(11)
    w = rng.integers(1 << 31, 1 << 32, size=300000, dtype=np.uint64)
    s1 = s2 = 0
    for j, x in enumerate(w.tolist()):
        s1 += x
        s2 += (j + 1) * x
    assert s2 >= M64  # the sum really wraps
    assert oracle.checksum(w.astype("<u4").view(np.uint8)) == (s1 % M64, s2 % M64)


def test_chunk_checksums_split_the_stream():
    rng = np.random.default_rng(2)
    s = rng.integers(0, 1 << 16, size=1000, dtype=np.uint16)
    cks = oracle.chunk_checksums(s, 64)
    assert len(cks) == -(-2000 // 64)
    assert cks[0] == oracle.checksum(s[:32]) and cks[-1] == oracle.checksum(s[-(1000 - 31 * 32):])


def test_moment_stream_order():
    w, S = 3, 512
    m = [np.full(S, i, dtype=np.float32) for i in range(w)]
    v = [np.full(S, 10 + i, dtype=np.float32) for i in range(w)]
    st = oracle.moment_stream(m, v).view(np.float32)
    assert st.size == 2 * w * S
    assert np.array_equal(st, np.repeat(np.array([0, 1, 2, 10, 11, 12], dtype=np.float32), S))
