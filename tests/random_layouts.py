"""Seeded random staging layouts for the parity sweeps: decoder shapes, shard counts, TP degrees
and chunk budgets that the library accepts, at sizes the oracle finishes in well under a second
but that still span many workgroup tiles with ragged tails, column-sliced o/down runs cut at
shard and chunk boundaries, and (for odd head widths) unaligned runs."""
from __future__ import annotations

import numpy as np

from paper_2607_22614_amd import datagen


def random_layout(rng: np.random.Generator, max_elems: int = 4_000_000, max_chunks: int = 2048):
    """(model, W, T, B) with T | Hq, Hkv, F, V, Hkv | Hq, H % 8 == 0, B % 16 == 0, at most
    max_elems padded training elements and at most max_chunks chunks of the rollout stream (the
    oracle checksums chunk by chunk; budgets down to 16 bytes are covered on small shapes)."""
    while True:
        t = int(rng.choice([1, 2, 3, 4, 8]))
        hkv = t * int(rng.integers(1, 3))
        hq = hkv * int(rng.choice([1, 2, 4]))
        d = int(rng.choice([2, 4, 6, 8, 16, 32, 64, 128], p=[.05, .1, .05, .1, .2, .2, .2, .1]))
        h = 8 * int(rng.integers(1, 97))
        f = t * int(rng.integers(1, 301))
        v = t * int(rng.integers(1, 601))
        layers = int(rng.integers(0, 4))
        w = int(rng.choice([1, 2, 3, 5, 8, 13, 64]))
        model = (layers, h, hq, hkv, d, f, v)
        n, npad = datagen.flat_sizes(model, w)
        if npad > max_elems:
            continue
        rollout_bytes = 2 * (n + (t - 1) * (2 * layers + 1) * h)  # norms are replicated on every rank
        # budgets log-uniform over 16 B .. 4 MiB, and now and then one chunk for everything
        b = 1 << 30 if rng.random() < 0.1 else 16 * int(2 ** rng.uniform(0, 18))
        b = max(b, 16 * -(-rollout_bytes // (16 * max_chunks)))
        return model, w, t, b


def random_reshard(rng: np.random.Generator, max_elems: int = 4_000_000, max_chunks: int = 2048):
    """(model, W, W', B) for a reshard plan (4-byte elements; at most max_chunks chunks)."""
    model, w, _, b = random_layout(rng, max_elems, max_chunks)
    w2 = int(rng.choice([1, 2, 3, 4, 6, 7, 8, 16, 64]))
    _, npad2 = datagen.flat_sizes(model, w2)
    return model, w, w2, max(b, 16 * -(-4 * npad2 // (16 * max_chunks)))
