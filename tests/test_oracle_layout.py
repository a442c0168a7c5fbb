"""Pins of the oracle's layout transform (O1, O3, O4) against things other than itself.

* closed-form sizes of the five workloads (tests/golden/workload_sizes.txt);
* a hand-worked example of both ranks of a tiny model (tests/golden/tiny_worked_layout.txt);
* brute force on a grid of tiny shapes with tagged sources: every output element
  is checked, one by one, against a direct per-element index formula, and the
  tags must cover each weight exactly once and each norm exactly T times;
* T = 1 reduces the transform to a plain cast of the unpadded flat buffer;
* the round-trip inverse (rollout -> training) equals a cast of the source;
* chunk spans: fixed size B except the last, contiguous, covering the stream.
"""
import itertools
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import Model
from paper_2607_22614_amd import datagen, workloads


def _model(w):
    return Model(*w.model)


# ------------------------------------------------------------------ closed-form sizes
def _sizes(golden_dir):
    out = {}
    with open(os.path.join(golden_dir, "workload_sizes.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, *vals = line.split()
            out[name] = [int(v) for v in vals]
    return out


@pytest.mark.parametrize("wl", workloads.ALL, ids=lambda w: w.name)
def test_workload_sizes(wl, golden_dir):
    N, Nn, Npad, S, per_rank, stream_bytes, nchunks, last = _sizes(golden_dir)[wl.name]
    m = _model(wl)
    _, n = oracle.training_offsets(m)
    assert n == N
    assert sum(int(np.prod(s)) for name, s in oracle.training_tensors(m) if len(s) == 1) == Nn
    assert oracle.padded_elems(n, wl.train_shards) == Npad
    assert Npad // wl.train_shards == S
    assert sum(int(np.prod(s)) for _, s in oracle.rollout_tensors(m, wl.tp)) == per_rank
    tbl = oracle.rollout_table(m, wl.tp)
    r, name, off, shape = tbl[-1]
    assert 2 * (off + int(np.prod(shape))) == stream_bytes
    spans = oracle.chunk_spans(stream_bytes, wl.chunk_bytes)
    assert len(spans) == nchunks
    assert spans[-1][1] - spans[-1][0] == last
    # conservation: every weight once, every norm once per rank
    assert wl.tp * per_rank == (N - Nn) + wl.tp * Nn
    # the input generator agrees on N / Npad (independent enumeration)
    assert datagen.flat_sizes(wl.model, wl.train_shards) == (N, Npad)


# ------------------------------------------------------------------ hand-worked example
def _expand(tokens):
    out = []
    for tok in tokens:
        if "+4i+" in tok:
            base, rest = tok.split("+4i+")
            cols = [int(c) for c in rest.split()[0].strip("{}").split(",")]
            out += [int(base) + 4 * i + c for i in range(8) for c in cols]
        elif ".." in tok:
            a, b = tok.split("..")
            out += list(range(int(a), int(b) + 1))
        else:
            out.append(int(tok))
    return out


def test_tiny_worked_example(golden_dir):
    m = Model(1, 8, 2, 2, 2, 4, 4)
    expected = {}
    with open(os.path.join(golden_dir, "tiny_worked_layout.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.split()
            r, name = int(parts[0]), parts[1]
            toks = [t for t in parts[2:] if not t.startswith("i=")]
            expected[(r, name)] = _expand(toks)
    flat = datagen.tagged_flat((1, 8, 2, 2, 2, 4, 4), 1).view(np.uint32)
    _, n = oracle.training_offsets(m)
    assert n == 312
    src = oracle.training_views(flat, m)
    for r in range(2):
        for name, arr in oracle.rollout_rank(src, m, 2, r):
            short = name.split(".")[-1]
            got = arr.ravel().astype(np.int64) - 1  # tag -> element index
            assert got.tolist() == expected[(r, short)], (r, name)


# ------------------------------------------------------------------ tagged brute force
def _grid():
    out = []
    for L, H, Hq, D, F, V in itertools.product((1, 2), (8, 16), (1, 2, 4), (2, 4, 8), (8, 12, 24), (8, 16, 24)):
        for Hkv in [h for h in (1, 2, 4) if Hq % h == 0]:
            for T in (1, 2, 3, 4, 6, 8):
                if Hq % T or Hkv % T or F % T or V % T:
                    continue
                out.append((Model(L, H, Hq, Hkv, D, F, V), T))
    return out


GRID = _grid()


def _source_index(m, offs, T, r, name, i, j):
    """Training element index read by output element (i, j) of rank r's tensor ``name``."""
    H, D, F = m.hidden, m.head_dim, m.ffn
    qh, kh, fr, vr = m.n_q_heads // T, m.n_kv_heads // T, F // T, m.vocab // T
    base = name.split(".")[-1]
    lay = name[: -len(base)]
    if base in ("ln1", "ln2", "final_norm"):
        return offs[name][0] + i
    if base == "embed":
        return offs["embed"][0] + (r * vr + i) * H + j
    if base == "lm_head":
        return offs["lm_head"][0] + (r * vr + i) * H + j
    if base == "qkv":
        if i < qh * D:                        # q rows of heads r*qh .. r*qh+qh-1
            head, d = divmod(i, D)
            return offs[lay + "q"][0] + ((r * qh + head) * D + d) * H + j
        i -= qh * D
        part = "k" if i < kh * D else "v"
        if part == "v":
            i -= kh * D
        head, d = divmod(i, D)
        return offs[lay + part][0] + ((r * kh + head) * D + d) * H + j
    if base == "o":                           # o[H, Hq*D]: input features of this rank's heads
        return offs[lay + "o"][0] + i * (m.n_q_heads * D) + r * qh * D + j
    if base == "gate_up":
        if i < fr:                            # gate rows of FFN units r*fr ..
            return offs[lay + "gate"][0] + (r * fr + i) * H + j
        return offs[lay + "up"][0] + (r * fr + i - fr) * H + j
    if base == "down":                        # down[H, F]: this rank's FFN units
        return offs[lay + "down"][0] + i * F + r * fr + j
    raise AssertionError(name)


def _check_tagged(m, T):
    L, H, Hq, Hkv, D, F, V = m
    flat = datagen.tagged_flat(tuple(m), 1).view(np.uint32)
    offs, n = oracle.training_offsets(m)
    src = oracle.training_views(flat, m)
    seen = np.zeros(n, dtype=np.int64)
    norms = np.zeros(n, dtype=bool)
    for name, (off, shape) in offs.items():
        if len(shape) == 1:
            norms[off:off + shape[0]] = True
    for r in range(T):
        for name, arr in oracle.rollout_rank(src, m, T, r):
            a2 = arr.reshape(arr.shape[0], -1) if arr.ndim == 2 else arr.reshape(-1, 1)
            rows, cols = a2.shape
            for i in range(rows):
                for j in range(cols):
                    e = _source_index(m, offs, T, r, name, i, j if arr.ndim == 2 else 0)
                    assert int(a2[i, j]) == e + 1, (m, T, r, name, i, j)
            np.add.at(seen, a2.ravel().astype(np.int64) - 1, 1)
    assert np.all(seen[~norms] == 1)
    assert np.all(seen[norms] == T)


@pytest.mark.parametrize("part", range(8))
def test_tagged_brute_force(part):
    for m, T in GRID[part::8]:
        _check_tagged(m, T)


def test_grid_covers_unaligned_runs():
    # column-slice runs (o: qh*D, down: F/T) that are not multiples of 4 are in the grid
    runs = {((m.n_q_heads // T) * m.head_dim) % 4 for m, T in GRID} | {(m.ffn // T) % 4 for m, T in GRID}
    assert runs - {0}
    assert len(GRID) > 1000


# ------------------------------------------------------------------ T = 1 identity
@pytest.mark.parametrize("wl", [workloads.TINY], ids=lambda w: w.name)
def test_single_rank_is_plain_cast(wl):
    m = _model(wl)
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=0.01).view(np.uint32)
    _, n = oracle.training_offsets(m)
    stream = oracle.rollout_stream(oracle.training_views(flat, m), m, 1)
    np.testing.assert_array_equal(stream, oracle.rne_bf16(flat[:n]))


# ------------------------------------------------------------------ round-trip inverse
@pytest.mark.parametrize("T", [1, 2, 4])
def test_round_trip_inverse(T):
    m = Model(2, 64, 8, 4, 16, 96, 128)
    flat = datagen.make_flat_numpy(tuple(m), 3, seed=7, specials_frac=0.05).view(np.uint32)
    src = oracle.training_views(flat, m)
    stream = oracle.rollout_stream(src, m, T)
    back = oracle.inverse(oracle.split_stream(stream, m, T), m, T)
    for name, _ in oracle.training_tensors(m):
        # the bf16 bits themselves, against the cast of the original
        np.testing.assert_array_equal(back[name], oracle.rne_bf16(src[name]), err_msg=name)
        # and as values: widened back to fp32 they equal torch's CPU round trip through bfloat16
        # (NaN compares equal to NaN here, whatever bits torch gives it)
        ref = torch.from_numpy(src[name].view(np.float32)).to(torch.bfloat16).to(torch.float32).numpy()
        np.testing.assert_array_equal(oracle.widen_bf16(back[name]).view(np.float32), ref, err_msg=name)


# ------------------------------------------------------------------ chunks
@pytest.mark.parametrize("total,budget", [(5264384, 262144), (48, 16), (16, 16), (64, 1 << 20), (1040, 32)])
def test_chunk_spans(total, budget):
    spans = oracle.chunk_spans(total, budget)
    assert spans[0][0] == 0 and spans[-1][1] == total
    assert len(spans) == -(-total // budget)
    for (a, b), (c, _) in zip(spans, spans[1:]):
        assert b == c and b - a == budget
    assert 0 < spans[-1][1] - spans[-1][0] <= budget


def test_padding_and_shards():
    m = _model(workloads.TINY)
    flat = datagen.make_flat_numpy(workloads.TINY.model, 4, 0)
    _, n = oracle.training_offsets(m)
    assert flat.size == oracle.padded_elems(n, 4) == 2631680
    assert np.all(flat[n:] == 0)
    sh = oracle.shards(flat, 4)
    assert [s.size for s in sh] == [657920] * 4
    assert np.shares_memory(sh[1], flat)


# ------------------------------------------------------------------ training -> training reshard
@pytest.mark.parametrize("w,w2", [(4, 3), (1, 8), (8, 1), (3, 64), (5, 5)])
def test_reshard_keeps_every_element_and_repads(w, w2):
    model = (2, 64, 8, 4, 16, 96, 128)
    flat = datagen.make_flat_numpy(model, w, seed=2, specials_frac=0.05)
    n, npad = datagen.flat_sizes(model, w)
    out = oracle.reshard(flat, n, w2)
    assert out.size == -(-n // (w2 * 256)) * (w2 * 256)  # closed form of the new padding
    assert out.size % (w2 * 256) == 0 and out.size - n < w2 * 256
    assert np.array_equal(out[:n].view(np.uint32), flat[:n].view(np.uint32))  # bit for bit, NaN included
    assert np.all(out[n:].view(np.uint32) == 0)
    back = oracle.reshard(out, n, w)  # and back again
    assert np.array_equal(back.view(np.uint32), flat.view(np.uint32))
    assert [s.size for s in oracle.shards(out, w2)] == [out.size // w2] * w2
