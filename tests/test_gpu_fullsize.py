"""Parity at the full workload sizes, in the launch configuration bench.py times.

8B shape (automatic tile depth: the deep tiling after a pause and depth 2 right
behind it, identical results) and 32B shape (196.6 GB resident, automatic tile
depth 4): every rollout tensor of every rank is compared with the oracle
byte for byte, and every chunk checksum with the oracle's.  The oracle's chunk
checksums are assembled from its per-tensor pieces with the concatenation law
s(A||B) = (s1A + s1B, s2A + s2B + |A|*s1B), which test_oracle_checksum pins.
The oracle runs on a pool of host threads (numpy releases the GIL in its array
work); the oracle itself is unchanged.
"""
import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _stage(wl):
    """dr_stage_all with the automatic tile depth.  A plan with two tilings stages twice: after a
    pause (deep tiling) and right behind that (depth 2); the two results must be identical, and
    the first is returned for the oracle comparison."""
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    flat = datagen.make_flat_torch(wl.model, wl.train_shards, wl.seed)
    S = info["shard_elems"]
    shards = [flat[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    depths = (4, 2) if info["deep_tile_elems"] else (info["tile_elems"] // 1024,)
    outs = [(torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda"),
             torch.full((info["num_chunks"], 2), -1, dtype=torch.int64, device="cuda")) for _ in depths]
    torch.cuda.synchronize()
    time.sleep(0.01)
    for depth, (dst, cks) in zip(depths, outs):
        say("stage_all", wl.name, "expecting tile depth", depth)
        dr.dr_stage_all(plan, shards, dst, cks)
        assert dr.dr_plan_get_info(plan)["last_tile_depth"] == depth
    torch.cuda.synchronize()
    dst, cks = outs[0]
    for other, other_cks in outs[1:]:
        assert torch.equal(other, dst) and torch.equal(other_cks, cks)
    del outs
    return plan, info, flat, dst, cks


_M64 = (1 << 64) - 1


def _needs(name):
    """Training tensors one rollout tensor reads."""
    prefix, _, base = name.rpartition(".")
    prefix = prefix + "." if prefix else ""
    return [prefix + t for t in {"qkv": ("q", "k", "v"), "gate_up": ("gate", "up")}.get(base, (base,))]


def _check_everything(wl, info, flat, dst, cks):
    m = oracle.Model(*wl.model)
    T, B = wl.tp, wl.chunk_bytes
    offs, _ = oracle.training_offsets(m)
    ranks_of = {}
    for r, name, off, _ in oracle.rollout_table(m, T):
        ranks_of.setdefault(name, []).append((r, off))

    def fetch(t):
        off, shape = offs[t]
        return flat[off:off + int(np.prod(shape))].cpu().numpy().view(np.uint32).reshape(shape)

    def one(name):
        """All ranks' copies of one rollout tensor: byte comparison, then the oracle's checksum
        contributions (chunk, s1, s2 shifted to the piece's word offset in the chunk)."""
        src = {t: fetch(t) for t in _needs(name)}
        parts, count = [], 0
        for r, off in ranks_of[name]:
            want = oracle.rollout_tensor(src, m, T, r, name).ravel()
            got = dst[2 * off:2 * (off + want.size)].cpu().numpy().view(np.uint16)
            if not np.array_equal(got, want):
                bad = np.flatnonzero(got != want)
                return f"rank {r} {name}: {bad.size} elements differ, first {bad[:4]}"
            raw = want.view(np.uint8)
            a, b = 2 * off, 2 * (off + want.size)
            while a < b:
                c = a // B
                e = min(b, (c + 1) * B)
                s1, s2 = oracle.checksum(raw[a - 2 * off:e - 2 * off])
                parts.append((c, s1, (s2 + (a - c * B) // 4 * s1) & _M64))
                a = e
            count += want.size
        return count, parts

    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    names = list(ranks_of)
    say("oracle over", len(names), "rollout tensors x", T, "ranks on", workers, "host threads")
    sums = [[0, 0] for _ in range(info["num_chunks"])]
    total = 0
    with ThreadPoolExecutor(workers) as ex:
        for i, res in enumerate(ex.map(one, names)):
            if isinstance(res, str):
                raise AssertionError(res)
            n, parts = res
            total += n
            for c, s1, s2 in parts:
                sums[c][0] = (sums[c][0] + s1) & _M64
                sums[c][1] = (sums[c][1] + s2) & _M64
            if i % 48 == 47:
                say("checked", i + 1, "of", len(names), "rollout tensors")
    assert 2 * total == info["rollout_bytes"]
    got = cks.cpu().numpy().view(np.uint64).reshape(-1, 2)
    assert [(int(x), int(y)) for x, y in got] == [tuple(v) for v in sums]


def test_8b_every_byte_and_every_checksum():
    """Both tilings against the oracle, then the bounded per-chunk form: 60 dr_stage_chunk calls
    (deep tiling) into their places of a fresh buffer, identical to the checked stream."""
    wl = workloads.EIGHT_B
    plan, info, flat, dst, cks = _stage(wl)
    assert (info["tile_elems"], info["deep_tile_elems"]) == (2048, 4096)
    _check_everything(wl, info, flat, dst, cks)
    S, B = info["shard_elems"], wl.chunk_bytes
    shards = [flat[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    out = torch.full_like(dst, 0xFF)
    out_cks = torch.full_like(cks, -1)
    say("stage_chunk over the 8b stream,", info["num_chunks"], "chunks")
    for c in range(info["num_chunks"]):
        dr.dr_stage_chunk(plan, c, shards, out[c * B:], out_cks[c])
        assert dr.dr_plan_get_info(plan)["last_tile_depth"] == 4
    torch.cuda.synchronize()
    assert torch.equal(out, dst) and torch.equal(out_cks, cks)


def test_32b_every_byte_and_every_checksum():
    wl = workloads.THIRTY_TWO_B
    plan, info, flat, dst, cks = _stage(wl)
    assert (info["tile_elems"], info["deep_tile_elems"]) == (4096, 0)
    _check_everything(wl, info, flat, dst, cks)
