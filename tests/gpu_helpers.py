"""Helpers for the GPU tests: device buffers, staging runs, host read-back, and the full-size
comparison of a staged stream with the oracle."""
from __future__ import annotations

import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle
from paper_2607_22614_amd import dr


def say(*a):
    """Names the case on stdout before a GPU step (flushed, so a dead box still shows it)."""
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def require_gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X; none is visible"
    name = torch.cuda.get_device_properties(0).gcnArchName
    assert name.startswith("gfx950"), name


def to_device_shards(flat: np.ndarray, w: int, separate: bool = True):
    """Upload a padded flat fp32 buffer as W device shards.

    separate=True: W independent allocations; False: W views of one allocation.
    Returns (shards, keepalive).
    """
    assert flat.size % w == 0
    s = flat.size // w
    t = torch.from_numpy(flat.view(np.float32))
    if separate:
        shards = [t[i * s:(i + 1) * s].to("cuda") for i in range(w)]
        return shards, shards
    whole = t.to("cuda")
    return [whole[i * s:(i + 1) * s] for i in range(w)], whole


def views_of(flat_dev, w: int):
    s = flat_dev.numel() // w
    return [flat_dev[i * s:(i + 1) * s] for i in range(w)]


def checksums_to_list(cks: torch.Tensor) -> list[tuple[int, int]]:
    a = cks.cpu().numpy().view(np.uint64).reshape(-1, 2)
    return [(int(x), int(y)) for x, y in a]


def new_checksums(n: int) -> torch.Tensor:
    # uint64 pairs (dr_checksum); filled with a pattern so unwritten slots show
    return torch.full((n, 2), -1, dtype=torch.int64, device="cuda")


def stage_all(plan, shards, poison: int = 0xFF):
    info = dr.dr_plan_get_info(plan)
    dst = torch.full((info["rollout_bytes"],), poison, dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    dr.dr_stage_all(plan, shards, dst, cks)
    torch.cuda.synchronize()
    return dst, cks


def as_u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


_M64 = (1 << 64) - 1


def _needs(name):
    """Training tensors one rollout tensor reads."""
    prefix, _, base = name.rpartition(".")
    prefix = prefix + "." if prefix else ""
    return [prefix + t for t in {"qkv": ("q", "k", "v"), "gate_up": ("gate", "up")}.get(base, (base,))]


def host_workers() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def check_against_oracle(wl, info, flat, dst, cks):
    """Every rollout tensor of every rank in `dst` (device bytes) against the oracle, byte for byte,
    and every chunk checksum in `cks` against the oracle's.  The oracle's chunk checksums are
    assembled from its per-tensor pieces with the concatenation law
    s(A||B) = (s1A + s1B, s2A + s2B + |A|*s1B), which test_oracle_checksum pins; the oracle runs on
    a pool of host threads, one rollout tensor at a time, so host memory stays bounded.  `flat` is
    the workload's flat fp32 source (device).  Returns the oracle's chunk checksums."""
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

    workers = host_workers()
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
    want_cks = [tuple(v) for v in sums]
    assert checksums_to_list(cks) == want_cks
    return want_cks


def oracle_chunk_checksums_of(raw: np.ndarray, budget: int) -> list[tuple[int, int]]:
    """oracle.checksum of every chunk of a host byte stream, chunks spread over host threads."""
    spans = oracle.chunk_spans(raw.size, budget)
    with ThreadPoolExecutor(host_workers()) as ex:
        return list(ex.map(lambda ab: oracle.checksum(raw[ab[0]:ab[1]]), spans))
