"""Helpers for the GPU tests: device buffers, staging runs and host read-back."""
from __future__ import annotations

import sys

import numpy as np
import torch

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
