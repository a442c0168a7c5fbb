"""Parity at the full workload sizes, in the launch configuration bench.py times.

8B shape (automatic tile depth: the deep tiling after a pause and depth 2 right
behind it, identical results) and 32B shape (196.6 GB resident, automatic tile
depth 4): every rollout tensor of every rank is compared with the oracle
byte for byte, and every chunk checksum with the oracle's.  The oracle's chunk
checksums are assembled from its per-tensor pieces with the concatenation law
s(A||B) = (s1A + s1B, s2A + s2B + |A|*s1B), which test_oracle_checksum pins.
The oracle runs on a pool of host threads (numpy releases the GIL in its array
work); the oracle itself is unchanged (tests/gpu_helpers.check_against_oracle).
"""
import time

import pytest
import torch

from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import check_against_oracle, require_gpu, say

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


def test_8b_every_byte_and_every_checksum():
    """Both tilings against the oracle, then the bounded per-chunk form: 60 dr_stage_chunk calls
    (deep tiling) into their places of a fresh buffer, identical to the checked stream."""
    wl = workloads.EIGHT_B
    plan, info, flat, dst, cks = _stage(wl)
    assert (info["tile_elems"], info["deep_tile_elems"]) == (2048, 4096)
    check_against_oracle(wl, info, flat, dst, cks)
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
    check_against_oracle(wl, info, flat, dst, cks)
