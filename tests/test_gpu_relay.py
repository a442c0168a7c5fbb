"""GPU tests of the weight path through host memory (dr_stage_through_host).

The relayed rollout stream and its checksums must equal the oracle's (small
workloads) and dr_stage_all's output (full 8B shape), byte for byte, whatever
the chunk budget, across repeated calls on one plan.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import Model
from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import (as_u16, check_against_oracle, checksums_to_list, new_checksums, require_gpu, say,
                               to_device_shards)
from tests.random_layouts import random_layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _relay_vs_oracle(model, w, t, b, flat, calls=1, tile_depth=0):
    say("stage_through_host", model, "W", w, "T", t, "B", b, "tile_depth", tile_depth)
    plan = dr.dr_plan_create(model, w, t, b, tile_depth=tile_depth)
    info = dr.dr_plan_get_info(plan)
    shards, keep = to_device_shards(flat, w)
    m = Model(*model)
    want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, t)
    want_cks = oracle.chunk_checksums(want, b)
    for _ in range(calls):
        dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
        cks = new_checksums(info["num_chunks"])
        dr.dr_stage_through_host(plan, shards, dst, cks)
        torch.cuda.synchronize()
        assert np.array_equal(as_u16(dst), want)
        assert checksums_to_list(cks) == want_cks


def test_tiny_workload_through_host():
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=0.001)
    _relay_vs_oracle(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat, calls=3)


def test_half_b_workload_through_host():
    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    _relay_vs_oracle(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat)


@pytest.mark.parametrize("b", [16, 48, 4096 + 16, 1 << 30])
def test_small_budgets_and_single_chunk(b):
    model = (2, 24, 8, 8, 3, 40, 64)
    flat = datagen.make_flat_numpy(model, 3, seed=12, specials_frac=0.02)
    _relay_vs_oracle(model, 3, 2, b, flat, calls=2)


def test_seeded_random_layouts_through_host():
    """20 seeded random layouts (tests/random_layouts.py) through the host relay, each relayed
    twice on its plan, automatic (chunks at depth 4) and depth 2 in turn; a budget past the stream
    is replaced by one just covering it (one chunk, without pinning a GiB per case)."""
    rng = np.random.default_rng(20260726)
    for i in range(20):
        model, w, t, b = random_layout(rng)
        flat = datagen.make_flat_numpy(model, w, seed=int(rng.integers(1 << 30)), specials_frac=0.003)
        info = dr.dr_plan_get_info(dr.dr_plan_create_host(model, w, t, b))
        if b >= info["rollout_bytes"]:
            b = 16 * -(-info["rollout_bytes"] // 16)
        _relay_vs_oracle(model, w, t, b, flat, calls=2, tile_depth=2 * (i % 2))


def test_relay_on_a_side_stream_then_read_on_main():
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed)
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    shards, keep = to_device_shards(flat, wl.train_shards)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    dst = torch.zeros(info["rollout_bytes"], dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    dr.dr_stage_through_host(plan, shards, dst, cks, stream=s)
    torch.cuda.current_stream().wait_stream(s)  # the stream saw the last reload
    copy = dst.clone()                            # read on the main stream
    torch.cuda.synchronize()
    m = Model(*wl.model)
    want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, wl.tp)
    assert np.array_equal(as_u16(copy), want)


def test_8b_through_host_against_the_oracle():
    """The paper's weight path at the 8B shape: dr_stage_through_host's every byte and every chunk
    checksum against the oracle (and equal to dr_stage_all's)."""
    wl = workloads.EIGHT_B
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    flat = datagen.make_flat_torch(wl.model, wl.train_shards, wl.seed)
    S = info["shard_elems"]
    shards = [flat[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    say("stage_through_host 8b")
    dr.dr_stage_through_host(plan, shards, dst, cks)
    torch.cuda.synchronize()
    check_against_oracle(wl, info, flat, dst, cks)
    ref = torch.empty_like(dst)
    ref_cks = new_checksums(info["num_chunks"])
    dr.dr_stage_all(plan, shards, ref, ref_cks)
    torch.cuda.synchronize()
    assert torch.equal(dst, ref) and torch.equal(cks, ref_cks)


def test_relay_waits_for_earlier_work_on_the_callers_stream():
    """Work queued on the caller's stream before the call, with no host synchronization, is ordered
    before the relay on both sides: a long run of kernels that finally writes the source is seen
    by the packing, and a reader of the old destination queued before the call still reads the
    old bytes, although the reload runs on the plan's own copy stream."""
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=0.001)
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    S = info["shard_elems"]
    real = torch.from_numpy(flat).cuda()
    src = torch.zeros_like(real)
    shards = [src[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    dst = torch.full((info["rollout_bytes"],), 0x5A, dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    snapshot = torch.empty_like(dst)
    torch.cuda.synchronize()
    say("relay behind 600 queued kernels, tiny")
    for _ in range(300):           # delay: the source is garbage until the last copy
        src.add_(1.0)
        src.mul_(0.5)
    src.copy_(real)
    snapshot.copy_(dst)            # a reader of the old destination, queued before the call
    dr.dr_stage_through_host(plan, shards, dst, cks)
    torch.cuda.synchronize()
    assert bool((snapshot == 0x5A).all()), "the reload overwrote the destination before an earlier reader"
    m = Model(*wl.model)
    want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, wl.tp)
    assert np.array_equal(as_u16(dst), want)
    assert checksums_to_list(cks) == oracle.chunk_checksums(want, wl.chunk_bytes)
