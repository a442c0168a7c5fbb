"""GPU parity of the training -> training reshard (dr_reshard) against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import checksums_to_list, new_checksums, oracle_chunk_checksums_of, require_gpu, say
from tests.random_layouts import random_reshard

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _run(model, w, w2, b, flat, views=False):
    say("reshard", model, w, "->", w2, "B", b)
    plan = dr.dr_reshard_plan_create(model, w, w2, b)
    info = dr.dr_plan_get_info(plan)
    n, npad = datagen.flat_sizes(model, w)
    S, S2 = info["shard_elems"], info["dst_shard_elems"]
    src = [torch.from_numpy(flat[i * S:(i + 1) * S]).cuda() for i in range(w)]
    if views:
        whole = torch.full((S2 * w2,), -1, dtype=torch.int32, device="cuda").view(torch.float32)
        dst = [whole[i * S2:(i + 1) * S2] for i in range(w2)]
    else:
        dst = [torch.full((S2,), -1, dtype=torch.int32, device="cuda").view(torch.float32) for _ in range(w2)]
    cks = new_checksums(info["num_chunks"])
    dr.dr_reshard(plan, src, dst, cks)
    torch.cuda.synchronize()
    want = oracle.reshard(flat, n, w2).view(np.uint32)
    got = np.concatenate([d.cpu().numpy().view(np.uint32) for d in dst])
    assert np.array_equal(got, want)
    assert checksums_to_list(cks) == oracle.chunk_checksums(want, b)


@pytest.mark.parametrize("w,w2,b", [(4, 3, 256 * 1024), (4, 4, 1 << 20), (1, 8, 4096 + 16), (8, 1, 1 << 16),
                                    (3, 64, 16 * 1000)])
def test_tiny_workload_reshard(w, w2, b):
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, w, wl.seed, specials_frac=0.01)
    _run(wl.model, w, w2, b, flat)


def test_small_budget_and_views():
    model = (1, 24, 4, 4, 6, 20, 8)
    flat = datagen.make_flat_numpy(model, 7, seed=3, specials_frac=0.1)
    _run(model, 7, 5, 16, flat)
    _run(model, 7, 5, 48, flat, views=True)


def test_seeded_random_reshards():
    """40 seeded random reshard layouts (tests/random_layouts.py) up to 4 M elements, W -> W' in
    both directions, budgets from 16 B up; shard allocations or views of one buffer."""
    rng = np.random.default_rng(20260725)
    for _ in range(40):
        model, w, w2, b = random_reshard(rng)
        flat = datagen.make_flat_numpy(model, w, seed=int(rng.integers(1 << 30)), specials_frac=0.003)
        _run(model, w, w2, b, flat, views=bool(rng.random() < 0.5))


def test_half_b_workload_reshard():
    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    _run(wl.model, wl.train_shards, 6, wl.chunk_bytes, flat)


def _check_8b_reshard(out, cks, want, want_cks, B):
    """Destination bytes against the oracle's, one chunk at a time, and every chunk checksum."""
    w32 = want.view(np.int32)
    e = B // 4
    for c in range(len(want_cks)):
        assert np.array_equal(out[c * e:(c + 1) * e].cpu().numpy(), w32[c * e:(c + 1) * e]), f"chunk {c}"
    assert checksums_to_list(cks) == want_cks


def test_8b_reshard_8_to_6_in_hbm_and_through_host():
    """The 8B training state re-cut from 8 to 6 shards, in HBM (dr_reshard) and through two pinned
    host buffers (dr_reshard_through_host): every destination byte and every one of the 120 chunk
    checksums of both against the oracle."""
    wl = workloads.EIGHT_B
    plan = dr.dr_reshard_plan_create(wl.model, 8, 6, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    n, S, S2, B = info["n_elems"], info["shard_elems"], info["dst_shard_elems"], wl.chunk_bytes
    flat = datagen.make_flat_torch(wl.model, 8, wl.seed)
    src = [flat[i * S:(i + 1) * S] for i in range(8)]
    say("oracle reshard of the 8b state, 8 -> 6")
    want = oracle.reshard(flat[:n].cpu().numpy(), n, 6)
    want_cks = oracle_chunk_checksums_of(want.view(np.uint8), B)
    assert len(want_cks) == info["num_chunks"] == 120
    for name, call in (("dr_reshard", dr.dr_reshard), ("dr_reshard_through_host", dr.dr_reshard_through_host)):
        out = torch.full((S2 * 6,), -1, dtype=torch.int32, device="cuda")
        dst = [out[i * S2:(i + 1) * S2].view(torch.float32) for i in range(6)]
        cks = new_checksums(info["num_chunks"])
        say(name, "8b 8->6")
        call(plan, src, dst, cks)
        torch.cuda.synchronize()
        _check_8b_reshard(out, cks, want, want_cks, B)
        del out, dst, cks


# ------------------------------------------------------------------ the same move through host memory
def _through_host(model, w, w2, b, flat, calls=1):
    say("reshard_through_host", model, w, "->", w2, "B", b)
    plan = dr.dr_reshard_plan_create(model, w, w2, b)
    info = dr.dr_plan_get_info(plan)
    n, _ = datagen.flat_sizes(model, w)
    S, S2 = info["shard_elems"], info["dst_shard_elems"]
    src = [torch.from_numpy(flat[i * S:(i + 1) * S]).cuda() for i in range(w)]
    want = oracle.reshard(flat, n, w2).view(np.uint32)
    want_cks = oracle.chunk_checksums(want, b)
    for _ in range(calls):
        whole = torch.full((S2 * w2,), -1, dtype=torch.int32, device="cuda").view(torch.float32)
        dst = [whole[i * S2:(i + 1) * S2] for i in range(w2)]
        cks = new_checksums(info["num_chunks"])
        dr.dr_reshard_through_host(plan, src, dst, cks)
        torch.cuda.synchronize()
        assert np.array_equal(whole.cpu().numpy().view(np.uint32), want)
        assert checksums_to_list(cks) == want_cks


@pytest.mark.parametrize("w,w2,b", [(4, 3, 256 * 1024), (1, 8, 4096 + 16), (8, 1, 1 << 16), (3, 64, 16 * 1000),
                                    (4, 4, 1 << 30)])
def test_tiny_workload_reshard_through_host(w, w2, b):
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, w, wl.seed, specials_frac=0.01)
    _through_host(wl.model, w, w2, b, flat, calls=2)


def test_half_b_workload_reshard_through_host():
    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    _through_host(wl.model, wl.train_shards, 6, wl.chunk_bytes, flat)
