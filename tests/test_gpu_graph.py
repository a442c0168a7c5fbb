"""dr_stage_all, dr_stage_chunk and dr_reshard recorded into a HIP graph and replayed.

These calls only enqueue kernels (no memset node, no allocation, no host
synchronization), so a caller may capture them.  Each replay runs after eager
work that rewrites the source and poisons the outputs, and is compared with the
oracle for the source it saw, and with an eager call of the same plan.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import Model
from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import as_u16, checksums_to_list, new_checksums, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def test_stage_and_reshard_replayed_from_a_graph():
    wl = workloads.TINY
    w, t, b, w2 = wl.train_shards, wl.tp, wl.chunk_bytes, 3
    m = Model(*wl.model)
    flats = [datagen.make_flat_numpy(wl.model, w, seed=s, specials_frac=0.01) for s in (20, 21, 22)]
    n, _ = datagen.flat_sizes(wl.model, w)

    plan = dr.dr_plan_create(wl.model, w, t, b)
    info = dr.dr_plan_get_info(plan)
    rplan = dr.dr_reshard_plan_create(wl.model, w, w2, b)
    rinfo = dr.dr_plan_get_info(rplan)
    S, S2 = info["shard_elems"], rinfo["dst_shard_elems"]
    chunk = 5
    chunk_len = min(b, info["rollout_bytes"] - chunk * b)

    src = torch.from_numpy(flats[0]).cuda()
    shards = [src[i * S:(i + 1) * S] for i in range(w)]
    dst = torch.empty(info["rollout_bytes"], dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    one = torch.empty(chunk_len, dtype=torch.uint8, device="cuda")
    one_ck = new_checksums(1)
    rdst = [torch.empty(S2, dtype=torch.float32, device="cuda") for _ in range(w2)]
    rcks = new_checksums(rinfo["num_chunks"])
    torch.cuda.synchronize()

    say("graph capture: dr_stage_all + dr_stage_chunk + dr_reshard, tiny workload")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st = torch.cuda.current_stream()
        dr.dr_stage_all(plan, shards, dst, cks, st)
        dr.dr_stage_chunk(plan, chunk, shards, one, one_ck, st)
        dr.dr_reshard(rplan, shards, rdst, rcks, st)
    torch.cuda.synchronize()

    edst = torch.empty_like(dst)
    ecks = new_checksums(info["num_chunks"])
    for i, flat in enumerate(flats * 2):
        say("graph replay", i)
        src.copy_(torch.from_numpy(flat))
        dst.fill_(0xEE)
        cks.fill_(-1)
        one.fill_(0xEE)
        one_ck.fill_(-1)
        for d in rdst:
            d.view(torch.int32).fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()

        bits = flat.view(np.uint32)
        want = oracle.rollout_stream(oracle.training_views(bits, m), m, t)
        want_cks = oracle.chunk_checksums(want, b)
        assert np.array_equal(as_u16(dst), want), f"replay {i}: rollout stream"
        assert checksums_to_list(cks) == want_cks, f"replay {i}: checksums"
        want_bytes = want.view(np.uint8)
        assert np.array_equal(one.cpu().numpy(), want_bytes[chunk * b:chunk * b + chunk_len]), f"replay {i}: chunk"
        assert checksums_to_list(one_ck) == [want_cks[chunk]]
        rwant = oracle.reshard(flat, n, w2).view(np.uint32)
        rgot = np.concatenate([d.cpu().numpy().view(np.uint32) for d in rdst])
        assert np.array_equal(rgot, rwant), f"replay {i}: reshard"
        assert checksums_to_list(rcks) == oracle.chunk_checksums(rwant, b)

        # the same plan used eagerly between replays gives the same bytes
        dr.dr_stage_all(plan, shards, edst, ecks)
        torch.cuda.synchronize()
        assert torch.equal(edst, dst)
        assert torch.equal(ecks, cks)
    del g
