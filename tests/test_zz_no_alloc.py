"""dr_stage_chunk_noalloc, the allocation-free variant of dr_stage_chunk, through the C ABI.

Two calls in a row, the second on a smaller chunk of another plan (fewer checksum slots than the
first used), each against dr_stage_chunk on the same chunk: identical bytes, identical checksum,
nothing written outside the chunk; the ragged last chunk too; the CPU-side refusals; the call
recorded into a HIP graph and replayed; and seeded random layouts against the oracle.
"""
import numpy as np
import pytest
import torch

from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import require_gpu, say, to_device_shards

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _case(wl, chunks):
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=0.001)
    shards, keep = to_device_shards(flat, wl.train_shards)
    B = wl.chunk_bytes
    for c in chunks:
        n = B if c + 1 < info["num_chunks"] else info["last_chunk_bytes"]
        say("stage_chunk_noalloc", wl.name, "chunk", c, "of", info["num_chunks"], n, "bytes")
        guard = 4096
        ref = torch.full((n + 2 * guard,), 0xA5, dtype=torch.uint8, device="cuda")
        got = torch.full((n + 2 * guard,), 0x5A, dtype=torch.uint8, device="cuda")
        ref_ck = torch.full((2,), -1, dtype=torch.int64, device="cuda")
        got_ck = torch.full((2,), -1, dtype=torch.int64, device="cuda")
        dr.dr_stage_chunk(plan, c, shards, ref[guard:guard + n], ref_ck)
        dr.dr_stage_chunk_noalloc(plan, c, shards, got[guard:guard + n], got_ck)
        torch.cuda.synchronize()
        assert torch.equal(got[guard:guard + n], ref[guard:guard + n]), (wl.name, c)
        assert torch.equal(got_ck, ref_ck), (wl.name, c)
        assert bool((got[:guard] == 0x5A).all()) and bool((got[guard + n:] == 0x5A).all()), "wrote outside the chunk"
    del keep
    plan.close()


def test_two_calls_in_a_row_the_second_smaller():
    _case(workloads.HALF_B, [0])      # 64 MiB chunk: about 8200 tiles, 256 checksum slots
    _case(workloads.TINY, [3])        # 256 KiB chunk: 32 tiles, 1 slot


def test_every_chunk_of_a_plan_and_the_ragged_last_one():
    wl = workloads.TINY
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    n = dr.dr_plan_get_info(plan)["num_chunks"]
    plan.close()
    _case(wl, list(range(n)))


def test_refusals_launch_nothing():
    wl = workloads.TINY
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed)
    shards, keep = to_device_shards(flat, wl.train_shards)
    dst = torch.empty(wl.chunk_bytes, dtype=torch.uint8, device="cuda")
    ck = torch.empty(2, dtype=torch.int64, device="cuda")
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(plan, info["num_chunks"], shards, dst, ck)
    assert e.value.code == dr.DR_ERANGE
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(plan, 0, shards, dst.data_ptr() + 8, ck)
    assert e.value.code == dr.DR_EINVAL
    host = dr.dr_plan_create_host(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(host, 0, shards, dst, ck)
    assert e.value.code == dr.DR_EINVAL and "host-only" in str(e.value)
    del keep


def test_recorded_in_a_graph_and_replayed():
    """The callers this entry point is for include code under HIP graph capture.  The recorded call
    (stage kernel and chunk sum) replays after eager work that rewrites the source and poisons the
    outputs, and after an eager call on a plan with a 4 MiB budget, which uses more slots of the
    same static array; every replay matches the oracle for the source it saw."""
    import oracle

    wl = workloads.TINY
    m = oracle.Model(*wl.model)
    w, t, b = wl.train_shards, wl.tp, wl.chunk_bytes
    flats = [datagen.make_flat_numpy(wl.model, w, seed=s, specials_frac=0.01) for s in (30, 31, 32)]
    plan = dr.dr_plan_create(wl.model, w, t, b)
    big = dr.dr_plan_create(wl.model, w, t, 4 << 20)
    info = dr.dr_plan_get_info(plan)
    S, chunk = info["shard_elems"], 7
    n = min(b, info["rollout_bytes"] - chunk * b)
    src = torch.from_numpy(flats[0]).cuda()
    shards = [src[i * S:(i + 1) * S] for i in range(w)]
    out = torch.empty(n, dtype=torch.uint8, device="cuda")
    ck = torch.empty(2, dtype=torch.int64, device="cuda")
    bbuf = torch.empty(4 << 20, dtype=torch.uint8, device="cuda")
    bck = torch.empty(2, dtype=torch.int64, device="cuda")
    ref = torch.empty_like(bbuf)
    ref_ck = torch.empty_like(bck)
    torch.cuda.synchronize()
    say("graph capture: dr_stage_chunk_noalloc, tiny workload, chunk", chunk)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dr.dr_stage_chunk_noalloc(plan, chunk, shards, out, ck, torch.cuda.current_stream())
    torch.cuda.synchronize()
    for i, flat in enumerate(flats * 2):
        say("graph replay", i)
        src.copy_(torch.from_numpy(flat))
        out.fill_(0xEE)
        ck.fill_(-1)
        dr.dr_stage_chunk_noalloc(big, 0, shards, bbuf, bck)  # eager: 4 MiB chunk, 32 slots against 1
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, t).view(np.uint8)
        piece = want[chunk * b:chunk * b + n]
        assert np.array_equal(out.cpu().numpy(), piece), f"replay {i}: chunk bytes"
        assert tuple(int(x) for x in ck.cpu().numpy().view(np.uint64)) == oracle.checksum(piece), f"replay {i}"
        assert tuple(int(x) for x in bck.cpu().numpy().view(np.uint64)) == oracle.checksum(want[:4 << 20])
        dr.dr_stage_chunk(big, 0, shards, ref, ref_ck)
        torch.cuda.synchronize()
        assert torch.equal(bbuf, ref) and torch.equal(bck, ref_ck), f"eager call {i}"
    del g
    plan.close()
    big.close()


def test_seeded_random_layouts_against_the_oracle():
    """30 seeded random layouts (shapes, shard counts, TP degrees, budgets from 16 B, all tile
    depths), so the static array serves chunks from one tile to thousands, with single packed slots
    and up to 256 slots of a line each: the first, the last and two other chunks of each, in
    guarded buffers, against the oracle's rollout stream and checksums."""
    import oracle
    from tests.random_layouts import random_layout

    rng = np.random.default_rng(20261202)
    guard = 256
    for i in range(30):
        model, w, t, b = random_layout(rng)
        depth = int(rng.choice([0, 2, 4]))
        flat = datagen.make_flat_numpy(model, w, seed=int(rng.integers(1 << 30)), specials_frac=0.003)
        plan = dr.dr_plan_create(model, w, t, b, tile_depth=depth)
        info = dr.dr_plan_get_info(plan)
        nc = info["num_chunks"]
        m = oracle.Model(*model)
        want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, t).view(np.uint8)
        shards, keep = to_device_shards(flat, w)
        chunks = sorted({0, nc - 1, int(rng.integers(nc)), int(rng.integers(nc))})
        say("noalloc random layout", i, model, "W", w, "T", t, "B", b, "depth", depth, "chunks", chunks, "of", nc)
        for c in chunks:
            lo, hi = c * b, min((c + 1) * b, want.size)
            buf = torch.full((hi - lo + 2 * guard,), 0x5A, dtype=torch.uint8, device="cuda")
            ck = torch.full((2,), -1, dtype=torch.int64, device="cuda")
            dr.dr_stage_chunk_noalloc(plan, c, shards, buf[guard:guard + hi - lo], ck)
            torch.cuda.synchronize()
            got = buf.cpu().numpy()
            assert np.array_equal(got[guard:guard + hi - lo], want[lo:hi]), (i, c)
            assert (got[:guard] == 0x5A).all() and (got[guard + hi - lo:] == 0x5A).all(), (i, c)
            assert tuple(int(x) for x in ck.cpu().numpy().view(np.uint64)) == oracle.checksum(want[lo:hi]), (i, c)
        del keep
        plan.close()
