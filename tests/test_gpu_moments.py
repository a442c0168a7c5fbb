"""GPU tests of the bounded moment offload and the deferred restore (bit-exact).

The host store must hold the oracle's moment stream m_0..m_{W-1} v_0..v_{W-1}
byte for byte after an offload, and a restore into poisoned shards must bring
back every byte, padding included.  Chunk sizes are chosen so chunks straddle
shard and m/v boundaries and the last chunk is ragged.
"""
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import check_against_oracle, checksums_to_list, new_checksums, require_gpu, say, stage_all
from tests.random_layouts import random_layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _moments_case(model, w, t, b, bm, seed, separate=True):
    say("moments", model, "W", w, "Bm", bm)
    plan = dr.dr_plan_create(model, w, t, b, bm)
    info = dr.dr_plan_get_info(plan)
    S, npad = info["shard_elems"], info["padded_elems"]
    m_host, v_host = datagen.make_moments_numpy(npad, seed)
    if separate:
        ms = [torch.from_numpy(m_host[i * S:(i + 1) * S]).cuda() for i in range(w)]
        vs = [torch.from_numpy(v_host[i * S:(i + 1) * S]).cuda() for i in range(w)]
        keep = (ms, vs)
    else:
        md, vd = torch.from_numpy(m_host).cuda(), torch.from_numpy(v_host).cuda()
        ms = [md[i * S:(i + 1) * S] for i in range(w)]
        vs = [vd[i * S:(i + 1) * S] for i in range(w)]
        keep = (md, vd)
    store = np.full(info["moment_bytes"], 0xEE, dtype=np.uint8)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    before = new_checksums(info["num_moment_chunks"])
    dr.dr_moment_checksums(plan, ms, vs, before)
    torch.cuda.synchronize()
    dr.dr_offload_moments(plan, ms, vs, store, side)
    want = oracle.moment_stream(oracle.shards(m_host, w), oracle.shards(v_host, w))
    assert store.size == want.size == 2 * npad * 4
    assert np.array_equal(store, want)
    # the moment chunks' checksums (O5 over fp32 words) against the oracle's
    assert checksums_to_list(before) == oracle.chunk_checksums(want, bm)
    for x in ms + vs:
        x.view(torch.int32).fill_(-1)  # poison: NaN bit patterns everywhere
    torch.cuda.synchronize()
    dr.dr_restore_moments(plan, store, ms, vs, side)
    for i in range(w):
        assert np.array_equal(ms[i].cpu().numpy().view(np.uint32), m_host[i * S:(i + 1) * S].view(np.uint32))
        assert np.array_equal(vs[i].cpu().numpy().view(np.uint32), v_host[i * S:(i + 1) * S].view(np.uint32))
    after = new_checksums(info["num_moment_chunks"])
    dr.dr_moment_checksums(plan, ms, vs, after)
    torch.cuda.synchronize()
    assert torch.equal(after, before)
    return plan, info, keep


def test_tiny_moments_ragged_chunks():
    wl = workloads.TINY
    # 1 MiB + 16: chunks straddle shard and m/v boundaries; last chunk ragged
    plan, info, _ = _moments_case(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, (1 << 20) + 16, seed=4)
    assert info["num_moment_chunks"] == -(-info["moment_bytes"] // ((1 << 20) + 16))
    assert info["moment_bytes"] % ((1 << 20) + 16) != 0


def test_moments_single_chunk_and_views():
    wl = workloads.TINY
    _moments_case(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, 1 << 30, seed=5, separate=False)


def test_moments_tiny_budget_many_chunks():
    model = (2, 64, 8, 4, 16, 96, 128)
    plan, info, _ = _moments_case(model, 3, 2, 4096, 4096 + 48, seed=6)
    assert info["num_moment_chunks"] > 100


def test_seeded_random_moment_budgets():
    """12 seeded random layouts (tests/random_layouts.py) with moment budgets log-uniform from 16 B
    up (at most 2048 moment chunks), so chunks start and end anywhere relative to the shard and
    m/v boundaries; separate allocations or views of one buffer."""
    rng = np.random.default_rng(20260727)
    for _ in range(12):
        model, w, t, b = random_layout(rng)
        npad = datagen.flat_sizes(model, w)[1]
        bm = max(16 * int(2 ** rng.uniform(0, 20)), 16 * -(-8 * npad // (16 * 2048)))
        _moments_case(model, w, t, b, bm, seed=int(rng.integers(1 << 30)), separate=bool(rng.random() < 0.5))


def test_offload_overlaps_staging_on_another_stream():
    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, 64 << 20)
    info = dr.dr_plan_get_info(plan)
    S, npad = info["shard_elems"], info["padded_elems"]
    dev = torch.from_numpy(flat).cuda()
    shards = [dev[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    m_host, v_host = datagen.make_moments_numpy(npad, 8)
    md, vd = torch.from_numpy(m_host).cuda(), torch.from_numpy(v_host).cuda()
    ms = [md[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    vs = [vd[i * S:(i + 1) * S] for i in range(wl.train_shards)]
    dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
    cks = torch.empty((info["num_chunks"], 2), dtype=torch.int64, device="cuda")
    store = np.empty(info["moment_bytes"], dtype=np.uint8)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    say("stage_all + offload overlapped, 0.5B")
    dr.dr_stage_all(plan, shards, dst, cks)          # main stream, asynchronous
    dr.dr_offload_moments(plan, ms, vs, store, side)  # side stream, blocks the host
    torch.cuda.synchronize()
    m = oracle.Model(*wl.model)
    want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, wl.tp)
    assert np.array_equal(dst.cpu().numpy().view(np.uint16), want)
    assert [tuple(int(x) for x in r) for r in cks.cpu().numpy().view(np.uint64)] == \
        oracle.chunk_checksums(want, wl.chunk_bytes)
    assert np.array_equal(store, oracle.moment_stream(oracle.shards(m_host, wl.train_shards),
                                                      oracle.shards(v_host, wl.train_shards)))


def test_offload_waits_for_work_queued_on_the_side_stream():
    """The copies read the moments only after the kernels queued before them on side_stream
    (here: a run of elementwise kernels that finally writes the real values) have finished."""
    wl = workloads.TINY
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, (1 << 20) + 16)
    info = dr.dr_plan_get_info(plan)
    S, npad, W = info["shard_elems"], info["padded_elems"], wl.train_shards
    m_host, v_host = datagen.make_moments_numpy(npad, 9)
    m_src, v_src = torch.from_numpy(m_host).cuda(), torch.from_numpy(v_host).cuda()
    md = torch.zeros(npad, dtype=torch.float32, device="cuda")
    vd = torch.zeros(npad, dtype=torch.float32, device="cuda")
    ms = [md[i * S:(i + 1) * S] for i in range(W)]
    vs = [vd[i * S:(i + 1) * S] for i in range(W)]
    store = np.full(info["moment_bytes"], 0xEE, dtype=np.uint8)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    say("offload after queued side-stream work, tiny")
    with torch.cuda.stream(side):
        for _ in range(200):
            md.add_(1.0)
            vd.add_(1.0)
        md.copy_(m_src)
        vd.copy_(v_src)
    dr.dr_offload_moments(plan, ms, vs, store, side)
    assert np.array_equal(store, oracle.moment_stream(oracle.shards(m_host, W), oracle.shards(v_host, W)))


def test_offload_from_another_thread_while_staging():
    """dr_offload_moments blocks its thread; run it on a second host thread while the main thread
    stages the 0.5B workload repeatedly on the main stream.  Both results are bit-exact."""
    import threading

    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, 32 << 20)
    info = dr.dr_plan_get_info(plan)
    S, npad, W = info["shard_elems"], info["padded_elems"], wl.train_shards
    dev = torch.from_numpy(flat).cuda()
    shards = [dev[i * S:(i + 1) * S] for i in range(W)]
    m_host, v_host = datagen.make_moments_numpy(npad, 10)
    md, vd = torch.from_numpy(m_host).cuda(), torch.from_numpy(v_host).cuda()
    ms = [md[i * S:(i + 1) * S] for i in range(W)]
    vs = [vd[i * S:(i + 1) * S] for i in range(W)]
    store = np.empty(info["moment_bytes"], dtype=np.uint8)
    dst = torch.empty(info["rollout_bytes"], dtype=torch.uint8, device="cuda")
    cks = torch.empty((info["num_chunks"], 2), dtype=torch.int64, device="cuda")
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    errors = []

    def offload():
        try:
            dr.dr_offload_moments(plan, ms, vs, store, side)
        except Exception as e:  # reported by the main thread
            errors.append(e)

    say("offload on a second thread while staging, 0.5B")
    th = threading.Thread(target=offload)
    th.start()
    for _ in range(20):
        dst.fill_(0xFF)
        dr.dr_stage_all(plan, shards, dst, cks)
    torch.cuda.synchronize()
    th.join()
    assert not errors, errors
    m = oracle.Model(*wl.model)
    want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, wl.tp)
    assert np.array_equal(dst.cpu().numpy().view(np.uint16), want)
    assert [tuple(int(x) for x in r) for r in cks.cpu().numpy().view(np.uint64)] == \
        oracle.chunk_checksums(want, wl.chunk_bytes)
    assert np.array_equal(store, oracle.moment_stream(oracle.shards(m_host, W), oracle.shards(v_host, W)))


def test_full_size_adam_workload():
    """The 8B + Adam role switch at full size (seed 4), as bench.py runs it: the offload of the
    64.24 GB moment stream through 512 MiB bounce chunks runs on a second host thread and the side
    stream while dr_stage_all packs the weights on the main stream.  Every byte and every chunk
    checksum of that pack is compared with the oracle, every one of the 120 chunks of the host
    store with the oracle's moment stream (O6; one chunk at a time so host memory stays bounded),
    and the restore into poisoned shards with the original moments, bit for bit."""
    import threading

    wl = workloads.EIGHT_B_ADAM
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, wl.moment_chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    assert info["num_moment_chunks"] == 120 and info["pinned_bytes"] == 2 * wl.moment_chunk_bytes
    S, npad, W = info["shard_elems"], info["padded_elems"], wl.train_shards
    flat = datagen.make_flat_torch(wl.model, W, wl.seed)
    shards = [flat[i * S:(i + 1) * S] for i in range(W)]
    m, v = datagen.make_moments_torch(npad, wl.seed)
    ms = [m[i * S:(i + 1) * S] for i in range(W)]
    vs = [v[i * S:(i + 1) * S] for i in range(W)]
    dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
    cks = torch.full((info["num_chunks"], 2), -1, dtype=torch.int64, device="cuda")
    say("allocating a", info["moment_bytes"], "byte host store")
    store = torch.empty(info["moment_bytes"], dtype=torch.uint8)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    errors = []

    def offload():
        try:
            dr.dr_offload_moments(plan, ms, vs, store, side)
        except Exception as e:  # reported on the main thread
            errors.append(e)

    mcks = new_checksums(info["num_moment_chunks"])
    say("moment checksums 8b_adam")
    dr.dr_moment_checksums(plan, ms, vs, mcks)
    torch.cuda.synchronize()
    say("offload 8b_adam on a second thread, pack on the main stream meanwhile")
    th = threading.Thread(target=offload)
    th.start()
    time.sleep(0.2)  # the offload is in full flow when the pack starts
    dr.dr_stage_all(plan, shards, dst, cks)
    torch.cuda.current_stream().synchronize()
    assert th.is_alive(), "the offload ended before the pack: nothing overlapped"
    th.join()
    assert not errors, errors
    say("pack under the offload against the oracle")
    check_against_oracle(wl, info, flat, dst, cks)
    del dst, cks, shards
    # the host store against the oracle's O6 stream, chunk by chunk: the stream's bytes [a, b) are
    # the O6 concatenation of the parts of every shard that fall inside [a, b)
    Bm, sb = wl.moment_chunk_bytes, 4 * S
    shard_bytes = [x.view(torch.uint8) for x in ms + vs]
    moment_cks = checksums_to_list(mcks)
    empty = np.empty(0, dtype=np.uint8)
    say("host store against the oracle,", info["num_moment_chunks"], "chunks")
    for k in range(info["num_moment_chunks"]):
        a, b = k * Bm, min((k + 1) * Bm, info["moment_bytes"])
        parts = []
        for i, x in enumerate(shard_bytes):
            lo, hi = max(a, i * sb), min(b, (i + 1) * sb)
            parts.append(x[lo - i * sb:hi - i * sb].cpu().numpy() if lo < hi else empty)
        want = oracle.moment_stream(parts[:W], parts[W:])
        assert want.size == b - a
        assert np.array_equal(store[a:b].numpy(), want), f"moment chunk {k}"
        assert moment_cks[k] == oracle.checksum(want), f"checksum of moment chunk {k}"
    m_ref, v_ref = m.clone(), v.clone()
    m.view(torch.int32).fill_(-1)
    v.view(torch.int32).fill_(-1)
    torch.cuda.synchronize()
    say("restore 8b_adam")
    dr.dr_restore_moments(plan, store, ms, vs, side)
    assert torch.equal(m.view(torch.int32), m_ref.view(torch.int32))
    assert torch.equal(v.view(torch.int32), v_ref.view(torch.int32))
    again = new_checksums(info["num_moment_chunks"])
    dr.dr_moment_checksums(plan, ms, vs, again)
    torch.cuda.synchronize()
    assert torch.equal(again, mcks)


def test_deferred_restore_overlaps_compute_on_the_main_stream():
    wl = workloads.TINY
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, (1 << 20) + 16)
    info = dr.dr_plan_get_info(plan)
    S, npad, W = info["shard_elems"], info["padded_elems"], wl.train_shards
    m_host, v_host = datagen.make_moments_numpy(npad, 11)
    md, vd = torch.from_numpy(m_host).cuda(), torch.from_numpy(v_host).cuda()
    ms = [md[i * S:(i + 1) * S] for i in range(W)]
    vs = [vd[i * S:(i + 1) * S] for i in range(W)]
    store = np.empty(info["moment_bytes"], dtype=np.uint8)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    dr.dr_offload_moments(plan, ms, vs, store, side)
    md.view(torch.int32).fill_(-1)
    vd.view(torch.int32).fill_(-1)
    torch.cuda.synchronize()
    a = torch.randn(2048, 2048, device="cuda")
    say("deferred restore with compute on the main stream")
    dr.dr_restore_moments_begin(plan, store, ms, vs, side)
    with pytest.raises(dr.DrError) as e:  # one at a time per plan
        dr.dr_restore_moments_begin(plan, store, ms, vs, side)
    assert "in flight" in str(e.value)
    with pytest.raises(dr.DrError) as e:  # the bounce buffers are taken until _end
        dr.dr_offload_moments(plan, ms, vs, store, side)
    assert e.value.code == dr.DR_EINVAL and "in flight" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_restore_moments(plan, store, ms, vs, side)
    assert e.value.code == dr.DR_EINVAL and "in flight" in str(e.value)
    x = a
    for _ in range(20):  # the "first step" runs meanwhile
        x = torch.tanh(x @ a) * 0.5
    dr.dr_restore_moments_end(plan)
    torch.cuda.synchronize()
    assert np.array_equal(md.cpu().numpy().view(np.uint32), m_host.view(np.uint32))
    assert np.array_equal(vd.cpu().numpy().view(np.uint32), v_host.view(np.uint32))
    assert bool(torch.isfinite(x).all())
    with pytest.raises(dr.DrError):
        dr.dr_restore_moments_end(plan)  # nothing left in flight


def test_plan_destroy_waits_for_a_deferred_restore():
    wl = workloads.TINY
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, 1 << 16)
    info = dr.dr_plan_get_info(plan)
    S, W = info["shard_elems"], wl.train_shards
    dev = torch.zeros(2 * S * W, dtype=torch.float32, device="cuda")
    ms = [dev[i * S:(i + 1) * S] for i in range(W)]
    vs = [dev[(W + i) * S:(W + i + 1) * S] for i in range(W)]
    store = np.arange(info["moment_bytes"] // 4, dtype=np.uint32)
    dr.dr_restore_moments_begin(plan, store, ms, vs, torch.cuda.Stream())
    plan.close()  # joins the restore thread
    torch.cuda.synchronize()
    assert np.array_equal(dev.cpu().numpy().view(np.uint32), store)


def test_offload_and_restore_resume_from_any_chunk():
    """An offload interrupted after chunk k and restarted at k fills the same host store as one
    call; ranges touch only their own chunks, in any order; a restore in ranges brings back every
    byte; ranges past the last chunk are refused (DR_ERANGE) before anything moves."""
    wl = workloads.TINY
    bm = (1 << 20) + 16
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, bm)
    info = dr.dr_plan_get_info(plan)
    S, npad, W, K = info["shard_elems"], info["padded_elems"], wl.train_shards, info["num_moment_chunks"]
    assert K > 12
    m_host, v_host = datagen.make_moments_numpy(npad, 11)
    md, vd = torch.from_numpy(m_host).cuda(), torch.from_numpy(v_host).cuda()
    ms = [md[i * S:(i + 1) * S] for i in range(W)]
    vs = [vd[i * S:(i + 1) * S] for i in range(W)]
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    want = oracle.moment_stream(oracle.shards(m_host, W), oracle.shards(v_host, W))
    say("moment ranges, tiny, K", K)
    store = np.full(info["moment_bytes"], 0xEE, dtype=np.uint8)
    dr.dr_offload_moments_range(plan, ms, vs, store, 0, 3, side)  # "interrupted" after chunk 3
    assert np.array_equal(store[:3 * bm], want[:3 * bm])
    assert bool((store[3 * bm:] == 0xEE).all()), "a range wrote past its chunks"
    dr.dr_offload_moments_range(plan, ms, vs, store, 3, K - 3, side)  # resumed
    assert np.array_equal(store, want)
    store2 = np.full(info["moment_bytes"], 0xEE, dtype=np.uint8)
    for first, count in ((10, K - 10), (0, 4), (4, 6), (K, 0)):
        dr.dr_offload_moments_range(plan, ms, vs, store2, first, count, side)
    assert np.array_equal(store2, want)
    for first, count in ((K, 1), (0, K + 1), (K + 1, 0)):
        with pytest.raises(dr.DrError) as e:
            dr.dr_offload_moments_range(plan, ms, vs, store2, first, count, side)
        assert e.value.code == dr.DR_ERANGE
        with pytest.raises(dr.DrError) as e:
            dr.dr_restore_moments_range(plan, store2, ms, vs, first, count, side)
        assert e.value.code == dr.DR_ERANGE
    md.view(torch.int32).fill_(-1)
    vd.view(torch.int32).fill_(-1)
    torch.cuda.synchronize()
    dr.dr_restore_moments_range(plan, store, ms, vs, 7, K - 7, side)
    dr.dr_restore_moments_range(plan, store, ms, vs, 0, 7, side)
    assert np.array_equal(md.cpu().numpy().view(np.uint32), m_host.view(np.uint32))
    assert np.array_equal(vd.cpu().numpy().view(np.uint32), v_host.view(np.uint32))
