"""GPU parity of the HIP staging path against the CPU oracle (bit-exact).

Every case runs the library through the C ABI (ctypes binding) on the GPU and
compares, byte for byte, the rollout stream and the per-chunk checksums with
what the oracle computes from the same seeded inputs.
"""
import gc
import time

import numpy as np
import pytest
import torch

import oracle
from oracle import Model
from paper_2607_22614_amd import datagen, dr, workloads
from tests.gpu_helpers import as_u16, checksums_to_list, new_checksums, require_gpu, say, to_device_shards
from tests.random_layouts import random_layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _oracle(flat_bits, model, t, chunk_bytes):
    m = Model(*model)
    stream = oracle.rollout_stream(oracle.training_views(flat_bits, m), m, t)
    return stream, oracle.chunk_checksums(stream, chunk_bytes)


def _run_and_compare(model, w, t, b, flat, separate=True, tile_depth=0):
    """Stages with the given tile depth and compares with the oracle.  An automatic plan that holds
    two tilings is run twice: after a pause (its deep tiling, depth 4) and right behind that call
    (depth 2); both results are compared."""
    say("stage_all", model, "W", w, "T", t, "B", b, "separate", separate, "tile_depth", tile_depth)
    plan = dr.dr_plan_create(model, w, t, b, tile_depth=tile_depth)
    info = dr.dr_plan_get_info(plan)
    if tile_depth:
        assert info["tile_elems"] == 1024 * tile_depth and info["deep_tile_elems"] == 0
    depths = (4, 2) if info["deep_tile_elems"] else (info["tile_elems"] // 1024,)
    shards, keep = to_device_shards(flat, w, separate)
    runs = [(torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda"),
             new_checksums(info["num_chunks"])) for _ in depths]
    torch.cuda.synchronize()
    time.sleep(0.005)  # more than the 2 ms after which an automatic plan takes its deep tiling
    for depth, (dst, cks) in zip(depths, runs):
        dr.dr_stage_all(plan, shards, dst, cks)  # the second call queues right behind the first
        assert dr.dr_plan_get_info(plan)["last_tile_depth"] == depth
    torch.cuda.synchronize()
    want, want_cks = _oracle(flat.view(np.uint32), model, t, b)
    for depth, (dst, cks) in zip(depths, runs):
        got = as_u16(dst)
        if not np.array_equal(got, want):
            bad = np.flatnonzero(got != want)
            raise AssertionError(f"depth {depth}: {bad.size} elements differ, first at {bad[:8]}: "
                                 f"got {got[bad[:8]]} want {want[bad[:8]]}")
        assert checksums_to_list(cks) == want_cks, f"depth {depth}"
    dst, cks = runs[-1]
    return plan, shards, keep, dst, cks


# ------------------------------------------------------------------ the five workloads' small members
@pytest.mark.parametrize("tile_depth", [0, 4])
def test_tiny_workload(tile_depth):
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed)
    _run_and_compare(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat, tile_depth=tile_depth)


def test_tiny_workload_shard_views_of_one_buffer():
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed)
    _run_and_compare(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat, separate=False)


@pytest.mark.parametrize("tile_depth", [0, 4])
def test_half_b_workload_with_special_values(tile_depth):
    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    bits = flat.view(np.uint32)
    nan = (bits & 0x7FFFFFFF) > 0x7F800000
    assert nan.sum() > 50000  # the recipe really carries NaN, ties, subnormals
    _run_and_compare(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat, tile_depth=tile_depth)


def test_automatic_depth_follows_the_issue_pattern():
    """An automatic plan's dr_stage_all takes its deep tiling (depth 4) after a pause and depth 2
    when queued behind another pack or issued within 2 ms of the previous one's end, whichever plan
    launched it (a chunk call included); dr_stage_chunk always takes depth 4; explicit depths never
    change.  Every result equals the oracle's."""
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=0.001)
    auto = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    fixed = {k: dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, tile_depth=k) for k in (2, 4)}
    info = dr.dr_plan_get_info(auto)
    assert (info["tile_elems"], info["deep_tile_elems"]) == (2048, 4096)
    shards, keep = to_device_shards(flat, wl.train_shards)
    want, want_cks = _oracle(flat.view(np.uint32), wl.model, wl.tp, wl.chunk_bytes)
    B, n = wl.chunk_bytes, info["num_chunks"]

    def fresh():
        return (torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda"), new_checksums(n))

    def check(out, what):
        assert np.array_equal(as_u16(out[0]), want), what
        assert checksums_to_list(out[1]) == want_cks, what

    def pause(seconds):
        torch.cuda.synchronize()
        time.sleep(seconds)

    def depth(plan):
        return dr.dr_plan_get_info(plan)["last_tile_depth"]

    say("automatic tile depth by issue pattern")
    outs = [fresh() for _ in range(8)]
    seen = []
    gc.disable()  # the hot cases need consecutive calls within 2 ms; no collector pause between them
    try:
        _issue_pattern(auto, fixed, shards, outs, seen, pause, depth, n, B, info)
    finally:
        gc.enable()
    assert seen == [4, 2, 2, 4, 2, 2] + [4] * n + [2]
    for i in range(8):
        check(outs[i], f"call {i}")
    del keep


def _issue_pattern(auto, fixed, shards, outs, seen, pause, depth, n, B, info):
    pause(0.01)
    dr.dr_stage_all(auto, shards, *outs[0]); seen.append(depth(auto))   # after a pause: deep
    dr.dr_stage_all(auto, shards, *outs[1]); seen.append(depth(auto))   # queued behind: depth 2
    torch.cuda.synchronize()
    dr.dr_stage_all(auto, shards, *outs[2]); seen.append(depth(auto))   # right after the end: depth 2
    pause(0.01)
    dr.dr_stage_all(fixed[4], shards, *outs[3]); seen.append(depth(fixed[4]))  # explicit: 4
    dr.dr_stage_all(auto, shards, *outs[4]); seen.append(depth(auto))   # behind another plan's pack: 2
    pause(0.01)
    dr.dr_stage_all(fixed[2], shards, *outs[5]); seen.append(depth(fixed[2]))  # explicit: 2, even after a pause
    pause(0.01)
    dst, cks = outs[6]
    for c in range(n):  # chunk by chunk: depth 4 after a pause and queued behind each other
        a, e = c * B, min((c + 1) * B, info["rollout_bytes"])
        dr.dr_stage_chunk(auto, c, shards, dst[a:e], cks[c])
        seen.append(depth(auto))
    dr.dr_stage_all(auto, shards, *outs[7]); seen.append(depth(auto))   # behind the chunk calls: 2
    torch.cuda.synchronize()


def test_two_threads_staging_their_own_plans():
    """Two host threads, each with its own automatic plan and stream, stage 12 times each at the
    same time (the per-device drain estimate is shared and raced on); every result equals the
    oracle's."""
    import threading

    cases = [(workloads.TINY, 3), (workloads.HALF_B, 4)]
    work = []
    for wl, seed in cases:
        flat = datagen.make_flat_numpy(wl.model, wl.train_shards, seed, specials_frac=0.01)
        plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
        info = dr.dr_plan_get_info(plan)
        shards, keep = to_device_shards(flat, wl.train_shards)
        outs = [(torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda"),
                 new_checksums(info["num_chunks"])) for _ in range(3)]
        stream = torch.cuda.Stream()
        stream.synchronize()
        work.append((wl, flat, plan, shards, keep, outs, stream))
    torch.cuda.synchronize()
    errors = []

    def run(plan, shards, outs, stream):
        try:
            for i in range(12):
                dst, cks = outs[i % 3]
                dr.dr_stage_all(plan, shards, dst, cks, stream=stream)
                if i % 4 == 3:
                    stream.synchronize()
                    time.sleep(0.003)
            stream.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    say("two threads staging tiny and 0.5B plans")
    threads = [threading.Thread(target=run, args=(w[2], w[3], w[5], w[6])) for w in work]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    for wl, flat, plan, shards, keep, outs, stream in work:
        want, want_cks = _oracle(flat.view(np.uint32), wl.model, wl.tp, wl.chunk_bytes)
        for dst, cks in outs:
            assert np.array_equal(as_u16(dst), want), wl.name
            assert checksums_to_list(cks) == want_cks, wl.name


def test_concurrent_calls_with_different_tilings_keep_their_checksums():
    """A chunk call (deep tiling) and a whole-stream call right behind it (depth 2) of one automatic
    plan, in flight at once on two streams.  Chunk 18's deep tiles have about the same tile indices
    as depth-2 tiles of the middle of the stream, so the tilings must keep separate per-tile
    partial slots: the chunk's and the stream's bytes and checksums equal the oracle's."""
    wl = workloads.HALF_B
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=wl.specials_frac)
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    assert info["deep_tile_elems"] and info["num_chunks"] == 19
    shards, keep = to_device_shards(flat, wl.train_shards)
    B = wl.chunk_bytes
    chunk = (torch.full((B,), 0xFF, dtype=torch.uint8, device="cuda"), new_checksums(1))
    whole = (torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda"),
             new_checksums(info["num_chunks"]))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for st in streams:
        st.synchronize()  # torch creates a stream on first use (about 3 ms): not between the two calls
    torch.cuda.synchronize()
    time.sleep(0.01)
    say("a chunk call and a whole-stream call in flight with different tilings, 0.5B")
    dr.dr_stage_chunk(plan, 18, shards, chunk[0], chunk[1], stream=streams[0])
    depths = [dr.dr_plan_get_info(plan)["last_tile_depth"]]
    dr.dr_stage_all(plan, shards, whole[0], whole[1], stream=streams[1])
    depths.append(dr.dr_plan_get_info(plan)["last_tile_depth"])
    torch.cuda.synchronize()
    assert depths == [4, 2]
    want, want_cks = _oracle(flat.view(np.uint32), wl.model, wl.tp, B)
    raw = want.view(np.uint8)
    n = info["rollout_bytes"] - 18 * B
    assert np.array_equal(chunk[0][:n].cpu().numpy(), raw[18 * B:18 * B + n])
    assert checksums_to_list(chunk[1])[0] == want_cks[18]
    assert np.array_equal(as_u16(whole[0]), want)
    assert checksums_to_list(whole[1]) == want_cks
    del keep


# ------------------------------------------------------------------ cast edge values
def test_every_special_category_and_nan_payload():
    model = (2, 64, 8, 4, 16, 96, 128)
    flat = datagen.make_flat_numpy(model, 2, seed=21, specials_frac=0.3)
    bits = flat.view(np.uint32)
    rng = np.random.default_rng(4)
    n = oracle.training_offsets(Model(*model))[1]
    extra = np.array([0x7F800001, 0xFF800001, 0x7FA00000, 0x7FFFFFFF, 0xFFFFFFFF, 0x7F7F8000, 0xFF7F8000,
                      0x7F7FFFFF, 0x007FFFFF, 0x807F8000, 0x00008000, 0x00018000, 0x3F808000, 0x3F818000],
                     dtype=np.uint32)
    pos = rng.choice(n, size=extra.size * 50, replace=False)
    bits[pos] = np.tile(extra, 50)
    for t in (1, 2, 4):
        for depth in (2, 4):
            _run_and_compare(model, 2, t, 4096, flat, tile_depth=depth)


def test_exhaustive_upper_halves_through_the_kernel():
    # every sign/exponent/top-mantissa pattern with the rounding-critical low halves
    hi = np.arange(1 << 16, dtype=np.uint32) << np.uint32(16)
    lows = (0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF)
    pats = np.concatenate([hi | np.uint32(lo) for lo in lows])
    # a T=1 model whose stream is the plain cast of its flat buffer
    model = (1, 64, 1, 1, 64, 64, 4096)
    n, npad = datagen.flat_sizes(model, 1)
    flat = np.zeros(npad, dtype=np.uint32)
    reps = -(-n // pats.size)
    flat[:n] = np.tile(pats, reps)[:n]
    assert n >= pats.size
    for depth in (2, 4):
        _run_and_compare(model, 1, 1, 1 << 16, flat.view(np.float32), tile_depth=depth)


# ------------------------------------------------------------------ layouts, budgets, alignment
_SHAPES = [(1, 8, 2, 2, 2, 4, 4), (2, 16, 4, 2, 2, 12, 8), (2, 16, 4, 4, 8, 24, 24), (2, 24, 8, 8, 3, 40, 64),
           (1, 24, 4, 4, 6, 20, 8)]


@pytest.mark.parametrize("model", _SHAPES)
def test_tagged_small_shapes(model):
    L, H, Hq, Hkv, D, F, V = model
    for w in (1, 3, 7):
        for t in [t for t in (1, 2, 4, 8) if Hq % t == 0 and Hkv % t == 0 and F % t == 0 and V % t == 0]:
            for b in (16, 48, 1024, 1 << 20):
                flat = datagen.tagged_flat(model, w)
                _run_and_compare(model, w, t, b, flat)
                if b in (48, 1 << 20):
                    _run_and_compare(model, w, t, b, flat, tile_depth=4)


def test_seeded_random_layouts():
    """100 seeded random layouts (tests/random_layouts.py) up to 4 M elements: hundreds to thousands
    of tiles each, ragged tails, column slices cut at shard and chunk boundaries, odd head widths;
    separate shard allocations or views of one buffer, automatic (both depths) or a fixed depth."""
    rng = np.random.default_rng(20260724)
    for i in range(100):
        model, w, t, b = random_layout(rng)
        flat = datagen.make_flat_numpy(model, w, seed=int(rng.integers(1 << 30)), specials_frac=0.003)
        say("random layout", i)
        _run_and_compare(model, w, t, b, flat, separate=bool(rng.random() < 0.5),
                         tile_depth=int(rng.choice([0, 0, 2, 4])))


def test_zero_layer_model():
    """The degenerate decoder with no layers (embed, final_norm, lm_head), both tile depths."""
    model = (0, 64, 4, 4, 16, 32, 96)
    flat = datagen.make_flat_numpy(model, 3, seed=13, specials_frac=0.02)
    for depth in (2, 4):
        for t, b in ((1, 16), (2, 4096 + 16), (4, 1 << 20)):
            _run_and_compare(model, 3, t, b, flat, tile_depth=depth)


def test_max_shards_and_single_chunk():
    model = (2, 64, 8, 4, 16, 96, 128)
    flat = datagen.make_flat_numpy(model, 64, seed=9, specials_frac=0.01)
    for depth in (2, 4):
        _run_and_compare(model, 64, 4, 1 << 30, flat, tile_depth=depth)  # one chunk covering everything
        _run_and_compare(model, 64, 2, 16, flat, tile_depth=depth)       # smallest budget: 16-byte chunks


@pytest.mark.parametrize("tile_depth", [0, 2])  # automatic plans stage chunks at depth 4
def test_chunk_calls_write_only_their_chunk(tile_depth):
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed, specials_frac=0.001)
    plan, shards, keep, dst, cks = _run_and_compare(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat,
                                                    tile_depth=tile_depth)
    info = dr.dr_plan_get_info(plan)
    full = dst.cpu().numpy()
    full_cks = checksums_to_list(cks)
    guard = 256
    B = wl.chunk_bytes
    for c in range(info["num_chunks"]):
        n = B if c < info["num_chunks"] - 1 else info["last_chunk_bytes"]
        buf = torch.full((guard + B + guard,), 0xA5, dtype=torch.uint8, device="cuda")
        ck = new_checksums(1)
        dr.dr_stage_chunk(plan, c, shards, buf[guard:], ck)
        assert dr.dr_plan_get_info(plan)["last_tile_depth"] == (tile_depth or 4)
        torch.cuda.synchronize()
        h = buf.cpu().numpy()
        assert np.all(h[:guard] == 0xA5) and np.all(h[guard + n:] == 0xA5), f"chunk {c} wrote outside its bytes"
        assert np.array_equal(h[guard:guard + n], full[c * B:c * B + n]), c
        assert checksums_to_list(ck)[0] == full_cks[c]


@pytest.mark.parametrize("tile_depth", [0, 2])
def test_restaging_is_idempotent_and_resumable(tile_depth):
    # stage chunks 0..k, "crash", start again at k: the bytes and checksums match one clean pass
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed)
    plan, shards, keep, dst, cks = _run_and_compare(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, flat,
                                                    tile_depth=tile_depth)
    info = dr.dr_plan_get_info(plan)
    B = wl.chunk_bytes
    out = torch.zeros(info["rollout_bytes"], dtype=torch.uint8, device="cuda")
    cks2 = new_checksums(info["num_chunks"])
    k = 7
    for c in list(range(0, k + 1)) + list(range(k, info["num_chunks"])):
        dr.dr_stage_chunk(plan, c, shards, out[c * B:], cks2[c])
    torch.cuda.synchronize()
    assert torch.equal(out, dst)
    assert checksums_to_list(cks2) == checksums_to_list(cks)


def test_stage_on_side_stream():
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, wl.seed)
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    shards, keep = to_device_shards(flat, wl.train_shards)
    info = dr.dr_plan_get_info(plan)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    dst = torch.empty(info["rollout_bytes"], dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    with torch.cuda.stream(s):
        dr.dr_stage_all(plan, shards, dst, cks, stream=s)
    s.synchronize()
    want, want_cks = _oracle(flat.view(np.uint32), wl.model, wl.tp, wl.chunk_bytes)
    assert np.array_equal(as_u16(dst), want)
    assert checksums_to_list(cks) == want_cks


def test_plan_device_and_errors_on_gpu():
    wl = workloads.TINY
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    assert info["device"] == torch.cuda.current_device()
    shards = [torch.zeros(info["shard_elems"], dtype=torch.float32, device="cuda") for _ in range(4)]
    dst = torch.empty(info["rollout_bytes"], dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_all(plan, shards[:3] + [None], dst, cks)
    assert e.value.code == dr.DR_EINVAL
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk(plan, info["num_chunks"], shards, dst, cks)
    assert e.value.code == dr.DR_ERANGE
    # the binding refuses device buffers it can see are wrong before the library runs anything
    with pytest.raises(ValueError, match="the plan needs"):
        dr.dr_stage_all(plan, shards, dst[:-16], cks)
    with pytest.raises(ValueError, match="the plan needs"):
        dr.dr_stage_all(plan, shards, dst, cks[:-1])
    with pytest.raises(ValueError, match="the plan needs"):
        dr.dr_stage_all(plan, [x[:-4] for x in shards], dst, cks)
    with pytest.raises(ValueError, match="not contiguous"):
        dr.dr_stage_all(plan, shards, torch.empty(2 * info["rollout_bytes"], dtype=torch.uint8, device="cuda")[::2],
                        cks)
    with pytest.raises(ValueError, match="the plan needs"):
        dr.dr_stage_chunk(plan, 0, shards, dst[:wl.chunk_bytes - 16], cks[0])


def test_every_fp32_pattern_through_the_kernel():
    """All 2^32 fp32 bit patterns pass through dr_stage_all (T=1: the stream is the cast of the flat
    buffer) with both tile depths, and every bf16 result equals the oracle's, NaN payloads included."""
    model = (1, 64, 1, 1, 64, 64, 1 << 25)  # N = 2^32 + 28800: embed + lm_head hold 2^32 elements
    plan = dr.dr_plan_create(model, 1, 1, 1 << 30, tile_depth=2)
    plan4 = dr.dr_plan_create(model, 1, 1, 1 << 30, tile_depth=4)
    info = dr.dr_plan_get_info(plan)
    n = info["n_elems"]
    assert n >= 1 << 32
    flat = torch.zeros(info["padded_elems"], dtype=torch.int32, device="cuda")
    blk = 1 << 28
    for b in range(0, 1 << 32, blk):
        x = torch.arange(b, b + blk, dtype=torch.int64, device="cuda")
        flat[b:b + blk] = torch.where(x >= (1 << 31), x - (1 << 32), x).to(torch.int32)
        del x
    dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
    cks = new_checksums(info["num_chunks"])
    dst4 = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
    cks4 = new_checksums(info["num_chunks"])
    say("all 2^32 patterns through stage_all, tile depths 2 and 4")
    dr.dr_stage_all(plan, [flat.view(torch.float32)], dst, cks)
    dr.dr_stage_all(plan4, [flat.view(torch.float32)], dst4, cks4)
    torch.cuda.synchronize()
    for b in range(0, 1 << 32, blk):
        src = flat[b:b + blk].cpu().numpy().view(np.uint32)
        want = oracle.rne_bf16(src)
        for out in (dst.view(torch.int16), dst4.view(torch.int16)):
            got = out[b:b + blk].cpu().numpy().view(np.uint16)
            if not np.array_equal(got, want):
                bad = np.flatnonzero(got != want)[:4]
                raise AssertionError(f"inputs {[hex(int(src[i])) for i in bad]} -> "
                                     f"{[hex(int(got[i])) for i in bad]}, want {[hex(int(want[i])) for i in bad]}")
    assert torch.equal(cks, cks4)


def test_largest_segment_at_both_depths():
    """Segments at the planner's cap: with T=1 and one shard, embed and lm_head are contiguous runs
    of exactly 2^30 elements, each one segment.  The stream (the plain cast of the flat buffer) is
    compared with the oracle element by element, for both tile depths."""
    model = (0, 16384, 8, 8, 128, 16384, 1 << 16)  # V*H = 2^30
    plan2 = dr.dr_plan_create(model, 1, 1, 1 << 34, tile_depth=2)
    plan4 = dr.dr_plan_create(model, 1, 1, 1 << 34, tile_depth=4)
    info = dr.dr_plan_get_info(plan2)
    sizes = [s["rows"] * s["cols"] for s in (dr.dr_plan_segment(plan2, i) for i in range(info["num_segments"]))]
    assert sizes.count(1 << 30) == 2 and max(sizes) == 1 << 30
    n = info["n_elems"]
    g = torch.Generator(device="cuda")
    g.manual_seed(31)
    flat = torch.randint(-(1 << 31), 1 << 31, (info["padded_elems"],), dtype=torch.int64, device="cuda",
                         generator=g).to(torch.int32)
    outs = []
    for plan in (plan2, plan4):
        dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
        cks = new_checksums(info["num_chunks"])
        say("2^30-element segments, tile_elems", dr.dr_plan_get_info(plan)["tile_elems"])
        dr.dr_stage_all(plan, [flat.view(torch.float32)], dst, cks)
        outs.append((dst, cks))
    torch.cuda.synchronize()
    blk = 1 << 27
    for b in range(0, n, blk):
        e = min(n, b + blk)
        want = oracle.rne_bf16(flat[b:e].cpu().numpy().view(np.uint32))
        for dst, _ in outs:
            assert np.array_equal(dst.view(torch.int16)[b:e].cpu().numpy().view(np.uint16), want), b
    assert torch.equal(outs[0][1], outs[1][1])


# ------------------------------------------------------------------ launch-grid caps
# A tile kernel launches at most 16777208 workgroups (2^32 - 1 lanes of 256, rounded down to a
# multiple of the 8 XCDs), and the chunk reduce at most 2^20; larger plans stride over the rest.
# With no layers, T = 1 and 16-byte chunks, every chunk is one tile, and a vocabulary of
# 2^23 - 1 rows of 8 gives 2^24 - 1 chunks: 7 tiles past the first pass of the grid and 16 chunks
# per reduce workgroup.
_STRIDE_MODEL = (0, 8, 1, 1, 8, 8, (1 << 23) - 1)
_MAX_GRID = (0xFFFFFFFF // 256) // 8 * 8


def _xcd_tile(b, n):
    per, rem, x = n // 8, n % 8, b % 8
    return x * per + min(x, rem) + b // 8


def _sampled_chunks(n_chunks, seed):
    """Chunks of the tiles the grid's second pass runs, the ends, and a random sample."""
    late = [_xcd_tile(b, n_chunks) for b in range(_MAX_GRID, n_chunks)]
    rng = np.random.default_rng(seed)
    return sorted(set(late + [0, 1, n_chunks - 2, n_chunks - 1] + rng.integers(0, n_chunks, 20000).tolist()))


def _check_sampled(raw, cks, chunk_bytes, chunks):
    got = cks.cpu().numpy().view(np.uint64).reshape(-1, 2)
    assert not np.any(np.all(got == np.uint64(0xFFFFFFFFFFFFFFFF), axis=1)), "a checksum slot was not written"
    for c in chunks:
        assert (int(got[c, 0]), int(got[c, 1])) == oracle.checksum(raw[c * chunk_bytes:(c + 1) * chunk_bytes]), c


def test_grids_that_stride_over_tiles_and_chunks():
    plan = dr.dr_plan_create(_STRIDE_MODEL, 1, 1, 16)
    info = dr.dr_plan_get_info(plan)
    nc = info["num_chunks"]
    assert nc == info["num_tiles"] == (1 << 24) - 1 and nc > _MAX_GRID
    n = info["n_elems"]
    g = torch.Generator(device="cuda")
    g.manual_seed(41)
    flat = torch.randint(-(1 << 31), 1 << 31, (info["padded_elems"],), dtype=torch.int64, device="cuda",
                         generator=g).to(torch.int32)
    dst = torch.full((info["rollout_bytes"],), 0xFF, dtype=torch.uint8, device="cuda")
    cks = new_checksums(nc)
    say("stage_all over", nc, "16-byte chunks (grid-stride tiles and chunks)")
    dr.dr_stage_all(plan, [flat.view(torch.float32)], dst, cks)
    torch.cuda.synchronize()
    want = oracle.rne_bf16(flat[:n].cpu().numpy().view(np.uint32))
    got = dst.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, want)
    _check_sampled(want.view(np.uint8), cks, 16, _sampled_chunks(nc, 1))


def test_reshard_grid_that_strides_over_tiles():
    """2 -> 1 shards in 32-byte chunks: 2^24 chunks and tiles (8 of them past the first pass)."""
    plan = dr.dr_reshard_plan_create(_STRIDE_MODEL, 2, 1, 32)
    info = dr.dr_plan_get_info(plan)
    nc = info["num_chunks"]
    assert nc == info["num_tiles"] == 1 << 24
    n, S, S2 = info["n_elems"], info["shard_elems"], info["dst_shard_elems"]
    g = torch.Generator(device="cuda")
    g.manual_seed(43)
    flat = torch.randint(-(1 << 31), 1 << 31, (2 * S,), dtype=torch.int64, device="cuda", generator=g).to(torch.int32)
    dst = torch.full((S2,), -1, dtype=torch.int32, device="cuda")
    cks = new_checksums(nc)
    say("dr_reshard over", nc, "32-byte chunks (grid-stride tiles and chunks)")
    dr.dr_reshard(plan, [flat[:S].view(torch.float32), flat[S:].view(torch.float32)], [dst.view(torch.float32)], cks)
    torch.cuda.synchronize()
    want = oracle.reshard(flat.cpu().numpy().view(np.uint32), n, 1)
    assert np.array_equal(dst.cpu().numpy().view(np.uint32), want)
    _check_sampled(want.view(np.uint8), cks, 32, _sampled_chunks(nc, 2))
