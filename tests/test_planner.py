"""CPU tests of the planner (segment table) and of the C ABI's host-side behaviour.

The segment table is read back through dr_plan_segment and interpreted here in
numpy (move row i of a segment from shard[src + i*stride ...] to the dense
stream position); the result must equal the oracle's rollout stream.  No GPU is
involved: plans are built with dr_plan_create_host.
"""
import ctypes
import os
import re
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from oracle import Model
from paper_2607_22614_amd import datagen, dr, workloads
from tests.random_layouts import random_layout, random_reshard

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _segments(plan):
    n = dr.dr_plan_get_info(plan)["num_segments"]
    return [dr.dr_plan_segment(plan, i) for i in range(n)]


def _walk(plan, shard_bits, info):
    """Interpret the segment table: returns the uint16 stream the table describes and a write count."""
    total = info["rollout_bytes"] // 2
    out = np.zeros(total, dtype=np.uint16)
    count = np.zeros(total, dtype=np.int32)
    for s in _segments(plan):
        src = shard_bits[s["shard"]]
        rows, cols, stride = s["rows"], s["cols"], s["src_row_stride"]
        idx = s["src_elem"] + (np.arange(rows, dtype=np.int64)[:, None] * stride + np.arange(cols)[None, :])
        vals = oracle.rne_bf16(src[idx.ravel()])
        out[s["dst_elem"]:s["dst_elem"] + rows * cols] = vals
        count[s["dst_elem"]:s["dst_elem"] + rows * cols] += 1
    return out, count


def _check_table(plan, w, info):
    S = info["shard_elems"]
    segs = _segments(plan)
    prev_end = 0
    for s in segs:
        n = s["rows"] * s["cols"]
        assert s["dst_elem"] == prev_end, "segments are dense and in stream order"
        prev_end += n
        assert 0 <= s["shard"] < w
        assert s["src_elem"] + (s["rows"] - 1) * s["src_row_stride"] + s["cols"] <= S, "segment crosses a shard"
        assert s["rows"] == 1 or s["src_row_stride"] >= s["cols"]
        assert n <= (1 << 30)
        vec = (s["src_elem"] % 4 == 0 and s["dst_elem"] % 4 == 0 and s["cols"] % 4 == 0
               and (s["rows"] == 1 or s["src_row_stride"] % 4 == 0))
        assert bool(s["flags"] & dr.DR_SEG_VEC4) == vec
    assert prev_end == info["rollout_bytes"] // 2
    return segs


def _check_chunks(segs, chunk_bytes):
    ce = chunk_bytes // 2
    for s in segs:
        first = s["dst_elem"]
        last = s["dst_elem"] + s["rows"] * s["cols"] - 1
        assert first // ce == last // ce == s["chunk"], "segment crosses a chunk boundary"


# ------------------------------------------------------------------ planner vs oracle
def _compare(model, w, t, chunk_bytes, seed=0, specials=0.0, tagged=False):
    m = Model(*model)
    plan = dr.dr_plan_create_host(model, w, t, chunk_bytes)
    info = dr.dr_plan_get_info(plan)
    flat = (datagen.tagged_flat(model, w) if tagged else
            datagen.make_flat_numpy(model, w, seed, specials_frac=specials)).view(np.uint32)
    assert info["padded_elems"] == flat.size
    assert info["shard_elems"] * w == flat.size
    segs = _check_table(plan, w, info)
    _check_chunks(segs, chunk_bytes)
    got, count = _walk(plan, oracle.shards(flat, w), info)
    assert np.all(count == 1), "every stream element is written exactly once"
    want = oracle.rollout_stream(oracle.training_views(flat, m), m, t)
    np.testing.assert_array_equal(got, want)
    # tensor descriptors agree with the oracle's table
    per_rank = 3 + 6 * m.n_layers
    table = oracle.rollout_table(m, t)
    for r in range(t):
        for i in range(per_rank):
            d = dr.dr_plan_tensor(plan, r, i)
            r2, name, off, shape = table[r * per_rank + i]
            assert (d["rank"], d["name"], d["byte_offset"]) == (r2, name, 2 * off)
            assert (d["rows"], d["cols"]) == (shape[0], shape[1] if len(shape) == 2 else 1)
    return info


def test_tiny_workload_against_oracle():
    wl = workloads.TINY
    info = _compare(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, seed=wl.seed, specials=0.001)
    assert info["num_chunks"] == 21 and info["last_chunk_bytes"] == 21504


_SMALL = [(1, 8, 2, 2, 2, 4, 4), (2, 16, 4, 2, 2, 12, 8), (1, 8, 1, 1, 2, 8, 8), (2, 16, 4, 4, 8, 24, 24),
          (1, 16, 2, 1, 4, 12, 16), (2, 8, 4, 1, 8, 8, 24)]


@pytest.mark.parametrize("model", _SMALL)
def test_tagged_small_shapes_all_layouts(model):
    L, H, Hq, Hkv, D, F, V = model
    for w in (1, 2, 3, 4, 7):
        for t in [t for t in (1, 2, 3, 4, 8) if Hq % t == 0 and Hkv % t == 0 and F % t == 0 and V % t == 0]:
            total = 2 * sum(int(np.prod(s)) for _, s in oracle.rollout_tensors(Model(*model), t)) * t
            for b in sorted({16, 32, 48, 80, 144, 1024, ((total + 15) // 16) * 16, 1 << 20}):
                _compare(model, w, t, b, tagged=True)


@pytest.mark.parametrize("w,t,b", [(1, 1, 16 * 1000), (3, 2, 4096 + 16), (64, 4, 1 << 16), (2, 8, 48)])
def test_unaligned_column_runs(w, t, b):
    # Hq*D/T and F/T not multiples of 4: o and down rows are unaligned runs
    model = (2, 24, 8, 8, 3, 40, 64)
    _compare(model, w, t, b, seed=3, specials=0.01)


def test_segment_splits_at_shard_boundaries_inside_rows():
    # shard length S = 256 with H = 24 (o rows of 24*... cross shard boundaries mid-row)
    model = (1, 24, 4, 4, 6, 20, 8)
    info = _compare(model, 7, 2, 160, seed=1)
    assert info["num_segments"] > 30


# ------------------------------------------------------------------ ABI errors (no HIP call happens)
def _create_rc(model, w=1, t=1, b=256, bm=0):
    h = ctypes.c_void_p()
    rc = dr._lib.dr_plan_create_host(ctypes.byref(dr.dr_model(*model)), ctypes.byref(dr.dr_layout(w, t, b, bm)),
                                     ctypes.byref(h))
    if rc == 0:
        dr._lib.dr_plan_destroy(h)
    return rc


GOOD = (2, 256, 4, 4, 64, 688, 2048)


@pytest.mark.parametrize("field", range(7))
def test_nonpositive_shape_fields(field):
    for bad in ((-1,) if field == 0 else (0, -1)):
        m = list(GOOD)
        m[field] = bad
        assert _create_rc(tuple(m)) == dr.DR_EINVAL
        assert ("must be >= 0" if field == 0 else "must be > 0") in dr.dr_last_error()


@pytest.mark.parametrize("w,t,b", [(1, 1, 16), (3, 2, 48), (4, 4, 1 << 20), (64, 2, 4096)])
def test_zero_layer_model(w, t, b):
    """The degenerate decoder with no layers: embed, final_norm and lm_head only."""
    info = _compare((0, 16, 4, 4, 4, 8, 24), w, t, b, seed=5, specials=0.05)
    assert info["norm_elems"] == 16 and info["n_elems"] == 2 * 24 * 16 + 16


@pytest.mark.parametrize("model,w,t,b,bm,msg", [
    ((2, 260, 4, 4, 64, 688, 2048), 1, 1, 256, 0, "multiple of 8"),
    ((2, 256, 6, 4, 64, 688, 2048), 1, 1, 256, 0, "multiple of n_kv_heads"),
    (GOOD, 1, 3, 256, 0, "divide n_q_heads"),
    ((2, 256, 8, 2, 64, 688, 2048), 1, 4, 256, 0, "divide n_kv_heads"),
    ((2, 256, 4, 4, 64, 687, 2048), 1, 2, 256, 0, "divide ffn"),
    ((2, 256, 4, 4, 64, 688, 2049), 1, 2, 256, 0, "divide vocab"),
    (GOOD, 0, 1, 256, 0, "train_shards"),
    (GOOD, 65, 1, 256, 0, "train_shards"),
    (GOOD, 1, 0, 256, 0, "tp must be"),
    (GOOD, 1, 1, 0, 0, "chunk_bytes"),
    (GOOD, 1, 1, 24, 0, "chunk_bytes"),
    (GOOD, 1, 1, 256, 20, "moment_chunk_bytes"),
    ((2000000000, 1 << 30, 1, 1, 1, 1 << 30, 1 << 30), 1, 1, 1 << 30, 0, "too large"),
    (GOOD, 1, 1, 16, 0, None),
    ((24, 896, 14, 2, 64, 4864, 151936), 1, 1, 16, 0, "chunks"),
    ((24, 896, 14, 2, 64, 4864, 151936), 1, 1, 1 << 20, 16, "moment chunks"),
])
def test_invalid_layouts(model, w, t, b, bm, msg):
    rc = _create_rc(model, w, t, b, bm)
    if msg is None:
        assert rc == dr.DR_OK
    else:
        assert rc == dr.DR_EINVAL, dr.dr_last_error()
        assert msg in dr.dr_last_error()


def test_introspection_ranges():
    plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024)
    with pytest.raises(dr.DrError) as e:
        dr.dr_plan_tensor(plan, 2, 0)
    assert e.value.code == dr.DR_ERANGE
    with pytest.raises(dr.DrError) as e:
        dr.dr_plan_tensor(plan, 0, 3 + 6 * 2)
    assert e.value.code == dr.DR_ERANGE
    n = dr.dr_plan_get_info(plan)["num_segments"]
    with pytest.raises(dr.DrError) as e:
        dr.dr_plan_segment(plan, n)
    assert e.value.code == dr.DR_ERANGE
    assert dr.dr_plan_get_info(plan)["device"] == -1


def test_staging_calls_validate_before_any_hip_call():
    plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, 1 << 20)
    info = dr.dr_plan_get_info(plan)
    fake = [0x1000 * (i + 1) for i in range(4)]  # aligned, never dereferenced
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk(plan, info["num_chunks"], fake, 0x10000, 0x20000, stream=0)
    assert e.value.code == dr.DR_ERANGE
    for args, frag in [((0, fake[:3] + [0], 0x10000, 0x20000), "shard 3"),
                       ((0, fake[:3] + [0x1008], 0x10000, 0x20000), "shard 3"),
                       ((0, fake, 0x10008, 0x20000), "dst_chunk"),
                       ((0, fake, 0x10000, 0), "d_ck"),
                       ((0, fake, 0x10000, 0x20000), "host-only")]:
        with pytest.raises(dr.DrError) as e:
            dr.dr_stage_chunk(plan, *args, stream=0)
        assert e.value.code == dr.DR_EINVAL and frag in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_all(plan, fake, 0x10000, 0x20004, stream=0)
    assert e.value.code == dr.DR_EINVAL and "d_cks" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_all(plan, fake, 0x10000, 0x20000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "host-only" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_offload_moments(plan, fake, fake, 0x30000, 0)
    assert "host-only" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_restore_moments(plan, 0, fake, fake, 0)
    assert "null host store" in str(e.value)
    plan0 = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024)  # no moment path
    with pytest.raises(dr.DrError) as e:
        dr.dr_offload_moments(plan0, fake, fake, 0x30000, 0)
    assert "moment_chunk_bytes = 0" in str(e.value)


def test_moment_sizes():
    wl = workloads.EIGHT_B_ADAM
    info = dr.dr_plan_get_info(dr.dr_plan_create_host(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes,
                                                       wl.moment_chunk_bytes))
    assert info["moment_bytes"] == 2 * 8030261248 * 4
    assert info["num_moment_chunks"] == 120
    assert info["moment_bytes"] - 119 * wl.moment_chunk_bytes == 354451456
    assert info["pinned_bytes"] == 2 * wl.moment_chunk_bytes


# ------------------------------------------------------------------ the library and its header agree
def _header_functions():
    text = open(os.path.join(ROOT, "include", "dr.h")).read()
    return sorted(set(re.findall(r"^(?:int|void|double|const char\*)\s+(dr_[a-z_]+)\s*\(", text, flags=re.M)))


def test_library_exports_every_header_function():
    names = _header_functions()
    assert "dr_stage_all" in names and "dr_offload_moments" in names
    out = subprocess.run(["nm", "-D", "--defined-only", dr.library_path()], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    assert set(dr.EXPORTED) == set(names)


def test_library_targets_gfx950_only(tmp_path):
    """Every offload bundle in libdr.so (one per HIP source) holds gfx950 code and nothing else."""
    llvm = "/opt/rocm/llvm/bin"
    fatbin = tmp_path / "lib.fatbin"
    subprocess.run([f"{llvm}/llvm-objcopy", f"--dump-section=.hip_fatbin={fatbin}", dr.library_path(),
                    str(tmp_path / "stripped.so")], check=True, capture_output=True)
    data = fatbin.read_bytes()
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    starts = [i for i in range(len(data)) if data.startswith(magic, i)]
    assert len(starts) >= 2  # stage.hip and reshard.hip
    for n, (a, b) in enumerate(zip(starts, starts[1:] + [len(data)])):
        part = tmp_path / f"b{n}.fatbin"
        part.write_bytes(data[a:b])
        out = subprocess.run([f"{llvm}/clang-offload-bundler", "--list", "--type=o", f"--input={part}"],
                             capture_output=True, text=True, check=True).stdout
        targets = [t for t in out.split() if "amdgcn" in t]
        assert targets == ["hipv4-amdgcn-amd-amdhsa--gfx950"], out


# ------------------------------------------------------------------ the kernel's row division is exact
def _div_cols(e, cols, magic):
    """The stage kernel's e / cols: q = umulhi(e, magic), then one correction step."""
    q = (e * magic) >> 32
    r = e - q * cols
    if r >= cols:
        q, r = q + 1, r - cols
    return q, r


def test_row_division_exact():
    rng = np.random.default_rng(0)
    cols_set = list(range(1, 2100)) + [3456, 3584, 4096, 4864, 27648, (1 << 30) - 1, 1 << 30] + \
        [int(c) for c in rng.integers(1, 1 << 30, size=300)]
    for cols in cols_set:
        magic = 0xFFFFFFFF if cols == 1 else (1 << 32) // cols
        es = [0, 1, cols - 1, cols, cols + 1, (1 << 30) - 1, (1 << 31) - 1, (1 << 32) - 1]
        es += [int(x) for x in rng.integers(0, 1 << 32, size=64)]
        for e in es:
            assert _div_cols(e, cols, magic) == divmod(e, cols), (e, cols)


def test_capped_grid_strides_over_every_tile_on_its_xcd():
    """A tile kernel's grid is capped at a multiple of the 8 XCDs; workgroup g runs tiles
    xcd_tile(g + k*grid, n).  Every tile must run exactly once, and on the XCD (g % 8) whose
    contiguous range holds it."""
    def xcd_tile(b, n):
        per, rem, x = n // 8, n % 8, b % 8
        return x * per + min(x, rem) + b // 8

    assert ((0xFFFFFFFF // 256) // 8 * 8) % 8 == 0
    for n in (9, 17, 100, 1001, 4099):
        starts = [x * (n // 8) + min(x, n % 8) for x in range(9)]
        for grid in (8, 16, 24, 8 * ((n // 8) - 1) or 8):
            seen = []
            for g in range(grid):
                for b in range(g, n, grid):
                    t = xcd_tile(b, n)
                    assert starts[g % 8] <= t < starts[g % 8 + 1], (n, grid, g, t)
                    seen.append(t)
            assert sorted(seen) == list(range(n)), (n, grid)


def test_xcd_tile_order_is_a_permutation():
    """The stage kernel runs tile xcd_tile(b, n) in workgroup b; every tile must run exactly once."""
    def xcd_tile(b, n):
        per, rem, x = n // 8, n % 8, b % 8
        return x * per + min(x, rem) + b // 8

    for n in list(range(1, 300)) + [980559, 4000473]:
        if n < 300:
            assert sorted(xcd_tile(b, n) for b in range(n)) == list(range(n))
        else:
            t = np.array([xcd_tile(b, n) for b in range(n)])
            assert np.array_equal(np.sort(t), np.arange(n))


# ------------------------------------------------------------------ reshard plans
def _walk_reshard(plan, src_shards, info, w2):
    S2 = info["dst_shard_elems"]
    out = np.full(S2 * w2, 0xDEADBEEF, dtype=np.uint32)
    count = np.zeros(S2 * w2, dtype=np.int32)
    ce = None
    for s in _segments(plan):
        n = s["rows"] * s["cols"]
        assert s["rows"] == 1
        a = s["dst_elem"]
        assert s["dst_shard"] == a // S2 == (a + n - 1) // S2, "segment crosses a destination shard"
        if s["op"] == dr.DR_OP_ZERO_F32:
            out[a:a + n] = 0
        else:
            assert s["op"] == dr.DR_OP_COPY_F32
            out[a:a + n] = src_shards[s["shard"]][s["src_elem"]:s["src_elem"] + n]
        count[a:a + n] += 1
        assert s["flags"] & dr.DR_SEG_VEC4
    return out, count


@pytest.mark.parametrize("model,w,w2,b", [
    ((2, 256, 4, 4, 64, 688, 2048), 4, 3, 256 * 1024),
    ((2, 64, 8, 4, 16, 96, 128), 1, 8, 16),
    ((2, 64, 8, 4, 16, 96, 128), 8, 1, 4096 + 16),
    ((2, 64, 8, 4, 16, 96, 128), 3, 64, 1 << 30),
    ((1, 24, 4, 4, 6, 20, 8), 7, 5, 48),
])
def test_reshard_plan_against_oracle(model, w, w2, b):
    plan = dr.dr_reshard_plan_create_host(model, w, w2, b)
    info = dr.dr_plan_get_info(plan)
    assert info["kind"] == dr.DR_PLAN_RESHARD
    n, npad = datagen.flat_sizes(model, w)
    flat = datagen.make_flat_numpy(model, w, seed=1, specials_frac=0.05).view(np.uint32)
    want = oracle.reshard(flat, n, w2)
    assert info["rollout_bytes"] == 4 * want.size and info["dst_shard_elems"] * w2 == want.size
    got, count = _walk_reshard(plan, oracle.shards(flat, w), info, w2)
    assert np.all(count == 1)
    assert np.array_equal(got, want)
    _check_chunks(_segments(plan), b // 2)  # b-byte chunks hold b/4 fp32 words (helper divides by 2)
    assert info["num_chunks"] == -(-4 * want.size // b)


def test_seeded_random_layouts_against_oracle():
    """120 seeded random layouts (shapes, W, T, budgets; tests/random_layouts.py): each segment table
    reproduces the oracle's stream exactly, writes every element once and respects the cuts."""
    rng = np.random.default_rng(20260722)
    for _ in range(120):
        model, w, t, b = random_layout(rng, max_elems=400_000)
        _compare(model, w, t, b, seed=int(rng.integers(1 << 30)), specials=0.01)


def test_seeded_random_reshard_plans_against_oracle():
    rng = np.random.default_rng(20260723)
    for _ in range(40):
        model, w, w2, b = random_reshard(rng, max_elems=400_000)
        plan = dr.dr_reshard_plan_create_host(model, w, w2, b)
        info = dr.dr_plan_get_info(plan)
        n, _ = datagen.flat_sizes(model, w)
        flat = datagen.make_flat_numpy(model, w, seed=int(rng.integers(1 << 30)), specials_frac=0.01).view(np.uint32)
        want = oracle.reshard(flat, n, w2)
        got, count = _walk_reshard(plan, oracle.shards(flat, w), info, w2)
        assert np.all(count == 1)
        assert np.array_equal(got, want), (model, w, w2, b)
        _check_chunks(_segments(plan), b // 2)


def test_reshard_plan_rejects_and_rollout_calls_refuse_it():
    m = (2, 64, 8, 4, 16, 96, 128)
    for bad in ((m, 0, 2, 256), (m, 2, 65, 256), (m, 2, 2, 24)):
        with pytest.raises(dr.DrError) as e:
            dr.dr_reshard_plan_create_host(*bad)
        assert e.value.code == dr.DR_EINVAL
    plan = dr.dr_reshard_plan_create_host(m, 2, 3, 256)
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_all(plan, [0x1000, 0x2000], 0x3000, 0x4000, stream=0)
    assert "not a rollout plan" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_plan_tensor(plan, 0, 0)
    assert "not a rollout plan" in str(e.value)
    rollout = dr.dr_plan_create_host(m, 2, 2, 256)
    with pytest.raises(dr.DrError) as e:
        dr.dr_reshard(rollout, [0x1000, 0x2000], [0x3000] * 3, 0x4000, stream=0)
    assert "not a reshard plan" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_reshard(plan, [0x1000, 0x2000], [0x3000, 0x3008, 0x3010], 0x4000, stream=0)
    assert "destination shard 1" in str(e.value)


def test_noalloc_chunk_call_validates_before_any_hip_call():
    """The allocation-free chunk call refuses on the host what dr_stage_chunk refuses."""
    plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024)
    info = dr.dr_plan_get_info(plan)
    fake = [0x1000 * (i + 1) for i in range(4)]
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(plan, info["num_chunks"], fake, 0x9000, 0xA000, stream=0)
    assert e.value.code == dr.DR_ERANGE
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(plan, 0, fake, 0x9008, 0xA000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "16-byte aligned" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(plan, 0, fake, 0x9000, 0xA000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "host-only" in str(e.value)
    reshard = dr.dr_reshard_plan_create_host(GOOD, 4, 3, 4096)
    with pytest.raises(dr.DrError) as e:
        dr.dr_stage_chunk_noalloc(reshard, 0, fake, 0x9000, 0xA000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "not a rollout plan" in str(e.value)


def test_moment_checksums_validate_before_any_hip_call():
    fake = [0x1000 * (i + 1) for i in range(4)]
    plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, 1 << 20)
    with pytest.raises(dr.DrError) as e:
        dr.dr_moment_checksums(plan, fake, fake, 0xA000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "host-only" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_moment_checksums(plan, fake, [0x1008] + fake[1:], 0xA000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "16-byte aligned" in str(e.value)
    without = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024)  # no moment path
    with pytest.raises(dr.DrError) as e:
        dr.dr_moment_checksums(without, fake, fake, 0xA000, stream=0)
    assert e.value.code == dr.DR_EINVAL and "no moment path" in str(e.value)
    with pytest.raises(ValueError, match="3 shard buffers given"):
        dr.dr_moment_checksums(plan, fake[:3], fake, 0xA000, stream=0)


def test_deferred_restore_calls_validate_on_cpu():
    plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, 1 << 20)
    fake = [0x1000 * (i + 1) for i in range(4)]
    with pytest.raises(dr.DrError) as e:
        dr.dr_restore_moments_begin(plan, 0x5000, fake, fake, 0)
    assert e.value.code == dr.DR_EINVAL and "host-only" in str(e.value)
    with pytest.raises(dr.DrError) as e:
        dr.dr_restore_moments_end(plan)
    assert e.value.code == dr.DR_EINVAL and "no deferred restore" in str(e.value)


class _DeferredRestoreStub:
    """Stands in for the library's two deferred-restore calls (everything else is the real library)."""

    def __init__(self, lib):
        self._lib = lib

    def __getattr__(self, name):
        return getattr(self._lib, name)

    def dr_restore_moments_begin(self, *args):
        return dr.DR_OK

    def dr_restore_moments_end(self, *args):
        return dr.DR_OK


def test_deferred_restore_binding_holds_its_buffers(monkeypatch):
    """dr_restore_moments_begin returns while a library thread still reads the host store and
    writes the shards: the binding keeps them alive until dr_restore_moments_end or close."""
    import gc
    import weakref

    monkeypatch.setattr(dr, "_lib", _DeferredRestoreStub(dr._lib))
    for finish in ("end", "close"):
        plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, 1 << 20)
        info = dr.dr_plan_get_info(plan)
        store = np.empty(info["moment_bytes"], np.uint8)
        alive = weakref.ref(store)
        fake = [0x1000 * (i + 1) for i in range(4)]
        dr.dr_restore_moments_begin(plan, store, fake, fake, 0)
        del store
        gc.collect()
        assert alive() is not None, "host store freed while the restore may still read it"
        if finish == "end":
            dr.dr_restore_moments_end(plan)
        else:
            plan.close()
        gc.collect()
        assert alive() is None, finish
        plan.close()


def test_plan_info_reports_the_layout():
    i = dr.dr_plan_get_info(dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, 1 << 20))
    assert (i["train_shards"], i["tp"], i["dst_shards"], i["chunk_bytes"], i["moment_chunk_bytes"]) == \
        (4, 2, 0, 256 * 1024, 1 << 20)
    r = dr.dr_plan_get_info(dr.dr_reshard_plan_create_host(GOOD, 4, 3, 4096))
    assert (r["train_shards"], r["tp"], r["dst_shards"], r["chunk_bytes"], r["moment_chunk_bytes"]) == \
        (4, 0, 3, 4096, 0)


def test_binding_checks_buffers_before_the_library_sees_them():
    """The C ABI carries no sizes: the binding checks what it can see (shard count, contiguity,
    device or host side, length) and raises ValueError before any call into the library."""
    import torch

    plan = dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, 1 << 20)
    info = dr.dr_plan_get_info(plan)
    fake = [0x1000 * (i + 1) for i in range(4)]
    with pytest.raises(ValueError, match="3 shard buffers given, the plan has 4"):
        dr.dr_stage_all(plan, fake[:3], 0x9000, 0xA000, stream=0)
    with pytest.raises(ValueError, match="expected a device tensor"):
        dr.dr_stage_all(plan, fake, torch.empty(info["rollout_bytes"], dtype=torch.uint8), 0xA000, stream=0)
    with pytest.raises(ValueError, match="numpy array is host memory"):
        dr.dr_stage_all(plan, fake, np.empty(info["rollout_bytes"], np.uint8), 0xA000, stream=0)
    with pytest.raises(ValueError, match="expected a device tensor"):
        dr.dr_stage_chunk(plan, 0, [torch.empty(info["shard_elems"])] * 4, 0x9000, 0xA000, stream=0)
    store = np.empty(info["moment_bytes"], np.uint8)
    with pytest.raises(ValueError, match="the plan needs"):
        dr.dr_offload_moments(plan, fake, fake, store[:-16], 0)
    with pytest.raises(ValueError, match="not contiguous"):
        dr.dr_offload_moments(plan, fake, fake, np.empty(2 * info["moment_bytes"], np.uint8)[::2], 0)
    with pytest.raises(ValueError, match="not contiguous"):
        dr.dr_restore_moments(plan, torch.empty(2 * info["moment_bytes"], dtype=torch.uint8)[::2], fake, fake, 0)
    with pytest.raises(ValueError, match="2 shard buffers given"):
        dr.dr_restore_moments_begin(plan, store, fake, fake[:2], 0)
    # a correctly sized host store reaches the library, which refuses the host-only plan
    with pytest.raises(dr.DrError) as e:
        dr.dr_offload_moments(plan, fake, fake, store, 0)
    assert e.value.code == dr.DR_EINVAL and "host-only" in str(e.value)
    rs = dr.dr_reshard_plan_create_host(GOOD, 4, 3, 4096)
    with pytest.raises(ValueError, match="4 shard buffers given, the plan has 3"):
        dr.dr_reshard(rs, fake, fake, 0xA000, stream=0)


def test_tile_depth_choice():
    """tile_depth is a launch-geometry choice: automatic (2 within 128 GiB), or 2 or 4 explicitly;
    other values and a nonzero reserved field are rejected before anything is built."""
    for depth, elems, deep in ((0, 2048, 4096), (2, 2048, 0), (4, 4096, 0)):
        i = dr.dr_plan_get_info(dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, tile_depth=depth))
        assert (i["tile_elems"], i["deep_tile_elems"], i["last_tile_depth"]) == (elems, deep, 0)
        assert (i["deep_num_tiles"] > 0) == (deep > 0)
    big = workloads.THIRTY_TWO_B  # 197 GB of source + rollout: automatic depth 4, one tiling
    i = dr.dr_plan_get_info(dr.dr_plan_create_host(big.model, big.train_shards, big.tp, big.chunk_bytes))
    assert (i["tile_elems"], i["deep_tile_elems"], i["deep_num_tiles"]) == (4096, 0, 0)
    assert dr.dr_plan_get_info(dr.dr_plan_create_host(big.model, big.train_shards, big.tp, big.chunk_bytes,
                                                      tile_depth=2))["tile_elems"] == 2048
    for bad in (-1, 1, 3, 8):
        with pytest.raises(dr.DrError) as e:
            dr.dr_plan_create_host(GOOD, 4, 2, 256 * 1024, tile_depth=bad)
        assert e.value.code == dr.DR_EINVAL and "tile_depth" in str(e.value)
    h = ctypes.c_void_p()
    lay = dr.dr_layout(4, 2, 256 * 1024, 0, 0, 7)
    assert dr._lib.dr_plan_create_host(ctypes.byref(dr.dr_model(*GOOD)), ctypes.byref(lay), ctypes.byref(h)) == \
        dr.DR_EINVAL
    assert "reserved" in dr.dr_last_error()
    # the segment table does not depend on the depth
    a = dr.dr_plan_create_host((2, 24, 8, 8, 3, 40, 64), 3, 2, 4096 + 16, tile_depth=2)
    b = dr.dr_plan_create_host((2, 24, 8, 8, 3, 40, 64), 3, 2, 4096 + 16, tile_depth=4)
    assert _segments(a) == _segments(b)


def test_automatic_plans_hold_both_tilings_and_count_them():
    """Within 128 GiB an automatic plan holds the depth-2 tiling (num_tiles) and the depth-4 one
    (deep_num_tiles): about half as many tiles, never fewer than one per segment, and both are
    counted in device_table_bytes, each with partial slots of its own."""
    wl = workloads.EIGHT_B
    auto = dr.dr_plan_get_info(dr.dr_plan_create_host(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes))
    two = dr.dr_plan_get_info(dr.dr_plan_create_host(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, tile_depth=2))
    four = dr.dr_plan_get_info(dr.dr_plan_create_host(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes, tile_depth=4))
    assert auto["num_tiles"] == two["num_tiles"] and auto["deep_num_tiles"] == four["num_tiles"]
    assert auto["num_segments"] <= four["num_tiles"] < two["num_tiles"] <= 2 * four["num_tiles"]
    seg_bytes = 64 * auto["num_segments"]

    def tiling_bytes(ntiles, nchunks, slots):
        # tiles; chunk index; `slots` checksum accumulators per chunk, a 128-byte line each
        return 8 * ntiles + 4 * (nchunks + 1) + nchunks * slots * 128

    # 60 chunks of about 65 536 (depth 2) and 32 768 (depth 4) tiles: 256 accumulator slots each
    # (about 256 tiles per slot, a power of two, at most 256)
    assert two["device_table_bytes"] == seg_bytes + tiling_bytes(two["num_tiles"], two["num_chunks"], 256)
    assert auto["device_table_bytes"] == two["device_table_bytes"] + tiling_bytes(four["num_tiles"],
                                                                                   four["num_chunks"], 256)
    rs = dr.dr_plan_get_info(dr.dr_reshard_plan_create_host(wl.model, 8, 6, wl.chunk_bytes))
    assert (rs["deep_tile_elems"], rs["deep_num_tiles"]) == (0, 0)


def test_binding_fails_loudly_without_the_library(tmp_path):
    """No fallback: a copy of the package without libdr.so cannot even be imported."""
    import shutil
    import sys

    pkg = tmp_path / "paper_2607_22614_amd"
    pkg.mkdir()
    for f in os.listdir(os.path.join(ROOT, "paper_2607_22614_amd")):
        if f.endswith(".py"):
            shutil.copy(os.path.join(ROOT, "paper_2607_22614_amd", f), pkg / f)
    r = subprocess.run([sys.executable, "-c", "import paper_2607_22614_amd.dr"], cwd=tmp_path, capture_output=True,
                       text=True, timeout=120, env={**os.environ, "PYTHONPATH": str(tmp_path)})
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "libdr.so" in r.stderr and "build" in r.stderr


def test_plans_beyond_the_tile_index_are_refused_before_allocating():
    """N ~ 2^45 fp32 elements need more than 2^32 workgroup tiles, which 32-bit tile indices
    cannot address: both planners refuse it (DR_EINVAL) before building any table."""
    import time

    m = (0, 8192, 8, 8, 128, 8192, (1 << 31) - 8)
    # 2^32 - 2^24 <= tiles < 2^32: addressable, but a grid-stride tile index could wrap
    near = (0, 65536, 8, 8, 128, 65536, 511 << 17)
    for make in (lambda: dr.dr_plan_create_host(m, 1, 1, 1 << 40),
                 lambda: dr.dr_reshard_plan_create_host(m, 1, 2, 1 << 40),
                 lambda: dr.dr_plan_create_host(near, 1, 1, 1 << 40, tile_depth=2)):
        t0 = time.perf_counter()
        with pytest.raises(dr.DrError) as e:
            make()
        assert e.value.code == dr.DR_EINVAL and "too many tiles" in str(e.value)
        assert time.perf_counter() - t0 < 5.0


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
@pytest.mark.parametrize("std", ["c99", "c11"])
def test_header_is_strict_c(tmp_path, std):
    """include/dr.h is a C header: it compiles as strict ISO C with every warning an error, with
    nothing else included (the plain-C consumer in tests/native links the library this way)."""
    src = tmp_path / "h.c"
    src.write_text('#include "dr.h"\nint main(void) { dr_plan_info i; (void)i; return (int)sizeof(dr_layout) - 32; }\n')
    r = subprocess.run(["gcc", f"-std={std}", "-pedantic-errors", "-Wall", "-Wextra", "-Werror", "-I",
                        os.path.join(ROOT, "include"), str(src), "-o", str(tmp_path / "h")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    assert subprocess.run([str(tmp_path / "h")]).returncode == 0
