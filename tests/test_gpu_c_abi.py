"""The C ABI from a plain C program (tests/native/c_consumer.c, built by build() with gcc).

The program links only libdr.so and the HIP runtime: it uploads the shards, stages the stream with
dr_stage_all, re-stages every chunk with dr_stage_chunk and checks it against that, round-trips the
moments through malloc'd host memory, and writes the stream and checksums to files.  Here those
files are compared with the oracle, byte for byte."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2607_22614_amd import datagen, workloads
from tests.gpu_helpers import require_gpu, say

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "c_consumer")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    assert os.path.exists(EXE), f"{EXE} is missing: run __graft_entry__.build() first"


@pytest.mark.parametrize("model,w,t,b,bm,specials", [
    (workloads.TINY.model, 4, 2, 256 * 1024, 48 * 1024 + 16, 0.001),
    ((2, 24, 3, 3, 2, 27, 48), 3, 3, 48, 1040, 0.3),  # column runs of 2 and 9 elements: unaligned paths
    (workloads.TINY.model, 1, 4, 16, 0, 0.0),          # 16-byte chunks, no moment path
])
def test_plain_c_consumer_matches_the_oracle(tmp_path, model, w, t, b, bm, specials):
    flat = datagen.make_flat_numpy(model, w, seed=7, specials_frac=specials)
    src = tmp_path / "flat.bin"
    flat.astype("<f4").tofile(src)
    out_stream, out_cks = tmp_path / "stream.bin", tmp_path / "cks.bin"
    args = [EXE, str(src), str(out_stream), str(out_cks), *map(str, model), str(w), str(t), str(b), str(bm)]
    say("c_consumer", model, "W", w, "T", t, "B", b, "Bm", bm)
    r = subprocess.run(args, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c_consumer ok" in r.stdout
    m = oracle.Model(*model)
    want = oracle.rollout_stream(oracle.training_views(flat.view(np.uint32), m), m, t)
    got = np.fromfile(out_stream, dtype="<u2")
    assert np.array_equal(got, want)
    cks = np.fromfile(out_cks, dtype="<u8").reshape(-1, 2)
    assert [(int(x), int(y)) for x, y in cks] == oracle.chunk_checksums(want, b)
