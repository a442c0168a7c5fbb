"""CPU checks of bench.py's contract pieces that need no GPU: the refusal of more than one GPU,
and the committed rocprofv3 summaries it reads the HBM traffic from."""
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def _fields(summary):
    fields = {}
    with open(os.path.join(ROOT, "profiles", summary)) as fh:
        for line in fh:
            if ": " in line:
                k, v = line.rsplit(": ", 1)
                fields[k.strip()] = v.strip()
    return fields


@pytest.mark.parametrize("summary,kernel,alg", [
    ("stage_kernel_8b_hbm_traffic.txt", "stage_kernel", 48183164928),
    ("stage_kernel_32b_hbm_traffic.txt", "stage_kernel", 196589752320),
    ("reshard_kernel_8b_8to6.txt", "reshard_kernel", 64242092032),
    ("moment_sum_kernel_8b_adam.txt", "moment_sum_kernel", 64242089984),
])
def test_traffic_summary_parses_and_matches_the_algorithmic_bytes(summary, kernel, alg):
    fields = _fields(summary)
    traffic = int(fields["traffic_bytes_per_launch"])
    assert int(fields.get("algorithmic_bytes_per_launch", alg)) == alg
    assert 1.0 <= traffic / alg < 1.05, "counted HBM bytes far from the algorithmic bytes"
    labels = [k for k in fields if k.startswith("kernel code sha256[:16]")]
    assert len(labels) == 1 and len(fields[labels[0]]) == 16
    current = labels[0] == bench.hash_label(kernel) and fields[labels[0]] == bench.kernel_source_hash(kernel)
    # bench reports the traffic only while the summary belongs to the kernel sources in the tree
    assert bench.profiled_traffic(summary, kernel) == (traffic if current else None)
    assert bench.profiled_traffic("no-such-summary.txt", kernel) is None


def test_the_kernel_hashes_cover_different_sources():
    hashes = {bench.kernel_source_hash(k) for k in ("stage_kernel", "reshard_kernel", "moment_sum_kernel")}
    assert len(hashes) == 3


def test_code_hash_ignores_comments_only():
    src = 'int f() { return 1; }  // one\n// two\nconst char* s = "a // b";\n'
    assert bench._code_only(src) == 'int f() { return 1; }\nconst char* s = "a // b";'
    assert bench._code_only(src + "// three\n") == bench._code_only(src)
    assert bench._code_only(src.replace("return 1", "return 2")) != bench._code_only(src)


def test_profile_summaries_name_their_commands():
    for name in os.listdir(os.path.join(ROOT, "profiles")):
        text = open(os.path.join(ROOT, "profiles", name)).read()
        assert "rocprofv3" in text and "bench.py" in text, name
        assert "_work" not in text, name


@pytest.mark.parametrize("workload,alg", [("8b", 48183164928), ("32b", 196589752320)])
def test_kernel_trace_summary_parses(workload, alg):
    """bench reports the profiled kernel mean (and its roofline fraction) from the committed trace
    summary only while the summary belongs to the kernel sources in the tree."""
    summary = f"stage_kernel_{workload}_kernel_trace.txt"
    fields = _fields(summary)
    mean_ms = float(fields["kernel_mean_us"]) / 1e3
    assert 0.5 < alg / mean_ms / 1e6 / 8000 < 1.0  # a fraction of the 8 TB/s peak
    current = fields.get(bench.hash_label("stage_kernel")) == bench.kernel_source_hash("stage_kernel")
    assert bench.profiled_kernel_ms(summary) == (mean_ms if current else None)
    assert bench.profiled_kernel_ms("no-such-summary.txt") is None
