"""Host-side parts of bench.py (CPU only): the one-GPU rule, the algorithmic
bytes and flops its roofline figures divide by, and the code hash that keeps
counter-based traffic figures tied to the sources they were taken on."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2502_06798_amd import synth  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("name,want", [
    # cache once + entry factors + queries (and scales) + top-k output, written out by hand
    ("b16_n10k_d768_f32", 10_000 * 768 * 4 + 4 * 10_000 + 16 * 768 * 4 + 8 * 16 * 5),
    ("b256_n100k_d768_f16", 154_413_696),
    ("b1024_n1m_d768_bf16", 1_000_000 * 1536 + 4_000_000 + 1024 * 1536 + 8 * 1024 * 10),
    ("b4096_n4m_d512_f16", 4_000_000 * 1024 + 16_000_000 + 4096 * 1024 + 8 * 4096 * 16),
    ("b16384_n10m_d768_e4m3", 7_736_842_752),
])
def test_algorithmic_bytes(name, want):
    assert bench.alg_bytes(synth.BY_NAME[name]) == want


def test_roofline_bound_per_workload():
    """The small batch is HBM-bound, the three large ones MFMA-bound (their
    arithmetic intensity against the ridge of the dtype's peak)."""
    bound = {}
    for name in ("b256_n100k_d768_f16", "b1024_n1m_d768_bf16", "b4096_n4m_d512_f16", "b16384_n10m_d768_e4m3"):
        w = synth.BY_NAME[name]
        ai = 2.0 * w.B * w.N * w.d / bench.alg_bytes(w)
        ridge = bench.PEAK_TFLOPS[w.dtype] * 1e12 / (bench.PEAK_HBM_GBS * 1e9)
        bound[name] = "hbm" if ai < ridge else "mfma"
    assert bound == {"b256_n100k_d768_f16": "hbm", "b1024_n1m_d768_bf16": "mfma",
                     "b4096_n4m_d512_f16": "mfma", "b16384_n10m_d768_e4m3": "mfma"}


def test_code_hash_ignores_comments_only(tmp_path):
    a, b, c = tmp_path / "a.h", tmp_path / "b.h", tmp_path / "c.h"
    a.write_text("int f(int x) { return x + 1; }\n")
    b.write_text("// a comment\n/* and\n   another */\n\nint f(int x) { return x + 1; }   // trailing\n")
    c.write_text("int f(int x) { return x + 2; }\n")
    assert bench.code_hash([str(a)]) == bench.code_hash([str(b)])
    assert bench.code_hash([str(a)]) != bench.code_hash([str(c)])


def test_traffic_table_covers_the_bench_workloads():
    assert set(bench.TRAFFIC_BYTES) == {"b256_n100k_d768_f16", "b1024_n1m_d768_bf16", "b4096_n4m_d512_f16",
                                        "b16384_n10m_d768_e4m3"}
    for name, nbytes in bench.TRAFFIC_BYTES.items():
        assert nbytes >= bench.alg_bytes(synth.BY_NAME[name])        # counters read at least the cache once
