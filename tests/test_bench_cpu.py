"""CPU checks of the benchmark script's contract: it refuses more than one
GPU without printing a result line, it reports measured HBM traffic only
while the kernel sources are the ones the counters were taken on, and its
algorithmic bytes (the roofline's numerator) follow the payload geometry."""
import os
import shutil
import subprocess
import sys

import pytest

import bench
import oracle
from paper_2606_08635_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""  # no result line


def test_measured_traffic_follows_the_kernel_sources(monkeypatch):
    key = ("mistral7b_32k", "unpack")
    nbytes, kernel_file, _ = bench.MEASURED_TRAFFIC[key]
    monkeypatch.setitem(bench.MEASURED_TRAFFIC, key, (nbytes, kernel_file, bench.source_digest(kernel_file)))
    assert bench.measured_traffic(*key) == nbytes
    monkeypatch.setitem(bench.MEASURED_TRAFFIC, key, (nbytes, kernel_file, "0" * 16))
    assert bench.measured_traffic(*key) is None
    assert bench.measured_traffic("no_such_workload", "unpack") is None


def test_source_digest_covers_the_kernel_and_every_header(tmp_path, monkeypatch):
    src = tmp_path / "csrc"
    shutil.copytree(bench.CSRC, src)
    monkeypatch.setattr(bench, "CSRC", str(src))
    before = bench.source_digest("unpack.hip")
    for name in ("unpack.hip", "row_codec.h"):
        path = src / name
        original = path.read_bytes()
        # a line of code changes the digest
        path.write_bytes(original + b"\nstatic_assert(true, \"\");\n")
        assert bench.source_digest("unpack.hip") != before, name
        # comments and blank space do not
        path.write_bytes(original + b"\n// a note\n/* another\n note */\n\n")
        assert bench.source_digest("unpack.hip") == before, name
        path.write_bytes(original)
        assert bench.source_digest("unpack.hip") == before


@pytest.mark.parametrize("name", ["mistral7b_32k", "qwen7b_b0.3", "gemma9b_b0.7"])
def test_algorithmic_bytes_follow_the_payload_geometry(name):
    w = workloads.WORKLOADS[name]
    ocfg = oracle.config(w.layers, w.kv_heads, w.head_dim, w.tokens, w.budget, first_ratio=w.first_ratio,
                         decay=w.decay, num_tiers=w.num_tiers)
    plan = oracle.plan(ocfg)
    payload = oracle.payload_size(ocfg)
    pack, unpack = bench.algorithmic_bytes(w, plan, payload, 16)
    L, H, d, n = w.layers, w.kv_heads, w.head_dim, w.tokens
    F = 4 * L * H * d * n  # fp16 K and V
    kept_rows = 2 * L * H * (n - plan["n_drop"])
    # pack reads every non-dropped fp16 row and the byte tier map, and writes the payload
    assert pack == kept_rows * 2 * d + n + payload
    # unpack reads the payload and the int32 block table, and writes the whole fp16 cache
    assert unpack == payload + 4 * ((n + 15) // 16) + F
    if name == "mistral7b_32k":  # the headline request: no drops at b = 0.5
        assert plan["n_drop"] == 0 and payload == 2213258496
        assert (pack, unpack) == (6508258560, 6508233984)
