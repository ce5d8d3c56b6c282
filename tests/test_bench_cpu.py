"""Host-side logic of bench.py: the one-GPU contract, the benchmarked
workload, the counter record and the oracle baseline leg.  Nothing here
touches a GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_30342_amd import synth  # noqa: E402


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    """The step runs on one GPU: --gpus N > 1 exits with a message, before
    anything is initialised."""
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 2
    assert "one GPU" in out.stderr
    assert out.stdout == ""


@pytest.mark.parametrize("dtype,esize,stream_bytes", [
    ("fp32", 4, 2_490_568_004),
    ("bf16", 2, 1_743_929_156),
])
def test_benchmarked_set_is_gpt2_small(dtype, esize, stream_bytes):
    """GPT-2 small: 124,439,808 parameters in 50 matrices and 98 bias /
    LayerNorm vectors.  A streaming pass must read x, g, p and write x, p
    (3 * esize + 8 bytes per matrix element) and read R and C (4 bytes per
    row and column); a vector element also reads and writes its friction
    xi (3 * esize + 16 bytes)."""
    specs = synth.gpt2_small(dtype)
    mats = [s for s in specs if not s.is_vector]
    vecs = [s for s in specs if s.is_vector]
    assert (len(mats), len(vecs)) == (50, 98)
    assert sum(s.numel for s in specs) == 124_439_808
    assert all(s.dtype == dtype for s in specs)
    total = (sum(s.numel * (3 * esize + 8) + 4 * (s.m + s.n) for s in mats)
             + sum(s.numel * (3 * esize + 16) for s in vecs))
    assert total == stream_bytes


def test_counter_record_applies_only_to_the_sources_it_was_taken_on(tmp_path, monkeypatch):
    rec = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(rec))
    assert bench.measured_traffic("fp32") is None                 # no record
    rec.write_text("{not json")
    assert bench.measured_traffic("fp32") is None                 # unreadable
    body = {"fp32": {"bytes_per_launch": 123.0}}
    rec.write_text(json.dumps(dict(body, kernel_source_hash="0" * 16)))
    assert bench.measured_traffic("fp32") is None                 # other sources
    rec.write_text(json.dumps(dict(body, kernel_source_hash=bench.kernel_source_hash())))
    assert bench.measured_traffic("fp32") == 123.0
    assert bench.measured_traffic("bf16") is None                 # dtype not recorded


def test_committed_counter_record_is_well_formed():
    with open(bench.TRAFFIC_FILE) as f:
        rec = json.load(f)
    assert len(rec["kernel_source_hash"]) == 16
    for dtype, floor in (("fp32", 2_490_568_004), ("bf16", 1_743_929_156)):
        b = rec[dtype]["bytes_per_launch"]
        # counted HBM bytes cover at least the compulsory bytes, and the
        # partial sums add about 1%
        assert floor <= b < 1.05 * floor


def test_cpu_baseline_leg_times_the_oracle_on_a_sample():
    r = bench.cpu_baseline(synth.gpt2_small(), dict(synth.HP_BASE), 0.5)
    assert r["kind"] == "oracle" and r["unit"] == "params/s"
    assert r["value"] > 0 and r["single_thread_value"] > 0
    assert r["cores"] == len(os.sched_getaffinity(0))
    # wpe and block 0's four matrices and eight vectors
    sample = [s for s in synth.gpt2_small() if s.name == "wpe" or s.name.startswith("h0.")]
    assert len(sample) == 13
    assert f"({sum(s.numel for s in sample)} params, 13 tensors)" in r["sample"]
