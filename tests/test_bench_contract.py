"""bench.py's command-line contract and its measurement bookkeeping, on the CPU.

The timed run itself needs a GPU; these tests cover what does not: the refusal
of several GPUs, the exit without a GPU, the counter records that feed
`roofline.traffic` (taken only when the kernel source is the one the counters
were measured on) and the algorithmic counts behind `roofline.achieved`."""
import hashlib
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2603_04427_amd import accounting as acc  # noqa: E402
from synth import WORKLOADS  # noqa: E402


def run_bench(*args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, timeout=300, env=e)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_torchrun_world_size_is_refused_too():
    r = run_bench(env={"WORLD_SIZE": "8"})
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU may be visible here")
def test_no_gpu_exits_nonzero_without_a_line():
    r = run_bench("--steps", "1", "--warmup", "0")
    assert r.returncode != 0
    assert not any(line.startswith("{") for line in r.stdout.splitlines())


def test_traffic_records_name_existing_summaries_and_kernels():
    with open(bench.TRAFFIC_FILE) as f:
        recs = json.load(f)
    assert recs, "no counter records"
    for name, rec in recs.items():
        assert os.path.exists(os.path.join(ROOT, rec["summary"])), name
        assert rec["kernel"].startswith("void tk::"), name
        assert rec["bytes_per_call"] == pytest.approx(rec["read_bytes_per_call"] + rec["write_bytes_per_call"],
                                                      abs=2)
        # the plain-copy calibration: FETCH_SIZE counts 32-byte units of a 64-byte read
        assert rec["fetch_factor"] == pytest.approx(2.0, abs=0.01)
        assert rec["write_factor"] == pytest.approx(1.0, abs=0.01)


def test_traffic_is_taken_only_for_the_measured_source(tmp_path, monkeypatch):
    rec = {"x_decode": {"kernel": "void tk::k", "bytes_per_call": 123, "read_bytes_per_call": 100,
                        "write_bytes_per_call": 23, "fetch_factor": 2.0, "write_factor": 1.0,
                        "source_sha256": bench.source_sha("decode"), "summary": "s.md"},
           "x_stale": {"kernel": "void tk::k", "bytes_per_call": 456, "read_bytes_per_call": 400,
                       "write_bytes_per_call": 56, "fetch_factor": 2.0, "write_factor": 1.0,
                       "source_sha256": hashlib.sha256(b"an older source").hexdigest(), "summary": "s.md"}}
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(p))
    assert bench.traffic_for("x_decode", "decode") == 123
    assert bench.traffic_for("x_stale", "decode") is None
    assert bench.traffic_for("absent", "decode") is None


def test_decode_workload_bytes_are_320_per_token_head():
    spec = WORKLOADS["mistral_decode_b16"]
    n = acc.decode_bytes(spec.lens, spec.h_q, spec.h_kv, spec.r, spec.d_v, spec.k_dtype)
    units = spec.batch * spec.h_kv * spec.ctx
    # K and V rows of every visible token once, plus Q, O and the lengths
    assert n == units * 320 + spec.batch * spec.h_q * spec.r * 2 + spec.batch * spec.h_q * spec.d_v * 2 + \
        spec.batch * 4


def test_prefill_workload_flops_are_320_per_causal_pair():
    spec = WORKLOADS["mistral_prefill_s8192"]
    f = acc.prefill_flops(spec.batch, spec.h_q, spec.seq_q, spec.seq_k, spec.r, spec.d_v, spec.causal)
    pairs = spec.batch * spec.h_q * spec.seq_q * (spec.seq_q + 1) // 2
    assert f == pairs * 320


def test_secondary_lines_time_at_least_their_minimum():
    # the headline keeps exactly its steps
    assert bench.plan_timed_calls(200, 32e-6, 0.0) == 200
    # a 17 us kernel is timed for at least 50 ms, a 1 ms one for 51 calls
    assert bench.plan_timed_calls(10, 17e-6, 0.05) == int(0.05 / 17e-6) + 1
    assert bench.plan_timed_calls(10, 1e-3, 0.05) == 51
    # never fewer than asked, never more than the cap
    assert bench.plan_timed_calls(100, 1.0, 0.05) == 100
    assert bench.plan_timed_calls(10, 1e-9, 0.05) == bench.MAX_TIMED_CALLS


def test_every_traffic_record_names_a_known_kernel_source():
    with open(bench.TRAFFIC_FILE) as f:
        recs = json.load(f)
    shas = {bench.source_sha(kind) for kind in bench.KERNEL_SOURCES}
    for name, rec in recs.items():
        assert len(rec["source_sha256"]) == 64, name
        # a record is either current for one of the kernel sources or stale; a stale one reports no traffic
        kind = next((k for k in bench.KERNEL_SOURCES if bench.source_sha(k) == rec["source_sha256"]), None)
        if kind is None:
            assert rec["source_sha256"] not in shas
        else:
            assert bench.traffic_for(name, kind) == rec["bytes_per_call"]


def test_event_fields_carry_mean_median_and_min():
    rec = bench.event_ms(30e-6, (29.5e-6, 28.25e-6))
    assert rec == {"kernel_ms": 0.03, "single_call_ms_median": 0.0295, "single_call_ms_min": 0.02825}
