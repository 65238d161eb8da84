#!/usr/bin/env python3
"""Benchmark of the thin-key attention hot path on one MI355X.

One step is one tk_attn_decode call on the Mistral-7B-shaped decode workload
(batch 16, 32 query / 8 KV heads, context 4096, r 32, d_v 128, bf16): the
workload the headline metric is quoted on. Inputs are generated on the GPU
before timing; the timed region rotates over several copies of the caches so
that the 168 MB step does not run out of the 256 MB last-level cache.

The JSON line reports, besides the contract fields:
  roofline      achieved algorithmic GB/s of the decode kernel (HIP events on
                the launch stream, averaged over the timed calls) against
                8 TB/s, the median and minimum of single calls timed one by
                one after the timed region, and the HBM traffic per call from
                rocprofv3 counters when they were taken on the current kernel
                sources;
  cpu_baseline  the fp64 oracle on the host cores, on a bounded sample of the
                same workload (not an optimisation target), with the CPU model,
                usable cores and OMP_NUM_THREADS; each secondary workload
                carries its own (whole decode steps; the whole GPT-2 prefill;
                64 rows of the 8192-token prefill, extrapolated);
  secondary     the other workloads, each with its own roofline: causal prefill
                at 8192 tokens (bf16 MFMA), the 131072-token paged decode, the
                fp8-key and 4-bit-key decodes, and the GPT-2 fp32 prefill;
  cache_append  the cache write before decode (tk_cache_append): 8192 new tokens
                per (sequence, KV head) of the prefill shape with bf16, fp8 and
                4-bit keys (quantised on write), and one decode token of the
                batch-16 shape;
  prefill_backward  the backward pass (dQ, dK, dV) of the 8192-token prefill,
                thin keys and the full-key control, against the bf16 MFMA peak
                with the algorithmic FLOPs 2 (3r + 2 d_v) per visible pair;
  decode_batch_sweep  the Mistral-shaped decode (context 4096) at batch 1, 4,
                8, 16 and 32 (the batch sizes of the paper's decode table), thin
                keys against standard-width keys, with the time ratio next to
                the byte ratio of the two caches;
  thin_projection  the three projections of a layer converted to thin keys
                (q' = x W_Q', k' = x W_K', v = x W_V, tk_project_heads) at the
                Mistral 8192-token and GPT-2 1024-token shapes, against the bf16
                MFMA peak;
  device        the part's CU count, architecture and engine clock levels, and
                the rates of torch's sum over 2 GiB and copy of 1 GiB on it
                (context for the fractions of the published peaks);
  fullkey_control  the batch-16 decode, the 8192-token prefill, the
                131072-token paged decode and the 4-bit-key decode again with
                standard-width bf16 keys (r = 128, same values), and the thin-key
                speedup over them next to the byte (decode) or FLOP (prefill)
                ratio that bounds it.
Every line but the headline times at least 50 ms of calls (more calls for the
short kernels, after a quarter as many extra warm-up calls) and reports the
number it timed in `timed_calls`; the headline times exactly --steps calls.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "thin-key decode-attn HBM GB/s (% peak); prefill-attn TFLOP/s (% MFMA peak)"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic.json")
SECONDARY_MIN_S = 0.05  # seconds of timed calls at least, for every line but the headline
KERNEL_SOURCES = {"decode": "paper_2603_04427_amd/csrc/decode.hip",
                  "prefill_bf16": "paper_2603_04427_amd/csrc/prefill_bf16.hip",
                  "prefill_f32": "paper_2603_04427_amd/csrc/prefill_f32.hip",
                  "prefill_bwd": "paper_2603_04427_amd/csrc/prefill_bwd.hip",
                  "append": "paper_2603_04427_amd/csrc/append.hip",
                  "project": "paper_2603_04427_amd/csrc/project.hip"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200, help="timed steps")
    ap.add_argument("--warmup", type=int, default=500,
                    help="untimed warm-up steps (enough for the GPU to reach its steady clocks; the "
                         "secondary workloads take a tenth of it, prefill at most 3, then the warm-up "
                         "that their 50 ms minimum of timed calls adds)")
    ap.add_argument("--rotate", type=int, default=8, help="cache copies cycled through in the timed loop")
    ap.add_argument("--only", default=None, help="time just this workload (e.g. for profiling)")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fullkey", action="store_true", help="skip the full-key (r = 128) control timings")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget for the oracle's host timing")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device three times (reads and writes a known number "
                         "of bytes, to scale the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


# Other units built from a kernel's file (decode_short.hip compiles decode.hip's
# eight-wave kernels), and the headers every kernel source includes: a change to
# any of them changes the kernels too.
EXTRA_SOURCES = {"decode": ("paper_2603_04427_amd/csrc/decode_short.hip",)}
SHARED_SOURCES = ("paper_2603_04427_amd/csrc/tk_device.hpp", "paper_2603_04427_amd/csrc/tk_internal.hpp")


def kernel_source_files(kind: str) -> tuple:
    """The files a kernel is built from, in the order source_sha hashes them."""
    return (KERNEL_SOURCES[kind],) + EXTRA_SOURCES.get(kind, ()) + SHARED_SOURCES


def source_sha(kind: str) -> str:
    """SHA-256 over the sources a kernel is built from (kernel_source_files)."""
    h = hashlib.sha256()
    for path in kernel_source_files(kind):
        with open(os.path.join(ROOT, path), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_for(workload: str, kind: str):
    """HBM bytes per call from committed rocprofv3 counter runs, if taken on this source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(workload)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha256") != source_sha(kind):
        return None
    return rec.get("bytes_per_call")


def event_ms(ev: float, one) -> dict:
    """Time fields of a roofline record: the mean over the back-to-back timed calls
    (the denominator of ``achieved``), and the median and minimum of single calls,
    each between its own events. A single call's figure also holds the gap the
    event between two calls leaves (the next launch no longer overlaps the end of
    the previous kernel), so it sits above the mean for short kernels."""
    return {"kernel_ms": round(ev * 1e3, 5), "single_call_ms_median": round(one[0] * 1e3, 5),
            "single_call_ms_min": round(one[1] * 1e3, 5)}


MAX_TIMED_CALLS = 5000
PER_CALL_MAX = 200  # single calls timed one by one after the timed region


def plan_timed_calls(steps: int, one_call_s: float, min_timed_s: float) -> int:
    """Timed calls for a line: ``steps``, raised (up to MAX_TIMED_CALLS) until
    they cover ``min_timed_s`` at ``one_call_s`` per call; unchanged when
    ``min_timed_s`` is 0 (the headline times exactly the steps it is given)."""
    if min_timed_s <= 0:
        return steps
    return max(steps, min(MAX_TIMED_CALLS, int(min_timed_s / max(one_call_s, 1e-6)) + 1))


def time_calls(calls, steps: int, warmup: int, min_timed_s: float = 0.0):
    """Warm up, then time ``steps`` calls (cycling through ``calls``).

    With ``min_timed_s`` > 0 (the secondary workloads; the headline line times
    exactly the steps it is given) the timed calls are raised, up to MAX_TIMED_CALLS, until
    they cover at least that many seconds, and as many extra warm-up calls as a
    quarter of them run first: a few calls of a kernel of some microseconds would
    otherwise time the host's launch gaps and the clock's ramp, not the kernel.

    Returns (wall seconds per step, event seconds per step, timed calls,
    (median, min) seconds of single calls). The wall clock is bracketed by device
    synchronisation; the events sit on the launch stream. After the timed region,
    as many calls again (at most PER_CALL_MAX) are timed one by one, an event
    recorded between consecutive calls, for the median and the minimum of a
    single call."""
    import torch
    n = len(calls)
    for i in range(warmup):
        calls[i % n]()
    torch.cuda.synchronize()
    if min_timed_s > 0:
        t = time.perf_counter()
        calls[0]()
        torch.cuda.synchronize()
        steps = plan_timed_calls(steps, time.perf_counter() - t, min_timed_s)
        for i in range(steps // 4):
            calls[i % n]()
        torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(st)
    for i in range(steps):
        calls[i % n]()
    e1.record(st)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    ev = e0.elapsed_time(e1) / 1e3 / steps
    m = min(steps, PER_CALL_MAX)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(m + 1)]
    marks[0].record(st)
    for i in range(m):
        calls[i % n]()
        marks[i + 1].record(st)
    torch.cuda.synchronize()
    one = sorted(marks[i].elapsed_time(marks[i + 1]) / 1e3 for i in range(m))
    return wall, ev, steps, (one[m // 2], one[0])


def decode_setup(spec, dev, rotate: int):
    import torch
    from paper_2603_04427_amd import prepare_decode, tk_attn_decode_workspace_bytes
    from synth import make_decode

    d = make_decode(spec, device=dev)
    d.pop("k_logical"), d.pop("v_logical"), d.pop("k_scale_logical")
    torch.cuda.empty_cache()
    ws = torch.zeros(tk_attn_decode_workspace_bytes(spec.batch, spec.h_q, spec.h_kv, spec.ctx, spec.d_v),
                     dtype=torch.uint8, device=dev)
    out = torch.empty(spec.batch, spec.h_q, spec.d_v, dtype=torch.bfloat16, device=dev)
    copies = [(d["k"], d["v"], d["k_scale"])]
    for _ in range(rotate - 1):
        copies.append((d["k"].clone(), d["v"].clone(), None if d["k_scale"] is None else d["k_scale"].clone()))
    calls = [prepare_decode(d["q"], k, v, d["ctx_lens"], max_ctx=spec.ctx, scale=spec.softmax_scale, k_scale=ks,
                            block_table=d["block_table"], block_size=spec.block_size if spec.paged else 0,
                            workspace=ws, O=out) for (k, v, ks) in copies]
    return calls


def decode_result(name, spec, calls, steps, warmup, min_timed_s=0.0):
    from paper_2603_04427_amd import accounting as acc
    wall, ev, steps, one = time_calls(calls, steps, warmup, min_timed_s)
    nbytes = acc.decode_bytes(spec.lens, spec.h_q, spec.h_kv, spec.r, spec.d_v, spec.k_dtype,
                              spec.blocks_per_seq if spec.paged else None)
    achieved = nbytes / ev / 1e9
    traffic = traffic_for(name, "decode")
    return {
        "workload": name, "value": round(nbytes / wall / 1e9, 1), "unit": "GB/s",
        "ms_per_call": round(wall * 1e3, 5), "timed_calls": steps,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": acc.HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / acc.HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes": nbytes, **event_ms(ev, one)},
    }


def prefill_result(name, spec, dev, steps, warmup, min_timed_s=0.0):
    import torch
    from paper_2603_04427_amd import accounting as acc
    from paper_2603_04427_amd import prepare_prefill
    from synth import make_prefill

    p = make_prefill(spec, device=dev)
    call = prepare_prefill(p["q"], p["k"], p["v"], causal=spec.causal, scale=spec.softmax_scale)
    wall, ev, steps, one = time_calls([call], steps, warmup, min_timed_s)
    flops = acc.prefill_flops(spec.batch, spec.h_q, spec.seq_q, spec.seq_k, spec.r, spec.d_v, spec.causal)
    peak = acc.BF16_MFMA_PEAK_TFLOPS if spec.dtype == "bf16" else acc.FP32_MFMA_PEAK_TFLOPS
    achieved = flops / ev / 1e12
    kind = "prefill_bf16" if spec.dtype == "bf16" else "prefill_f32"
    del p, call
    torch.cuda.empty_cache()
    return {
        "workload": name, "value": round(flops / wall / 1e12, 2), "unit": "TFLOP/s",
        "ms_per_call": round(wall * 1e3, 5), "timed_calls": steps, "dtype": spec.dtype,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": traffic_for(name, kind),
                     "algorithmic_flops": flops, **event_ms(ev, one)},
    }


def backward_result(name, spec, dev, steps, warmup, min_timed_s=0.0):
    """tk_attn_prefill_backward (both kernels) on a prefill shape; the forward with
    log-sum-exp runs once, untimed, to produce O and lse."""
    import torch
    from paper_2603_04427_amd import accounting as acc
    from paper_2603_04427_amd import prepare_prefill_backward, tk_attn_prefill_lse
    from synth import make_prefill, make_prefill_grad

    p = make_prefill(spec, device=dev)
    do = make_prefill_grad(spec, device=dev)
    o, lse = tk_attn_prefill_lse(p["q"], p["k"], p["v"], causal=spec.causal, scale=spec.softmax_scale)
    call = prepare_prefill_backward(p["q"], p["k"], p["v"], o, do, lse, causal=spec.causal,
                                    scale=spec.softmax_scale)
    wall, ev, steps, one = time_calls([call], steps, warmup, min_timed_s)
    flops = acc.prefill_backward_flops(spec.batch, spec.h_q, spec.seq_q, spec.seq_k, spec.r, spec.d_v,
                                       spec.causal)
    peak = acc.BF16_MFMA_PEAK_TFLOPS
    achieved = flops / ev / 1e12
    del p, do, o, lse, call
    torch.cuda.empty_cache()
    return {
        "workload": name, "value": round(flops / wall / 1e12, 2), "unit": "TFLOP/s",
        "ms_per_call": round(wall * 1e3, 5), "timed_calls": steps, "dtype": spec.dtype,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": traffic_for(name, "prefill_bwd"),
                     "algorithmic_flops": flops, **event_ms(ev, one),
                     "kernels": "bwd_dq_kernel + bwd_dkdv_kernel"},
    }


SWEEP_BATCHES = (1, 4, 8, 16, 32)


def batch_sweep(dev, steps, warmup, rotate):
    """Decode at the batch sizes of the paper's decode table (Mistral-7B shape,
    context 4096): thin keys (r 32) against standard-width keys (r 128, same
    values), with the ratio of the two times next to the ratio of the bytes
    the two caches hold (the attention-only form of Eq. 10)."""
    import torch
    from dataclasses import replace
    from paper_2603_04427_amd import accounting as acc
    from synth import WORKLOADS

    base = WORKLOADS["mistral_decode_b16"]
    out = []
    for B in SWEEP_BATCHES:
        row = {"batch": B}
        for tag, r in (("thin", 32), ("full", 128)):
            spec = replace(base, name=f"decode_b{B}_{tag}", batch=B, r=r)
            calls = decode_setup(spec, dev, rotate)
            res = decode_result(spec.name, spec, calls, steps, warmup, SECONDARY_MIN_S)
            del calls
            torch.cuda.empty_cache()
            row[tag] = {"kernel_ms": res["roofline"]["kernel_ms"], "GBps": res["roofline"]["achieved"],
                        "frac": res["roofline"]["frac"]}
        nb = lambda r: acc.decode_bytes((base.ctx,) * B, base.h_q, base.h_kv, r, base.d_v, "bf16")
        row["thin_key_speedup"] = round(row["full"]["kernel_ms"] / row["thin"]["kernel_ms"], 3)
        row["byte_ratio"] = round(nb(128) / nb(32), 3)
        out.append(row)
    return out


PROJECTION_CASES = {  # (B, S, d_model, h_q, h_kv, r, d_v): a converted layer's three projections
    "thin_projection_mistral_s8192": (4, 8192, 4096, 32, 8, 32, 128),
    "thin_projection_gpt2_s1024": (1, 1024, 768, 12, 12, 16, 64),
}


def projection_result(name, B, S, d_model, h_q, h_kv, r, dv, dev, steps, warmup, min_timed_s=0.0):
    """q' = x W_Q', k' = x W_K' and v = x W_V of a layer converted to thin keys:
    three tk_project_heads calls per step, random bf16 weights of the converted shapes."""
    import torch
    from paper_2603_04427_amd import accounting as acc
    from paper_2603_04427_amd import prepare_project_heads
    from synth import normal, stream_key

    x = normal(stream_key(21, 0), B * S * d_model, device=dev).view(B, S, d_model).to(torch.bfloat16)
    calls, cols = [], 0
    for t, (n, w) in enumerate(((h_q, r), (h_kv, r), (h_kv, dv))):
        wt = (normal(stream_key(21, 1 + t), n * w * d_model, device=dev).view(n * w, d_model) *
              d_model ** -0.5).to(torch.bfloat16)
        calls.append(prepare_project_heads(x, wt, n))
        cols += n * w

    def step():
        for c in calls:
            c()
    wall, ev, steps, one = time_calls([step], steps, warmup, min_timed_s)
    flops = 2 * B * S * d_model * cols
    achieved = flops / ev / 1e12
    del x, calls
    torch.cuda.empty_cache()
    return {
        "workload": name, "value": round(flops / wall / 1e12, 2), "unit": "TFLOP/s",
        "ms_per_call": round(wall * 1e3, 5), "timed_calls": steps, "dtype": "bf16",
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": acc.BF16_MFMA_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / acc.BF16_MFMA_PEAK_TFLOPS, 4),
                     "traffic": traffic_for(name, "project"), "algorithmic_flops": flops,
                     **event_ms(ev, one), "kernels": "project_kernel x 3 (q', k', v)"},
    }


APPEND_CASES = {"cache_append_s8192": (4, 8192, "bf16"), "cache_append_fp8_s8192": (4, 8192, "fp8"),
                "cache_append_int4_s8192": (4, 8192, "int4"), "cache_append_decode_b16": (16, 1, "bf16")}


def append_result(name, B, Hkv, T, r, dv, kdt, dev, steps, warmup, min_timed_s=0.0, rotate=8):
    """tk_cache_append of T new tokens per (sequence, KV head) into a contiguous cache
    with bf16, fp8 or 4-bit keys (``kdt``). The timed calls cycle through ``rotate``
    copies of the new rows and of the cache (each copy its own buffers), so that a
    call's reads do not find the previous call's lines in the last-level cache."""
    import torch
    from paper_2603_04427_amd import prepare_cache_append
    from synth import normal, stream_key

    kn0 = normal(stream_key(20, 0), B * Hkv * T * r, device=dev).view(B, Hkv, T, r).to(torch.bfloat16)
    vn0 = normal(stream_key(20, 1), B * Hkv * T * dv, device=dev).view(B, Hkv, T, dv).to(torch.bfloat16)
    quant = kdt != "bf16"
    pos = torch.zeros(B, dtype=torch.int32, device=dev)
    bufs, calls = [], []
    for i in range(max(1, rotate)):
        kn, vn = (kn0, vn0) if i == 0 else (kn0.clone(), vn0.clone())
        kc = torch.zeros(B, Hkv, T, r // 2 if kdt == "int4" else r, dtype=torch.uint8 if quant else torch.bfloat16,
                         device=dev)
        vc = torch.zeros(B, Hkv, T, dv, dtype=torch.bfloat16, device=dev)
        ks = torch.zeros(B, Hkv, T, dtype=torch.float32, device=dev) if quant else None
        bufs.append((kn, vn, kc, vc, ks))
        calls.append(prepare_cache_append(kn, vn, pos, kc, vc, k_scale=ks))
    wall, ev, steps, one = time_calls(calls, steps, warmup, min_timed_s)
    tokens = B * Hkv * T
    key_out = {"bf16": r * 2, "fp8": r + 4, "int4": r // 2 + 4}[kdt]
    nbytes = tokens * (r * 2 + dv * 2) + B * 4 + tokens * key_out + tokens * dv * 2
    del kn0, vn0, bufs, calls
    torch.cuda.empty_cache()
    from paper_2603_04427_amd import accounting as acc
    return {
        "workload": name, "value": round(nbytes / wall / 1e9, 1), "unit": "GB/s",
        "ms_per_call": round(wall * 1e3, 5), "timed_calls": steps, "rotate": max(1, rotate),
        "roofline": {"bound": "hbm", "achieved": round(nbytes / ev / 1e9, 1), "peak": acc.HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(nbytes / ev / 1e9 / acc.HBM_PEAK_GBS, 4),
                     "traffic": traffic_for(name, "append"), "algorithmic_bytes": nbytes,
                     **event_ms(ev, one)},
    }


def host_info():
    """The host the oracle runs on: CPU model, cores this process may use, OpenMP threads."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    nproc = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"cpu_model": model, "nproc": nproc, "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def _repeat(fn, budget_s: float):
    """Runs fn until budget_s has passed (at least once); returns (runs, seconds)."""
    reps, t0 = 0, time.perf_counter()
    while True:
        fn()
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            return reps, el


def cpu_baseline(spec, budget_s: float, dev=None):
    """The fp64 oracle on the host cores, timed on a bounded sample of the workload.

    Decode: whole steps (every sequence and head), inputs drawn on the GPU when one
    is given and copied to the host once. Prefill: the whole call when it is small
    (the GPT-2 shape), otherwise the last 64 query rows of sequence 0, all heads
    (bottom-right aligned, so each row sees its full causal prefix), with the
    whole call's time extrapolated from the sample's FLOP rate."""
    import torch
    from oracle import oracle
    from paper_2603_04427_amd import accounting as acc
    from synth import make_decode, make_prefill

    info = {"cores": oracle.max_threads(), "kind": "oracle", **host_info()}
    if hasattr(spec, "ctx"):
        d = make_decode(spec, device=dev if dev is not None else "cpu")
        q, v, lens = d["q"].cpu(), d["v_logical"].cpu(), d["ctx_lens"].cpu()
        k = d["k_logical"].cpu()
        ks = None if d["k_scale_logical"] is None else d["k_scale_logical"].cpu()
        del d
        torch.cuda.empty_cache() if torch.cuda.is_available() else None
        keys = oracle.Int4(k) if spec.k_dtype == "int4" else k
        nbytes = acc.decode_bytes(spec.lens, spec.h_q, spec.h_kv, spec.r, spec.d_v, spec.k_dtype,
                                  spec.blocks_per_seq if spec.paged else None)
        reps, el = _repeat(lambda: oracle.decode(q, keys, v, lens, scale=spec.softmax_scale, k_scale=ks), budget_s)
        del q, k, v, keys
        return {"value": round(nbytes * reps / el / 1e9, 3), "unit": "GB/s", **info,
                "sample": f"{reps} whole decode steps of {spec.name} (fp64 C oracle, OpenMP, on the contiguous "
                          f"logical cache), {el:.1f} s", "seconds_per_step": round(el / reps, 4)}
    p = make_prefill(spec, device=dev if dev is not None else "cpu")
    whole = spec.batch * spec.h_q * spec.seq_q * spec.seq_k <= (1 << 26)
    if whole:
        q, kk, vv = p["q"].cpu(), p["k"].cpu(), p["v"].cpu()
        flops = acc.prefill_flops(spec.batch, spec.h_q, spec.seq_q, spec.seq_k, spec.r, spec.d_v, spec.causal)
        what = f"the whole {spec.name} call"
    else:
        n = 64
        q, kk, vv = p["q"][:1, :, -n:].cpu(), p["k"][:1].cpu(), p["v"][:1].cpu()
        flops = acc.prefill_flops(1, spec.h_q, n, spec.seq_k, spec.r, spec.d_v, spec.causal)
        what = f"the last {n} query rows of sequence 0 of {spec.name}, all {spec.h_q} heads"
    del p
    torch.cuda.empty_cache() if torch.cuda.is_available() else None
    reps, el = _repeat(lambda: oracle.prefill(q, kk, vv, causal=spec.causal, scale=spec.softmax_scale), budget_s)
    rate = flops * reps / el
    full = acc.prefill_flops(spec.batch, spec.h_q, spec.seq_q, spec.seq_k, spec.r, spec.d_v, spec.causal)
    return {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", **info,
            "sample": f"{reps} runs of {what} (fp64 C oracle, OpenMP), {el:.1f} s",
            "seconds_per_step": round(full / rate, 3),
            "seconds_per_step_is": "measured" if whole else "extrapolated from the sample's FLOP rate"}


def copy_calibration(mib: int, dev):
    """A plain streaming kernel of known size: each launch reads ``mib`` MiB once and
    writes ``mib`` MiB once (an elementwise bitwise-not, so it is a shader kernel and
    not a DMA-engine copy)."""
    import torch
    n = mib << 20
    src = torch.ones(n // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.bitwise_not(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n, "launches": 3}))


PROBE_LIB = os.path.join(ROOT, "paper_2603_04427_amd", "libtkprobe.so")


def stream_read_rates(dev, nbytes: int = 167936064, copies: int = 8, grid: int = 256, reps: int = 50) -> dict:
    """A plain streaming read of ``nbytes`` (the batch-16 decode step's bytes) with
    the probe kernel (libtkprobe: ``grid`` workgroups, four 16-byte loads in flight
    per lane, grid-stride), cycling through ``copies`` buffers so that no read is
    served from the last-level cache; with ordinary and with non-temporal loads.
    The mean over ``reps`` back-to-back launches, from HIP events."""
    import ctypes
    import torch
    lib = ctypes.CDLL(PROBE_LIB)  # built beside libtkattn; a missing probe is an error
    lib.tkprobe_threads.restype = ctypes.c_int
    lib.tkprobe_stream_read.restype = ctypes.c_int
    lib.tkprobe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_void_p]
    n = nbytes // 16 * 16
    bufs = [torch.ones(n, dtype=torch.uint8, device=dev) for _ in range(copies)]
    sink = torch.empty(grid * lib.tkprobe_threads(), dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream()
    out = {"bytes": n, "copies": copies, "workgroups": grid, "threads": lib.tkprobe_threads()}
    for nt, key in ((0, "GBps"), (1, "non_temporal_GBps")):
        def call(i):
            rc = lib.tkprobe_stream_read(ctypes.c_void_p(bufs[i % copies].data_ptr()), n,
                                         ctypes.c_void_p(sink.data_ptr()), grid, nt, ctypes.c_void_p(st.cuda_stream))
            if rc != 0:
                raise RuntimeError(f"tkprobe_stream_read returned {rc}")
        for i in range(2 * copies):
            call(i)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for i in range(reps):
            call(i)
        e1.record(st)
        torch.cuda.synchronize()
        out[key] = round(n / (e0.elapsed_time(e1) / 1e3 / reps) / 1e9, 1)
    del bufs, sink
    torch.cuda.empty_cache()
    return out


def device_context(dev):
    """What the part reports and plain streaming rates measured on it, as context
    for the roofline fractions (which use the published peaks): CU count and
    architecture, the engine clock levels the driver lists, a plain streaming
    read of the decode step's size by a probe kernel (``stream_read``), and the
    rates of torch's own kernels for a read-only sum over 2 GiB and a 1 GiB copy
    (best of 5, HIP events), which are library kernels, not the part's ceiling."""
    import glob
    import torch
    props = torch.cuda.get_device_properties(dev)
    ctx = {"name": props.name, "arch": props.gcnArchName, "cus": props.multi_processor_count,
           "sclk_mhz_levels": None, "stream_read": None, "torch_sum_read_GBps": None, "torch_copy_GBps": None}
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            with open(path) as f:
                levels = [int(t.rstrip("*").lower().replace("mhz", ""))
                          for line in f for t in line.split()[1:2] if t.lower().rstrip("*").endswith("mhz")]
            if levels:
                ctx["sclk_mhz_levels"] = levels
                break
        except (OSError, ValueError):
            continue

    def best(fn, nbytes):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()
        torch.cuda.synchronize()
        t = []
        for _ in range(5):
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1) / 1e3)
        return round(nbytes / min(t) / 1e9, 1)

    ctx["stream_read"] = stream_read_rates(dev)
    x = torch.ones((2 << 30) // 4, dtype=torch.float32, device=dev)
    ctx["torch_sum_read_GBps"] = best(lambda: x.sum(), x.numel() * 4)
    del x
    src = torch.ones((1 << 30) // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    ctx["torch_copy_GBps"] = best(lambda: dst.copy_(src), 2 * src.numel() * 4)
    del src, dst
    torch.cuda.empty_cache()
    return ctx


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: measures one GPU only; the thin-key attention kernels are not sharded across "
              "GPUs. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    from synth import FULLKEY, INT4KEY, WORKLOADS
    workloads = {**WORKLOADS, **INT4KEY, **FULLKEY}

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda", 0)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, dev)
        return
    if args.only and args.only.startswith("cache_append"):
        B, T, kdt = APPEND_CASES[args.only]
        res = append_result(args.only, B, 8, T, 32, 128, kdt, dev, args.steps, args.warmup, rotate=args.rotate)
        print(json.dumps({"metric": "cache append HBM GB/s", "value": res["value"], "unit": "GB/s", "n_gpus": 1,
                          "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_call"],
                          "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
                          "data": "synthetic", "config": {"workload": args.only}, "roofline": res["roofline"]}),
              flush=True)
        return
    if args.only and args.only.startswith("thin_projection"):
        res = projection_result(args.only, *PROJECTION_CASES[args.only], dev, args.steps, min(args.warmup, 5))
        print(json.dumps({"metric": "thin projection TFLOP/s", "value": res["value"], "unit": "TFLOP/s",
                          "n_gpus": 1, "steps": args.steps, "warmup": min(args.warmup, 5),
                          "ms_per_step": res["ms_per_call"], "higher_is_better": True, "scaling": "weak",
                          "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                          "config": {"workload": args.only}, "roofline": res["roofline"]}), flush=True)
        return
    if args.only and args.only.endswith("_backward"):
        spec = workloads[args.only[:-len("_backward")]]
        res = backward_result(args.only, spec, dev, args.steps, min(args.warmup, 3))
        print(json.dumps({"metric": "prefill backward TFLOP/s", "value": res["value"], "unit": "TFLOP/s",
                          "n_gpus": 1, "steps": args.steps, "warmup": min(args.warmup, 3),
                          "ms_per_step": res["ms_per_call"], "higher_is_better": True, "scaling": "weak",
                          "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                          "config": {"workload": args.only}, "roofline": res["roofline"]}), flush=True)
        return
    main_name = args.only or "mistral_decode_b16"
    results = {}
    order = [main_name] if (args.no_secondary or args.only) else \
        [main_name] + [n for n in ("mistral_prefill_s8192", "longctx_paged_decode", "fp8key_decode",
                                   "int4key_decode", "gpt2_prefill_f32") if n != main_name]
    def run(name, spec, main=False):
        print(f"bench: timing {name}", file=sys.stderr, flush=True)
        if hasattr(spec, "ctx"):
            big = spec.batch * spec.h_kv * spec.ctx * (spec.r + spec.d_v) * 2 > (1 << 30)
            calls = decode_setup(spec, dev, 1 if big else args.rotate)
            steps = args.steps if main else max(10, args.steps // 10)
            res = decode_result(name, spec, calls, steps, args.warmup if main else max(10, args.warmup // 10),
                                0.0 if main else SECONDARY_MIN_S)
            res["rotate"] = len(calls)
            del calls
            torch.cuda.empty_cache()
        else:
            steps = args.steps if main else max(5, args.steps // 20)
            res = prefill_result(name, spec, dev, steps, min(args.warmup, 3), 0.0 if main else SECONDARY_MIN_S)
        return res

    for name in order:
        results[name] = run(name, workloads[name], main=name == main_name)
    fullkey = []
    if not (args.no_fullkey or args.only or args.no_secondary):
        from paper_2603_04427_amd import accounting as acc
        for name, spec in FULLKEY.items():
            thin = results[name[:-len("_fullkey")]]
            full = run(name, spec)
            tspec = workloads[name[:-len("_fullkey")]]
            if hasattr(spec, "ctx"):
                ideal = acc.decode_bytes(spec.lens, spec.h_q, spec.h_kv, spec.r, spec.d_v, spec.k_dtype) / \
                    acc.decode_bytes(tspec.lens, tspec.h_q, tspec.h_kv, tspec.r, tspec.d_v, tspec.k_dtype)
            else:
                ideal = (spec.r + spec.d_v) / (tspec.r + tspec.d_v)
            full["thin_key_speedup"] = round(full["roofline"]["kernel_ms"] / thin["roofline"]["kernel_ms"], 3)
            full["ideal_speedup"] = round(ideal, 3)
            fullkey.append(full)
    backward = []
    if not (args.only or args.no_secondary):
        for base in ("mistral_prefill_s8192", "mistral_prefill_s8192_fullkey"):
            print(f"bench: timing {base}_backward", file=sys.stderr, flush=True)
            backward.append(backward_result(base + "_backward", workloads[base], dev, max(5, args.steps // 20),
                                            min(args.warmup, 3), SECONDARY_MIN_S))
        if len(backward) == 2:
            thin, full = backward
            full["thin_key_speedup"] = round(full["roofline"]["kernel_ms"] / thin["roofline"]["kernel_ms"], 3)
            tspec, fspec = workloads["mistral_prefill_s8192"], workloads["mistral_prefill_s8192_fullkey"]
            full["ideal_speedup"] = round((3 * fspec.r + 2 * fspec.d_v) / (3 * tspec.r + 2 * tspec.d_v), 3)
    appends = []
    if not (args.only or args.no_secondary):
        for name, (B, T, kdt) in APPEND_CASES.items():
            print(f"bench: timing {name}", file=sys.stderr, flush=True)
            appends.append(append_result(name, B, 8, T, 32, 128, kdt, dev, max(10, args.steps // 10),
                                         args.warmup, SECONDARY_MIN_S, rotate=args.rotate))
    projections = []
    if not (args.only or args.no_secondary):
        for name, shape in PROJECTION_CASES.items():
            print(f"bench: timing {name}", file=sys.stderr, flush=True)
            projections.append(projection_result(name, *shape, dev, max(10, args.steps // 10), min(args.warmup, 5),
                                                 SECONDARY_MIN_S))
    sweep = []
    if not (args.only or args.no_secondary or args.no_fullkey):
        print("bench: timing the decode batch sweep", file=sys.stderr, flush=True)
        sweep = batch_sweep(dev, max(20, args.steps // 4), max(20, args.warmup // 10), args.rotate)
    m = results[main_name]
    spec = workloads[main_name]
    is_decode = hasattr(spec, "ctx")
    line = {
        "metric": METRIC, "value": m["value"], "unit": m["unit"], "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": m["ms_per_call"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": (spec.dtype if not is_decode else
                                       "bf16" if spec.k_dtype == "bf16" else f"{spec.k_dtype}-keys/bf16"),
        "data": ("synthetic (seeded N(0,1) draws shaped like the paper's Mistral-7B decode)"
                 if main_name == "mistral_decode_b16" else f"synthetic (seeded N(0,1) draws, workload {main_name})"),
        "config": ({"workload": main_name, "batch": spec.batch, "h_q": spec.h_q, "h_kv": spec.h_kv,
                    "ctx": spec.ctx, "r": spec.r, "d_v": spec.d_v, "k_dtype": spec.k_dtype,
                    "layout": "paged" if spec.paged else "contiguous", "rotate": m.get("rotate")}
                   if is_decode else
                   {"workload": main_name, "batch": spec.batch, "h_q": spec.h_q, "h_kv": spec.h_kv,
                    "seq": spec.seq_q, "r": spec.r, "d_v": spec.d_v, "causal": spec.causal}),
        "roofline": m["roofline"],
    }
    if not args.no_cpu_baseline:
        print(f"bench: oracle on the host cores ({main_name})", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(spec, args.cpu_seconds, dev)
        for n in order:
            if n != main_name:
                print(f"bench: oracle on the host cores ({n})", file=sys.stderr, flush=True)
                results[n]["cpu_baseline"] = cpu_baseline(workloads[n], args.cpu_seconds / 2, dev)
    line["secondary"] = [results[n] for n in order if n != main_name]
    if fullkey:
        line["fullkey_control"] = fullkey
    if backward:
        line["prefill_backward"] = backward
    if appends:
        line["cache_append"] = appends
    if projections:
        line["thin_projection"] = projections
    if sweep:
        line["decode_batch_sweep"] = sweep
    line["device"] = device_context(dev)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
