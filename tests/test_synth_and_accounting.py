"""Seeded input generator, fp8 key quantisation, and the paper's byte accounting."""
import hashlib
import json
import math
import os

import numpy as np
import pytest
import torch

from paper_2603_04427_amd import accounting as acc
from synth import (WORKLOADS, make_decode, make_prefill, normal, normal_at, quantize_e4m3, splitmix64,
                   stream_key, with_shape)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- generator

def test_splitmix64_published_vector():
    """SplitMix64 seeded with 1234567: the first outputs of the reference implementation."""
    want = [6457827717110365317, 3203168211198807973, 9817491932198370423,
            4593380528125082431, 16408922859458223821]
    got = [x & ((1 << 64) - 1) for x in splitmix64(1234567, torch.arange(5)).tolist()]
    assert got == want


def test_splitmix64_matches_exact_integer_arithmetic():
    key = stream_key(3, 1)
    idx = torch.tensor([0, 1, 2, 1000, 2 ** 40 + 7, 2 ** 62 - 3])
    got = [x & ((1 << 64) - 1) for x in splitmix64(key, idx).tolist()]
    M = (1 << 64) - 1
    for i, g in zip(idx.tolist(), got):
        z = (key + (i + 1) * 0x9E3779B97F4A7C15) & M
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        assert g == z ^ (z >> 31)


def test_normal_is_slice_and_thread_independent():
    key = stream_key(2, 2)
    n = 100_003
    full = normal(key, n, chunk=1 << 14)
    old = torch.get_num_threads()
    try:
        torch.set_num_threads(1)
        one = normal(key, n, chunk=7777)
    finally:
        torch.set_num_threads(old)
    assert torch.equal(full, one)
    idx = torch.tensor([0, 5, 99_999, 77])
    assert torch.equal(normal_at(key, idx), full[idx])
    # moments of a standard normal
    assert abs(full.mean().item()) < 0.02 and abs(full.std().item() - 1) < 0.02


def test_stored_hashes():
    """First 4096 draws of each workload's Q/K/V streams (written by tests/golden/make_synth_hashes.py)."""
    with open(os.path.join(GOLDEN, "synth_sha256.json")) as f:
        stored = json.load(f)
    for name, spec in WORKLOADS.items():
        for t in range(3):
            x = normal(stream_key(spec.config_id, t), 4096).numpy().tobytes()
            assert hashlib.sha256(x).hexdigest() == stored[f"{name}/{t}"]


def test_workload_layouts():
    s = with_shape(WORKLOADS["longctx_paged_decode"], batch=2, ctx=1024, ctx_lens=(1024, 700))
    d = make_decode(s)
    tb, bs = d["block_table"], s.block_size
    assert sorted(tb.flatten().tolist()) == list(range(8))
    for b in range(2):
        for t in (0, 255, 256, 699, 1023):
            assert torch.equal(d["k"][tb[b, t // bs], 5, t % bs], d["k_logical"][b, 5, t])
            assert torch.equal(d["v"][tb[b, t // bs], 5, t % bs], d["v_logical"][b, 5, t])
    p = make_prefill(with_shape(WORKLOADS["mistral_prefill_s8192"], batch=1, seq_q=32, seq_k=32))
    assert p["q"].shape == (1, 32, 32, 32) and p["v"].shape == (1, 8, 32, 128)
    assert p["q"].dtype == torch.bfloat16
    assert abs(p["k"].float().std().item() - 0.5) < 0.05


# ----------------------------------------------------------------- fp8 quantisation

def test_e4m3_quantisation_round_trip_bound():
    k = normal(stream_key(77, 1), 64 * 1000).view(1000, 64)
    k[3] = 0.0
    codes, sc = quantize_e4m3(k)
    khat = codes.view(torch.float8_e4m3fn).to(torch.float64) * sc.double().unsqueeze(-1)
    err = (khat - k.double()).abs()
    bound = torch.maximum(k.double().abs() * 2.0 ** -4, sc.double().unsqueeze(-1) * 2.0 ** -10)
    assert (err <= bound * (1 + 1e-12)).all()
    # each row's largest magnitude lands exactly on +-448
    mx = codes.view(torch.float8_e4m3fn).to(torch.float64).abs().amax(-1)
    assert (mx[torch.arange(1000) != 3] == 448.0).all()
    assert sc[3].item() == 1.0 and (codes[3] == 0).all()


def test_e4m3_encode_ties_round_to_even():
    """Midpoints between neighbouring E4M3 values round to the even code."""
    vals = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64)
    pos = sorted(set(v for v in vals.tolist() if v >= 0 and math.isfinite(v)))
    for a, b in zip(pos[:-1], pos[1:]):
        mid = torch.tensor([(a + b) / 2], dtype=torch.float32)
        code = mid.to(torch.float8_e4m3fn).view(torch.uint8).item()
        ca = torch.tensor([a], dtype=torch.float32).to(torch.float8_e4m3fn).view(torch.uint8).item()
        cb = torch.tensor([b], dtype=torch.float32).to(torch.float8_e4m3fn).view(torch.uint8).item()
        assert code == (ca if ca % 2 == 0 else cb)


# ----------------------------------------------------------------- paper accounting

def golden():
    with open(os.path.join(GOLDEN, "paper_kv_accounting.json")) as f:
        return json.load(f)


def test_kvcache_per_user_table():
    """Sec. 4.1 per-user table. As printed, its totals and savings are sums and
    differences of the already-rounded components (33.6 + 33.6 = 67.2 while
    2 x 33.55 GB rounds to 67.1; 524 - 328 = 196), so the check rounds the same way."""
    g = golden()["kvcache_per_user"]
    base = {}
    for row in g["rows"]:
        n, ds = row["n"], row["d_select"]
        std = acc.kv_cache_bytes_standard(n, g["d_model"], g["layers"], g["bytes_per"])
        thin = acc.kv_cache_bytes_thin(n, ds, g["d_model"], g["layers"], g["bytes_per"])
        k = n * ds * g["layers"] * g["bytes_per"]
        v = thin - k
        assert v == std / 2                      # values keep full width
        if n == 128000:
            kr, vr = round(k / 1e9, 1), round(v / 1e9, 1)
            assert (kr, vr) == (row["k_gb"], row["v_gb"])
            tot = round(kr + vr, 1)
            assert tot == row["total_gb"]
        else:
            tot = round(thin / 1e9)
            assert tot == row["total_gb"]
        if ds == g["d_model"]:
            assert thin == std
            base[n] = tot
        if "saved_gb" in row:
            assert round(base[n] - tot, 1) == row["saved_gb"]
            assert round(100 * (std - thin) / std, 1) == row["saved_pct"]


def test_kv_7b_analytical_table():
    g = golden()["kv_7b_analytical"]
    gib = 2.0 ** 30
    mha = None
    for row in g["rows"]:
        tot = acc.kv_cache_bytes(g["n"], g["layers"], g["bytes_per"], row["k_width"], row["v_width"])
        if mha is None:
            mha = tot
        assert round(tot / gib, 1) == row["total_gib"]
        if "k_gib" in row:
            assert round(g["n"] * row["k_width"] * g["layers"] * g["bytes_per"] / gib, 1) == row["k_gib"]
        if "saved_pct" in row:
            assert round(100 * (1 - tot / mha), 1) == row["saved_pct"]


def test_decode_bandwidth_model_eq10():
    g = golden()["mistral_decode_model"]
    c = acc.mistral_c_kv(g["n"], g["layers"], g["n_kv"], g["d_head"], g["d_head"], g["beta"])
    c256 = acc.mistral_c_kv(g["n"], g["layers"], g["n_kv"], 32, g["d_head"], g["beta"])
    c512 = acc.mistral_c_kv(g["n"], g["layers"], g["n_kv"], 64, g["d_head"], g["beta"])
    assert round(c / 1e6) == g["c_kv_mb"] and round(c256 / 1e6) == g["c_kv_r256_mb"]
    w, w256 = g["w_gb"] * 1e9, g["w_r256_gb"] * 1e9
    w512 = w - (w - w256) * 2 / 3
    # Nine of the ten printed predictions are Eq. 10 on the stated inputs rounded to two
    # places; r256 at b=8 is printed 1.17 where the stated inputs give 1.164, so every
    # entry is checked to within 0.006.
    for b, p256, p512 in zip(g["batches"], g["predicted_r256"], g["predicted_r512"]):
        assert abs(acc.decode_speedup(w, c, w256, c256, b) - p256) < 0.006
        assert round(acc.decode_speedup(w, c, w512, c512, b), 2) == p512
    assert round(c / c256, 2) == g["asymptote_r256"]


def test_kernel_work_figures():
    c2 = WORKLOADS["mistral_decode_b16"]
    assert acc.decode_bytes(c2.lens, 32, 8, 32, 128) == 16 * 8 * 4096 * 320 + 16 * 32 * 32 * 2 + 16 * 32 * 128 * 2 + 64
    c3 = WORKLOADS["mistral_prefill_s8192"]
    f = acc.prefill_flops(c3.batch, c3.h_q, c3.seq_q, c3.seq_k, c3.r, c3.d_v)
    assert f == 4 * 32 * (8192 * 8193 // 2) * 320
    # backward: five products per visible pair, 3 of width r and 2 of width d_v
    fb = acc.prefill_backward_flops(c3.batch, c3.h_q, c3.seq_q, c3.seq_k, c3.r, c3.d_v)
    assert fb == 4 * 32 * (8192 * 8193 // 2) * 2 * (3 * 32 + 2 * 128)
    assert acc.prefill_backward_flops(1, 1, 3, 3, 4, 8, causal=False) == 9 * 2 * (12 + 16)
    assert acc.causal_pairs(5, 8) == sum(min(8, i + 3 + 1) for i in range(5)) == 4 + 5 + 6 + 7 + 8
    c5 = WORKLOADS["fp8key_decode"]
    assert acc.decode_bytes(c5.lens, 32, 8, 32, 128, "fp8") == 32 * 8 * 32768 * 292 + 32 * 32 * 32 * 2 + 32 * 32 * 256 + 128
    # 4-bit keys: 16 bytes of codes and a 4-byte scale per key row
    assert acc.decode_bytes(c5.lens, 32, 8, 32, 128, "int4") == 32 * 8 * 32768 * 276 + 32 * 32 * 32 * 2 + 32 * 32 * 256 + 128
