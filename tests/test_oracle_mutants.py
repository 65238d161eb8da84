"""The oracle's pins are sharp: each plausible slip planted in a copy of the C
oracle (built on the CPU) makes the pin suite fail.

Every mutant below is compiled from tk_oracle.c with one textual change, then
tests/test_oracle_pins.py runs against it in a subprocess and must fail."""
import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "tk_oracle.c")

MUTANTS = {
    "causal_off_by_one": ("long n_keys = causal ? i + (Sk - Sq) + 1 : Sk;",
                          "long n_keys = causal ? i + (Sk - Sq) : Sk;"),
    "causal_top_left": ("long n_keys = causal ? i + (Sk - Sq) + 1 : Sk;",
                        "long n_keys = causal ? i + 1 : Sk;"),
    "gqa_modulo_map": ("long h = idx % Hq, b = idx / Hq, g = h / G;",
                       "long h = idx % Hq, b = idx / Hq, g = h % Hkv;"),
    "gqa_modulo_map_prefill": ("            long g = h / G;", "            long g = h % Hkv;"),
    "scale_dropped": ("s[j] = scale * acc;", "s[j] = acc;"),
    "normaliser_dropped": ("double w = s[j] / l;", "double w = s[j];"),
    "value_columns_reversed": ("(size_t)row * dv + c)", "(size_t)row * dv + (dv - 1 - c))"),
    "key_dims_shifted": ("(size_t)row * r + c)", "(size_t)row * r + (c + 1) % r)"),
    "page_slot_wrong": ("rows[t] = (blk * Hkv + g) * block_size + t % block_size;",
                        "rows[t] = (blk * Hkv + g) * block_size + (t + 1) % block_size;"),
    "contiguous_layout_transposed": ("rows[t] = (b * Hkv + g) * max_ctx + t;",
                                     "rows[t] = (g * B + b) * max_ctx + t;"),
    "key_scale_ignored": ("double ks = kv->k_scale ? (double)kv->k_scale[row] : 1.0;", "double ks = 1.0;"),
    "e4m3_bias": ("mag = ldexp(1.0 + (double)m / 8.0, e - 7);", "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    "e4m3_subnormal": ("mag = ldexp((double)m / 8.0, -6);", "mag = ldexp((double)m / 8.0, -7);"),
    "max_not_subtracted_uses_first": ("m = s[j] > m ? s[j] : m;", "m = s[0];"),
    "int4_nibble_order": ("const int n = (i & 1) ? (byte >> 4) : (byte & 15);",
                          "const int n = (i & 1) ? (byte & 15) : (byte >> 4);"),
    "int4_excess": ("return (double)(n - 8);", "return (double)(n - 7);"),
    "bf16_widening": ("uint32_t w = (uint32_t)bits << 16;", "uint32_t w = ((uint32_t)bits << 16) | 0x8000u;"),
}

# slips in the backward, each caught by tests/test_oracle_backward.py
BACKWARD_MUTANTS = {
    "bwd_dq_D_dropped": ("const double ds = s[j] * (dp[j] - D);", "const double ds = s[j] * dp[j];"),
    "bwd_dk_D_dropped": ("const double ds = p * (dpv - Dr[idx]);", "const double ds = p * dpv;"),
    "bwd_dq_scale_dropped": ("dQ[(size_t)idx * r + c] += scale * ds *", "dQ[(size_t)idx * r + c] += ds *"),
    "bwd_dk_uses_key": ("dk[c] += scale * ds * ld(Q, q_dt, idx * r + c);",
                        "dk[c] += scale * ds * ld(K, k_dt, (size_t)kidx * r + c);"),
    "bwd_dv_unnormalised": ("const double p = exp(scale * acc - lse[idx]);", "const double p = exp(scale * acc);"),
    "bwd_causal_rows": ("long i0 = causal ? j - off : 0;", "long i0 = causal ? j - off + 1 : 0;"),
    "bwd_gqa_one_head": ("for (long h = g * G; h < (g + 1) * G; h++) {",
                         "for (long h = g * G; h < g * G + 1; h++) {"),
    "bwd_lse_max_only": ("const double ls = m + log(l);", "const double ls = m;"),
    "bwd_score_scale_dropped": ("s[j] = acc * scale;", "s[j] = acc;"),
    "bwd_dv_value_row": ("dvv[c] += p * ld(dO, do_dt, idx * dv + c);",
                         "dvv[c] += p * ld(V, v_dt, (size_t)kidx * dv + c);"),
    "bwd_stored_o_ignored": ("            if (O) {\n                D = 0.0;", "            if (0) {\n                D = 0.0;"),
}
PIN_FILES = {**{n: "test_oracle_pins.py" for n in MUTANTS}, **{n: "test_oracle_backward.py" for n in BACKWARD_MUTANTS}}
ALL_MUTANTS = {**MUTANTS, **BACKWARD_MUTANTS}


def run_mutant(name, tmp):
    old, new = ALL_MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = os.path.join(tmp, f"{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = os.path.join(tmp, f"lib_{name}.so")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", lib, path, "-lm"])
    env = dict(os.environ, TKO_ORACLE_LIB=lib, OMP_NUM_THREADS="1")
    p = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", PIN_FILES[name])],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    return name, p.returncode


def test_every_mutant_is_caught():
    with tempfile.TemporaryDirectory() as tmp:
        with cf.ThreadPoolExecutor(max_workers=6) as ex:
            results = list(ex.map(lambda n: run_mutant(n, tmp), ALL_MUTANTS))
    survivors = [n for n, rc in results if rc == 0]
    errors = [(n, rc) for n, rc in results if rc not in (0, 1)]
    assert not errors, errors
    assert not survivors, f"pins did not catch: {survivors}"
