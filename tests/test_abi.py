"""The C ABI without a GPU: the library loads, exports what include/tk_attn.h
declares, and rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2603_04427_amd import binding as tb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tk_attn.h")

P = ctypes.c_void_p(0x10000)       # aligned, never dereferenced on these paths
P_ODD = ctypes.c_void_p(0x10008)   # 8-byte aligned only


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tk_[a-z0-9_]+)\s*\(", text)))


def test_exports_match_header():
    names = declared_functions()
    assert names == sorted(tb.SIGNATURES), names
    lib = tb.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    assert tb.tk_status_str(0) == "ok"
    assert tb.tk_status_str(tb.TK_ERR_WORKSPACE).startswith("workspace")
    assert tb.tk_status_str(99) == "unknown status"
    assert tb.tk_version() >= 100


def prefill(**kw):
    a = dict(Q=P, K=P, V=P, O=P, batch=1, H_q=4, H_kv=2, seq_q=8, seq_k=8, r=32, d_v=128, causal=1,
             scale=0.0, dtype=tb.TK_BF16, stream=None)
    a.update(kw)
    return tb.lib().tk_attn_prefill(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(H_q=3, H_kv=2), tb.TK_ERR_INVALID_ARG),
    (dict(H_kv=0), tb.TK_ERR_INVALID_ARG),
    (dict(batch=-1), tb.TK_ERR_INVALID_ARG),
    (dict(seq_q=9, seq_k=8), tb.TK_ERR_INVALID_ARG),           # causal needs Sq <= Sk
    (dict(seq_k=0, causal=0), tb.TK_ERR_INVALID_ARG),
    (dict(Q=None), tb.TK_ERR_INVALID_ARG),
    (dict(O=P_ODD), tb.TK_ERR_INVALID_ARG),
    (dict(r=24), tb.TK_ERR_UNSUPPORTED),
    (dict(d_v=96), tb.TK_ERR_UNSUPPORTED),
    (dict(dtype=tb.TK_FP8_E4M3), tb.TK_ERR_UNSUPPORTED),
    (dict(dtype=7), tb.TK_ERR_INVALID_ARG),
    (dict(batch=0), tb.TK_OK),                                 # nothing to do, no launch
    (dict(seq_q=0), tb.TK_OK),
])
def test_prefill_validation(kw, status):
    assert prefill(**kw) == status


def prefill_lse(**kw):
    a = dict(Q=P, K=P, V=P, O=P, lse=P, batch=1, H_q=4, H_kv=2, seq_q=8, seq_k=8, r=32, d_v=128, causal=1,
             scale=0.0, stream=None)
    a.update(kw)
    return tb.lib().tk_attn_prefill_lse(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(lse=None), tb.TK_ERR_INVALID_ARG),
    (dict(lse=ctypes.c_void_p(0x10002)), tb.TK_ERR_INVALID_ARG),   # not 4-byte aligned
    (dict(H_q=3), tb.TK_ERR_INVALID_ARG),
    (dict(seq_q=9), tb.TK_ERR_INVALID_ARG),
    (dict(r=24), tb.TK_ERR_UNSUPPORTED),
    (dict(seq_q=0, lse=None), tb.TK_OK),
])
def test_prefill_lse_validation(kw, status):
    assert prefill_lse(**kw) == status


def backward(**kw):
    a = dict(Q=P, K=P, V=P, O=P, dO=P, lse=P, dQ=P, dK=P, dV=P, batch=1, H_q=4, H_kv=2, seq_q=8, seq_k=8,
             r=32, d_v=128, causal=1, scale=0.0, ws=P, ws_bytes=1 << 20, stream=None)
    a.update(kw)
    return tb.lib().tk_attn_prefill_backward(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(H_q=3), tb.TK_ERR_INVALID_ARG),
    (dict(seq_q=9), tb.TK_ERR_INVALID_ARG),                    # causal needs Sq <= Sk
    (dict(seq_k=0, causal=0), tb.TK_ERR_INVALID_ARG),
    (dict(dO=None), tb.TK_ERR_INVALID_ARG),
    (dict(lse=None), tb.TK_ERR_INVALID_ARG),
    (dict(dK=P_ODD), tb.TK_ERR_INVALID_ARG),
    (dict(lse=ctypes.c_void_p(0x10002)), tb.TK_ERR_INVALID_ARG),
    (dict(ws=None), tb.TK_ERR_WORKSPACE),
    (dict(ws_bytes=16), tb.TK_ERR_WORKSPACE),
    (dict(r=16), tb.TK_ERR_UNSUPPORTED),
    (dict(d_v=96), tb.TK_ERR_UNSUPPORTED),
    (dict(batch=0), tb.TK_OK),
    (dict(seq_q=0, seq_k=0, Q=None, O=None, dO=None, lse=None, dQ=None), tb.TK_OK),
])
def test_backward_validation(kw, status):
    assert backward(**kw) == status


def test_backward_workspace_query():
    ws = tb.tk_attn_prefill_backward_workspace_bytes
    assert ws(4, 32, 8192) == 4 * 32 * 8192 * 8
    assert ws(1, 3, 5) == 256
    assert ws(0, 4, 10) == 256 and ws(1, 4, 0) == 256
    assert ws(-1, 4, 10) == 0 and ws(1, 0, 10) == 0


def decode(**kw):
    a = dict(Q=P, K=P, V=P, O=P, batch=2, H_q=32, H_kv=8, ctx_lens=P, max_ctx=4096, r=32, d_v=128,
             scale=0.0, k_dtype=tb.TK_BF16, k_scale=None, block_table=None, block_size=0,
             max_blocks=0, num_blocks=0, ws=P, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return tb.lib().tk_attn_decode(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(H_q=30), tb.TK_ERR_INVALID_ARG),
    (dict(max_ctx=-1), tb.TK_ERR_INVALID_ARG),
    (dict(k_dtype=tb.TK_FP8_E4M3), tb.TK_ERR_INVALID_ARG),     # fp8 without scales
    (dict(k_scale=P), tb.TK_ERR_INVALID_ARG),                  # scales without fp8
    (dict(k_dtype=tb.TK_INT4), tb.TK_ERR_INVALID_ARG),         # 4-bit keys without scales
    (dict(k_dtype=tb.TK_F32), tb.TK_ERR_UNSUPPORTED),
    (dict(block_size=256), tb.TK_ERR_INVALID_ARG),             # layout args without a table
    (dict(block_table=P, block_size=0, max_blocks=16, num_blocks=32), tb.TK_ERR_INVALID_ARG),
    (dict(block_table=P, block_size=256, max_blocks=8, num_blocks=32), tb.TK_ERR_INVALID_ARG),  # 2048 < ctx
    (dict(block_table=P, block_size=32, max_blocks=128, num_blocks=256), tb.TK_ERR_UNSUPPORTED),
    (dict(block_table=P, block_size=96, max_blocks=64, num_blocks=256), tb.TK_ERR_UNSUPPORTED),
    (dict(ctx_lens=None), tb.TK_ERR_INVALID_ARG),
    (dict(V=P_ODD), tb.TK_ERR_INVALID_ARG),
    (dict(r=48), tb.TK_ERR_UNSUPPORTED),
    (dict(d_v=256), tb.TK_ERR_UNSUPPORTED),
    (dict(ws=None), tb.TK_ERR_WORKSPACE),
    (dict(ws_bytes=16), tb.TK_ERR_WORKSPACE),
    (dict(ws=ctypes.c_void_p(0x10010)), tb.TK_ERR_WORKSPACE),  # not 256-byte aligned
    (dict(batch=0), tb.TK_OK),
])
def test_decode_validation(kw, status):
    assert decode(**kw) == status


def decode_noalloc(**kw):
    a = dict(Q=P, K=P, V=P, O=P, batch=2, H_q=32, H_kv=8, ctx_lens=P, max_ctx=4096, r=32, d_v=128,
             scale=0.0, k_dtype=tb.TK_BF16, k_scale=None, block_table=None, block_size=0,
             max_blocks=0, num_blocks=0, stream=None)
    a.update(kw)
    return tb.lib().tk_attn_decode_noalloc(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(H_q=30), tb.TK_ERR_INVALID_ARG),
    (dict(max_ctx=-1), tb.TK_ERR_INVALID_ARG),
    (dict(k_dtype=tb.TK_FP8_E4M3), tb.TK_ERR_INVALID_ARG),     # fp8 without scales
    (dict(k_scale=P), tb.TK_ERR_INVALID_ARG),                  # scales without fp8
    (dict(k_dtype=tb.TK_F32), tb.TK_ERR_UNSUPPORTED),
    (dict(block_size=256), tb.TK_ERR_INVALID_ARG),             # layout args without a table
    (dict(block_table=P, block_size=256, max_blocks=8, num_blocks=32), tb.TK_ERR_INVALID_ARG),  # 2048 < ctx
    (dict(block_table=P, block_size=96, max_blocks=64, num_blocks=256), tb.TK_ERR_UNSUPPORTED),
    (dict(ctx_lens=None), tb.TK_ERR_INVALID_ARG),
    (dict(O=P_ODD), tb.TK_ERR_INVALID_ARG),
    (dict(r=48), tb.TK_ERR_UNSUPPORTED),
    (dict(batch=0), tb.TK_OK),
])
def test_decode_noalloc_validation(kw, status):
    """The no-allocation decode rejects what tk_attn_decode rejects, on the host,
    before it looks up its scratch (the first HIP call of that path)."""
    assert decode_noalloc(**kw) == status


def project(**kw):
    a = dict(X=P, Wt=P, Y=P, batch=2, seq=128, d_model=1024, n_heads=8, width=32, stream=None)
    a.update(kw)
    return tb.lib().tk_project_heads(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), tb.TK_ERR_INVALID_ARG),
    (dict(d_model=0), tb.TK_ERR_INVALID_ARG),
    (dict(n_heads=0), tb.TK_ERR_INVALID_ARG),
    (dict(width=0), tb.TK_ERR_INVALID_ARG),
    (dict(X=None), tb.TK_ERR_INVALID_ARG),
    (dict(Y=P_ODD), tb.TK_ERR_INVALID_ARG),
    (dict(d_model=1000), tb.TK_ERR_UNSUPPORTED),     # not a multiple of 32
    (dict(width=30), tb.TK_ERR_UNSUPPORTED),         # not a multiple of 4
    (dict(d_model=1 << 23), tb.TK_ERR_UNSUPPORTED),  # copy offsets would not fit 32 bits
    (dict(batch=0), tb.TK_OK),
    (dict(seq=0), tb.TK_OK),
])
def test_project_validation(kw, status):
    assert project(**kw) == status


def test_workspace_query_is_pure_and_sized():
    ws = tb.tk_attn_decode_workspace_bytes
    a = ws(16, 32, 8, 4096, 128)
    assert a == ws(16, 32, 8, 4096, 128) > 0
    # a fixed leading region of 512 arrival counters (4 B) for every shape, then
    # [B, Hq, n_split, d_v + 2] fp32 partials
    counters = 2048
    assert (a - counters) % (16 * 32 * 130 * 4) == 0
    assert ws(16, 30, 8, 4096, 128) == 0 and ws(0, 32, 8, 4096, 128) == 0
    assert ws(8, 32, 8, 131072, 128) >= 8 * 32 * 130 * 4
    assert ws(1, 32, 8, 0, 128) == counters + 32 * 130 * 4      # empty caches: one split
    assert ws(200, 64, 8, 64, 64) == counters + 200 * 64 * 66 * 4  # many pairs: one split


def append(**kw):
    a = dict(K_new=P, V_new=P, batch=2, H_kv=8, n_new=1, r=32, d_v=128, positions=P, K=P, V=P, max_ctx=4096,
             k_dtype=tb.TK_BF16, k_scale=None, block_table=None, block_size=0, max_blocks=0, num_blocks=0,
             stream=None)
    a.update(kw)
    return tb.lib().tk_cache_append(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(n_new=-1), tb.TK_ERR_INVALID_ARG),
    (dict(H_kv=0), tb.TK_ERR_INVALID_ARG),
    (dict(max_ctx=-1), tb.TK_ERR_INVALID_ARG),
    (dict(k_dtype=tb.TK_FP8_E4M3), tb.TK_ERR_INVALID_ARG),     # fp8 without scales
    (dict(k_scale=P), tb.TK_ERR_INVALID_ARG),                  # scales without fp8
    (dict(k_dtype=tb.TK_INT4), tb.TK_ERR_INVALID_ARG),         # 4-bit keys without scales
    (dict(k_dtype=tb.TK_F32), tb.TK_ERR_UNSUPPORTED),
    (dict(block_size=64), tb.TK_ERR_INVALID_ARG),              # layout args without a table
    (dict(block_table=P, block_size=0, max_blocks=4, num_blocks=8), tb.TK_ERR_INVALID_ARG),
    (dict(block_table=P, block_size=48, max_blocks=4, num_blocks=8), tb.TK_ERR_UNSUPPORTED),
    (dict(positions=None), tb.TK_ERR_INVALID_ARG),
    (dict(V_new=P_ODD), tb.TK_ERR_INVALID_ARG),
    (dict(r=24), tb.TK_ERR_UNSUPPORTED),
    (dict(d_v=32), tb.TK_ERR_UNSUPPORTED),
    (dict(batch=4096, H_kv=32), tb.TK_ERR_UNSUPPORTED),        # more than 65535 (sequence, head) pairs
    (dict(batch=0), tb.TK_OK),                                 # nothing to do, no launch
    (dict(n_new=0), tb.TK_OK),
])
def test_append_validation(kw, status):
    assert append(**kw) == status


def test_stream_probe_library_loads_and_rejects_bad_arguments():
    """The benchmark's streaming-read probe (a separate library, not the attention
    ABI) loads and rejects bad arguments before any HIP call."""
    path = os.path.join(ROOT, "paper_2603_04427_amd", "libtkprobe.so")
    if not os.path.exists(path):
        pytest.skip("probe library not built")
    lib = ctypes.CDLL(path)
    lib.tkprobe_threads.restype = ctypes.c_int
    assert lib.tkprobe_threads() == 512
    f = lib.tkprobe_stream_read
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    assert f(None, 4096, P, 256, 0, None) == 1        # no buffer
    assert f(P, 4096, None, 256, 0, None) == 1        # no sink
    assert f(P, 4100, P, 256, 0, None) == 1           # not a multiple of 16 bytes
    assert f(P_ODD, 4096, P, 256, 0, None) == 1       # misaligned
    assert f(P, 4096, P, 0, 1, None) == 1             # empty grid
    assert f(P, 0, P, 256, 1, None) == 1              # nothing to read
