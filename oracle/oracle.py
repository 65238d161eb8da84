"""Python access to the fp64 C oracle (``tk_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
CPU-baseline leg of the benchmark, never by the GPU library. It shares no code
with the GPU path; inputs are passed exactly as the GPU receives them (fp32,
bf16 bit patterns, E4M3 or packed 4-bit integer codes with fp32 scales) and
widened inside the oracle.

Each call is the plain definition of thin-key attention (Sec. 2.1, Eq. 4): see
the header of ``tk_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tk_oracle.c")
_LIB = os.path.join(_HERE, "libtkoracle.so")

F64, F32, BF16, E4M3, INT4 = 0, 1, 2, 3, 4
_lib = None


class Int4:
    """Marks a uint8 tensor [..., r / 2] as packed 4-bit key codes (excess-8, low
    nibble first); the key entry is (nibble - 8) * its row's scale."""

    def __init__(self, packed: torch.Tensor):
        self.packed = packed

    @property
    def shape(self):  # shape in key entries
        return (*self.packed.shape[:-1], self.packed.shape[-1] * 2)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP). Returns the library path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("TKO_ORACLE_LIB")  # an alternate build (the mutation tests use it)
        if path is None:
            path = _LIB
            if not os.path.exists(path):
                build()
        L = ctypes.CDLL(path)
        vp, i, l, d = ctypes.c_void_p, ctypes.c_int, ctypes.c_long, ctypes.c_double
        L.tko_prefill.argtypes = [vp, i, vp, i, vp, vp, i, vp, l, l, l, l, l, l, l, i, d, i]
        L.tko_prefill.restype = i
        L.tko_decode.argtypes = [vp, i, vp, i, vp, vp, i, vp, l, l, l, vp, l, l, l, d, vp, l, l, i]
        L.tko_decode.restype = i
        L.tko_e4m3_value.argtypes = [ctypes.c_uint8]
        L.tko_e4m3_value.restype = d
        L.tko_int4_value.argtypes = [vp, ctypes.c_size_t]
        L.tko_int4_value.restype = d
        L.tko_max_threads.restype = i
        L.tko_prefill_backward.argtypes = [vp, i, vp, i, vp, i, vp, i, vp, i, vp, vp, vp, vp,
                                           l, l, l, l, l, l, l, i, d, l, i]
        L.tko_prefill_backward.restype = i
        _lib = L
    return _lib


def _typed(x):
    """(pointer, dtype code, keep-alive tensor) for a CPU tensor."""
    if isinstance(x, Int4):
        p = x.packed.detach().cpu().contiguous().view(torch.uint8)
        return ctypes.c_void_p(p.data_ptr()), INT4, p
    x = x.detach().cpu().contiguous()
    if x.dtype == torch.float64:
        code = F64
    elif x.dtype == torch.float32:
        code = F32
    elif x.dtype == torch.bfloat16:
        code = BF16
    elif x.dtype in (torch.uint8, torch.float8_e4m3fn):
        x = x.view(torch.uint8)
        code = E4M3
    else:
        raise TypeError(f"oracle: unsupported dtype {x.dtype}")
    return ctypes.c_void_p(x.data_ptr()), code, x


def e4m3_value(code: int) -> float:
    """The oracle's decode of one OCP E4M3FN code."""
    return lib().tko_e4m3_value(code)


def int4_value(packed_row: torch.Tensor, i: int) -> float:
    """The oracle's decode of entry i of a packed 4-bit code row."""
    p = packed_row.detach().cpu().contiguous().view(torch.uint8)
    return lib().tko_int4_value(ctypes.c_void_p(p.data_ptr()), i)


def max_threads() -> int:
    return lib().tko_max_threads()


def prefill(q, k, v, causal=True, scale=None, k_scale=None, threads=0) -> torch.Tensor:
    """O [B,Hq,Sq,dv] fp64 for Q [B,Hq,Sq,r], K [B,Hkv,Sk,r], V [B,Hkv,Sk,dv]."""
    B, Hq, Sq, r = q.shape
    _, Hkv, Sk, _ = k.shape
    dv = v.shape[-1]
    if scale is None:
        scale = r ** -0.5
    pq, cq, q_ = _typed(q)
    pk, ck, k_ = _typed(k)
    pv, cv, v_ = _typed(v)
    ks = None if k_scale is None else k_scale.detach().cpu().to(torch.float32).contiguous()
    o = torch.empty(B, Hq, Sq, dv, dtype=torch.float64)
    rc = lib().tko_prefill(pq, cq, pk, ck, None if ks is None else ctypes.c_void_p(ks.data_ptr()),
                           pv, cv, ctypes.c_void_p(o.data_ptr()),
                           B, Hq, Hkv, Sq, Sk, r, dv, int(bool(causal)), float(scale), int(threads))
    if rc != 0:
        raise ValueError("oracle prefill: invalid shapes")
    return o


def decode(q, k, v, ctx_lens, scale=None, k_scale=None, block_table=None, block_size=0,
           threads=0) -> torch.Tensor:
    """O [B,Hq,dv] fp64 for one query token per sequence against a (paged) cache."""
    B, Hq, r = q.shape
    dv = v.shape[-1]
    Hkv = k.shape[1]
    if scale is None:
        scale = r ** -0.5
    lens = ctx_lens.detach().cpu().to(torch.int32).contiguous()
    pq, cq, q_ = _typed(q)
    pk, ck, k_ = _typed(k)
    pv, cv, v_ = _typed(v)
    ks = None if k_scale is None else k_scale.detach().cpu().to(torch.float32).contiguous()
    if block_table is None:
        max_ctx, tb, mb = k.shape[2], None, 0
    else:
        tb = block_table.detach().cpu().to(torch.int32).contiguous()
        mb = tb.shape[1]
        max_ctx = mb * block_size
    o = torch.empty(B, Hq, dv, dtype=torch.float64)
    rc = lib().tko_decode(pq, cq, pk, ck, None if ks is None else ctypes.c_void_p(ks.data_ptr()),
                          pv, cv, ctypes.c_void_p(o.data_ptr()), B, Hq, Hkv,
                          ctypes.c_void_p(lens.data_ptr()), max_ctx, r, dv, float(scale),
                          None if tb is None else ctypes.c_void_p(tb.data_ptr()),
                          int(block_size), int(mb), int(threads))
    if rc != 0:
        raise ValueError("oracle decode: invalid shapes or lengths")
    return o


def prefill_backward(q, k, v, do, causal=True, scale=None, row_lo=0, threads=0, o=None):
    """Gradients (dQ [B,Hq,Sq,r], dK [B,Hkv,Sk,r], dV [B,Hkv,Sk,dv]) of the prefill
    attention for the output gradient dO [B,Hq,Sq,dv], and the forward's
    log-sum-exp [B,Hq,Sq] (natural log), all fp64; see ``tko_prefill_backward``.
    ``o`` (optional, [B,Hq,Sq,dv]): a stored forward output whose rowsum(dO * O)
    is used as D (by default D is the exact sum of P * dP).
    Only query rows >= row_lo are processed (dQ and lse of lower rows are NaN, and
    dK, dV hold those rows' contributions: for a causal mask the full gradient of
    keys >= row_lo + Sk - Sq)."""
    B, Hq, Sq, r = q.shape
    _, Hkv, Sk, _ = k.shape
    dv = v.shape[-1]
    if scale is None:
        scale = r ** -0.5
    pq, cq, q_ = _typed(q)
    pk, ck, k_ = _typed(k)
    pv, cv, v_ = _typed(v)
    pd, cd, d_ = _typed(do)
    po, co, o_ = (None, 0, None) if o is None else _typed(o)
    dq = torch.full((B, Hq, Sq, r), float("nan"), dtype=torch.float64)
    dk = torch.empty(B, Hkv, Sk, r, dtype=torch.float64)
    dvv = torch.empty(B, Hkv, Sk, dv, dtype=torch.float64)
    lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float64)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    rc = lib().tko_prefill_backward(pq, cq, pk, ck, pv, cv, pd, cd, po, co, ptr(dq), ptr(dk), ptr(dvv), ptr(lse),
                                    B, Hq, Hkv, Sq, Sk, r, dv, int(bool(causal)), float(scale), int(row_lo),
                                    int(threads))
    if rc != 0:
        raise ValueError("oracle prefill_backward: invalid shapes")
    return dq, dk, dvv, lse
