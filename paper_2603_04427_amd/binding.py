"""ctypes binding of libtkattn.so, with the C entry points' names.

Argument marshalling only: shapes are read from the tensors, checked for
consistency, and passed with the tensors' device pointers and torch's current
HIP stream to the C ABI declared in include/tk_attn.h. Every step of the
computation runs in the HIP kernels; there is no other code path. If the
library has not been built, the first call raises instead of falling back.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtkattn.so")

TK_OK, TK_ERR_INVALID_ARG, TK_ERR_UNSUPPORTED, TK_ERR_WORKSPACE, TK_ERR_HIP = 0, 1, 2, 3, 4
TK_F32, TK_BF16, TK_FP8_E4M3, TK_INT4 = 0, 1, 2, 3

# exported functions and their ctypes signatures (kept in step with include/tk_attn.h)
_vp, _i, _f, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
SIGNATURES = {
    "tk_attn_prefill": ([_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _f, _i, _vp], _i),
    "tk_attn_prefill_lse": ([_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _f, _vp], _i),
    "tk_attn_prefill_backward_workspace_bytes": ([_i, _i, _i], _sz),
    "tk_attn_prefill_backward": ([_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _f,
                                  _vp, _sz, _vp], _i),
    "tk_attn_decode_workspace_bytes": ([_i, _i, _i, _i, _i], _sz),
    "tk_attn_decode": ([_vp, _vp, _vp, _vp, _i, _i, _i, _vp, _i, _i, _i, _f, _i, _vp, _vp, _i, _i, _i,
                        _vp, _sz, _vp], _i),
    "tk_attn_decode_noalloc": ([_vp, _vp, _vp, _vp, _i, _i, _i, _vp, _i, _i, _i, _f, _i, _vp, _vp, _i, _i, _i,
                                _vp], _i),
    "tk_cache_append": ([_vp, _vp, _i, _i, _i, _i, _i, _vp, _vp, _vp, _i, _i, _vp, _vp, _i, _i, _i, _vp], _i),
    "tk_project_heads": ([_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp], _i),
    "tk_status_str": ([_i], ctypes.c_char_p),
    "tk_version": ([], _i),
}

_lib = None


class TkError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {tk_status_str(status)} (status {status})")


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"libtkattn.so not found at {_LIB_PATH}; build it with "
                               "`python -m paper_2603_04427_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def tk_status_str(status: int) -> str:
    return lib().tk_status_str(int(status)).decode()


def tk_version() -> int:
    return lib().tk_version()


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(t: torch.Tensor, name: str, dtypes, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class PreparedCall:
    """A C entry point with its arguments marshalled once; calling it launches again
    with the same tensors (for timing loops and graph-free replay)."""

    def __init__(self, name: str, args, keep, result=None):
        self.name = name
        self.fn = getattr(lib(), name)
        self.args = args
        self.keep = keep  # tensors whose memory the pointers refer to
        self.result = keep[-1] if result is None else result

    def __call__(self):
        st = self.fn(*self.args)
        if st != TK_OK:
            raise TkError(st, self.name)
        return self.result


def prepare_prefill(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, O: Optional[torch.Tensor] = None,
                    causal: bool = True, scale: float = 0.0, stream=None) -> PreparedCall:
    dts = (torch.bfloat16, torch.float32)
    _check(Q, "Q", dts, 4)
    _check(K, "K", (Q.dtype,), 4)
    _check(V, "V", (Q.dtype,), 4)
    B, Hq, Sq, r = Q.shape
    _, Hkv, Sk, dv = V.shape
    if K.shape != (B, Hkv, Sk, r) or V.shape[0] != B:
        raise ValueError(f"shape mismatch Q{tuple(Q.shape)} K{tuple(K.shape)} V{tuple(V.shape)}")
    if O is None:
        O = torch.empty(B, Hq, Sq, dv, dtype=Q.dtype, device=Q.device)
    _check(O, "O", (Q.dtype,), 4)
    if O.shape != (B, Hq, Sq, dv):
        raise ValueError("O has the wrong shape")
    args = (_ptr(Q), _ptr(K), _ptr(V), _ptr(O), B, Hq, Hkv, Sq, Sk, r, dv, int(bool(causal)), float(scale),
            TK_BF16 if Q.dtype == torch.bfloat16 else TK_F32, _stream(stream))
    return PreparedCall("tk_attn_prefill", args, (Q, K, V, O))


def tk_attn_prefill(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, O: Optional[torch.Tensor] = None,
                    causal: bool = True, scale: float = 0.0, stream=None) -> torch.Tensor:
    """O = softmax(scale Q K^T [causal]) V for Q [B,Hq,Sq,r], K [B,Hkv,Sk,r], V [B,Hkv,Sk,dv]."""
    return prepare_prefill(Q, K, V, O, causal, scale, stream)()


def _prefill_shapes(Q, K, V):
    B, Hq, Sq, r = Q.shape
    _, Hkv, Sk, dv = V.shape
    if K.shape != (B, Hkv, Sk, r) or V.shape[0] != B:
        raise ValueError(f"shape mismatch Q{tuple(Q.shape)} K{tuple(K.shape)} V{tuple(V.shape)}")
    return B, Hq, Hkv, Sq, Sk, r, dv


def prepare_prefill_lse(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, O: Optional[torch.Tensor] = None,
                        lse: Optional[torch.Tensor] = None, causal: bool = True, scale: float = 0.0,
                        stream=None) -> PreparedCall:
    bf = (torch.bfloat16,)
    for t, n in ((Q, "Q"), (K, "K"), (V, "V")):
        _check(t, n, bf, 4)
    B, Hq, Hkv, Sq, Sk, r, dv = _prefill_shapes(Q, K, V)
    if O is None:
        O = torch.empty(B, Hq, Sq, dv, dtype=torch.bfloat16, device=Q.device)
    if lse is None:
        lse = torch.empty(B, Hq, Sq, dtype=torch.float32, device=Q.device)
    _check(O, "O", bf, 4)
    _check(lse, "lse", (torch.float32,), 3)
    if O.shape != (B, Hq, Sq, dv) or lse.shape != (B, Hq, Sq):
        raise ValueError("O or lse has the wrong shape")
    args = (_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(lse), B, Hq, Hkv, Sq, Sk, r, dv, int(bool(causal)),
            float(scale), _stream(stream))
    return PreparedCall("tk_attn_prefill_lse", args, (Q, K, V, O, lse), result=(O, lse))


def tk_attn_prefill_lse(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, O: Optional[torch.Tensor] = None,
                        lse: Optional[torch.Tensor] = None, causal: bool = True, scale: float = 0.0,
                        stream=None):
    """bf16 prefill that also returns each row's log-sum-exp (fp32 [B, Hq, Sq]): (O, lse)."""
    return prepare_prefill_lse(Q, K, V, O, lse, causal, scale, stream)()


def tk_attn_prefill_backward_workspace_bytes(batch: int, H_q: int, seq_q: int) -> int:
    return int(lib().tk_attn_prefill_backward_workspace_bytes(batch, H_q, seq_q))


def prepare_prefill_backward(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, O: torch.Tensor,
                             dO: torch.Tensor, lse: torch.Tensor, causal: bool = True, scale: float = 0.0,
                             dQ: Optional[torch.Tensor] = None, dK: Optional[torch.Tensor] = None,
                             dV: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                             stream=None) -> PreparedCall:
    bf = (torch.bfloat16,)
    for t, n in ((Q, "Q"), (K, "K"), (V, "V"), (O, "O"), (dO, "dO")):
        _check(t, n, bf, 4)
    _check(lse, "lse", (torch.float32,), 3)
    B, Hq, Hkv, Sq, Sk, r, dv = _prefill_shapes(Q, K, V)
    if O.shape != (B, Hq, Sq, dv) or dO.shape != O.shape or lse.shape != (B, Hq, Sq):
        raise ValueError("O, dO or lse has the wrong shape")
    dQ = torch.empty_like(Q) if dQ is None else dQ
    dK = torch.empty_like(K) if dK is None else dK
    dV = torch.empty_like(V) if dV is None else dV
    for t, n, ref in ((dQ, "dQ", Q), (dK, "dK", K), (dV, "dV", V)):
        _check(t, n, bf, 4)
        if t.shape != ref.shape:
            raise ValueError(f"{n} has the wrong shape")
    if workspace is None:
        workspace = torch.empty(tk_attn_prefill_backward_workspace_bytes(B, Hq, Sq), dtype=torch.uint8,
                                device=Q.device)
    args = (_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(lse), _ptr(dQ), _ptr(dK), _ptr(dV),
            B, Hq, Hkv, Sq, Sk, r, dv, int(bool(causal)), float(scale), _ptr(workspace),
            workspace.numel() * workspace.element_size(), _stream(stream))
    return PreparedCall("tk_attn_prefill_backward", args, (Q, K, V, O, dO, lse, dQ, dK, dV, workspace),
                        result=(dQ, dK, dV))


def tk_attn_prefill_backward(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, O: torch.Tensor,
                             dO: torch.Tensor, lse: torch.Tensor, causal: bool = True, scale: float = 0.0,
                             dQ: Optional[torch.Tensor] = None, dK: Optional[torch.Tensor] = None,
                             dV: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                             stream=None):
    """Gradients (dQ, dK, dV) of the bf16 prefill given O, dO and the forward's lse."""
    return prepare_prefill_backward(Q, K, V, O, dO, lse, causal, scale, dQ, dK, dV, workspace, stream)()


def tk_attn_decode_workspace_bytes(batch: int, H_q: int, H_kv: int, max_ctx: int, d_v: int) -> int:
    return int(lib().tk_attn_decode_workspace_bytes(batch, H_q, H_kv, max_ctx, d_v))


def _key_format(K_cache: torch.Tensor, r: int) -> int:
    """bf16 rows, E4M3 codes (uint8 / float8_e4m3fn, r per row) or packed 4-bit codes (uint8, r/2 per row)."""
    if K_cache.dtype == torch.bfloat16:
        return TK_BF16
    if K_cache.shape[-1] == r:
        return TK_FP8_E4M3
    if K_cache.dtype == torch.uint8 and K_cache.shape[-1] * 2 == r:
        return TK_INT4
    raise ValueError(f"K_cache rows of {K_cache.shape[-1]} {K_cache.dtype} do not hold {r} key entries")


def prepare_decode(Q: torch.Tensor, K_cache: torch.Tensor, V_cache: torch.Tensor, ctx_lens: torch.Tensor,
                   max_ctx: Optional[int] = None, scale: float = 0.0, k_scale: Optional[torch.Tensor] = None,
                   block_table: Optional[torch.Tensor] = None, block_size: int = 0,
                   workspace: Optional[torch.Tensor] = None, O: Optional[torch.Tensor] = None,
                   stream=None, noalloc: bool = False) -> PreparedCall:
    """One decode step, marshalled. Q [B,Hq,r] bf16; K_cache bf16, uint8 E4M3 codes or uint8 packed 4-bit
    codes [.., r/2] (quantised keys with k_scale fp32); contiguous [B,Hkv,max_ctx,*] or paged
    [nblk,Hkv,bs,*] with block_table [B, mb] int32. With ``noalloc`` the call goes to
    tk_attn_decode_noalloc (the library's fixed scratch; no workspace)."""
    _check(Q, "Q", (torch.bfloat16,), 3)
    _check(K_cache, "K_cache", (torch.bfloat16, torch.uint8, torch.float8_e4m3fn), 4)
    _check(V_cache, "V_cache", (torch.bfloat16,), 4)
    _check(ctx_lens, "ctx_lens", (torch.int32,), 1)
    B, Hq, r = Q.shape
    Hkv, dv = V_cache.shape[1], V_cache.shape[3]
    kf = _key_format(K_cache, r)
    if kf != TK_BF16:
        if k_scale is None:
            raise ValueError("quantised keys need k_scale")
        _check(k_scale, "k_scale", (torch.float32,), 3)
        K_cache = K_cache.view(torch.uint8)
    elif k_scale is not None:
        raise ValueError("k_scale is only for quantised keys")
    if K_cache.shape[1] != Hkv or K_cache.shape[:3] != V_cache.shape[:3]:
        raise ValueError(f"cache shapes K{tuple(K_cache.shape)} V{tuple(V_cache.shape)} do not match r={r}")
    if k_scale is not None and tuple(k_scale.shape) != tuple(K_cache.shape[:3]):
        raise ValueError("k_scale must be [*, Hkv, tokens]")
    if ctx_lens.shape[0] != B:
        raise ValueError("ctx_lens must have one entry per sequence")
    if block_table is None:
        if K_cache.shape[0] != B:
            raise ValueError("contiguous cache must be [B, Hkv, max_ctx, *]")
        cap = K_cache.shape[2]
        mb = nblk = 0
        block_size = 0
    else:
        _check(block_table, "block_table", (torch.int32,), 2)
        if block_table.shape[0] != B:
            raise ValueError("block_table must be [B, max_blocks_per_seq]")
        if block_size != K_cache.shape[2]:
            raise ValueError("block_size must equal the cache's slot dimension")
        mb = block_table.shape[1]
        nblk = K_cache.shape[0]
        cap = mb * block_size
    if max_ctx is None:
        max_ctx = cap
    if max_ctx > cap:
        raise ValueError("max_ctx exceeds the cache capacity")
    if O is None:
        O = torch.empty(B, Hq, dv, dtype=torch.bfloat16, device=Q.device)
    _check(O, "O", (torch.bfloat16,), 3)
    head = (_ptr(Q), _ptr(K_cache), _ptr(V_cache), _ptr(O), B, Hq, Hkv, _ptr(ctx_lens), int(max_ctx), r, dv,
            float(scale), kf, _ptr(k_scale), _ptr(block_table), int(block_size), int(mb), int(nblk))
    if noalloc:
        if workspace is not None:
            raise ValueError("tk_attn_decode_noalloc takes no workspace")
        return PreparedCall("tk_attn_decode_noalloc", head + (_stream(stream),),
                            (Q, K_cache, V_cache, ctx_lens, k_scale, block_table, O))
    need = tk_attn_decode_workspace_bytes(B, Hq, Hkv, max_ctx, dv)
    if workspace is None:
        workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=Q.device)
    if workspace.device.type != "cuda":
        raise ValueError("workspace must be on the GPU")
    args = head + (_ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    return PreparedCall("tk_attn_decode", args, (Q, K_cache, V_cache, ctx_lens, k_scale, block_table, workspace, O))


def tk_attn_decode(Q: torch.Tensor, K_cache: torch.Tensor, V_cache: torch.Tensor, ctx_lens: torch.Tensor,
                   max_ctx: Optional[int] = None, scale: float = 0.0, k_scale: Optional[torch.Tensor] = None,
                   block_table: Optional[torch.Tensor] = None, block_size: int = 0,
                   workspace: Optional[torch.Tensor] = None, O: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    """One decode step. Q [B,Hq,r] bf16; K_cache bf16, uint8 E4M3 codes or uint8 packed 4-bit codes
    [.., r/2] (quantised keys with k_scale fp32); contiguous [B,Hkv,max_ctx,*] or paged [nblk,Hkv,bs,*]
    with block_table [B, mb] int32.
    A workspace passed in must have been zeroed before its first use (see include/tk_attn.h)."""
    return prepare_decode(Q, K_cache, V_cache, ctx_lens, max_ctx, scale, k_scale, block_table, block_size,
                          workspace, O, stream)()


def tk_attn_decode_noalloc(Q: torch.Tensor, K_cache: torch.Tensor, V_cache: torch.Tensor, ctx_lens: torch.Tensor,
                           max_ctx: Optional[int] = None, scale: float = 0.0, k_scale: Optional[torch.Tensor] = None,
                           block_table: Optional[torch.Tensor] = None, block_size: int = 0,
                           O: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """tk_attn_decode on the library's fixed scratch: the C call allocates nothing (pass O to keep this
    wrapper from allocating the output). Calls that may overlap on one GPU race (see include/tk_attn.h)."""
    return prepare_decode(Q, K_cache, V_cache, ctx_lens, max_ctx, scale, k_scale, block_table, block_size,
                          None, O, stream, noalloc=True)()


def prepare_cache_append(K_new: torch.Tensor, V_new: torch.Tensor, positions: torch.Tensor,
                         K_cache: torch.Tensor, V_cache: torch.Tensor, k_scale: Optional[torch.Tensor] = None,
                         block_table: Optional[torch.Tensor] = None, block_size: int = 0,
                         stream=None) -> PreparedCall:
    """Append marshalled. K_new [B,Hkv,T,r], V_new [B,Hkv,T,dv] bf16; positions [B] int32; caches as for
    decode: contiguous [B,Hkv,max_ctx,*] or paged [nblk,Hkv,bs,*] with block_table [B, mb] int32. A uint8 /
    float8_e4m3fn K_cache with r entries per row receives E4M3 codes, a uint8 K_cache with r/2 bytes per
    row packed 4-bit codes, each quantised per row with its scale written to k_scale (fp32)."""
    _check(K_new, "K_new", (torch.bfloat16,), 4)
    _check(V_new, "V_new", (torch.bfloat16,), 4)
    _check(positions, "positions", (torch.int32,), 1)
    _check(K_cache, "K_cache", (torch.bfloat16, torch.uint8, torch.float8_e4m3fn), 4)
    _check(V_cache, "V_cache", (torch.bfloat16,), 4)
    B, Hkv, T, r = K_new.shape
    dv = V_new.shape[3]
    if tuple(V_new.shape[:3]) != (B, Hkv, T) or positions.shape[0] != B:
        raise ValueError(f"shape mismatch K_new{tuple(K_new.shape)} V_new{tuple(V_new.shape)} "
                         f"positions{tuple(positions.shape)}")
    kf = _key_format(K_cache, r)
    if kf != TK_BF16:
        if k_scale is None:
            raise ValueError("quantised keys need k_scale")
        _check(k_scale, "k_scale", (torch.float32,), 3)
        K_cache = K_cache.view(torch.uint8)
    elif k_scale is not None:
        raise ValueError("k_scale is only for quantised keys")
    if K_cache.shape[1] != Hkv or K_cache.shape[:3] != V_cache.shape[:3] or V_cache.shape[3] != dv:
        raise ValueError(f"cache shapes K{tuple(K_cache.shape)} V{tuple(V_cache.shape)} do not match the rows")
    if k_scale is not None and tuple(k_scale.shape) != tuple(K_cache.shape[:3]):
        raise ValueError("k_scale must be [*, Hkv, tokens]")
    if block_table is None:
        if K_cache.shape[0] != B:
            raise ValueError("contiguous cache must be [B, Hkv, max_ctx, *]")
        max_ctx, mb, nblk, block_size = K_cache.shape[2], 0, 0, 0
    else:
        _check(block_table, "block_table", (torch.int32,), 2)
        if block_table.shape[0] != B or block_size != K_cache.shape[2]:
            raise ValueError("block_table must be [B, mb] and block_size the cache's slot dimension")
        max_ctx, mb, nblk = 0, block_table.shape[1], K_cache.shape[0]
    args = (_ptr(K_new), _ptr(V_new), B, Hkv, T, r, dv, _ptr(positions), _ptr(K_cache), _ptr(V_cache),
            int(max_ctx), kf, _ptr(k_scale), _ptr(block_table), int(block_size),
            int(mb), int(nblk), _stream(stream))
    return PreparedCall("tk_cache_append", args, (K_new, V_new, positions, k_scale, block_table, K_cache))


def tk_cache_append(K_new: torch.Tensor, V_new: torch.Tensor, positions: torch.Tensor, K_cache: torch.Tensor,
                    V_cache: torch.Tensor, k_scale: Optional[torch.Tensor] = None,
                    block_table: Optional[torch.Tensor] = None, block_size: int = 0, stream=None) -> None:
    """Write T new tokens per sequence into the cache at positions[b] + t (see include/tk_attn.h)."""
    prepare_cache_append(K_new, V_new, positions, K_cache, V_cache, k_scale, block_table, block_size, stream)()


def prepare_project_heads(X: torch.Tensor, Wt: torch.Tensor, n_heads: int, Y: Optional[torch.Tensor] = None,
                          stream=None) -> PreparedCall:
    """One thin projection, marshalled: X [B, S, d_model] bf16, Wt [n_heads * width, d_model] bf16
    (the weight transposed) -> Y [B, n_heads, S, width] bf16."""
    _check(X, "X", (torch.bfloat16,), 3)
    _check(Wt, "Wt", (torch.bfloat16,), 2)
    B, S, d_model = X.shape
    if Wt.shape[1] != d_model:
        raise ValueError(f"Wt {tuple(Wt.shape)} does not match d_model {d_model}")
    if n_heads <= 0 or Wt.shape[0] % n_heads:
        raise ValueError(f"{Wt.shape[0]} weight rows do not split into {n_heads} heads")
    width = Wt.shape[0] // n_heads
    if Y is None:
        Y = torch.empty(B, n_heads, S, width, dtype=torch.bfloat16, device=X.device)
    _check(Y, "Y", (torch.bfloat16,), 4)
    if tuple(Y.shape) != (B, n_heads, S, width):
        raise ValueError(f"Y must be {(B, n_heads, S, width)}")
    args = (_ptr(X), _ptr(Wt), _ptr(Y), B, S, d_model, n_heads, width, _stream(stream))
    return PreparedCall("tk_project_heads", args, (X, Wt, Y))


def tk_project_heads(X: torch.Tensor, Wt: torch.Tensor, n_heads: int, Y: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
    """Y[b, h, s, :] = X[b, s, :] @ Wt[h * width:(h + 1) * width, :].T, head-major bf16."""
    return prepare_project_heads(X, Wt, n_heads, Y, stream)()
