"""The synthetic workloads: shapes, value recipes and layouts.

Shapes follow the paper's models (GPT-2 small: 12 heads, d_head 64, 16 key
dimensions per head after factoring; Mistral-7B: 32 query heads over 8 KV heads,
d_head 128, 32 key dimensions per head), stated in Sec. 3 (Exp. 5 and Exp. 8)
and the decode table of Sec. 4.2. Real activations are absent, so every tensor
is an i.i.d. draw; the "structured" variants plant a peaked attention pattern
(a needle for decode, the copy-back offset of Exp. 1 for prefill) so that
outputs are O(1) and a wrong index or a dropped block shows up as a large error.

Layouts are head-major:
  prefill  Q [B, Hq, Sq, r]   K [B, Hkv, Sk, r]   V [B, Hkv, Sk, dv]
  decode   Q [B, Hq, r]       contiguous K [B, Hkv, ctx, r], V [B, Hkv, ctx, dv]
           paged K [nblk, Hkv, bs, r], V [nblk, Hkv, bs, dv], table [B, ctx/bs]
  fp8 keys are OCP E4M3FN codes (uint8) with one fp32 scale per (token, KV head),
  scale = max|k| / 448 over the r entries (1 where the row is all zero).
Nothing here computes scores, softmax or outputs.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

import torch

from .gen import normal, permutation, stream_key, uniform_int

E4M3_MAX = 448.0

# tensor ids inside one workload's seed family
T_Q, T_K, T_V, T_PERM, T_STRUCT, T_DO = 0, 1, 2, 3, 4, 5


@dataclass(frozen=True)
class PrefillSpec:
    name: str
    config_id: int
    batch: int
    h_q: int
    h_kv: int
    seq_q: int
    seq_k: int
    r: int
    d_v: int
    dtype: str = "bf16"          # "bf16" or "f32"
    amp: float = 1.0             # entries are amp * N(0, 1)
    causal: bool = True
    scale: Optional[float] = None  # None -> 1/sqrt(r)

    @property
    def softmax_scale(self) -> float:
        return self.scale if self.scale is not None else 1.0 / math.sqrt(self.r)


@dataclass(frozen=True)
class DecodeSpec:
    name: str
    config_id: int
    batch: int
    h_q: int
    h_kv: int
    ctx: int                     # max context (sizes the contiguous cache)
    r: int
    d_v: int
    k_dtype: str = "bf16"        # "bf16", "fp8" (E4M3) or "int4"
    paged: bool = False
    block_size: int = 256
    ctx_lens: Optional[Tuple[int, ...]] = None  # ragged lengths; None -> all ctx
    scale: Optional[float] = None

    @property
    def softmax_scale(self) -> float:
        return self.scale if self.scale is not None else 1.0 / math.sqrt(self.r)

    @property
    def lens(self) -> Tuple[int, ...]:
        return self.ctx_lens if self.ctx_lens is not None else (self.ctx,) * self.batch

    @property
    def blocks_per_seq(self) -> int:
        return -(-self.ctx // self.block_size)


# The five workloads, by what they are.
WORKLOADS = {
    # GPT-2 small, one layer of causal prefill, fp32 (Exp. 5 shape: 12 heads, r/head 16).
    "gpt2_prefill_f32": PrefillSpec("gpt2_prefill_f32", 1, 1, 12, 12, 1024, 1024, 16, 64,
                                    dtype="f32", amp=1.0),
    # Mistral-7B decode step, batch 16, context 4096 (Exp. 8 shape, r256 -> 32 per head).
    "mistral_decode_b16": DecodeSpec("mistral_decode_b16", 2, 16, 32, 8, 4096, 32, 128),
    # Mistral-7B causal prefill, batch 4, 8192 tokens, bf16 entries 0.5 * N(0,1).
    "mistral_prefill_s8192": PrefillSpec("mistral_prefill_s8192", 3, 4, 32, 8, 8192, 8192, 32, 128,
                                         dtype="bf16", amp=0.5),
    # 7B long-context decode, 131072 tokens in 256-token pages with a permuted block table.
    "longctx_paged_decode": DecodeSpec("longctx_paged_decode", 4, 8, 32, 8, 131072, 32, 128,
                                       paged=True, block_size=256),
    # Thin keys composed with 8-bit quantisation: fp8-e4m3 keys, per-token-head scale.
    "fp8key_decode": DecodeSpec("fp8key_decode", 5, 32, 32, 8, 32768, 32, 128, k_dtype="fp8"),
}

# Thin keys composed with 4-bit quantisation (the composition the discussion in
# Sec. 6 proposes): the fp8-key workload with 4-bit integer keys.
INT4KEY = {"int4key_decode": DecodeSpec("int4key_decode", 5, 32, 32, 8, 32768, 32, 128, k_dtype="int4")}


# Full-key controls: the same workloads with standard-width keys (r = d_head =
# 128, scale 1/sqrt(128)) and the same value streams, so that thin-key and
# full-key attention can be timed side by side (the decode saving the paper
# predicts from the byte ratio, Eq. 8-10, and the prefill selection cost).
# The 4-bit-key decode's control has standard-width bf16 keys: it measures the
# composition of thin keys with 4-bit quantisation (Sec. 6) against plain keys.
FULLKEY = {
    name + "_fullkey": replace(WORKLOADS[name], name=name + "_fullkey", r=128)
    for name in ("mistral_decode_b16", "mistral_prefill_s8192", "longctx_paged_decode")
}
FULLKEY["int4key_decode_fullkey"] = replace(INT4KEY["int4key_decode"], name="int4key_decode_fullkey", r=128,
                                            k_dtype="bf16")


def _draw(spec_id: int, tensor: int, shape, device, amp: float = 1.0) -> torch.Tensor:
    n = 1
    for s in shape:
        n *= s
    x = normal(stream_key(spec_id, tensor), n, device=device).view(*shape)
    if amp != 1.0:
        x = x * amp
    return x


def quantize_e4m3(k: torch.Tensor):
    """Per-row (last axis) OCP E4M3FN codes and fp32 scales: scale = max|k| / 448.

    Encoding is torch's float8_e4m3fn cast (round to nearest even). Returns
    (codes uint8 [..., r], scales fp32 [...])."""
    amax = k.abs().amax(dim=-1)
    scale = torch.where(amax > 0, amax / E4M3_MAX, torch.ones_like(amax)).to(torch.float32)
    codes = (k / scale.unsqueeze(-1)).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, scale


INT4_MAX = 7.0


def quantize_int4(k: torch.Tensor):
    """Per-row (last axis, even length) 4-bit integer codes and fp32 scales:
    scale = max|k| / 7 (1 where the row is all zero), code = k / scale rounded
    half-to-even and clipped to [-7, 7], stored excess-8 two per byte (entry 2j in
    the low nibble of byte j). Returns (packed uint8 [..., r / 2], scales fp32 [...])."""
    k = k.to(torch.float32)
    amax = k.abs().amax(dim=-1)
    scale = torch.where(amax > 0, amax / INT4_MAX, torch.ones_like(amax)).to(torch.float32)
    n = torch.round(k / scale.unsqueeze(-1)).clamp(-7, 7).to(torch.int32) + 8
    return (n[..., 0::2] | (n[..., 1::2] << 4)).to(torch.uint8), scale


def make_prefill(spec: PrefillSpec, device="cpu", structured: bool = False, needle_logit: Optional[float] = None):
    """Q, K, V of a prefill workload, in the workload's dtype, on ``device``.

    ``structured`` plants the copy-back pattern; by default its planted logit is
    about 2 sqrt(r) over noise logits of standard deviation 2 (rows close to
    one-hot). ``needle_logit`` sets the planted logit's expected size instead
    (noise standard deviation needle_logit / sqrt(r)), for moderately peaked rows."""
    B, Hq, Hkv, Sq, Sk, r, dv = spec.batch, spec.h_q, spec.h_kv, spec.seq_q, spec.seq_k, spec.r, spec.d_v
    dt = torch.float32 if spec.dtype == "f32" else torch.bfloat16
    q = _draw(spec.config_id, T_Q, (B, Hq, Sq, r), device, spec.amp)
    k = _draw(spec.config_id, T_K, (B, Hkv, Sk, r), device, spec.amp)
    v = _draw(spec.config_id, T_V, (B, Hkv, Sk, dv), device, spec.amp)
    k = k.to(dt)
    if structured:
        # copy-back (Exp. 1: y_t = x_{t-8}): query row i points at key row i - 8 of its
        # KV head, scaled so that the noise logits have standard deviation about 2.
        G = Hq // Hkv
        off = 8 + (Sk - Sq)
        lam = 2.0 / (spec.amp * spec.amp * math.sqrt(r) * spec.softmax_scale)
        if needle_logit is not None:
            lam = needle_logit / (spec.amp * spec.amp * r * spec.softmax_scale)
        kk = k.to(torch.float32).repeat_interleave(G, dim=1)  # [B, Hq, Sk, r]
        i0 = max(0, -off + 0)
        rows = torch.arange(Sq, device=device)
        src = rows + (Sk - Sq) - 8
        ok = src >= 0
        q[:, :, rows[ok]] = lam * kk[:, :, src[ok]]
        del kk, i0
    return {"q": q.to(dt), "k": k, "v": v.to(dt)}


def make_prefill_grad(spec: PrefillSpec, device="cpu"):
    """The loss gradient dO [B, Hq, Sq, dv] of a prefill workload for the backward
    pass: i.i.d. N(0, 1) entries in the workload's dtype."""
    dt = torch.float32 if spec.dtype == "f32" else torch.bfloat16
    return _draw(spec.config_id, T_DO, (spec.batch, spec.h_q, spec.seq_q, spec.d_v), device).to(dt)


def _to_pages(x: torch.Tensor, table: torch.Tensor, bs: int, n_blocks: int) -> torch.Tensor:
    """Scatter a logical [B, H, ctx, w] cache into pages [n_blocks, H, bs, w] per ``table``."""
    B, H, ctx, w = x.shape
    mb = table.shape[1]
    pad = mb * bs - ctx
    if pad:
        x = torch.nn.functional.pad(x, (0, 0, 0, pad)) if x.dtype.is_floating_point else \
            torch.cat([x, x.new_zeros(B, H, pad, w)], dim=2)
    blocks = x.view(B, H, mb, bs, w).permute(0, 2, 1, 3, 4).reshape(B * mb, H, bs, w)
    pages = x.new_zeros(n_blocks, H, bs, w)
    pages[table.reshape(-1).to(torch.int64).to(x.device)] = blocks
    return pages


def make_decode(spec: DecodeSpec, device="cpu", structured: bool = False):
    """Query, caches, lengths and (paged) block table of a decode workload.

    Returns a dict with q [B,Hq,r] bf16, k (bf16 or uint8 codes), k_scale (fp32
    or None), v bf16, ctx_lens int32 [B], block_table int32 [B, mb] or None, and
    k_logical / v_logical: the contiguous [B, Hkv, ctx, *] views of the same
    values (for paged workloads these are extra copies; for contiguous ones they
    alias k / v)."""
    B, Hq, Hkv, ctx, r, dv = spec.batch, spec.h_q, spec.h_kv, spec.ctx, spec.r, spec.d_v
    lens = torch.tensor(spec.lens, dtype=torch.int32)
    assert lens.numel() == B and int(lens.max()) <= ctx and int(lens.min()) >= 0
    q = _draw(spec.config_id, T_Q, (B, Hq, r), device)
    kf = _draw(spec.config_id, T_K, (B, Hkv, ctx, r), device)
    v = _draw(spec.config_id, T_V, (B, Hkv, ctx, dv), device).to(torch.bfloat16)
    if structured:
        G = Hq // Hkv
        pos = uniform_int(stream_key(spec.config_id, T_STRUCT), B * Hq, 1 << 30, device="cpu")
        pos = pos.view(B, Hq) % lens.clamp(min=1).view(B, 1).to(torch.int64)
        lam = 2.0 / (math.sqrt(r) * spec.softmax_scale)
        for b in range(B):
            if int(lens[b]) == 0:
                continue
            for h in range(Hq):
                q[b, h] = lam * kf[b, h // G, int(pos[b, h])]
    q = q.to(torch.bfloat16)
    if spec.k_dtype == "fp8":
        k, k_scale = quantize_e4m3(kf)
    elif spec.k_dtype == "int4":
        k, k_scale = quantize_int4(kf)
    else:
        k, k_scale = kf.to(torch.bfloat16), None
    del kf
    out = {"q": q, "ctx_lens": lens.to(device), "k_logical": k, "v_logical": v,
           "k_scale_logical": k_scale}
    if spec.paged:
        mb = spec.blocks_per_seq
        n_blocks = B * mb
        table = permutation(stream_key(spec.config_id, T_PERM), n_blocks).view(B, mb).to(torch.int32)
        bs = spec.block_size
        out["k"] = _to_pages(k, table, bs, n_blocks)
        out["v"] = _to_pages(v, table, bs, n_blocks)
        out["k_scale"] = None if k_scale is None else \
            _to_pages(k_scale.unsqueeze(-1), table, bs, n_blocks).squeeze(-1)
        out["block_table"] = table.to(device)
    else:
        out["k"], out["v"], out["k_scale"], out["block_table"] = k, v, k_scale, None
    return out


def with_shape(spec, **kw):
    """A copy of ``spec`` with some fields replaced (for test sweeps)."""
    return replace(spec, **kw)
