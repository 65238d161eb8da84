"""Cache append, written out plainly (test infrastructure only).

What the write before decode computes, for the thin-key / full-value cache of
Sec. 2.4 (Eq. 9): the key row (r entries) and value row (d_v entries) of new
token t of sequence b and KV head g go to cache position positions[b] + t,
either in a contiguous cache [B, Hkv, max_ctx, *] or, through a block table, in
a paged cache [num_blocks, Hkv, block_size, *]. A position outside
[0, capacity) or a table entry outside [0, num_blocks) is skipped.

fp8 keys (thin keys composed with quantisation, the suggestion of Sec. 6): per
key row, scale = max|k| / 448 (1 for an all-zero row) and code = E4M3(k / scale)
with round-to-nearest-even, every step in fp32 (IEEE division), so that the
integer codes are decided in the same precision as on the GPU. The rounding to
E4M3 uses torch's float8_e4m3fn conversion as a library step.

4-bit integer keys: per key row, scale = max|k| / 7 (1 for an all-zero row) and
code c = k / scale rounded half-to-even and clipped to [-7, 7], in fp32; stored
excess-8 (nibble c + 8), entry 2j in the low and entry 2j + 1 in the high nibble
of byte j.

Nothing here is shared with the GPU library; only the tests use it.
"""
from __future__ import annotations

from typing import Optional, Tuple

import torch

E4M3_MAX = 448.0


def quantize_rows(k: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per-row (last axis) E4M3 codes (uint8) and fp32 scales of fp32 rows ``k``."""
    k = k.to(torch.float32)
    amax = k.abs().amax(dim=-1)
    scale = torch.where(amax > 0, amax / torch.tensor(E4M3_MAX, dtype=torch.float32),
                        torch.ones_like(amax))
    codes = (k / scale.unsqueeze(-1)).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, scale


def quantize_rows_int4(k: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per-row (last axis, even length) packed 4-bit codes (uint8 [..., r / 2]) and
    fp32 scales of fp32 rows ``k``."""
    k = k.to(torch.float32)
    amax = k.abs().amax(dim=-1)
    scale = torch.where(amax > 0, amax / torch.tensor(7.0, dtype=torch.float32), torch.ones_like(amax))
    c = torch.round(k / scale.unsqueeze(-1)).clamp(-7, 7).to(torch.int32) + 8  # round: half to even
    packed = (c[..., 0::2] | (c[..., 1::2] << 4)).to(torch.uint8)
    return packed, scale


def cache_append(k_new: torch.Tensor, v_new: torch.Tensor, positions: torch.Tensor, k_cache: torch.Tensor,
                 v_cache: torch.Tensor, k_scale: Optional[torch.Tensor] = None,
                 block_table: Optional[torch.Tensor] = None, block_size: int = 0, k_format: str = "auto"):
    """Returns copies of (k_cache, v_cache, k_scale) with the new rows written.

    k_new [B, Hkv, T, r], v_new [B, Hkv, T, dv] (bf16); positions [B] int; caches on
    the CPU. ``k_cache`` of dtype uint8 holds E4M3 codes [.., r] or, with
    k_format="int4", packed 4-bit codes [.., r / 2], with ``k_scale``."""
    k_cache, v_cache = k_cache.clone(), v_cache.clone()
    k_scale = None if k_scale is None else k_scale.clone()
    B, Hkv, T, r = k_new.shape
    fp8 = k_cache.dtype == torch.uint8
    if fp8:
        if k_format == "int4":
            codes, scales = quantize_rows_int4(k_new.to(torch.float32))
        else:
            codes, scales = quantize_rows(k_new.to(torch.float32))
    if block_table is None:
        capacity = k_cache.shape[2]
    else:
        capacity = block_size * block_table.shape[1]
        n_blocks = k_cache.shape[0]
    for b in range(B):
        for t in range(T):
            pos = int(positions[b]) + t
            if pos < 0 or pos >= capacity:
                continue
            if block_table is None:
                blk, slot, ok = b, pos, True
            else:
                blk = int(block_table[b, pos // block_size])
                slot = pos % block_size
                ok = 0 <= blk < n_blocks
            if not ok:
                continue
            # every KV head of the token (heads share the position and the table entry)
            v_cache[blk, :, slot] = v_new[b, :, t]
            if fp8:
                k_cache[blk, :, slot] = codes[b, :, t]
                k_scale[blk, :, slot] = scales[b, :, t]
            else:
                k_cache[blk, :, slot] = k_new[b, :, t]
    return k_cache, v_cache, k_scale
