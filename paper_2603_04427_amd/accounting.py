"""Byte and FLOP accounting for thin-key attention.

Two kinds of figures live here:

* The paper's analytical cache model: the KV-cache sizes of Eq. 8-9
  (Sec. 2.4), the per-user tables of Sec. 4.1 and of the GQA/MLA comparison
  (Sec. 3, Exp. 7b), and the decode bandwidth model of Eq. 10 (Sec. 4.2).
* The algorithmic work of one kernel call, used as the numerator of achieved
  GB/s and TFLOP/s: decode moves every visible key row (r elements of the key
  dtype, half a byte each for 4-bit keys, plus one fp32 scale per row for
  quantised keys) and every value row (d_v
  bf16) once per KV head, plus the queries, outputs, lengths and block table;
  causal prefill performs 2 (r + d_v) FLOPs for each (query head, visible key)
  pair, the diagonal included, with no credit for masked work.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

# ---------------------------------------------------------------- Eq. 8-9


def kv_cache_bytes_standard(n: int, d_model: int, layers: int, bytes_per: float) -> float:
    """Standard KV cache: 2 n d_model L b bytes (Eq. 8)."""
    return 2.0 * n * d_model * layers * bytes_per


def kv_cache_bytes_thin(n: int, d_select: int, d_model: int, layers: int, bytes_per: float) -> float:
    """Asymmetric KV cache: n (d_select + d_model) L b bytes (Eq. 9)."""
    return float(n) * (d_select + d_model) * layers * bytes_per


def kv_cache_bytes(n: int, layers: int, bytes_per: float, k_width: int, v_width: int) -> float:
    """K and V cache bytes for per-token key/value widths summed over KV heads."""
    return float(n) * (k_width + v_width) * layers * bytes_per


# ---------------------------------------------------------------- Eq. 10


def mistral_c_kv(n: int, layers: int, n_kv: int, d_k: int, d_v: int, beta: float) -> float:
    """Per-sequence cache bytes at context n: L n_kv (d_k + d_v) n beta.

    With d_k = d_v = d_head this is the 2 L n_kv d_head n beta of Sec. 4.2."""
    return float(layers) * n_kv * (d_k + d_v) * n * beta


def decode_speedup(w: float, c_kv: float, w_thin: float, c_kv_thin: float, batch: float) -> float:
    """(W + b C_kv) / (W' + b C'_kv): Eq. 10."""
    return (w + batch * c_kv) / (w_thin + batch * c_kv_thin)


# ---------------------------------------------------------------- kernel work

KEY_BYTES = {"bf16": 2, "fp8": 1, "int4": 0.5, "f32": 4}


def decode_bytes(ctx_lens: Sequence[int], h_q: int, h_kv: int, r: int, d_v: int,
                 k_dtype: str = "bf16", paged_blocks_per_seq: Optional[int] = None) -> int:
    """Algorithmic bytes of one decode call (bf16 queries, values and outputs)."""
    kb = KEY_BYTES[k_dtype]
    per_token = h_kv * (int(r * kb) + (4 if k_dtype in ("fp8", "int4") else 0) + d_v * 2)
    total = sum(int(L) for L in ctx_lens) * per_token
    B = len(ctx_lens)
    total += B * h_q * r * 2 + B * h_q * d_v * 2 + B * 4
    if paged_blocks_per_seq is not None:
        total += B * paged_blocks_per_seq * 4
    return total


def causal_pairs(seq_q: int, seq_k: int) -> int:
    """Visible (query, key) pairs of one head under bottom-right causal masking."""
    off = seq_k - seq_q
    return sum(min(seq_k, i + off + 1) for i in range(seq_q)) if off else seq_q * (seq_q + 1) // 2


def prefill_flops(batch: int, h_q: int, seq_q: int, seq_k: int, r: int, d_v: int, causal: bool = True) -> int:
    """Algorithmic FLOPs: 2 (r + d_v) per visible (query head, key) pair."""
    pairs = causal_pairs(seq_q, seq_k) if causal else seq_q * seq_k
    return batch * h_q * pairs * 2 * (r + d_v)


def prefill_backward_flops(batch: int, h_q: int, seq_q: int, seq_k: int, r: int, d_v: int,
                           causal: bool = True) -> int:
    """Algorithmic FLOPs of the backward pass: per visible (query head, key) pair the
    five products S = Q K^T (2r), dP = dO V^T (2 d_v), dV = P^T dO (2 d_v),
    dQ = dS K (2r) and dK = dS^T Q (2r), so 2 (3r + 2 d_v). Work a kernel repeats
    (recomputing S and dP in a second pass) is not counted."""
    pairs = causal_pairs(seq_q, seq_k) if causal else seq_q * seq_k
    return batch * h_q * pairs * 2 * (3 * r + 2 * d_v)


def prefill_bytes(batch: int, h_q: int, h_kv: int, seq_q: int, seq_k: int, r: int, d_v: int,
                  elem_bytes: int) -> int:
    """Compulsory bytes of a prefill call: Q, K, V read once and O written once."""
    return elem_bytes * batch * (h_q * seq_q * (r + d_v) + h_kv * seq_k * (r + d_v))


# ---------------------------------------------------------------- MI355X peaks

HBM_PEAK_GBS = 8000.0            # 8 TB/s HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0   # dense bf16 matrix
FP32_MFMA_PEAK_TFLOPS = 157.3    # fp32 matrix / vector


def frac(achieved: float, peak: float) -> float:
    return achieved / peak if peak > 0 and math.isfinite(achieved) else float("nan")
