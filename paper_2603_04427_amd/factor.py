"""Offline conversion of a pretrained attention layer to thin keys (Sec. 2.3, Eq. 5-7).

For every KV head g the key projection block W_K^(g) [d_model, d_head] is
replaced by its rank-r truncated SVD, U_r S_r V_r^T. The cached key becomes
k' = x W_K'^(g) with W_K'^(g) = U_r S_r [d_model, r], and the remaining factor
V_r^T is absorbed into the query projection of every query head h of the group:
W_Q'^(h) = W_Q^(h) V_r [d_model, r]. Then q' . k' = x_i W_Q V_r V_r^T W_K^T x_j^T,
which equals the original logit q . k when W_K^(g) has rank at most r, and
otherwise differs by at most |x_i W_Q^(h)| sigma_{r+1} |x_j| (Eckart-Young).

The factorisation is per KV head (the per-head key widths of the paper's
tables, and the grouping of GQA); the query heads of a group share its factor.
Values and the output projection are untouched: V keeps its full width.

The factorisation is weight preprocessing, done once on the host before
serving. `project_thin` applies the converted projections on the GPU with the
library's projection kernel (tk_project_heads) to produce the head-major bf16
Q, K and V that `tk_attn_prefill` and `tk_cache_append` take. The softmax scale that preserves
a pretrained model's attention is the original 1/sqrt(d_head), passed to the
kernels explicitly.
"""
from __future__ import annotations

import torch

from .binding import tk_project_heads


def _head_blocks(w: torch.Tensor, n_heads: int) -> torch.Tensor:
    """[d_model, n_heads * d_head] -> [n_heads, d_model, d_head] (head h owns
    columns h d_head .. (h + 1) d_head - 1, the usual head-major split)."""
    d_model, width = w.shape
    if width % n_heads:
        raise ValueError(f"projection width {width} is not a multiple of {n_heads} heads")
    return w.reshape(d_model, n_heads, width // n_heads).permute(1, 0, 2)


def factor_layer(w_q: torch.Tensor, w_k: torch.Tensor, r: int, h_q: int, h_kv: int):
    """Thin query and key projections of one layer.

    w_q [d_model, h_q d_head] and w_k [d_model, h_kv d_head] map a token's
    hidden state (a row vector x) to its queries and keys, x @ w. Query head h
    reads KV head h // (h_q / h_kv). The SVD runs in float64 on the host.

    Returns (w_q_thin [d_model, h_q r], w_k_thin [d_model, h_kv r],
    sigma [h_kv, min(d_model, d_head)]: the singular values of every key head,
    whose tail beyond r bounds the logit error), all float64 on the CPU."""
    if h_kv <= 0 or h_q % h_kv:
        raise ValueError("h_q must be a positive multiple of h_kv")
    wq = _head_blocks(w_q.detach().to("cpu", torch.float64), h_q)
    wk = _head_blocks(w_k.detach().to("cpu", torch.float64), h_kv)
    d_model, d_head = wk.shape[1], wk.shape[2]
    if wq.shape[2] != d_head:
        raise ValueError("query and key heads must have the same width before factoring")
    if not 0 < r <= min(d_model, d_head):
        raise ValueError(f"rank {r} outside 1..{min(d_model, d_head)}")
    u, s, vh = torch.linalg.svd(wk, full_matrices=False)  # per head: wk = u diag(s) vh
    k_thin = u[:, :, :r] * s[:, None, :r]                 # [h_kv, d_model, r]
    v_r = vh[:, :r, :].transpose(1, 2)                    # [h_kv, d_head, r]
    group = h_q // h_kv
    q_thin = torch.matmul(wq, v_r.repeat_interleave(group, dim=0))  # [h_q, d_model, r]
    return (q_thin.permute(1, 0, 2).reshape(d_model, h_q * r),
            k_thin.permute(1, 0, 2).reshape(d_model, h_kv * r), s)


def logit_error_bound(x_q: torch.Tensor, w_q: torch.Tensor, x_k: torch.Tensor, sigma_next: float) -> torch.Tensor:
    """Eckart-Young bound on |q . k - q' . k'| for one query head: for query
    rows x_q [n, d_model] with that head's block w_q [d_model, d_head] and key
    rows x_k [m, d_model], |x_q w_q| sigma_{r+1} |x_k| as an [n, m] matrix."""
    qn = torch.linalg.vector_norm(x_q @ w_q, dim=-1)
    kn = torch.linalg.vector_norm(x_k, dim=-1)
    return qn[:, None] * sigma_next * kn[None, :]


def transposed_bf16(w: torch.Tensor, device) -> torch.Tensor:
    """A projection weight w [d_model, n_heads * width] as the kernel takes it:
    transposed, [n_heads * width, d_model], bf16, contiguous, on ``device``
    (done once per layer, with the conversion)."""
    return w.detach().t().to(device=device, dtype=torch.bfloat16).contiguous()


def project_thin(x: torch.Tensor, w_q_thin: torch.Tensor, w_k_thin: torch.Tensor, w_v: torch.Tensor,
                 h_q: int, h_kv: int):
    """Queries, thin keys and values of hidden states x [B, S, d_model], head-major
    bf16 on x's device: Q [B, h_q, S, r], K [B, h_kv, S, r], V [B, h_kv, S, d_v].

    Each projection is one tk_project_heads call (bf16 matrix cores, fp32
    accumulation, one rounding to bf16) on the weights as ``factor_layer``
    returns them, [d_model, n * width], converted with ``transposed_bf16``
    (a serving loop converts once and calls tk_project_heads directly); x is
    taken in bf16."""
    xb = x.to(torch.bfloat16).contiguous()

    def heads(w, n):
        return tk_project_heads(xb, transposed_bf16(w, x.device), n)

    return heads(w_q_thin, h_q), heads(w_k_thin, h_kv), heads(w_v, h_kv)
