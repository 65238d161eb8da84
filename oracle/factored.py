"""Factored keys: truncated SVD of a key projection and query absorption (fp64).

TEST INFRASTRUCTURE ONLY. Follows Sec. 2.3 (Eq. 5-7): a key projection is
factored as W_K ~= A B with A = U_r S_r (the thin key projection, whose outputs
are cached) and B = V_r^T; B^T is absorbed into the query projection,
W_Q' = W_Q B^T, so that q' k'^T = x_i W_Q B^T A^T x_j^T, which equals the
original q k^T whenever W_K has rank at most r.

Reading of the paper used here: the factorisation is taken per KV head (one
d_model x d_head block of W_K per head, r columns kept per head), matching the
per-head key widths that the paper's tables quote and the GQA grouping; every
query head of a group absorbs that group's B. The library routine numpy.linalg.svd
(LAPACK, fp64) is the SVD step.
"""
from __future__ import annotations

import numpy as np


def factor_key_projection(w_k: np.ndarray, r: int):
    """Truncated SVD of one head's key projection w_k [d_model, d_head].

    Returns (A [d_model, r], B [r, d_head], singular values)."""
    u, s, vt = np.linalg.svd(np.asarray(w_k, dtype=np.float64), full_matrices=False)
    a = u[:, :r] * s[:r]
    b = vt[:r, :]
    return a, b, s


def absorb_query(w_q: np.ndarray, b: np.ndarray) -> np.ndarray:
    """W_Q' = W_Q B^T: [d_model, d_head] x [d_head, r] -> [d_model, r]."""
    return np.asarray(w_q, dtype=np.float64) @ b.T


def thin_projections(x: np.ndarray, w_q_heads, w_k_heads, r: int, group: int = 1):
    """Thin queries and keys for every head.

    x [n, d_model]; w_q_heads: list of Hq matrices [d_model, d_head];
    w_k_heads: list of Hkv matrices. Query head h uses KV head h // group.
    Returns (q' [Hq, n, r], k' [Hkv, n, r], per-KV-head singular values)."""
    ks, bs, sv = [], [], []
    for w_k in w_k_heads:
        a, b, s = factor_key_projection(w_k, r)
        ks.append(x @ a)
        bs.append(b)
        sv.append(s)
    qs = [x @ absorb_query(w_q, bs[h // group]) for h, w_q in enumerate(w_q_heads)]
    return np.stack(qs), np.stack(ks), sv


def project_heads(x: np.ndarray, w: np.ndarray, n_heads: int) -> np.ndarray:
    """One projection of a layer, head-major, in fp64: x [B, S, d_model] and
    w [d_model, n_heads * width] give Y [B, n_heads, S, width] with
    Y[b, h, s, :] = x[b, s, :] w[:, h width : (h + 1) width] (the layout the
    attention calls take). The product is numpy's fp64 matmul."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, S, d_model = x.shape
    width = w.shape[1] // n_heads
    y = x.reshape(B * S, d_model) @ w
    return y.reshape(B, S, n_heads, width).transpose(0, 2, 1, 3).copy()
