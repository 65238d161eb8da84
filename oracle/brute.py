"""Pure-Python brute force for tiny thin-key attention problems.

TEST INFRASTRUCTURE ONLY. An evaluator written independently of ``tk_oracle.c``:
it builds the whole score matrix with an explicit -inf mask, exponentiates with
``math.exp`` and sums with ``math.fsum`` (exactly rounded sums), then normalises.
It follows the definition of Sec. 2.1 (Eq. 4) with causal masking aligned to the
bottom-right corner and consecutive GQA grouping. Meant for sizes of a few
dozen rows; it is the brute-force pin of the C oracle.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

Matrix = List[List[float]]


def head_attention(q: Matrix, k: Matrix, v: Matrix, scale: float, causal: bool) -> Matrix:
    """softmax(scale * q k^T, masked) v for one head; q [Sq][r], k [Sk][r], v [Sk][dv]."""
    sq, sk = len(q), len(k)
    dv = len(v[0]) if sk else 0
    neg_inf = float("-inf")
    scores = [[neg_inf] * sk for _ in range(sq)]
    for i in range(sq):
        for j in range(sk):
            if causal and j > i + (sk - sq):
                continue
            scores[i][j] = scale * math.fsum(a * b for a, b in zip(q[i], k[j]))
    out = []
    for i in range(sq):
        row = scores[i]
        finite = [x for x in row if x != neg_inf]
        if not finite:
            out.append([0.0] * dv)
            continue
        m = max(finite)
        w = [math.exp(x - m) if x != neg_inf else 0.0 for x in row]
        z = math.fsum(w)
        out.append([math.fsum(w[j] * v[j][c] for j in range(sk)) / z for c in range(dv)])
    return out


def attention(Q, K, V, scale: float, causal: bool):
    """Nested lists Q [B][Hq][Sq][r], K [B][Hkv][Sk][r], V [B][Hkv][Sk][dv]."""
    B, Hq, Hkv = len(Q), len(Q[0]), len(K[0])
    G = Hq // Hkv
    return [[head_attention(Q[b][h], K[b][h // G], V[b][h // G], scale, causal)
             for h in range(Hq)] for b in range(B)]


def decode(Q, K, V, ctx_lens: Sequence[int], scale: float,
           block_table: Optional[Sequence[Sequence[int]]] = None, block_size: int = 0):
    """One query per sequence. Q [B][Hq][r]; K, V contiguous [B][Hkv][ctx][*] or,
    with ``block_table``, pages [nblk][Hkv][bs][*]."""
    B, Hq, Hkv = len(Q), len(Q[0]), len(K[0])
    G = Hq // Hkv
    out = []
    for b in range(B):
        L = ctx_lens[b]
        row = []
        for h in range(Hq):
            g = h // G
            if block_table is None:
                kk = [K[b][g][t] for t in range(L)]
                vv = [V[b][g][t] for t in range(L)]
            else:
                kk = [K[block_table[b][t // block_size]][g][t % block_size] for t in range(L)]
                vv = [V[block_table[b][t // block_size]][g][t % block_size] for t in range(L)]
            if L == 0:
                row.append([0.0] * len(V[0][0][0]))
            else:
                row.append(head_attention([Q[b][h]], kk, vv, scale, False)[0])
        out.append(row)
    return out
