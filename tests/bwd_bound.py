"""Error bound for the prefill backward run end to end (GPU forward, then
backward) against the exact gradient.

The backward's contract (as in every flash-style backward) forms
D_i = sum_c dO_ic O_ic from the output O it is handed, i.e. the forward's
stored bf16 output, not the exact one. The exact gradient differs from the
gradient of that contract only through D:

    dS_ij = P_ij (dP_ij - D_i)   =>   delta dS_ij = -P_ij delta D_i,
    delta dQ_ic = -scale delta D_i  sum_j P_ij K_jc,
    delta dK_jc = -scale sum_i P_ij delta D_i Q_ic   (summed over the group's heads),
    delta dV    = 0,
    |delta D_i| <= sum_c |dO_ic| eps_ic,   eps_ic >= |O_stored,ic - O_ic|.

The forward rounds each weight to bf16 before both the value product and the
row sum (relative error u = 2^-8 each), so its fp32 output is a weighted mean
with weights off by at most 2u/(1-u) relative: |O_fp32 - O| <= 2.02 u sum_j
P_ij |V_jc - O_ic|. Rounding that output to bf16 adds u |O|, and fp32
accumulation adds well under 1e-6 max|V|. Everything on the right-hand side is
computed here from the exact (fp64 oracle) P and O, never from GPU output.

gate_end_to_end applies, per gradient tensor, with B that bound:
    |got - exact| <= B + 2e-2 max|exact|      (element by element)
    ||got - exact|| <= ||B|| + 1e-2 ||exact||  (L2)
the same max-abs and rel-L2 bars as the isolated backward tests, widened by
exactly the D term. A case is only admissible when the L2 bar stays below half
of ||exact||, so that an all-zero (or otherwise unrelated) gradient fails it."""
from __future__ import annotations

import torch

from oracle import oracle as orc

U_BF16 = 2.0 ** -8


def exact_terms(q, k, v, do, causal, scale):
    """Exact gradients (fp64 oracle) and the D-term bounds (B_dQ, B_dK, B_dV).

    With a causal mask, q and do may hold only the last rows of the sequences
    (bottom-right alignment places them at their original positions); dK and dV
    are then the full gradients of the keys those rows alone see."""
    dq, dk, dv, lse = orc.prefill_backward(q, k, v, do, causal=causal, scale=scale)
    o = orc.prefill(q, k, v, causal=causal, scale=scale)               # [B,Hq,Sq,dv] fp64
    qd, kd, vd, dod = (t.double() for t in (q, k, v, do))
    B, Hq, Sq, r = qd.shape
    Hkv, Sk = kd.shape[1], kd.shape[2]
    G = Hq // Hkv
    kx = kd.repeat_interleave(G, dim=1)
    vx = vd.repeat_interleave(G, dim=1)
    s = scale * torch.matmul(qd, kx.transpose(-1, -2))                  # [B,Hq,Sq,Sk]
    if causal:
        i = torch.arange(Sq).view(-1, 1) + (Sk - Sq)
        j = torch.arange(Sk).view(1, -1)
        s = s.masked_fill(j > i, float("-inf"))
    p = torch.exp(s - lse.unsqueeze(-1))
    dp = torch.matmul(dod, vx.transpose(-1, -2))                        # [B,Hq,Sq,Sk]
    dd = (dod * o).sum(-1, keepdim=True)                                # exact D
    # weight rounding enters D as sum_j w_ij (dP_ij - D_i), |w_ij| <= 2.02 u P_ij;
    # output rounding as sum_c dO_ic rho_ic, |rho_ic| <= u |O_fp32,ic|
    w_term = 2.02 * U_BF16 * (p * (dp - dd).abs()).sum(-1)
    # |O_fp32| <= |O| + 2.02 u sum_j P_ij |V_jc - O_ic| <= (1 + 2.02 u) |O| + 2.02 u (P |V|)_ic
    o32 = (1 + 2.02 * U_BF16) * o.abs() + 2.02 * U_BF16 * torch.matmul(p, vx.abs())
    rho_term = U_BF16 * (dod.abs() * o32).sum(-1)
    dD = w_term + rho_term + 1e-6 * vd.abs().max() * dod.abs().sum(-1)  # [B,Hq,Sq]
    b_dq = scale * dD.unsqueeze(-1) * torch.matmul(p, kx.abs())         # [B,Hq,Sq,r]
    b_dk = scale * torch.matmul((p * dD.unsqueeze(-1)).transpose(-1, -2), qd.abs())   # [B,Hq,Sk,r]
    b_dk = b_dk.view(B, Hkv, G, Sk, r).sum(2)
    return (dq, dk, dv), (b_dq, b_dk, torch.zeros_like(dv))


def bars(exact, bound):
    """(elementwise bar, L2 bar) of one gradient tensor."""
    return bound + 2e-2 * exact.abs().max(), bound.norm() + 1e-2 * exact.norm()


def admissible(exact, bound) -> bool:
    """True when an all-zero gradient fails the L2 bar with margin (bar < ||exact|| / 2)."""
    return bool(bars(exact, bound)[1] < 0.5 * exact.norm())


def check(got, exact, bound):
    """(ok, message) for one gradient tensor against the end-to-end bars."""
    g = got.detach().double().cpu()
    if not torch.isfinite(g).all():
        return False, "non-finite"
    el, l2 = bars(exact, bound)
    d = (g - exact).abs()
    worst = (d - el).max().item()
    n = (g - exact).norm().item()
    ok = worst <= 0 and n <= l2.item()
    return ok, (f"L2 err {n:.3e} (bar {l2.item():.3e}, ||exact|| {exact.norm().item():.3e}); "
                f"worst element over its bar by {worst:.2e}")
