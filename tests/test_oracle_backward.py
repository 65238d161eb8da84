"""Pins of the oracle's prefill backward (``oracle.prefill_backward``) against
things other than itself: central finite differences of the forward oracle,
fp64 autograd through a textbook attention expression (torch), the closed form
for equal value rows, the log-sum-exp against torch.logsumexp, and the partial
(row_lo) evaluation against the full one."""
import math

import pytest
import torch

from oracle import oracle

pytestmark = []


def rand(shape, seed, dtype=torch.float64):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g, dtype=torch.float64).to(dtype)


def textbook(q, k, v, causal, scale):
    """softmax(scale Q K^T [bottom-right causal mask]) V with K, V repeated over each
    group of consecutive query heads, in fp64."""
    Hq, Hkv = q.shape[1], k.shape[1]
    kr = k.repeat_interleave(Hq // Hkv, dim=1)
    vr = v.repeat_interleave(Hq // Hkv, dim=1)
    s = (q @ kr.transpose(-1, -2)) * scale
    if causal:
        Sq, Sk = q.shape[2], k.shape[2]
        i = torch.arange(Sq).view(-1, 1)
        j = torch.arange(Sk).view(1, -1)
        s = s.masked_fill(j > i + (Sk - Sq), float("-inf"))
    return torch.softmax(s, dim=-1) @ vr, torch.logsumexp(s, dim=-1)


CASES = [  # B, Hq, Hkv, Sq, Sk, r, dv, causal
    (1, 2, 1, 5, 5, 3, 4, True),
    (2, 4, 2, 7, 7, 4, 6, True),
    (1, 3, 3, 4, 9, 2, 5, True),      # bottom-right: 4 new rows after 5 cached keys
    (1, 2, 2, 6, 8, 5, 3, False),
    (1, 8, 2, 33, 33, 16, 64, True),  # G = 4, thin keys r < d_v
]


@pytest.mark.parametrize("case", CASES)
def test_backward_matches_autograd(case):
    B, Hq, Hkv, Sq, Sk, r, dv, causal = case
    q, k, v = rand((B, Hq, Sq, r), 1), rand((B, Hkv, Sk, r), 2), rand((B, Hkv, Sk, dv), 3)
    do = rand((B, Hq, Sq, dv), 4)
    scale = 0.7 / math.sqrt(r)
    dq, dk, dv_, lse = oracle.prefill_backward(q, k, v, do, causal=causal, scale=scale)
    qq, kk, vv = (t.clone().requires_grad_() for t in (q, k, v))
    o, lse_ref = textbook(qq, kk, vv, causal, scale)
    (o * do).sum().backward()
    for got, ref in ((dq, qq.grad), (dk, kk.grad), (dv_, vv.grad)):
        assert (got - ref).abs().max().item() <= 1e-12 * max(1.0, ref.abs().max().item())
    assert (lse - lse_ref.detach()).abs().max().item() <= 1e-12


@pytest.mark.parametrize("causal", [True, False])
def test_backward_matches_finite_differences_of_the_forward(causal):
    """d/dx of sum(O * W) by central differences of the forward oracle, for every
    entry of Q, K and V of a small GQA case."""
    B, Hq, Hkv, Sq, Sk, r, dv = 1, 4, 2, 4, 6, 3, 2
    q, k, v = rand((B, Hq, Sq, r), 11), rand((B, Hkv, Sk, r), 12), rand((B, Hkv, Sk, dv), 13)
    w = rand((B, Hq, Sq, dv), 14)
    scale = 1.3
    if causal:  # bottom-right needs Sq <= Sk: it holds
        pass
    dq, dk, dv_, _ = oracle.prefill_backward(q, k, v, w, causal=causal, scale=scale)
    eps = 1e-6

    def loss(qq, kk, vv):
        return float((oracle.prefill(qq, kk, vv, causal=causal, scale=scale) * w).sum())

    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv_)):
        flat = x.reshape(-1)
        for idx in range(flat.numel()):
            xp, xm = flat.clone(), flat.clone()
            xp[idx] += eps
            xm[idx] -= eps
            args = {"q": q, "k": k, "v": v}
            args[name] = xp.view_as(x)
            lp = loss(args["q"], args["k"], args["v"])
            args[name] = xm.view_as(x)
            lm = loss(args["q"], args["k"], args["v"])
            num = (lp - lm) / (2 * eps)
            assert abs(num - grad.reshape(-1)[idx].item()) <= 1e-7 * max(1.0, abs(num)), (name, idx)


def test_equal_value_rows_give_zero_query_and_key_gradients():
    """With every value row equal, O is that row whatever the scores, so the loss
    does not depend on Q or K; dV_j is the attention-weighted sum of dO rows."""
    B, Hq, Hkv, S, r, dv = 1, 4, 2, 12, 8, 6
    q, k = rand((B, Hq, S, r), 21), rand((B, Hkv, S, r), 22)
    row = rand((dv,), 23)
    v = row.expand(B, Hkv, S, dv).contiguous()
    do = rand((B, Hq, S, dv), 24)
    dq, dk, dv_, _ = oracle.prefill_backward(q, k, v, do, causal=True)
    assert dq.abs().max().item() <= 1e-13
    assert dk.abs().max().item() <= 1e-13
    # dV summed over keys equals dO summed over every row of the group (the weights of a row sum to 1)
    tot = dv_.sum(dim=2)
    ref = do.view(B, Hkv, Hq // Hkv, S, dv).sum(dim=(2, 3))
    assert (tot - ref).abs().max().item() <= 1e-12


def test_partial_rows_agree_with_the_full_gradients():
    B, Hq, Hkv, Sq, Sk, r, dv = 1, 4, 2, 40, 56, 8, 16
    q, k, v = rand((B, Hq, Sq, r), 31), rand((B, Hkv, Sk, r), 32), rand((B, Hkv, Sk, dv), 33)
    do = rand((B, Hq, Sq, dv), 34)
    full = oracle.prefill_backward(q, k, v, do, causal=True)
    lo = 25
    part = oracle.prefill_backward(q, k, v, do, causal=True, row_lo=lo)
    assert torch.equal(part[0][:, :, lo:], full[0][:, :, lo:])
    assert torch.equal(part[3][:, :, lo:], full[3][:, :, lo:])
    first_key = lo + (Sk - Sq)
    assert torch.equal(part[1][:, :, first_key:], full[1][:, :, first_key:])
    assert torch.equal(part[2][:, :, first_key:], full[2][:, :, first_key:])
    assert torch.isnan(part[0][:, :, :lo]).all()


def test_bf16_inputs_are_widened_exactly():
    B, Hq, Hkv, S, r, dv = 1, 2, 1, 10, 16, 32
    q, k, v = (rand(s, n, torch.bfloat16) for s, n in (((B, Hq, S, r), 41), ((B, Hkv, S, r), 42),
                                                         ((B, Hkv, S, dv), 43)))
    do = rand((B, Hq, S, dv), 44, torch.bfloat16)
    a = oracle.prefill_backward(q, k, v, do, causal=True)
    b = oracle.prefill_backward(q.double(), k.double(), v.double(), do.double(), causal=True)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_stored_output_enters_through_D_only():
    """With O given, D = rowsum(dO * O). With the exact forward output this is the
    default gradient; a perturbation Delta of O moves D_i by dO_i . Delta_i, which
    leaves dV unchanged and moves dQ_i by -scale * (dO_i . Delta_i) * sum_j P_ij k_j and
    dK_j by -scale * sum_i P_ij (dO_i . Delta_i) q_i (first order is exact: D enters
    linearly)."""
    B, Hq, Hkv, Sq, Sk, r, dv = 1, 4, 2, 9, 13, 4, 6
    q, k, v = rand((B, Hq, Sq, r), 51), rand((B, Hkv, Sk, r), 52), rand((B, Hkv, Sk, dv), 53)
    do = rand((B, Hq, Sq, dv), 54)
    scale = 0.6
    o = oracle.prefill(q, k, v, causal=True, scale=scale)
    base = oracle.prefill_backward(q, k, v, do, causal=True, scale=scale)
    same = oracle.prefill_backward(q, k, v, do, causal=True, scale=scale, o=o)
    for x, y in zip(base, same):
        assert (x - y).abs().max().item() <= 1e-12
    delta = 1e-2 * rand((B, Hq, Sq, dv), 55)
    moved = oracle.prefill_backward(q, k, v, do, causal=True, scale=scale, o=o + delta)
    dD = (do * delta).sum(-1)                                    # [B, Hq, Sq]
    G = Hq // Hkv
    kr = k.repeat_interleave(G, dim=1)
    s = (q @ kr.transpose(-1, -2)) * scale
    i = torch.arange(Sq).view(-1, 1)
    j = torch.arange(Sk).view(1, -1)
    p = torch.softmax(s.masked_fill(j > i + (Sk - Sq), float("-inf")), dim=-1)
    exp_dq = base[0] - scale * dD.unsqueeze(-1) * (p @ kr)
    exp_dk = base[1] - scale * ((p * dD.unsqueeze(-1)).transpose(-1, -2) @ q).view(B, Hkv, G, Sk, r).sum(2)
    assert (moved[0] - exp_dq).abs().max().item() <= 1e-12
    assert (moved[1] - exp_dk).abs().max().item() <= 1e-12
    assert (moved[2] - base[2]).abs().max().item() <= 1e-12
    assert (moved[0] - base[0]).abs().max().item() > 1e-4      # the perturbation is visible
