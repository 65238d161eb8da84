"""The offline thin-key conversion (Sec. 2.3, Eq. 5-7) on the CPU.

Pinned by what the mathematics fixes, independently of the oracle: a key
projection of rank at most r is reproduced exactly (logits to rounding), r =
d_head is exact for any weights, a full-rank projection stays within the
Eckart-Young bound, and the query heads of a group share their KV head's
factor. The oracle's own factorisation (a separate implementation) must give
the same logits, which are invariant to the SVD's sign choices."""
import math

import pytest
import torch

from oracle import factored
from paper_2603_04427_amd import factor
from synth import normal, stream_key


def draw(tensor: int, *shape, std=1.0):
    n = math.prod(shape)
    return (normal(stream_key(41, tensor), n).view(*shape) * std).to(torch.float64)


def layer(d_model, d_head, h_q, h_kv, key_rank=None):
    """Seeded W_Q [d_model, h_q d_head] and W_K [d_model, h_kv d_head]; with
    key_rank, every key head is a product of two random factors of that rank."""
    w_q = draw(0, d_model, h_q * d_head, std=d_model ** -0.5)
    if key_rank is None:
        w_k = draw(1, d_model, h_kv * d_head, std=d_model ** -0.5)
    else:
        a = draw(2, h_kv, d_model, key_rank, std=d_model ** -0.5)
        b = draw(3, h_kv, key_rank, d_head, std=key_rank ** -0.5)
        w_k = torch.matmul(a, b).permute(1, 0, 2).reshape(d_model, h_kv * d_head)
    return w_q, w_k


def logits(x, w_q, w_k, h_q, h_kv):
    """[h_q, n, n] logits x W_Q^(h) (x W_K^(h // G))^T."""
    n = x.shape[0]
    q = (x @ w_q).reshape(n, h_q, -1).permute(1, 0, 2)
    k = (x @ w_k).reshape(n, h_kv, -1).permute(1, 0, 2)
    k = k.repeat_interleave(h_q // h_kv, dim=0)
    return q @ k.transpose(1, 2)


@pytest.mark.parametrize("h_q,h_kv", [(4, 4), (8, 2)])
def test_exact_rank_keys_keep_every_logit(h_q, h_kv):
    d_model, d_head, r = 96, 32, 8
    w_q, w_k = layer(d_model, d_head, h_q, h_kv, key_rank=r)
    x = draw(4, 40, d_model)
    q_t, k_t, sigma = factor.factor_layer(w_q, w_k, r, h_q, h_kv)
    assert q_t.shape == (d_model, h_q * r) and k_t.shape == (d_model, h_kv * r)
    ref = logits(x, w_q, w_k, h_q, h_kv)
    got = logits(x, q_t, k_t, h_q, h_kv)
    assert (got - ref).abs().max() <= 1e-10 * ref.abs().max()
    # the key heads really have rank r: the tail of their spectra is rounding
    assert sigma[:, r:].max() <= 1e-12 * sigma[:, 0].max()


def test_full_width_is_exact_for_any_weights():
    d_model, d_head, h = 64, 16, 3
    w_q, w_k = layer(d_model, d_head, h, h)
    x = draw(5, 30, d_model)
    q_t, k_t, _ = factor.factor_layer(w_q, w_k, d_head, h, h)
    ref = logits(x, w_q, w_k, h, h)
    assert (logits(x, q_t, k_t, h, h) - ref).abs().max() <= 1e-10 * ref.abs().max()


def test_full_rank_keys_stay_within_eckart_young():
    d_model, d_head, h, r = 80, 32, 2, 6
    w_q, w_k = layer(d_model, d_head, h, h)
    x = draw(6, 50, d_model)
    q_t, k_t, sigma = factor.factor_layer(w_q, w_k, r, h, h)
    err = (logits(x, q_t, k_t, h, h) - logits(x, w_q, w_k, h, h)).abs()
    assert err.max() > 1e-3  # truncation really changed something
    for hh in range(h):
        bound = factor.logit_error_bound(x, w_q[:, hh * d_head:(hh + 1) * d_head], x, float(sigma[hh, r]))
        assert bool((err[hh] <= bound * (1 + 1e-12) + 1e-12).all())


def test_group_shares_its_key_factor():
    """Query heads 0 and 1 of a group with identical W_Q blocks get identical thin blocks."""
    d_model, d_head, r = 48, 16, 4
    w_q, w_k = layer(d_model, d_head, 4, 2)
    w_q[:, d_head:2 * d_head] = w_q[:, :d_head]
    q_t, _, _ = factor.factor_layer(w_q, w_k, r, 4, 2)
    assert torch.equal(q_t[:, :r], q_t[:, r:2 * r])


@pytest.mark.parametrize("h_q,h_kv,r", [(4, 4, 8), (8, 2, 5)])
def test_logits_match_the_oracle_factorisation(h_q, h_kv, r):
    d_model, d_head = 72, 24
    w_q, w_k = layer(d_model, d_head, h_q, h_kv)
    x = draw(7, 25, d_model)
    q_t, k_t, sigma = factor.factor_layer(w_q, w_k, r, h_q, h_kv)
    qh = [w_q[:, i * d_head:(i + 1) * d_head].numpy() for i in range(h_q)]
    kh = [w_k[:, i * d_head:(i + 1) * d_head].numpy() for i in range(h_kv)]
    qo, ko, so = factored.thin_projections(x.numpy(), qh, kh, r, group=h_q // h_kv)
    ref = torch.from_numpy(qo) @ torch.from_numpy(ko).repeat_interleave(h_q // h_kv, dim=0).transpose(1, 2)
    got = logits(x, q_t, k_t, h_q, h_kv)
    assert (got - ref).abs().max() <= 1e-10 * ref.abs().max()
    assert torch.allclose(sigma, torch.from_numpy(__import__("numpy").stack(so)), rtol=1e-12, atol=1e-12)


def test_transposed_weights_layout():
    """The projection kernel takes each weight transposed ([n_heads * width, d_model])
    in bf16: entry (n, k) is w[k, n] rounded once."""
    w = draw(9, 32, 4 * 8).to(torch.float32)
    wt = factor.transposed_bf16(w, "cpu")
    assert wt.shape == (32, 32) and wt.dtype == torch.bfloat16 and wt.is_contiguous()
    for n, k in ((0, 0), (5, 17), (31, 3), (12, 31)):
        assert wt[n, k].item() == w[k, n].to(torch.bfloat16).item()


def test_oracle_projection_is_head_major():
    """oracle.factored.project_heads against explicit loops (pure Python sums) on a
    tiny input: Y[b, h, s, w] = sum_k X[b, s, k] W[k, h * width + w]."""
    import numpy as np
    B, S, d_model, heads, width = 2, 3, 5, 2, 4
    x = draw(12, B, S, d_model).numpy()
    w = draw(13, d_model, heads * width).numpy()
    y = factored.project_heads(x, w, heads)
    assert y.shape == (B, heads, S, width)
    for b in range(B):
        for h in range(heads):
            for s_ in range(S):
                for c in range(width):
                    want = math.fsum(float(x[b, s_, k]) * float(w[k, h * width + c]) for k in range(d_model))
                    assert abs(y[b, h, s_, c] - want) <= 1e-13 * (1 + abs(want))
    assert np.array_equal(factored.project_heads(x[:, :0], w, heads), np.zeros((B, heads, 0, width)))


def test_bad_arguments_are_rejected():
    w_q, w_k = layer(32, 8, 4, 2)
    with pytest.raises(ValueError):
        factor.factor_layer(w_q, w_k, 9, 4, 2)       # rank above d_head
    with pytest.raises(ValueError):
        factor.factor_layer(w_q, w_k, 4, 4, 3)       # heads do not group
    with pytest.raises(ValueError):
        factor.factor_layer(w_q[:, :30], w_k, 4, 4, 2)  # width not a multiple of the heads
