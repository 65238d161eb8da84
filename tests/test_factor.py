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


def test_project_thin_is_head_major():
    B, S, d_model, h_q, h_kv, r, d_v = 2, 7, 32, 4, 2, 8, 16
    x = draw(8, B, S, d_model).to(torch.float32)
    w_q = draw(9, d_model, h_q * r).to(torch.float32)
    w_k = draw(10, d_model, h_kv * r).to(torch.float32)
    w_v = draw(11, d_model, h_kv * d_v).to(torch.float32)
    q, k, v = factor.project_thin(x, w_q, w_k, w_v, h_q, h_kv, dtype=torch.float32)
    assert q.shape == (B, h_q, S, r) and k.shape == (B, h_kv, S, r) and v.shape == (B, h_kv, S, d_v)
    assert q.is_contiguous() and k.is_contiguous() and v.is_contiguous()
    assert torch.allclose(q[1, 3, 5], x[1, 5] @ w_q[:, 3 * r:4 * r], rtol=1e-5, atol=1e-5)
    assert torch.allclose(v[0, 1, 2], x[0, 2] @ w_v[:, d_v:2 * d_v], rtol=1e-5, atol=1e-5)


def test_bad_arguments_are_rejected():
    w_q, w_k = layer(32, 8, 4, 2)
    with pytest.raises(ValueError):
        factor.factor_layer(w_q, w_k, 9, 4, 2)       # rank above d_head
    with pytest.raises(ValueError):
        factor.factor_layer(w_q, w_k, 4, 4, 3)       # heads do not group
    with pytest.raises(ValueError):
        factor.factor_layer(w_q[:, :30], w_k, 4, 4, 2)  # width not a multiple of the heads
