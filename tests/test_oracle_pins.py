"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Every check here compares the oracle with something other than itself: a
library routine (torch SDPA in fp64, numpy's SVD), an independent pure-Python
brute force, a closed form, or an invariant of the definition (Sec. 2.1, Eq. 4;
Sec. 2.3, Eq. 6-7). Each is chosen so that a plausible slip in the oracle (a
dropped term, a wrong sign, a transposed operand, an off-by-one in the causal
bound, a wrong GQA map or page index) fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import brute, factored
from oracle import oracle as orc
from synth import normal, stream_key

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def rnd(tag, *shape, dtype=torch.float64):
    n = int(np.prod(shape))
    return normal(stream_key(900, tag), n).view(*shape).to(dtype)


def bottom_right_mask(sq, sk):
    i = torch.arange(sq).view(-1, 1)
    j = torch.arange(sk).view(1, -1)
    return j <= i + (sk - sq)


def sdpa(q, k, v, causal, scale):
    """Library reference: torch SDPA in fp64 with GQA expanded by repeat_interleave."""
    G = q.shape[1] // k.shape[1]
    k = k.double().repeat_interleave(G, dim=1)
    v = v.double().repeat_interleave(G, dim=1)
    mask = bottom_right_mask(q.shape[2], k.shape[2]) if causal else None
    return F.scaled_dot_product_attention(q.double(), k, v, attn_mask=mask, scale=scale)


# ----------------------------------------------------------------- P1: reduction to MHA

def test_reduces_to_standard_mha_sdpa():
    """r = d_v = d_head: the method is standard multi-head attention (Sec. 2.1)."""
    n, d_model, H, dh = 96, 768, 12, 64
    x = rnd(1, n, d_model) / math.sqrt(d_model)
    wq, wk, wv = rnd(2, H, d_model, dh), rnd(3, H, d_model, dh), rnd(4, H, d_model, dh)
    q = torch.einsum("nd,hde->hne", x, wq).unsqueeze(0)
    k = torch.einsum("nd,hde->hne", x, wk).unsqueeze(0)
    v = torch.einsum("nd,hde->hne", x, wv).unsqueeze(0)
    for causal in (False, True):
        o = orc.prefill(q, k, v, causal=causal, scale=1 / math.sqrt(dh))
        ref = sdpa(q, k, v, causal, 1 / math.sqrt(dh))
        assert (o - ref).abs().max().item() < 1e-12
        # the textbook formula with an explicit additive mask
        s = q @ k.transpose(-1, -2) / math.sqrt(dh)
        if causal:
            s = s.masked_fill(~bottom_right_mask(n, n), float("-inf"))
        text = torch.softmax(s, dim=-1) @ v
        assert (o - text).abs().max().item() < 1e-12


@pytest.mark.parametrize("r,dv,hq,hkv,sq,sk,causal", [
    (16, 64, 4, 4, 33, 33, True),
    (32, 128, 8, 2, 40, 40, True),
    (8, 24, 6, 3, 17, 29, True),     # bottom-right aligned, S_q < S_k
    (32, 128, 4, 1, 21, 50, False),
    (128, 64, 2, 2, 9, 9, True),
])
def test_thin_keys_match_sdpa(r, dv, hq, hkv, sq, sk, causal):
    """r != d_v and GQA: SDPA accepts E != Ev; the oracle must agree."""
    q, k, v = rnd(10, 2, hq, sq, r), rnd(11, 2, hkv, sk, r), rnd(12, 2, hkv, sk, dv)
    o = orc.prefill(q, k, v, causal=causal, scale=0.3)
    ref = sdpa(q, k, v, causal, 0.3)
    assert (o - ref).abs().max().item() < 1e-12
    if hq != hkv:
        g = F.scaled_dot_product_attention(q, k, v, scale=0.3, enable_gqa=True,
                                           attn_mask=bottom_right_mask(sq, sk) if causal else None)
        assert (o - g).abs().max().item() < 1e-12


# ----------------------------------------------------------------- P2: factored keys

def test_query_absorption_exact_rank():
    """W_K of rank r: truncated SVD, absorbing B^T into W_Q reproduces logits and outputs (Eq. 6-7)."""
    n, d_model, H, dh, r = 64, 768, 12, 64, 16
    x = rnd(20, n, d_model).numpy() / math.sqrt(d_model)
    wq = [rnd(21 + h, d_model, dh).numpy() for h in range(H)]
    wk = [(rnd(40 + h, d_model, r) @ rnd(60 + h, r, dh)).numpy() / math.sqrt(r) for h in range(H)]
    wv = [rnd(80 + h, d_model, dh).numpy() for h in range(H)]
    qt, kt, sv = factored.thin_projections(x, wq, wk, r)
    for h in range(H):
        a, b, s = factored.factor_key_projection(wk[h], r)
        assert np.linalg.norm(a @ b - wk[h]) / np.linalg.norm(wk[h]) < 1e-12
        assert s[r] / s[0] < 1e-13          # exact rank r
        full = (x @ wq[h]) @ (x @ wk[h]).T
        thin = qt[h] @ kt[h].T
        assert np.abs(thin - full).max() / np.abs(full).max() < 1e-10
    q_full = torch.from_numpy(np.stack([x @ w for w in wq]))[None]
    k_full = torch.from_numpy(np.stack([x @ w for w in wk]))[None]
    v = torch.from_numpy(np.stack([x @ w for w in wv]))[None]
    # unscaled logits are what absorption preserves; the same scale on both sides
    for causal in (True, False):
        o_full = orc.prefill(q_full, k_full, v, causal=causal, scale=0.125)
        o_thin = orc.prefill(torch.from_numpy(qt)[None], torch.from_numpy(kt)[None], v,
                             causal=causal, scale=0.125)
        assert (o_full - o_thin).abs().max().item() < 1e-12


def test_query_absorption_eckart_young_bound():
    """Full-rank W_K: |q.k - q'.k'| <= ||x_i W_Q|| sigma_{r+1} ||x_j|| (spectral norm of the residual)."""
    n, d_model, dh, r = 48, 256, 64, 8
    x = rnd(100, n, d_model).numpy()
    wq, wk = rnd(101, d_model, dh).numpy(), rnd(102, d_model, dh).numpy()
    qt, kt, sv = factored.thin_projections(x, [wq], [wk], r)
    err = np.abs(qt[0] @ kt[0].T - (x @ wq) @ (x @ wk).T)
    bound = np.linalg.norm(x @ wq, axis=1)[:, None] * sv[0][r] * np.linalg.norm(x, axis=1)[None, :]
    assert (err <= bound * (1 + 1e-9) + 1e-9).all()
    assert err.max() > 0.01 * bound.max()   # the bound is not vacuous here


# ----------------------------------------------------------------- P3: invariants

def test_softmax_rows_sum_to_one_and_affine_in_v():
    q, k = rnd(110, 1, 4, 37, 16), rnd(111, 1, 2, 37, 16)
    ones = torch.ones(1, 2, 37, 64, dtype=torch.float64)
    o = orc.prefill(q, k, ones, causal=True, scale=0.7)
    assert (o - 1).abs().max().item() < 1e-14
    v = rnd(112, 1, 2, 37, 64)
    a, c = -2.5, 0.75
    o1 = orc.prefill(q, k, v, causal=True, scale=0.7)
    o2 = orc.prefill(q, k, a * v + c, causal=True, scale=0.7)
    assert (o2 - (a * o1 + c)).abs().max().item() < 1e-13


def test_causal_future_perturbation_is_invisible():
    q, k, v = rnd(120, 1, 2, 40, 32), rnd(121, 1, 2, 40, 32), rnd(122, 1, 2, 40, 128)
    o = orc.prefill(q, k, v, causal=True)
    i = 23
    k2, v2 = k.clone(), v.clone()
    k2[:, :, i + 1:] = rnd(123, 1, 2, 40 - i - 1, 32) * 7
    v2[:, :, i + 1:] = -100.0
    o2 = orc.prefill(q, k2, v2, causal=True)
    assert torch.equal(o[:, :, :i + 1], o2[:, :, :i + 1])
    assert not torch.equal(o[:, :, i + 1:], o2[:, :, i + 1:])


def test_gqa_equals_repeated_kv_mha_bitwise():
    q, k, v = rnd(130, 2, 8, 19, 16), rnd(131, 2, 2, 19, 16), rnd(132, 2, 2, 19, 24)
    o = orc.prefill(q, k, v, causal=True)
    o2 = orc.prefill(q, k.repeat_interleave(4, 1), v.repeat_interleave(4, 1), causal=True)
    assert torch.equal(o, o2)
    # a wrong map (h % Hkv instead of h / G) gives a different answer
    o3 = orc.prefill(q, k.repeat(1, 4, 1, 1), v.repeat(1, 4, 1, 1), causal=True)
    assert not torch.allclose(o, o3)


def test_paged_equals_contiguous_bitwise():
    B, Hq, Hkv, ctx, r, dv, bs = 3, 4, 2, 40, 16, 32, 8
    q, k, v = rnd(140, B, Hq, r), rnd(141, B, Hkv, ctx, r), rnd(142, B, Hkv, ctx, dv)
    lens = torch.tensor([40, 17, 0], dtype=torch.int32)
    mb = ctx // bs
    perm = torch.randperm(B * mb, generator=torch.Generator().manual_seed(5))
    table = perm.view(B, mb).to(torch.int32)
    kp = torch.zeros(B * mb, Hkv, bs, r, dtype=torch.float64)
    vp = torch.zeros(B * mb, Hkv, bs, dv, dtype=torch.float64)
    for b in range(B):
        for t in range(ctx):
            kp[table[b, t // bs], :, t % bs] = k[b, :, t]
            vp[table[b, t // bs], :, t % bs] = v[b, :, t]
    o = orc.decode(q, k, v, lens)
    o2 = orc.decode(q, kp, vp, lens, block_table=table, block_size=bs)
    assert torch.equal(o, o2)
    assert (o[2] == 0).all()     # empty context writes zeros


def test_last_prefill_row_equals_decode():
    q, k, v = rnd(150, 2, 8, 30, 32), rnd(151, 2, 2, 30, 32), rnd(152, 2, 2, 30, 128)
    o = orc.prefill(q, k, v, causal=True)
    d = orc.decode(q[:, :, -1].contiguous(), k, v, torch.tensor([30, 30], dtype=torch.int32))
    assert torch.equal(o[:, :, -1], d)


# ----------------------------------------------------------------- P4: closed forms

def test_closed_forms_row0_and_uniform_query():
    q, k, v = rnd(160, 1, 3, 25, 16), rnd(161, 1, 3, 25, 16), rnd(162, 1, 3, 25, 20)
    o = orc.prefill(q, k, v, causal=True)
    assert torch.equal(o[:, :, 0], v[:, :, 0])       # row 0 sees only key 0
    oz = orc.prefill(torch.zeros_like(q), k, v, causal=True)
    mean = torch.cumsum(v, dim=2) / torch.arange(1, 26, dtype=torch.float64).view(1, 1, -1, 1)
    assert (oz - mean).abs().max().item() < 1e-14


def test_needle_bound():
    """One key with logit margin D over n-1 others: |O - v_needle| <= (n-1) e^-D 2 max|V|."""
    n, r, dv = 300, 32, 64
    k = rnd(170, 1, 1, n, r)
    k = k / k.norm(dim=-1, keepdim=True)
    v = rnd(171, 1, 1, n, dv)
    j = 123
    q = (12.0 * k[:, :, j]).contiguous()
    s = (k[0, 0] @ q[0, 0])
    margin = (s[j] - torch.cat([s[:j], s[j + 1:]]).max()).item()
    o = orc.decode(q, k, v, torch.tensor([n], dtype=torch.int32), scale=1.0)
    bound = (n - 1) * math.exp(-margin) * 2 * v.abs().max().item()
    assert margin > 3
    assert (o[0, 0] - v[0, 0, j]).abs().max().item() <= bound


def test_large_logits_select_the_arg_max():
    """Logits thousands apart: softmax is one-hot on the best key and stays finite."""
    n, r, dv = 50, 16, 12
    k, v = rnd(175, 1, 2, n, r), rnd(176, 1, 2, n, dv)
    q = 500.0 * rnd(177, 1, 4, r)
    o = orc.decode(q, k, v, torch.tensor([n], dtype=torch.int32), scale=1.0)
    for h in range(4):
        j = int(torch.argmax(k[0, h // 2] @ q[0, h]))
        assert torch.isfinite(o[0, h]).all()
        assert torch.equal(o[0, h], v[0, h // 2, j])


def test_copy_back_pattern():
    """Exp. 1's copy-back offset: q_i proportional to k_{i-8} attends (almost) only to i-8."""
    S, r, dv = 64, 16, 8
    k = rnd(180, 1, 1, S, r)
    k = k / k.norm(dim=-1, keepdim=True)
    v = rnd(181, 1, 1, S, dv)
    q = torch.zeros(1, 1, S, r, dtype=torch.float64)
    q[:, :, 8:] = 40.0 * k[:, :, :-8]
    o = orc.prefill(q, k, v, causal=True, scale=1.0)
    assert (o[0, 0, 8:] - v[0, 0, :-8]).abs().max().item() < 0.05


# ----------------------------------------------------------------- P5: brute force

def nested(x):
    return x.tolist()


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Sk,r,dv,causal", [
    (1, 1, 1, 1, 1, 1, 1, True),
    (1, 2, 1, 5, 5, 2, 5, True),
    (2, 4, 2, 9, 9, 3, 1, True),
    (1, 4, 1, 3, 8, 16, 5, True),
    (1, 2, 2, 7, 4, 16, 64, False),
    (1, 1, 1, 6, 6, 16, 64, True),
])
def test_brute_force_prefill(B, Hq, Hkv, Sq, Sk, r, dv, causal):
    q, k, v = rnd(200, B, Hq, Sq, r), rnd(201, B, Hkv, Sk, r), rnd(202, B, Hkv, Sk, dv)
    scale = 1.0 / math.sqrt(r)
    o = orc.prefill(q, k, v, causal=causal, scale=scale)
    ref = torch.tensor(brute.attention(nested(q), nested(k), nested(v), scale, causal), dtype=torch.float64)
    assert (o - ref).abs().max().item() < 1e-13


@pytest.mark.parametrize("bs", [1, 2, 4])
@pytest.mark.parametrize("G", [1, 2, 4])
def test_brute_force_paged_decode(bs, G):
    B, Hkv, r, dv = 3, 2, 3, 5
    Hq = Hkv * G
    lens = [9, 4, 1]
    mb = -(-9 // bs)
    nblk = B * mb
    q = rnd(210, B, Hq, r)
    kp, vp = rnd(211, nblk, Hkv, bs, r), rnd(212, nblk, Hkv, bs, dv)
    perm = torch.randperm(nblk, generator=torch.Generator().manual_seed(bs * 10 + G))
    table = perm.view(B, mb).to(torch.int32)
    o = orc.decode(q, kp, vp, torch.tensor(lens, dtype=torch.int32), scale=0.6,
                   block_table=table, block_size=bs)
    ref = brute.decode(nested(q), nested(kp), nested(vp), lens, 0.6, table.tolist(), bs)
    assert (o - torch.tensor(ref, dtype=torch.float64)).abs().max().item() < 1e-13


def test_brute_force_fp8_keys():
    """E4M3 keys with per-(token, head) scales; the brute force dequantises with torch's own cast."""
    B, Hq, Hkv, ctx, r, dv = 2, 4, 2, 7, 16, 6
    kf = rnd(220, B, Hkv, ctx, r).float()
    amax = kf.abs().amax(-1)
    sc = (amax / 448).float()
    codes = (kf / sc.unsqueeze(-1)).to(torch.float8_e4m3fn)
    khat = codes.to(torch.float64) * sc.double().unsqueeze(-1)
    q, v = rnd(221, B, Hq, r), rnd(222, B, Hkv, ctx, dv)
    lens = torch.tensor([7, 3], dtype=torch.int32)
    o = orc.decode(q, codes.view(torch.uint8), v, lens, scale=0.25, k_scale=sc)
    ref = brute.decode(nested(q), nested(khat), nested(v), [7, 3], 0.25)
    assert (o - torch.tensor(ref, dtype=torch.float64)).abs().max().item() < 1e-13


def test_brute_force_int4_keys():
    """4-bit integer keys (excess-8 nibbles, low nibble first) with per-(token, head)
    scales; codes and packing written here independently, brute force on c * scale."""
    import random
    B, Hq, Hkv, ctx, r, dv = 2, 4, 2, 7, 16, 6
    rng = random.Random(240)
    codes = [[[[rng.randint(-7, 7) for _ in range(r)] for _ in range(ctx)] for _ in range(Hkv)] for _ in range(B)]
    packed = torch.tensor([[[[(row[2 * j] + 8) | ((row[2 * j + 1] + 8) << 4) for j in range(r // 2)]
                             for row in head] for head in seq] for seq in codes], dtype=torch.uint8)
    sc = torch.rand(B, Hkv, ctx, generator=torch.Generator().manual_seed(241)).float() + 0.1
    khat = [[[[c * float(sc[b, g, t]) for c in codes[b][g][t]] for t in range(ctx)] for g in range(Hkv)]
            for b in range(B)]
    q, v = rnd(242, B, Hq, r), rnd(243, B, Hkv, ctx, dv)
    o = orc.decode(q, orc.Int4(packed), v, torch.tensor([7, 3], dtype=torch.int32), scale=0.25, k_scale=sc)
    ref = brute.decode(nested(q), khat, nested(v), [7, 3], 0.25)
    assert (o - torch.tensor(ref, dtype=torch.float64)).abs().max().item() < 1e-13


def test_int4_decode_every_nibble():
    for n in range(16):
        row = torch.tensor([n | ((15 - n) << 4)], dtype=torch.uint8)
        assert orc.int4_value(row, 0) == n - 8 and orc.int4_value(row, 1) == 7 - n


def test_bf16_and_f32_inputs_widen_exactly():
    q, k, v = rnd(230, 1, 2, 11, 16), rnd(231, 1, 2, 11, 16), rnd(232, 1, 2, 11, 32)
    for dt in (torch.bfloat16, torch.float32):
        qd, kd, vd = q.to(dt), k.to(dt), v.to(dt)
        o = orc.prefill(qd, kd, vd, causal=True)
        o64 = orc.prefill(qd.double(), kd.double(), vd.double(), causal=True)
        assert torch.equal(o, o64)


# ----------------------------------------------------------------- P6: E4M3 decode

def test_e4m3_decode_all_codes_vs_torch():
    codes = torch.arange(256, dtype=torch.uint8)
    lib_vals = codes.view(torch.float8_e4m3fn).to(torch.float64)
    for c in range(256):
        mine = orc.e4m3_value(c)
        ref = lib_vals[c].item()
        if math.isnan(ref):
            assert math.isnan(mine), c
        else:
            assert mine == ref, (c, mine, ref)
    assert orc.e4m3_value(0x7E) == 448.0 and orc.e4m3_value(0x01) == 2.0 ** -9
