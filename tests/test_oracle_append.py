"""Pins of the cache-append oracle against facts fixed outside it: rows read back
by position, the paged/contiguous equivalence, a hand-computed E4M3 row, the
quantisation error bound, and a brute-force nearest-code search."""
import math

import pytest
import torch

from oracle import append as oa
from oracle import oracle as orc
from synth import normal, permutation, stream_key


def bf16(shape, key, amp=1.0):
    n = math.prod(shape)
    return (normal(stream_key(key, 0), n).view(*shape) * amp).to(torch.bfloat16)


def test_bf16_rows_land_at_their_positions_and_nothing_else_moves():
    B, Hkv, T, r, dv, cap = 3, 2, 5, 16, 64, 12
    k, v = bf16((B, Hkv, T, r), 1), bf16((B, Hkv, T, dv), 2)
    kc, vc = bf16((B, Hkv, cap, r), 3), bf16((B, Hkv, cap, dv), 4)
    pos = torch.tensor([0, 9, -2], dtype=torch.int32)  # sequence 1 overflows, sequence 2 starts before 0
    k2, v2, _ = oa.cache_append(k, v, pos, kc, vc)
    for b in range(B):
        for p in range(cap):
            t = p - int(pos[b])
            if 0 <= t < T:
                assert torch.equal(k2[b, :, p], k[b, :, t]) and torch.equal(v2[b, :, p], v[b, :, t])
            else:
                assert torch.equal(k2[b, :, p], kc[b, :, p]) and torch.equal(v2[b, :, p], vc[b, :, p])


def test_paged_equals_contiguous_through_the_table():
    B, Hkv, T, r, dv, bs, mb = 2, 3, 40, 32, 64, 16, 4
    k, v = bf16((B, Hkv, T, r), 5), bf16((B, Hkv, T, dv), 6)
    pos = torch.tensor([3, 20], dtype=torch.int32)
    kc, vc = torch.zeros(B, Hkv, bs * mb, r, dtype=torch.bfloat16), torch.zeros(B, Hkv, bs * mb, dv, dtype=torch.bfloat16)
    kc2, vc2, _ = oa.cache_append(k, v, pos, kc, vc)
    table = permutation(stream_key(7, 3), B * mb).view(B, mb).to(torch.int32)
    kp = torch.zeros(B * mb, Hkv, bs, r, dtype=torch.bfloat16)
    vp = torch.zeros(B * mb, Hkv, bs, dv, dtype=torch.bfloat16)
    kp2, vp2, _ = oa.cache_append(k, v, pos, kp, vp, block_table=table, block_size=bs)
    for b in range(B):
        for p in range(bs * mb):
            blk, slot = int(table[b, p // bs]), p % bs
            assert torch.equal(kp2[blk, :, slot], kc2[b, :, p]) and torch.equal(vp2[blk, :, slot], vc2[b, :, p])


def test_bad_table_entry_is_skipped():
    k, v = bf16((1, 1, 4, 16), 8), bf16((1, 1, 4, 64), 9)
    kp, vp = torch.zeros(2, 1, 4, 16, dtype=torch.bfloat16), torch.zeros(2, 1, 4, 64, dtype=torch.bfloat16)
    table = torch.tensor([[1, 5]], dtype=torch.int32)  # second block outside [0, 2)
    kp2, vp2, _ = oa.cache_append(k, v, torch.tensor([2], dtype=torch.int32), kp, vp, block_table=table, block_size=4)
    assert torch.equal(kp2[1, 0, 2:], k[0, 0, :2]) and torch.equal(kp2[0], kp[0]) and torch.equal(kp2[1, 0, :2], kp[1, 0, :2])


def test_e4m3_hand_computed_row():
    """k = (1, -2, 0.5, 0, ...): max|k| = 2, scale = 2/448, k/scale = (224, -448, 112, 0):
    224 = 1.75 * 2^7 -> exponent field 14, mantissa 6: 0x76; -448 -> 0xFE; 112 -> 0x6E."""
    k = torch.zeros(1, 1, 1, 16, dtype=torch.bfloat16)
    k[0, 0, 0, :3] = torch.tensor([1.0, -2.0, 0.5])
    kc = torch.zeros(1, 1, 4, 16, dtype=torch.uint8)
    ks = torch.zeros(1, 1, 4, dtype=torch.float32)
    v = torch.zeros(1, 1, 1, 64, dtype=torch.bfloat16)
    kc2, _, ks2 = oa.cache_append(k, v, torch.tensor([1], dtype=torch.int32), kc, torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16), k_scale=ks)
    assert kc2[0, 0, 1, :4].tolist() == [0x76, 0xFE, 0x6E, 0x00]
    assert ks2[0, 0, 1].item() == pytest.approx(2.0 / 448.0, rel=1e-7)
    assert float(torch.tensor(2.0, dtype=torch.float32) / torch.tensor(448.0)) == ks2[0, 0, 1].item()


def test_zero_row_scale_one():
    codes, scale = oa.quantize_rows(torch.zeros(3, 32))
    assert torch.all(codes == 0) and torch.all(scale == 1.0)


def test_quantisation_error_bound_and_peak_code():
    k = bf16((64, 32), 10, amp=3.0).to(torch.float32)
    codes, scale = oa.quantize_rows(k)
    dec = torch.tensor([[orc.e4m3_value(int(c)) for c in row] for row in codes.tolist()], dtype=torch.float64)
    kh = dec * scale.double().unsqueeze(-1)
    bound = torch.maximum(k.double().abs() * 2.0 ** -4, scale.double().unsqueeze(-1) * 2.0 ** -10)
    assert torch.all((kh - k.double()).abs() <= bound)
    # the largest magnitude of every row encodes as +-448
    peak = k.abs().argmax(dim=-1)
    assert torch.all((codes.gather(1, peak.unsqueeze(1)).squeeze(1) & 0x7F) == 0x7E)


def test_rounding_matches_brute_force_nearest_even_code():
    """For fp32 values near every E4M3 midpoint, the oracle's code is the nearest
    finite code, ties going to the even code (brute force over the code table)."""
    table = [(c, orc.e4m3_value(c)) for c in range(0x7F)]  # non-negative finite codes 0 .. 0x7E
    vals = []
    for (c0, a), (c1, b) in zip(table, table[1:]):
        mid = (a + b) / 2
        for x in (mid, math.nextafter(mid, 0), math.nextafter(mid, 1e9), a, b):
            vals.append(x)
    x = torch.tensor(vals, dtype=torch.float32)
    scale = torch.ones(1)
    got = (x / scale).to(torch.float8_e4m3fn).view(torch.uint8).tolist()
    for xv, g in zip(x.tolist(), got):
        best = min(table, key=lambda cv: (abs(cv[1] - xv), cv[0] & 1))
        assert g == best[0], (xv, g, best)


def test_int4_hand_computed_row():
    """k = (1, -2, 0.5, 0.15, 0, ...): max|k| = 2 and scale = fp32(2/7), which lies just
    above 2/7, so in fp32 k/scale = (3.4999998, -6.9999998, 1.7499999, 0.525): the
    codes are (3, -7, 2, 1), not the 4 an exact 3.5 would give; stored excess-8 as
    nibbles (11, 1, 10, 9): bytes 0x1B, 0x9A."""
    k = torch.zeros(1, 16)
    k[0, :4] = torch.tensor([1.0, -2.0, 0.5, 0.15])
    packed, scale = oa.quantize_rows_int4(k)
    assert packed[0, :3].tolist() == [0x1B, 0x9A, 0x88]
    assert scale.item() == float(torch.tensor(2.0) / torch.tensor(7.0))


def test_int4_round_half_even_and_bound():
    """Ties go to the even integer (2.5 -> 2, 3.5 -> 4, -0.5 -> 0); every decoded entry
    lies within scale / 2 of the input, and the peak entry codes to +-7."""
    x = torch.tensor([[7.0, 2.5, 3.5, -0.5, 0.5, -2.5, 6.5, -6.5]])
    packed, scale = oa.quantize_rows_int4(x)
    assert scale.item() == 1.0
    c = [int(orc.int4_value(packed[0], i)) for i in range(8)]
    assert c == [7, 2, 4, 0, 0, -2, 6, -6]
    k = (normal(stream_key(12, 0), 64 * 32).view(64, 32) * 3).float()
    packed, scale = oa.quantize_rows_int4(k)
    dec = torch.tensor([[orc.int4_value(packed[i], j) for j in range(32)] for i in range(64)], dtype=torch.float64)
    err = (dec * scale.double().unsqueeze(-1) - k.double()).abs()
    assert torch.all(err <= scale.double().unsqueeze(-1) / 2 * (1 + 1e-6))
    peak = k.abs().argmax(dim=-1)
    assert torch.all(dec.gather(1, peak.unsqueeze(1)).abs() == 7)
