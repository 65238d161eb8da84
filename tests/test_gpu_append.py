"""Cache-append parity on the GPU: tk_cache_append against the oracle on the same
seeded inputs, bit for bit (bf16 rows are copies; E4M3 codes and scales are
integer and fp32 decisions taken in the same precision on both sides), over the
whole cache so that untouched rows are checked too; then append followed by
decode against the oracle's decode of the oracle's cache."""
import math

import pytest
import torch

from gpu_cases import device, gate, say
from oracle import append as oa
from oracle import oracle as orc
from synth import normal, permutation, stream_key

pytestmark = pytest.mark.gpu


def bf16(shape, key, amp=1.0, device="cpu"):
    n = math.prod(shape)
    return (normal(stream_key(key, 0), n, device=device).view(*shape) * amp).to(torch.bfloat16)


def fill_bytes(shape, key, dtype):
    """A cache filled with arbitrary finite bytes (so that untouched rows are checked)."""
    n = math.prod(shape)
    x = normal(stream_key(key, 1), n).view(*shape)
    if dtype == torch.uint8:
        return (x.abs() * 37).to(torch.int32).remainder(126).to(torch.uint8)
    return x.to(dtype)


def run(B, Hkv, T, r, dv, kdt, paged, positions, bs=16, mb=None, key=0, bad=None):
    """kdt: "bf16", "fp8" (True) or "int4" key cache."""
    from paper_2603_04427_amd import tk_cache_append
    dev = device()
    k = bf16((B, Hkv, T, r), 100 + key, amp=2.0)
    v = bf16((B, Hkv, T, dv), 200 + key)
    pos = torch.tensor(positions, dtype=torch.int32)
    if paged:
        mb = mb or 8
        nblk = B * mb
        table = permutation(stream_key(300 + key, 3), nblk).view(B, mb).to(torch.int32)
        if bad is not None:
            table[bad] = nblk + 3
        shape_k, shape_v = (nblk, Hkv, bs, r), (nblk, Hkv, bs, dv)
    else:
        table = None
        cap = mb or 64
        shape_k, shape_v = (B, Hkv, cap, r), (B, Hkv, cap, dv)
    kdt = {True: "fp8", False: "bf16"}.get(kdt, kdt)
    fp8 = kdt != "bf16"
    if kdt == "int4":
        shape_k = (*shape_k[:3], r // 2)
    kc = fill_bytes(shape_k, 400 + key, torch.uint8 if fp8 else torch.bfloat16)
    vc = fill_bytes(shape_v, 500 + key, torch.bfloat16)
    ks = normal(stream_key(600 + key, 1), math.prod(shape_k[:3])).view(*shape_k[:3]).abs() if fp8 else None
    ref = oa.cache_append(k, v, pos, kc, vc, k_scale=ks, block_table=table, block_size=bs if paged else 0,
                          k_format=kdt)
    gk, gv = kc.to(dev), vc.to(dev)
    gs = None if ks is None else ks.to(dev)
    say(f"append B={B} Hkv={Hkv} T={T} r={r} dv={dv} keys={kdt} paged={paged} pos={positions}")
    tk_cache_append(k.to(dev), v.to(dev), pos.to(dev), gk, gv, k_scale=gs,
                    block_table=None if table is None else table.to(dev), block_size=bs if paged else 0)
    torch.cuda.synchronize()
    assert torch.equal(gk.cpu(), ref[0]), "key cache differs"
    assert torch.equal(gv.cpu(), ref[1]), "value cache differs"
    if fp8:
        assert torch.equal(gs.cpu(), ref[2]), "scales differ"


@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("dv", [64, 128])
@pytest.mark.parametrize("kdt", ["bf16", "fp8", "int4"])
@pytest.mark.parametrize("paged", [False, True])
def test_sweep_bitexact(r, dv, kdt, paged):
    run(3, 2, 37, r, dv, kdt, paged, positions=[0, 50, 90], key=r + dv)


@pytest.mark.parametrize("T,positions", [(1, [0, 5, 127]), (1, [-1, 128, 64]), (300, [-7, 0, 100]),
                                          (128, [0, 0, 0])])
def test_positions_and_capacity(T, positions):
    run(3, 4, T, 32, 128, True, True, positions, bs=16, mb=8, key=T)  # capacity 128 per sequence
    run(3, 4, T, 32, 128, False, False, positions, mb=128, key=T + 1)


def test_bad_block_entry_skipped():
    run(2, 2, 64, 32, 128, True, True, [0, 0], bs=16, mb=4, bad=(1, 2))


def test_prefill_scale_append_bitexact():
    """The 8192-token, 4 x 8 KV-head shape of the prefill workload, bf16, fp8 and 4-bit keys."""
    for kdt in ("bf16", "fp8", "int4"):
        run(4, 8, 8192, 32, 128, kdt, False, [0, 0, 0, 0], mb=8192, key=11)


def test_append_then_decode():
    """A cache built by appends (a prefill chunk, then one decode token per sequence)
    decoded on the GPU equals the oracle's decode of the oracle-built cache."""
    from paper_2603_04427_amd import tk_attn_decode, tk_cache_append
    dev = device()
    B, Hq, Hkv, r, dv, bs, mb = 3, 8, 2, 32, 128, 64, 8
    for kdt in ("bf16", "fp8", "int4"):
        fp8 = kdt != "bf16"
        lens = [300, 511, 1]
        T0 = max(lens) - 1
        k0, v0 = bf16((B, Hkv, T0, r), 700, amp=2.0), bf16((B, Hkv, T0, dv), 701)
        k1, v1 = bf16((B, Hkv, 1, r), 702, amp=2.0), bf16((B, Hkv, 1, dv), 703)
        q = bf16((B, Hq, r), 704, amp=2.0)
        table = permutation(stream_key(705, 3), B * mb).view(B, mb).to(torch.int32)
        kc = torch.zeros(B * mb, Hkv, bs, r // 2 if kdt == "int4" else r,
                         dtype=torch.uint8 if fp8 else torch.bfloat16)
        vc = torch.zeros(B * mb, Hkv, bs, dv, dtype=torch.bfloat16)
        ks = torch.ones(B * mb, Hkv, bs) if fp8 else None
        pos0 = torch.zeros(B, dtype=torch.int32)
        pos1 = torch.tensor([L - 1 for L in lens], dtype=torch.int32)
        rk, rv, rs = oa.cache_append(k0, v0, pos0, kc, vc, ks, table, bs, k_format=kdt)
        rk, rv, rs = oa.cache_append(k1, v1, pos1, rk, rv, rs, table, bs, k_format=kdt)
        gk, gv, gs, gt = kc.to(dev), vc.to(dev), None if ks is None else ks.to(dev), table.to(dev)
        say(f"append+decode keys={kdt}")
        tk_cache_append(k0.to(dev), v0.to(dev), pos0.to(dev), gk, gv, gs, gt, bs)
        tk_cache_append(k1.to(dev), v1.to(dev), pos1.to(dev), gk, gv, gs, gt, bs)
        lens_t = torch.tensor(lens, dtype=torch.int32)
        out = tk_attn_decode(q.to(dev), gk, gv, lens_t.to(dev), max_ctx=max(lens), k_scale=gs, block_table=gt,
                             block_size=bs)
        torch.cuda.synchronize()
        # oracle: gather the logical cache through the table and decode it
        logical_k = torch.stack([torch.cat([rk[int(table[b, j])] for j in range(mb)], dim=1) for b in range(B)])
        logical_v = torch.stack([torch.cat([rv[int(table[b, j])] for j in range(mb)], dim=1) for b in range(B)])
        logical_s = None if rs is None else torch.stack(
            [torch.cat([rs[int(table[b, j])] for j in range(mb)], dim=1) for b in range(B)])
        ref = orc.decode(q, orc.Int4(logical_k) if kdt == "int4" else logical_k, logical_v, lens_t,
                         k_scale=logical_s)
        gate(out, ref, kdt, f"append+decode keys={kdt}")
