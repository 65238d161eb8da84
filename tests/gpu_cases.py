"""Shared helpers for the GPU parity tests: device checks, calls through the
binding, oracle references and the error gates.

Gates (max-abs against the fp64 oracle on the same inputs): 1e-4 for fp32
outputs, 2e-2 for bf16 outputs, 5e-2 with fp8 or 4-bit keys. Because i.i.d. inputs give
near-uniform attention and small outputs, a relative L2 gate is applied too
(1e-5 fp32, 1e-2 otherwise), and the structured inputs make outputs O(1)."""
from __future__ import annotations

import sys

import pytest
import torch

from oracle import oracle as orc

TOL = {"f32": (1e-4, 1e-5), "bf16": (2e-2, 1e-2), "fp8": (5e-2, 1e-2), "int4": (5e-2, 1e-2)}


def device():
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    return torch.device("cuda", 0)


def say(msg: str):
    """Name the case before a GPU step (flushed, so it survives a crash)."""
    print(msg, flush=True)
    sys.stdout.flush()


def errors(out: torch.Tensor, ref: torch.Tensor):
    o = out.detach().double().cpu()
    d = (o - ref).abs()
    rel = (o - ref).norm() / ref.norm().clamp(min=1e-30)
    return d.max().item(), rel.item()


def gate(out, ref, kind: str, what: str = ""):
    mx, rel = errors(out, ref)
    tmax, trel = TOL[kind]
    assert torch.isfinite(out.detach().double().cpu()).all(), f"{what}: non-finite output"
    assert mx <= tmax, f"{what}: max-abs {mx:.3e} > {tmax:.1e} (rel-L2 {rel:.2e})"
    assert rel <= trel, f"{what}: rel-L2 {rel:.3e} > {trel:.1e} (max-abs {mx:.2e})"
    return mx, rel


def decode_on_gpu(d, spec, dev, **kw):
    from paper_2603_04427_amd import tk_attn_decode
    g = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in d.items()}
    return tk_attn_decode(g["q"], g["k"], g["v"], g["ctx_lens"], max_ctx=spec.ctx, scale=spec.softmax_scale,
                          k_scale=g["k_scale"], block_table=g["block_table"],
                          block_size=spec.block_size if spec.paged else 0, **kw)


def decode_oracle(d, spec, batches=None):
    """fp64 oracle on the logical (contiguous) cache; ``batches`` selects sequences."""
    q, k, v, ks, lens = d["q"], d["k_logical"], d["v_logical"], d["k_scale_logical"], d["ctx_lens"]
    if batches is not None:
        idx = torch.tensor(batches)
        q, k, v, lens = q[idx], k[idx], v[idx], lens.cpu()[idx]
        ks = None if ks is None else ks[idx]
    k = k.cpu()
    if getattr(spec, "k_dtype", "bf16") == "int4":
        k = orc.Int4(k)
    return orc.decode(q.cpu(), k, v.cpu(), lens.cpu(), scale=spec.softmax_scale,
                      k_scale=None if ks is None else ks.cpu())


def prefill_on_gpu(p, spec, dev):
    from paper_2603_04427_amd import tk_attn_prefill
    return tk_attn_prefill(p["q"].to(dev), p["k"].to(dev), p["v"].to(dev), causal=spec.causal,
                           scale=spec.softmax_scale)


def prefill_oracle(p, spec):
    return orc.prefill(p["q"].cpu(), p["k"].cpu(), p["v"].cpu(), causal=spec.causal, scale=spec.softmax_scale)


def prefill_rows_oracle(p, spec, b: int, rows):
    """Oracle for selected query rows of sequence b, all heads: row i of a causal
    prefill is a decode over keys 0..i + (Sk - Sq). The sequence's own K and V
    serve every row as one cache page of Sk tokens (block table all zeros), so
    nothing is copied per row."""
    q = p["q"][b, :, rows].permute(1, 0, 2).contiguous().cpu()   # [n, Hq, r]
    n = len(rows)
    k = p["k"][b:b + 1].cpu().contiguous()                       # one page [1, Hkv, Sk, r]
    v = p["v"][b:b + 1].cpu().contiguous()
    off = spec.seq_k - spec.seq_q
    lens = torch.tensor([i + off + 1 if spec.causal else spec.seq_k for i in rows], dtype=torch.int32)
    table = torch.zeros(n, 1, dtype=torch.int32)
    return orc.decode(q, k, v, lens, scale=spec.softmax_scale, block_table=table,
                      block_size=spec.seq_k)                      # [n, Hq, dv]
