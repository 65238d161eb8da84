"""Decode calls captured into a HIP graph replay to the eager result.

The C ABI promises that calls can be captured: sequence lengths live on the
device, the host sizes only the grid, and the split-K arrival counters are
reset by the kernel itself (no memset is recorded). The graph here holds
several calls on rotated cache copies sharing one workspace; it is replayed
several times with eager calls and synchronisations in between, and every
replay must equal the eager output bit for bit (the kernel is deterministic)."""
import pytest
import torch

from gpu_cases import device, say
from paper_2603_04427_amd import prepare_decode, tk_attn_decode_workspace_bytes
from synth import WORKLOADS, make_decode, with_shape

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,kw", [
    ("mistral_decode_b16", dict(batch=4, ctx=3000, ctx_lens=(3000, 1, 0, 1777))),
    ("longctx_paged_decode", dict(batch=2, ctx=4096, ctx_lens=(4096, 2500))),
    ("fp8key_decode", dict(batch=3, ctx=2048, ctx_lens=(2048, 700, 1))),
])
def test_captured_decode_replays_bitwise(name, kw):
    dev = device()
    spec = with_shape(WORKLOADS[name], **kw)
    d = make_decode(spec, device=dev, structured=True)
    ws = torch.zeros(tk_attn_decode_workspace_bytes(spec.batch, spec.h_q, spec.h_kv, spec.ctx, spec.d_v),
                     dtype=torch.uint8, device=dev)
    copies = [(d["k"], d["v"], d["k_scale"])]
    for _ in range(2):
        copies.append((d["k"].clone(), d["v"].clone(), None if d["k_scale"] is None else d["k_scale"].clone()))

    def calls(outs):
        return [prepare_decode(d["q"], k, v, d["ctx_lens"], max_ctx=spec.ctx, scale=spec.softmax_scale, k_scale=ks,
                               block_table=d["block_table"], block_size=spec.block_size if spec.paged else 0,
                               workspace=ws, O=o) for (k, v, ks), o in zip(copies, outs)]

    say(f"graph capture {spec}")
    eager_out = [torch.empty(spec.batch, spec.h_q, spec.d_v, dtype=torch.bfloat16, device=dev) for _ in copies]
    eager = calls(eager_out)
    for c in eager:
        c()
    torch.cuda.synchronize()
    ref = [o.clone() for o in eager_out]

    graph_out = [torch.empty_like(o) for o in eager_out]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture's side stream
        for c in calls(graph_out):
            c()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for c in calls(graph_out):
            c()
    torch.cuda.synchronize()

    for rep in range(4):
        for o in graph_out:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (o, r) in enumerate(zip(graph_out, ref)):
            assert torch.equal(o, r), f"replay {rep}, call {i}"
        for c in eager:  # eager work on the same workspace between replays
            c()
        torch.cuda.synchronize()
