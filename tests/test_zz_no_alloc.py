"""tk_attn_decode_noalloc (the library's fixed scratch instead of a caller's
workspace) against tk_attn_decode, through the C ABI: two calls in a row, the
second with a smaller input, each bitwise equal to tk_attn_decode's output (same
kernels, same split) and within the bf16 gate of the oracle. Both calls split
the context, so the scratch's partials and arrival counters are used, and the
second call finds what the first left there."""
import pytest
import torch

from gpu_cases import decode_oracle, device, gate, say
from synth import WORKLOADS, make_decode, with_shape

pytestmark = pytest.mark.gpu


def run_both(spec, structured):
    from paper_2603_04427_amd import tk_attn_decode, tk_attn_decode_noalloc, tk_attn_decode_workspace_bytes
    dev = device()
    d = make_decode(spec, structured=structured)
    g = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in d.items()}
    kw = dict(max_ctx=spec.ctx, scale=spec.softmax_scale, k_scale=g["k_scale"], block_table=g["block_table"],
              block_size=spec.block_size if spec.paged else 0)
    say(f"decode noalloc {spec} structured={structured}")
    out = torch.full((spec.batch, spec.h_q, spec.d_v), 7.0, dtype=torch.bfloat16, device=dev)
    got = tk_attn_decode_noalloc(g["q"], g["k"], g["v"], g["ctx_lens"], O=out, **kw)
    ws = torch.zeros(tk_attn_decode_workspace_bytes(spec.batch, spec.h_q, spec.h_kv, spec.ctx, spec.d_v),
                     dtype=torch.uint8, device=dev)
    want = tk_attn_decode(g["q"], g["k"], g["v"], g["ctx_lens"], workspace=ws, **kw)
    torch.cuda.synchronize()
    assert got.data_ptr() == out.data_ptr()
    assert torch.equal(got, want), f"{spec.name}: not bitwise equal to tk_attn_decode"
    gate(got, decode_oracle(d, spec), spec.k_dtype, spec.name)


def test_two_calls_second_smaller():
    big = WORKLOADS["mistral_decode_b16"]                       # 2 splits of 2048 tokens
    small = with_shape(big, config_id=1500, batch=3, ctx=3000, ctx_lens=(3000, 1234, 0))   # 12 splits
    run_both(big, structured=False)
    run_both(small, structured=True)


def test_paged_quantised_after_the_others():
    spec = with_shape(WORKLOADS["mistral_decode_b16"], config_id=1501, batch=2, ctx=2048, ctx_lens=(2048, 777),
                      k_dtype="fp8", paged=True, block_size=128)
    run_both(spec, structured=True)
    run_both(with_shape(spec, batch=1, ctx=1024, ctx_lens=(1000,)), structured=False)
