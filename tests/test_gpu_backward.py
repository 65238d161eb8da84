"""Prefill backward parity on the GPU against the fp64 oracle on the same seeded
inputs.

* The training forward (tk_attn_prefill_lse): O bitwise equal to tk_attn_prefill,
  and lse within 4e-3 of the oracle's (the kernel sums bf16-rounded weights, a
  relative error below 2^-9 in the sum, so below 2^-8 in its logarithm).
* The backward kernels in isolation: Q, K, V, dO seeded; O the oracle's forward
  output rounded to bf16 and lse the oracle's log-sum-exp, handed to both sides
  (the oracle then forms D = rowsum(dO * O) from the same O). Every output against
  the oracle: relative L2 <= 1e-2 and max-abs <= 2e-2 * max|ref| per tensor. The
  kernels round one operand of each product (P or dS) to bf16 (relative error
  up to 2^-8) and each output once more, so errors of a few 2^-9 relative per
  entry are expected.
* End to end (GPU forward, then backward) against the exact gradient, with
  i.i.d. and moderately peaked inputs: the same bars widened by the derived
  bound on what the stored bf16 output changes through D = rowsum(dO * O)
  (bwd_bound), on inputs where that bound leaves the test discriminating (an
  all-zero gradient fails). With sharply peaked rows dP - D cancels and that
  rounding term is the whole of dQ and dK; the isolated tests cover that regime,
  with the same bf16 O given to both sides.
* The Mistral 8192-token shape in the benchmark's launch configuration: the last
  rows of every sequence (all heads), with the key gradients those rows
  determine, end to end against the exact gradient; the dV column sums of every
  KV head (they equal the dO sums of its rows, since each row's weights sum to
  one); bitwise reproducibility."""
import pytest
import torch

from bwd_bound import admissible, check, exact_terms
from gpu_cases import device, say
from oracle import oracle as orc
from synth import WORKLOADS, PrefillSpec, make_prefill, make_prefill_grad, with_shape

pytestmark = pytest.mark.gpu

BASE = PrefillSpec("bwd", 900, 1, 4, 2, 300, 300, 32, 128, dtype="bf16", amp=0.5)


def gate_grad(out, ref, what, trel=1e-2, tmax=2e-2):
    o = out.detach().double().cpu()
    assert torch.isfinite(o).all(), f"{what}: non-finite output"
    scale = ref.abs().max().item()
    mx = (o - ref).abs().max().item()
    rel = ((o - ref).norm() / ref.norm().clamp(min=1e-30)).item()
    assert rel <= trel, f"{what}: rel-L2 {rel:.3e} > {trel:.0e} (max-abs {mx:.2e}, max|ref| {scale:.2e})"
    assert mx <= tmax * max(scale, 1e-30), f"{what}: max-abs {mx:.3e} > {tmax:.0e} * {scale:.2e} (rel {rel:.2e})"
    return mx, rel


def inputs(spec, structured=False):
    p = make_prefill(spec, structured=structured)
    return p["q"], p["k"], p["v"], make_prefill_grad(spec)


def gpu_backward(q, k, v, o, do, lse, spec, dev):
    from paper_2603_04427_amd import tk_attn_prefill_backward
    g = [t.to(dev).contiguous() for t in (q, k, v, o, do, lse)]
    return tk_attn_prefill_backward(*g, causal=spec.causal, scale=spec.softmax_scale)


def isolated(spec, structured):
    dev = device()
    q, k, v, do = inputs(spec, structured)
    o = orc.prefill(q, k, v, causal=spec.causal, scale=spec.softmax_scale).to(torch.bfloat16)
    ref = orc.prefill_backward(q, k, v, do, causal=spec.causal, scale=spec.softmax_scale, o=o)
    say(f"backward isolated {spec} structured={structured}")
    got = gpu_backward(q, k, v, o, do, ref[3].float(), spec, dev)
    torch.cuda.synchronize()
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref[:3]):
        gate_grad(g, r, f"{name} {spec} structured={structured}")


@pytest.mark.parametrize("structured", [False, True])
@pytest.mark.parametrize("r", [32, 64, 128])
@pytest.mark.parametrize("dv", [64, 128])
def test_backward_widths(r, dv, structured):
    isolated(with_shape(BASE, config_id=900 + r + dv, r=r, d_v=dv), structured)


SHAPES = [  # (B, Hq, Hkv, Sq, Sk, causal)
    (1, 1, 1, 1, 1, True),
    (1, 2, 1, 31, 31, True),
    (2, 4, 4, 33, 33, True),
    (1, 8, 2, 100, 100, False),
    (1, 4, 2, 64, 200, True),     # bottom-right: 64 new rows after 136 cached keys
    (1, 4, 1, 5, 300, True),
    (2, 6, 2, 257, 257, True),    # G = 3
    (1, 16, 2, 130, 130, True),   # G = 8
    (1, 2, 2, 65, 129, False),
    (1, 4, 1, 129, 129, True),    # one row past a 128-key block
]


@pytest.mark.parametrize("shape", SHAPES)
def test_backward_shapes_and_masks(shape):
    B, Hq, Hkv, Sq, Sk, causal = shape
    spec = with_shape(BASE, config_id=1000, batch=B, h_q=Hq, h_kv=Hkv, seq_q=Sq, seq_k=Sk, causal=causal)
    isolated(spec, structured=True)


def forward_lse(q, k, v, spec, dev):
    from paper_2603_04427_amd import tk_attn_prefill_lse
    return tk_attn_prefill_lse(q.to(dev), k.to(dev), v.to(dev), causal=spec.causal, scale=spec.softmax_scale)


@pytest.mark.parametrize("r,dv", [(32, 128), (64, 64), (128, 128)])
@pytest.mark.parametrize("shape", [(1, 4, 2, 300, 300, True), (1, 4, 2, 70, 200, True), (2, 2, 1, 90, 90, False)])
def test_forward_lse(r, dv, shape):
    from paper_2603_04427_amd import tk_attn_prefill
    dev = device()
    B, Hq, Hkv, Sq, Sk, causal = shape
    spec = with_shape(BASE, config_id=1100 + r, batch=B, h_q=Hq, h_kv=Hkv, seq_q=Sq, seq_k=Sk, causal=causal,
                      r=r, d_v=dv)
    for structured in (False, True):
        q, k, v, do = inputs(spec, structured)
        say(f"forward lse {spec} structured={structured}")
        o, lse = forward_lse(q, k, v, spec, dev)
        o_plain = tk_attn_prefill(q.to(dev), k.to(dev), v.to(dev), causal=causal, scale=spec.softmax_scale)
        torch.cuda.synchronize()
        assert torch.equal(o, o_plain)
        ref = orc.prefill_backward(q, k, v, do, causal=causal, scale=spec.softmax_scale)[3]
        err = (lse.double().cpu() - ref).abs().max().item()
        assert err <= 4e-3, f"lse max-abs {err:.2e}"


def gate_end_to_end(got, exact, bound, what):
    for name, g, e, b in zip(("dQ", "dK", "dV"), got, exact, bound):
        assert admissible(e, b), f"{what} {name}: the bound does not discriminate on these inputs"
        ok, msg = check(g, e, b)
        assert ok, f"{what} {name}: {msg}"
        say(f"  {name} {msg}")


@pytest.mark.parametrize("structured", [False, True])
@pytest.mark.parametrize("r,dv", [(32, 128), (64, 128), (128, 64)])
def test_end_to_end(r, dv, structured):
    dev = device()
    spec = with_shape(BASE, config_id=1200 + r, r=r, d_v=dv, h_q=8, h_kv=2, seq_q=333, seq_k=333)
    p = make_prefill(spec, structured=structured, needle_logit=6.0)
    q, k, v, do = p["q"], p["k"], p["v"], make_prefill_grad(spec)
    exact, bound = exact_terms(q, k, v, do, True, spec.softmax_scale)
    say(f"backward end to end {spec} structured={structured}")
    o, lse = forward_lse(q, k, v, spec, dev)
    got = gpu_backward(q, k, v, o, do, lse, spec, dev)
    torch.cuda.synchronize()
    gate_end_to_end(got, exact, bound, f"{spec} structured={structured}")


def test_mid_size_every_output():
    """2048 tokens, 4 query heads over one KV head, thin keys: every output end to end."""
    dev = device()
    spec = PrefillSpec("bwd_s2048", 1300, 1, 4, 1, 2048, 2048, 32, 128, dtype="bf16", amp=0.5)
    q, k, v, do = inputs(spec)
    exact, bound = exact_terms(q, k, v, do, True, spec.softmax_scale)
    say(f"backward end to end {spec}")
    o, lse = forward_lse(q, k, v, spec, dev)
    got = gpu_backward(q, k, v, o, do, lse, spec, dev)
    torch.cuda.synchronize()
    gate_end_to_end(got, exact, bound, spec.name)


def test_mistral_s8192_sampled():
    """Batch 4, 32/8 heads, 8192 tokens, r 32, d_v 128: the whole backward on the GPU
    (the benchmark's launch), the last 96 rows of every sequence (all heads) and
    the keys only those rows see, end to end against the exact gradient."""
    dev = device()
    spec = WORKLOADS["mistral_prefill_s8192"]
    B, S = spec.batch, spec.seq_q
    p = make_prefill(spec, device=dev)
    do = make_prefill_grad(spec, device=dev)
    say(f"backward full {spec.name}")
    o, lse = forward_lse(p["q"], p["k"], p["v"], spec, dev)
    got = gpu_backward(p["q"], p["k"], p["v"], o, do, lse, spec, dev)
    torch.cuda.synchronize()
    again = gpu_backward(p["q"], p["k"], p["v"], o, do, lse, spec, dev)
    torch.cuda.synchronize()
    for a, b in zip(got, again):
        assert torch.equal(a, b), "backward is not bitwise reproducible"
    lo = S - 96
    for b in range(B):
        sl = slice(b, b + 1)
        # the last rows alone, bottom-right aligned, sit at their own positions
        exact, bound = exact_terms(p["q"][sl, :, lo:].cpu(), p["k"][sl].cpu(), p["v"][sl].cpu(),
                                   do[sl, :, lo:].cpu(), True, spec.softmax_scale)
        ref = orc.prefill_backward(p["q"][sl, :, lo:].cpu(), p["k"][sl].cpu(), p["v"][sl].cpu(),
                                   do[sl, :, lo:].cpu(), causal=True, scale=spec.softmax_scale)
        mine = (got[0][sl, :, lo:], got[1][sl, :, lo:], got[2][sl, :, lo:])
        gate_end_to_end(mine, [t[:, :, lo:] if i else t for i, t in enumerate(exact)],
                        [t[:, :, lo:] if i else t for i, t in enumerate(bound)], f"rows >= {lo} b={b}")
        err = (lse[sl, :, lo:].double().cpu() - ref[3]).abs().max().item()
        assert err <= 4e-3, f"lse b={b}: {err:.2e}"
    # every KV head: sum over keys of dV = sum over the group's rows of dO
    G = spec.h_q // spec.h_kv
    col = got[2].double().sum(dim=2)                                           # [B, Hkv, dv]
    want = do.double().view(B, spec.h_kv, G, S, -1).sum(dim=(2, 3))
    bound = do.double().abs().view(B, spec.h_kv, G, S, -1).sum(dim=(2, 3))
    assert ((col - want).abs() <= 1e-2 * bound).all()


def test_empty_rows_zero_key_gradients_and_errors():
    from paper_2603_04427_amd import TkError, tk_attn_prefill_backward, tk_attn_prefill_backward_workspace_bytes
    dev = device()
    bf = dict(dtype=torch.bfloat16, device=dev)
    q = torch.empty(1, 4, 0, 32, **bf)
    o = torch.empty(1, 4, 0, 128, **bf)
    k = torch.randn(1, 2, 70, 32, **bf)
    v = torch.randn(1, 2, 70, 128, **bf)
    lse = torch.empty(1, 4, 0, dtype=torch.float32, device=dev)
    dk = torch.full_like(k, 7.0)
    dv = torch.full_like(v, 7.0)
    say("backward with no query rows")
    tk_attn_prefill_backward(q, k, v, o, o, lse, dK=dk, dV=dv)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dk) == 0 and torch.count_nonzero(dv) == 0
    # host-side rejections: nothing is launched
    q16 = torch.randn(1, 2, 8, 16, **bf)
    k16 = torch.randn(1, 1, 8, 16, **bf)
    v16 = torch.randn(1, 1, 8, 64, **bf)
    o16 = torch.randn(1, 2, 8, 64, **bf)
    l16 = torch.zeros(1, 2, 8, dtype=torch.float32, device=dev)
    with pytest.raises(TkError, match="unsupported"):
        tk_attn_prefill_backward(q16, k16, v16, o16, o16, l16)
    ws = torch.empty(tk_attn_prefill_backward_workspace_bytes(1, 4, 300) - 256, dtype=torch.uint8, device=dev)
    q32 = torch.randn(1, 4, 300, 32, **bf)
    k32 = torch.randn(1, 2, 300, 32, **bf)
    v32 = torch.randn(1, 2, 300, 128, **bf)
    o32 = torch.randn(1, 4, 300, 128, **bf)
    l32 = torch.zeros(1, 4, 300, dtype=torch.float32, device=dev)
    with pytest.raises(TkError, match="workspace"):
        tk_attn_prefill_backward(q32, k32, v32, o32, o32, l32, workspace=ws)
