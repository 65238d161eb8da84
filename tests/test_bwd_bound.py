"""CPU checks of the end-to-end backward bars (bwd_bound).

* Every end-to-end case the GPU tests run is admissible: an all-zero gradient,
  and the exact gradient with one row's sign flipped, fail its bars, while the
  exact gradient passes.
* The isolated backward gate (rel-L2 1e-2 and max-abs 2e-2 max|ref|) fails an
  all-zero gradient by construction; checked on one strongly peaked case.
* The bound covers a rounding model of the kernels' arithmetic (fp32 scores,
  weights rounded to bf16 before both the value product and the row sum, the
  output rounded to bf16, D from that rounded output, dS rounded to bf16) on
  every fuzzed case, against the exact gradient. On the strongly peaked
  copy-back inputs the same model lands far outside the isolated bars, which is
  why the end-to-end tests widen them by the bound and keep to admissible
  inputs."""
import math

import pytest
import torch

from bwd_bound import admissible, bars, check, exact_terms
from oracle import oracle as orc
from synth import PrefillSpec, make_prefill, make_prefill_grad, with_shape
from test_gpu_backward import BASE, gate_grad
from test_gpu_fuzz import backward_cases, backward_inputs


def end_to_end_cases():
    out = []
    for spec in backward_cases():
        out.append((spec.name, spec, backward_inputs(spec)))
    for structured in (False, True):
        for r, dv in ((32, 128), (64, 128), (128, 64)):
            spec = with_shape(BASE, config_id=1200 + r, r=r, d_v=dv, h_q=8, h_kv=2, seq_q=333, seq_k=333)
            p = make_prefill(spec, structured=structured, needle_logit=6.0)
            out.append((f"e2e_r{r}_dv{dv}_s{int(structured)}", spec,
                        (p["q"], p["k"], p["v"], make_prefill_grad(spec))))
    return out


CASES = end_to_end_cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_cases_admissible_and_discriminating(case):
    name, spec, (q, k, v, do) = case
    exact, bound = exact_terms(q, k, v, do, spec.causal, spec.softmax_scale)
    for what, e, b in zip(("dQ", "dK", "dV"), exact, bound):
        assert admissible(e, b), f"{name} {what}"
        assert check(e, e, b)[0], f"{name} {what}: the exact gradient fails"
        assert not check(torch.zeros_like(e), e, b)[0], f"{name} {what}: zero passes"
        flipped = e.clone()
        row = e.flatten(0, -2).norm(dim=-1).argmax()
        flipped.view(-1, e.shape[-1])[row] *= -1
        assert not check(flipped, e, b)[0], f"{name} {what}: a sign-flipped row passes"


def test_isolated_gate_rejects_zero_on_peaked_rows():
    spec = with_shape(BASE, config_id=932, r=32, d_v=128)
    p = make_prefill(spec, structured=True)
    do = make_prefill_grad(spec)
    o = orc.prefill(p["q"], p["k"], p["v"], causal=True, scale=spec.softmax_scale).to(torch.bfloat16)
    ref = orc.prefill_backward(p["q"], p["k"], p["v"], do, causal=True, scale=spec.softmax_scale, o=o)
    for r in ref[:3]:
        gate_grad(r.float(), r, "reference against itself")
        with pytest.raises(AssertionError):
            gate_grad(torch.zeros_like(r), r, "zero")


def _bf(t):
    return t.to(torch.bfloat16).float()


def rounding_model(q, k, v, do, causal, scale):
    """The kernels' rounding points, in torch fp32 (a model, not the kernels)."""
    q, k, v, do = (t.float() for t in (q, k, v, do))
    B, Hq, Sq, r = q.shape
    Hkv, Sk = k.shape[1], k.shape[2]
    G = Hq // Hkv
    kx, vx = k.repeat_interleave(G, 1), v.repeat_interleave(G, 1)
    s = torch.matmul(q, kx.transpose(-1, -2))
    if causal:
        i = torch.arange(Sq).view(-1, 1) + (Sk - Sq)
        s = s.masked_fill(torch.arange(Sk).view(1, -1) > i, float("-inf"))
    c = scale * math.log2(math.e)
    m = s.amax(-1, keepdim=True)
    p = _bf(torch.exp2(s * c - m * c))
    l = p.sum(-1, keepdim=True)
    o = _bf(torch.matmul(p, vx) / l)
    lse = m * scale + torch.log(l)
    pp = torch.exp(s * scale - lse)
    dv = torch.matmul(_bf(pp).transpose(-1, -2), do).view(B, Hkv, G, Sk, -1).sum(2)
    ds = _bf(pp * (torch.matmul(do, vx.transpose(-1, -2)) - (do * o).sum(-1, keepdim=True)))
    dq = scale * torch.matmul(ds, kx)
    dk = (scale * torch.matmul(ds.transpose(-1, -2), q)).view(B, Hkv, G, Sk, -1).sum(2)
    return dq, dk, dv


@pytest.mark.parametrize("spec", backward_cases(), ids=lambda s: s.name)
def test_bound_covers_the_rounding_model(spec):
    q, k, v, do = backward_inputs(spec)
    exact, bound = exact_terms(q, k, v, do, spec.causal, spec.softmax_scale)
    for what, g, e, b in zip(("dQ", "dK", "dV"), rounding_model(q, k, v, do, spec.causal, spec.softmax_scale),
                             exact, bound):
        ok, msg = check(g, e, b)
        assert ok, f"{spec.name} {what}: {msg}"


def test_peaked_rows_need_the_bound():
    """Strongly peaked copy-back rows: the rounding model misses the exact dQ by
    more than the isolated bars allow, but stays inside the widened bars."""
    spec = PrefillSpec("peaked", 3208, 1, 4, 1, 14, 302, 128, 64, dtype="bf16", amp=0.5)
    p = make_prefill(spec, structured=True)
    q, k, v, do = p["q"], p["k"], p["v"], make_prefill_grad(spec)
    exact, bound = exact_terms(q, k, v, do, True, spec.softmax_scale)
    dq = rounding_model(q, k, v, do, True, spec.softmax_scale)[0].double()
    assert (dq - exact[0]).norm() > 1e-2 * exact[0].norm()
    assert check(dq, exact[0], bound[0])[0]
    assert not admissible(exact[0], bound[0])
    assert bars(exact[0], bound[0])[1] > exact[0].norm()
