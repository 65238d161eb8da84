"""Seeded random shapes against the oracle: the combinations the parametrised
sweeps do not cross.

* decode: key format (bf16, E4M3, 4-bit) x contiguous or paged (64-256-token
  blocks) x GQA group 1-8 x r x d_v x ragged lengths (empty sequences included);
* prefill: bf16 or fp32 x head counts and groups x r x d_v x causal (with
  bottom-right alignment) or not x lengths up to a few hundred;
* backward: the same for the bf16 training step, run end to end (GPU forward,
  then backward) against the exact fp64 gradient, on i.i.d. inputs and on
  moderately peaked copy-back inputs (planted logit about 6, so that the
  gradient does not cancel to nothing). The bars widen the isolated backward's
  by the derived bound on the stored bf16 output's effect through D
  (bwd_bound); every case is checked to be admissible, i.e. an all-zero
  gradient fails it.

Every case is drawn from a fixed seed, so the set is the same on every run; the
case is printed before its GPU call. Gates as everywhere else (gpu_cases)."""
import random

import pytest
import torch

from bwd_bound import admissible, check, exact_terms
from gpu_cases import decode_on_gpu, decode_oracle, device, gate, prefill_on_gpu, prefill_oracle, say
from synth import DecodeSpec, PrefillSpec, make_decode, make_prefill, make_prefill_grad

pytestmark = pytest.mark.gpu


def decode_cases(n=24, seed=26034427):
    rng = random.Random(seed)
    out = []
    for i in range(n):
        h_kv = rng.choice([1, 2, 3])
        G = rng.choice([1, 2, 3, 4, 8])
        B = rng.randint(1, 4)
        ctx = rng.randint(1, 2500)
        lens = tuple(rng.choice([0, ctx, rng.randint(1, ctx)]) for _ in range(B))
        out.append(DecodeSpec(f"fuzz_decode_{i}", 3000 + i, B, h_kv * G, h_kv, ctx,
                              rng.choice([16, 32, 64, 128]), rng.choice([64, 128]),
                              k_dtype=rng.choice(["bf16", "fp8", "int4"]), paged=rng.random() < 0.5,
                              block_size=rng.choice([64, 128, 256]), ctx_lens=lens))
    return out


def prefill_cases(n=24, seed=44272603):
    rng = random.Random(seed)
    out = []
    for i in range(n):
        h_kv = rng.choice([1, 2])
        G = rng.choice([1, 2, 3, 4, 8])
        causal = rng.random() < 0.75
        sk = rng.randint(1, 600)
        sq = rng.randint(1, sk) if causal else rng.randint(1, 600)
        out.append(PrefillSpec(f"fuzz_prefill_{i}", 3100 + i, rng.randint(1, 3), h_kv * G, h_kv, sq, sk,
                               rng.choice([16, 32, 64, 128]), rng.choice([64, 128]),
                               dtype=rng.choice(["bf16", "f32"]), amp=0.5, causal=causal))
    return out


def backward_cases(n=10, seed=27182818):
    rng = random.Random(seed)
    out = []
    for i in range(n):
        h_kv = rng.choice([1, 2])
        G = rng.choice([1, 2, 4])
        causal = rng.random() < 0.75
        sk = rng.randint(1, 400)
        sq = rng.randint(1, sk) if causal else rng.randint(1, 400)
        out.append(PrefillSpec(f"fuzz_backward_{i}", 3200 + i, rng.randint(1, 2), h_kv * G, h_kv, sq, sk,
                               rng.choice([32, 64, 128]), rng.choice([64, 128]), dtype="bf16", amp=0.5,
                               causal=causal))
    return out


@pytest.mark.parametrize("spec", decode_cases(), ids=lambda s: s.name)
def test_decode_random_shapes(spec):
    dev = device()
    d = make_decode(spec, structured=spec.config_id % 2 == 0)
    say(f"fuzz {spec}")
    out = decode_on_gpu(d, spec, dev)
    torch.cuda.synchronize()
    gate(out, decode_oracle(d, spec), spec.k_dtype, spec.name)


@pytest.mark.parametrize("spec", prefill_cases(), ids=lambda s: s.name)
def test_prefill_random_shapes(spec):
    dev = device()
    p = make_prefill(spec, structured=spec.config_id % 2 == 0)
    say(f"fuzz {spec}")
    out = prefill_on_gpu(p, spec, dev)
    torch.cuda.synchronize()
    gate(out, prefill_oracle(p, spec), spec.dtype, spec.name)


def backward_inputs(spec):
    """Inputs of a fuzzed backward case: odd ids i.i.d., even ids moderately peaked."""
    p = make_prefill(spec, structured=spec.config_id % 2 == 0, needle_logit=6.0)
    return p["q"], p["k"], p["v"], make_prefill_grad(spec)


@pytest.mark.parametrize("spec", backward_cases(), ids=lambda s: s.name)
def test_backward_random_shapes(spec):
    from paper_2603_04427_amd import tk_attn_prefill_backward, tk_attn_prefill_lse
    dev = device()
    q, k, v, do = backward_inputs(spec)
    exact, bound = exact_terms(q, k, v, do, spec.causal, spec.softmax_scale)
    for name, e, b in zip(("dQ", "dK", "dV"), exact, bound):
        assert admissible(e, b), f"{spec.name} {name}: the bound does not discriminate on these inputs"
    say(f"fuzz {spec}")
    g = [t.to(dev) for t in (q, k, v)]
    o, lse = tk_attn_prefill_lse(*g, causal=spec.causal, scale=spec.softmax_scale)
    grads = tk_attn_prefill_backward(*g, o, do.to(dev), lse, causal=spec.causal, scale=spec.softmax_scale)
    torch.cuda.synchronize()
    for name, got, e, b in zip(("dQ", "dK", "dV"), grads, exact, bound):
        ok, msg = check(got, e, b)
        assert ok, f"{spec.name} {name}: {msg}"
