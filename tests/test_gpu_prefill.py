"""Prefill parity on the GPU: tk_attn_prefill against the fp64 oracle on the same
seeded inputs — every output at sweep sizes and at the GPT-2 fp32 size, and
65 rows of every sequence (all heads) at the Mistral 8192-token size in the launch
configuration the benchmark times — plus causal invariants."""
import pytest
import torch

from gpu_cases import device, gate, prefill_on_gpu, prefill_oracle, prefill_rows_oracle, say
from synth import FULLKEY, WORKLOADS, PrefillSpec, make_prefill, with_shape

pytestmark = pytest.mark.gpu

BASE = PrefillSpec("sweep", 600, 2, 4, 2, 200, 200, 32, 128, dtype="bf16", amp=1.0)


def run_full(spec, structured=False):
    dev = device()
    p = make_prefill(spec, structured=structured)
    say(f"prefill {spec} structured={structured}")
    out = prefill_on_gpu(p, spec, dev)
    torch.cuda.synchronize()
    return out, prefill_oracle(p, spec)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("dv", [64, 128])
def test_sweep_widths(dtype, r, dv):
    spec = with_shape(BASE, config_id=600 + r + dv, r=r, d_v=dv, dtype=dtype)
    for structured in (False, True):
        out, ref = run_full(spec, structured)
        gate(out, ref, dtype, f"{spec} structured={structured}")


SHAPES = [  # (B, Hq, Hkv, Sq, Sk, causal)
    (1, 1, 1, 1, 1, True),
    (1, 2, 1, 31, 31, True),
    (2, 4, 4, 33, 33, True),
    (1, 8, 2, 100, 100, False),
    (1, 4, 2, 64, 200, True),     # bottom-right alignment: 64 new rows after 136 cached keys
    (1, 4, 1, 5, 300, True),
    (2, 6, 2, 257, 257, True),    # G = 3
    (1, 16, 2, 130, 130, True),   # G = 8
    (1, 2, 2, 65, 129, False),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES)
def test_shapes_and_masks(dtype, shape):
    B, Hq, Hkv, Sq, Sk, causal = shape
    spec = with_shape(BASE, config_id=700, batch=B, h_q=Hq, h_kv=Hkv, seq_q=Sq, seq_k=Sk, causal=causal,
                      dtype=dtype, r=32 if dtype == "bf16" else 16, d_v=128 if dtype == "bf16" else 64)
    out, ref = run_full(spec, structured=True)
    gate(out, ref, dtype, str(spec))


def test_gpt2_prefill_f32_full():
    """GPT-2 small shape, fp32, every output against the oracle (gate 1e-4)."""
    spec = WORKLOADS["gpt2_prefill_f32"]
    for structured in (False, True):
        out, ref = run_full(spec, structured)
        mx, rel = gate(out, ref, "f32", f"gpt2 structured={structured}")
        say(f"  max-abs {mx:.2e} rel-L2 {rel:.2e}")


# first and last row of 32-row wave blocks (and of 64-key tiles) at causal depths
# from the first tile to the last, plus interior rows: 65 rows per sequence
BLOCKS = [0, 1, 2, 3, 7, 15, 31, 32, 63, 64, 100, 127, 128, 129, 191, 200, 223, 240, 250, 253, 254, 255]
ROWS = sorted({32 * kb + d for kb in BLOCKS for d in (0, 31)} | {5, 17, 47, 48, 95, 1000, 2049, 3071, 4096,
                                                                    4111, 5000, 6143, 7000, 7777, 8000,
                                                                    8100, 8129, 8150, 8160, 8175, 8180,
                                                                    8185, 8189, 8190, 2, 33, 1023, 1024, 4095})


@pytest.mark.parametrize("structured", [False, True])
@pytest.mark.parametrize("name", ["mistral_prefill_s8192", "mistral_prefill_s8192_fullkey"])
def test_mistral_prefill_s8192_full_sampled(name, structured):
    """Batch 4, 32/8 heads, 8192 tokens, d_v 128, bf16, thin keys (r 32) and the
    full-key control (r 128): the whole call on the GPU, 65 rows of every sequence
    (all heads) against the oracle."""
    dev = device()
    spec = {**WORKLOADS, **FULLKEY}[name]
    p = make_prefill(spec, device=dev, structured=structured)
    say(f"prefill full {spec.name} structured={structured}")
    out = prefill_on_gpu(p, spec, dev)
    torch.cuda.synchronize()
    assert len(ROWS) >= 64
    for b in range(spec.batch):
        ref = prefill_rows_oracle(p, spec, b, ROWS)                  # [n, Hq, dv]
        got = out[b, :, ROWS].permute(1, 0, 2)
        mx, rel = gate(got, ref, "bf16", f"b={b}")
        say(f"  b={b} max-abs {mx:.2e} rel-L2 {rel:.2e}")


def test_causal_future_perturbation_bitwise():
    dev = device()
    spec = with_shape(BASE, config_id=800, seq_q=300, seq_k=300)
    p = make_prefill(spec, structured=True)
    a = prefill_on_gpu(p, spec, dev)
    i = 150
    p2 = {k: v.clone() for k, v in p.items()}
    p2["k"][:, :, i + 1:] = 3.0
    p2["v"][:, :, i + 1:] = -7.0
    say("prefill future perturbation")
    b = prefill_on_gpu(p2, spec, dev)
    assert torch.equal(a[:, :, :i + 1], b[:, :, :i + 1])
    assert not torch.equal(a[:, :, i + 1:], b[:, :, i + 1:])
    assert torch.equal(a, prefill_on_gpu(p, spec, dev))   # deterministic
