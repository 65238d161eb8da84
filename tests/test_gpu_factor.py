"""Thin keys from a converted pretrained layer, end to end on the GPU (Sec. 2.3, Eq. 5-7).

A synthetic layer whose key heads have exact rank r is converted offline
(`factor.factor_layer`), its thin projections are applied to hidden states
(`factor.project_thin`, bf16), and `tk_attn_prefill` runs on the result with
the layer's original softmax scale 1/sqrt(d_head). Two comparisons:

* kernel parity: the GPU output against the fp64 oracle on the same bf16 thin
  inputs (the bf16 gate);
* the method: the same GPU output against the fp64 oracle on the *unfactored*
  queries and keys of the original layer. Absorption is exact for rank-r keys,
  so the two differ only by the bf16 rounding of the projected inputs; with
  values of unit scale that stays inside the same bf16 gate.
"""
import math

import pytest
import torch

from gpu_cases import device, gate, say
from oracle import oracle as orc
from paper_2603_04427_amd import factor, tk_attn_prefill
from synth import normal, stream_key

pytestmark = pytest.mark.gpu


def draw(tensor: int, *shape, std=1.0):
    n = math.prod(shape)
    return (normal(stream_key(42, tensor), n).view(*shape) * std).to(torch.float64)


def heads(y, B, S, n):
    return y.reshape(B, S, n, -1).permute(0, 2, 1, 3).contiguous()


@pytest.mark.parametrize("B,S,d_model,h_q,h_kv,d_head,r", [
    (1, 256, 768, 12, 12, 64, 16),     # GPT-2-small layer, r/head 16
    (2, 300, 1024, 8, 2, 128, 32),     # Mistral-like GQA 4:1, d_head 128 -> r 32, ragged length
])
def test_converted_layer_matches_the_unfactored_attention(B, S, d_model, h_q, h_kv, d_head, r):
    dev = device()
    say(f"factored layer B={B} S={S} d_model={d_model} heads={h_q}/{h_kv} d_head={d_head} r={r}")
    x = draw(0, B, S, d_model)
    w_q = draw(1, d_model, h_q * d_head, std=d_model ** -0.5)
    a = draw(2, h_kv, d_model, r, std=d_model ** -0.5)
    b = draw(3, h_kv, r, d_head, std=r ** -0.5)
    w_k = torch.matmul(a, b).permute(1, 0, 2).reshape(d_model, h_kv * d_head)  # rank-r key heads
    w_v = draw(4, d_model, h_kv * d_head, std=0.5 * d_model ** -0.5)
    scale = d_head ** -0.5

    # the original layer in fp64 (reference of the method)
    q = heads(x @ w_q, B, S, h_q)
    k = heads(x @ w_k, B, S, h_kv)
    v = heads(x @ w_v, B, S, h_kv)
    ref_unfactored = orc.prefill(q, k, v, causal=True, scale=scale)

    # converted offline, projected and attended on the GPU
    q_t, k_t, sigma = factor.factor_layer(w_q, w_k, r, h_q, h_kv)
    assert sigma[:, r:].max() <= 1e-12 * sigma[:, 0].max()
    qg, kg, vg = factor.project_thin(x.to(dev, torch.float32), q_t, k_t, w_v, h_q, h_kv)
    assert qg.shape == (B, h_q, S, r) and kg.shape == (B, h_kv, S, r) and vg.shape == (B, h_kv, S, d_head)
    out = tk_attn_prefill(qg, kg, vg, causal=True, scale=scale)
    torch.cuda.synchronize()

    ref_same_inputs = orc.prefill(qg.cpu(), kg.cpu(), vg.cpu(), causal=True, scale=scale)
    gate(out, ref_same_inputs, "bf16", "kernel on the thin inputs")
    gate(out, ref_unfactored, "bf16", "thin keys against the unfactored layer")
