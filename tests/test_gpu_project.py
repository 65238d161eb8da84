"""The thin-projection kernel (tk_project_heads) on the GPU against the fp64
oracle on the same seeded inputs (Sec. 2.3, Eq. 6-7).

* Kernel parity: Y = X W head-major for bf16 X and W, element by element
  against oracle.factored.project_heads on the same bf16 values widened
  exactly. The bar is derived from the arithmetic: fp32 accumulation of d_model
  exact products (at most d_model * 2^-24 of sum |x||w|) and one rounding to
  bf16 (at most 2^-8 of the value):
      |Y_gpu - Y| <= 2^-8 |Y| + (1 + 2^-8) d_model 2^-24 (|X| |W|).
  Shapes cover both tile shapes the kernel picks (128 x 128 and 256 x 256),
  tile tails in tokens and columns, odd numbers of k-tiles, head widths 4-128
  and a single token.
* The converted layer: factor.factor_layer on a layer whose key heads have exact
  rank r, then factor.project_thin (three kernel calls) against
  oracle.factored.thin_projections, which redoes the SVD with numpy in fp64.
  Singular vectors are unique up to sign, so each thin column's sign is
  aligned on the keys (and carried to the group's queries) before the element
  comparison; the logits q' k'^T, which are unique, are compared as well. The
  bar adds the bf16 rounding of x and of the converted weights to the one above.
"""
import math

import numpy as np
import pytest
import torch

from gpu_cases import device, say
from oracle import factored
from paper_2603_04427_amd import TkError, factor, tk_project_heads
from synth import normal, stream_key

pytestmark = pytest.mark.gpu

U = 2.0 ** -8


def draw(seed: int, tensor: int, *shape, std=1.0):
    n = math.prod(shape)
    return normal(stream_key(seed, tensor), n).view(*shape) * std


def check(got, ref, bar, what):
    g = got.detach().double().cpu().numpy()
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    over = np.abs(g - ref) - bar
    assert over.max() <= 0, f"{what}: worst element over its bar by {over.max():.3e} (max-abs {np.abs(g - ref).max():.3e})"
    return np.abs(g - ref).max()


SHAPES = [  # (B, S, d_model, heads, width)
    (1, 256, 768, 12, 16),    # GPT-2 small: q' and k' (r 16 per head)
    (1, 256, 768, 12, 64),    # GPT-2 small: values
    (2, 300, 1024, 8, 32),    # GQA-like queries, ragged token tile
    (2, 300, 1024, 2, 128),   # full-width values of 2 KV heads
    (3, 77, 4096, 32, 32),    # Mistral-7B d_model, 32 query heads of r 32
    (1, 1, 64, 1, 4),         # one token, one narrow head
    (1, 129, 160, 3, 20),     # an odd number of 32-wide k-tiles, 60 columns, ragged tokens
    (2, 2048, 1024, 32, 128),  # 256 x 256 workgroup tiles (at least one per CU)
    (1, 4100, 256, 64, 68),   # 256 x 256 tiles with tails in tokens and columns
    (1, 4100, 160, 64, 68),   # 256 x 256 tiles over an odd number (5) of k-tiles
    (1, 4096, 32, 64, 64),    # 256 x 256 tiles over a single k-tile
    (2, 16350, 288, 7, 36),   # 256 x 128 tiles (narrow and long): ragged columns and tokens, 9 k-tiles
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_projection_against_oracle(shape):
    B, S, d_model, heads, width = shape
    dev = device()
    seed = 1600 + sum(shape)
    x = draw(seed, 0, B, S, d_model).to(torch.bfloat16)
    w = draw(seed, 1, d_model, heads * width, std=d_model ** -0.5).to(torch.bfloat16)
    xd, wd = x.double().numpy(), w.double().numpy()
    ref = factored.project_heads(xd, wd, heads)
    bar = U * np.abs(ref) + (1 + U) * d_model * 2.0 ** -24 * factored.project_heads(np.abs(xd), np.abs(wd), heads)
    say(f"project {shape}")
    y = tk_project_heads(x.to(dev), w.t().contiguous().to(dev), heads)
    torch.cuda.synchronize()
    assert tuple(y.shape) == (B, heads, S, width)
    mx = check(y, ref, bar, str(shape))
    say(f"  max-abs {mx:.2e}")


def test_empty_and_rejected():
    dev = device()
    x = torch.zeros(2, 0, 64, dtype=torch.bfloat16, device=dev)
    wt = torch.zeros(8, 64, dtype=torch.bfloat16, device=dev)
    assert tk_project_heads(x, wt, 2).shape == (2, 2, 0, 4)
    with pytest.raises(TkError, match="unsupported"):   # width 3 is not a multiple of 4
        tk_project_heads(torch.zeros(1, 4, 64, dtype=torch.bfloat16, device=dev),
                         torch.zeros(6, 64, dtype=torch.bfloat16, device=dev), 2)
    with pytest.raises(TkError, match="unsupported"):   # d_model 40 is not a multiple of 32
        tk_project_heads(torch.zeros(1, 4, 40, dtype=torch.bfloat16, device=dev),
                         torch.zeros(8, 40, dtype=torch.bfloat16, device=dev), 2)


@pytest.mark.parametrize("B,S,d_model,h_q,h_kv,d_head,r", [
    (1, 256, 768, 12, 12, 64, 16),     # GPT-2-small layer, r/head 16
    (2, 300, 1024, 8, 2, 128, 32),     # Mistral-like GQA 4:1, d_head 128 -> r 32
])
def test_converted_layer_projections(B, S, d_model, h_q, h_kv, d_head, r):
    dev = device()
    seed = 1700 + r
    x = draw(seed, 0, B, S, d_model).double()
    w_q = draw(seed, 1, d_model, h_q * d_head, std=d_model ** -0.5).double()
    a = draw(seed, 2, h_kv, d_model, r, std=d_model ** -0.5).double()
    b = draw(seed, 3, h_kv, r, d_head, std=r ** -0.5).double()
    w_k = torch.matmul(a, b).permute(1, 0, 2).reshape(d_model, h_kv * d_head)   # rank-r key heads
    w_v = draw(seed, 4, d_model, h_kv * d_head, std=0.5 * d_model ** -0.5).double()
    G = h_q // h_kv

    q_t, k_t, _ = factor.factor_layer(w_q, w_k, r, h_q, h_kv)
    say(f"converted layer projections B={B} S={S} d_model={d_model} heads={h_q}/{h_kv} r={r}")
    qg, kg, vg = factor.project_thin(x.to(dev), q_t, k_t, w_v, h_q, h_kv)
    torch.cuda.synchronize()

    qh = [w_q[:, i * d_head:(i + 1) * d_head].numpy() for i in range(h_q)]
    kh = [w_k[:, i * d_head:(i + 1) * d_head].numpy() for i in range(h_kv)]
    xs = x.reshape(B * S, d_model).numpy()
    qo, ko, _ = factored.thin_projections(xs, qh, kh, r, group=G)       # [h, B*S, r]
    ko = ko.reshape(h_kv, B, S, r).transpose(1, 0, 2, 3)                  # [B, h_kv, S, r]
    qo = qo.reshape(h_q, B, S, r).transpose(1, 0, 2, 3)
    # the converted weights the oracle implies, for the bar (|x| |W'|, sign-free)
    wk_or = np.concatenate([factored.factor_key_projection(k_, r)[0] for k_ in kh], axis=1)
    wq_or = np.concatenate([factored.absorb_query(qh[i], factored.factor_key_projection(kh[i // G], r)[1])
                            for i in range(h_q)], axis=1)
    xa = np.abs(x.numpy())
    rel = 2 * U + U * U + d_model * 2.0 ** -24 * (1 + U) ** 2

    kgd = kg.double().cpu().numpy()
    sign = np.sign(np.einsum("bhsc,bhsc->hc", kgd, ko))                    # [h_kv, r]
    assert (sign != 0).all()
    k_al = ko * sign[None, :, None, :]
    q_al = qo * np.repeat(sign, G, axis=0)[None, :, None, :]
    bars = {}
    for got, ref, wo, n, what in ((kg, k_al, wk_or, h_kv, "k'"), (qg, q_al, wq_or, h_q, "q'")):
        bars[what] = U * np.abs(ref) + (1 + U) * rel * factored.project_heads(xa, np.abs(wo), n)
        mx = check(got, ref, bars[what], what)
        say(f"  {what} max-abs {mx:.2e}")
    # values: the plain projection of the same x
    ref_v = factored.project_heads(x.numpy(), w_v.numpy(), h_kv)
    bar_v = U * np.abs(ref_v) + (1 + U) * rel * factored.project_heads(xa, np.abs(w_v.numpy()), h_kv)
    check(vg, ref_v, bar_v, "v")
    # logits of the thin projections are unique: compare them directly, with the
    # bar the element bars imply, |dq||k| + |q||dk| + |dq||dk| summed over r
    def mm(a_, b_):
        return torch.matmul(torch.from_numpy(np.ascontiguousarray(a_)),
                            torch.from_numpy(np.ascontiguousarray(b_)).repeat_interleave(G, dim=1).transpose(-1, -2))
    lg = torch.matmul(qg.double().cpu(), kg.double().cpu().repeat_interleave(G, dim=1).transpose(-1, -2))
    lo = mm(qo, ko)
    bq, bk = bars["q'"], bars["k'"]
    lbar = mm(bq, np.abs(ko)) + mm(np.abs(qo), bk) + mm(bq, bk)
    assert ((lg - lo).abs() <= lbar).all()
