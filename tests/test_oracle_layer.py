"""Pins of the OpenLM block oracle (oracle/layer.py).

* the parameter count of Table "openlm1b" (1,439,893,504) from the block
  readings, 24 blocks, untied 50,432-token embeddings and a final norm weight;
* an independent formulation: the whole block in float64 torch with
  scaled_dot_product_attention and RoPE as complex multiplication, forward and
  autograd gradients;
* finite differences of sum(dy * y) on a tiny block.
"""
import numpy as np
import pytest
import torch

from oracle import layer as OL

RNG = np.random.default_rng(77)


def weights(d, h, scale=0.2):
    r = lambda *s: RNG.standard_normal(s) * scale
    return dict(ln1_w=1 + r(d), ln1_b=r(d), w_qkv=r(d, 3 * d), w_o=r(d, d),
                ln2_w=1 + r(d), ln2_b=r(d), w_1=r(d, h), w_3=r(d, h), w_2=r(h, d))


def test_openlm1b_parameter_count():
    d, layers, vocab, hidden = 2048, 24, 50432, 5632
    total = 2 * vocab * d + layers * OL.openlm_block_params(d, hidden) + d
    assert total == 1_439_893_504


def reference_block(x, w, H, base):
    """Independent float64 formulation: SDPA + complex-number RoPE."""
    B, L, d = x.shape
    D = d // H
    a = torch.nn.functional.layer_norm(x, (d,), w["ln1_w"], w["ln1_b"], 1e-5)
    q, k, v = (a @ w["w_qkv"]).split(d, dim=-1)
    q, k, v = (t.reshape(B, L, H, D) for t in (q, k, v))
    if base:
        theta = base ** (-torch.arange(D // 2, dtype=torch.float64) * 2 / D)
        rot = torch.polar(torch.ones(L, D // 2, dtype=torch.float64),
                          torch.arange(L, dtype=torch.float64)[:, None] * theta)
        def rope(t):
            z = torch.view_as_complex(t.reshape(B, L, H, D // 2, 2).contiguous())
            return torch.view_as_real(z * rot[None, :, None, :]).reshape(B, L, H, D)
        q, k = rope(q), rope(k)
    o = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(1, 2), k.transpose(1, 2), v.transpose(1, 2), is_causal=True).transpose(1, 2)
    h = x + o.reshape(B, L, d) @ w["w_o"]
    m = torch.nn.functional.layer_norm(h, (d,), w["ln2_w"], w["ln2_b"], 1e-5)
    return h + (torch.nn.functional.silu(m @ w["w_1"]) * (m @ w["w_3"])) @ w["w_2"]


@pytest.mark.parametrize("base", [None, 10000.0])
def test_block_matches_independent_formulation(base):
    B, L, d, H, h = 2, 9, 16, 2, 24
    x, dy = RNG.standard_normal((B, L, d)), RNG.standard_normal((B, L, d))
    w = weights(d, h)
    y, g = OL.block_fwd_bwd(x, w, dy, H, base)
    xt = torch.tensor(x, requires_grad=True)
    wt = {n: torch.tensor(a, requires_grad=True) for n, a in w.items()}
    yr = reference_block(xt, wt, H, base)
    yr.backward(torch.tensor(dy))
    np.testing.assert_allclose(y, yr.detach().numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(g["x"], xt.grad.numpy(), rtol=1e-9, atol=1e-10)
    for n in w:
        np.testing.assert_allclose(g[n], wt[n].grad.numpy(), rtol=1e-9, atol=1e-10, err_msg=n)


def test_block_gradients_finite_differences():
    B, L, d, H, h = 1, 4, 8, 2, 6
    x, dy = RNG.standard_normal((B, L, d)), RNG.standard_normal((B, L, d))
    w = weights(d, h, 0.3)
    _, g = OL.block_fwd_bwd(x, w, dy, H, 100.0)
    f = lambda xx, ww: float((OL.block_fwd_bwd(xx, ww, dy, H, 100.0)[0] * dy).sum())
    eps = 1e-6
    for name in ("x", "w_qkv", "w_2", "ln1_b"):
        base = x if name == "x" else w[name]
        num = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            p, m = base.copy(), base.copy()
            p[idx] += eps
            m[idx] -= eps
            if name == "x":
                num[idx] = (f(p, w) - f(m, w)) / (2 * eps)
            else:
                num[idx] = (f(x, {**w, name: p}) - f(x, {**w, name: m})) / (2 * eps)
        np.testing.assert_allclose(g[name], num, rtol=1e-5, atol=1e-7, err_msg=name)
