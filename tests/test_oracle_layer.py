"""Pins of the OpenLM block oracle (oracle/layer.py).

* the parameter count of Table "openlm1b" (1,439,893,504) from the block
  readings, 24 blocks, untied 50,432-token embeddings and a final norm weight;
* an independent forward in plain float64 numpy written from the
  definitions: LayerNorm as mean and biased variance with eps 1e-5, SiLU as
  u / (1 + exp(-u)), RoPE as explicit cos/sin pair rotations, attention as a
  dense causal score matrix with -inf above the diagonal and a softmax;
* an independent formulation for the gradients: the whole block in float64
  torch autograd with the LayerNorm and SiLU written out the same way (no
  torch layer_norm or silu call), scaled_dot_product_attention and RoPE as
  complex multiplication;
* finite differences of sum(dy * y) on a tiny block;
* closed forms: a row of equal values normalises to the LayerNorm bias, and
  a block whose projections are zero is the identity.
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


def np_layer_norm(x, w, b, eps=1e-5):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)  # biased
    return (x - mu) / np.sqrt(var + eps) * w + b


def np_silu(u):
    return u / (1.0 + np.exp(-u))


def np_rope(t, base):
    """Rotate components (2j, 2j+1) of every head vector by pos * base^(-2j/D)."""
    B, L, H, D = t.shape
    out = t.copy()
    for j in range(D // 2):
        ang = np.arange(L, dtype=np.float64) * base ** (-2.0 * j / D)
        c, s = np.cos(ang)[None, :, None], np.sin(ang)[None, :, None]
        x0, x1 = t[..., 2 * j], t[..., 2 * j + 1]
        out[..., 2 * j] = x0 * c - x1 * s
        out[..., 2 * j + 1] = x0 * s + x1 * c
    return out


def np_causal_attention(q, k, v):
    B, L, H, D = q.shape
    o = np.zeros_like(q)
    future = np.triu(np.ones((L, L), dtype=bool), 1)
    for b in range(B):
        for h in range(H):
            s = q[b, :, h] @ k[b, :, h].T / np.sqrt(D)
            s[future] = -np.inf
            p = np.exp(s - s.max(axis=1, keepdims=True))
            o[b, :, h] = (p / p.sum(axis=1, keepdims=True)) @ v[b, :, h]
    return o


def numpy_block(x, w, H, base):
    """The block's forward in plain float64 numpy."""
    B, L, d = x.shape
    D = d // H
    a = np_layer_norm(x, w["ln1_w"], w["ln1_b"])
    qkv = a @ w["w_qkv"]
    q, k, v = (qkv[..., i * d:(i + 1) * d].reshape(B, L, H, D) for i in range(3))
    if base:
        q, k = np_rope(q, base), np_rope(k, base)
    h = x + np_causal_attention(q, k, v).reshape(B, L, d) @ w["w_o"]
    m = np_layer_norm(h, w["ln2_w"], w["ln2_b"])
    return h + (np_silu(m @ w["w_1"]) * (m @ w["w_3"])) @ w["w_2"]


def reference_block(x, w, H, base):
    """Independent float64 torch formulation (autograd): LayerNorm and SiLU
    written out, SDPA and complex-number RoPE."""
    B, L, d = x.shape
    D = d // H

    def layer_norm(t, g, b):
        mu = t.mean(dim=-1, keepdim=True)
        var = ((t - mu) ** 2).mean(dim=-1, keepdim=True)
        return (t - mu) / torch.sqrt(var + 1e-5) * g + b

    a = layer_norm(x, w["ln1_w"], w["ln1_b"])
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
    m = layer_norm(h, w["ln2_w"], w["ln2_b"])
    u = m @ w["w_1"]
    return h + (u / (1 + torch.exp(-u)) * (m @ w["w_3"])) @ w["w_2"]


@pytest.mark.parametrize("base", [None, 10000.0])
def test_block_forward_matches_numpy(base):
    B, L, d, H, h = 2, 11, 16, 2, 24
    x, dy = RNG.standard_normal((B, L, d)), RNG.standard_normal((B, L, d))
    w = weights(d, h, 0.3)
    y, _ = OL.block_fwd_bwd(x, w, dy, H, base)
    np.testing.assert_allclose(y, numpy_block(x, w, H, base), rtol=1e-11, atol=1e-11)


def test_block_closed_forms():
    B, L, d, H, h = 1, 5, 8, 2, 6
    w = weights(d, h)
    # A row of equal values has zero variance: LayerNorm returns its bias.
    x = np.full((B, L, d), 3.25)
    np.testing.assert_allclose(np_layer_norm(x, w["ln1_w"], w["ln1_b"]),
                               np.broadcast_to(w["ln1_b"], x.shape), atol=1e-12)
    # With zero output projections the block is the identity, so dy reaches x
    # unchanged and the input projections get no gradient.
    zero = {**w, "w_o": np.zeros((d, d)), "w_2": np.zeros((h, d))}
    x = RNG.standard_normal((B, L, d))
    dy = RNG.standard_normal((B, L, d))
    y, g = OL.block_fwd_bwd(x, zero, dy, H, 100.0)
    np.testing.assert_allclose(y, x, atol=1e-14)
    np.testing.assert_allclose(g["x"], dy, atol=1e-12)
    for n in ("w_qkv", "w_1", "w_3", "ln1_w", "ln1_b", "ln2_w", "ln2_b"):
        assert np.abs(g[n]).max() < 1e-12, n
    # silu(u) = u * sigmoid(u): sigmoid(0) = 1/2, so silu(0) = 0, silu(u) -> u
    assert np_silu(0.0) == 0.0 and abs(np_silu(40.0) - 40.0) < 1e-12


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
