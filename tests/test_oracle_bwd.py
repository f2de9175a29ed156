"""Pins of the oracle backward.

* brute force: central finite differences of f = sum(dO * O) in float64;
* a library routine: torch autograd through scaled_dot_product_attention in
  float64 on the CPU;
* closed forms: L = 1 and Q = 0;
* invariants: keys' gradients sum to zero per document segment (each row of
  dS sums to zero), and causality of dQ.
"""
import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(99)


def rand(*shape):
    return RNG.standard_normal(shape)


def fwd_full(q, k, v, causal, cu):
    B, L, H, D = q.shape
    o, _ = oracle.attn_fwd(q, k, v, causal=causal, cu_doclens=cu)
    return oracle.to_blhd(o, B, H)


@pytest.mark.parametrize("causal,cu", [(True, None), (False, None),
                                       (True, [0, 2, 7, 12]), (False, [0, 4, 12])])
def test_bwd_matches_finite_differences(causal, cu):
    B, L, H, D = 2, 6, 1, 3
    q, k, v, do = (rand(B, L, H, D) for _ in range(4))
    dq, dk, dv = (oracle.to_blhd(x, B, H)
                  for x in oracle.attn_bwd(q, k, v, do, causal=causal, cu_doclens=cu))
    eps = 1e-6
    for name, base, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            args = {"q": q, "k": k, "v": v}
            plus = base.copy(); plus[idx] += eps
            minus = base.copy(); minus[idx] -= eps
            args[name] = plus
            fp = (fwd_full(args["q"], args["k"], args["v"], causal, cu) * do).sum()
            args[name] = minus
            fm = (fwd_full(args["q"], args["k"], args["v"], causal, cu) * do).sum()
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-8, err_msg=name)


@pytest.mark.parametrize("B,L,H,D,causal", [(2, 21, 2, 8, True), (1, 48, 1, 64, True),
                                            (1, 13, 2, 16, False)])
def test_bwd_matches_sdpa_autograd(B, L, H, D, causal):
    q, k, v, do = (rand(B, L, H, D) for _ in range(4))
    t = [torch.from_numpy(x.copy()).permute(0, 2, 1, 3).requires_grad_(True) for x in (q, k, v)]
    o = torch.nn.functional.scaled_dot_product_attention(*t, is_causal=causal)
    o.backward(torch.from_numpy(do).permute(0, 2, 1, 3))
    ref = [x.grad.permute(0, 2, 1, 3).numpy() for x in t]
    got = [oracle.to_blhd(x, B, H) for x in oracle.attn_bwd(q, k, v, do, causal=causal)]
    for g, r, n in zip(got, ref, "qkv"):
        np.testing.assert_allclose(g, r, rtol=0, atol=1e-11, err_msg=n)


def test_length_one_closed_form():
    B, L, H, D = 3, 1, 2, 8
    q, k, v, do = (rand(B, L, H, D) for _ in range(4))
    dq, dk, dv = (oracle.to_blhd(x, B, H) for x in oracle.attn_bwd(q, k, v, do))
    assert np.all(dq == 0) and np.all(dk == 0)
    np.testing.assert_array_equal(dv, do)


def test_q_zero_closed_form():
    B, L, H, D = 1, 11, 1, 4
    q = np.zeros((B, L, H, D))
    k, v, do = (rand(B, L, H, D) for _ in range(3))
    dq, dk, dv = (oracle.to_blhd(x, B, H) for x in oracle.attn_bwd(q, k, v, do))
    np.testing.assert_allclose(dk, 0.0, atol=1e-14)
    for j in range(L):
        expect = sum(do[0, i, 0] / (i + 1) for i in range(j, L))
        np.testing.assert_allclose(dv[0, j, 0], expect, atol=1e-13)


def test_dk_sums_to_zero_per_segment():
    B, L, H, D = 2, 20, 2, 8
    cu = [0, 3, 11, 26, 40]
    q, k, v, do = (rand(B, L, H, D) for _ in range(4))
    _, dk, _ = oracle.attn_bwd(q, k, v, do, cu_doclens=cu)
    dkf = oracle.to_blhd(dk, B, H).reshape(B * L, H, D)
    cuts = sorted(set(cu) | {L})
    for a, z in zip(cuts[:-1], cuts[1:]):
        np.testing.assert_allclose(dkf[a:z].sum(axis=0), 0.0, atol=1e-12)


def test_dq_causality():
    B, L, H, D = 1, 16, 1, 4
    q, k, v, do = (rand(B, L, H, D) for _ in range(4))
    dq1, _, _ = oracle.attn_bwd(q, k, v, do)
    v2, do2 = v.copy(), do.copy()
    v2[:, 9:] += 1.5
    do2[:, 9:] *= 3.0
    dq2, _, _ = oracle.attn_bwd(q, k, v2, do2)
    np.testing.assert_array_equal(dq1[:, :9], dq2[:, :9])
