"""Pins of the oracle forward against things other than itself.

* a library routine: torch's scaled_dot_product_attention in float64 on the
  CPU (causal, non-causal, and with a boolean document mask);
* closed forms: Q = 0, L = 1, constant V, one-hot V (which exposes P);
* invariants: key shift, causality, permutation of b and h, and the
  DD <-> document-masked-chunk equivalence (Sec. 2.1: each DD sequence is a
  subsequence of one document; Sec. 3.6: document masking removes
  cross-document attention inside a chunk).
Every case here is small enough to run in well under a second.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth

RNG = np.random.default_rng(1234)


def rand(*shape):
    return RNG.standard_normal(shape)


def sdpa_ref(q, k, v, causal, mask=None):
    """torch SDPA in float64; q,k,v [B,L,H,D] -> o [B,L,H,D]."""
    t = [torch.from_numpy(np.ascontiguousarray(x)).permute(0, 2, 1, 3) for x in (q, k, v)]
    o = torch.nn.functional.scaled_dot_product_attention(
        *t, attn_mask=mask, is_causal=causal and mask is None)
    return o.permute(0, 2, 1, 3).numpy()


def blhd(o, B, H):
    return oracle.to_blhd(o, B, H)


@pytest.mark.parametrize("B,L,H,D,causal", [
    (2, 37, 3, 8, True), (1, 64, 2, 64, True), (2, 19, 2, 16, False),
    (1, 1, 1, 4, True), (3, 5, 1, 128, True)])
def test_fwd_matches_sdpa(B, L, H, D, causal):
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    o, lse = oracle.attn_fwd(q, k, v, causal=causal)
    ref = sdpa_ref(q, k, v, causal)
    np.testing.assert_allclose(blhd(o, B, H), ref, rtol=0, atol=1e-12)


def doc_mask_matrix(B, L, cu, causal):
    """Boolean [B,1,L,L] mask from doc ids (for the library routine only)."""
    ids = np.searchsorted(np.asarray(cu), np.arange(B * L), side="right") - 1
    ids = ids.reshape(B, L)
    m = ids[:, :, None] == ids[:, None, :]
    if causal:
        m = m & np.tril(np.ones((L, L), dtype=bool))[None]
    return torch.from_numpy(m[:, None])


@pytest.mark.parametrize("causal", [True, False])
def test_fwd_doc_mask_matches_sdpa(causal):
    B, L, H, D = 2, 30, 2, 8
    cu = [0, 7, 8, 25, 41, 60]  # documents crossing the row edge at 30
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    o, _ = oracle.attn_fwd(q, k, v, causal=causal, cu_doclens=cu)
    ref = sdpa_ref(q, k, v, causal, mask=doc_mask_matrix(B, L, cu, causal))
    np.testing.assert_allclose(blhd(o, B, H), ref, rtol=0, atol=1e-12)


def test_q_zero_gives_prefix_mean():
    B, L, H, D = 1, 23, 2, 5
    q = np.zeros((B, L, H, D))
    k, v = rand(B, L, H, D), rand(B, L, H, D)
    o, lse = oracle.attn_fwd(q, k, v, causal=True)
    o = blhd(o, B, H)
    lse = oracle.to_blhd(lse, B, H)
    for i in range(L):
        np.testing.assert_allclose(o[0, i], v[0, : i + 1].mean(axis=0), atol=1e-13)
        np.testing.assert_allclose(lse[0, i], math.log(i + 1), atol=1e-13)
    o2, lse2 = oracle.attn_fwd(q, k, v, causal=False)
    np.testing.assert_allclose(blhd(o2, B, H)[0], np.broadcast_to(v[0].mean(axis=0), (L, H, D)),
                               atol=1e-13)
    np.testing.assert_allclose(lse2, math.log(L), atol=1e-13)


def test_length_one_returns_v():
    B, L, H, D = 5, 1, 3, 64
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    o, lse = oracle.attn_fwd(q, k, v)
    np.testing.assert_array_equal(blhd(o, B, H), v)
    expect = (q * k).sum(-1) / math.sqrt(D)
    np.testing.assert_allclose(oracle.to_blhd(lse, B, H), expect, atol=1e-13)


def test_constant_v_rows():
    B, L, H, D = 2, 17, 2, 6
    q, k = rand(B, L, H, D), rand(B, L, H, D)
    c = rand(D)
    v = np.broadcast_to(c, (B, L, H, D)).copy()
    o, _ = oracle.attn_fwd(q, k, v, cu_doclens=[0, 3, 20, 34])
    np.testing.assert_allclose(blhd(o, B, H), v, atol=1e-13)


@pytest.mark.parametrize("causal", [True, False])
def test_one_hot_v_exposes_probabilities(causal):
    # V = identity (D = L) makes o_i the probability row p_i.
    B, L, H = 1, 12, 1
    cu = [0, 5, 12]
    q, k = rand(B, L, H, L), rand(B, L, H, L)
    v = np.eye(L)[None, :, None, :].copy()
    o, _ = oracle.attn_fwd(q, k, v, causal=causal, cu_doclens=cu)
    p = o[0]
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-14)
    doc = np.searchsorted(cu, np.arange(L), side="right") - 1
    for i in range(L):
        for j in range(L):
            ok = doc[i] == doc[j] and (not causal or j <= i)
            if not ok:
                assert p[i, j] == 0.0
            else:
                assert p[i, j] > 0.0


def test_key_shift_invariance():
    B, L, H, D = 2, 15, 2, 8
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    c = rand(D)
    o1, l1 = oracle.attn_fwd(q, k, v)
    o2, l2 = oracle.attn_fwd(q, k + c, v)
    np.testing.assert_allclose(o2, o1, atol=1e-12)
    shift = (q @ c) / math.sqrt(D)  # [B, L, H]
    np.testing.assert_allclose(oracle.to_blhd(l2 - l1, B, H), shift, atol=1e-12)


def test_causality_future_perturbation_is_exact():
    B, L, H, D = 1, 40, 2, 8
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    o1, l1 = oracle.attn_fwd(q, k, v)
    k2, v2, q2 = k.copy(), v.copy(), q.copy()
    k2[:, 20:] += 3.0
    v2[:, 20:] -= 2.0
    q2[:, 20:] *= -1.0
    o2, l2 = oracle.attn_fwd(q2, k2, v2)
    np.testing.assert_array_equal(o1[:, :20], o2[:, :20])
    np.testing.assert_array_equal(l1[:, :20], l2[:, :20])
    assert not np.allclose(o1[:, 20:], o2[:, 20:])


def test_permutation_of_batch_and_heads():
    B, L, H, D = 3, 9, 4, 4
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    pb, ph = [2, 0, 1], [3, 1, 0, 2]
    o1, _ = oracle.attn_fwd(q, k, v)
    perm = lambda x: x[pb][:, :, ph]
    o2, _ = oracle.attn_fwd(perm(q), perm(k), perm(v))
    np.testing.assert_array_equal(perm(blhd(o1, B, H)), blhd(o2, B, H))


def test_dd_buckets_equal_masked_chunks_zero_copy():
    # A packed [Bc, L] batch whose documents all have length ell is, byte for
    # byte, the DD bucket batch [Bc*L/ell, ell] without any mask.
    Bc, L, H, D, ell = 2, 32, 2, 8, 8
    q, k, v = rand(Bc, L, H, D), rand(Bc, L, H, D), rand(Bc, L, H, D)
    cu = np.arange(0, Bc * L + 1, ell)
    o1, l1 = oracle.attn_fwd(q, k, v, cu_doclens=cu)
    r = lambda x: x.reshape(Bc * L // ell, ell, H, D)
    o2, l2 = oracle.attn_fwd(r(q), r(k), r(v))
    np.testing.assert_array_equal(blhd(o1, Bc, H).reshape(-1, H, D),
                                  blhd(o2, Bc * L // ell, H).reshape(-1, H, D))
    np.testing.assert_array_equal(oracle.to_blhd(l1, Bc, H).reshape(-1, H),
                                  oracle.to_blhd(l2, Bc * L // ell, H).reshape(-1, H))


def test_masked_chunk_equals_separate_documents():
    B, L, H, D = 2, 24, 2, 8
    cu = [0, 5, 6, 19, 30, 48]
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    o, lse = oracle.attn_fwd(q, k, v, cu_doclens=cu)
    o, lse = blhd(o, B, H), oracle.to_blhd(lse, B, H)
    flat = lambda x: x.reshape(B * L, H, -1)
    of, lf = flat(o), lse.reshape(B * L, H)
    qf, kf, vf = flat(q), flat(k), flat(v)
    for s, e in zip(cu[:-1], cu[1:]):
        # a document crossing a row edge is split there (concat-and-chunk)
        cuts = sorted({s, e} | {x for x in range(0, B * L + 1, L) if s < x < e})
        for a, z in zip(cuts[:-1], cuts[1:]):
            seg = lambda x: x[a:z][None]
            od, ld = oracle.attn_fwd(seg(qf), seg(kf), seg(vf))
            np.testing.assert_allclose(of[a:z], blhd(od, 1, H)[0], atol=1e-13)
            np.testing.assert_allclose(lf[a:z], oracle.to_blhd(ld, 1, H)[0], atol=1e-13)


def test_bf16_entry_equals_f64_entry_on_widened_values():
    B, L, H, D = 2, 33, 2, 64
    x = synth.attention_inputs(B, L, H, D, seed=7, with_grad=False)
    w = {n: synth.f32_from_bf16_bits(a).astype(np.float64) for n, a in x.items()}
    bh = [(1, 0), (0, 1)]
    o1, l1 = oracle.attn_fwd(x["q"], x["k"], x["v"], bh=bh)
    o2, l2 = oracle.attn_fwd(w["q"], w["k"], w["v"], bh=bh)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_bad_arguments_raise():
    q = np.zeros((1, 4, 1, 2))
    with pytest.raises(ValueError):
        oracle.attn_fwd(q, q, q, bh=[(1, 0)])


@pytest.mark.parametrize("causal", [True, False])
def test_lse_matches_library_logsumexp(causal):
    B, L, H, D = 2, 26, 2, 16
    cu = [0, 9, 10, 31, 52]
    q, k, v = rand(B, L, H, D), rand(B, L, H, D), rand(B, L, H, D)
    _, lse = oracle.attn_fwd(q, k, v, causal=causal, cu_doclens=cu)
    s = torch.einsum("blhd,bmhd->bhlm", torch.from_numpy(q), torch.from_numpy(k)) / math.sqrt(D)
    m = doc_mask_matrix(B, L, cu, causal)  # [B,1,L,L]
    s = s.masked_fill(~m, float("-inf"))
    ref = torch.logsumexp(s, dim=-1).permute(0, 2, 1).numpy()  # [B,L,H]
    np.testing.assert_allclose(oracle.to_blhd(lse, B, H), ref, rtol=0, atol=1e-12)
