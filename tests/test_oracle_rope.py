"""Pins of the RoPE oracle (arXiv 2405.13226, Sec. 3 "Positional encoding").

* a second formulation: pairs as complex numbers multiplied by exp(i a);
* closed forms: position 0 is the identity; D = 2 rotates by the position
  itself; pair j of D = 4 at base 10^4 turns 0.01 rad per position;
* invariants: pair norms are kept; scores of rotated q and k depend only on
  the position difference; the inverse undoes the rotation;
* positions: row-local and document-local on an explicit example;
* brute force: finite differences of sum(dO * O) through rotation and
  attention pin the backward's transposed rotation;
* the DD / masked-chunk equivalence with document-local positions.
"""
import numpy as np
import pytest

import oracle
from oracle import rope as R

RNG = np.random.default_rng(2024)


def rand(*shape):
    return RNG.standard_normal(shape)


def test_complex_form():
    B, L, H, D, base = 2, 7, 3, 8, 10000.0
    x = rand(B, L, H, D)
    pos = np.arange(L)
    y = R.rope(x, base)
    z = x[..., 0::2] + 1j * x[..., 1::2]
    theta = base ** (-np.arange(D // 2) * 2.0 / D)
    w = z * np.exp(1j * pos[None, :, None, None] * theta)
    np.testing.assert_allclose(y[..., 0::2], w.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(y[..., 1::2], w.imag, rtol=0, atol=1e-12)


def test_position_zero_identity_and_norms():
    x = rand(1, 5, 2, 16)
    y = R.rope(x, 100000.0)
    np.testing.assert_array_equal(y[:, 0], x[:, 0])
    n_x = x[..., 0::2] ** 2 + x[..., 1::2] ** 2
    n_y = y[..., 0::2] ** 2 + y[..., 1::2] ** 2
    np.testing.assert_allclose(n_y, n_x, rtol=1e-12)


def test_closed_form_angles():
    # D = 2: theta_0 = 1, so position m turns by m radians.
    x = np.zeros((1, 4, 1, 2)); x[..., 0] = 1.0
    y = R.rope(x, 10000.0)
    for m in range(4):
        np.testing.assert_allclose(y[0, m, 0], [np.cos(m), np.sin(m)], atol=1e-15)
    # D = 4, base 1e4: pair 1 has theta = 1e4^(-1/2) = 0.01; position 100 -> 1 rad.
    x = np.zeros((1, 101, 1, 4)); x[..., 2] = 1.0
    y = R.rope(x, 10000.0)
    np.testing.assert_allclose(y[0, 100, 0], [0.0, 0.0, np.cos(1.0), np.sin(1.0)], atol=1e-13)


def test_scores_depend_on_position_difference():
    D, base = 16, 10000.0
    q, k = rand(D), rand(D)
    def score(m, n):
        qm = R.rotate(q, R.angles(m, D, base))
        kn = R.rotate(k, R.angles(n, D, base))
        return float(qm @ kn)
    for m, n, c in ((5, 2, 7), (0, 0, 100), (40, 39, 1000), (3, 9, 12)):
        assert abs(score(m, n) - score(m + c, n + c)) < 1e-9


def test_inverse():
    x = rand(2, 9, 2, 8)
    cu = [0, 4, 11, 18]
    y = R.rope(x, 500.0, cu, doc_positions=True)
    B, L, H, D = x.shape
    ang = R.angles(R.positions(B, L, cu, True), D, 500.0)[:, :, None, :]
    np.testing.assert_allclose(R.rotate(y, ang, inverse=True), x, atol=1e-12)


def test_positions():
    # rows of 6 tokens; documents start at 0, 4, 9
    cu = [0, 4, 9, 12]
    np.testing.assert_array_equal(R.positions(2, 6), [[0, 1, 2, 3, 4, 5]] * 2)
    np.testing.assert_array_equal(R.positions(2, 6, cu, doc_positions=True),
                                  [[0, 1, 2, 3, 0, 1], [0, 1, 2, 0, 1, 2]])
    # without the flag, document offsets do not change positions
    np.testing.assert_array_equal(R.positions(2, 6, cu, doc_positions=False),
                                  R.positions(2, 6))


def _f(q, k, v, do, base, cu, docpos):
    B, L, H, D = q.shape
    o, _ = R.attn_fwd(q, k, v, base, True, cu, docpos, round_rotated=False)
    return float((oracle.to_blhd(o, B, H) * do).sum())


@pytest.mark.parametrize("cu,docpos", [(None, False), ([0, 3, 7, 10], True), ([0, 3, 7, 10], False)])
def test_bwd_matches_finite_differences(cu, docpos):
    B, L, H, D, base = 2, 5, 1, 4, 10.0
    q, k, v, do = (rand(B, L, H, D) for _ in range(4))
    dq, dk, dv = (oracle.to_blhd(x, B, H)
                  for x in R.attn_bwd(q, k, v, do, base, True, cu, docpos, round_rotated=False))
    eps = 1e-6
    for name, grad in (("q", dq), ("k", dk), ("v", dv)):
        args = {"q": q, "k": k, "v": v}
        num = np.zeros_like(args[name])
        it = np.nditer(args[name], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            a = dict(args)
            p = args[name].copy(); p[idx] += eps
            m = args[name].copy(); m[idx] -= eps
            a[name] = p
            fp = _f(a["q"], a["k"], a["v"], do, base, cu, docpos)
            a[name] = m
            fm = _f(a["q"], a["k"], a["v"], do, base, cu, docpos)
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-8, err_msg=name)


def test_rope_changes_attention():
    # a nonzero base frequency must change the result (guards against a no-op rotation)
    q, k, v = (rand(1, 6, 1, 8) for _ in range(3))
    o0, _ = oracle.attn_fwd(q, k, v)
    o1, _ = R.attn_fwd(q, k, v, 10000.0, round_rotated=False)
    assert np.abs(o1 - o0).max() > 1e-3
    np.testing.assert_allclose(o1[:, 0], o0[:, 0], atol=1e-12)  # row 0 sees only itself


def test_dd_equivalence_with_document_positions():
    # a masked chunk with document-local positions equals separate per-document
    # calls with row positions
    L, H, D, base = 14, 2, 8, 10000.0
    cu = [0, 5, 9, 14]
    q, k, v, do = (rand(1, L, H, D) for _ in range(4))
    o, lse = R.attn_fwd(q, k, v, base, True, cu, True)
    g = R.attn_bwd(q, k, v, do, base, True, cu, True)
    o, lse = oracle.to_blhd(o, 1, H), oracle.to_blhd(lse, 1, H)
    g = [oracle.to_blhd(x, 1, H) for x in g]
    for a, z in zip(cu[:-1], cu[1:]):
        sl = (slice(None), slice(a, z))
        od, ld = R.attn_fwd(q[sl], k[sl], v[sl], base)
        gd = R.attn_bwd(q[sl], k[sl], v[sl], do[sl], base)
        np.testing.assert_allclose(o[sl], oracle.to_blhd(od, 1, H), atol=1e-12)
        np.testing.assert_allclose(lse[sl], oracle.to_blhd(ld, 1, H), atol=1e-12)
        for x, y in zip(g, gd):
            np.testing.assert_allclose(x[sl], oracle.to_blhd(y, 1, H), atol=1e-12)


def test_round_bf16_closed_forms():
    one = 1.0
    cases = [(one, one), (one + 2.0 ** -8, one),                  # tie -> even (1.0)
             (one + 3 * 2.0 ** -8, one + 2.0 ** -6),              # tie -> even (odd below)
             (one + 2.0 ** -8 + 2.0 ** -20, one + 2.0 ** -7),     # just above the tie
             (-3.0 - 2.0 ** -7, -3.0), (0.1, 0.10009765625), (1000.7, 1000.0)]
    got = R.round_bf16([c[0] for c in cases])
    np.testing.assert_array_equal(got, [c[1] for c in cases])
    # every result is a bf16 value: its float32 bits have 16 zero low bits
    x = rand(1000) * 100
    bits = R.round_bf16(x).astype(np.float32).view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)
    assert np.all(np.abs(R.round_bf16(x) - x) <= np.abs(x) * 2.0 ** -8)


def test_rounding_of_rotated_inputs_is_the_only_difference():
    q, k, v = (rand(1, 9, 2, 8) for _ in range(3))
    exact, _ = R.attn_fwd(q, k, v, 10000.0, round_rotated=False)
    qr = R.round_bf16(R.rope(q, 10000.0))
    kr = R.round_bf16(R.rope(k, 10000.0))
    ref, _ = oracle.attn_fwd(qr, kr, v)
    got, _ = R.attn_fwd(q, k, v, 10000.0)
    np.testing.assert_array_equal(got, ref)
    assert np.abs(got - exact).max() < 0.05


def test_selected_rows_match_full():
    q, k, v, do = (rand(3, 10, 2, 8) for _ in range(4))
    cu = [0, 4, 13, 22, 30]
    bh = [(2, 1), (0, 0)]
    full = R.attn_fwd(q, k, v, 10.0, True, cu, True)
    part = R.attn_fwd(q, k, v, 10.0, True, cu, True, bh=bh)
    gfull = R.attn_bwd(q, k, v, do, 10.0, True, cu, True)
    gpart = R.attn_bwd(q, k, v, do, 10.0, True, cu, True, bh=bh)
    idx = [b * 2 + h for b, h in bh]
    for a, z in zip(full + gfull, part + gpart):
        np.testing.assert_array_equal(a[idx], z)


def test_widen_bf16_exact():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x4049], dtype=np.uint16)
    np.testing.assert_array_equal(R.widen(bits), [1.0, -2.0, 0.0, 3.140625])
