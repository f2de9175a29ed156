"""GPU parity of rotary position embedding (Sec. 3, "Positional encoding")
through the C ABI against the fp64 oracle (oracle/rope.py).

* dd_rope alone: every element is the oracle's exact rotation rounded to
  bf16, up to half a bf16 ulp plus the fp32 evaluation error of the rotation
  (angle reduced in double, fp32 sine/cosine: 2^-17 of the pair's magnitude);
  positions up to 16,383 exercise the angle reduction.
* Attention over rotated q, k (dd_rope of k, dd_attn_fwd_rope rotating q
  as it loads it, dd_attn_bwd_rope): the tolerances of tests/parity.py
  against the oracle with the rotated q, k rounded to bf16 (its stated
  reading of the precision); the fused query rotation is bit-identical to a
  dd_rope pass followed by dd_attn_fwd.
* The DD / masked-chunk equivalence with document-local positions.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import rope as R
from paper_2405_13226_amd import dd

from parity import (BWD_RTOL, FWD_ATOL, LSE_ATOL, half_ulp_bf16, log, rel_l2, select_bh,
                    to_dev, to_f64)

pytestmark = pytest.mark.gpu

ROT_REL = 2.0 ** -17  # fp32 evaluation of a rotated pair, relative to the pair's norm


def rope_bound(x_bits, ref):
    x = R.widen(x_bits)
    pair = np.sqrt(x[..., 0::2] ** 2 + x[..., 1::2] ** 2)
    pair = np.repeat(pair, 2, axis=-1)
    return half_ulp_bf16(ref) + ROT_REL * pair + 1e-30


@pytest.mark.parametrize("B,L,H,D,base,docs,doc_pos,inverse", [
    (2, 300, 3, 64, 10000.0, False, False, False),
    (2, 300, 3, 128, 100000.0, False, False, True),
    (3, 512, 2, 128, 10000.0, True, True, False),
    (3, 512, 2, 64, 10000.0, True, False, False),
    (1, 16384, 1, 128, 10000.0, False, False, False),
    (1, 16384, 1, 64, 200000.0, False, False, True),
])
def test_rope_kernel_matches_oracle(cuda, B, L, H, D, base, docs, doc_pos, inverse):
    import paper_2405_13226_amd as pkg
    log(f"rope B={B} L={L} H={H} D={D} base={base} docs={docs} doc_pos={doc_pos} inv={inverse}")
    x = synth.normal_bf16((B, L, H, D), seed=B * 7 + D, stream=11)
    cu = None
    if docs:
        lens = synth.lognormal_doc_lengths(3, total_tokens=B * L, median=100, sigma=1.0)
        cu = dd.chunk_doclens(lens, B * L)
    y = pkg.rope(to_dev(x, cuda), base, cu, doc_pos, inverse)
    torch.cuda.synchronize()
    ref = R.rope(x, base, cu, doc_pos, inverse)
    got = to_f64(y)
    err = np.abs(got - ref)
    bound = rope_bound(x, ref)
    log(f"  max err {err.max():.3g}, max err/bound {(err / bound).max():.3f}")
    assert np.all(err <= bound)


def test_rope_in_place_and_inverse(cuda):
    import paper_2405_13226_amd as pkg
    x = synth.normal_bf16((2, 257, 2, 128), seed=5, stream=12)
    t = to_dev(x, cuda).clone()
    y = pkg.rope(t, 10000.0)
    pkg.rope(t, 10000.0, out=t)  # in place
    torch.cuda.synchronize()
    assert torch.equal(t, y)
    back = to_f64(pkg.rope(y, 10000.0, inverse=True))
    # R^T(bf16(R x)) returns x up to the rounding of the rotated values
    assert np.abs(back - R.widen(x)).max() <= 2.0 ** -7 * np.abs(R.widen(x)).max()


def run_rope_attention(B, L, H, D, base, cu=None, doc_pos=False, seed=0, bh=None):
    import paper_2405_13226_amd as pkg
    tag = f"B={B} L={L} H={H} D={D} base={base:g} docs={None if cu is None else len(cu) - 1} doc_pos={doc_pos}"
    log(f"rope attention {tag}")
    inp = synth.attention_inputs(B, L, H, D, seed=seed, with_grad=True)
    q, k, v, do = (to_dev(inp[n], cuda_dev()) for n in ("q", "k", "v", "do"))
    o, lse, qr, kr = pkg.forward_rope(q, k, v, base, True, cu, doc_pos)
    dq, dk, dv = pkg.backward_rope(qr, kr, v, o, lse, do, base, True, cu, doc_pos)
    torch.cuda.synchronize()
    if bh is None:
        bh = [(b, h) for b in range(B) for h in range(H)]
    o_ref, lse_ref = R.attn_fwd(inp["q"], inp["k"], inp["v"], base, True, cu, doc_pos, bh)
    g_ref = R.attn_bwd(inp["q"], inp["k"], inp["v"], inp["do"], base, True, cu, doc_pos, bh)
    got_o = select_bh(to_f64(o), bh)
    err = np.abs(got_o - o_ref)
    res = {"o_excess": float((err - (FWD_ATOL + half_ulp_bf16(o_ref))).max()),
           "o_maxabs": float(err.max()),
           "lse_maxabs": float(np.abs(select_bh(lse.cpu().numpy().astype(np.float64), bh)
                                      - lse_ref).max())}
    for n, t, ref in zip(("dq", "dk", "dv"), (dq, dk, dv), g_ref):
        res[n + "_rel"] = rel_l2(select_bh(to_f64(t), bh), ref)
    log("  " + "  ".join(f"{k}={v:.3g}" for k, v in res.items()))
    assert res["o_excess"] <= 0 and res["lse_maxabs"] <= LSE_ATOL, res
    for n in ("dq", "dk", "dv"):
        assert res[n + "_rel"] <= BWD_RTOL, res
    return (o, lse, dq, dk, dv), res


def cuda_dev():
    return torch.device("cuda:0")


@pytest.mark.parametrize("B,L,H,D,base", [(2, 256, 2, 64, 10000.0), (1, 300, 2, 128, 100000.0),
                                          (3, 129, 1, 64, 100000.0), (2, 512, 2, 128, 10000.0)])
def test_attention_rope_parity(cuda, B, L, H, D, base):
    run_rope_attention(B, L, H, D, base, seed=L + D)


@pytest.mark.parametrize("D,doc_pos", [(64, True), (128, True), (128, False)])
def test_attention_rope_masked_chunks(cuda, D, doc_pos):
    B, L, H = 3, 512, 2
    lens = synth.lognormal_doc_lengths(7, total_tokens=B * L, median=150, sigma=1.0)
    cu = dd.chunk_doclens(lens, B * L)
    run_rope_attention(B, L, H, D, 10000.0, cu, doc_pos, seed=D)


@pytest.mark.parametrize("B,D", [(48, 128), (48, 64)])
def test_attention_rope_persistent_dkdv(cuda, B, D):
    # 864 ragged key blocks: the dK RoPE epilogue runs once per item inside
    # the persistent dK/dV kernels' item loop.
    run_rope_attention(B, 700, 3, D, 100000.0, seed=5,
                       bh=[(0, 0), (B // 2, 1), (B - 8, 2), (B - 1, 2)])


def test_attention_rope_full_bucket_sampled(cuda):
    B, L, H, D = 8, 8192, 16, 128
    run_rope_attention(B, L, H, D, 100000.0, seed=0, bh=[(0, 0), (7, 15), (3, 8)])


@pytest.mark.parametrize("B,L,H,D,base,docs,doc_pos", [
    (2, 300, 3, 64, 10000.0, False, False),     # persistent forward
    (2, 300, 3, 128, 100000.0, True, True),
    (48, 700, 3, 64, 100000.0, True, False),    # several items per workgroup
    (1, 4100, 2, 64, 10000.0, False, False),    # one block per workgroup, ragged
    (1, 16384, 1, 128, 10000.0, True, True),    # long positions
    (3, 1000, 2, 128, 500000.0, False, False),
])
def test_fused_query_rotation_is_bit_identical(cuda, B, L, H, D, base, docs, doc_pos):
    # The forward that rotates q as it loads it gives the same rotated q, O
    # and LSE, bit for bit, as a dd_rope pass followed by dd_attn_fwd.
    import paper_2405_13226_amd as pkg
    log(f"fused rope forward B={B} L={L} H={H} D={D} base={base:g} docs={docs} doc_pos={doc_pos}")
    inp = synth.attention_inputs(B, L, H, D, seed=L + D, with_grad=False)
    q, k, v = (to_dev(inp[n], cuda_dev()) for n in ("q", "k", "v"))
    cu = None
    if docs:
        lens = synth.lognormal_doc_lengths(L, total_tokens=B * L, median=200, sigma=1.0)
        cu = dd.chunk_doclens(lens, B * L)
    f = pkg.forward_rope(q, k, v, base, True, cu, doc_pos, fused=True)
    u = pkg.forward_rope(q, k, v, base, True, cu, doc_pos, fused=False)
    torch.cuda.synchronize()
    for name, a, b in zip(("o", "lse", "q_rot", "k_rot"), f, u):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b), name


def test_rope_dd_equals_masked_chunk_with_document_positions(cuda):
    # Equal-length documents packed in chunks with document-local positions are
    # the same bytes as the DD batch of those documents with row positions.
    import paper_2405_13226_amd as pkg
    Bc, L, H, D, ell, base = 2, 1024, 2, 128, 256, 10000.0
    inp = synth.attention_inputs(Bc, L, H, D, seed=9, with_grad=True)
    q, k, v, do = (to_dev(inp[n], cuda_dev()) for n in ("q", "k", "v", "do"))
    cu = np.arange(0, Bc * L + 1, ell)
    m = pkg.forward_rope(q, k, v, base, True, cu, True)
    mg = pkg.backward_rope(m[2], m[3], v, m[0], m[1], do, base, True, cu, True)
    view = lambda t: t.view(Bc * L // ell, ell, H, D)
    d = pkg.forward_rope(view(q), view(k), view(v), base)
    dg = pkg.backward_rope(d[2], d[3], view(v), d[0], d[1], view(do), base)
    torch.cuda.synchronize()
    # rotations agree bitwise (same positions); attention outputs within tolerance
    assert torch.equal(view(m[2]), d[2]) and torch.equal(view(m[3]), d[3])
    for a, b in zip((m[0],) + tuple(mg), (d[0],) + tuple(dg)):
        a, b = to_f64(view(a)), to_f64(b)
        assert rel_l2(a, b) <= 1e-2, rel_l2(a, b)


def test_autograd_matches_functional(cuda):
    import paper_2405_13226_amd as pkg
    B, L, H, D, base = 2, 200, 2, 64, 10000.0
    inp = synth.attention_inputs(B, L, H, D, seed=4, with_grad=True)
    q, k, v, do = (to_dev(inp[n], cuda_dev()) for n in ("q", "k", "v", "do"))
    qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
    out = pkg.attention(qa, ka, va, rope_base=base)
    out.backward(do)
    o, lse, qr, kr = pkg.forward_rope(q, k, v, base)
    g = pkg.backward_rope(qr, kr, v, o, lse, do, base)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), o)
    for a, b in zip((qa.grad, ka.grad, va.grad), g):
        assert torch.equal(a, b)


def _rope_cases(n=12, seed=239):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        D = int(rng.choice([64, 128]))
        L = int(rng.choice([int(rng.integers(1, 200)), int(rng.integers(200, 1500))]))
        B, H = int(rng.integers(1, 30)), int(rng.integers(1, 7))
        base = float(rng.choice([10000.0, 100000.0]))
        cu, doc_pos = None, False
        if rng.random() < 0.5 and B * L >= 2:
            lens = synth.lognormal_doc_lengths(int(rng.integers(1 << 30)), total_tokens=B * L,
                                               median=float(rng.choice([60, 300])), sigma=1.0)
            cu = dd.chunk_doclens(lens, B * L)
            doc_pos = bool(rng.random() < 0.5)
        bh = sorted({(int(rng.integers(B)), int(rng.integers(H))) for _ in range(3)})
        out.append((i, B, L, H, D, base, cu, doc_pos, bh))
    return out


@pytest.mark.parametrize("case", _rope_cases(), ids=lambda c: f"case{c[0]}")
def test_attention_rope_random_configuration(cuda, case):
    # Seeded random shapes, bases and document layouts (row or document-local
    # positions), three sampled (b, h) slices each.
    i, B, L, H, D, base, cu, doc_pos, bh = case
    run_rope_attention(B, L, H, D, base, cu, doc_pos, seed=300 + i, bh=bh)
