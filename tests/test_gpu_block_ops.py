"""GPU parity of the block kernels around the attention (the bf16 GEMM, the
LayerNorm and the SwiGLU of one OpenLM block) through the C ABI, against
plain float64 numpy definitions of the same operations on the same bf16
inputs.

Tolerances: every output is rounded to bf16 once (RMS relative rounding
error 2^-9 / sqrt(3) ~ 1.1e-3 over a binade, measured 1.66e-3 relative L2 on
N(0,1) products); fp32 accumulation adds far less at these depths.  Bound:
relative L2 <= 3e-3 per output.  The LayerNorm parameter gradients (sums
over all rows) and the outputs with a residual (two roundings) use 5e-3.
"""
import numpy as np
import pytest
import torch

from paper_2405_13226_amd import block_ops as ops

from parity import log, rel_l2

pytestmark = pytest.mark.gpu
RTOL, RTOL2 = 3e-3, 5e-3


def bf16(shape, seed, scale=1.0):
    g = torch.Generator(device="cpu").manual_seed(seed)
    return (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)


def f64(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("M,N,K,ta,tb", [
    (256, 256, 64, 0, 0), (512, 768, 320, 0, 1), (768, 512, 192, 1, 0),
    (1024, 512, 8192, 1, 0),      # long K: split over several workgroups
    # 40 tile rows (5 per XCD: a band of 4 rows and one of 1) and 11 tile
    # columns (column groups of 8 and 3) in the grouped tile order
    (10240, 2816, 128, 0, 0), (10240, 2816, 128, 0, 1),
    (65536, 2048, 2048, 0, 0),    # the block's output projection at 65,536 tokens
    (2048, 2048, 65536, 1, 0),    # its weight gradient
])
def test_gemm(cuda, M, N, K, ta, tb):
    log(f"gemm M={M} N={N} K={K} ta={ta} tb={tb}")
    a = bf16((K, M) if ta else (M, K), M + K)
    b = bf16((N, K) if tb else (K, N), N + K + 1)
    c = ops.gemm(a.to(cuda), b.to(cuda), bool(ta), bool(tb))
    torch.cuda.synchronize()
    if M * N * K > 2 ** 33:  # sampled rows at full size
        rows = np.random.default_rng(0).choice(M, 64, replace=False)
        an = f64(a.t() if ta else a)[rows]
        ref = an @ f64(b.t() if tb else b)
        got = f64(c)[rows]
    else:
        ref = f64(a.t() if ta else a) @ f64(b.t() if tb else b)
        got = f64(c)
    err = rel_l2(got, ref)
    log(f"  rel-L2 {err:.3g}")
    assert err <= RTOL


def test_gemm_strided_slices_and_residual(cuda):
    # Column slices of wider matrices as operands and output (row strides
    # passed through), and the residual added in place.
    M, K, N, W = 512, 256, 256, 768
    a = bf16((M, K), 1).to(cuda)
    wide = bf16((K, W), 2).to(cuda)
    out = torch.zeros((M, W), dtype=torch.bfloat16, device=cuda)
    res = bf16((M, N), 3).to(cuda)
    acc = res.clone()
    ops.gemm(a, wide[:, 256:512], out=out[:, 512:768])
    ops.gemm(a, wide[:, 0:256], residual=acc, out=acc)
    torch.cuda.synchronize()
    ref = f64(a) @ f64(wide)[:, 256:512]
    assert rel_l2(f64(out)[:, 512:768], ref) <= RTOL
    assert np.all(f64(out)[:, :512] == 0)  # nothing written outside the slice
    ref2 = f64(a) @ f64(wide)[:, 0:256] + f64(res)
    assert rel_l2(f64(acc), ref2) <= RTOL2


def ln_ref(x, w, b, dy, dres, eps=1e-5):
    mu = x.mean(1, keepdims=True)
    var = ((x - mu) ** 2).mean(1, keepdims=True)
    rstd = 1 / np.sqrt(var + eps)
    xh = (x - mu) * rstd
    y = xh * w + b
    g = dy * w
    dx = rstd * (g - g.mean(1, keepdims=True) - xh * (g * xh).mean(1, keepdims=True)) + dres
    return y, dx, (dy * xh).sum(0), dy.sum(0), mu[:, 0], rstd[:, 0]


@pytest.mark.parametrize("rows,d", [(100, 512), (777, 1024), (4096, 2048)])
def test_layer_norm(cuda, rows, d):
    x = bf16((rows, d), rows, 2.0) + 0.5
    w, b = bf16((d,), 5) * 0.3 + 1, bf16((d,), 6) * 0.3
    dy, dres = bf16((rows, d), 7), bf16((rows, d), 8)
    X, W_, B_ = x.to(cuda), w.to(cuda), b.to(cuda)
    y, mean, rstd = ops.layer_norm(X, W_, B_)
    dx, dw, db = ops.layer_norm_backward(X, W_, mean, rstd, dy.to(cuda), dres.to(cuda))
    torch.cuda.synchronize()
    ry, rdx, rdw, rdb, rmu, rrs = ln_ref(f64(x), f64(w), f64(b), f64(dy), f64(dres))
    res = {"y": rel_l2(f64(y), ry), "dx": rel_l2(f64(dx), rdx), "dw": rel_l2(f64(dw), rdw),
           "db": rel_l2(f64(db), rdb),
           "mean": float(np.abs(mean.cpu().numpy() - rmu).max()),
           "rstd": float(np.abs(rstd.cpu().numpy() / rrs - 1).max())}
    log(f"  layernorm rows={rows} d={d}: " + "  ".join(f"{k}={v:.3g}" for k, v in res.items()))
    assert res["y"] <= RTOL and res["dx"] <= RTOL2
    assert res["dw"] <= RTOL2 and res["db"] <= RTOL2
    assert res["mean"] <= 1e-5 and res["rstd"] <= 1e-5


@pytest.mark.parametrize("R,C,pad", [(64, 64, 0), (192, 320, 0), (2048, 5632, 0),
                                     (5632, 2048, 64)])
def test_transpose(cuda, R, C, pad):
    # bit-exact against the transposed copy; pad > 0: strided views in and out
    x = bf16((R, C + pad), 7)
    xd = x.to(cuda)[:, pad // 2:pad // 2 + C]
    y = torch.empty((C, R + 2 * pad), dtype=torch.bfloat16, device=cuda)[:, :R]
    ops.transpose(xd, out=y)
    torch.cuda.synchronize()
    ref = x[:, pad // 2:pad // 2 + C].view(torch.int16).numpy().T
    assert np.array_equal(y.cpu().view(torch.int16).numpy(), ref)


def test_swiglu(cuda):
    n = 3 * 1024 * 8 + 64
    u, v, dy = bf16((n,), 1, 3.0), bf16((n,), 2), bf16((n,), 3)
    y = ops.swiglu(u.to(cuda), v.to(cuda))
    du, dv = ops.swiglu_backward(u.to(cuda), v.to(cuda), dy.to(cuda))
    torch.cuda.synchronize()
    U, V, DY = f64(u), f64(v), f64(dy)
    sig = 1 / (1 + np.exp(-U))
    assert rel_l2(f64(y), U * sig * V) <= RTOL
    assert rel_l2(f64(du), DY * V * sig * (1 + U * (1 - sig))) <= RTOL
    assert rel_l2(f64(dv), DY * U * sig) <= RTOL
