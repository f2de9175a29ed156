"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
on seeded inputs and compare with the fp64 oracle.

Tolerances (bf16 inputs, fp32 accumulation):
* forward O: |o - o_ref| <= 1e-2 + half a bf16 ulp of o_ref, elementwise.
  The extra half ulp is the rounding of the bf16 output format itself, which
  alone exceeds 1e-2 once |o| >= 4 (early causal rows with few keys).
* LSE: max-abs <= 1e-3 (fp32 output).
* dQ, dK, dV: relative L2 error <= 1e-2 per tensor over the compared rows,
  and the same bound on the worst (b, h) slice and on the worst block of
  ROW_BLOCK consecutive rows of a slice, so that a local error (one wrong key
  block, one wrong slice) cannot hide in the pooled norm; where the exact
  gradient is identically zero (L = 1), max-abs <= 1e-5.  Slices and blocks
  whose exact gradient is identically zero are held to the max-abs bound
  instead.
"""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle
import synth

FWD_ATOL = 1e-2
LSE_ATOL = 1e-3
BWD_RTOL = 1e-2
ZERO_ATOL = 1e-5  # bound where the exact gradient is identically zero
ROW_BLOCK = 128   # rows per block of the blockwise gradient check


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(bits, device):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device)
    return t.view(torch.bfloat16)


def to_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def half_ulp_bf16(x):
    ax = np.abs(x)
    e = np.floor(np.log2(np.maximum(ax, 2.0 ** -126)))
    return 0.5 * 2.0 ** (e - 7)


def rel_l2(a, b):
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-30))


def local_errors(got, ref, rows=ROW_BLOCK):
    """Worst relative L2 error over the (b, h) slices of [n_bh, L, D] arrays,
    and over blocks of `rows` consecutive rows of each slice; a ragged tail
    joins the block before it, so every block holds at least `rows` rows (or
    the whole slice).  A block is kept that long because one row's relative
    error is not bounded by the tolerance: delta = rowsum(dO * O) is formed
    from the bf16-rounded forward output, which moves dP - delta by an
    absolute amount, so a key seen by one query with a small dP - delta (a
    dK row of norm ~0.01) can carry a few per cent of relative error while
    the 128-row block around it stays far below 1e-2.  Slices or blocks whose
    reference is exactly zero are left out of the relative figures; the
    largest absolute error on them is returned as the third value (0 if
    there are none)."""
    worst_slice = worst_block = zero_abs = 0.0
    for g, r in zip(got, ref):
        n = r.shape[0]
        starts = list(range(0, max(n - rows, 0) + 1, rows)) if n >= rows else [0]
        ends = starts[1:] + [n]
        spans = [(0, n)] + list(zip(starts, ends))
        for k, (lo, hi) in enumerate(spans):
            den = float(np.linalg.norm(r[lo:hi].ravel()))
            diff = g[lo:hi] - r[lo:hi]
            if den == 0.0:
                zero_abs = max(zero_abs, float(np.abs(diff).max()))
            elif k == 0:
                worst_slice = max(worst_slice, float(np.linalg.norm(diff.ravel())) / den)
            else:
                worst_block = max(worst_block, float(np.linalg.norm(diff.ravel())) / den)
    return worst_slice, worst_block, zero_abs


def gpu_run(inputs, causal, cu, device, backward=True):
    import paper_2405_13226_amd as dd
    q, k, v = (to_dev(inputs[n], device) for n in ("q", "k", "v"))
    o, lse = dd.forward(q, k, v, causal=causal, cu_doclens=cu)
    out = {"o": o, "lse": lse}
    if backward:
        do = to_dev(inputs["do"], device)
        dq, dk, dv = dd.backward(q, k, v, o, lse, do, causal=causal, cu_doclens=cu)
        out.update(dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize(device)
    return out


def select_bh(x, bh):
    """[B, L, H, ...] -> [n_bh, L, ...] for the listed pairs."""
    return np.stack([x[b, :, h] for b, h in bh])


def compare(inputs, out, causal, cu, bh, backward=True, tag=""):
    """Oracle on the listed (b, h) pairs vs the GPU outputs; returns errors."""
    t0 = time.time()
    o_ref, lse_ref = oracle.attn_fwd(inputs["q"], inputs["k"], inputs["v"],
                                     causal=causal, cu_doclens=cu, bh=bh)
    o = select_bh(to_f64(out["o"]), bh)
    lse = select_bh(out["lse"].cpu().numpy().astype(np.float64), bh)
    err_o = np.abs(o - o_ref)
    bound = FWD_ATOL + half_ulp_bf16(o_ref)
    res = {"o_maxabs": float(err_o.max()), "o_excess": float((err_o - bound).max()),
           "lse_maxabs": float(np.abs(lse - lse_ref).max())}
    if backward:
        g_ref = oracle.attn_bwd(inputs["q"], inputs["k"], inputs["v"], inputs["do"],
                                causal=causal, cu_doclens=cu, bh=bh)
        for name, ref in zip(("dq", "dk", "dv"), g_ref):
            got = select_bh(to_f64(out[name]), bh)
            if np.linalg.norm(ref.ravel()) > 0:
                res[name + "_rel"] = rel_l2(got, ref)
                sl, bl, za = local_errors(got, ref)
                res[name + "_slice"] = sl
                res[name + "_block"] = bl
                res[name + "_zabs"] = za
            else:  # zero reference (e.g. L = 1): relative error undefined
                res[name + "_abs"] = float(np.abs(got - ref).max())
    log(f"  [{tag}] oracle {time.time() - t0:.1f}s  " +
        "  ".join(f"{k}={v:.3g}" for k, v in res.items()))
    return res


def assert_ok(res, backward=True):
    assert res["o_excess"] <= 0.0, res
    assert res["lse_maxabs"] <= LSE_ATOL, res
    if backward:
        for n in ("dq", "dk", "dv"):
            if n + "_rel" in res:
                assert res[n + "_rel"] <= BWD_RTOL, res
                assert res[n + "_slice"] <= BWD_RTOL, res
                assert res[n + "_block"] <= BWD_RTOL, res
                assert res[n + "_zabs"] <= ZERO_ATOL, res
            else:
                assert res[n + "_abs"] <= ZERO_ATOL, res


def check_case(B, L, H, D, causal=True, cu=None, seed=0, bh=None, device="cuda:0",
               backward=True, tag=None):
    tag = tag or f"B={B} L={L} H={H} D={D} causal={int(causal)} docs={None if cu is None else len(cu) - 1}"
    log(f"case {tag} seed={seed}")
    inputs = synth.attention_inputs(B, L, H, D, seed=seed, with_grad=backward)
    out = gpu_run(inputs, causal, cu, device, backward)
    for n, t in out.items():
        assert torch.isfinite(t.float()).all(), f"{n} has non-finite values"
    if bh is None:
        bh = [(b, h) for b in range(B) for h in range(H)]
    res = compare(inputs, out, causal, cu, bh, backward, tag)
    assert_ok(res, backward)
    return inputs, out, res
