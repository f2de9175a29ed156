"""Tensors of 2^32 elements (8 GiB each at D = 128): element offsets past 2^31
and byte offsets past 2^32 in every kernel (forward, delta, dK/dV, dQ),
checked against the fp64 oracle on (b, h) slices at the start, past 2^31
elements, and at the very end of the tensors.

The inputs are drawn on the device (seeded torch normal in bf16); the oracle
receives the exact bf16 values of the sampled slices, packed as a small batch
[n, L, 1, D] (pairs are independent and positions are row-local, so the
packed batch computes the same numbers as those slices of the large one).
"""
import numpy as np
import pytest
import torch

from parity import assert_ok, compare, log

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def test_offsets_beyond_32_bits(cuda):
    import paper_2405_13226_amd as dd

    B, L, H, D = 8192, 256, 16, 128
    n_elem = B * L * H * D
    assert n_elem == 1 << 32
    dev = torch.device("cuda:0")
    need = 8 * n_elem * 2 + (3 << 30)  # 8 bf16 tensors, LSE and workspace
    free, _ = torch.cuda.mem_get_info(dev)
    if free < need:
        pytest.skip(f"needs {need / 2**30:.0f} GiB of device memory, {free / 2**30:.0f} free")
    log(f"large case B={B} L={L} H={H} D={D}: {n_elem} elements per tensor")
    g = torch.Generator(device=dev).manual_seed(2024)
    ins = {}
    for name in ("q", "k", "v", "do"):
        t = torch.empty(B, L, H, D, dtype=torch.bfloat16, device=dev)
        for b0 in range(0, B, 1024):
            t[b0:b0 + 1024].normal_(generator=g)
        ins[name] = t
    o, lse = dd.forward(ins["q"], ins["k"], ins["v"])
    dq, dk, dv = dd.backward(ins["q"], ins["k"], ins["v"], o, lse, ins["do"])
    torch.cuda.synchronize(dev)
    log("  large case: kernels done")

    # (b, h) slices: the first, one past 2^31 elements, and the last ones
    # (their bytes lie past 2^32).
    bh = [(0, 0), (B // 2, 1), (B - 1, 0), (B - 1, H - 1)]
    assert (B // 2) * L * H * D >= 1 << 31 and 2 * (B - 1) * L * H * D > 1 << 32
    small_in = {n: np.stack([_bits(t[b, :, h])[:, None, :] for b, h in bh])
                for n, t in ins.items()}
    small_out = {n: torch.stack([t[b, :, h] for b, h in bh]).unsqueeze(2)
                 for n, t in (("o", o), ("dq", dq), ("dk", dk), ("dv", dv))}
    small_out["lse"] = torch.stack([lse[b, :, h] for b, h in bh]).unsqueeze(2)
    del ins, o, lse, dq, dk, dv
    torch.cuda.empty_cache()
    res = compare(small_in, small_out, True, None, [(i, 0) for i in range(len(bh))],
                  tag="large, 2^32 elements")
    assert_ok(res)
