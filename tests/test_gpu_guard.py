"""Guard bands and a closed form on the GPU.

* Out-of-bounds writes: every output of dd_attn_fwd, dd_attn_bwd(_rope) and
  dd_rope is placed inside a larger buffer whose bytes before and after it
  hold a canary pattern; after the calls, every canary byte must be intact.
  Shapes are ragged (L not a multiple of any tile, B*L odd, documents crossing
  rows) so that partial tiles and clamped rows are exercised.
* Q = 0: every score is 0, so row i of O is the mean of the V rows its query
  may see and LSE_i = ln |A_i| (exact up to the bf16 output rounding).
"""
import ctypes

import numpy as np
import pytest
import torch

import synth
from paper_2405_13226_amd import dd as ddhost
import paper_2405_13226_amd as dd

from parity import half_ulp_bf16, log, to_dev, to_f64

pytestmark = pytest.mark.gpu

PAD = 4096  # canary bytes on each side (multiple of 256 keeps alignment)
CANARY = 0xA5


class Guarded:
    """A tensor of `shape`/`dtype` inside a byte buffer with canary bands."""

    def __init__(self, shape, dtype, dev):
        n = int(np.prod(shape)) * torch.empty(0, dtype=dtype).element_size()
        self.raw = torch.full((PAD + n + PAD,), CANARY, dtype=torch.uint8, device=dev)
        self.t = self.raw[PAD:PAD + n].view(dtype).view(shape)

    def intact(self):
        head, tail = self.raw[:PAD], self.raw[-PAD:]
        return bool((head == CANARY).all() and (tail == CANARY).all())


# (90, 200, 3, 64): 270 slices for the persistent one-kernel backward's 256
# workgroups, so some take a second slice (staged during their first).
@pytest.mark.parametrize("B,L,H,D,docs", [(3, 77, 3, 64, False), (1, 1, 1, 128, False),
                                          (5, 129, 2, 128, True), (2, 1000, 1, 64, True),
                                          (90, 200, 3, 64, True), (90, 200, 3, 64, False)])
def test_outputs_stay_inside_their_buffers(cuda, B, L, H, D, docs):
    log(f"guard B={B} L={L} H={H} D={D} docs={docs}")
    x = {n: to_dev(a, cuda) for n, a in synth.attention_inputs(B, L, H, D, seed=L).items()}
    cu = None
    if docs:
        lens = synth.lognormal_doc_lengths(1, total_tokens=B * L, median=60, sigma=1.0)
        cu = ddhost.chunk_doclens(lens, B * L)
    P = ctypes.c_void_p
    lib = dd.lib()
    st = P(torch.cuda.current_stream().cuda_stream)
    docs_d = dd.DocLens(cu, B * L, cuda) if cu is not None else None
    cup, nd = (P(docs_d.dev.data_ptr()), docs_d.n_docs) if docs_d else (None, 0)
    o, lse = Guarded((B, L, H, D), torch.bfloat16, cuda), Guarded((B, L, H), torch.float32, cuda)
    assert lib.dd_attn_fwd(P(x["q"].data_ptr()), P(x["k"].data_ptr()), P(x["v"].data_ptr()),
                           P(o.t.data_ptr()), P(lse.t.data_ptr()), B, L, H, D, 1, cup, nd, st) == 0
    ws_bytes = lib.dd_attn_bwd_workspace_bytes(B, L, H, D)
    ws = Guarded((ws_bytes,), torch.uint8, cuda)
    grads = [Guarded((B, L, H, D), torch.bfloat16, cuda) for _ in range(3)]
    args = [P(t.data_ptr()) for t in (x["q"], x["k"], x["v"], o.t, x["do"], lse.t)]
    args += [P(gt.t.data_ptr()) for gt in grads]
    assert lib.dd_attn_bwd(*args, B, L, H, D, 1, cup, nd, P(ws.t.data_ptr()),
                           ctypes.c_size_t(ws_bytes), st) == 0
    grads_r = [Guarded((B, L, H, D), torch.bfloat16, cuda) for _ in range(3)]
    args_r = args[:6] + [P(gt.t.data_ptr()) for gt in grads_r]
    assert lib.dd_attn_bwd_rope(*args_r, B, L, H, D, 1, cup, nd, 10000.0, 1 if docs else 0,
                                P(ws.t.data_ptr()), ctypes.c_size_t(ws_bytes), st) == 0
    rot = Guarded((B, L, H, D), torch.bfloat16, cuda)
    assert lib.dd_rope(P(x["q"].data_ptr()), P(rot.t.data_ptr()), B, L, H, D, 10000.0, 0, cup,
                       nd, 1 if docs else 0, st) == 0
    torch.cuda.synchronize()
    for name, g in [("o", o), ("lse", lse), ("ws", ws), ("rot", rot)] + \
            [(f"grad{i}", gg) for i, gg in enumerate(grads + grads_r)]:
        assert g.intact(), name
    assert torch.isfinite(o.t.float()).all()


@pytest.mark.parametrize("D,docs", [(64, False), (128, True)])
def test_zero_queries_give_prefix_means(cuda, D, docs):
    B, L, H = 2, 300, 2
    x = synth.attention_inputs(B, L, H, D, seed=D, with_grad=False)
    cu = None
    if docs:
        cu = ddhost.chunk_doclens(synth.lognormal_doc_lengths(2, total_tokens=B * L, median=70,
                                                              sigma=1.0), B * L)
    q = torch.zeros(B, L, H, D, dtype=torch.bfloat16, device=cuda)
    o, lse = dd.forward(q, to_dev(x["k"], cuda), to_dev(x["v"], cuda), cu_doclens=cu)
    torch.cuda.synchronize()
    v = x["v"]
    vf = (v.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    # allowed keys of query i in row b: [start of its document in the row, i]
    starts = np.zeros((B, L), dtype=np.int64)
    if cu is not None:
        cu = np.asarray(cu)
        for b in range(B):
            for i in range(L):
                t = b * L + i
                starts[b, i] = max(cu[cu <= t].max(), b * L) - b * L
    exp_o = np.empty((B, L, H, D))
    for b in range(B):
        cs = np.cumsum(vf[b], axis=0)  # [L, H, D]
        for i in range(L):
            s = starts[b, i]
            tot = cs[i] - (cs[s - 1] if s > 0 else 0)
            exp_o[b, i] = tot / (i - s + 1)
    exp_lse = np.log((np.arange(L)[None, :] - starts + 1).astype(np.float64))[:, :, None]
    got_o = to_f64(o)
    assert np.all(np.abs(got_o - exp_o) <= 1e-2 + half_ulp_bf16(exp_o))
    assert np.abs(lse.cpu().numpy() - exp_lse).max() <= 1e-5
