"""fp64 oracle for one OpenLM transformer block (forward and backward).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never imports it.

The paper trains OpenLM models (Sec. 3.1; Appendix, Tables "openlm1b" etc.:
OpenLM-1B has hidden dimension 2048, 24 layers, 16 heads and 1,439,893,504
parameters) with RoPE (Sec. 3, "Positional encoding").  Readings where the
paper is silent, fixed by matching that parameter count exactly with a
50,432-token vocabulary and untied embeddings:
  * pre-norm block: x + Attn(LN1(x)), then h + MLP(LN2(h));
  * LayerNorm with weight and bias (eps 1e-5); projections without bias;
  * attention: q, k, v = LN1(x) W_qkv split into H heads of D = d / H, RoPE on
    q and k, causal (document-masked) softmax attention, output W_o;
  * SwiGLU MLP with hidden width 5632: (silu(x W_1) * (x W_3)) W_2;
so a block holds 4 d^2 + 3 d h + 4 d = 51,388,416 parameters at d = 2048.

Arithmetic: float64 throughout; attention and RoPE come from the pinned
attention oracle (``oracle.rope``, exact rotation).  Weights are passed in as
arrays; weight matrices map rows (tokens) by right multiplication.
"""
from __future__ import annotations

import numpy as np
import torch

from . import to_blhd
from . import rope as _rope

LN_EPS = 1e-5


def openlm_block_params(d: int, hidden: int) -> int:
    """Parameters of one block under the readings above."""
    return 4 * d * d + 3 * d * hidden + 4 * d


class _Attention(torch.autograd.Function):
    """Attention over rotated q, k via the fp64 oracle (numpy)."""

    @staticmethod
    def forward(ctx, q, k, v, base, cu, doc_positions):
        B, L, H, D = q.shape
        args = (q.detach().numpy(), k.detach().numpy(), v.detach().numpy())
        if base:
            o, _ = _rope.attn_fwd(*args, base, True, cu, doc_positions, round_rotated=False)
        else:
            from . import attn_fwd
            o, _ = attn_fwd(*args, causal=True, cu_doclens=cu)
        ctx.save_for_backward(q, k, v)
        ctx.cfg = (base, cu, doc_positions)
        return torch.from_numpy(to_blhd(o, B, H))

    @staticmethod
    def backward(ctx, do):
        q, k, v = ctx.saved_tensors
        base, cu, docpos = ctx.cfg
        B, L, H, D = q.shape
        args = (q.numpy(), k.numpy(), v.numpy(), do.contiguous().numpy())
        if base:
            g = _rope.attn_bwd(*args, base, True, cu, docpos, round_rotated=False)
        else:
            from . import attn_bwd
            g = attn_bwd(*args, causal=True, cu_doclens=cu)
        dq, dk, dv = (torch.from_numpy(to_blhd(x, B, H)) for x in g)
        return dq, dk, dv, None, None, None


def block_forward(x, w, H: int, rope_base=None, cu_doclens=None, doc_positions=False):
    """One block on x [B, L, d] (float64 torch tensors; w: dict of tensors
    ln1_w, ln1_b, w_qkv [d, 3d], w_o [d, d], ln2_w, ln2_b, w_1 [d, h],
    w_3 [d, h], w_2 [h, d]).  Differentiable with torch autograd."""
    B, L, d = x.shape
    D = d // H
    a = torch.nn.functional.layer_norm(x, (d,), w["ln1_w"], w["ln1_b"], LN_EPS)
    qkv = a @ w["w_qkv"]
    q, k, v = (t.reshape(B, L, H, D).contiguous() for t in qkv.split(d, dim=-1))
    o = _Attention.apply(q, k, v, rope_base, cu_doclens, doc_positions)
    h = x + o.reshape(B, L, d) @ w["w_o"]
    m = torch.nn.functional.layer_norm(h, (d,), w["ln2_w"], w["ln2_b"], LN_EPS)
    y = h + (torch.nn.functional.silu(m @ w["w_1"]) * (m @ w["w_3"])) @ w["w_2"]
    return y


def block_fwd_bwd(x, w, dy, H: int, rope_base=None, cu_doclens=None, doc_positions=False):
    """Forward output and gradients of sum(dy * y) with respect to x and every
    weight.  Inputs are numpy arrays (any float dtype) widened to float64."""
    xt = torch.tensor(np.asarray(x, dtype=np.float64), requires_grad=True)
    wt = {n: torch.tensor(np.asarray(a, dtype=np.float64), requires_grad=True)
          for n, a in w.items()}
    y = block_forward(xt, wt, H, rope_base, cu_doclens, doc_positions)
    y.backward(torch.tensor(np.asarray(dy, dtype=np.float64)))
    grads = {n: t.grad.numpy() for n, t in wt.items()}
    grads["x"] = xt.grad.numpy()
    return y.detach().numpy(), grads
