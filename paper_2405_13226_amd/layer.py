"""One OpenLM transformer block on the GPU (forward and backward).

The paper's models are OpenLM transformers (Sec. 3.1; Table "openlm1b":
hidden dimension 2048, 24 layers, 16 heads, 1,439,893,504 parameters) with
RoPE (Sec. 3, "Positional encoding").  The block, with the readings that
reproduce that parameter count exactly (50,432-token vocabulary, untied
embeddings):

    a = LayerNorm_1(x);  q, k, v = a W_qkv   (H heads of D = d / H)
    h = x + Attention(RoPE(q), RoPE(k), v) W_o
    m = LayerNorm_2(h);  y = h + (silu(m W_1) * (m W_3)) W_2

LayerNorms have weight and bias, projections have none, the SwiGLU width is
5632 at d = 2048.  Every step runs in this library's HIP kernels: the
projections and the MLP products in its bf16 GEMM (the residual additions in
the GEMM epilogue; the forward multiplies by transposed copies of the weights,
made by its transpose kernel at the start of the step, so that both operands
of every forward product are read along rows, the GEMM's faster form), the
LayerNorms and the SwiGLU in its elementwise kernels,
RoPE and attention in the attention kernels; the backward is written out
step by step (one autograd node for the whole block).  The block exists to
place the attention hot path in a full layer step: its time as a share of
the step, and the step time's growth with the sequence length at a fixed
token budget.  Shapes: B*L, d and the SwiGLU width multiples of 256, d in
{512, 1024, 2048}, d / H in {64, 128}.
"""
from __future__ import annotations

import torch

from . import block_ops as ops
from .attention import _doclens, backward_rope, forward_rope

LN_EPS = 1e-5
OPENLM_1B = dict(d=2048, H=16, hidden=5632)


class _BlockFunction(torch.autograd.Function):
    """Forward and backward of one block on x [T, d] (T = B * L tokens)."""

    @staticmethod
    def forward(ctx, x, ln1_w, ln1_b, w_qkv, w_o, ln2_w, ln2_b, w_1, w_3, w_2, shape, base,
                docs, doc_pos):
        B, L, H, D = shape
        d = H * D
        # transposed weight copies: every forward product then reads both of
        # its operands along rows (the GEMM's faster operand form)
        t_qkv, t_o, t_1, t_3, t_2 = (ops.transpose(w) for w in (w_qkv, w_o, w_1, w_3, w_2))
        a, mean1, rstd1 = ops.layer_norm(x, ln1_w, ln1_b, LN_EPS)
        q, k, v = (ops.gemm(a, t_qkv[i * d:(i + 1) * d], trans_b=True) for i in range(3))
        o, lse, qr, kr = forward_rope(q.view(B, L, H, D), k.view(B, L, H, D),
                                      v.view(B, L, H, D), base, True, docs, doc_pos)
        o2 = o.view(B * L, d)
        h = ops.gemm(o2, t_o, trans_b=True, residual=x)
        m, mean2, rstd2 = ops.layer_norm(h, ln2_w, ln2_b, LN_EPS)
        u1, u3 = ops.gemm(m, t_1, trans_b=True), ops.gemm(m, t_3, trans_b=True)
        g = ops.swiglu(u1, u3)
        y = ops.gemm(g, t_2, trans_b=True, residual=h)
        del t_qkv, t_o, t_1, t_3, t_2
        ctx.save_for_backward(x, ln1_w, w_qkv, w_o, ln2_w, w_1, w_3, w_2, a, mean1, rstd1, qr,
                              kr, v, o, lse, h, m, mean2, rstd2, u1, u3, g)
        ctx.cfg = (shape, base, docs, doc_pos)
        return y

    @staticmethod
    def backward(ctx, dy):
        (x, ln1_w, w_qkv, w_o, ln2_w, w_1, w_3, w_2, a, mean1, rstd1, qr, kr, v, o, lse, h, m,
         mean2, rstd2, u1, u3, g) = ctx.saved_tensors
        (B, L, H, D), base, docs, doc_pos = ctx.cfg
        d = H * D
        dy = dy.contiguous()
        # MLP: y = h + swiglu(m W1, m W3) W2
        dg = ops.gemm(dy, w_2, trans_b=True)
        dw_2 = ops.gemm(g, dy, trans_a=True)
        du1, du3 = ops.swiglu_backward(u1, u3, dg)
        dm = ops.gemm(du1, w_1, trans_b=True)
        ops.gemm(du3, w_3, trans_b=True, residual=dm, out=dm)
        dw_1 = ops.gemm(m, du1, trans_a=True)
        dw_3 = ops.gemm(m, du3, trans_a=True)
        dh, dln2_w, dln2_b = ops.layer_norm_backward(h, ln2_w, mean2, rstd2, dm, dres=dy)
        # attention: h = x + attn(RoPE(q), RoPE(k), v) Wo
        do = ops.gemm(dh, w_o, trans_b=True)
        dw_o = ops.gemm(o.view(B * L, d), dh, trans_a=True)
        dq, dk, dv = backward_rope(qr, kr, v.view(B, L, H, D), o, lse, do.view(B, L, H, D),
                                   base, True, docs, doc_pos)
        grads = [t.view(B * L, d) for t in (dq, dk, dv)]
        da = ops.gemm(grads[0], w_qkv[:, :d], trans_b=True)
        for i in (1, 2):
            ops.gemm(grads[i], w_qkv[:, i * d:(i + 1) * d], trans_b=True, residual=da, out=da)
        dw_qkv = torch.empty_like(w_qkv)
        for i in range(3):
            ops.gemm(a, grads[i], trans_a=True, out=dw_qkv[:, i * d:(i + 1) * d])
        dx, dln1_w, dln1_b = ops.layer_norm_backward(x, ln1_w, mean1, rstd1, da, dres=dh)
        return (dx, dln1_w, dln1_b, dw_qkv, dw_o, dln2_w, dln2_b, dw_1, dw_3, dw_2,
                None, None, None, None)


class OpenLMBlock(torch.nn.Module):
    def __init__(self, d: int = 2048, H: int = 16, hidden: int = 5632, rope_base=100000.0,
                 device="cuda", dtype=torch.bfloat16, seed: int = 0, init_scale: float = 0.02):
        super().__init__()
        if d % H:
            raise ValueError("d must be a multiple of H")
        self.d, self.H, self.D, self.hidden = d, H, d // H, hidden
        self.rope_base = rope_base
        g = torch.Generator(device="cpu").manual_seed(seed)

        def mat(*shape):
            w = torch.randn(*shape, generator=g) * init_scale
            return torch.nn.Parameter(w.to(device=device, dtype=dtype))

        def vec(fill):
            return torch.nn.Parameter(torch.full((d,), fill, device=device, dtype=dtype))

        # weights map rows by right multiplication: x [T, in] @ W [in, out]
        self.ln1_w, self.ln1_b = vec(1.0), vec(0.0)
        self.w_qkv = mat(d, 3 * d)
        self.w_o = mat(d, d)
        self.ln2_w, self.ln2_b = vec(1.0), vec(0.0)
        self.w_1 = mat(d, hidden)
        self.w_3 = mat(d, hidden)
        self.w_2 = mat(hidden, d)

    def weights(self) -> dict:
        return {n: p for n, p in self.named_parameters()}

    def forward(self, x, cu_doclens=None, doc_positions: bool = False):
        B, L, d = x.shape
        docs = _doclens(cu_doclens, B, L, x.device)
        y = _BlockFunction.apply(x.reshape(B * L, d), self.ln1_w, self.ln1_b, self.w_qkv,
                                 self.w_o, self.ln2_w, self.ln2_b, self.w_1, self.w_3, self.w_2,
                                 (B, L, self.H, self.D), self.rope_base, docs, doc_positions)
        return y.view(B, L, d)

    def gemm_flops(self, tokens: int) -> int:
        """Forward FLOPs of the projections and the MLP (backward: twice this)."""
        d, h = self.d, self.hidden
        return 2 * tokens * (4 * d * d + 3 * d * h)
