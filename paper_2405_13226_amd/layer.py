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
5632 at d = 2048.  Attention and RoPE run in this library's HIP kernels (the
autograd wrapper of ``attention.py``); the projections and the MLP are plain
2-D bf16 GEMMs and the norms and SiLU are elementwise, all through torch
(vendor-library GEMMs).  The block exists to place the attention hot path in
a full layer step: its time as a share of the step, and the step time's
growth with the sequence length at a fixed token budget.
"""
from __future__ import annotations

import torch
import torch.nn.functional as F

from .attention import attention

LN_EPS = 1e-5
OPENLM_1B = dict(d=2048, H=16, hidden=5632)


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
        H, D = self.H, self.D
        t = x.reshape(B * L, d)
        a = F.layer_norm(t, (d,), self.ln1_w, self.ln1_b, LN_EPS)
        qkv = a @ self.w_qkv
        q, k, v = (s.reshape(B, L, H, D).contiguous() for s in qkv.split(d, dim=-1))
        o = attention(q, k, v, True, cu_doclens, self.rope_base, doc_positions)
        h = t + o.reshape(B * L, d) @ self.w_o
        m = F.layer_norm(h, (d,), self.ln2_w, self.ln2_b, LN_EPS)
        y = h + (F.silu(m @ self.w_1) * (m @ self.w_3)) @ self.w_2
        return y.reshape(B, L, d)

    def gemm_flops(self, tokens: int) -> int:
        """Forward FLOPs of the projections and the MLP (backward: twice this)."""
        d, h = self.d, self.hidden
        return 2 * tokens * (4 * d * d + 3 * d * h)
