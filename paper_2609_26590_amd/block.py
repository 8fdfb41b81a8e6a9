"""One GTR block (paper Sec. 3.1) as a sequence of libgtr calls.

    n1 = LN1(x)                                   gtr_layernorm
    [q k v z] = n1 W_qkvr^T                       gtr_gemm, then gtr_heads_split
    a = (n1 W_a1^T) W_a2^T + b_a                  gtr_gemm x 2 (low-rank gate logits), gtr_heads_split
    u = SiLU(z) * RMSNorm(GLA(q, k, v; a))        gtr_gla_fwd: gate fusion (tau) and the output-gate epilogue
    x1 = x + concat_heads(u) W_o^T                gtr_heads_merge, gtr_gemm with the residual
    x2 = x1 + SpatialSwiGLU(LN2(x1))              gtr_layernorm, gtr_spatial_swiglu, gtr_add

Every step runs in the library's kernels; this module only marshals
arguments. The block's normalisation and residual placement are a reading of
the paper (it names the parts of the block, not their order): pre-norm layer
normalisation before the token mixer and before the Spatial SwiGLU, a residual
around each. The gate's rank-16 projection pair is zero-padded to 64 once,
when the weights are prepared (the product kernel takes K and N in multiples
of 64; the padding adds exact zeros).
"""
from __future__ import annotations

import torch

from . import (gtr_add, gtr_gemm, gtr_gla_fwd, gtr_heads_merge, gtr_heads_split, gtr_layernorm,
               gtr_spatial_swiglu)

GATE_PAD = 64


def prepare(p: dict) -> dict:
    """Device weights for ``forward``: the gate's rank-16 pair padded to 64."""
    q = dict(p)
    r, d = p["w_a1"].shape
    a1 = torch.zeros((GATE_PAD, d), dtype=p["w_a1"].dtype, device=p["w_a1"].device)
    a1[:r] = p["w_a1"]
    a2 = torch.zeros((d, GATE_PAD), dtype=p["w_a2"].dtype, device=p["w_a2"].device)
    a2[:, :r] = p["w_a2"]
    q["w_a1"], q["w_a2"] = a1, a2.contiguous()
    return q


def forward(x: torch.Tensor, p: dict, *, H: int, W: int, heads: int, scan: str, tau: float = 16.0,
            ln_eps: float = 1e-6, norm_eps: float = 1e-5, stream=None) -> torch.Tensor:
    """x [B, H*W, d] (fp16 or bf16, spatial order) -> the block's output, same
    shape and dtype. ``p`` from ``prepare``."""
    B, L, d = x.shape
    dh = d // heads
    M = B * L
    x2d = x.reshape(M, d)
    n1 = gtr_layernorm(x2d, p["ln1_w"], p["ln1_b"], eps=ln_eps, stream=stream)
    proj = gtr_gemm(n1, p["w_qkvr"], stream=stream)                       # [M, 4d]
    qkvz = gtr_heads_split(proj, parts=4, B=B, heads=heads, dh=dh, stream=stream)
    a1 = gtr_gemm(n1, p["w_a1"], stream=stream)                           # [M, 64]
    a = gtr_gemm(a1, p["w_a2"], bias=p["b_a"], stream=stream)             # [M, d]
    g = gtr_heads_split(a, parts=1, B=B, heads=heads, dh=dh, stream=stream)[0]
    u, _ = gtr_gla_fwd(qkvz[0], qkvz[1], qkvz[2], g, H=H, W=W, scale=dh ** -0.5, scan=scan,
                       gate_tau=tau, out_gate=qkvz[3], norm_weight=p["norm_w"],
                       norm_eps=norm_eps, stream=stream)
    um = gtr_heads_merge(u, stream=stream)                               # [M, d]
    x1 = gtr_gemm(um, p["w_o"], res=x2d, stream=stream)
    n2 = gtr_layernorm(x1, p["ln2_w"], p["ln2_b"], eps=ln_eps, stream=stream)
    y = gtr_spatial_swiglu(n2.reshape(B, L, d), p["w_g"], p["w_v"], p["w_out"], p["conv_w"], p["conv_b"],
                           H=H, W=W, stream=stream)
    return gtr_add(x1.reshape(B, L, d), y, stream=stream)
