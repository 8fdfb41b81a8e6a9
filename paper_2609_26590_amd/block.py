"""One GTR block (paper Sec. 3.1) as a sequence of libgtr calls.

    [q k v z a] = LN1(x) [W_qkvr; W_a]^T + [0; b_a]   one gtr_gemm that normalises the rows of x inside the
                                                  product (LN1's weights folded into the matrix and the bias
                                                  in ``prepare``), stored head-major; W_a = W_a2 W_a1, the
                                                  low-rank gate's factors multiplied once in ``prepare``
    u = SiLU(z) * RMSNorm(GLA(q, k, v; a))        gtr_gla_fwd: gate fusion (tau) and the output-gate epilogue
    x1 = x + concat_heads(u) W_o^T                gtr_gemm reading u head-major, the residual in its epilogue
    x2 = x1 + SpatialSwiGLU(LN2(x1))              gtr_layernorm, gtr_spatial_swiglu with the residual

Every step runs in the library's kernels; this module only marshals
arguments. The block's normalisation and residual placement are a reading of
the paper (it names the parts of the block, not their order): pre-norm layer
normalisation before the token mixer and before the Spatial SwiGLU, a residual
around each. The gate's rank-16 factors are multiplied into one d x d matrix
when the weights are prepared: the same logits in real arithmetic, with the
product's fp16 rounding in place of the rank-16 intermediate's. LN1's weights
gamma, beta are folded the usual way, LN1(x) W^T + c = norm(x) (W diag(gamma))^T
+ (c + W beta): the same values in real arithmetic, with the folded matrix
rounded to the input dtype in place of the rounding of LN1(x).
"""
from __future__ import annotations

import torch

from . import gtr_gemm, gtr_gla_fwd, gtr_layernorm, gtr_spatial_swiglu

GATE_PAD = 64


def prepare(p: dict) -> dict:
    """Device weights for ``forward`` (once per block), all products through
    gtr_gemm: the gate's rank-16 factors multiplied into one d x d matrix
    W_a = W_a2 W_a1 (the rank zero-padded to 64) and appended to the
    projections as a fifth part, with the gate bias as that part's bias, so one
    product gives q, k, v, z and the gate logits; then LN1's weights folded
    into that matrix and bias: W diag(gamma) and c + W beta."""
    r, d = p["w_a1"].shape
    dev, dt = p["w_a1"].device, p["w_a1"].dtype
    a2 = torch.zeros((d, GATE_PAD), dtype=dt, device=dev)
    a2[:, :r] = p["w_a2"]
    a1t = torch.zeros((d, GATE_PAD), dtype=dt, device=dev)
    a1t[:, :r] = p["w_a1"].t()
    w_a = gtr_gemm(a2, a1t)  # [d, d] = W_a2 W_a1
    w_proj = torch.cat([p["w_qkvr"], w_a]).contiguous()
    b_proj = torch.cat([torch.zeros(4 * d, device=dev), p["b_a"].float()]).contiguous()
    gamma = torch.diag(p["ln1_w"].float()).to(dt).contiguous()
    q = dict(p)
    q["w_proj"] = gtr_gemm(w_proj, gamma)  # W diag(gamma)
    beta = p["ln1_b"].to(dt).reshape(1, d).contiguous()
    q["b_proj"] = gtr_gemm(beta, w_proj, bias=b_proj, out_dtype=torch.float32).reshape(-1)  # c + W beta
    return q


def forward(x: torch.Tensor, p: dict, *, H: int, W: int, heads: int, scan: str, tau: float = 16.0,
            ln_eps: float = 1e-6, norm_eps: float = 1e-5, stream=None) -> torch.Tensor:
    """x [B, H*W, d] (fp16 or bf16, spatial order) -> the block's output, same
    shape and dtype. ``p`` from ``prepare``."""
    B, L, d = x.shape
    dh = d // heads
    M = B * L
    x2d = x.reshape(M, d)
    # one product over the normalised rows of x, stored head-major ([5, B, heads, L, dh]: q, k, v, z and
    # the gate logits)
    proj = gtr_gemm(x2d, p["w_proj"], bias=p["b_proj"], heads_out=(L, heads, dh), row_norm_eps=ln_eps,
                    stream=stream)
    u, _ = gtr_gla_fwd(proj[0], proj[1], proj[2], proj[4], H=H, W=W, scale=dh ** -0.5, scan=scan,
                       gate_tau=tau, out_gate=proj[3], norm_weight=p["norm_w"],
                       norm_eps=norm_eps, stream=stream)
    # the head concat read in place by W_o, the residual in its epilogue
    x1 = gtr_gemm(u, p["w_o"], res=x2d, stream=stream)
    n2 = gtr_layernorm(x1, p["ln2_w"], p["ln2_b"], eps=ln_eps, stream=stream)
    x1 = x1.reshape(B, L, d)
    return gtr_spatial_swiglu(n2.reshape(B, L, d), p["w_g"], p["w_v"], p["w_out"], p["conv_w"], p["conv_b"],
                              H=H, W=W, residual=x1, stream=stream)
