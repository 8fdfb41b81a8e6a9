"""Seeded synthetic inputs for the chunkwise GLA hot path.

This module holds the input recipe only: shapes, value distributions, seeds and
dtype casts. It performs none of the method's arithmetic, so both the HIP path
and the CPU oracle can consume exactly the same rounded values.

Recipe (one ``numpy.random.Generator(PCG64(seed))`` per input set):

* draw order: q, k, v, gate noise, then S0 (only when the workload has one);
* every draw is float64 standard normal, scaled as the workload states;
* the log-gate is ``g = logsigmoid(mu + std * z)`` evaluated in float64
  (the key-side log-decay log(gamma) of the recurrence in the paper's Sec. 3.1,
  with gamma in (0, 1));
* values are cast float64 -> float32 -> the workload dtype (round to nearest even);
* arrays are C-order ``[B, heads, L, d]`` in spatial (row-major grid) order,
  ``L = H * W``; S0 is float32 ``[B, heads, d_k, d_v]``.

The shapes follow the paper's backbone: a 640x640 image at patch stride 16 is a
40x40 token grid (L = 1600), 1280x1280 is 80x80 (L = 6400), and the larger GTR
models use head width 64. Trained activations are not available, so these
distributions stand in for them.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Sequence

import numpy as np
import torch

SCANS = ("row", "col", "row_rev", "col_rev")

_TORCH_DTYPES = {
    "f32": torch.float32,
    "f16": torch.float16,
    "bf16": torch.bfloat16,
}


@dataclass(frozen=True)
class Workload:
    """One synthetic GLA input set and the call options it is run with."""

    name: str
    B: int
    heads: int
    H: int
    W: int
    dk: int
    dv: int
    dtype: str            # q, k, v and g dtype: "f32" | "f16" | "bf16"
    odtype: str           # output dtype
    gate_mu: float
    gate_std: float
    qk_std: float
    v_std: float
    s0_std: Optional[float] = None   # None: zero initial state
    want_final: bool = False
    chunk: int = 64
    scans: Sequence[str] = ("row",)
    seed: int = 0
    calls: int = 1        # consecutive calls per step (one per scan direction)
    extra_chunks: Sequence[int] = field(default_factory=tuple)

    @property
    def L(self) -> int:
        return self.H * self.W

    @property
    def scale(self) -> float:
        return self.dk ** -0.5

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The workload shapes. ``tiny`` is small enough for the oracle to finish in
# well under a second; ``kbench`` is the 40x40-token operator benchmark with head
# width 64 (fp16 inputs, chunk 64); ``op*`` are the paper's own operator shape
# (d_k = 32, d_v = 64) at its three benchmark lengths.
WORKLOADS = {
    "tiny": Workload("tiny", B=1, heads=2, H=16, W=16, dk=32, dv=32, dtype="f32", odtype="f32",
                     gate_mu=2.0, gate_std=1.0, qk_std=32 ** -0.5, v_std=32 ** -0.5,
                     chunk=64, seed=1),
    "kbench": Workload("kbench", B=1, heads=6, H=40, W=40, dk=64, dv=64, dtype="f16", odtype="f16",
                       gate_mu=3.0, gate_std=1.0, qk_std=1 / 8, v_std=1.0, chunk=64, seed=2),
    "directions": Workload("directions", B=1, heads=12, H=40, W=40, dk=64, dv=64, dtype="bf16",
                           odtype="f32", gate_mu=3.0, gate_std=1.0, qk_std=1 / 8, v_std=1.0,
                           chunk=64, scans=SCANS, calls=4, seed=3),
    "highres": Workload("highres", B=1, heads=6, H=80, W=80, dk=64, dv=64, dtype="f16", odtype="f16",
                        gate_mu=4.0, gate_std=1.0, qk_std=1 / 8, v_std=1.0, chunk=64,
                        extra_chunks=(32, 128), seed=4),
    "batched": Workload("batched", B=8, heads=12, H=40, W=40, dk=64, dv=64, dtype="bf16", odtype="f32",
                        gate_mu=2.0, gate_std=2.0, qk_std=1 / 8, v_std=1.0, s0_std=0.1,
                        want_final=True, chunk=64, seed=5),
    # the paper's own operator shape (its operator appendix): d_k = 32, d_v = 64,
    # 6 heads, fp16, C = 64, at 256, 1.6K and 16.4K tokens (16x16, 40x40, 128x128)
    "op256": Workload("op256", B=1, heads=6, H=16, W=16, dk=32, dv=64, dtype="f16", odtype="f16",
                      gate_mu=3.0, gate_std=1.0, qk_std=1 / 8, v_std=1.0, chunk=64, seed=6),
    "op1600": Workload("op1600", B=1, heads=6, H=40, W=40, dk=32, dv=64, dtype="f16", odtype="f16",
                       gate_mu=3.0, gate_std=1.0, qk_std=1 / 8, v_std=1.0, chunk=64, seed=7),
    "op16k": Workload("op16k", B=1, heads=6, H=128, W=128, dk=32, dv=64, dtype="f16", odtype="f16",
                      gate_mu=3.0, gate_std=1.0, qk_std=1 / 8, v_std=1.0, chunk=64, seed=8),
}


def _logsigmoid(x: np.ndarray) -> np.ndarray:
    # log(1 / (1 + e^-x)) = -log(1 + e^-x), in a form that does not overflow.
    return -np.logaddexp(0.0, -x)


def _cast(a: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(_TORCH_DTYPES[dtype])


def make_inputs(wl: Workload, seed: Optional[int] = None) -> dict:
    """Draw one input set for ``wl`` as CPU tensors (see the module docstring)."""
    rng = np.random.Generator(np.random.PCG64(wl.seed if seed is None else seed))
    shp_k = (wl.B, wl.heads, wl.L, wl.dk)
    shp_v = (wl.B, wl.heads, wl.L, wl.dv)
    q = rng.standard_normal(shp_k) * wl.qk_std
    k = rng.standard_normal(shp_k) * wl.qk_std
    v = rng.standard_normal(shp_v) * wl.v_std
    z = rng.standard_normal(shp_k)
    g = _logsigmoid(wl.gate_mu + wl.gate_std * z)
    out = {
        "q": _cast(q, wl.dtype),
        "k": _cast(k, wl.dtype),
        "v": _cast(v, wl.dtype),
        "g": _cast(g, wl.dtype),
        "s0": None,
    }
    if wl.s0_std is not None:
        s0 = rng.standard_normal((wl.B, wl.heads, wl.dk, wl.dv)) * wl.s0_std
        out["s0"] = _cast(s0, "f32")
    return out


def torch_dtype(name: str) -> torch.dtype:
    return _TORCH_DTYPES[name]


def algorithmic_flops(wl: Workload, chunk: Optional[int] = None) -> float:
    """FLOPs of one chunkwise forward call (causal halves counted once).

    Per token and head: 2*C*... is folded into (d_k + d_v)(C + 1) for the two
    causal intra-chunk products plus 4 d_k d_v for the chunk summary and the
    state readout.
    """
    C = wl.chunk if chunk is None else chunk
    per = (wl.dk + wl.dv) * (C + 1) + 4 * wl.dk * wl.dv
    return float(per) * wl.B * wl.heads * wl.L


def algorithmic_bytes(wl: Workload) -> float:
    """HBM bytes one call must move: q, k, g, v in, o out, optional S0/S_final."""
    s_in = torch.tensor([], dtype=_TORCH_DTYPES[wl.dtype]).element_size()
    s_out = torch.tensor([], dtype=_TORCH_DTYPES[wl.odtype]).element_size()
    per = (3 * wl.dk + wl.dv) * s_in + wl.dv * s_out
    total = float(per) * wl.B * wl.heads * wl.L
    seq_state = wl.dk * wl.dv * 4 * wl.B * wl.heads
    if wl.s0_std is not None:
        total += seq_state
    if wl.want_final:
        total += seq_state
    return total


# ---------------------------------------------------------------------------
# One GTR block with random weights (GTR-S: d 192, 3 heads; GTR-L: d 384, 6
# heads; head width 64, Spatial SwiGLU expansion 4, gate rank 16). Draw order:
# x, then the weights in the order of BLOCK_WEIGHTS; projections N(0, 1/fan_in),
# layer-norm and RMSNorm weights 1 + N(0, 0.1), biases N(0, 0.1), the gate bias
# N(2, 0.5) (decays of about 0.98 to 0.998 per token after the
# temperature), depthwise conv weights N(0, 1/9). Every tensor is cast to its
# dtype once; fp16 / bf16 weights and float32 norm weights and biases.
# ---------------------------------------------------------------------------
BLOCK_SIZES = {"gtr_s": (192, 3), "gtr_l": (384, 6)}
GATE_RANK = 16


def make_block(name: str, H: int, W: int, B: int = 1, dtype: str = "f16", seed: int = 11) -> tuple:
    """(x [B, H*W, d], weights dict) for one block; see the recipe above."""
    d, heads = BLOCK_SIZES[name]
    hidden = 4 * d
    rng = np.random.Generator(np.random.PCG64(seed))
    n = lambda *shape, std=1.0, mu=0.0: mu + std * rng.standard_normal(shape)
    x = _cast(n(B, H * W, d), dtype)
    p = {
        "ln1_w": n(d, std=0.1, mu=1.0), "ln1_b": n(d, std=0.1),
        "w_qkvr": n(4 * d, d, std=d ** -0.5),
        "w_a1": n(GATE_RANK, d, std=d ** -0.5), "w_a2": n(d, GATE_RANK, std=GATE_RANK ** -0.5),
        "b_a": n(d, std=0.5, mu=2.0),
        "norm_w": n(d // heads, std=0.1, mu=1.0),
        "w_o": n(d, d, std=d ** -0.5),
        "ln2_w": n(d, std=0.1, mu=1.0), "ln2_b": n(d, std=0.1),
        "w_g": n(hidden, d, std=d ** -0.5), "w_v": n(hidden, d, std=d ** -0.5),
        "w_out": n(d, hidden, std=hidden ** -0.5),
        "conv_w": n(hidden, 3, 3, std=1.0 / 3), "conv_b": n(hidden, std=0.1),
    }
    f32 = ("ln1_w", "ln1_b", "b_a", "norm_w", "ln2_w", "ln2_b", "conv_w", "conv_b")
    return x, {k: _cast(v, "f32" if k in f32 else dtype) for k, v in p.items()}
