"""CPU oracle for the chunkwise GLA hot path.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may use this package; the product library never
does. It shares no code with the HIP path (the two meet only through the seeded
input module, which holds no arithmetic of the method).

* :func:`scan_order` - the four directional scan orders (paper Sec. 3.1,
  "Directional scanning": left-to-right, right-to-left, top-to-bottom,
  bottom-to-top), as the permutation "scan position -> spatial index".
* :func:`permute` - gather / scatter of token rows by that permutation.
* :func:`gla` - the key-only GLA recurrence (Sec. 3.1), float64, token by token,
  in ``gla_oracle.c``.
* :func:`log_decay_from_logits` - the retention gate of Sec. 3.1,
  gamma = sigmoid(a)^(1/tau), as the log-decay g = log gamma the recurrence uses.
* :func:`output_gate` - the output gate of Sec. 3.1, u = SiLU(x W_r) * RMSNorm(o).
* :func:`spatial_swiglu` (with :func:`dwconv3x3`) - the Spatial SwiGLU of Sec. 3.1,
  Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o on the patch grid.

Readings taken where the paper is not explicit (each is listed with its reason
in the design notes of the repository):

* right-to-left is the full reversal of the row-major sequence, bottom-to-top
  the full reversal of the column-major one (not per-row "snakes");
* column-major visits column 0 top to bottom, then column 1, ...;
* S0 is applied before the first token in scan order and S_final is the state
  after the last token in scan order;
* ``scale`` is explicit; the paper's value is d_k^{-1/2};
* RMSNorm of the output gate normalises each token of each head over its d_v
  channels, with an explicit epsilon and an optional per-channel weight (the
  paper names RMSNorm without its axis or epsilon);
* the depthwise convolution of Spatial SwiGLU is a cross-correlation (as in
  common deep-learning libraries) with zero padding and an optional bias.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gla_oracle.c")
_LIB = os.path.join(_HERE, "_build", "liboracle.so")

SCAN_IDS = {"row": 0, "col": 1, "row_rev": 2, "col_rev": 3}


def build(force: bool = True) -> str:
    """Compile ``gla_oracle.c`` with gcc into ``oracle/_build/liboracle.so``."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    os.makedirs(os.path.dirname(_LIB), exist_ok=True)
    tmp = _LIB + f".tmp{os.getpid()}"
    # Plain -O2, no fast-math: the oracle keeps IEEE float64 semantics.
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-Wall",
                           "-o", tmp, _SRC, "-lm", "-lpthread"])
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        fn = lib.oracle_gla_forward
        P = ctypes.c_void_p
        fn.argtypes = [P, P, P, P, P, P, P, ctypes.c_long, ctypes.c_long, ctypes.c_int,
                       ctypes.c_int, ctypes.c_double, P, ctypes.c_int]
        fn.restype = ctypes.c_int
        _lib = lib
    return _lib


def scan_order(H: int, W: int, scan: str) -> np.ndarray:
    """order[s] = spatial (row-major) index of the token visited at scan step s.

    row:     s -> s                         (left-to-right, rows top to bottom)
    col:     s = j*H + i -> i*W + j         (top-to-bottom, columns left to right)
    row_rev: s -> L-1-s                     (right-to-left = reversed row scan)
    col_rev: s -> col(L-1-s)                (bottom-to-top = reversed column scan)
    """
    L = H * W
    s = np.arange(L, dtype=np.int64)
    if scan == "row":
        return s
    if scan == "col":
        j, i = np.divmod(s, H)
        return i * W + j
    if scan == "row_rev":
        return (L - 1) - s
    if scan == "col_rev":
        return scan_order(H, W, "col")[::-1].copy()
    raise ValueError(f"unknown scan {scan!r}")


def permute(x: np.ndarray, H: int, W: int, scan: str, inverse: bool = False) -> np.ndarray:
    """Reorder the token axis (axis -2) of ``x`` [..., L, E].

    forward: out[..., s, :] = x[..., order[s], :]   (spatial -> scan order)
    inverse: out[..., order[s], :] = x[..., s, :]   (scan order -> spatial)
    """
    order = scan_order(H, W, scan)
    if not inverse:
        return x[..., order, :].copy()
    out = np.empty_like(x)
    out[..., order, :] = x
    return out


def _f64(a) -> np.ndarray:
    if a is None:
        return None
    if hasattr(a, "detach"):  # torch tensor: take the exact values it holds
        a = a.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(a, dtype=np.float64)


def gla(q, k, v, g, s0=None, *, scale: float, H: int, W: int, scan: str = "row",
        threads: Optional[int] = None, want_final: bool = True):
    """Float64 recurrence over [B, heads, L, d] inputs in spatial order.

    Returns ``(o [B, heads, L, d_v], s_final [B, heads, d_k, d_v] or None)`` as
    float64 numpy arrays, ``o`` in spatial order.
    """
    q, k, v, g, s0 = (_f64(x) for x in (q, k, v, g, s0))
    B, Hh, L, dk = q.shape
    dv = v.shape[-1]
    if L != H * W:
        raise ValueError("L must equal H*W")
    if k.shape != q.shape or g.shape != q.shape or v.shape[:3] != q.shape[:3]:
        raise ValueError("shape mismatch")
    if s0 is not None and s0.shape != (B, Hh, dk, dv):
        raise ValueError("s0 shape mismatch")
    order = np.ascontiguousarray(scan_order(H, W, scan), dtype=np.int64)
    o = np.empty((B, Hh, L, dv), dtype=np.float64)
    sf = np.empty((B, Hh, dk, dv), dtype=np.float64) if want_final else None
    if threads is None:
        threads = max(1, len(os.sched_getaffinity(0)))
    ptr = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
    rc = _load().oracle_gla_forward(ptr(q), ptr(k), ptr(v), ptr(g), ptr(s0), ptr(o), ptr(sf),
                                    B * Hh, L, dk, dv, float(scale), ptr(order), int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle_gla_forward failed with {rc}")
    return o, sf


def log_decay_from_logits(a, tau: float) -> np.ndarray:
    """g = log gamma for gamma = sigmoid(a)^(1/tau) (Sec. 3.1, retention gate).

    Written as -log(1 + exp(-a)) / tau, with log(1 + exp(-a)) evaluated as
    logaddexp(0, -a) so that large |a| neither overflows nor loses the value.
    """
    a = _f64(a)
    return -np.logaddexp(0.0, -a) / float(tau)


def output_gate(o, z, weight=None, eps: float = 1e-5) -> np.ndarray:
    """u = SiLU(z) * RMSNorm(o) per token (Sec. 3.1, output gate).

    ``o`` and ``z`` are [..., d_v] (``z`` = x W_r, the gate before its SiLU);
    RMSNorm(o)_j = o_j / sqrt(mean_i o_i^2 + eps) * w_j over the last axis, with
    w = ``weight`` (ones if None). SiLU(z) = z * sigmoid(z) = z / (1 + exp(-z)).
    """
    o, z = _f64(o), _f64(z)
    w = np.ones(o.shape[-1]) if weight is None else _f64(weight)
    rms = np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + float(eps))
    silu = z / (1.0 + np.exp(-z))
    return silu * (o / rms) * w


def dwconv3x3(v, conv_w, conv_b=None, *, H: int, W: int) -> np.ndarray:
    """Depthwise 3x3 convolution of token features on the H x W patch grid (Sec. 3.1,
    Spatial SwiGLU): v [B, H*W, C] in row-major grid order, conv_w [C, 3, 3],
    zero padding, out[b, i, j, c] = sum_{u, w in 0..2} v[b, i+u-1, j+w-1, c] conv_w[c, u, w]
    (+ conv_b[c]); written as the nine shifted copies of the grid, one term each."""
    v = _f64(v)
    B, L, C = v.shape
    if L != H * W:
        raise ValueError("L must equal H*W")
    grid = v.reshape(B, H, W, C)
    pad = np.zeros((B, H + 2, W + 2, C))
    pad[:, 1:H + 1, 1:W + 1] = grid
    cw = _f64(conv_w)
    out = np.zeros((B, H, W, C))
    for u in range(3):
        for w_ in range(3):
            out += pad[:, u:u + H, w_:w_ + W, :] * cw[:, u, w_]
    if conv_b is not None:
        out += _f64(conv_b)
    return out.reshape(B, L, C)


def spatial_swiglu(x, w_gate, w_value, w_out, conv_w, conv_b=None, *, H: int, W: int) -> np.ndarray:
    """Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o (Sec. 3.1, Spatial SwiGLU), float64.

    x [B, H*W, d] in row-major grid order; weights in the layout of a linear
    layer (output features first): w_gate, w_value [h, d], w_out [d, h];
    conv_w [h, 3, 3], conv_b [h] or None. Returns y [B, H*W, d]."""
    x = _f64(x)
    g = x @ _f64(w_gate).T
    v = x @ _f64(w_value).T
    hidden = (g / (1.0 + np.exp(-g))) * dwconv3x3(v, conv_w, conv_b, H=H, W=W)
    return hidden @ _f64(w_out).T


def layer_norm(x, weight=None, bias=None, eps: float = 1e-6) -> np.ndarray:
    """Layer normalisation over the last axis: (x - mean) / sqrt(var + eps) * w + b,
    mean and variance (biased, divided by d) of each row. The block's
    normalisation before the token mixer and before the Spatial SwiGLU (the
    paper names neither; see the block's reading of Sec. 3.1)."""
    x = _f64(x)
    d = x.shape[-1]
    w = np.ones(d) if weight is None else _f64(weight)
    b = np.zeros(d) if bias is None else _f64(bias)
    mean = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mean) ** 2, axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + float(eps)) * w + b


def gtr_block(x, p: dict, *, H: int, W: int, heads: int, scan: str, tau: float = 16.0, ln_eps: float = 1e-6,
              norm_eps: float = 1e-5) -> np.ndarray:
    """One GTR block (Sec. 3.1), float64, composed from the functions above:
        n1 = LN1(x);  q, k, v, z = n1 W_q^T, n1 W_k^T, n1 W_v^T, n1 W_r^T
        a  = (n1 W_a1^T) W_a2^T + b_a                 (gate logits, low rank)
        o  = GLA(q, k, v, log gamma = logsigmoid(a) / tau) per head, in ``scan``
             order, scale d_k^-1/2
        u  = SiLU(z) * RMSNorm(o) per head (weight norm_w)
        x1 = x + concat_heads(u) W_o^T
        x2 = x1 + SpatialSwiGLU(LN2(x1))
    x [B, H*W, d] in spatial order; ``p`` holds the weights in linear-layer
    layout (output features first): w_qkvr [4d, d] (rows q, k, v, r), w_a1 [r, d],
    w_a2 [d, r], b_a [d], norm_w [d / heads], w_o [d, d], ln1_w, ln1_b, ln2_w, ln2_b
    [d], and the Spatial SwiGLU's w_g, w_v [h, d], w_out [d, h], conv_w [h, 3, 3],
    conv_b [h]."""
    x = _f64(x)
    B, L, d = x.shape
    dh = d // heads
    n1 = layer_norm(x, p["ln1_w"], p["ln1_b"], ln_eps)
    proj = n1 @ _f64(p["w_qkvr"]).T  # [B, L, 4d]

    def split(t):  # [B, L, heads * dh] -> [B, heads, L, dh]
        return t.reshape(B, L, heads, dh).transpose(0, 2, 1, 3)

    q, k, v, z = (split(proj[..., i * d:(i + 1) * d]) for i in range(4))
    a = (n1 @ _f64(p["w_a1"]).T) @ _f64(p["w_a2"]).T + _f64(p["b_a"])
    g = log_decay_from_logits(split(a), tau)
    o, _ = gla(q, k, v, g, None, scale=dh ** -0.5, H=H, W=W, scan=scan, want_final=False)
    u = output_gate(o, z, p["norm_w"], norm_eps)  # [B, heads, L, dh]
    x1 = x + u.transpose(0, 2, 1, 3).reshape(B, L, d) @ _f64(p["w_o"]).T
    n2 = layer_norm(x1, p["ln2_w"], p["ln2_b"], ln_eps)
    return x1 + spatial_swiglu(n2, p["w_g"], p["w_v"], p["w_out"], p["conv_w"], p["conv_b"], H=H, W=W)
