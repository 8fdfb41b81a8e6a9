"""Python binding of libgtr: chunkwise key-only GLA forward on MI355X (gfx950).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libgtr.so``. PyTorch supplies device memory and streams. There is
no CPU fallback: if the library is not built, every call raises.

Entry points (same names as the C ABI in ``include/gtr.h``):

* :func:`gtr_scan_permute` - token rows to / from the four scan orders
  (paper Sec. 3.1, "Directional scanning"), bit-exact.
* :func:`gtr_gla_fwd` - the chunkwise forward of the recurrence
  ``S_t = Diag(exp g_t) S_{t-1} + k_t^T v_t, o_t = scale q_t S_t``
  (Sec. 3.1, evaluated with the chunkwise schedule of Sec. 3.3).
* :func:`gtr_gla_workspace_size`, :func:`gtr_gla_workspace_init`,
  :func:`gtr_gla_workspace_fault`, :func:`gtr_status_string`.
* :func:`gtr_spatial_swiglu` - the Spatial SwiGLU channel mixer (Sec. 3.1),
  with :func:`gtr_spatial_swiglu_workspace_size` in the C ABI.

:class:`Workspace` keeps a caller-owned, zero-initialised workspace buffer.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgtr.so")

F32, F16, BF16 = 0, 1, 2
SCANS = {"row": 0, "col": 1, "row_rev": 2, "col_rev": 3}
PATHS = {"auto": 0, "fused": 1, "staged": 2, "inline": 3}
STATUS = {0: "GTR_OK", 1: "GTR_ERR_NULL", 2: "GTR_ERR_SHAPE", 3: "GTR_ERR_UNSUPPORTED",
          4: "GTR_ERR_ALIAS", 5: "GTR_ERR_WORKSPACE", 6: "GTR_ERR_HIP", 7: "GTR_ERR_SCRATCH"}

_DT = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}
_DT_BACK = {F32: torch.float32, F16: torch.float16, BF16: torch.bfloat16}

EXPORTS = ("gtr_scan_permute", "gtr_gla_workspace_size", "gtr_gla_workspace_init", "gtr_gla_fwd", "gtr_gla_fwd_noalloc",
           "gtr_gla_schedule", "gtr_gla_value_parts", "gtr_gla_workspace_fault", "gtr_status_string", "gtr_spatial_swiglu_workspace_size",
           "gtr_spatial_swiglu", "gtr_gemm", "gtr_layernorm", "gtr_heads_split", "gtr_heads_merge", "gtr_add")


class GtrError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {STATUS.get(status, status)}")


class GlaArgs(ctypes.Structure):
    """Mirror of ``gtr_gla_args`` (include/gtr.h)."""
    _fields_ = [
        ("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("g", ctypes.c_void_p), ("o", ctypes.c_void_p),
        ("s0", ctypes.c_void_p), ("s_final", ctypes.c_void_p),
        ("qkv_dtype", ctypes.c_int), ("g_dtype", ctypes.c_int), ("o_dtype", ctypes.c_int),
        ("B", ctypes.c_int32), ("heads", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32),
        ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
        ("scale", ctypes.c_float), ("scan", ctypes.c_int), ("path", ctypes.c_int),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
        ("g_kind", ctypes.c_int), ("gate_tau", ctypes.c_float),
        ("out_gate", ctypes.c_void_p), ("out_gate_dtype", ctypes.c_int),
        ("norm_eps", ctypes.c_float), ("norm_weight", ctypes.c_void_p),
        ("spin_limit", ctypes.c_uint32),
    ]


class SwigluArgs(ctypes.Structure):
    """Mirror of ``gtr_swiglu_args`` (include/gtr.h)."""
    _fields_ = [
        ("x", ctypes.c_void_p), ("w_gate", ctypes.c_void_p), ("w_value", ctypes.c_void_p),
        ("w_out", ctypes.c_void_p), ("conv_w", ctypes.c_void_p), ("conv_b", ctypes.c_void_p),
        ("y", ctypes.c_void_p), ("dtype", ctypes.c_int), ("y_dtype", ctypes.c_int),
        ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32), ("d", ctypes.c_int32),
        ("hidden", ctypes.c_int32), ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
        ("residual", ctypes.c_void_p),
    ]


class GemmArgs(ctypes.Structure):
    """Mirror of ``gtr_gemm_args`` (include/gtr.h)."""
    _fields_ = [
        ("a", ctypes.c_void_p), ("b", ctypes.c_void_p), ("c", ctypes.c_void_p), ("bias", ctypes.c_void_p),
        ("res", ctypes.c_void_p), ("a_dtype", ctypes.c_int), ("b_dtype", ctypes.c_int), ("c_dtype", ctypes.c_int),
        ("M", ctypes.c_int64), ("N", ctypes.c_int32), ("K", ctypes.c_int32),
        ("a_tokens", ctypes.c_int64), ("c_tokens", ctypes.c_int64), ("c_heads", ctypes.c_int32),
        ("c_head_dim", ctypes.c_int32), ("row_norm_eps", ctypes.c_float), ("row_norm", ctypes.c_int32),
    ]


_lib = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libgtr.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2609_26590_amd.build` "
                           "(or __graft_entry__.build()); there is no fallback implementation")
    lib = ctypes.CDLL(p)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.gtr_scan_permute.argtypes = [P, P, I64, I32, I32, I64, ctypes.c_int, ctypes.c_int, I32, P]
    lib.gtr_scan_permute.restype = ctypes.c_int
    lib.gtr_gla_workspace_size.argtypes = [ctypes.POINTER(GlaArgs)]
    lib.gtr_gla_workspace_size.restype = ctypes.c_size_t
    lib.gtr_gla_workspace_init.argtypes = [P, ctypes.c_size_t, P]
    lib.gtr_gla_workspace_init.restype = ctypes.c_int
    lib.gtr_gla_fwd.argtypes = [ctypes.POINTER(GlaArgs), P]
    lib.gtr_gla_fwd.restype = ctypes.c_int
    lib.gtr_gla_fwd_noalloc.argtypes = [ctypes.POINTER(GlaArgs), P]
    lib.gtr_gla_fwd_noalloc.restype = ctypes.c_int
    lib.gtr_gla_schedule.argtypes = [ctypes.POINTER(GlaArgs)]
    lib.gtr_gla_schedule.restype = ctypes.c_int
    lib.gtr_gla_value_parts.argtypes = [ctypes.POINTER(GlaArgs)]
    lib.gtr_gla_value_parts.restype = ctypes.c_int
    lib.gtr_gla_workspace_fault.argtypes = [P, ctypes.c_size_t]
    lib.gtr_gla_workspace_fault.restype = ctypes.c_int
    lib.gtr_status_string.argtypes = [ctypes.c_int]
    lib.gtr_status_string.restype = ctypes.c_char_p
    lib.gtr_spatial_swiglu_workspace_size.argtypes = [ctypes.POINTER(SwigluArgs)]
    lib.gtr_spatial_swiglu_workspace_size.restype = ctypes.c_size_t
    lib.gtr_spatial_swiglu.argtypes = [ctypes.POINTER(SwigluArgs), P]
    lib.gtr_spatial_swiglu.restype = ctypes.c_int
    lib.gtr_gemm.argtypes = [ctypes.POINTER(GemmArgs), P]
    lib.gtr_gemm.restype = ctypes.c_int
    lib.gtr_layernorm.argtypes = [P, P, P, P, I64, I32, ctypes.c_float, ctypes.c_int, P]
    lib.gtr_layernorm.restype = ctypes.c_int
    lib.gtr_heads_split.argtypes = [P, P, I32, I32, I32, I64, I32, I64, ctypes.c_int, P]
    lib.gtr_heads_split.restype = ctypes.c_int
    lib.gtr_heads_merge.argtypes = [P, P, I32, I32, I64, I32, ctypes.c_int, P]
    lib.gtr_heads_merge.restype = ctypes.c_int
    lib.gtr_add.argtypes = [P, P, P, I64, ctypes.c_int, P]
    lib.gtr_add.restype = ctypes.c_int
    _lib = lib
    return lib


def _stream_ptr(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def gtr_status_string(status: int) -> str:
    return load().gtr_status_string(status).decode()


def gtr_scan_permute(src: torch.Tensor, H: int, W: int, scan: str, inverse: bool = False,
                     out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Reorder axis -2 (tokens, L = H*W) of a contiguous [..., L, E] device tensor."""
    if not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous device tensor")
    if src.dim() < 2 or src.shape[-2] != H * W:
        raise ValueError("src must be [..., H*W, E]")
    dst = torch.empty_like(src) if out is None else out
    _check("out", dst, tuple(src.shape), (src.dtype,), src.device)
    outer = src.numel() // (src.shape[-2] * src.shape[-1]) if src.numel() else 0
    st = load().gtr_scan_permute(_ptr(src), _ptr(dst), outer, H, W, src.shape[-1], _DT[src.dtype],
                                 SCANS[scan], int(bool(inverse)), _stream_ptr(stream))
    if st:
        raise GtrError("gtr_scan_permute", st)
    return dst


GATE_LOG_DECAY, GATE_LOGITS = 0, 1


def make_args(q, k, v, g, *, H, W, scale, chunk=64, scan="row", s0=None, o=None, s_final=None,
              path="auto", workspace=None, gate_tau=None, out_gate=None, norm_weight=None,
              norm_eps=1e-5, spin_limit=0) -> GlaArgs:
    B, heads, L, dk = q.shape
    a = GlaArgs()
    a.q, a.k, a.v, a.g = _ptr(q), _ptr(k), _ptr(v), _ptr(g)
    a.o, a.s0, a.s_final = _ptr(o), _ptr(s0), _ptr(s_final)
    a.qkv_dtype = _DT[q.dtype]
    a.g_dtype = _DT[g.dtype]
    a.o_dtype = _DT[o.dtype] if o is not None else a.qkv_dtype
    a.B, a.heads, a.H, a.W = B, heads, H, W
    a.dk, a.dv, a.chunk = dk, v.shape[-1], chunk
    a.scale = float(scale)
    a.scan = SCANS[scan]
    a.path = PATHS[path]
    a.spin_limit = int(spin_limit)
    if workspace is not None:
        a.workspace = workspace.data_ptr()
        a.workspace_bytes = workspace.numel()
    if gate_tau is not None:  # g holds gate logits: log gamma = logsigmoid(g) / gate_tau
        a.g_kind = GATE_LOGITS
        a.gate_tau = float(gate_tau)
    if out_gate is not None:  # o receives SiLU(out_gate) * RMSNorm(o)
        a.out_gate = _ptr(out_gate)
        a.out_gate_dtype = _DT[out_gate.dtype]
        a.norm_weight = _ptr(norm_weight)
        a.norm_eps = float(norm_eps)
    return a


def gtr_gla_workspace_size(args: GlaArgs) -> int:
    return int(load().gtr_gla_workspace_size(ctypes.byref(args)))


def gtr_gla_workspace_init(ws: torch.Tensor, stream=None) -> None:
    st = load().gtr_gla_workspace_init(_ptr(ws), ws.numel(), _stream_ptr(stream))
    if st:
        raise GtrError("gtr_gla_workspace_init", st)


def gtr_gla_workspace_fault(ws: torch.Tensor) -> int:
    """Fault bits of the calls on ``ws`` since its initialisation (1: a bounded
    wait ran out, 2: a bf16 input outside the fp16 range); blocks until the
    device is idle."""
    return int(load().gtr_gla_workspace_fault(_ptr(ws), ws.numel()))


class Workspace:
    """A growable, zero-initialised device workspace for :func:`gtr_gla_fwd`,
    used on one stream: it is allocated and zero-filled on that stream, so
    the caching allocator never hands its memory to another stream while a
    call on this one may still use it."""

    def __init__(self, device=None, stream=None):
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.stream = stream
        self.buf: Optional[torch.Tensor] = None

    def get(self, nbytes: int, stream=None) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            s = stream if stream is not None else (self.stream or torch.cuda.current_stream(self.device))
            n = max(256, (nbytes + 255) // 256 * 256)
            with torch.cuda.stream(s):
                # 256-byte aligned: torch's caching allocator hands out 512-byte aligned blocks
                self.buf = torch.empty(n, dtype=torch.uint8, device=self.device)
                gtr_gla_workspace_init(self.buf, s)
        return self.buf


# default workspaces, one per (device, stream): calls on different streams
# never share one
_default_ws: dict = {}


def _default_workspace(kind: str, device: torch.device, stream) -> Workspace:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    key = (kind, device, int(s.cuda_stream))
    ws = _default_ws.get(key)
    if ws is None:
        ws = _default_ws[key] = Workspace(device, s)
    return ws


def _check(name: str, t: Optional[torch.Tensor], shape, dtypes, device) -> None:
    if t is None:
        return
    if not t.is_cuda or t.device != device:
        raise ValueError(f"{name} must be on {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {list(dtypes)}")


def gtr_gla_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor, *, H: int, W: int,
                scale: Optional[float] = None, chunk: int = 64, scan: str = "row",
                s0: Optional[torch.Tensor] = None, want_final: bool = False,
                o_dtype: Optional[torch.dtype] = None, path: str = "auto",
                out: Optional[torch.Tensor] = None, s_final: Optional[torch.Tensor] = None,
                workspace: Optional[Workspace] = None, stream=None, gate_tau: Optional[float] = None,
                out_gate: Optional[torch.Tensor] = None, norm_weight: Optional[torch.Tensor] = None,
                norm_eps: float = 1e-5, spin_limit: int = 0, check: bool = False):
    """Chunkwise GLA forward. Inputs [B, heads, H*W, d] in spatial order on the GPU.

    ``gate_tau``: g holds gate logits a, log gamma = logsigmoid(a) / gate_tau.
    ``out_gate`` ([B, heads, H*W, dv], x W_r) with optional ``norm_weight`` ([dv],
    float32): the output is u = SiLU(out_gate) * RMSNorm(o) instead of o.
    ``spin_limit``: polls of a one-launch wait before it gives up (0: default).
    ``check``: synchronise and raise if the workspace's fault word is set.
    Returns ``(o, s_final)``; ``s_final`` is None unless requested.
    """
    if q.dim() != 4:
        raise ValueError("q must be [B, heads, H*W, d_k]")
    B, heads, L, dk = q.shape
    dv = v.shape[-1] if v.dim() == 4 else -1
    dev = q.device
    if L != H * W:
        raise ValueError(f"q has {L} tokens, H*W = {H * W}")
    if q.dtype not in _DT:
        raise ValueError(f"unsupported dtype {q.dtype}")
    qdt = (q.dtype,)
    _check("q", q, (B, heads, L, dk), qdt, dev)
    _check("k", k, (B, heads, L, dk), qdt, dev)
    _check("v", v, (B, heads, L, dv), qdt, dev)
    _check("g", g, (B, heads, L, dk), (q.dtype, torch.float32), dev)
    _check("s0", s0, (B, heads, dk, dv), (torch.float32,), dev)
    _check("out_gate", out_gate, (B, heads, L, dv), (q.dtype, torch.float32), dev)
    _check("norm_weight", norm_weight, (dv,), (torch.float32,), dev)
    if scale is None:
        scale = dk ** -0.5
    odt = o_dtype or (out.dtype if out is not None else q.dtype)
    o = out if out is not None else torch.empty((B, heads, L, dv), dtype=odt, device=dev)
    _check("out", o, (B, heads, L, dv), (q.dtype, torch.float32), dev)
    sf = s_final
    if want_final and sf is None:
        sf = torch.empty((B, heads, dk, dv), dtype=torch.float32, device=dev)
    _check("s_final", sf, (B, heads, dk, dv), (torch.float32,), dev)
    args = make_args(q, k, v, g, H=H, W=W, scale=scale, chunk=chunk, scan=scan, s0=s0, o=o,
                     s_final=sf, path=path, gate_tau=gate_tau, out_gate=out_gate,
                     norm_weight=norm_weight, norm_eps=norm_eps, spin_limit=spin_limit)
    need = gtr_gla_workspace_size(args)
    if need == 0:
        raise GtrError("gtr_gla_workspace_size", 2)
    if workspace is None:
        workspace = _default_workspace("gla", dev, stream)
    buf = workspace.get(need, stream)
    args.workspace = buf.data_ptr()
    args.workspace_bytes = buf.numel()
    st = load().gtr_gla_fwd(ctypes.byref(args), _stream_ptr(stream))
    if st:
        raise GtrError("gtr_gla_fwd", st)
    if check:
        f = gtr_gla_workspace_fault(buf)
        if f:
            raise RuntimeError(f"gtr_gla_fwd: fault word {f} (1: a wait ran out, 2: bf16 input outside fp16 range)")
    return o, sf


SCHEDULES = {1: "fused", 2: "staged", 3: "inline"}


def _schedule_args(q, k, v, g, H, W, chunk, scan, s0, want_final, o_dtype, path):
    o = torch.empty((0,), dtype=o_dtype or q.dtype, device=q.device)
    sf = torch.empty((0,), dtype=torch.float32, device=q.device) if want_final else None
    return make_args(q, k, v, g, H=H, W=W, scale=1.0, chunk=chunk, scan=scan, s0=s0, o=o, s_final=sf, path=path)


def gtr_gla_schedule(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor, *, H: int, W: int,
                     chunk: int = 64, scan: str = "row", s0: Optional[torch.Tensor] = None,
                     want_final: bool = False, o_dtype: Optional[torch.dtype] = None, path: str = "auto") -> str:
    """The schedule gtr_gla_fwd runs for these arguments: "fused", "staged" or "inline"."""
    args = _schedule_args(q, k, v, g, H, W, chunk, scan, s0, want_final, o_dtype, path)
    r = int(load().gtr_gla_schedule(ctypes.byref(args)))
    if r not in SCHEDULES:
        raise GtrError("gtr_gla_schedule", 3)
    return SCHEDULES[r]


def gtr_gla_value_parts(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor, *, H: int, W: int,
                        chunk: int = 64, scan: str = "row", s0: Optional[torch.Tensor] = None,
                        want_final: bool = False, o_dtype: Optional[torch.dtype] = None, path: str = "auto") -> int:
    """Work-groups per chunk's value columns in that schedule: 2 under the inline value split, else 1."""
    args = _schedule_args(q, k, v, g, H, W, chunk, scan, s0, want_final, o_dtype, path)
    r = int(load().gtr_gla_value_parts(ctypes.byref(args)))
    if r not in (1, 2):
        raise GtrError("gtr_gla_value_parts", 3)
    return r


def gtr_spatial_swiglu(x: torch.Tensor, w_gate: torch.Tensor, w_value: torch.Tensor, w_out: torch.Tensor,
                       conv_w: torch.Tensor, conv_b: Optional[torch.Tensor] = None, *, H: int, W: int,
                       y_dtype: Optional[torch.dtype] = None, out: Optional[torch.Tensor] = None,
                       residual: Optional[torch.Tensor] = None,
                       workspace: Optional["Workspace"] = None, stream=None) -> torch.Tensor:
    """Spatial SwiGLU (Sec. 3.1): y = [SiLU(x W_g^T) * DWConv3x3(x W_v^T)] W_o^T.

    x [B, H*W, d] (fp16/bf16, spatial order), w_gate/w_value [hidden, d],
    w_out [d, hidden] (same dtype), conv_w [hidden, 3, 3] and conv_b [hidden]
    float32. Returns y [B, H*W, d] in ``y_dtype`` (default: x's dtype), plus
    ``residual`` ([B, H*W, d] in that dtype, may be ``out``) when given.
    """
    for name, t in (("x", x), ("w_gate", w_gate), ("w_value", w_value), ("w_out", w_out), ("conv_w", conv_w)) + \
            ((("conv_b", conv_b),) if conv_b is not None else ()):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous device tensor")
    B, L, d = x.shape
    y = out if out is not None else torch.empty((B, L, d), dtype=y_dtype or x.dtype, device=x.device)
    a = SwigluArgs()
    a.x, a.w_gate, a.w_value, a.w_out = _ptr(x), _ptr(w_gate), _ptr(w_value), _ptr(w_out)
    a.conv_w, a.conv_b, a.y = _ptr(conv_w), _ptr(conv_b), _ptr(y)
    a.dtype, a.y_dtype = _DT[x.dtype], _DT[y.dtype]
    a.B, a.H, a.W, a.d, a.hidden = B, H, W, d, w_gate.shape[0]
    if residual is not None:  # y = residual + SwiGLU(x)
        _check("residual", residual, (B, L, d), (y.dtype,), x.device)
        a.residual = _ptr(residual)
    lib = load()
    need = int(lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(a)))
    if need == 0:
        raise GtrError("gtr_spatial_swiglu_workspace_size", 2)
    if workspace is None:
        workspace = _default_workspace("swiglu", x.device, stream)
    buf = workspace.get(need, stream)
    a.workspace, a.workspace_bytes = buf.data_ptr(), buf.numel()
    st = lib.gtr_spatial_swiglu(ctypes.byref(a), _stream_ptr(stream))
    if st:
        raise GtrError("gtr_spatial_swiglu", st)
    return y


# ---------------------------------------------------------------------------
# the small calls of one GTR block (gtr_gemm, gtr_layernorm, gtr_heads_split /
# gtr_heads_merge, gtr_add): argument marshalling only
# ---------------------------------------------------------------------------
def _dev_contig(name: str, t: torch.Tensor) -> None:
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")


def gtr_gemm(a: torch.Tensor, b: torch.Tensor, *, bias: Optional[torch.Tensor] = None,
             res: Optional[torch.Tensor] = None, out_dtype: Optional[torch.dtype] = None,
             out: Optional[torch.Tensor] = None, heads_out: Optional[tuple] = None,
             row_norm_eps: Optional[float] = None, stream=None) -> torch.Tensor:
    """c = a b^T (+ bias) (+ res): a [M, K], b [N, K] (fp16 or bf16, same dtype),
    bias [N] float32, res [M, N] in the output dtype (may be ``out``).

    ``row_norm_eps`` set: every row of a is first normalised over its K
    columns, (a - mean) / sqrt(var + row_norm_eps) (a layer normalisation whose
    weights the caller folds into b and bias).

    a may also be head-major [B, K / 64, L, 64] (a head concat read in place:
    M = B * L). ``heads_out = (L, heads, dh)`` stores c head-major as
    [N / (heads * dh), M / L, heads, L, dh] instead of [M, N]."""
    for name, t in (("a", a), ("b", b)) + ((("bias", bias),) if bias is not None else ()) + \
            ((("res", res),) if res is not None else ()):
        _dev_contig(name, t)
    a_tokens = 0
    if a.dim() == 4:
        Bi, nh, L, w = a.shape
        if w != 64:
            raise ValueError("a head-major operand has heads of width 64")
        M, K, a_tokens = Bi * L, nh * 64, L
    else:
        M, K = a.shape
    N = b.shape[0]
    if b.shape[1] != K:
        raise ValueError(f"b has {b.shape[1]} columns, a has {K}")
    if heads_out is not None:
        L, nh, dh = heads_out
        shape = (N // (nh * dh), M // L, nh, L, dh)
    else:
        shape = (M, N)
    c = out if out is not None else torch.empty(shape, dtype=out_dtype or a.dtype, device=a.device)
    _check("out", c, shape, (torch.float32, torch.float16, torch.bfloat16), a.device)
    _check("bias", bias, (N,), (torch.float32,), a.device)
    _check("res", res, (M, N), (c.dtype,), a.device)
    g = GemmArgs()
    g.a, g.b, g.c, g.bias, g.res = _ptr(a), _ptr(b), _ptr(c), _ptr(bias), _ptr(res)
    g.a_dtype, g.b_dtype, g.c_dtype = _DT[a.dtype], _DT[b.dtype], _DT[c.dtype]
    g.M, g.N, g.K = M, N, K
    g.a_tokens = a_tokens
    if row_norm_eps is not None:
        g.row_norm, g.row_norm_eps = 1, float(row_norm_eps)
    if heads_out is not None:
        g.c_tokens, g.c_heads, g.c_head_dim = heads_out
    st = load().gtr_gemm(ctypes.byref(g), _stream_ptr(stream))
    if st:
        raise GtrError("gtr_gemm", st)
    return c


def gtr_layernorm(x: torch.Tensor, weight: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None, *,
                  eps: float = 1e-6, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Layer normalisation over the last dimension of x (fp16 or bf16)."""
    _dev_contig("x", x)
    d = x.shape[-1]
    y = out if out is not None else torch.empty_like(x)
    _check("out", y, tuple(x.shape), (x.dtype,), x.device)
    _check("weight", weight, (d,), (torch.float32,), x.device)
    _check("bias", bias, (d,), (torch.float32,), x.device)
    st = load().gtr_layernorm(_ptr(x), _ptr(weight), _ptr(bias), _ptr(y), x.numel() // d, d, float(eps), _DT[x.dtype],
                              _stream_ptr(stream))
    if st:
        raise GtrError("gtr_layernorm", st)
    return y


def gtr_heads_split(x: torch.Tensor, *, parts: int, B: int, heads: int, dh: int, stream=None) -> torch.Tensor:
    """x [B*L, ld] (token-major product; part p, head h at columns
    (p*heads + h)*dh ...) -> [parts, B, heads, L, dh]."""
    _dev_contig("x", x)
    M, ld = x.shape
    L = M // B
    y = torch.empty((parts, B, heads, L, dh), dtype=x.dtype, device=x.device)
    st = load().gtr_heads_split(_ptr(x), _ptr(y), parts, B, heads, L, dh, ld, _DT[x.dtype], _stream_ptr(stream))
    if st:
        raise GtrError("gtr_heads_split", st)
    return y


def gtr_heads_merge(u: torch.Tensor, stream=None) -> torch.Tensor:
    """u [B, heads, L, dh] -> [B*L, heads*dh] (the head concat)."""
    _dev_contig("u", u)
    B, H, L, dh = u.shape
    y = torch.empty((B * L, H * dh), dtype=u.dtype, device=u.device)
    st = load().gtr_heads_merge(_ptr(u), _ptr(y), B, H, L, dh, _DT[u.dtype], _stream_ptr(stream))
    if st:
        raise GtrError("gtr_heads_merge", st)
    return y


def gtr_add(a: torch.Tensor, b: torch.Tensor, *, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """a + b elementwise (fp16 or bf16, same shape); ``out`` may be a or b."""
    _dev_contig("a", a)
    _check("b", b, tuple(a.shape), (a.dtype,), a.device)
    y = out if out is not None else torch.empty_like(a)
    _check("out", y, tuple(a.shape), (a.dtype,), a.device)
    st = load().gtr_add(_ptr(a), _ptr(b), _ptr(y), a.numel(), _DT[a.dtype], _stream_ptr(stream))
    if st:
        raise GtrError("gtr_add", st)
    return y
