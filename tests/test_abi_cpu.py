"""The C ABI on the CPU: the library loads, exports every declared entry point,
and every host-side validation path returns its status without launching.

Only invalid argument sets are passed here (pointers are fake, never
dereferenced): validation happens before any HIP call, so nothing runs.
"""
import ctypes
import os
import re

import pytest

import paper_2609_26590_amd as gtr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gtr.h")

OK, NULL, SHAPE, UNSUP, ALIAS, WS = 0, 1, 2, 3, 4, 5


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(gtr.LIB_PATH):
        pytest.fail("libgtr.so is not built (run __graft_entry__.build())")
    return gtr.load()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gtr_\w+)\s*\(", src)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(gtr.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code, name in gtr.STATUS.items():
        assert gtr.gtr_status_string(code).startswith(name)


# ---------------------------------------------------------------------------
# gtr_gla_fwd / gtr_gla_workspace_size
# ---------------------------------------------------------------------------

FAKE = 1 << 40  # never dereferenced


def base_args(B=1, heads=2, H=4, W=5, dk=64, dv=64, chunk=64, dt=gtr.F16, ws_bytes=None):
    a = gtr.GlaArgs()
    L = H * W
    n_in = B * heads * L * 64 * 4
    a.q, a.k, a.v, a.g = FAKE, FAKE + n_in, FAKE + 2 * n_in, FAKE + 3 * n_in
    a.o = FAKE + 4 * n_in
    a.s0 = None
    a.s_final = None
    a.qkv_dtype = a.g_dtype = a.o_dtype = dt
    a.B, a.heads, a.H, a.W = B, heads, H, W
    a.dk, a.dv, a.chunk = dk, dv, chunk
    a.scale = 0.125
    a.scan = 0
    a.path = 0
    need = gtr.load().gtr_gla_workspace_size(ctypes.byref(a))
    a.workspace = FAKE + 6 * n_in
    a.workspace_bytes = need if ws_bytes is None else ws_bytes
    return a


def fwd(lib, a):
    return lib.gtr_gla_fwd(ctypes.byref(a), None)


def test_workspace_size_formula(lib):
    a = base_args(B=2, heads=3, H=40, W=40, dk=64, dv=64, chunk=64)
    BH, nc = 6, 25
    a256 = lambda x: (x + 255) // 256 * 256
    # header, done counters of 1024 sequences, chunk flags of 1024 x 256, then
    # the summaries (fp16 for 16-bit inputs, float32 for float32 inputs), the
    # chunk records ((decay, scale) pairs per key dim, two per chunk for the
    # value split) and the float32 states
    fixed = 256 + 1024 * 16 + 1024 * 256 * 4
    rec = a256(2 * BH * nc * (2 * 64) * 4)
    states = BH * nc * 64 * 64 * 4
    want = fixed + a256(BH * nc * 64 * 64 * 2) + rec + states
    assert a.qkv_dtype != gtr.F32 and lib.gtr_gla_workspace_size(ctypes.byref(a)) == want
    a.qkv_dtype = a.g_dtype = a.o_dtype = gtr.F32
    want = fixed + BH * nc * 64 * 64 * 4 + rec + states
    assert lib.gtr_gla_workspace_size(ctypes.byref(a)) == want
    a.dk = 48
    assert lib.gtr_gla_workspace_size(ctypes.byref(a)) == 0


def test_schedule_query_without_device(lib):
    """gtr_gla_schedule: -1 for invalid arguments. AUTO is length-aware: INLINE
    up to 32 chunks per sequence when the whole grid is resident at once, FUSED
    up to 64 chunks (256 for 16-bit inputs at chunk 64), STAGED beyond; an
    explicit one-launch path that does not
    fit (more than 256 chunks) reports -1. Without a usable device residency is
    unknown (so AUTO takes FUSED) and the value split is off."""
    assert lib.gtr_gla_schedule(None) == -1
    a = base_args(B=1, heads=6, H=40, W=40)  # 25 chunks
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 1
    a.path = 3
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 3
    a.path = 0
    a.H, a.W = 40, 80  # 50 chunks
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 1
    a.H = a.W = 80  # 100 chunks: FUSED (grouped look-back) for 16-bit inputs at chunk 64
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 1
    a.qkv_dtype = a.g_dtype = a.o_dtype = gtr.F32  # STAGED for float32
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 2
    a.path = 1  # an explicit one-launch path still fits
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 1
    a.path = 0
    a.qkv_dtype = a.g_dtype = a.o_dtype = gtr.F16
    a.H = a.W = 200  # 625 chunks
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 2
    a.path = 1
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == -1
    a.path, a.H, a.W = 2, 40, 40
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == 2
    a.path, a.dk = 0, 48
    assert lib.gtr_gla_schedule(ctypes.byref(a)) == -1
    assert lib.gtr_gla_value_parts(None) == -1
    assert lib.gtr_gla_value_parts(ctypes.byref(a)) == -1
    a.dk = 64
    assert lib.gtr_gla_value_parts(ctypes.byref(a)) == 1


def test_sequence_rows_beyond_descriptor_range(lib):
    """One sequence's rows are addressed through a 32-bit buffer descriptor:
    L * max(dk, dv) * 4 bytes must stay below 0x7fffff00."""
    a = base_args(B=1, heads=1, H=4096, W=2048, dk=64, dv=64)  # 8.4M tokens: 2.1 GB of float32 rows
    assert lib.gtr_gla_workspace_size(ctypes.byref(a)) == 0
    assert lib.gtr_gla_fwd(ctypes.byref(a), None) == SHAPE
    a.W = 2047
    assert lib.gtr_gla_workspace_size(ctypes.byref(a)) > 0


def test_null_struct(lib):
    assert lib.gtr_gla_fwd(None, None) == NULL


@pytest.mark.parametrize("field", ["q", "k", "v", "g", "o"])
def test_null_tensor(lib, field):
    a = base_args()
    setattr(a, field, None)
    assert fwd(lib, a) == NULL


@pytest.mark.parametrize("field,val", [("B", 0), ("heads", -1), ("H", 0), ("W", 0), ("chunk", 0)])
def test_bad_shape(lib, field, val):
    a = base_args()
    setattr(a, field, val)
    assert fwd(lib, a) == SHAPE


def test_shape_overflow(lib):
    a = base_args()
    a.B, a.heads, a.H, a.W = 2 ** 30, 2 ** 30, 2 ** 30, 2 ** 30
    assert fwd(lib, a) == SHAPE


@pytest.mark.parametrize("field,val", [("dk", 48), ("dv", 128), ("chunk", 96), ("qkv_dtype", 7),
                                       ("scan", 4), ("path", 9)])
def test_unsupported(lib, field, val):
    a = base_args()
    setattr(a, field, val)
    assert fwd(lib, a) == UNSUP


def test_unsupported_dtype_mix(lib):
    a = base_args(dt=gtr.F16)
    a.g_dtype = gtr.BF16
    assert fwd(lib, a) == UNSUP
    a = base_args(dt=gtr.F16)
    a.o_dtype = gtr.BF16
    assert fwd(lib, a) == UNSUP


def test_misaligned_tensor(lib):
    a = base_args()
    a.v = a.v + 2
    assert fwd(lib, a) == UNSUP


def test_output_aliases_input(lib):
    a = base_args()
    a.o = a.k + 64
    assert fwd(lib, a) == ALIAS


def test_final_state_aliases_output(lib):
    a = base_args()
    a.s_final = a.o
    assert fwd(lib, a) == ALIAS


def test_workspace_aliases_input(lib):
    a = base_args()
    a.workspace = a.q
    assert fwd(lib, a) == ALIAS


def test_workspace_missing_small_misaligned(lib):
    a = base_args()
    a.workspace = None
    assert fwd(lib, a) == WS
    a = base_args()
    a.workspace_bytes -= 1
    assert fwd(lib, a) == WS
    a = base_args()
    a.workspace += 128
    assert fwd(lib, a) == WS


def test_workspace_init_validation(lib):
    assert lib.gtr_gla_workspace_init(None, 256, None) == NULL
    assert lib.gtr_gla_workspace_init(FAKE + 16, 256, None) == WS
    assert lib.gtr_gla_workspace_init(FAKE, 250, None) == WS


def test_workspace_fault_rejects_bad_args(lib):
    assert lib.gtr_gla_workspace_fault(None, 256) == -1
    assert lib.gtr_gla_workspace_fault(FAKE, 16) == -1


# ---------------------------------------------------------------------------
# gtr_scan_permute
# ---------------------------------------------------------------------------

def perm(lib, src=FAKE, dst=FAKE + (1 << 30), outer=1, H=3, W=4, row=8, dt=gtr.F16, d=0, inv=0):
    return lib.gtr_scan_permute(src, dst, outer, H, W, row, dt, d, inv, None)


def test_permute_validation(lib):
    assert perm(lib, src=None) == NULL
    assert perm(lib, dst=None) == NULL
    assert perm(lib, outer=0) == SHAPE
    assert perm(lib, H=0) == SHAPE
    assert perm(lib, W=-2) == SHAPE
    assert perm(lib, row=0) == SHAPE
    assert perm(lib, outer=2 ** 62, H=2 ** 30, W=2 ** 30) == SHAPE
    assert perm(lib, dt=5) == UNSUP
    assert perm(lib, d=7) == UNSUP
    assert perm(lib, inv=2) == UNSUP
    assert perm(lib, dst=FAKE + 64) == ALIAS


# ---------------------------------------------------------------------------
# gate fusion and output-gate epilogue arguments
# ---------------------------------------------------------------------------

def test_gate_kind_and_tau_checked(lib):
    a = base_args()
    a.g_kind = 2
    assert fwd(lib, a) == UNSUP
    for tau in (0.0, -1.0, float("nan"), float("inf")):
        a = base_args()
        a.g_kind = gtr.GATE_LOGITS
        a.gate_tau = tau
        assert fwd(lib, a) == UNSUP, tau
        assert lib.gtr_gla_workspace_size(ctypes.byref(a)) == 0


def epilogue_args(**kw):
    a = base_args(**kw)
    n_in = a.B * a.heads * a.H * a.W * 64 * 4
    a.out_gate = FAKE + 5 * n_in
    a.out_gate_dtype = a.qkv_dtype
    a.norm_eps = 1e-5
    return a


def test_epilogue_arguments_checked(lib):
    a = epilogue_args()
    a.out_gate_dtype = gtr.BF16  # neither the input dtype (fp16) nor float32
    assert fwd(lib, a) == UNSUP
    for eps in (0.0, -1e-5, float("nan"), float("inf")):
        a = epilogue_args()
        a.norm_eps = eps
        assert fwd(lib, a) == UNSUP, eps
    a = epilogue_args()
    a.out_gate += 8  # the epilogue reads 16-byte pieces
    assert fwd(lib, a) == UNSUP
    a = epilogue_args()
    a.norm_weight = FAKE + 4  # misaligned weight
    assert fwd(lib, a) == UNSUP


def test_epilogue_gate_must_not_overlap_output(lib):
    a = epilogue_args()
    a.out_gate = a.o + 64
    assert fwd(lib, a) == ALIAS
    a = epilogue_args()
    a.norm_weight = a.o
    assert fwd(lib, a) == ALIAS


# ---------------------------------------------------------------------------
# gtr_spatial_swiglu
# ---------------------------------------------------------------------------

def swiglu_args(B=1, H=4, W=5, d=64, hidden=128, dt=gtr.F16):
    a = gtr.SwigluArgs()
    M = B * H * W
    step = 1 << 30
    a.x, a.w_gate, a.w_value, a.w_out = FAKE, FAKE + step, FAKE + 2 * step, FAKE + 3 * step
    a.conv_w, a.conv_b, a.y = FAKE + 4 * step, None, FAKE + 5 * step
    a.dtype, a.y_dtype = dt, dt
    a.B, a.H, a.W, a.d, a.hidden = B, H, W, d, hidden
    need = gtr.load().gtr_spatial_swiglu_workspace_size(ctypes.byref(a))
    a.workspace, a.workspace_bytes = FAKE + 6 * step, need
    return a


def sw(lib, a):
    return lib.gtr_spatial_swiglu(ctypes.byref(a), None)


def test_swiglu_workspace_size(lib):
    a = swiglu_args(B=2, H=40, W=40, d=384, hidden=1536)
    M = 2 * 1600
    a256 = lambda x: (x + 255) // 256 * 256
    # H in fp16 (G and V stay on chip); the output product splits K only when
    # its 64 x 64 tiles give fewer than 64 work-groups: 50 x 6 = 300 do not
    base = a256(M * 1536 * 2)
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(a)) == base
    one = swiglu_args(B=1, H=40, W=40, d=384, hidden=1536)  # 25 x 6 work-groups: no split
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(one)) == a256(1600 * 1536 * 2)
    small = swiglu_args(B=1, H=16, W=16, d=384, hidden=1536)  # 4 x 6 work-groups: 4 slices
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(small)) == \
        a256(a256(256 * 1536 * 2) + 4 * 256 * 384 * 4)
    tiny = swiglu_args(B=1, H=8, W=8, d=64, hidden=2048)  # 1 work-group: 8 slices (the most)
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(tiny)) == \
        a256(a256(64 * 2048 * 2) + 8 * 64 * 64 * 4)
    big = swiglu_args(B=8, H=40, W=40, d=384, hidden=1536)  # 100 x 6 work-groups: no split
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(big)) == a256(12800 * 1536 * 2)


@pytest.mark.parametrize("field,val,want", [("B", 0, SHAPE), ("H", -1, SHAPE), ("d", 48, UNSUP),
                                            ("hidden", 100, UNSUP), ("dtype", gtr.F32, UNSUP)])
def test_swiglu_bad_arguments(lib, field, val, want):
    a = swiglu_args()
    setattr(a, field, val)
    assert sw(lib, a) == want


def test_swiglu_grid_bounds(lib):
    """Launch sizes are checked on the host: 2^30 one-token images at hidden
    192 would need 3 * 2^30 gated-convolution work-groups (more than 2^31 - 1):
    GTR_ERR_SHAPE, with no launch; at hidden 64 (2^30 work-groups) the shape
    is accepted."""
    a = swiglu_args(B=1 << 30, H=1, W=1, d=64, hidden=192)
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(a)) == 0
    assert sw(lib, a) == SHAPE
    a = swiglu_args(B=1 << 30, H=1, W=1, d=64, hidden=64)
    assert lib.gtr_spatial_swiglu_workspace_size(ctypes.byref(a)) > 0


def test_swiglu_nulls_alignment_alias_workspace(lib):
    a = swiglu_args()
    a.w_out = None
    assert sw(lib, a) == NULL
    a = swiglu_args()
    a.conv_b = FAKE + 8
    assert sw(lib, a) == UNSUP
    a = swiglu_args()
    a.y = a.x  # output over the input
    assert sw(lib, a) == ALIAS
    a = swiglu_args()
    a.workspace_bytes -= 256
    assert sw(lib, a) == WS
    a = swiglu_args()
    a.y_dtype = gtr.BF16  # neither fp16 (the input dtype) nor float32
    assert sw(lib, a) == UNSUP


# ---------------------------------------------------------------------------
# gtr_gla_fwd_noalloc: validation before any HIP call
# ---------------------------------------------------------------------------

def test_noalloc_validation(lib):
    assert lib.gtr_gla_fwd_noalloc(None, None) == 1  # GTR_ERR_NULL
    a = base_args(B=8, heads=12, H=40, W=40)  # a batch of 8 images of 12 heads: about 80 MB of workspace
    assert lib.gtr_gla_workspace_size(ctypes.byref(a)) > 32 << 20
    assert lib.gtr_gla_fwd_noalloc(ctypes.byref(a), None) == 7  # GTR_ERR_SCRATCH, nothing launched
    a = base_args(B=1, heads=6, H=40, W=40)
    a.dk = 48
    assert lib.gtr_gla_fwd_noalloc(ctypes.byref(a), None) == UNSUP
    a = base_args(B=1, heads=6, H=40, W=40)
    a.workspace, a.workspace_bytes = None, 0  # ignored by this entry point
    assert lib.gtr_gla_workspace_size(ctypes.byref(a)) <= 32 << 20


# ---------------------------------------------------------------------------
# gtr_gemm: the row normalisation's argument checks (before any HIP call)
# ---------------------------------------------------------------------------

def gemm_args(M=200, N=128, K=192):
    g = gtr.GemmArgs()
    step = 1 << 30
    g.a, g.b, g.c = FAKE, FAKE + step, FAKE + 2 * step
    g.a_dtype = g.b_dtype = g.c_dtype = gtr.F16
    g.M, g.N, g.K = M, N, K
    g.row_norm, g.row_norm_eps = 1, 1e-6
    return g


@pytest.mark.parametrize("field,val", [("a_tokens", 100), ("row_norm_eps", -1.0), ("row_norm_eps", float("nan")),
                                       ("row_norm", 2)])
def test_gemm_row_norm_rejects(lib, field, val):
    g = gemm_args()
    setattr(g, field, val)
    assert lib.gtr_gemm(ctypes.byref(g), None) == UNSUP
