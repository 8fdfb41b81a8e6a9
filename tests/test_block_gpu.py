"""GPU parity of one GTR block (Sec. 3.1) and of the calls it is made of.

The block's reading (pre-norm layer normalisation before the token mixer and
before the Spatial SwiGLU, a residual around each) and its parts are pinned in
tests/test_oracle_pins.py; here the HIP path runs them through the C ABI and
is compared with the float64 oracle on the same seeded values.

Tolerances: the helpers round once into fp16 (2^-11 relative) after float32
arithmetic. The block rounds about ten intermediates to fp16 (the normalised
inputs, the projections, the gate logits, the gated GLA output, the residual
sums, and the Spatial SwiGLU's own fp16 products) and each product adds the
rounding of its inputs times sqrt(K)-sized sums of random signs; the last
rounding alone (x2 in fp16, |x2| up to about 8) is half an ulp of 2^-9 x 8.
The output is held to 5e-3 of the largest |x2 - x| (what the block adds to
its input) and to 2e-3 of the largest |x2| (measured: about 1.1e-3 and 0.8e-3
of those at the GTR-S and GTR-L widths).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_26590_amd as gtr
from paper_2609_26590_amd import block
from paper_2609_26590_amd.workloads import SCANS, make_block

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda")


def rnd(rng, *shape, std=1.0, dtype=torch.float16):
    return torch.from_numpy(rng.standard_normal(shape) * std).to(torch.float32).to(dtype)


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("M,N,K,bias,res,cdt", [(200, 128, 192, True, True, None), (1600, 1536, 384, False, False, None),
                                                 (37, 64, 64, True, False, torch.float32), (1, 384, 64, False, True, None)])
def test_gemm_parity(dtype, M, N, K, bias, res, cdt):
    rng = np.random.default_rng(M + N + K)
    a, b = rnd(rng, M, K, dtype=dtype), rnd(rng, N, K, std=K ** -0.5, dtype=dtype)
    bi = rnd(rng, N, dtype=torch.float32) if bias else None
    cdt = cdt or dtype
    rs = rnd(rng, M, N, dtype=cdt) if res else None
    c = gtr.gtr_gemm(a.to(DEV), b.to(DEV), bias=None if bi is None else bi.to(DEV),
                     res=None if rs is None else rs.to(DEV), out_dtype=cdt)
    torch.cuda.synchronize()
    want = a.double().numpy() @ b.double().numpy().T
    if bias:
        want = want + bi.double().numpy()
    if res:
        want = want + rs.double().numpy()
    got = c.double().cpu().numpy()
    ulp = 2.0 ** -8 if cdt == torch.bfloat16 else (2.0 ** -11 if cdt == torch.float16 else 0.0)
    err = np.max(np.abs(got - want) / (np.abs(want) * ulp + 1e-3 * np.max(np.abs(want))))
    assert err <= 1.0, err


def test_gemm_residual_in_place():
    rng = np.random.default_rng(3)
    a, b = rnd(rng, 300, 128).to(DEV), rnd(rng, 192, 128, std=128 ** -0.5).to(DEV)
    r = rnd(rng, 300, 192).to(DEV)
    want = gtr.gtr_gemm(a, b, res=r)
    got = r.clone()
    gtr.gtr_gemm(a, b, res=got, out=got)
    torch.cuda.synchronize()
    assert torch.equal(got, want)


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("M,N,K,offset", [(1600, 1920, 384, 1.0), (200, 128, 192, 40.0), (37, 64, 64, 0.0),
                                          (1, 384, 384, 5.0), (3200, 384, 192, 300.0)])
def test_gemm_row_norm(dtype, M, N, K, offset):
    """gtr_gemm with row_norm: the layer normalisation (no affine weights) of
    every row of a, then the product, against the float64 oracle's
    layer_norm. Row means up to 300 times the spread check the shifted
    squares; every seventh row is constant (variance zero, the result is the
    bias alone); grids below and above 256 tiles run both kernel shapes."""
    rng = np.random.default_rng(M + K)
    a = (rnd(rng, M, K, dtype=torch.float32) * 3 + torch.from_numpy(rng.uniform(-1, 1, (M, 1)) * offset).float())
    a[::7] = torch.from_numpy(rng.uniform(-4, 4, (len(range(0, M, 7)), 1))).float()  # constant rows: zero spread
    a = a.to(dtype)
    b = rnd(rng, N, K, std=K ** -0.5, dtype=dtype)
    bi = rnd(rng, N, dtype=torch.float32)
    c = gtr.gtr_gemm(a.to(DEV), b.to(DEV), bias=bi.to(DEV), row_norm_eps=1e-6)
    torch.cuda.synchronize()
    want = oracle.layer_norm(a.double().numpy(), None, None, 1e-6) @ b.double().numpy().T + bi.double().numpy()
    got = c.double().cpu().numpy()
    ulp = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -11
    err = np.max(np.abs(got - want) / (np.abs(want) * ulp + 1e-3 * np.max(np.abs(want))))
    assert err <= 1.0, err


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("B,L,heads,parts", [(1, 1600, 6, 4), (2, 207, 3, 1)])
def test_gemm_head_major_operands(dtype, B, L, heads, parts):
    """gtr_gemm storing c head-major and reading a head-major a: the same
    products, placed as a reshape and transpose of the row-major ones."""
    rng = np.random.default_rng(L + parts)
    d = 64 * heads
    a = rnd(rng, B * L, d, dtype=dtype).to(DEV)
    w = rnd(rng, parts * d, d, std=d ** -0.5, dtype=dtype).to(DEV)
    bias = rnd(rng, parts * d, dtype=torch.float32).to(DEV)
    plain = gtr.gtr_gemm(a, w, bias=bias)
    hm = gtr.gtr_gemm(a, w, bias=bias, heads_out=(L, heads, 64))
    torch.cuda.synchronize()
    assert torch.equal(hm, plain.reshape(B, L, parts, heads, 64).permute(2, 0, 3, 1, 4))
    # a head-major a (as the GLA output) against its head concat
    u = hm[0].contiguous()                       # [B, heads, L, 64]
    wo = rnd(rng, d, d, std=d ** -0.5, dtype=dtype).to(DEV)
    got = gtr.gtr_gemm(u, wo, res=a)
    want = gtr.gtr_gemm(u.permute(0, 2, 1, 3).reshape(B * L, d).contiguous(), wo, res=a)
    torch.cuda.synchronize()
    assert torch.equal(got, want)


@pytest.mark.parametrize("B,H,W", [(1, 40, 40), (2, 9, 23)])
def test_spatial_swiglu_residual(B, H, W):
    """y = residual + SwiGLU(x), in place on the residual too."""
    rng = np.random.default_rng(H * W)
    d, h = 192, 768
    x = rnd(rng, B, H * W, d).to(DEV)
    wg, wv = rnd(rng, h, d, std=d ** -0.5).to(DEV), rnd(rng, h, d, std=d ** -0.5).to(DEV)
    wo = rnd(rng, d, h, std=h ** -0.5).to(DEV)
    cw = rnd(rng, h, 3, 3, std=1 / 3, dtype=torch.float32).to(DEV)
    r = rnd(rng, B, H * W, d).to(DEV)
    y0 = gtr.gtr_spatial_swiglu(x, wg, wv, wo, cw, H=H, W=W, y_dtype=torch.float32)
    y1 = gtr.gtr_spatial_swiglu(x, wg, wv, wo, cw, H=H, W=W, residual=r)
    y2 = r.clone()
    gtr.gtr_spatial_swiglu(x, wg, wv, wo, cw, H=H, W=W, residual=y2, out=y2)
    torch.cuda.synchronize()
    want = (y0.double() + r.double()).cpu().numpy()
    tol = 2.0 ** -11 * np.abs(want) + 1e-6
    assert np.all(np.abs(y1.double().cpu().numpy() - want) <= tol)
    assert torch.equal(y1, y2)


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("M,d,affine", [(1600, 384, True), (33, 192, False), (5, 2048, True), (4, 8, True)])
def test_layernorm_parity(dtype, M, d, affine):
    rng = np.random.default_rng(M * d)
    x = (rnd(rng, M, d, dtype=torch.float32) * 3 + 1).to(dtype)
    w = rnd(rng, d, std=0.1, dtype=torch.float32) + 1 if affine else None
    b = rnd(rng, d, std=0.1, dtype=torch.float32) if affine else None
    y = gtr.gtr_layernorm(x.to(DEV), None if w is None else w.to(DEV), None if b is None else b.to(DEV), eps=1e-6)
    torch.cuda.synchronize()
    want = oracle.layer_norm(x.double().numpy(), None if w is None else w.numpy(), None if b is None else b.numpy(),
                             1e-6)
    ulp = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -11
    err = np.max(np.abs(y.double().cpu().numpy() - want))
    assert err <= 2 * ulp * np.max(np.abs(want)) + 1e-5, err


@pytest.mark.parametrize("parts,B,heads,L,dh", [(4, 1, 6, 1600, 64), (1, 2, 3, 37, 64), (2, 3, 2, 5, 8)])
def test_heads_split_and_merge_are_exact(parts, B, heads, L, dh):
    rng = np.random.default_rng(parts * 100 + L)
    ld = parts * heads * dh + (8 if parts == 2 else 0)  # a padded row pitch for one case
    src = rnd(rng, B * L, ld)
    got = gtr.gtr_heads_split(src.to(DEV), parts=parts, B=B, heads=heads, dh=dh)
    want = src[:, :parts * heads * dh].reshape(B, L, parts, heads, dh).permute(2, 0, 3, 1, 4)
    assert torch.equal(got.cpu(), want)
    back = gtr.gtr_heads_merge(got[0].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(back.cpu(), src[:, :heads * dh])


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
def test_add_parity(dtype):
    rng = np.random.default_rng(9)
    a, b = rnd(rng, 1600, 384, dtype=dtype), rnd(rng, 1600, 384, dtype=dtype)
    y = gtr.gtr_add(a.to(DEV), b.to(DEV))
    torch.cuda.synchronize()
    want = (a.double() + b.double()).numpy()
    ulp = 2.0 ** -8 if dtype == torch.bfloat16 else 2.0 ** -11
    assert np.all(np.abs(y.double().cpu().numpy() - want) <= ulp * np.abs(want) + 1e-7)


def run_block(name, scan, H=40, W=40, B=1, dtype="f16"):
    x, p = make_block(name, H, W, B=B, dtype=dtype)
    heads = {"gtr_s": 3, "gtr_l": 6}[name]
    pd = block.prepare({k: v.to(DEV) for k, v in p.items()})
    y = block.forward(x.to(DEV), pd, H=H, W=W, heads=heads, scan=scan)
    torch.cuda.synchronize()
    want = oracle.gtr_block(x.double().numpy(), {k: v.double().numpy() for k, v in p.items()}, H=H, W=W, heads=heads,
                            scan=scan)
    return x.double().numpy(), y.double().cpu().numpy(), want


@pytest.mark.parametrize("scan", SCANS)
@pytest.mark.parametrize("name", ["gtr_s", "gtr_l"])
def test_block_parity(name, scan):
    x, got, want = run_block(name, scan)
    err = np.max(np.abs(got - want))
    inc = np.max(np.abs(want - x))
    print(f"{name} {scan}: max err {err:.3e}, max |increment| {inc:.3e}, max |out| {np.max(np.abs(want)):.3e}")
    assert err <= 5e-3 * inc, (err, inc)
    assert err <= 2e-3 * np.max(np.abs(want)), err


def test_block_ragged_grid_two_images():
    """Two images on a grid whose chunks and tiles do not divide it."""
    x, got, want = run_block("gtr_s", "col", H=9, W=23, B=2)
    err = np.max(np.abs(got - want))
    assert err <= 5e-3 * np.max(np.abs(want - x)), err


@pytest.mark.parametrize("scan", ["row_rev", "col"])
def test_block_parity_bf16(scan):
    """bf16 activations and weights (the products on bf16 MFMA, the GLA on fp16
    operands with its range check): one bf16 rounding (2^-8 relative) per
    stored intermediate, so the bars are 8x the fp16 ones."""
    x, got, want = run_block("gtr_l", scan, dtype="bf16")
    err = np.max(np.abs(got - want))
    inc = np.max(np.abs(want - x))
    print(f"gtr_l bf16 {scan}: max err {err:.3e}, max |increment| {inc:.3e}")
    assert err <= 4e-2 * inc, (err, inc)
    assert err <= 1.6e-2 * np.max(np.abs(want)), err


def test_block_graph_replays_match_eager():
    """The whole block captured in one HIP graph (the layer norm, the products,
    the GLA call with its default workspace, the Spatial SwiGLU) replays to the
    eager result bit for bit, several times, with eager blocks in between."""
    x, p = make_block("gtr_s", 9, 23, B=2)
    pd = block.prepare({k: v.to(DEV) for k, v in p.items()})
    x = x.to(DEV)
    run = lambda: block.forward(x, pd, H=9, W=23, heads=3, scan="col_rev")
    want = run().clone()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        y = run()
    for rep in range(4):
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, want), f"replay {rep} differs"
        assert torch.equal(run(), want)  # eager work between replays
        torch.cuda.synchronize()
