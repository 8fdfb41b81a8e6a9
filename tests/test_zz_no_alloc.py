"""gtr_gla_fwd_noalloc (the entry point for callers that cannot allocate)
against gtr_gla_fwd, through the C ABI: two calls in a row, the second on a
smaller input, each compared with gtr_gla_fwd on the same arguments. Both run
the same kernels, so the results agree bit for bit (the chunk schedule of these
shapes sums every state in a fixed order); the first call is also checked
against the oracle at the parity bar."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_26590_amd.workloads import WORKLOADS, make_inputs, torch_dtype

pytestmark = pytest.mark.gpu


def _call(gtr, fn, wl, inp, o, sf, ws):
    dev = torch.device("cuda")
    q, k, v, g = (inp[n] for n in ("q", "k", "v", "g"))
    a = gtr.make_args(q, k, v, g, H=wl.H, W=wl.W, scale=wl.scale, chunk=wl.chunk, s0=inp["s0"], o=o,
                      s_final=sf, path="auto", workspace=ws)
    st = fn(ctypes.byref(a), ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    torch.cuda.synchronize()
    return st


def test_noalloc_matches_gtr_gla_fwd_twice(gtr):
    lib = gtr.load()
    dev = torch.device("cuda")
    cases = [WORKLOADS["kbench"].with_(s0_std=0.1, want_final=True),             # 6 heads, 40 x 40
             WORKLOADS["tiny"].with_(dtype="f16", odtype="f16", s0_std=0.1, want_final=True)]  # smaller
    for i, wl in enumerate(cases):
        inp = {n: (None if t is None else t.to(dev)) for n, t in make_inputs(wl).items()}
        outs = []
        for fn in (lib.gtr_gla_fwd_noalloc, lib.gtr_gla_fwd):
            o = torch.full((wl.B, wl.heads, wl.L, wl.dv), float("nan"), dtype=torch_dtype(wl.odtype), device=dev)
            sf = torch.full((wl.B, wl.heads, wl.dk, wl.dv), float("nan"), dtype=torch.float32, device=dev)
            ws = None
            if fn is lib.gtr_gla_fwd:
                probe = gtr.make_args(inp["q"], inp["k"], inp["v"], inp["g"], H=wl.H, W=wl.W, scale=wl.scale,
                                      chunk=wl.chunk, s0=inp["s0"], o=o, s_final=sf)
                ws = torch.empty(gtr.gtr_gla_workspace_size(probe), dtype=torch.uint8, device=dev)
                gtr.gtr_gla_workspace_init(ws)
            assert _call(gtr, fn, wl, inp, o, sf, ws) == 0
            outs.append((o, sf))
        (o1, s1), (o2, s2) = outs
        assert torch.equal(o1, o2), f"call {i}: outputs differ"
        assert torch.equal(s1, s2), f"call {i}: final states differ"
        if i == 0:
            cpu = make_inputs(wl)
            o_ref, s_ref = oracle.gla(cpu["q"], cpu["k"], cpu["v"], cpu["g"], cpu["s0"], scale=wl.scale, H=wl.H,
                                      W=wl.W)
            err = np.max(np.abs(o1.double().cpu().numpy() - o_ref)) / (np.max(np.abs(o_ref)) + 1e-6)
            assert err <= 2e-3, err


def test_noalloc_rejects_a_call_beyond_its_scratch(gtr):
    lib = gtr.load()
    dev = torch.device("cuda")
    wl = WORKLOADS["batched"]  # 96 sequences: about 80 MB of workspace
    mk = lambda d: torch.empty((wl.B, wl.heads, wl.L, d), dtype=torch_dtype(wl.dtype), device=dev)
    o = torch.full((wl.B, wl.heads, wl.L, wl.dv), 7.0, dtype=torch.float32, device=dev)
    a = gtr.make_args(mk(64), mk(64), mk(64), mk(64), H=wl.H, W=wl.W, scale=wl.scale, o=o)
    assert lib.gtr_gla_fwd_noalloc(ctypes.byref(a), ctypes.c_void_p(0)) == 7  # GTR_ERR_SCRATCH
    torch.cuda.synchronize()
    assert torch.all(o == 7.0)  # nothing was launched
