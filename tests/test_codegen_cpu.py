"""CPU check of the generated gfx950 code: every memory address that the GLA
kernels form is defined for every active lane and lies inside its buffer.

The kernels are compiled to gfx950 assembly with the library's own flags and
executed wave by wave in ``gfx950_wave`` (an emulator of our own listing, run
on the CPU). This guards against a class of defect that source-level review
cannot see: the compiler once produced, for the bf16 instantiation only, a
global address from a register pair that was written on the fp16 and float32
paths but not on the bf16 one (for the lanes that used it). The first test pins
that the emulator reports exactly that pattern.
"""
from __future__ import annotations

import hashlib
import os
import re
import shutil
import struct
import subprocess

import pytest

import gfx950_wave as emu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_26590_amd", "csrc")
BUILD = os.path.join(ROOT, "paper_2609_26590_amd", "_build")

# ---------------------------------------------------------------------------
# the emulator catches the defect class (a hand-written kernel)
# ---------------------------------------------------------------------------
SNIPPET = """
{name}:
	s_load_dwordx2 s[4:5], s[0:1], 0x0
	{pre}
	v_cmp_gt_u32_e32 vcc, 32, v0
	s_and_saveexec_b64 s[6:7], vcc
	v_mov_b32_e32 v2, v0
	v_mov_b32_e32 v3, 0
	s_or_b64 exec, exec, s[6:7]
	s_waitcnt lgkmcnt(0)
	v_lshl_add_u64 v[2:3], v[2:3], 2, s[4:5]
	global_load_dword v4, v[2:3], off
	s_endpgm
.Lfunc_end0:
	.amdhsa_kernel {name}
		.amdhsa_group_segment_fixed_size 0
		.amdhsa_private_segment_fixed_size 0
		.amdhsa_kernarg_size 8
		.amdhsa_user_sgpr_count 2
		.amdhsa_user_sgpr_kernarg_segment_ptr 1
		.amdhsa_system_sgpr_workgroup_id_x 1
	.end_amdhsa_kernel
"""


def run_snippet(pre: str) -> emu.Report:
    name = "_Zsnippet"
    text = "\n" + SNIPPET.format(name=name, pre=pre)
    prog, labels, desc = emu.parse_kernel(text, name)
    base = 0x1000_0000_0000
    regions = [emu.Region("buf", base, 64 * 4, "r"), emu.Region("kernarg", emu.KERNARG_BASE, 8, "r")]
    rep = emu.Report()
    emu.run_wave(prog, labels, desc, struct.pack("<Q", base), regions, 0, (0, 0, 0), 0, rep)
    return rep


def test_emulator_flags_address_from_lanes_left_unwritten():
    # v[2:3] is written under the mask of lanes 0..31 only, then all 64 lanes
    # use it as an address: lanes 32..63 read whatever an earlier wave left
    rep = run_snippet("s_nop 0")
    assert rep.counts.get("ERR-UNDEF-ADDR", 0) == 1
    (_, raw, detail), = rep.items["ERR-UNDEF-ADDR"]
    assert raw.startswith("global_load_dword") and "32" in detail


def test_emulator_passes_the_same_code_with_every_lane_written():
    rep = run_snippet("v_mov_b32_e32 v2, v0\n\tv_mov_b32_e32 v3, 0")
    assert not [k for k in rep.counts if k.startswith("ERR")], dict(rep.counts)


def test_emulator_flags_out_of_bounds():
    # every lane writes its address (word tid + 1), lane 63 lands one word past
    # the 64-word buffer; v0 = 64 leaves the masked block with no lanes
    rep = run_snippet("v_add_u32_e32 v2, 1, v0\n\tv_mov_b32_e32 v3, 0\n\tv_mov_b32_e32 v0, 64")
    assert rep.counts.get("ERR-OOB", 0) >= 1


WINDOW_SNIPPET = """
{name}:
	s_load_dwordx2 s[4:5], s[0:1], 0x0
	s_waitcnt lgkmcnt(0)
	v_mov_b32_e32 v2, s4
	v_mov_b32_e32 v3, s5
	global_load_dword v4, v[2:3], off
	s_mov_b32 s8, s4
	s_and_b32 s9, s5, 0xffff
	s_mov_b32 s10, {nrec}
	s_mov_b32 s11, 0x20000
	s_waitcnt vmcnt(0)
	buffer_load_dword v5, v4, s[8:11], 0 offen
	s_endpgm
.Lfunc_end0:
	.amdhsa_kernel {name}
		.amdhsa_group_segment_fixed_size 0
		.amdhsa_private_segment_fixed_size 0
		.amdhsa_kernarg_size 8
		.amdhsa_user_sgpr_count 2
		.amdhsa_user_sgpr_kernarg_segment_ptr 1
		.amdhsa_system_sgpr_workgroup_id_x 1
	.end_amdhsa_kernel
"""


def test_emulator_bounds_a_data_dependent_buffer_offset_by_its_descriptor():
    # the offset of the buffer load is loaded data (unknown): safe exactly when
    # the descriptor's whole window lies inside the 256-byte buffer
    for nrec, bad in ((256, False), (260, True)):
        name = "_Zwindow"
        prog, labels, desc = emu.parse_kernel("\n" + WINDOW_SNIPPET.format(name=name, nrec=nrec), name)
        base = 0x1000_0000_0000
        regions = [emu.Region("buf", base, 64 * 4, "r"), emu.Region("kernarg", emu.KERNARG_BASE, 8, "r")]
        rep = emu.Report()
        emu.run_wave(prog, labels, desc, struct.pack("<Q", base), regions, 0, (0, 0, 0), 0, rep)
        assert (rep.counts.get("ERR-OOB", 0) >= 1) == bad, (nrec, dict(rep.counts))
        assert (rep.counts.get("INFO-DATA-OFFSET", 0) >= 1) == (not bad), (nrec, dict(rep.counts))
        assert "WARN-DATA-ADDR" not in rep.counts


# ---------------------------------------------------------------------------
# the library's kernels
# ---------------------------------------------------------------------------
DT = {"f32": (0, 4), "f16": (1, 2), "bf16": (2, 2)}
SCAN = {"row": 0, "col": 1, "row_rev": 2, "col_rev": 3}
KERNARG_BYTES = 216  # sizeof(GlaParams)


def a256(x):
    return (x + 255) & ~255


def device_asm() -> str:
    """gfx950 assembly of the GLA kernels (gla_fwd.hip, gla_lean.hip) with the
    library's flags, cached by source hash."""
    from paper_2609_26590_amd import build as b
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    with open(os.path.join(ROOT, "include", "gtr.h"), "rb") as fh:
        h.update(fh.read())
    h.update(" ".join(b.HIPCC_FLAGS).encode())
    os.makedirs(BUILD, exist_ok=True)
    texts = []
    for src in ("gla_fwd.hip", "gla_lean.hip"):
        path = os.path.join(BUILD, f"{src[:-4]}.gfx950.{h.hexdigest()[:16]}.s")
        if not os.path.exists(path):
            hipcc = b._hipcc() if shutil.which("hipcc") or os.path.exists("/opt/rocm/bin/hipcc") else None
            if hipcc is None:
                pytest.skip("hipcc is not available")
            tmp = path + f".tmp{os.getpid()}"
            r = subprocess.run([hipcc, *b.HIPCC_FLAGS, "-S", "--cuda-device-only", os.path.join(CSRC, src),
                                "-o", tmp], capture_output=True, text=True)
            assert r.returncode == 0, r.stderr[-2000:]
            os.replace(tmp, path)
        with open(path) as fh:
            texts.append(fh.read())
    return "\n".join(texts)


class Shape:
    def __init__(self, B, heads, H, W, dk, dv, chunk, dt, gdt, odt, scan, s0, sfinal, logits=False, zdt=None,
                 weighted=False):
        self.logits, self.zdt, self.weighted = logits, zdt, weighted
        self.B, self.heads, self.H, self.W = B, heads, H, W
        self.dk, self.dv, self.chunk = dk, dv, chunk
        self.dt, self.gdt, self.odt, self.scan, self.s0, self.sfinal = dt, gdt, odt, scan, s0, sfinal
        self.BH = B * heads
        self.L = H * W
        self.NC = (self.L + chunk - 1) // chunk


class Launch:
    """How the one-launch kernel is run: value parts, descending chunk order
    (every work-group resident), inclusive states published, the value every
    chunk flag reads as (FLAG_SUMMARY: summaries only, the look-back walks back
    to the start; FLAG_ALL: inclusive states everywhere as well, it stops at the
    nearest; FLAG_NONE: nothing is ever ready, every wait runs out after the
    spin limit), the XCDs of the sequence-per-XCD grid (0: chunk-major) and the
    grouped look-back of the 16-bit kernel (FLAG_GROUP: every group aggregate
    is stored)."""

    def __init__(self, vparts=1, desc=0, publish=1, flag=1, nxcd=0, group=0):
        self.vparts, self.desc, self.publish, self.flag, self.nxcd = vparts, desc, publish, flag, nxcd
        self.group = group


def kernel_args(c: Shape, ln: Launch = Launch()):
    """GlaParams for shape c with every buffer at its own base, and the buffers."""
    regions = []
    nxt = [0x1000_0000_0000]

    def alloc(name, size, mode):
        base = nxt[0]
        nxt[0] += 0x10_0000_0000
        if size:
            regions.append(emu.Region(name, base, size, mode))
        return base if size else 0

    esz = DT[c.dt][1]
    q = alloc("q", c.BH * c.L * c.dk * esz, "r")
    k = alloc("k", c.BH * c.L * c.dk * esz, "r")
    v = alloc("v", c.BH * c.L * c.dv * esz, "r")
    g = alloc("g", c.BH * c.L * c.dk * DT[c.gdt][1], "r")
    o = alloc("o", c.BH * c.L * c.dv * DT[c.odt][1], "w")
    s0 = alloc("s0", c.BH * c.dk * c.dv * 4, "r") if c.s0 else 0
    sf = alloc("s_final", c.BH * c.dk * c.dv * 4, "w") if c.sfinal else 0
    z = alloc("out_gate", c.BH * c.L * c.dv * DT[c.zdt][1], "r") if c.zdt else 0
    nw = alloc("norm_weight", c.dv * 4, "r") if c.zdt and c.weighted else 0
    # workspace layout of gla_workspace_layout(): header (fault word), done
    # counters, chunk flags, summaries, chunk records, states
    sync = 256
    flags = a256(sync + 1024 * 16)
    agg = a256(flags + 1024 * 256 * 4)
    tiles = c.BH * c.NC
    rec = a256(agg + tiles * c.dk * c.dv * (4 if c.dt == "f32" else 2))
    states = a256(rec + 2 * tiles * (2 * c.dk) * 4)
    total = a256(states + tiles * c.dk * c.dv * 4)
    ws = alloc("workspace", total, "rw")
    ns = c.BH * ln.vparts
    regions.insert(0, emu.Region("flags", ws + flags, 1024 * 256 * 4, "rw", load_value=ln.flag))
    regions.insert(0, emu.Region("sync", ws + sync, ns * 16, "rw"))
    regions.insert(0, emu.Region("fault", ws, 256, "rw"))
    regions.append(emu.Region("kernarg", emu.KERNARG_BASE, KERNARG_BYTES, "r"))
    kern = struct.pack("<7Q6iqifi4x6Qif2Qif6iIi", q, k, v, g, o, s0, sf, DT[c.dt][0], DT[c.gdt][0],
                       DT[c.odt][0], c.BH, c.H, c.W, c.L, c.NC, c.dk ** -0.5, SCAN[c.scan],
                       ws + agg, ws + rec, ws + states, ws + sync, ws + flags, ws,
                       1 if c.logits else 0, 1.0 / 16, z, nw, DT[c.zdt][0] if c.zdt else 0, 1e-5,
                       c.dv, ln.vparts, ns, ln.desc, ln.publish, ln.nxcd, 8, ln.group)
    assert len(kern) == KERNARG_BYTES
    return kern, regions


def mangled(kind: str, c: Shape) -> str:
    t = f"ILi{c.dk}ELi{c.dv}ELi{c.chunk}ELi{DT[c.dt][0]}E"
    if kind == "summary":
        return f"_ZN3gtr18gla_summary_kernel{t}EEvNS_9GlaParamsE"
    if kind == "output":
        return f"_ZN3gtr17gla_output_kernel{t}EEvNS_9GlaParamsE"
    if kind == "scan":
        return f"_ZN3gtr15gla_scan_kernelILi{c.dk}ELi{c.dv}ELb{int(c.dt != 'f32')}EEEvNS_9GlaParamsE"
    if kind == "chain_split":  # d_v / 2 columns per work-group
        return f"_ZN3gtr16gla_chain_kernelILi{c.dk}ELi{c.dv // 2}ELi{c.chunk}ELi{DT[c.dt][0]}EEEvNS_9GlaParamsE"
    if kind in ("lean_split", "lean4_split"):
        occ = 4 if kind.startswith("lean4") else 3
        return f"_ZN3gtr15gla_lean_kernelILi{c.dk}ELi{c.dv // 2}ELi{c.chunk}ELi{DT[c.dt][0]}ELi{occ}EEEvNS_9GlaParamsE"
    if kind in ("lean", "lean4"):
        occ = 4 if kind == "lean4" else 3
        return f"_ZN3gtr15gla_lean_kernelILi{c.dk}ELi{c.dv}ELi{c.chunk}ELi{DT[c.dt][0]}ELi{occ}EEEvNS_9GlaParamsE"
    return f"_ZN3gtr16gla_chain_kernel{t}EEvNS_9GlaParamsE"


def work_groups(kind: str, c: Shape, ln: Launch):
    """Staged kernels: first, second and last chunk of the first and last
    sequence. One-launch kernels: first and second chunk of the first sequence
    and the last chunk of the last (+ the last chunk of the first group for the
    grouped look-back, + one block of the XCD-ordered grid that has no
    sequence)."""
    nw = c.chunk // 16
    cs = sorted({0, 1 % c.NC, c.NC - 1} | ({15} if ln.group and c.NC > 16 else set()))  # 15: a group's last chunk
    bhs = sorted({0, c.BH - 1})
    if kind in ("summary", "output"):
        return [((cc, bh, 0), nw) for cc in cs for bh in bhs]
    if kind == "scan":
        eb = (c.dk * c.dv + 255) // 256
        return [((x, bh, 0), 2) for x in sorted({0, eb - 1}) for bh in bhs]  # 128 threads
    ns = c.BH * ln.vparts
    # one-launch kernels: the first chunks (and a group's last) of the first
    # sequence, the last chunk of the last sequence
    pairs = sorted({(cc, 0) for cc in cs if cc != c.NC - 1 or c.NC == 1} | {(c.NC - 1, ns - 1)})
    row = lambda cc: (c.NC - 1 - cc) if ln.desc else cc
    if ln.nxcd > 1:
        # sequence-per-XCD grid: block (row * nx + j) * nxcd + x runs sequence
        # x + nxcd * j, nx = the sequences of XCD x; blocks past an XCD's share return
        nx = lambda x: (ns - x + ln.nxcd - 1) // ln.nxcd
        blocks = ln.nxcd * ((ns + ln.nxcd - 1) // ln.nxcd) * c.NC
        out = [(((row(cc) * nx(sq % ln.nxcd) + sq // ln.nxcd) * ln.nxcd + sq % ln.nxcd, 0, 0), nw)
               for cc, sq in pairs]
        pad = [(nx(x) * c.NC) * ln.nxcd + x for x in range(ln.nxcd)]
        out += [((bb, 0, 0), nw) for bb in pad if bb < blocks][:1]
        return out
    # chunk-major grid: block row * ns + seq, row = chunk (or NC - 1 - chunk)
    return [((row(cc) * ns + sq, 0, 0), nw) for cc, sq in pairs]


# (shape, kernels): the bf16 instantiations, float32 gates with 16-bit inputs,
# every chunk size, reversed and column scans, S0 / S_final, partial chunks;
# the one-launch kernels in both chunk orders, every flag state, the value split
# and (16-bit kernel) the sequence-per-XCD grid
CHAIN = ("chain", "chain_x", "chain_i")
# the 16-bit kernel at chunk 64: every launch variant on one shape, one variant on the others
LEAN = ("lean", "lean_n", "lean_x", "lean_i", "lean_xcd", "lean_split", "lean_g", "lean_gs", "lean4")
CHECKS = [
    (Shape(1, 12, 40, 40, 64, 64, 64, "bf16", "bf16", "f32", "row", False, False),
     ("summary", "scan", "output") + CHAIN + ("chain_split",) + LEAN),
    (Shape(8, 12, 40, 40, 64, 64, 64, "bf16", "bf16", "f32", "col_rev", True, True), ("output",) + CHAIN + ("lean_x", "lean_g")),
    (Shape(2, 9, 12, 20, 32, 32, 32, "bf16", "f32", "f32", "col", True, True), ("summary", "output") + CHAIN),
    (Shape(1, 2, 20, 20, 32, 64, 128, "bf16", "bf16", "bf16", "row_rev", False, False), ("output",) + CHAIN),
    (Shape(1, 6, 40, 40, 64, 64, 64, "f16", "f16", "f16", "row", False, False),
     CHAIN + ("chain_split", "lean_split")),
    (Shape(1, 5, 9, 23, 32, 64, 64, "f16", "f32", "f32", "row_rev", True, True), ("lean", "lean_split", "lean4", "lean4_gs")),
    (Shape(3, 3, 16, 16, 32, 32, 64, "bf16", "f32", "bf16", "col", False, True), ("lean_xcd",)),
    (Shape(1, 3, 7, 9, 64, 64, 128, "f16", "f32", "f32", "col", True, True), ("output",) + CHAIN + ("chain_split",)),
    (Shape(1, 2, 13, 11, 64, 64, 32, "f32", "f32", "f32", "row_rev", True, True), CHAIN + ("chain_split",)),
    (Shape(1, 2, 13, 11, 32, 32, 32, "f32", "f32", "f32", "row", False, True), ("summary", "output") + CHAIN),
    (Shape(1, 6, 80, 80, 64, 64, 64, "f16", "f16", "f16", "row", False, False), ("scan",) + CHAIN + ("lean", "lean_g", "lean4_g")),
    # gate fusion and the output-gate epilogue
    (Shape(1, 12, 40, 40, 64, 64, 64, "bf16", "bf16", "f32", "col", True, True, True, "bf16", True),
     ("summary", "output") + CHAIN + ("lean_i",)),
    (Shape(2, 3, 8, 8, 64, 64, 64, "f16", "f32", "f16", "row", False, False, True, "f32", False), ("lean",)),
    (Shape(1, 3, 7, 9, 32, 64, 32, "f16", "f32", "f16", "row_rev", False, False, True, "f32", False),
     ("summary", "output", "chain")),
]


# summaries only; summaries and inclusive states; nothing; summaries and group aggregates
FLAG_SUMMARY, FLAG_ALL, FLAG_NONE, FLAG_GROUP = 1, 3, 0, 9


def launches(kind: str, c: Shape):
    """The launch variants a kind stands for."""
    if kind == "chain":  # ascending chunks, summaries only: the look-back reads back to the start
        return [Launch(flag=FLAG_SUMMARY), Launch(flag=FLAG_NONE)]
    if kind == "chain_x":  # descending chunks, inclusive states everywhere
        return [Launch(desc=1, flag=FLAG_ALL)]
    if kind == "chain_i":  # no inclusive states published (the inline form)
        return [Launch(desc=1, publish=0, flag=FLAG_SUMMARY)]
    if kind == "chain_split":
        return [Launch(vparts=2, flag=FLAG_SUMMARY), Launch(vparts=2, desc=1, flag=FLAG_ALL)]
    if kind == "lean":
        return [Launch(flag=FLAG_SUMMARY)]
    if kind == "lean_n":
        return [Launch(flag=FLAG_NONE)]
    if kind == "lean_x":
        return [Launch(desc=1, flag=FLAG_ALL)]
    if kind == "lean_i":
        return [Launch(desc=1, publish=0, flag=FLAG_SUMMARY)]
    if kind == "lean_xcd":  # eight XCDs, every sequence's chunks on one
        return [Launch(desc=1, flag=FLAG_SUMMARY, nxcd=8)]
    if kind == "lean_split":
        return [Launch(vparts=2, desc=1, flag=FLAG_ALL, nxcd=8)]
    if kind == "lean_g":  # grouped look-back: aggregates back to the start; inclusive states; nothing ready
        return [Launch(group=1, flag=FLAG_GROUP), Launch(group=1, desc=1, flag=FLAG_ALL | FLAG_GROUP),
                Launch(group=1, flag=FLAG_NONE)]
    if kind == "lean_gs":  # grouped look-back with the value split
        return [Launch(vparts=2, group=1, flag=FLAG_GROUP)]
    if kind == "lean4":  # four work-groups per CU: summaries back to the start, inclusive states
        return [Launch(flag=FLAG_SUMMARY), Launch(desc=1, flag=FLAG_ALL)]
    if kind == "lean4_g":
        return [Launch(group=1, flag=FLAG_GROUP), Launch(group=1, flag=FLAG_NONE)]
    if kind == "lean4_gs":
        return [Launch(vparts=2, group=1, flag=FLAG_GROUP | FLAG_ALL)]
    return [Launch()]


def split_name(kind):
    """The kernel a kind runs: the value-split instantiation for the split kinds
    (lean4: the four-per-CU instantiation of the 16-bit kernel)."""
    if kind in ("chain_split", "lean_split", "lean_gs", "lean4_gs"):
        return kind if kind == "chain_split" else kind.split("_")[0] + "_split"
    return kind.split("_")[0]


@pytest.fixture(scope="module")
def asm_text():
    return device_asm()


_JOBS = {}  # kernel listings shared with the forked workers


def _wave_job(job):
    name, kern, regions, wg, wave = job
    prog, labels, desc = _JOBS[name]
    rep = emu.Report()
    emu.run_wave(prog, labels, desc, kern, regions, desc["amdhsa_group_segment_fixed_size"], wg, wave, rep)
    return dict(rep.items), dict(rep.counts)


def run_waves(jobs):
    """Run independent waves (in forked worker processes where there are enough
    CPUs); the findings per job, in order."""
    workers = min(len(jobs), max(1, (os.cpu_count() or 1) // int(os.environ.get("PYTEST_XDIST_WORKER_COUNT", "1"))),
                  8)
    if workers <= 1:
        return [_wave_job(j) for j in jobs]
    import multiprocessing
    with multiprocessing.get_context("fork").Pool(workers) as pool:
        return pool.map(_wave_job, jobs, chunksize=1)


@pytest.mark.parametrize("case", range(len(CHECKS)))
def test_gla_kernel_addresses(asm_text, case):
    c, kinds = CHECKS[case]
    names = set(emu.kernel_names(asm_text))
    jobs, keys = [], []
    for kind in kinds:
        name = mangled(split_name(kind), c)
        assert name in names, f"no kernel {name} in the listing"
        if name not in _JOBS:
            _JOBS[name] = emu.parse_kernel(asm_text, name)
        assert _JOBS[name][2]["amdhsa_kernarg_size"] == KERNARG_BYTES
        for li, ln in enumerate(launches(kind, c)):
            kern, regions = kernel_args(c, ln)
            for wg, nw in work_groups(kind.split("_")[0], c, ln):
                for wave in range(nw):
                    jobs.append((name, kern, regions, wg, wave))
                    keys.append((kind, li))
    found = {}
    for key, (items, counts) in zip(keys, run_waves(jobs)):
        f = found.setdefault(key, ({}, set()))
        for k, v in items.items():
            if k.startswith(("ERR", "WARN", "NOTIMPL")):
                f[0].setdefault(k, set()).update(v)
        f[1].update(counts)
    for (kind, li), (bad, counts) in found.items():
        assert not bad, f"{kind} launch {li}: { {k: sorted(v)[:4] for k, v in bad.items()} }"
        assert "INFO-PATHLIMIT" not in counts, f"{kind} launch {li}: not every branch outcome was explored"


# ---------------------------------------------------------------------------
# Spatial SwiGLU kernels (swiglu.hip)
# ---------------------------------------------------------------------------
def swiglu_asm() -> str:
    from paper_2609_26590_amd import build as b
    src = os.path.join(CSRC, "swiglu.hip")
    h = hashlib.sha256()
    for f in ("swiglu.hip", "gtr_device.h", "gtr_internal.h"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "gtr.h"), "rb") as fh:
        h.update(fh.read())
    h.update(" ".join(b.HIPCC_FLAGS).encode())
    os.makedirs(BUILD, exist_ok=True)
    path = os.path.join(BUILD, f"swiglu.gfx950.{h.hexdigest()[:16]}.s")
    if not os.path.exists(path):
        tmp = path + f".tmp{os.getpid()}"
        r = subprocess.run([b._hipcc(), *b.HIPCC_FLAGS, "-S", "--cuda-device-only", src, "-o", tmp],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        os.replace(tmp, path)
    with open(path) as fh:
        return fh.read()


def check_kernel(text, name, kern, regions, wgs, waves=4):
    prog, labels, desc = emu.parse_kernel(text, name)
    rep = emu.Report()
    for wg in wgs:
        for wave in range(waves):
            emu.run_wave(prog, labels, desc, kern, regions, desc["amdhsa_group_segment_fixed_size"], wg, wave, rep)
    bad = {k: sorted(v)[:4] for k, v in rep.items.items() if k.startswith(("ERR", "WARN", "NOTIMPL"))}
    assert not bad, f"{name}: {bad}"
    assert "INFO-PATHLIMIT" not in rep.counts


@pytest.mark.parametrize("adt,bdt,mt,bn,M,N,K,cdt,ks,epi", [(1, 2, 1, 64, 126, 256, 64, 0, 1, 0),
                                                            (1, 1, 1, 64, 1600, 384, 1536, 1, 4, 0),
                                                            (1, 2, 1, 64, 63, 64, 128, 2, 1, 0),
                                                            (1, 1, 1, 64, 200, 192, 192, 1, 2, 0),
                                                            # gtr_gemm: bias and residual epilogue
                                                            (1, 1, 1, 64, 1600, 1536, 384, 1, 1, 3),
                                                            (2, 2, 2, 64, 37, 64, 64, 0, 1, 1),
                                                            (2, 2, 2, 64, 1, 384, 64, 2, 1, 2),
                                                            # head-major operands (the block's projections)
                                                            (1, 1, 1, 64, 1600, 1536, 384, 1, 1, 8),
                                                            (1, 1, 1, 64, 3200, 384, 384, 1, 1, 6),
                                                            (2, 2, 2, 64, 414, 384, 64, 2, 1, 9),
                                                            # 4 waves per tile at 256 tiles and more
                                                            (2, 2, 2, 64, 3200, 384, 64, 2, 1, 1),
                                                            (1, 2, 1, 64, 4096, 384, 128, 0, 1, 0),
                                                            # rows of A normalised (the block's first layer norm)
                                                            (1, 1, 1, 64, 1600, 1920, 384, 1, 1, 16 | 8 | 1),
                                                            (2, 2, 2, 64, 37, 128, 192, 2, 1, 16 | 2),
                                                            (1, 1, 1, 64, 200, 384, 64, 0, 1, 16)])
def test_swiglu_gemm_addresses(adt, bdt, mt, bn, M, N, K, cdt, ks, epi):
    """epi: bit 0 a bias, bit 1 a residual (gtr_gemm's epilogue), bits 2 / 3 head-major A / C, bit 4 the
    rows of A normalised."""
    text = swiglu_asm()
    base = 0x1000_0000_0000
    es = {0: 4, 1: 2, 2: 2}
    A, B, C, P, BI, R = (base + i * 0x10_0000_0000 for i in range(6))
    regions = [emu.Region("A", A, M * K * 2, "r"), emu.Region("B", B, N * K * 2, "r"),
               emu.Region("C", C, M * N * es[cdt], "w"),
               emu.Region("part", P, ks * M * N * 4, "w"),  # K-split partials are float32
               emu.Region("bias", BI, N * 4, "r"), emu.Region("res", R, M * N * es[cdt], "r"),
               emu.Region("kernarg", emu.KERNARG_BASE, 64, "r")]
    # epi bit 2: head-major A, bit 3: head-major C (6 heads of 64), two images of M / 2 tokens (one if M is odd)
    at = (M // 2 if M % 2 == 0 else M) if epi & 4 else 0
    ct = (M // 2 if M % 2 == 0 else M) if epi & 8 else 0
    kern = struct.pack("<QQQQiiiii4xQQqqiifi", A, B, C, P, M, N, K, cdt, ks, BI if epi & 1 else 0,
                       R if epi & 2 else 0, at, ct, 6 if ct else 0, 64 if ct else 0, 1e-6 if epi & 16 else 0.0, 0)
    # 8 waves per tile below 256 tiles (the K halves on separate waves), 4 above
    kw = 2 if ((M + 63) // 64) * (N // bn) * ks < 256 else 1
    name = f"_ZN3gtr14gemm_nt_kernelILi{adt}ELi{bdt}ELi{mt}ELi64ELi{bn}ELi{kw}ELi{1 if epi & 16 else 0}EEEvNS_8GemmArgsE"
    assert name in emu.kernel_names(text)
    gx, gy = (M + 63) // 64, N // bn
    T = gx * gy * ks

    def block_of(x, y, z):
        """The 1-D block id whose tile is (x, y, z): XCD k = b % 8 runs tile
        positions k (T // 8) + min(k, T % 8) + b // 8, column blocks fastest."""
        j = (z * gx + x) * gy + y
        for k in range(8):
            start, count = k * (T // 8) + min(k, T % 8), (T - k + 7) // 8
            if start <= j < start + count:
                return (j - start) * 8 + k
        raise AssertionError(j)

    ids = sorted({block_of(x, y, z) for x in sorted({0, gx - 1}) for y in sorted({0, gy - 1})
                  for z in sorted({0, ks - 1})})
    assert all(0 <= b < T for b in ids)
    check_kernel(text, name, kern, regions, [(b, 0, 0) for b in ids], waves=4 * kw)


@pytest.mark.parametrize("dt,B,H,W,d,hidden", [(1, 2, 7, 9, 64, 128), (2, 1, 40, 40, 384, 192),
                                                (1, 1, 16, 3, 128, 64), (2, 1, 9, 33, 64, 64)])
def test_swiglu_gated_conv_addresses(dt, B, H, W, d, hidden):
    text = swiglu_asm()
    M = B * H * W
    base = 0x1000_0000_0000
    X, WG, WV, CW, CB, HO = (base + i * 0x10_0000_0000 for i in range(6))
    regions = [emu.Region("X", X, M * d * 2, "r"), emu.Region("Wg", WG, hidden * d * 2, "r"),
               emu.Region("Wv", WV, hidden * d * 2, "r"), emu.Region("cw", CW, hidden * 9 * 4, "r"),
               emu.Region("cb", CB, hidden * 4, "r"), emu.Region("H", HO, M * hidden * 2, "w"),
               emu.Region("kernarg", emu.KERNARG_BASE, 64, "r")]
    kern = struct.pack("<QQQQQQiiiii4x", X, WG, WV, CW, CB, HO, H, W, d, hidden, B)
    name = [n for n in emu.kernel_names(text) if "gated_conv_kernel" in n and f"ILi{dt}E" in n][0]
    with open(os.path.join(CSRC, "swiglu.hip")) as fh:
        fn = int(re.search(r"constexpr int kFN = (\d+);", fh.read()).group(1))
    tx, ty = (W + 15) // 16, (H + 7) // 8  # one work-group per 8 x 16 tokens x kFN channels
    nt, nc = B * tx * ty, hidden // fn
    T = nt * nc

    def block_of(tile, cb):
        """1-D block id of (tile, channel block): XCD k = b % 8 runs positions
        k (T // 8) + min(k, T % 8) + b // 8 of the order, channel blocks fastest."""
        j = tile * nc + cb
        for k in range(8):
            start, count = k * (T // 8) + min(k, T % 8), (T - k + 7) // 8
            if start <= j < start + count:
                return (j - start) * 8 + k
        raise AssertionError(j)

    ids = sorted({block_of(t, c) for t in (0, tx - 1, nt - 1, nt // 2) for c in (0, nc - 1)})
    assert all(0 <= b < T for b in ids)
    check_kernel(text, name, kern, regions, [(b, 0, 0) for b in ids])


@pytest.mark.parametrize("cdt", [0, 1, 2])
def test_swiglu_ksplit_reduce_addresses(cdt):
    text = swiglu_asm()
    M, N, ks = 100, 64, 4
    n4 = M * N // 4
    es = {0: 4, 1: 2, 2: 2}
    base = 0x1000_0000_0000
    P, C = base, base + 0x10_0000_0000
    regions = [emu.Region("part", P, ks * M * N * 4, "r"), emu.Region("C", C, M * N * es[cdt], "w"),
               emu.Region("kernarg", emu.KERNARG_BASE, 40, "r")]
    R = base + 0x20_0000_0000
    regions.append(emu.Region("res", R, M * N * es[cdt], "r"))
    kern = struct.pack("<QQqiiQ", P, C, n4, ks, cdt, R if cdt else 0)
    name = [n for n in emu.kernel_names(text) if "ksplit_reduce_kernel" in n][0]
    nblk = (n4 + 255) // 256
    check_kernel(text, name, kern, regions, [(0, 0, 0), (nblk - 1, 0, 0)])


# ---------------------------------------------------------------------------
# the block's small kernels (block.hip)
# ---------------------------------------------------------------------------
def block_asm() -> str:
    from paper_2609_26590_amd import build as b
    h = hashlib.sha256()
    for f in ("block.hip", "gtr_device.h", "gtr_internal.h"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "gtr.h"), "rb") as fh:
        h.update(fh.read())
    h.update(" ".join(b.HIPCC_FLAGS).encode())
    os.makedirs(BUILD, exist_ok=True)
    path = os.path.join(BUILD, f"block.gfx950.{h.hexdigest()[:16]}.s")
    if not os.path.exists(path):
        tmp = path + f".tmp{os.getpid()}"
        r = subprocess.run([b._hipcc(), *b.HIPCC_FLAGS, "-S", "--cuda-device-only", os.path.join(CSRC, "block.hip"),
                            "-o", tmp], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        os.replace(tmp, path)
    with open(path) as fh:
        return fh.read()


def _kname(text, sub):
    return [n for n in emu.kernel_names(text) if sub in n][0]


@pytest.mark.parametrize("M,d,dt,affine", [(1600, 384, 1, True), (33, 192, 2, False), (5, 2048, 1, True),
                                           (4, 8, 2, True)])
def test_block_layernorm_addresses(M, d, dt, affine):
    text = block_asm()
    base = 0x1000_0000_0000
    X, Wt, Bt, Y = (base + i * 0x10_0000_0000 for i in range(4))
    regions = [emu.Region("x", X, M * d * 2, "r"), emu.Region("w", Wt, d * 4, "r"), emu.Region("b", Bt, d * 4, "r"),
               emu.Region("y", Y, M * d * 2, "w"), emu.Region("kernarg", emu.KERNARG_BASE, 64, "r")]
    kern = struct.pack("<QQQQqifi4x", X, Wt if affine else 0, Bt if affine else 0, Y, M, d, 1e-6, dt)
    nb = (M + 3) // 4
    check_kernel(text, _kname(text, "layernorm_kernel"), kern, regions, [(0, 0, 0), (nb - 1, 0, 0)])


@pytest.mark.parametrize("parts,B,H,L,dh,pad,merge", [(4, 1, 6, 1600, 64, 0, 0), (2, 3, 2, 5, 8, 8, 0),
                                                      (1, 2, 3, 37, 64, 0, 1), (1, 3, 2, 5, 8, 0, 1)])
def test_block_heads_addresses(parts, B, H, L, dh, pad, merge):
    text = block_asm()
    base = 0x1000_0000_0000
    S, D = base, base + 0x10_0000_0000
    ld = parts * H * dh + pad
    n = parts * B * H * L * dh
    src_elems = n if merge else B * L * ld
    regions = [emu.Region("src", S, src_elems * 2, "r"), emu.Region("dst", D, n * 2, "w"),
               emu.Region("kernarg", emu.KERNARG_BASE, 64, "r")]
    total = n // 8
    kern = struct.pack("<QQqiiqi4xqii", S, D, total, B, H, L, dh // 8, ld // 8, parts, merge)
    nb = (total + 255) // 256
    check_kernel(text, _kname(text, "heads_kernel"), kern, regions, sorted({(0, 0, 0), (nb - 1, 0, 0)}))


@pytest.mark.parametrize("n,dt", [(614400, 1), (8, 2), (2056, 1)])
def test_block_add_addresses(n, dt):
    text = block_asm()
    base = 0x1000_0000_0000
    A, Bv, Y = (base + i * 0x10_0000_0000 for i in range(3))
    regions = [emu.Region("a", A, n * 2, "r"), emu.Region("b", Bv, n * 2, "r"), emu.Region("y", Y, n * 2, "w"),
               emu.Region("kernarg", emu.KERNARG_BASE, 64, "r")]
    kern = struct.pack("<QQQqi4x", A, Bv, Y, n // 8, dt)
    nb = (n // 8 + 255) // 256
    check_kernel(text, _kname(text, "add_kernel"), kern, regions, sorted({(0, 0, 0), (nb - 1, 0, 0)}))
