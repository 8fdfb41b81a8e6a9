"""Wave-level emulator of gfx950 assembly, for checking the addresses of the
kernels this package compiles (test infrastructure; reads the `hipcc -S`
listing of our own sources, runs on the CPU, never touches a GPU).

One wave (64 lanes) of one work-group is executed instruction by instruction.
Every lane of every register carries two flags besides its value:
  * defined - written for this lane since the wave started (writes honour the
    exec mask, so a value produced under a partial mask is defined only for
    the lanes that were active);
  * opaque  - derived from memory contents or other data, value unknown.
Integer and address arithmetic (including the float steps of the compiler's
integer division) is emulated exactly; loaded data is opaque. A branch or an
exec-mask change that depends on opaque data forks the path: every outcome is
explored by re-running the wave with a list of decisions (loops fork a bounded
number of times per site, then leave by the less-taken direction).

Reported per instruction:
  ERR-UNDEF-ADDR  an active lane forms a memory address (global, buffer,
                  scratch, LDS, permute index) from an undefined value
  ERR-OOB         an active lane's address lies outside every registered
                  buffer (buffer-descriptor accesses: only the in-range ones)
  ERR-MODE        a store to a read-only buffer
  ERR-LDS         an LDS address beyond the work-group's allocation
  ERR-UNDEF-CTRL  a branch or exec change reads an undefined value
  WARN-DATA-ADDR  an address depends on loaded data
  WARN-UNDEF-DATA stored data (active lanes) is undefined
  INFO-BUFFER-OOR buffer accesses dropped by the descriptor's range check
  INFO-DATA-OFFSET a buffer access whose offset depends on loaded data, with
                  the descriptor's whole range inside one registered buffer
Barriers, waits and cache maintenance are no-ops; atomics return opaque data
unless the buffer they hit has a fixed load value.
"""
from __future__ import annotations

import re
import struct
import sys
from collections import defaultdict

import numpy as np

NL = 64
M32 = 0xFFFFFFFF
M64 = (1 << 64) - 1
LANES = np.arange(NL)

# ---------------------------------------------------------------------------
# parsing
# ---------------------------------------------------------------------------
REG_RE = re.compile(r'^(-)?(\|)?([vsa])(?:\[(\d+):(\d+)\]|(\d+))(\|)?$')


class Inst:
    __slots__ = ("op", "ops", "mods", "raw", "idx")

    def __init__(self, op, ops, mods, raw, idx):
        self.op, self.ops, self.mods, self.raw, self.idx = op, ops, mods, raw, idx


def parse_inst(t, idx):
    # DPP quad permutations print as quad_perm:[a,b,c,d]: keep them one modifier
    t = re.sub(r'quad_perm:\[(\d),(\d),(\d),(\d)\]', r'quad_perm:\1\2\3\4', t)
    parts = t.split(None, 1)
    op = parts[0]
    ops, mods = [], {}
    if len(parts) > 1:
        for k, piece in enumerate(parts[1].split(',')):
            toks = piece.split()
            if not toks:
                continue
            # first token of a comma piece is an operand unless it is a modifier
            first = toks[0]
            if ':' in first and not first.startswith(('s[', 'v[', 'a[')) and not re.match(r'^-?\|?[vsa]\[', first):
                rest = toks
            else:
                ops.append(first)
                rest = toks[1:]
            for m in rest:
                if ':' in m:
                    a, b = m.split(':', 1)
                    mods[a] = b
                else:
                    mods[m] = True
    return Inst(op, ops, mods, t, idx)


def parse_kernel(text, name):
    i = text.find('\n' + name + ':')
    assert i >= 0, name
    j = text.find('.Lfunc_end', i)
    prog, labels = [], {}
    for raw in text[i + 1:j].splitlines()[1:]:
        t = raw.split(';')[0].strip()
        if not t:
            continue
        if t.endswith(':'):
            labels[t[:-1]] = len(prog)
            continue
        if t.startswith('.'):
            continue
        prog.append(parse_inst(t, len(prog)))
    d = {}
    k = text.find('.amdhsa_kernel ' + name + '\n')
    e = text.find('.end_amdhsa_kernel', k)
    for l in text[k:e].splitlines():
        m = re.match(r'\s*\.(amdhsa_\w+)\s+(-?\d\S*)$', l)
        if m:
            d[m.group(1)] = int(m.group(2), 0)
    return prog, labels, d


def kernel_names(text):
    return re.findall(r'^(_Z\S+):\s', text, re.M)


# ---------------------------------------------------------------------------
# values
# ---------------------------------------------------------------------------
class VVal:
    """32-bit per-lane value."""
    __slots__ = ("v", "d", "o")

    def __init__(self, v, d, o):
        self.v, self.d, self.o = v, d, o


FLOAT_CONST = {'0.5': 0x3F000000, '-0.5': 0xBF000000, '1.0': 0x3F800000, '-1.0': 0xBF800000,
               '2.0': 0x40000000, '-2.0': 0xC0000000, '4.0': 0x40800000, '-4.0': 0xC0800000,
               '0.15915494': 0x3E22F983}


class Region:
    def __init__(self, name, base, size, mode, load_value=None):
        self.name, self.base, self.size, self.mode = name, base, size, mode
        self.load_value = load_value   # loads from here return this concrete value


class Report:
    def __init__(self):
        self.items = defaultdict(set)
        self.counts = defaultdict(int)

    def add(self, kind, inst, detail=""):
        key = (inst.idx, inst.raw)
        self.counts[kind] += 1
        if len(self.items[kind]) < 2000:
            self.items[kind].add((inst.idx, inst.raw, detail))


class Wave:
    def __init__(self, prog, labels, desc, kernarg: bytes, regions, lds_size, wg_ids, wave_in_wg,
                 decisions, report, max_steps=2_000_000, fork_limit=2):
        self.prog, self.labels, self.desc = prog, labels, desc
        self.kernarg = kernarg
        self.regions = regions
        self.lds_size = lds_size
        self.rep = report
        self.decisions = decisions
        self.dpos = 0
        self.new_decisions = []   # (position, n_options) encountered beyond the list
        self.site_count = defaultdict(int)
        self.dir_count = defaultdict(int)
        self.max_steps = max_steps
        self.fork_limit = fork_limit
        # register files
        self.V = np.zeros((1024, NL), np.uint32)   # v0..v511, a0..a511 at 512+
        self.VD = np.zeros((1024, NL), bool)
        self.VO = np.zeros((1024, NL), bool)
        self.S = [0] * 128       # value
        self.SO = [0] * 128      # opaque bit mask
        self.SD = [False] * 128  # defined
        self.exec = M64
        self.scc = (0, False, True)  # value, opaque, defined
        self.m0 = None
        self.gpr_idx = None
        self.scratch = {}
        self.scratch_size = desc.get('amdhsa_private_segment_fixed_size', 0)
        # ABI initial state
        n = 0
        if desc.get('amdhsa_user_sgpr_private_segment_buffer', 0):
            n += 4
        if desc.get('amdhsa_user_sgpr_dispatch_ptr', 0):
            n += 2
        if desc.get('amdhsa_user_sgpr_queue_ptr', 0):
            n += 2
        if desc.get('amdhsa_user_sgpr_kernarg_segment_ptr', 0):
            self.sset(n, KERNARG_BASE & M32)
            self.sset(n + 1, KERNARG_BASE >> 32)
            n += 2
        n = desc.get('amdhsa_user_sgpr_count', n)
        for axis in 'xyz':
            if desc.get('amdhsa_system_sgpr_workgroup_id_' + axis, 0):
                self.sset(n, wg_ids['xyz'.index(axis)])
                n += 1
        tid = wave_in_wg * NL + LANES
        self.V[0] = tid.astype(np.uint32)
        self.VD[0] = True
        self.pc = 0

    # ---- scalar helpers
    def sset(self, i, val, ob=0, d=True):
        self.S[i] = val & M32
        self.SO[i] = ob & M32
        self.SD[i] = d

    def decide(self, inst, n=2, forced=None):
        """Index of the option to take at an opaque decision."""
        key = inst.idx
        self.site_count[key] += 1
        if self.site_count[key] > self.fork_limit and forced is not None:
            c = min(range(n), key=lambda k: self.dir_count[(key, k)])
            self.dir_count[(key, c)] += 1
            return c
        if self.dpos < len(self.decisions):
            c = self.decisions[self.dpos]
            self.dpos += 1
            self.dir_count[(key, c)] += 1
            return c
        self.new_decisions.append((self.dpos, n))
        self.dpos += 1
        self.decisions = self.decisions + [0]
        self.dir_count[(key, 0)] += 1
        return 0

    # ---- operand access
    def sreg_index(self, tok):
        if tok in ('vcc', 'vcc_lo'):
            return 106
        if tok == 'vcc_hi':
            return 107
        if tok == 'm0':
            return 124
        m = re.match(r'^s(\d+)$', tok)
        if m:
            return int(m.group(1))
        return None

    def s64(self, tok, inst):
        """(value, opaque-bits, defined) of a 64-bit scalar operand."""
        if tok == 'exec':
            return self.exec, 0, True
        if tok == 'vcc':
            tok = 's[106:107]'
        m = re.match(r'^s\[(\d+):(\d+)\]$', tok)
        if m:
            a = int(m.group(1))
            return (self.S[a] | (self.S[a + 1] << 32), self.SO[a] | (self.SO[a + 1] << 32),
                    self.SD[a] and self.SD[a + 1])
        v = self.literal(tok)
        if v is None:
            raise NotImplementedError(f"s64 operand {tok}: {inst.raw}")
        v &= M64
        return v, 0, True

    def s64set(self, tok, val, ob=0, d=True):
        val &= M64
        ob &= M64
        if tok == 'exec':
            if ob:
                raise RuntimeError("opaque exec")
            self.exec = val
            return
        if tok == 'vcc':
            tok = 's[106:107]'
        m = re.match(r'^s\[(\d+):(\d+)\]$', tok)
        a = int(m.group(1))
        self.sset(a, val & M32, ob & M32, d)
        self.sset(a + 1, val >> 32, ob >> 32, d)

    def s32(self, tok, inst):
        if tok == 'exec_lo':
            return self.exec & M32, 0, True
        if tok == 'exec_hi':
            return self.exec >> 32, 0, True
        i = self.sreg_index(tok)
        if i is not None:
            return self.S[i], self.SO[i], self.SD[i]
        v = self.literal(tok)
        if v is None:
            raise NotImplementedError(f"s32 operand {tok}: {inst.raw}")
        return v & M32, 0, True

    def s32set(self, tok, val, ob=0, d=True):
        if tok == 'exec_lo':
            assert not ob
            self.exec = (self.exec & ~M32 & M64) | (val & M32)
            return
        if tok == 'exec_hi':
            assert not ob
            self.exec = (self.exec & M32) | ((val & M32) << 32)
            return
        i = self.sreg_index(tok)
        assert i is not None, tok
        self.sset(i, val, ob, d)

    @staticmethod
    def literal(tok):
        if tok in FLOAT_CONST:
            return FLOAT_CONST[tok]
        try:
            return int(tok, 0)
        except ValueError:
            return None

    def vidx(self, tok):
        m = REG_RE.match(tok)
        if not m:
            return None
        kind = m.group(3)
        if kind == 's':
            return None
        lo = int(m.group(4) if m.group(4) is not None else m.group(6))
        hi = int(m.group(5)) if m.group(5) is not None else lo
        base = 512 if kind == 'a' else 0
        return base + lo, base + hi

    def v32(self, tok, inst):
        """32-bit per-lane source (VGPR, SGPR broadcast or literal) with abs/neg."""
        neg = tok.startswith('-') and (tok[1:2] in ('v', 's', 'a', '|') or tok[1:] in ('vcc', 'vcc_lo', 'vcc_hi', 'm0'))
        t = tok[1:] if neg else tok
        ab = t.startswith('|') and t.endswith('|')
        if ab:
            t = t[1:-1]
        r = self.vidx(t)
        if r is not None:
            i = r[0]
            v, d, o = self.V[i].copy(), self.VD[i].copy(), self.VO[i].copy()
        else:
            sv, so, sd = self.s32(t, inst)
            v = np.full(NL, sv, np.uint32)
            d = np.full(NL, sd)
            o = np.full(NL, bool(so))
        if ab:
            v = v & np.uint32(0x7FFFFFFF)
        if neg:
            v = v ^ np.uint32(0x80000000)
        return VVal(v, d, o)

    def v64(self, tok, inst):
        """64-bit per-lane source as uint64 arrays."""
        r = self.vidx(tok)
        if r is not None:
            i = r[0]
            v = self.V[i].astype(np.uint64) | (self.V[i + 1].astype(np.uint64) << np.uint64(32))
            return v, self.VD[i] & self.VD[i + 1], self.VO[i] | self.VO[i + 1]
        m = re.match(r'^s\[(\d+):(\d+)\]$', tok)
        if m or tok in ('vcc', 'exec'):
            sv, so, sd = self.s64(tok, inst)
            return np.full(NL, sv, np.uint64), np.full(NL, sd), np.full(NL, bool(so))
        lit = self.literal(tok)
        if lit is None:
            raise NotImplementedError(f"v64 operand {tok}: {inst.raw}")
        return np.full(NL, lit & M64, np.uint64), np.ones(NL, bool), np.zeros(NL, bool)

    def v64w(self, tok, inst):
        """64-bit per-lane source with per-word flags: (value, d_lo, d_hi, o_lo, o_hi)."""
        r = self.vidx(tok)
        if r is not None:
            i = r[0]
            v = self.V[i].astype(np.uint64) | (self.V[i + 1].astype(np.uint64) << np.uint64(32))
            return v, self.VD[i], self.VD[i + 1], self.VO[i], self.VO[i + 1]
        v, d, o = self.v64(tok, inst)
        return v, d, d, o, o

    def vwrite64w(self, tok, v, d_lo, d_hi, o_lo, o_hi, lanes=None):
        r = self.vidx(tok)
        m = self.active() if lanes is None else lanes
        i = r[0]
        v = np.asarray(v, np.uint64)
        self.V[i][m] = (v & np.uint64(M32)).astype(np.uint32)[m]
        self.V[i + 1][m] = (v >> np.uint64(32)).astype(np.uint32)[m]
        self.VD[i][m], self.VO[i][m] = d_lo[m], o_lo[m]
        self.VD[i + 1][m], self.VO[i + 1][m] = d_hi[m], o_hi[m]

    def active(self):
        return ((np.uint64(self.exec) >> LANES.astype(np.uint64)) & np.uint64(1)).astype(bool)

    def vwrite(self, tok, val: VVal, lanes=None):
        r = self.vidx(tok)
        assert r is not None, tok
        m = self.active() if lanes is None else lanes
        i = r[0]
        self.V[i][m] = val.v[m]
        self.VD[i][m] = val.d[m]
        self.VO[i][m] = val.o[m]

    def vwrite64(self, tok, v, d, o, lanes=None):
        r = self.vidx(tok)
        m = self.active() if lanes is None else lanes
        i = r[0]
        v = np.asarray(v, np.uint64)
        self.V[i][m] = (v & np.uint64(M32)).astype(np.uint32)[m]
        self.V[i + 1][m] = (v >> np.uint64(32)).astype(np.uint32)[m]
        for j in (i, i + 1):
            self.VD[j][m] = d[m]
            self.VO[j][m] = o[m]

    def vwrite_multi(self, tok, d, o, lanes):
        r = self.vidx(tok)
        for j in range(r[0], r[1] + 1):
            self.VD[j][lanes] = d[lanes]
            self.VO[j][lanes] = o[lanes]
            self.V[j][lanes] = 0

    # ---- masks written by compares
    def write_mask(self, tok, bits, obits, dbits):
        """bits/obits: uint64 python ints for active lanes; inactive lanes read 0."""
        self.s64set(tok, bits, obits, dbits)

    # ---- memory checks
    def check_window(self, inst, base, size, mode):
        """A buffer descriptor's whole range [base, base + size): inside one
        registered buffer that allows `mode` (INFO-DATA-OFFSET), else ERR-OOB."""
        for rg in self.regions:
            if rg.base <= base and base + size <= rg.base + rg.size:
                if mode == 'w' and 'w' not in rg.mode:
                    self.rep.add('ERR-MODE', inst, rg.name)
                else:
                    self.rep.add('INFO-DATA-OFFSET', inst, rg.name)
                return
        self.rep.add('ERR-OOB', inst, f"descriptor window {base:#x}+{size:#x} {near(self.regions, base)}")

    def check_addr(self, inst, addr, d, o, size, mode, lanes):
        """addr uint64[64]; returns nothing; reports."""
        act = lanes
        if not act.any():
            return
        if (~d & act).any():
            self.rep.add('ERR-UNDEF-ADDR', inst, f"lanes {np.nonzero(~d & act)[0][:8].tolist()}")
            return
        if (o & act).any():
            self.rep.add('WARN-DATA-ADDR', inst)
            return
        a = addr[act].astype(object)
        found = set()
        for x in set(a.tolist()):
            ok = False
            for rg in self.regions:
                if rg.base <= x and x + size <= rg.base + rg.size:
                    if mode not in rg.mode:
                        self.rep.add('ERR-MODE', inst, f"{rg.name} {mode}")
                    ok = True
                    found.add(rg)
                    break
            if not ok:
                self.rep.add('ERR-OOB', inst, f"addr 0x{x:x} size {size} ({near(self.regions, x)})")
                return None
        return found.pop() if len(found) == 1 else None

    def check_data(self, inst, tok, lanes, nregs=1):
        r = self.vidx(tok)
        if r is None:
            return
        for j in range(r[0], r[0] + nregs):
            if (~self.VD[j] & lanes).any():
                self.rep.add('WARN-UNDEF-DATA', inst, tok)
                return

    # ---- run
    def run(self):
        prog = self.prog
        steps = 0
        while True:
            if self.pc >= len(prog):
                raise RuntimeError("fell off the end")
            inst = prog[self.pc]
            self.pc += 1
            steps += 1
            if steps > self.max_steps:
                self.rep.add('INFO-STEPLIMIT', inst)
                return
            try:
                if self.step(inst):
                    return
            except NotImplementedError as e:
                self.rep.add('NOTIMPL', inst, str(e))
                raise
            except Exception as e:  # noqa
                raise RuntimeError(f"at {inst.idx}: {inst.raw}: {e!r}") from e

    def branch(self, label):
        self.pc = self.labels[label]

    def step(self, inst):
        op = inst.op
        if self.gpr_idx is not None and op.startswith('v_') and op not in ('v_readfirstlane_b32',):
            off, modes = self.gpr_idx
            ops = list(inst.ops)
            for pos, mode in enumerate(('DST', 'SRC0', 'SRC1', 'SRC2')):
                if mode in modes and pos < len(ops):
                    m = REG_RE.match(ops[pos])
                    if m and m.group(3) == 'v':
                        lo = int(m.group(4) if m.group(4) is not None else m.group(6)) + off
                        if m.group(4) is not None:
                            hi = int(m.group(5)) + off
                            ops[pos] = f"v[{lo}:{hi}]"
                        else:
                            ops[pos] = f"v{lo}"
            inst = Inst(op, ops, inst.mods, inst.raw + f"  [gpr_idx {off}]", inst.idx)
        h = HANDLERS.get(op)
        if h is None:
            for prefix, fn in PREFIX_HANDLERS:
                if op.startswith(prefix):
                    h = fn
                    break
        if h is None:
            raise NotImplementedError(op)
        return h(self, inst)


def near(regions, x):
    best = None
    for rg in regions:
        dist = min(abs(x - rg.base), abs(x - (rg.base + rg.size)))
        if best is None or dist < best[0]:
            best = (dist, rg.name, x - rg.base)
    return f"nearest {best[1]} offset {best[2]}"


KERNARG_BASE = 0x7E00_0000_0000

HANDLERS = {}
PREFIX_HANDLERS = []


def handler(*names):
    def deco(fn):
        for n in names:
            HANDLERS[n] = fn
        return fn
    return deco


# ---------------------------------------------------------------------------
# control
# ---------------------------------------------------------------------------
@handler('s_endpgm')
def _endpgm(w, i):
    return True


@handler('s_nop', 's_waitcnt', 's_barrier', 's_sleep', 's_setprio', 's_waitcnt_vscnt', 's_sethalt', 'buffer_wbl2', 'buffer_inv', 'buffer_gl0_inv', 'buffer_gl1_inv')
def _nop(w, i):
    return False


@handler('s_bitset1_b32', 's_bitset0_b32')
def _bitset(w, i):
    # sdst[ssrc & 31] = 1 (bitset1) or 0 (bitset0); the other bits keep their value
    r = w.sreg_index(i.ops[0])
    bit, bo, bd = w.s32(i.ops[1], i)
    old, oo, od = w.s32(i.ops[0], i)
    m = 1 << (bit & 31)
    val = (old | m) if i.op == 's_bitset1_b32' else (old & ~m & M32)
    w.sset(r, val, (oo | (M32 if bo else 0)) & M32, od and bd)


HWREG_VALUE = 0  # what s_getreg_b32 reads: the emulated wave runs on XCC 0


@handler('s_getreg_b32')
def _getreg(w, i):
    r = w.sreg_index(i.ops[0])
    w.sset(r, HWREG_VALUE, 0, True)


@handler('s_branch')
def _br(w, i):
    w.branch(i.ops[0])


def cond_branch(w, i, concrete, opaque, defined):
    """Take the branch if `concrete`; opaque conditions fork (1 = taken)."""
    if not defined:
        w.rep.add('ERR-UNDEF-CTRL', i, 'branch condition')
    if opaque:
        tgt = w.labels[i.ops[0]]
        taken = bool(w.decide(i, 2, 1 if tgt > i.idx else 0))
    else:
        taken = concrete
    if taken:
        w.branch(i.ops[0])


@handler('s_cbranch_scc0')
def _bscc0(w, i):
    v, o, d = w.scc
    cond_branch(w, i, v == 0, o, d)


@handler('s_cbranch_scc1')
def _bscc1(w, i):
    v, o, d = w.scc
    cond_branch(w, i, v != 0, o, d)


@handler('s_cbranch_vccz')
def _bvccz(w, i):
    v, o, d = w.s64('vcc', i)
    known1 = v & ~o
    cond_branch(w, i, v == 0, bool(o) and not known1, d)


@handler('s_cbranch_vccnz')
def _bvccnz(w, i):
    v, o, d = w.s64('vcc', i)
    known1 = v & ~o
    cond_branch(w, i, v != 0, bool(o) and not known1, d)


@handler('s_cbranch_execz')
def _bexz(w, i):
    if w.exec == 0:
        w.branch(i.ops[0])


@handler('s_cbranch_execnz')
def _bexnz(w, i):
    if w.exec != 0:
        w.branch(i.ops[0])


# ---------------------------------------------------------------------------
# scalar ALU
# ---------------------------------------------------------------------------
def sx(v):
    v &= M32
    return v - (1 << 32) if v & 0x80000000 else v


def sx64(v):
    v &= M64
    return v - (1 << 64) if v >> 63 else v


def set_scc(w, val, opaque=False, d=True):
    w.scc = (1 if val else 0, bool(opaque), d)


def _sbfe(a, b, signed):
    """Scalar bit-field extract: offset b[4:0], width b[22:16] (sign-extended if signed)."""
    off, wid = b & 31, (b >> 16) & 127
    if wid == 0:
        return 0
    x = (a >> off) & ((1 << min(wid, 32)) - 1)
    if signed and wid < 32 and (x >> (wid - 1)) & 1:
        x -= 1 << wid
    return x & M32


def salu32(fn, scc_mode=None):
    def h(w, i):
        a = [w.s32(t, i) for t in i.ops[1:]]
        vals = [x[0] for x in a]
        ob = any(x[1] for x in a)
        d = all(x[2] for x in a)
        if scc_mode == 'carry_in':
            vals.append(w.scc[0])
            ob = ob or w.scc[1]
            d = d and w.scc[2]
        res, scc = fn(*vals)
        w.s32set(i.ops[0], res & M32, M32 if ob else 0, d)
        if scc is not None:
            set_scc(w, scc, ob, d)
    return h


def salu64(fn):
    def h(w, i):
        a = [w.s64(t, i) for t in i.ops[1:]]
        vals = [x[0] for x in a]
        ob = any(x[1] for x in a)
        d = all(x[2] for x in a)
        res, scc = fn(*vals)
        w.s64set(i.ops[0], res & M64, M64 if ob else 0, d)
        if scc is not None:
            set_scc(w, scc, ob, d)
    return h


def salu64_shift(fn):
    """64-bit shifts: the shift amount is a 32-bit operand."""
    def h(w, i):
        a = w.s64(i.ops[1], i)
        b = w.s32(i.ops[2], i)
        ob = bool(a[1]) or bool(b[1])
        d = bool(a[2]) and bool(b[2])
        res, scc = fn(a[0], b[0])
        w.s64set(i.ops[0], res & M64, M64 if ob else 0, d)
        set_scc(w, scc, ob, d)
    return h


HANDLERS.update({
    's_add_u32': salu32(lambda a, b: (a + b, (a + b) >> 32)),
    's_addc_u32': salu32(lambda a, b, c: (a + b + c, (a + b + c) >> 32), 'carry_in'),
    's_sub_u32': salu32(lambda a, b: (a - b, 1 if b > a else 0)),
    's_subb_u32': salu32(lambda a, b, c: (a - b - c, 1 if b + c > a else 0), 'carry_in'),
    's_add_i32': salu32(lambda a, b: (sx(a) + sx(b), not (-2**31 <= sx(a) + sx(b) < 2**31))),
    's_sub_i32': salu32(lambda a, b: (sx(a) - sx(b), not (-2**31 <= sx(a) - sx(b) < 2**31))),
    's_mul_i32': salu32(lambda a, b: (sx(a) * sx(b), None)),
    's_mul_hi_u32': salu32(lambda a, b: ((a * b) >> 32, None)),
    's_mul_hi_i32': salu32(lambda a, b: ((sx(a) * sx(b)) >> 32, None)),
    's_lshl_b32': salu32(lambda a, b: ((a << (b & 31)) & M32, ((a << (b & 31)) & M32) != 0)),
    's_lshr_b32': salu32(lambda a, b: (a >> (b & 31), (a >> (b & 31)) != 0)),
    's_ashr_i32': salu32(lambda a, b: (sx(a) >> (b & 31), (sx(a) >> (b & 31)) != 0)),
    's_and_b32': salu32(lambda a, b: (a & b, (a & b) != 0)),
    's_or_b32': salu32(lambda a, b: (a | b, (a | b) != 0)),
    's_xor_b32': salu32(lambda a, b: (a ^ b, (a ^ b) != 0)),
    's_min_i32': salu32(lambda a, b: (min(sx(a), sx(b)), sx(a) < sx(b))),
    's_max_i32': salu32(lambda a, b: (max(sx(a), sx(b)), sx(a) > sx(b))),
    's_min_u32': salu32(lambda a, b: (min(a, b), a < b)),
    's_max_u32': salu32(lambda a, b: (max(a, b), a > b)),
    's_abs_i32': salu32(lambda a: (abs(sx(a)), abs(sx(a)) != 0)),
    's_not_b32': salu32(lambda a: (~a & M32, (~a & M32) != 0)),
    's_andn2_b32': salu32(lambda a, b: (a & ~b & M32, (a & ~b & M32) != 0)),
    's_orn2_b32': salu32(lambda a, b: ((a | ~b) & M32, ((a | ~b) & M32) != 0)),
    's_bfe_u32': salu32(lambda a, b: (_sbfe(a, b, False), _sbfe(a, b, False) != 0)),
    's_bfe_i32': salu32(lambda a, b: (_sbfe(a, b, True), _sbfe(a, b, True) != 0)),
    's_lshl_b64': salu64_shift(lambda a, b: ((a << (b & 63)) & M64, ((a << (b & 63)) & M64) != 0)),
    's_lshr_b64': salu64_shift(lambda a, b: (a >> (b & 63), (a >> (b & 63)) != 0)),
})


@handler('s_mov_b32', 's_movk_i32')
def _smov(w, i):
    v, o, d = w.s32(i.ops[1], i)
    if i.op == 's_movk_i32':
        v &= 0xFFFF
        v = (v - 0x10000 if v & 0x8000 else v) & M32
    w.s32set(i.ops[0], v, o, d)


@handler('s_mulk_i32')
def _smulk(w, i):
    v, o, d = w.s32(i.ops[0], i)
    k = w.literal(i.ops[1])
    k = k - 0x10000 if k >= 0x8000 else k
    w.s32set(i.ops[0], (sx(v) * k) & M32, o, d)


@handler('s_addk_i32')
def _saddk(w, i):
    v, o, d = w.s32(i.ops[0], i)
    k = w.literal(i.ops[1])
    k = k - 0x10000 if k >= 0x8000 else k
    r = sx(v) + k
    w.s32set(i.ops[0], r & M32, o, d)
    set_scc(w, not (-2**31 <= r < 2**31), o, d)


@handler('s_cselect_b32')
def _scsel32(w, i):
    sv, so, sd = w.scc
    a, b = w.s32(i.ops[1], i), w.s32(i.ops[2], i)
    if so:
        w.s32set(i.ops[0], 0, M32, sd and a[2] and b[2])
        return
    r = a if sv else b
    w.s32set(i.ops[0], r[0], r[1], r[2] and sd)


@handler('s_cselect_b64')
def _scsel64(w, i):
    sv, so, sd = w.scc
    a, b = w.s64(i.ops[1], i), w.s64(i.ops[2], i)
    if so:
        # per-bit opaque where the two choices differ
        diff = (a[0] ^ b[0]) | a[1] | b[1]
        w.s64set(i.ops[0], a[0] & b[0], diff, sd and a[2] and b[2])
        return
    r = a if sv else b
    w.s64set(i.ops[0], r[0], r[1], r[2] and sd)


@handler('s_bcnt1_i32_b64')
def _sbcnt(w, i):
    v, o, d = w.s64(i.ops[1], i)
    r = bin(v).count('1')
    w.s32set(i.ops[0], r, M32 if o else 0, d)
    set_scc(w, r != 0, o, d)


@handler('s_bitcmp1_b32', 's_bitcmp0_b32')
def _sbitcmp(w, i):
    v, o, d = w.s32(i.ops[0], i)
    b, bo, bd = w.s32(i.ops[1], i)
    bit = (v >> (b & 31)) & 1
    set_scc(w, bit == (1 if i.op == 's_bitcmp1_b32' else 0), bool(o) or bool(bo), bool(d) and bool(bd))


@handler('s_ff1_i32_b64', 's_ff1_i32_b32')
def _sff1(w, i):
    if i.op.endswith('b64'):
        v, o, d = w.s64(i.ops[1], i)
    else:
        v, o, d = w.s32(i.ops[1], i)
    r = (v & -v).bit_length() - 1 if v else M32  # index of the lowest set bit, -1 if none
    w.s32set(i.ops[0], r & M32, M32 if o else 0, d)


@handler('s_mov_b64')
def _smov64(w, i):
    v, o, d = w.s64(i.ops[1], i)
    if i.ops[0] == 'exec':
        set_exec(w, i, v, o, d)
        return
    w.s64set(i.ops[0], v, o, d)


def bit_and(a, ao, b, bo):
    known0 = (~a & ~ao) | (~b & ~bo)
    v = a & b
    o = (ao | bo) & ~known0
    return v & M64, o & M64


def bit_or(a, ao, b, bo):
    known1 = (a & ~ao) | (b & ~bo)
    v = a | b
    o = (ao | bo) & ~known1
    return v & M64, o & M64


def bit_not(a, ao):
    return (~a) & M64, ao


def set_exec(w, i, v, o, d):
    if not d:
        w.rep.add('ERR-UNDEF-CTRL', i, 'exec from undefined')
    if o:
        c = w.decide(i, 2, 1)
        v = (v & ~o) | (o if c else 0)
    w.exec = v & M64


def logic64(kind):
    def h(w, i):
        dst = i.ops[0]
        a = w.s64(i.ops[1], i)
        b = w.s64(i.ops[2], i)
        if kind == 'and':
            v, o = bit_and(a[0], a[1], b[0], b[1])
        elif kind == 'or':
            v, o = bit_or(a[0], a[1], b[0], b[1])
        elif kind == 'xor':
            v, o = (a[0] ^ b[0]) & M64, a[1] | b[1]
        elif kind == 'andn2':
            nb = bit_not(b[0], b[1])
            v, o = bit_and(a[0], a[1], nb[0], nb[1])
        elif kind == 'orn2':
            nb = bit_not(b[0], b[1])
            v, o = bit_or(a[0], a[1], nb[0], nb[1])
        elif kind == 'nor':
            v, o = bit_or(a[0], a[1], b[0], b[1])
            v, o = bit_not(v, o)
        elif kind == 'nand':
            v, o = bit_and(a[0], a[1], b[0], b[1])
            v, o = bit_not(v, o)
        elif kind == 'xnor':
            v, o = (~(a[0] ^ b[0])) & M64, a[1] | b[1]
        d = a[2] and b[2]
        if dst == 'exec':
            set_exec(w, i, v, o, d)
            set_scc(w, w.exec != 0)
            return
        w.s64set(dst, v, o, d)
        known1 = v & ~o
        if known1:
            set_scc(w, 1, False, d)
        else:
            set_scc(w, 0, bool(o), d)
    return h


@handler('s_not_b64')
def _s_not_b64(w, i):
    a = w.s64(i.ops[1], i)
    v, o = bit_not(a[0], a[1])
    w.s64set(i.ops[0], v, o, a[2])
    known1 = v & ~o
    set_scc(w, 1 if known1 else 0, bool(o) and not known1, a[2])


HANDLERS.update({'s_and_b64': logic64('and'), 's_or_b64': logic64('or'), 's_xor_b64': logic64('xor'),
                 's_andn2_b64': logic64('andn2'), 's_orn2_b64': logic64('orn2'), 's_nor_b64': logic64('nor'),
                 's_nand_b64': logic64('nand'), 's_xnor_b64': logic64('xnor')})


def saveexec(kind):
    def h(w, i):
        dst = i.ops[0]
        s = w.s64(i.ops[1], i)
        old = w.exec
        w.s64set(dst, old, 0, True)
        if kind == 'and':
            v, o = bit_and(s[0], s[1], old, 0)
        elif kind == 'or':
            v, o = bit_or(s[0], s[1], old, 0)
        elif kind == 'andn2':
            v, o = bit_and(s[0], s[1], (~old) & M64, 0)
        elif kind == 'xor':
            v, o = (s[0] ^ old) & M64, s[1]
        set_exec(w, i, v, o, s[2])
        set_scc(w, w.exec != 0)
    return h


HANDLERS.update({'s_and_saveexec_b64': saveexec('and'), 's_or_saveexec_b64': saveexec('or'),
                 's_andn2_saveexec_b64': saveexec('andn2'), 's_xor_saveexec_b64': saveexec('xor')})


def scmp(fn, wide=False):
    def h(w, i):
        if wide:
            a, b = w.s64(i.ops[0], i), w.s64(i.ops[1], i)
        else:
            a, b = w.s32(i.ops[0], i), w.s32(i.ops[1], i)
        o = bool(a[1] or b[1])
        set_scc(w, fn(a[0], b[0]) if not o else 0, o, a[2] and b[2])
    return h


HANDLERS.update({
    's_cmp_eq_u32': scmp(lambda a, b: a == b), 's_cmp_lg_u32': scmp(lambda a, b: a != b),
    's_cmp_gt_u32': scmp(lambda a, b: a > b), 's_cmp_ge_u32': scmp(lambda a, b: a >= b),
    's_cmp_lt_u32': scmp(lambda a, b: a < b), 's_cmp_le_u32': scmp(lambda a, b: a <= b),
    's_cmp_eq_i32': scmp(lambda a, b: a == b), 's_cmp_lg_i32': scmp(lambda a, b: a != b),
    's_cmp_gt_i32': scmp(lambda a, b: sx(a) > sx(b)), 's_cmp_ge_i32': scmp(lambda a, b: sx(a) >= sx(b)),
    's_cmp_lt_i32': scmp(lambda a, b: sx(a) < sx(b)), 's_cmp_le_i32': scmp(lambda a, b: sx(a) <= sx(b)),
    's_cmp_eq_u64': scmp(lambda a, b: a == b, True), 's_cmp_lg_u64': scmp(lambda a, b: a != b, True),
})


def scmpk(fn, signed):
    """s_cmpk_*: SGPR against a 16-bit immediate (sign-extended for the _i32 forms)."""
    def h(w, i):
        a = w.s32(i.ops[0], i)
        k = int(i.ops[1], 0) & 0xFFFF
        if signed and k & 0x8000:
            k -= 0x10000
        set_scc(w, fn(sx(a[0]) if signed else a[0], k) if not a[1] else 0, bool(a[1]), a[2])
    return h


for _n, _f in [('eq', lambda a, b: a == b), ('lg', lambda a, b: a != b), ('gt', lambda a, b: a > b),
               ('ge', lambda a, b: a >= b), ('lt', lambda a, b: a < b), ('le', lambda a, b: a <= b)]:
    HANDLERS[f's_cmpk_{_n}_i32'] = scmpk(_f, True)
    HANDLERS[f's_cmpk_{_n}_u32'] = scmpk(_f, False)


@handler('s_set_gpr_idx_on')
def _gidx_on(w, i):
    v, o, d = w.s32(i.ops[0], i)
    if o or not d:
        w.rep.add('ERR-UNDEF-CTRL', i, 'gpr index')
    modes = re.findall(r'(DST|SRC0|SRC1|SRC2)', i.raw)
    w.gpr_idx = (v & 0xFF, set(modes))


@handler('s_set_gpr_idx_off')
def _gidx_off(w, i):
    w.gpr_idx = None


def scratch_op(nregs, store):
    def h(w, i):
        lanes = w.active()
        if store:
            vaddr, data, saddr = i.ops[0], i.ops[1], i.ops[2]
        else:
            data, vaddr, saddr = i.ops[0], i.ops[1], i.ops[2]
        assert vaddr == 'off' and saddr == 'off', i.raw
        off = int(i.mods.get('offset', 0))
        if off < 0 or off + 4 * nregs > w.scratch_size:
            w.rep.add('ERR-OOB', i, f"scratch offset {off}")
        r = w.vidx(data)
        for k in range(nregs):
            key = off + 4 * k
            if store:
                old = w.scratch.get(key)
                v = np.where(lanes, w.V[r[0] + k], old[0] if old else 0).astype(np.uint32)
                d = np.where(lanes, w.VD[r[0] + k], old[1] if old else False)
                o = np.where(lanes, w.VO[r[0] + k], old[2] if old else False)
                w.scratch[key] = (v, d, o)
            else:
                old = w.scratch.get(key, (np.zeros(NL, np.uint32), np.zeros(NL, bool), np.zeros(NL, bool)))
                w.vwrite(f"v{r[0] + k}", VVal(old[0].copy(), old[1].copy(), old[2].copy()), lanes)
    return h


HANDLERS.update({'scratch_load_dword': scratch_op(1, False), 'scratch_load_dwordx2': scratch_op(2, False),
                 'scratch_load_dwordx4': scratch_op(4, False), 'scratch_store_dword': scratch_op(1, True),
                 'scratch_store_dwordx2': scratch_op(2, True), 'scratch_store_dwordx4': scratch_op(4, True)})


# ---------------------------------------------------------------------------
# scalar memory
# ---------------------------------------------------------------------------
def sload(n):
    def h(w, i):
        dst = i.ops[0]
        base, bo, bd = w.s64(i.ops[1], i)
        off = w.literal(i.ops[2]) if w.literal(i.ops[2]) is not None else w.s32(i.ops[2], i)[0]
        if not bd or bo:
            w.rep.add('ERR-UNDEF-ADDR' if not bd else 'WARN-DATA-ADDR', i, 'scalar load base')
            vals = [0] * n
            ok = False
        else:
            a = base + off - KERNARG_BASE
            if 0 <= a and a + 4 * n <= len(w.kernarg):
                vals = list(struct.unpack_from('<%dI' % n, w.kernarg, a))
                ok = True
            else:
                w.rep.add('ERR-OOB', i, f"scalar load offset {a:#x}")
                vals = [0] * n
                ok = False
        m = re.match(r'^s\[(\d+):(\d+)\]$', dst)
        first = int(m.group(1)) if m else w.sreg_index(dst)
        for k in range(n):
            w.sset(first + k, vals[k], 0, ok)
    return h


HANDLERS.update({'s_load_dword': sload(1), 's_load_dwordx2': sload(2), 's_load_dwordx4': sload(4),
                 's_load_dwordx8': sload(8), 's_load_dwordx16': sload(16)})


# ---------------------------------------------------------------------------
# vector ALU
# ---------------------------------------------------------------------------
def vres(v, *srcs, d=None):
    dd = np.ones(NL, bool) if d is None else d
    oo = np.zeros(NL, bool)
    for s in srcs:
        dd = dd & s.d
        oo = oo | s.o
    v = np.asarray(v)
    if v.dtype != np.uint32:
        if v.dtype.kind == 'i':
            v = v.astype(np.int64).astype(np.uint64)
        v = v.astype(np.uint64).astype(np.uint32)
    return VVal(v, dd, oo)


def valu(fn, nsrc):
    def h(w, i):
        srcs = [w.v32(t, i) for t in i.ops[1:1 + nsrc]]
        with np.errstate(all='ignore'):
            v = fn(*[s.v for s in srcs])
        w.vwrite(i.ops[0], vres(v, *srcs))
    return h


def _bfe_i32(a, b, c):
    """Signed bit-field extract: width c & 31 bits of a from offset b & 31, sign-extended."""
    off = (b & np.uint32(31)).astype(np.int64)
    wid = (c & np.uint32(31)).astype(np.int64)
    x = (a.astype(np.int64) >> off) & ((np.int64(1) << wid) - 1)
    sign = np.where(wid > 0, (x >> np.maximum(wid - 1, 0)) & 1, 0)
    x = np.where(sign == 1, x - (np.int64(1) << wid), x)
    return (x & M32).astype(np.uint32)


def u64(x):
    return x.astype(np.uint64)


def i64(x):
    return x.view(np.int32).astype(np.int64)


def fl(x):
    return x.view(np.float32)


def fo(x):
    return np.asarray(x, np.float32).view(np.uint32)


def fop(fn, nsrc):
    def h(w, i):
        srcs = [w.v32(t, i) for t in i.ops[1:1 + nsrc]]
        with np.errstate(all='ignore'):
            v = fo(fn(*[fl(s.v) for s in srcs]))
        w.vwrite(i.ops[0], vres(v, *srcs))
    return h


HANDLERS.update({
    'v_mov_b32_e32': valu(lambda a: a, 1),
    'v_mov_b32_e64': valu(lambda a: a, 1),
    'v_not_b32_e32': valu(lambda a: ~a, 1),
    'v_and_b32_e32': valu(lambda a, b: a & b, 2), 'v_and_b32_e64': valu(lambda a, b: a & b, 2),
    'v_or_b32_e32': valu(lambda a, b: a | b, 2), 'v_or_b32_e64': valu(lambda a, b: a | b, 2),
    'v_xor_b32_e32': valu(lambda a, b: a ^ b, 2), 'v_xor_b32_e64': valu(lambda a, b: a ^ b, 2),
    'v_or3_b32': valu(lambda a, b, c: a | b | c, 3),
    'v_add_u32_e32': valu(lambda a, b: a + b, 2), 'v_add_u32_e64': valu(lambda a, b: a + b, 2),
    'v_sub_u32_e32': valu(lambda a, b: a - b, 2), 'v_sub_u32_e64': valu(lambda a, b: a - b, 2),
    'v_subrev_u32_e32': valu(lambda a, b: b - a, 2), 'v_subrev_u32_e64': valu(lambda a, b: b - a, 2),
    'v_add3_u32': valu(lambda a, b, c: a + b + c, 3),
    'v_add_u16_e32': valu(lambda a, b: (a + b) & np.uint32(0xFFFF), 2),
    'v_add_u16_e64': valu(lambda a, b: (a + b) & np.uint32(0xFFFF), 2),
    'v_lshlrev_b32_e32': valu(lambda a, b: b << (a & np.uint32(31)), 2),
    'v_lshlrev_b32_e64': valu(lambda a, b: b << (a & np.uint32(31)), 2),
    'v_lshrrev_b32_e32': valu(lambda a, b: b >> (a & np.uint32(31)), 2),
    'v_lshrrev_b32_e64': valu(lambda a, b: b >> (a & np.uint32(31)), 2),
    'v_ashrrev_i32_e32': valu(lambda a, b: (b.view(np.int32) >> (a & np.uint32(31)).astype(np.int32)).view(np.uint32), 2),
    'v_ashrrev_i32_e64': valu(lambda a, b: (b.view(np.int32) >> (a & np.uint32(31)).astype(np.int32)).view(np.uint32), 2),
    'v_lshl_add_u32': valu(lambda a, b, c: (a << (b & np.uint32(31))) + c, 3),
    'v_lshl_or_b32': valu(lambda a, b, c: (a << (b & np.uint32(31))) | c, 3),
    'v_add_lshl_u32': valu(lambda a, b, c: (a + b) << (c & np.uint32(31)), 3),
    'v_and_or_b32': valu(lambda a, b, c: (a & b) | c, 3),
    'v_bfe_i32': valu(lambda a, b, c: _bfe_i32(a, b, c), 3),
    'v_bfe_u32': valu(lambda a, b, c: (a >> (b & np.uint32(31))) & ((np.uint64(1) << u64(c & np.uint32(31))) - np.uint64(1)).astype(np.uint32), 3),
    'v_mul_lo_u32': valu(lambda a, b: (u64(a) * u64(b)) & np.uint64(M32), 2),
    'v_mul_hi_u32': valu(lambda a, b: (u64(a) * u64(b)) >> np.uint64(32), 2),
    'v_mul_u32_u24_e32': valu(lambda a, b: u64(a & np.uint32(0xFFFFFF)) * u64(b & np.uint32(0xFFFFFF)) & np.uint64(M32), 2),
    'v_mul_u32_u24_e64': valu(lambda a, b: u64(a & np.uint32(0xFFFFFF)) * u64(b & np.uint32(0xFFFFFF)) & np.uint64(M32), 2),
    'v_mul_i32_i24_e32': valu(lambda a, b: (s24(a) * s24(b)).astype(np.uint64) & np.uint64(M32), 2),
    'v_mad_u32_u24': valu(lambda a, b, c: (u64(a & np.uint32(0xFFFFFF)) * u64(b & np.uint32(0xFFFFFF)) + u64(c)) & np.uint64(M32), 3),
    'v_mad_i32_i24': valu(lambda a, b, c: ((s24(a) * s24(b) + c.view(np.int32).astype(np.int64)).astype(np.uint64)) & np.uint64(M32), 3),
    'v_alignbit_b32': valu(lambda a, b, c: ((u64(a) << np.uint64(32) | u64(b)) >> u64(c & np.uint32(31))) & np.uint64(M32), 3),
    'v_min_u32_e32': valu(lambda a, b: np.minimum(a, b), 2),
    'v_max_u32_e32': valu(lambda a, b: np.maximum(a, b), 2),
    'v_min_i32_e32': valu(lambda a, b: np.minimum(a.view(np.int32), b.view(np.int32)).view(np.uint32), 2),
    'v_max_i32_e32': valu(lambda a, b: np.maximum(a.view(np.int32), b.view(np.int32)).view(np.uint32), 2),
    'v_xad_u32': valu(lambda a, b, c: (u64(a ^ b) + u64(c)) & np.uint64(M32), 3),
    'v_med3_u32': valu(lambda a, b, c: np.maximum(np.minimum(a, b), np.minimum(np.maximum(a, b), c)), 3),
    'v_med3_i32': valu(lambda a, b, c: np.maximum(np.minimum(a.view(np.int32), b.view(np.int32)),
                                                  np.minimum(np.maximum(a.view(np.int32), b.view(np.int32)),
                                                             c.view(np.int32))).view(np.uint32), 3),
    # float
    'v_add_f32_e32': fop(lambda a, b: a + b, 2), 'v_add_f32_e64': fop(lambda a, b: a + b, 2),
    'v_sub_f32_e32': fop(lambda a, b: a - b, 2), 'v_sub_f32_e64': fop(lambda a, b: a - b, 2),
    'v_subrev_f32_e32': fop(lambda a, b: b - a, 2),
    'v_mul_f32_e32': fop(lambda a, b: a * b, 2), 'v_mul_f32_e64': fop(lambda a, b: a * b, 2),
    'v_max_f32_e32': fop(np.maximum, 2), 'v_max_f32_e64': fop(np.maximum, 2),
    'v_min_f32_e32': fop(np.minimum, 2), 'v_min_f32_e64': fop(np.minimum, 2),
    'v_max3_f32': fop(lambda a, b, c: np.maximum(np.maximum(a, b), c), 3),
    'v_fma_f32': fop(lambda a, b, c: (a.astype(np.float64) * b + c).astype(np.float32), 3),
    'v_exp_f32_e32': fop(lambda a: np.exp2(a), 1),
    'v_rcp_f32_e32': fop(lambda a: np.float32(1) / a, 1),
    'v_rcp_iflag_f32_e32': fop(lambda a: np.float32(1) / a, 1),
    'v_trunc_f32_e32': fop(np.trunc, 1),
    'v_rndne_f32_e32': fop(np.rint, 1),
    'v_sqrt_f32_e32': fop(np.sqrt, 1),
    'v_log_f32_e32': fop(np.log2, 1),
})


def s24(x):
    y = (x & np.uint32(0xFFFFFF)).astype(np.int64)
    return np.where(y & 0x800000, y - 0x1000000, y)


@handler('v_fmac_f32_e32', 'v_fmac_f32_e64')
def _fmac(w, i):
    a, b, c = w.v32(i.ops[1], i), w.v32(i.ops[2], i), w.v32(i.ops[0], i)
    with np.errstate(all='ignore'):
        v = fo((fl(a.v).astype(np.float64) * fl(b.v) + fl(c.v)).astype(np.float32))
    w.vwrite(i.ops[0], vres(v, a, b, c))


@handler('v_fmamk_f32')
def _fmamk(w, i):  # d = a * K + b
    a, k, b = w.v32(i.ops[1], i), w.v32(i.ops[2], i), w.v32(i.ops[3], i)
    with np.errstate(all='ignore'):
        v = fo((fl(a.v).astype(np.float64) * fl(k.v) + fl(b.v)).astype(np.float32))
    w.vwrite(i.ops[0], vres(v, a, k, b))


@handler('v_fmaak_f32')
def _fmaak(w, i):  # d = a * b + K
    a, b, k = w.v32(i.ops[1], i), w.v32(i.ops[2], i), w.v32(i.ops[3], i)
    with np.errstate(all='ignore'):
        v = fo((fl(a.v).astype(np.float64) * fl(b.v) + fl(k.v)).astype(np.float32))
    w.vwrite(i.ops[0], vres(v, a, b, k))


@handler('v_ldexp_f32')
def _ldexp(w, i):
    a, b = w.v32(i.ops[1], i), w.v32(i.ops[2], i)
    with np.errstate(all='ignore'):
        v = fo(np.ldexp(fl(a.v), b.v.view(np.int32)))
    w.vwrite(i.ops[0], vres(v, a, b))


@handler('v_cvt_f32_u32_e32', 'v_cvt_f32_u32_e64')
def _cvtfu(w, i):
    a = w.v32(i.ops[1], i)
    w.vwrite(i.ops[0], vres(fo(a.v.astype(np.float32)), a))


@handler('v_cvt_f32_i32_e32', 'v_cvt_f32_i32_e64')
def _cvtfi(w, i):
    a = w.v32(i.ops[1], i)
    w.vwrite(i.ops[0], vres(fo(a.v.view(np.int32).astype(np.float32)), a))


@handler('v_cvt_f32_ubyte0_e32', 'v_cvt_f32_ubyte0_e64')
def _cvtub0(w, i):
    a = w.v32(i.ops[1], i)
    w.vwrite(i.ops[0], vres(fo((a.v & np.uint32(0xff)).astype(np.float32)), a))


@handler('v_cvt_u32_f32_e32', 'v_cvt_u32_f32_e64')
def _cvtuf(w, i):
    a = w.v32(i.ops[1], i)
    f = fl(a.v).astype(np.float64)
    f = np.where(np.isnan(f), 0, f)
    v = np.clip(np.trunc(f), 0, M32).astype(np.uint64).astype(np.uint32)
    w.vwrite(i.ops[0], vres(v, a))


@handler('v_cvt_i32_f32_e32', 'v_cvt_i32_f32_e64')
def _cvtif(w, i):
    a = w.v32(i.ops[1], i)
    f = fl(a.v).astype(np.float64)
    f = np.where(np.isnan(f), 0, f)
    v = np.clip(np.trunc(f), -2**31, 2**31 - 1).astype(np.int64).astype(np.int32).view(np.uint32)
    w.vwrite(i.ops[0], vres(v, a))


def dataop(nsrc, first=1):
    """Ops whose result only matters as data: result is opaque (defined iff sources)."""
    def h(w, i):
        srcs = [w.v32(t, i) for t in i.ops[first:first + nsrc] if t not in ('off',)]
        r = vres(np.zeros(NL, np.uint32), *srcs)
        r.o = np.ones(NL, bool)
        preserve = i.mods.get('dst_unused') == 'UNUSED_PRESERVE' or i.op.startswith(('v_fma_mixlo', 'v_fma_mixhi'))
        if preserve:
            old = w.v32(i.ops[0], i)
            r.d = r.d & old.d
        w.vwrite(i.ops[0], r)
    return h


for _n, _k in [('v_cvt_f32_f16_e32', 1), ('v_cvt_f32_f16_e64', 1), ('v_cvt_f32_f16_sdwa', 1), ('v_cvt_f16_f32_e32', 1),
               ('v_cvt_pk_f16_f32', 2), ('v_pack_b32_f16', 2), ('v_perm_b32', 3), ('v_or_b32_sdwa', 2),
               ('v_fma_mixlo_f16', 3), ('v_fma_mixhi_f16', 3), ('v_fma_mix_f32', 3), ('v_cvt_f32_bf16', 1),
               ('v_pk_mul_f16', 2)]:
    HANDLERS[_n] = dataop(_k)


@handler('v_mov_b64_e32', 'v_mov_b64_e64')
def _vmov64(w, i):
    v, d, o = w.v64(i.ops[1], i)
    w.vwrite64(i.ops[0], v, d, o)


# 64-bit results: the low word depends only on the low words of the 64-bit
# sources (and on the 32-bit ones), the high word on everything.
@handler('v_lshl_add_u64')
def _lshladd64(w, i):
    a, adl, adh, aol, aoh = w.v64w(i.ops[1], i)
    s = w.v32(i.ops[2], i)
    b, bdl, bdh, bol, boh = w.v64w(i.ops[3], i)
    v = (a << (u64(s.v) & np.uint64(63))) + b
    dl, ol = adl & bdl & s.d, aol | bol | s.o
    w.vwrite64w(i.ops[0], v, dl, dl & adh & bdh, ol, ol | aoh | boh)


@handler('v_lshlrev_b64')
def _lshlrev64(w, i):
    s = w.v32(i.ops[1], i)
    a, adl, adh, aol, aoh = w.v64w(i.ops[2], i)
    v = a << (u64(s.v) & np.uint64(63))
    dl, ol = adl & s.d, aol | s.o
    w.vwrite64w(i.ops[0], v, dl, dl & adh, ol, ol | aoh)


@handler('v_lshrrev_b64')
def _lshrrev64(w, i):
    s = w.v32(i.ops[1], i)
    a, ad, ao = w.v64(i.ops[2], i)
    v = a >> (u64(s.v) & np.uint64(63))
    w.vwrite64(i.ops[0], v, ad & s.d, ao | s.o)


@handler('v_ashrrev_i64')
def _ashrrev64(w, i):
    s = w.v32(i.ops[1], i)
    a, ad, ao = w.v64(i.ops[2], i)
    v = (a.view(np.int64) >> (u64(s.v) & np.uint64(63)).astype(np.int64)).view(np.uint64)
    w.vwrite64(i.ops[0], v, ad & s.d, ao | s.o)


def carry_out(w, tok, bits, d, o):
    m = w.active()
    b = 0
    ob = 0
    for l in range(NL):
        if m[l]:
            if bits[l]:
                b |= 1 << l
            if o[l]:
                ob |= 1 << l
    w.s64set(tok, b, ob, bool((d | ~m).all()))


@handler('v_mad_u64_u32', 'v_mad_i64_i32')
def _mad64(w, i):
    a, b = w.v32(i.ops[2], i), w.v32(i.ops[3], i)
    c, cdl, cdh, col, coh = w.v64w(i.ops[4], i)
    if i.op == 'v_mad_u64_u32':
        p = a.v.astype(object) * b.v.astype(object)
    else:
        p = a.v.view(np.int32).astype(object) * b.v.view(np.int32).astype(object)
    full = p + (c.astype(object) if i.op == 'v_mad_u64_u32' else c.view(np.int64).astype(object))
    v = np.array([int(x) & M64 for x in full], dtype=np.uint64)
    carry = np.array([(int(x) >> 64) & 1 if i.op == 'v_mad_u64_u32' else 0 for x in full], bool)
    dl, ol = a.d & b.d & cdl, a.o | b.o | col
    d, o = dl & cdh, ol | coh
    w.vwrite64w(i.ops[0], v, dl, d, ol, o)
    carry_out(w, i.ops[1], carry, d, o)


def addsub_co(kind):
    """v_add_co_u32 / v_sub_co_u32 / v_subrev_co_u32 (+ carry-in forms)."""
    def h(w, i):
        dst, cdst = i.ops[0], i.ops[1]
        a, b = w.v32(i.ops[2], i), w.v32(i.ops[3], i)
        cin = np.zeros(NL, np.int64)
        cd, co = np.ones(NL, bool), np.zeros(NL, bool)
        if kind in ('addc', 'subb', 'subbrev'):
            sv, so, sd = w.s64(i.ops[4], i)
            cin = ((np.uint64(sv) >> LANES.astype(np.uint64)) & np.uint64(1)).astype(np.int64)
            co = ((np.uint64(so) >> LANES.astype(np.uint64)) & np.uint64(1)).astype(bool)
            cd = np.full(NL, sd)
        A = a.v.astype(np.int64)
        B = b.v.astype(np.int64)
        if kind in ('add', 'addc'):
            r = A + B + cin
            carry = r >> 32
        elif kind in ('sub', 'subb'):
            r = A - B - cin
            carry = (r < 0)
        else:  # subrev, subbrev
            r = B - A - cin
            carry = (r < 0)
        v = (r & M32).astype(np.uint32)
        d = a.d & b.d & cd
        o = a.o | b.o | co
        w.vwrite(dst, VVal(v, d, o))
        carry_out(w, cdst, np.asarray(carry, bool), d, o)
    return h


for _pfx, _k in [('v_add_co_u32', 'add'), ('v_addc_co_u32', 'addc'), ('v_sub_co_u32', 'sub'),
                 ('v_subb_co_u32', 'subb'), ('v_subrev_co_u32', 'subrev'), ('v_subbrev_co_u32', 'subbrev')]:
    HANDLERS[_pfx + '_e32'] = addsub_co(_k)
    HANDLERS[_pfx + '_e64'] = addsub_co(_k)


@handler('v_cndmask_b32_e32', 'v_cndmask_b32_e64')
def _cnd(w, i):
    a, b = w.v32(i.ops[1], i), w.v32(i.ops[2], i)
    mtok = i.ops[3] if len(i.ops) > 3 else 'vcc'
    sv, so, sd = w.s64(mtok, i)
    sel = ((np.uint64(sv) >> LANES.astype(np.uint64)) & np.uint64(1)).astype(bool)
    sop = ((np.uint64(so) >> LANES.astype(np.uint64)) & np.uint64(1)).astype(bool)
    v = np.where(sel, b.v, a.v)
    d = np.where(sop, a.d & b.d, np.where(sel, b.d, a.d)) & sd
    o = np.where(sop, True, np.where(sel, b.o, a.o))
    w.vwrite(i.ops[0], VVal(v.astype(np.uint32), d, o))


def vcmp(fn, kind):
    """kind: 'u32','i32','u64','i64','f32'."""
    def h(w, i):
        dst = i.ops[0]
        if kind in ('u64', 'i64'):
            a, ad, ao = w.v64(i.ops[1], i)
            b, bd, bo = w.v64(i.ops[2], i)
            if kind == 'i64':
                a, b = a.view(np.int64), b.view(np.int64)
            with np.errstate(all='ignore'):
                r = fn(a, b)
            d, o = ad & bd, ao | bo
        else:
            A, B = w.v32(i.ops[1], i), w.v32(i.ops[2], i)
            a, b = A.v, B.v
            if kind == 'i32':
                a, b = a.view(np.int32), b.view(np.int32)
            elif kind == 'f32':
                a, b = fl(a), fl(b)
            with np.errstate(all='ignore'):
                r = fn(a, b)
            d, o = A.d & B.d, A.o | B.o
        m = w.active()
        bits = ob = 0
        for l in range(NL):
            if m[l]:
                if o[l]:
                    ob |= 1 << l
                elif r[l]:
                    bits |= 1 << l
        dd = bool((d | ~m).all())
        if not dd:
            # undefined compare inputs on active lanes: keep going but note it
            w.rep.add('WARN-UNDEF-CMP', i)
        w.s64set(dst, bits, ob, dd)
    return h


_CMPS = {
    'eq': lambda a, b: a == b, 'ne': lambda a, b: a != b, 'lg': lambda a, b: a != b,
    'gt': lambda a, b: a > b, 'ge': lambda a, b: a >= b, 'lt': lambda a, b: a < b, 'le': lambda a, b: a <= b,
    'nlt': lambda a, b: ~(a < b), 'ngt': lambda a, b: ~(a > b), 'nle': lambda a, b: ~(a <= b),
    'nge': lambda a, b: ~(a >= b), 'u': lambda a, b: np.isnan(a) | np.isnan(b), 'o': lambda a, b: ~(np.isnan(a) | np.isnan(b)),
}
for _c, _f in _CMPS.items():
    for _t in ('u32', 'i32', 'u64', 'i64', 'f32'):
        for _e in ('_e32', '_e64'):
            HANDLERS[f'v_cmp_{_c}_{_t}{_e}'] = vcmp(_f, _t)


@handler('v_readfirstlane_b32')
def _rfl(w, i):
    src = w.v32(i.ops[1], i)
    m = w.active()
    l = int(np.argmax(m)) if m.any() else 0
    if not src.d[l]:
        w.rep.add('WARN-UNDEF-READLANE', i)
    w.s32set(i.ops[0], int(src.v[l]), M32 if src.o[l] else 0, bool(src.d[l]))


@handler('v_readlane_b32')
def _rl(w, i):
    src = w.v32(i.ops[1], i)
    ln, lo, ld = w.s32(i.ops[2], i)
    l = ln & 63
    w.s32set(i.ops[0], int(src.v[l]), M32 if src.o[l] else 0, bool(src.d[l]))


@handler('v_writelane_b32')
def _wl(w, i):
    sv, so, sd = w.s32(i.ops[1], i)
    ln, lo, ld = w.s32(i.ops[2], i)
    lanes = np.zeros(NL, bool)
    lanes[ln & 63] = True
    w.vwrite(i.ops[0], VVal(np.full(NL, sv, np.uint32), np.full(NL, sd), np.full(NL, bool(so))), lanes)


@handler('v_mbcnt_lo_u32_b32', 'v_mbcnt_hi_u32_b32')
def _mbcnt(w, i):
    mv, mo, md = w.s32(i.ops[1], i)
    src = w.v32(i.ops[2], i)
    out = np.zeros(NL, np.uint32)
    for l in range(NL):
        if i.op == 'v_mbcnt_lo_u32_b32':
            k = min(l, 32)
        else:
            k = max(0, min(l - 32, 32))
        out[l] = bin(mv & ((1 << k) - 1)).count('1')
    w.vwrite(i.ops[0], VVal(out + src.v, src.d & md, src.o | bool(mo)))


@handler('v_accvgpr_read_b32', 'v_accvgpr_write_b32', 'v_accvgpr_mov_b32')
def _acc(w, i):
    w.vwrite(i.ops[0], w.v32(i.ops[1], i))


def dpp_src(w, i, tok):
    """Source value after the DPP lane shuffle; returns (VVal, write-enable mask)."""
    src = w.v32(tok, i)
    act = w.active()
    bound0 = i.mods.get('bound_ctrl') in ('1', '0', True)  # printed bound_ctrl:1 means zero fill
    idx = LANES.copy()
    valid = np.ones(NL, bool)
    if 'row_shr' in i.mods:
        n = int(i.mods['row_shr'], 0)
        valid = (LANES % 16) >= n
        idx = np.where(valid, LANES - n, LANES)
    elif 'row_shl' in i.mods:
        n = int(i.mods['row_shl'], 0)
        valid = (LANES % 16) + n < 16
        idx = np.where(valid, LANES + n, LANES)
    elif 'row_newbcast' in i.mods:
        n = int(i.mods['row_newbcast'], 0)
        idx = (LANES // 16) * 16 + n
    elif 'quad_perm' in i.mods:
        perm = np.array([int(ch) for ch in i.mods['quad_perm']])
        idx = (LANES // 4) * 4 + perm[LANES % 4]
    elif 'row_half_mirror' in i.mods:
        idx = (LANES // 8) * 8 + 7 - LANES % 8
    elif 'row_mirror' in i.mods:
        idx = (LANES // 16) * 16 + 15 - LANES % 16
    elif 'row_bcast' in i.mods or 'wave_shr' in i.mods or 'row_ror' in i.mods:
        raise NotImplementedError(f"dpp {i.mods}")
    valid = valid & act[idx]
    v = src.v[idx].copy()
    d = src.d[idx].copy()
    o = src.o[idx].copy()
    if bound0:
        v = np.where(valid, v, 0).astype(np.uint32)
        d = np.where(valid, d, True)
        o = np.where(valid, o, False)
        we = act
    else:
        we = act & valid
    return VVal(v, d, o), we


@handler('v_mov_b32_dpp')
def _movdpp(w, i):
    s, we = dpp_src(w, i, i.ops[1])
    w.vwrite(i.ops[0], s, we)


@handler('v_add_f32_dpp')
def _adddpp(w, i):
    s, we = dpp_src(w, i, i.ops[1])
    b = w.v32(i.ops[2], i)
    with np.errstate(all='ignore'):
        v = fo(fl(s.v) + fl(b.v))
    w.vwrite(i.ops[0], vres(v, s, b), we)


@handler('v_max_f32_dpp')
def _maxdpp(w, i):
    s, we = dpp_src(w, i, i.ops[1])
    b = w.v32(i.ops[2], i)
    v = fo(np.maximum(fl(s.v), fl(b.v)))
    w.vwrite(i.ops[0], vres(v, s, b), we)


def mfma(i, w):
    # v_mfma_* dst, A, B, C : result opaque; defined iff every lane of A, B and C is defined
    dst, A, B, C = i.ops[:4]
    ok = True
    for t in (A, B, C):
        r = w.vidx(t)
        if r is None:
            continue
        for j in range(r[0], r[1] + 1):
            ok = ok and bool(w.VD[j].all())
    r = w.vidx(dst)
    lanes = np.ones(NL, bool)
    w.vwrite_multi(dst, np.full(NL, ok), np.ones(NL, bool), lanes)
    if not ok:
        w.rep.add('WARN-UNDEF-MFMA', i)


PREFIX_HANDLERS.append(('v_mfma_', lambda w, i: mfma(i, w)))


# ---------------------------------------------------------------------------
# LDS
# ---------------------------------------------------------------------------
def lds_check(w, i, addr: VVal, offs, size, lanes):
    if not lanes.any():
        return
    if (~addr.d & lanes).any():
        w.rep.add('ERR-UNDEF-ADDR', i, 'lds')
        return
    if (addr.o & lanes).any():
        w.rep.add('WARN-DATA-ADDR', i, 'lds')
        return
    for off in offs:
        a = addr.v[lanes].astype(np.int64) + off
        if (a < 0).any() or (a + size > w.lds_size).any():
            w.rep.add('ERR-LDS', i, f"max {int(a.max()) + size} > {w.lds_size}")
            return


def ds_read(nregs, size, two=False, st64=False):
    def h(w, i):
        dst, vaddr = i.ops[0], i.ops[1]
        addr = w.v32(vaddr, i)
        lanes = w.active()
        if two:
            mul = size * (64 if st64 else 1)
            offs = [int(i.mods.get('offset0', 0)) * mul, int(i.mods.get('offset1', 0)) * mul]
        else:
            offs = [int(i.mods.get('offset', 0))]
        lds_check(w, i, addr, offs, size, lanes)
        d = addr.d.copy()
        w.vwrite_multi(dst, d, np.ones(NL, bool), lanes)
    return h


def ds_write(size, two=False, st64=False):
    def h(w, i):
        vaddr = i.ops[0]
        addr = w.v32(vaddr, i)
        lanes = w.active()
        if two:
            mul = size * (64 if st64 else 1)
            offs = [int(i.mods.get('offset0', 0)) * mul, int(i.mods.get('offset1', 0)) * mul]
        else:
            offs = [int(i.mods.get('offset', 0))]
        lds_check(w, i, addr, offs, size, lanes)
        for t in i.ops[1:]:
            w.check_data(i, t, lanes, max(1, size // 4))
    return h


HANDLERS.update({
    'ds_read_b32': ds_read(1, 4), 'ds_read_b64': ds_read(2, 8), 'ds_read_b128': ds_read(4, 16),
    'ds_read_b96': ds_read(3, 12),
    # transposing read: each lane reads 8 bytes of the row block; same address rules as ds_read_b64
    'ds_read_b64_tr_b16': ds_read(2, 8),
    'ds_read2_b32': ds_read(2, 4, True), 'ds_read2st64_b32': ds_read(2, 4, True, True),
    'ds_read2_b64': ds_read(4, 8, True),
    'ds_read_u16': ds_read(1, 2), 'ds_read_u16_d16': ds_read(1, 2), 'ds_read_u16_d16_hi': ds_read(1, 2),
    'ds_write_b32': ds_write(4), 'ds_write_b64': ds_write(8), 'ds_write_b128': ds_write(16),
    'ds_write_b16': ds_write(2), 'ds_write_b16_d16_hi': ds_write(2), 'ds_write_b8': ds_write(1),
    'ds_write2_b32': ds_write(4, True), 'ds_write2st64_b32': ds_write(4, True, True),
    'ds_write2_b64': ds_write(8, True), 'ds_write_b96': ds_write(12),
    'ds_write2st64_b64': ds_write(8, True, True), 'ds_read2st64_b64': ds_read(4, 8, True, True),
})


@handler('ds_bpermute_b32')
def _bperm(w, i):
    dst, addr_t, data_t = i.ops[0], i.ops[1], i.ops[2]
    addr, data = w.v32(addr_t, i), w.v32(data_t, i)
    lanes = w.active()
    if (~addr.d & lanes).any():
        w.rep.add('ERR-UNDEF-ADDR', i, 'bpermute index')
    off = int(i.mods.get('offset', 0))
    src = ((addr.v.astype(np.int64) + off) // 4) % 64
    act = lanes
    v = data.v[src]
    d = data.d[src] & act[src] & addr.d
    o = data.o[src] | addr.o
    w.vwrite(dst, VVal(v.astype(np.uint32), d, o))


# ---------------------------------------------------------------------------
# global / buffer memory
# ---------------------------------------------------------------------------
def gaddr(w, i, vaddr_tok, saddr_tok):
    off = int(i.mods.get('offset', 0))
    if saddr_tok in (None, 'off'):
        a, d, o = w.v64(vaddr_tok, i)
        return a + np.uint64(off & M64) if off >= 0 else a - np.uint64(-off), d, o
    sb, so, sd = w.s64(saddr_tok, i)
    v = w.v32(vaddr_tok, i)
    a = np.uint64(sb) + u64(v.v) + np.uint64(off) if off >= 0 else np.uint64(sb) + u64(v.v) - np.uint64(-off)
    return a, v.d & sd, v.o | bool(so)


def gload(nregs, nbytes=None):
    def h(w, i):
        dst, vaddr = i.ops[0], i.ops[1]
        saddr = i.ops[2] if len(i.ops) > 2 else 'off'
        lanes = w.active()
        a, d, o = gaddr(w, i, vaddr, saddr)
        rg = w.check_addr(i, a, d, o, nbytes or 4 * nregs, 'r', lanes)
        if rg is not None and rg.load_value is not None:
            r = w.vidx(dst)
            for j in range(r[0], r[1] + 1):
                w.V[j][lanes] = rg.load_value
                w.VD[j][lanes] = d[lanes]
                w.VO[j][lanes] = False
        else:
            w.vwrite_multi(dst, d, np.ones(NL, bool), lanes)
    return h


def gstore(nregs, nbytes=None):
    def h(w, i):
        vaddr, data = i.ops[0], i.ops[1]
        saddr = i.ops[2] if len(i.ops) > 2 else 'off'
        lanes = w.active()
        a, d, o = gaddr(w, i, vaddr, saddr)
        w.check_addr(i, a, d, o, nbytes or 4 * nregs, 'w', lanes)
        w.check_data(i, data, lanes, nregs)
    return h


def gatomic(w, i):
    # global_atomic_add [vdst,] vaddr, vdata, saddr|off
    ret = 'sc0' in i.mods or 'glc' in i.mods
    ops = i.ops
    if ret:
        dst, vaddr, data = ops[0], ops[1], ops[2]
        saddr = ops[3] if len(ops) > 3 else 'off'
    else:
        dst, vaddr, data = None, ops[0], ops[1]
        saddr = ops[2] if len(ops) > 2 else 'off'
    lanes = w.active()
    a, d, o = gaddr(w, i, vaddr, saddr)
    w.check_addr(i, a, d, o, 4, 'w', lanes)
    w.check_data(i, data, lanes)
    if dst:
        w.vwrite_multi(dst, d, np.ones(NL, bool), lanes)


HANDLERS.update({'global_load_dword': gload(1), 'global_load_dwordx2': gload(2), 'global_load_dwordx3': gload(3),
                 'global_load_dwordx4': gload(4), 'global_load_ushort': gload(1, 2),
                 'global_load_short_d16': gload(1, 2), 'global_load_short_d16_hi': gload(1, 2),
                 'global_store_dword': gstore(1), 'global_store_dwordx2': gstore(2),
                 'global_store_dwordx3': gstore(3), 'global_store_dwordx4': gstore(4),
                 'global_store_short': gstore(1, 2), 'global_store_short_d16_hi': gstore(1, 2),
                 'global_store_byte': gstore(1, 1)})
PREFIX_HANDLERS.append(('global_atomic_', gatomic))


def rsrc(w, i, tok):
    m = re.match(r'^s\[(\d+):(\d+)\]$', tok)
    a = int(m.group(1))
    ws = [w.S[a + k] for k in range(4)]
    d = all(w.SD[a + k] for k in range(4))
    o = any(w.SO[a + k] for k in range(4))
    base = ws[0] | ((ws[1] & 0xFFFF) << 32)
    stride = (ws[1] >> 16) & 0x3FFF
    nrec = ws[2]
    return base, stride, nrec, d, o


def buffer_op(nregs, store):
    def h(w, i):
        vdata, vaddr, rs, soff = i.ops[0], i.ops[1], i.ops[2], i.ops[3]
        lanes = w.active()
        base, stride, nrec, rd, ro = rsrc(w, i, rs)
        if not rd:
            w.rep.add('ERR-UNDEF-ADDR', i, 'rsrc')
        if ro:
            w.rep.add('WARN-DATA-ADDR', i, 'rsrc')
        assert stride == 0, i.raw
        so_v, so_o, so_d = w.s32(soff, i)
        imm = int(i.mods.get('offset', 0))
        if 'offen' in i.mods:
            v = w.v32(vaddr, i)
            voff, vd, vo = u64(v.v), v.d, v.o
        else:
            voff, vd, vo = np.zeros(NL, np.uint64), np.ones(NL, bool), np.zeros(NL, bool)
        d = vd & so_d & rd
        o = vo | bool(so_o) | ro
        if (~d & lanes).any():
            w.rep.add('ERR-UNDEF-ADDR', i, f"lanes {np.nonzero(~d & lanes)[0][:8].tolist()}")
        elif (o & lanes).any() and not ro and not so_o and lanes.any():
            # an offset that depends on loaded data: the descriptor still
            # confines every access to [base, base + num_records), so the whole
            # window must lie inside one buffer the access may touch
            w.check_window(i, base + so_v, nrec, 'w' if store else 'r')
        elif (o & lanes).any():
            w.rep.add('WARN-DATA-ADDR', i)
        else:
            rng = voff + np.uint64(imm)            # range-checked part
            inr = lanes & (rng + np.uint64(4 * nregs) <= np.uint64(nrec))
            if (lanes & ~inr).any():
                w.rep.add('INFO-BUFFER-OOR', i)
            addr = np.uint64(base) + rng + np.uint64(so_v)
            w.check_addr(i, addr, d, o, 4 * nregs, 'w' if store else 'r', inr)
        if store:
            w.check_data(i, vdata, lanes, nregs)
        else:
            w.vwrite_multi(vdata, d, np.ones(NL, bool), lanes)
    return h


HANDLERS.update({'buffer_load_dword': buffer_op(1, False), 'buffer_load_dwordx2': buffer_op(2, False),
                 'buffer_load_dwordx4': buffer_op(4, False),
                 'buffer_store_dword': buffer_op(1, True), 'buffer_store_dwordx2': buffer_op(2, True),
                 'buffer_store_dwordx4': buffer_op(4, True)})


# ---------------------------------------------------------------------------
# driver
# ---------------------------------------------------------------------------
def run_wave(prog, labels, desc, kernarg, regions, lds_size, wg, wave, report, max_paths=200, fork_limit=2):
    """Explore every decision path of one wave. Returns the number of paths."""
    todo = [[]]
    paths = 0
    while todo:
        dec = todo.pop()
        w = Wave(prog, labels, desc, kernarg, regions, lds_size, wg, wave, dec, report, fork_limit=fork_limit)
        w.run()
        paths += 1
        for pos, n in w.new_decisions:
            for c in range(1, n):
                todo.append(w.decisions[:pos] + [c])
        if paths >= max_paths:
            report.add('INFO-PATHLIMIT', prog[0], str(len(todo)))
            break
    return paths


_SDWA_SEL = {'DWORD': (0, 32), 'WORD_0': (0, 16), 'WORD_1': (16, 16), 'BYTE_0': (0, 8), 'BYTE_1': (8, 8),
             'BYTE_2': (16, 8), 'BYTE_3': (24, 8)}


def sdwa_int(fn, nsrc):
    """Integer SDWA ops: each source field is zero-extended from its src*_sel;
    only a full-dword destination is supported."""
    def h(w, i):
        if i.mods.get('dst_sel', 'DWORD') != 'DWORD' or any('sext' in t for t in i.ops):
            raise NotImplementedError(i.raw)
        srcs = [w.v32(t, i) for t in i.ops[1:1 + nsrc]]
        vals = []
        for k, sv in enumerate(srcs):
            sh, nb = _SDWA_SEL[i.mods.get(f'src{k}_sel', 'DWORD')]
            vals.append((sv.v >> np.uint32(sh)) & np.uint32((1 << nb) - 1) if nb < 32 else sv.v)
        with np.errstate(all='ignore'):
            v = fn(*vals)
        w.vwrite(i.ops[0], vres(np.asarray(v, np.uint32), *srcs))
    return h


def _bitop3(a, b, c, tt):
    """Three-input bitwise function by truth table: result bit = bit
    (4 a + 2 b + c) of tt (a <-> 0xF0, b <-> 0xCC, c <-> 0xAA)."""
    r = np.zeros_like(a)
    for idx in range(8):
        if (tt >> idx) & 1:
            r |= (a if idx & 4 else ~a) & (b if idx & 2 else ~b) & (c if idx & 1 else ~c)
    return r


@handler('v_bitop3_b32')
def _vbitop3(w, i):
    tt = int(i.mods['bitop3'], 0)
    valu(lambda a, b, c: _bitop3(a, b, c, tt), 3)(w, i)


HANDLERS.update({
    'v_add_u32_sdwa': sdwa_int(lambda a, b: a + b, 2),
    'v_sub_u32_sdwa': sdwa_int(lambda a, b: a - b, 2),
    'v_mov_b32_sdwa': sdwa_int(lambda a: a, 1),
    'v_and_b32_sdwa': sdwa_int(lambda a, b: a & b, 2),
    'v_mul_i32_i24_sdwa': sdwa_int(lambda a, b: ((s24(a) * s24(b)).astype(np.uint64) & np.uint64(M32))
                                   .astype(np.uint32), 2),
    'v_mul_u32_u24_sdwa': sdwa_int(lambda a, b: ((u64(a & np.uint32(0xFFFFFF)) * u64(b & np.uint32(0xFFFFFF)))
                                                 & np.uint64(M32)).astype(np.uint32), 2),
    'v_mul_lo_u16_sdwa': sdwa_int(lambda a, b: (u64(a & np.uint32(0xFFFF)) * u64(b & np.uint32(0xFFFF))
                                                & np.uint64(0xFFFF)).astype(np.uint32), 2),
    # 16-bit VOP2 ops of this generation write the low half and zero the high half
    'v_mul_lo_u16_e32': valu(lambda a, b: (u64(a & np.uint32(0xFFFF)) * u64(b & np.uint32(0xFFFF))
                                          & np.uint64(0xFFFF)).astype(np.uint32), 2),
    'v_sub_u16_e32': valu(lambda a, b: (a - b) & np.uint32(0xFFFF), 2),
    'v_lshrrev_b16_e32': valu(lambda a, b: (b & np.uint32(0xFFFF)) >> (a & np.uint32(15)), 2),
})


@handler('v_cndmask_b32_sdwa')
def _cnd_sdwa(w, i):
    # select of 16-bit fields: data only
    _cnd(w, Inst('v_cndmask_b32_e64', i.ops[:4], {}, i.raw, i.idx))
    r = w.vidx(i.ops[0])
    m = w.active()
    w.VO[r[0]][m] = True


def dataop_wide(nsrc, first=1):
    """Data ops with register-pair operands (float64 helpers of the math library):
    every destination register is opaque, defined iff every source register is."""
    def h(w, i):
        lanes = w.active()
        d = np.ones(NL, bool)
        for t in i.ops[first:first + nsrc]:
            r = w.vidx(t)
            if r is None:
                sv, so, sd = w.s32(t, i) if not t.startswith('s[') else (0, 0, w.s64(t, i)[2])
                d &= sd
                continue
            for j in range(r[0], r[1] + 1):
                d &= w.VD[j]
        w.vwrite_multi(i.ops[0], d, np.ones(NL, bool), lanes)
    return h


for _n, _k in [('v_frexp_mant_f32_e32', 1), ('v_frexp_exp_i32_f32_e32', 1), ('v_cvt_f64_f32_e32', 1),
               ('v_frexp_exp_i32_f64_e32', 1), ('v_div_fixup_f32', 3), ('v_rsq_f32_e32', 1)]:
    HANDLERS[_n] = dataop_wide(_k)


@handler('v_div_scale_f32')
def _divscale(w, i):
    # v_div_scale_f32 vdst, sdst, s0, s1, s2: data result plus a per-lane flag mask
    lanes = w.active()
    srcs = [w.v32(t, i) for t in i.ops[2:5]]
    d = np.ones(NL, bool)
    for x in srcs:
        d &= x.d
    w.vwrite_multi(i.ops[0], d, np.ones(NL, bool), lanes)
    ob = 0
    for l in range(NL):
        if lanes[l]:
            ob |= 1 << l
    w.s64set(i.ops[1], 0, ob, bool((d | ~lanes).all()))


@handler('v_div_fmas_f32')
def _divfmas(w, i):
    # reads VCC (the flag mask of v_div_scale) besides its three sources
    vv, vo, vd = w.s64('vcc', i)
    if not vd:
        w.rep.add('WARN-UNDEF-CMP', i, 'vcc')
    dataop_wide(3)(w, i)


for _t in ('f32',):
    for _e in ('_e32', '_e64'):
        HANDLERS[f'v_cmp_neq_{_t}{_e}'] = vcmp(lambda a, b: ~(a == b), _t)
        HANDLERS[f'v_cmp_class_{_t}{_e}'] = vcmp(lambda a, b: np.zeros(a.shape, bool), 'u32')
