"""Pins for the CPU oracle: it is checked against things other than itself.

* brute force: the quadratic masked form of the recurrence with *explicit
  products* of the gates (not exponentials of sums), pure-Python loops, tiny
  shapes - the unrolled form of the paper's Sec. 3.1 recurrence;
* closed forms: all gates 1 (g = 0) is causal linear attention
  ``tril(Q K^T) V``; gates ~ 0 (g = -60) leaves ``o_t = (q_t . k_t) v_t``; one
  scalar gate shared by all dimensions is retention ``sum_j gamma^(t-j) ...``;
* direction identities: the reversed scans are flip - run - flip, the
  column scan is the row scan of the transposed grid;
* state split: run the first L1 tokens, resume from the returned final state;
* L = 1 and linearity in v and in S0;
* a hand-written scan-order fixture (tests/golden/scan_order.txt).

``test_pins_reject_planted_mistakes`` shows that each pin family has power: a
Python copy of the recurrence with one planted mistake (wrong gate placement,
wrong exponent sign, swapped q/k, dropped S0, dropped scale, the previous token's gate)
fails at least one of the same checks the oracle passes.
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL = 1e-11


def rel_err(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b)) / (np.max(np.abs(b)) + 1e-300))


def rand_inputs(rng, BH, L, dk, dv, gate_lo=-2.0, gate_hi=0.0, with_s0=True):
    q = rng.standard_normal((1, BH, L, dk))
    k = rng.standard_normal((1, BH, L, dk))
    v = rng.standard_normal((1, BH, L, dv))
    g = rng.uniform(gate_lo, gate_hi, size=(1, BH, L, dk))
    s0 = rng.standard_normal((1, BH, dk, dv)) if with_s0 else None
    return q, k, v, g, s0


# ----------------------------------------------------------------------------
# independent references
# ----------------------------------------------------------------------------

def brute_force(q, k, v, g, s0, scale):
    """One sequence already in scan order: quadratic form, explicit gate products."""
    L, dk = q.shape
    dv = v.shape[1]
    gam = [[math.exp(g[t][i]) for i in range(dk)] for t in range(L)]
    o = [[0.0] * dv for _ in range(L)]
    for t in range(L):
        for j in range(t + 1):
            for i in range(dk):
                w = 1.0
                for u in range(j + 1, t + 1):
                    w *= gam[u][i]
                c = q[t][i] * w * k[j][i]
                for m in range(dv):
                    o[t][m] += c * v[j][m]
        if s0 is not None:
            for i in range(dk):
                w = 1.0
                for u in range(0, t + 1):
                    w *= gam[u][i]
                for m in range(dv):
                    o[t][m] += q[t][i] * w * s0[i][m]
        for m in range(dv):
            o[t][m] *= scale
    S = [[0.0] * dv for _ in range(dk)]
    for j in range(L):
        for i in range(dk):
            w = 1.0
            for u in range(j + 1, L):
                w *= gam[u][i]
            for m in range(dv):
                S[i][m] += w * k[j][i] * v[j][m]
    if s0 is not None:
        for i in range(dk):
            w = 1.0
            for u in range(L):
                w *= gam[u][i]
            for m in range(dv):
                S[i][m] += w * s0[i][m]
    return np.array(o), np.array(S)


def brute_force_grid(q, k, v, g, s0, scale, H, W, scan):
    """Brute force on [1, BH, L, d] spatial-order inputs for a scan direction."""
    order = oracle.scan_order(H, W, scan)
    BH = q.shape[1]
    o = np.zeros(v.shape)
    S = np.zeros((1, BH, q.shape[-1], v.shape[-1]))
    for b in range(BH):
        ob, Sb = brute_force(q[0, b][order], k[0, b][order], v[0, b][order], g[0, b][order],
                             None if s0 is None else s0[0, b], scale)
        o[0, b][order] = ob
        S[0, b] = Sb
    return o, S


# ----------------------------------------------------------------------------
# pin checks, parameterised by the implementation under test
# ----------------------------------------------------------------------------

def pin_brute_force(fn, seed):
    rng = np.random.default_rng(100 + seed)
    cases = [(2, 3, 2, "row"), (3, 2, 3, "col"), (2, 3, 3, "row_rev"), (3, 3, 2, "col_rev"),
             (1, 5, 4, "row")]
    for (H, W, dk, scan) in cases:
        dv = dk + 1
        q, k, v, g, s0 = rand_inputs(rng, 2, H * W, dk, dv, -1.5, 0.0)
        scale = 0.7
        o, S = fn(q, k, v, g, s0, scale=scale, H=H, W=W, scan=scan)
        ob, Sb = brute_force_grid(q, k, v, g, s0, scale, H, W, scan)
        if rel_err(o, ob) > TOL or rel_err(S, Sb) > TOL:
            return False
    return True


def pin_linear_attention(fn):
    rng = np.random.default_rng(7)
    H, W, dk, dv = 4, 5, 6, 3
    q, k, v, _, _ = rand_inputs(rng, 2, H * W, dk, dv, with_s0=False)
    g = np.zeros_like(q)
    o, S = fn(q, k, v, g, None, scale=1.0, H=H, W=W, scan="row")
    for b in range(2):
        ref = np.tril(q[0, b] @ k[0, b].T) @ v[0, b]
        if rel_err(o[0, b], ref) > TOL:
            return False
        if rel_err(S[0, b], k[0, b].T @ v[0, b]) > TOL:
            return False
    return True


def pin_forgetting(fn):
    rng = np.random.default_rng(8)
    H, W, dk, dv = 3, 4, 5, 4
    q, k, v, _, s0 = rand_inputs(rng, 2, H * W, dk, dv)
    g = np.full_like(q, -60.0)
    o, S = fn(q, k, v, g, s0, scale=0.5, H=H, W=W, scan="row")
    for b in range(2):
        ref = 0.5 * np.sum(q[0, b] * k[0, b], axis=1, keepdims=True) * v[0, b]
        if rel_err(o[0, b], ref) > 1e-9:
            return False
        if rel_err(S[0, b], np.outer(k[0, b, -1], v[0, b, -1])) > 1e-9:
            return False
    return True


def pin_retention(fn):
    rng = np.random.default_rng(9)
    H, W, dk, dv = 3, 5, 4, 5
    q, k, v, _, _ = rand_inputs(rng, 1, H * W, dk, dv, with_s0=False)
    gamma = 0.83
    g = np.full_like(q, math.log(gamma))
    o, _ = fn(q, k, v, g, None, scale=1.0, H=H, W=W, scan="row")
    L = H * W
    t = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    decay = np.where(t >= j, np.power(gamma, np.maximum(t - j, 0)), 0.0)
    ref = ((q[0, 0] @ k[0, 0].T) * decay) @ v[0, 0]
    return rel_err(o[0, 0], ref) <= TOL


def pin_directions(fn):
    rng = np.random.default_rng(10)
    H, W, dk, dv = 3, 5, 4, 3
    q, k, v, g, s0 = rand_inputs(rng, 2, H * W, dk, dv, -1.0, 0.0)
    sc = 0.9
    run = lambda xs, scan, HH, WW: fn(*xs, s0, scale=sc, H=HH, W=WW, scan=scan)
    flip = lambda x: x[:, :, ::-1, :].copy()
    o_row, S_row = run((q, k, v, g), "row", H, W)
    o_rr, S_rr = run((q, k, v, g), "row_rev", H, W)
    o_fl, S_fl = run((flip(q), flip(k), flip(v), flip(g)), "row", H, W)
    if rel_err(o_rr, flip(o_fl)) > TOL or rel_err(S_rr, S_fl) > TOL:
        return False

    def tgrid(x, HH, WW):  # spatial [.., H*W, E] -> transposed grid [.., W*H, E]
        sh = x.shape
        return x.reshape(sh[0], sh[1], HH, WW, sh[-1]).transpose(0, 1, 3, 2, 4).reshape(sh)

    o_col, S_col = run((q, k, v, g), "col", H, W)
    o_t, S_t = run(tuple(tgrid(x, H, W) for x in (q, k, v, g)), "row", W, H)
    if rel_err(o_col, tgrid(o_t, W, H)) > TOL or rel_err(S_col, S_t) > TOL:
        return False
    o_cr, S_cr = run((q, k, v, g), "col_rev", H, W)
    o_tr, S_tr = run(tuple(tgrid(x, H, W) for x in (q, k, v, g)), "row_rev", W, H)
    return rel_err(o_cr, tgrid(o_tr, W, H)) <= TOL and rel_err(S_cr, S_tr) <= TOL


def pin_state_split(fn):
    rng = np.random.default_rng(11)
    L, dk, dv = 23, 5, 6
    q, k, v, g, s0 = rand_inputs(rng, 2, L, dk, dv, -0.8, 0.0)
    o, S = fn(q, k, v, g, s0, scale=0.3, H=1, W=L, scan="row")
    for L1 in (1, 9, 22):
        o1, S1 = fn(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], g[:, :, :L1], s0,
                    scale=0.3, H=1, W=L1, scan="row")
        L2 = L - L1
        o2, S2 = fn(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], g[:, :, L1:], S1,
                    scale=0.3, H=1, W=L2, scan="row")
        if rel_err(np.concatenate([o1, o2], axis=2), o) > TOL or rel_err(S2, S) > TOL:
            return False
    return True


def pin_single_token(fn):
    rng = np.random.default_rng(12)
    dk, dv = 4, 3
    q, k, v, g, s0 = rand_inputs(rng, 3, 1, dk, dv)
    o, S = fn(q, k, v, g, s0, scale=1.3, H=1, W=1, scan="col_rev")
    for b in range(3):
        Sb = np.exp(g[0, b, 0])[:, None] * s0[0, b] + np.outer(k[0, b, 0], v[0, b, 0])
        if rel_err(S[0, b], Sb) > TOL or rel_err(o[0, b, 0], 1.3 * q[0, b, 0] @ Sb) > TOL:
            return False
    return True


def pin_linearity(fn):
    rng = np.random.default_rng(13)
    H, W, dk, dv = 2, 6, 3, 4
    q, k, v, g, s0 = rand_inputs(rng, 1, H * W, dk, dv)
    _, _, v2, _, s02 = rand_inputs(rng, 1, H * W, dk, dv)
    a, b = 0.37, -1.9
    run = lambda vv, ss: fn(q, k, vv, g, ss, scale=1.0, H=H, W=W, scan="col")
    o1, S1 = run(v, s0)
    o2, S2 = run(v2, s02)
    o3, S3 = run(a * v + b * v2, a * s0 + b * s02)
    return rel_err(o3, a * o1 + b * o2) <= 1e-10 and rel_err(S3, a * S1 + b * S2) <= 1e-10


ALL_PINS = {
    "brute_force": lambda fn: all(pin_brute_force(fn, s) for s in range(2)),
    "linear_attention": pin_linear_attention,
    "forgetting": pin_forgetting,
    "retention": pin_retention,
    "directions": pin_directions,
    "state_split": pin_state_split,
    "single_token": pin_single_token,
    "linearity": pin_linearity,
}


def oracle_fn(q, k, v, g, s0, *, scale, H, W, scan):
    return oracle.gla(q, k, v, g, s0, scale=scale, H=H, W=W, scan=scan, threads=2)


# ----------------------------------------------------------------------------
# the oracle passes every pin
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", sorted(ALL_PINS))
def test_oracle_pin(name):
    assert ALL_PINS[name](oracle_fn), name


def test_scan_order_golden():
    with open(os.path.join(GOLDEN, "scan_order.txt")) as f:
        rows = [ln for ln in f if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 8
    for ln in rows:
        head, idx = ln.split(":")
        H, W, scan = head.split()
        want = np.array([int(x) for x in idx.split()])
        np.testing.assert_array_equal(oracle.scan_order(int(H), int(W), scan), want)


@pytest.mark.parametrize("H,W", [(1, 1), (1, 7), (7, 1), (7, 9), (40, 40), (16, 5)])
def test_scan_order_properties(H, W):
    L = H * W
    row = oracle.scan_order(H, W, "row")
    col = oracle.scan_order(H, W, "col")
    np.testing.assert_array_equal(row, np.arange(L))
    for scan in oracle.SCAN_IDS:
        o = oracle.scan_order(H, W, scan)
        np.testing.assert_array_equal(np.sort(o), np.arange(L))  # a bijection
    # column-major order is the row-major order of the transposed grid
    np.testing.assert_array_equal(col, np.arange(L).reshape(H, W).T.reshape(-1))
    np.testing.assert_array_equal(oracle.scan_order(H, W, "row_rev"), row[::-1])
    np.testing.assert_array_equal(oracle.scan_order(H, W, "col_rev"), col[::-1])


@pytest.mark.parametrize("scan", sorted(oracle.SCAN_IDS))
def test_permute_roundtrip(scan):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, 7 * 9, 5))
    y = oracle.permute(x, 7, 9, scan)
    np.testing.assert_array_equal(oracle.permute(y, 7, 9, scan, inverse=True), x)
    order = oracle.scan_order(7, 9, scan)
    for s in (0, 11, 62):
        np.testing.assert_array_equal(y[:, :, s], x[:, :, order[s]])


def test_oracle_threads_do_not_change_results():
    rng = np.random.default_rng(5)
    q, k, v, g, s0 = rand_inputs(rng, 7, 40, 8, 8, -0.5, 0.0)
    o1, S1 = oracle.gla(q, k, v, g, s0, scale=0.2, H=5, W=8, scan="col", threads=1)
    o4, S4 = oracle.gla(q, k, v, g, s0, scale=0.2, H=5, W=8, scan="col", threads=4)
    np.testing.assert_array_equal(o1, o4)
    np.testing.assert_array_equal(S1, S4)


# ----------------------------------------------------------------------------
# the pins have power: planted mistakes are caught
# ----------------------------------------------------------------------------

def py_recurrence(q, k, v, g, s0, *, scale, H, W, scan, mistake=None):
    """A Python copy of the recurrence in which one mistake can be planted."""
    order = oracle.scan_order(H, W, scan)
    B, BH, L, dk = q.shape
    dv = v.shape[-1]
    o = np.zeros((B, BH, L, dv))
    Sf = np.zeros((B, BH, dk, dv))
    for b in range(BH):
        S = np.zeros((dk, dv)) if (s0 is None or mistake == "drop_s0") else s0[0, b].copy()
        for s in range(L):
            t = order[s]
            qt, kt, vt, gt = q[0, b, t], k[0, b, t], v[0, b, t], g[0, b, t]
            if mistake == "swap_qk":
                qt, kt = kt, qt
            gam = np.exp(-gt) if mistake == "neg_exp" else np.exp(gt)
            if mistake == "gate_after_add":
                S = gam[:, None] * (S + np.outer(kt, vt))
            elif mistake == "previous_gate":
                gp = np.exp(g[0, b, order[s - 1]]) if s > 0 else np.ones(dk)
                S = gp[:, None] * S + np.outer(kt, vt)
            else:
                S = gam[:, None] * S + np.outer(kt, vt)
            o[0, b, t] = (1.0 if mistake == "drop_scale" else scale) * (qt @ S)
        Sf[0, b] = S
    return o, Sf


@pytest.mark.parametrize("mistake", ["gate_after_add", "neg_exp", "swap_qk", "drop_s0",
                                     "drop_scale", "previous_gate"])
def test_pins_reject_planted_mistakes(mistake):
    fn = lambda *a, **kw: py_recurrence(*a, mistake=mistake, **kw)
    failed = [n for n, pin in ALL_PINS.items() if not pin(fn)]
    assert failed, f"no pin caught the planted mistake {mistake!r}"


def test_py_recurrence_without_mistake_passes_pins():
    # guards the mutation test itself: the unmutated copy passes every pin
    fn = lambda *a, **kw: py_recurrence(*a, **kw)
    assert all(pin(fn) for pin in ALL_PINS.values())


# ---------------------------------------------------------------------------
# gate fusion: g = log gamma for gamma = sigmoid(a)^(1/tau) (Sec. 3.1)
# ---------------------------------------------------------------------------

def test_log_decay_from_logits_matches_the_power_form():
    from scipy.special import expit
    a = np.random.default_rng(11).normal(0.0, 4.0, size=1000)
    for tau in (1.0, 16.0):
        g = oracle.log_decay_from_logits(a, tau)
        # gamma written as the paper's power of a sigmoid, evaluated independently
        np.testing.assert_allclose(np.exp(g), expit(a) ** (1.0 / tau), rtol=1e-13)
        assert np.all(g < 0)


def test_log_decay_from_logits_special_values():
    g = oracle.log_decay_from_logits(np.array([0.0, -60.0, 60.0]), 16.0)
    assert g[0] == pytest.approx(-np.log(2.0) / 16.0, rel=1e-15)
    assert g[1] == pytest.approx(-60.0 / 16.0, rel=1e-15)           # log sigmoid(a) -> a for a -> -inf
    assert g[2] == pytest.approx(-np.exp(-60.0) / 16.0, rel=1e-12)  # -> -e^-a for a -> +inf, not 0


# ---------------------------------------------------------------------------
# output gate: u = SiLU(x W_r) * RMSNorm(o) (Sec. 3.1)
# ---------------------------------------------------------------------------

def epilogue_pins(fn):
    """Each returns True when ``fn(o, z, weight, eps)`` behaves as the definition."""
    from scipy.special import expit
    rng = np.random.default_rng(12)
    o = rng.normal(size=(3, 5, 64)) * rng.uniform(0.1, 10.0, size=(3, 5, 1))
    z = rng.normal(size=(3, 5, 64)) * 3.0
    w = rng.uniform(0.5, 2.0, size=64)
    u = fn(o, z, None, 0.0)
    pins = []
    # SiLU of the gate: u / (o / rms) is z * sigmoid(z), checked against scipy
    rms = np.sqrt(np.mean(o * o, axis=-1, keepdims=True))
    pins.append(np.allclose(u / (o / rms), z * expit(z), rtol=1e-12))
    # RMSNorm is over the channels of one token: u / SiLU(z) has unit RMS per token
    pins.append(np.allclose(np.sqrt(np.mean((u / (z * expit(z))) ** 2, axis=-1)), 1.0, rtol=1e-12))
    # the weight scales channel j by w_j
    pins.append(np.allclose(fn(o, z, w, 0.0), u * w, rtol=1e-12))
    # epsilon enters under the root: a constant row c gives c / sqrt(c^2 + eps)
    c = np.full((1, 64), 0.5)
    zz = np.full((1, 64), 50.0)  # SiLU(50) = 50 (1 - 2e-22)
    pins.append(np.allclose(fn(c, zz, None, 0.75), 50.0 * 0.5 / np.sqrt(0.25 + 0.75), rtol=1e-12))
    # a zero output stays zero
    pins.append(np.all(fn(np.zeros((1, 64)), zz, None, 1e-5) == 0.0))
    return all(pins)


def py_output_gate(o, z, weight, eps, mistake=None):
    w = np.ones(o.shape[-1]) if weight is None else weight
    axis = -2 if mistake == "token_axis" else -1
    e = 0.0 if mistake == "drop_eps" else eps
    ms = np.mean(o * o, axis=axis, keepdims=True)
    rms = np.sqrt(ms) + e if mistake == "eps_outside" else np.sqrt(ms + e)
    gate = 1.0 / (1.0 + np.exp(-z)) if mistake == "sigmoid_only" else z / (1.0 + np.exp(z) if mistake == "sign" else 1.0 + np.exp(-z))
    return gate * (o / rms) * w


def test_output_gate_oracle_passes_its_pins():
    assert epilogue_pins(lambda o, z, w, eps: oracle.output_gate(o, z, w, eps))


@pytest.mark.parametrize("mistake", ["token_axis", "drop_eps", "eps_outside", "sigmoid_only", "sign"])
def test_output_gate_pins_reject_planted_mistakes(mistake):
    assert not epilogue_pins(lambda o, z, w, eps: py_output_gate(o, z, w, eps, mistake))


def test_output_gate_python_copy_passes_pins():
    assert epilogue_pins(lambda o, z, w, eps: py_output_gate(o, z, w, eps))


# ---------------------------------------------------------------------------
# Spatial SwiGLU (Sec. 3.1): Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o
# ---------------------------------------------------------------------------

def test_dwconv_matches_scipy_per_channel():
    from scipy.signal import correlate2d
    rng = np.random.default_rng(21)
    B, H, W, C = 2, 5, 7, 3
    v = rng.normal(size=(B, H * W, C))
    cw = rng.normal(size=(C, 3, 3))
    cb = rng.normal(size=C)
    out = oracle.dwconv3x3(v, cw, cb, H=H, W=W)
    for b in range(B):
        for c in range(C):
            want = correlate2d(v[b, :, c].reshape(H, W), cw[c], mode="same", boundary="fill", fillvalue=0) + cb[c]
            np.testing.assert_allclose(out[b, :, c].reshape(H, W), want, rtol=1e-13, atol=1e-13)


def test_dwconv_is_not_its_flip():
    # a kernel with one off-centre tap moves features in a known direction:
    # out[i, j] = v[i - 1, j + 1] for the tap at (u, w) = (0, 2)
    H, W = 4, 5
    v = np.arange(H * W, dtype=float).reshape(1, H * W, 1) + 1
    cw = np.zeros((1, 3, 3))
    cw[0, 0, 2] = 1.0
    out = oracle.dwconv3x3(v, cw, H=H, W=W).reshape(H, W)
    g = v.reshape(H, W)
    assert out[2, 1] == g[1, 2] and out[0, 1] == 0.0 and out[1, W - 1] == 0.0


def swiglu_weights(rng, d, h):
    return (rng.normal(size=(h, d)) / np.sqrt(d), rng.normal(size=(h, d)) / np.sqrt(d),
            rng.normal(size=(d, h)) / np.sqrt(h), rng.normal(size=(h, 3, 3)) / 3.0, rng.normal(size=h) * 0.1)


def test_spatial_swiglu_with_identity_conv_is_plain_swiglu():
    from scipy.special import expit
    rng = np.random.default_rng(22)
    B, H, W, d, h = 1, 3, 4, 8, 16
    x = rng.normal(size=(B, H * W, d))
    wg, wv, wo, _, _ = swiglu_weights(rng, d, h)
    ident = np.zeros((h, 3, 3))
    ident[:, 1, 1] = 1.0
    y = oracle.spatial_swiglu(x, wg, wv, wo, ident, None, H=H, W=W)
    # the textbook SwiGLU, token by token with explicit sums
    want = np.zeros_like(y)
    for t in range(H * W):
        gt = np.array([sum(x[0, t, k] * wg[j, k] for k in range(d)) for j in range(h)])
        vt = np.array([sum(x[0, t, k] * wv[j, k] for k in range(d)) for j in range(h)])
        ht = gt * expit(gt) * vt
        want[0, t] = [sum(ht[j] * wo[i, j] for j in range(h)) for i in range(d)]
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-12)


def test_spatial_swiglu_transposes_with_the_grid():
    # transposing the grid (and each 3x3 kernel) transposes the output tokens
    rng = np.random.default_rng(23)
    B, H, W, d, h = 2, 3, 5, 8, 8
    x = rng.normal(size=(B, H * W, d))
    wg, wv, wo, cw, cb = swiglu_weights(rng, d, h)
    y = oracle.spatial_swiglu(x, wg, wv, wo, cw, cb, H=H, W=W)
    xt = x.reshape(B, H, W, d).transpose(0, 2, 1, 3).reshape(B, H * W, d)
    yt = oracle.spatial_swiglu(xt, wg, wv, wo, cw.transpose(0, 2, 1), cb, H=W, W=H)
    np.testing.assert_allclose(yt, y.reshape(B, H, W, d).transpose(0, 2, 1, 3).reshape(B, H * W, d), rtol=1e-12,
                               atol=1e-12)


def test_spatial_swiglu_is_local():
    # changing one token changes outputs only within its 3x3 neighbourhood
    rng = np.random.default_rng(24)
    B, H, W, d, h = 1, 6, 6, 8, 8
    x = rng.normal(size=(B, H * W, d))
    wg, wv, wo, cw, cb = swiglu_weights(rng, d, h)
    y0 = oracle.spatial_swiglu(x, wg, wv, wo, cw, cb, H=H, W=W)
    x2 = x.copy()
    x2[0, 2 * W + 3] += 1.0
    diff = np.abs(oracle.spatial_swiglu(x2, wg, wv, wo, cw, cb, H=H, W=W) - y0).max(axis=-1).reshape(H, W)
    changed = np.argwhere(diff > 0)
    assert changed.min(axis=0).tolist() == [1, 2] and changed.max(axis=0).tolist() == [3, 4]


def swiglu_by_loops(x, wg, wv, wo, cw, cb, H, W):
    """Eq. spatial_swiglu written out token by token with scalar loops: the value
    branch X W_v is convolved over the 3 x 3 neighbourhood (zero outside the grid),
    then gated by SiLU of the token's own X W_g, then mapped by W_o."""
    import math
    B, L, d = x.shape
    h = wg.shape[0]
    y = np.zeros((B, L, d))
    for b in range(B):
        val = [[sum(x[b, t, k] * wv[c, k] for k in range(d)) for c in range(h)] for t in range(L)]
        for i in range(H):
            for j in range(W):
                t = i * W + j
                hid = []
                for c in range(h):
                    conv = cb[c] if cb is not None else 0.0
                    for u in range(3):
                        for w_ in range(3):
                            ii, jj = i + u - 1, j + w_ - 1
                            if 0 <= ii < H and 0 <= jj < W:
                                conv += val[ii * W + jj][c] * cw[c, u, w_]
                    gate = sum(x[b, t, k] * wg[c, k] for k in range(d))
                    hid.append(gate / (1.0 + math.exp(-gate)) * conv)
                for o_ in range(d):
                    y[b, t, o_] = sum(hid[c] * wo[o_, c] for c in range(h))
    return y


def swiglu_composition_pin(fn):
    """True when ``fn`` (the oracle's signature) agrees with the scalar loops on a
    3 x 4 grid with a non-identity 3 x 3 kernel per channel."""
    rng = np.random.default_rng(25)
    B, H, W, d, h = 1, 3, 4, 2, 3
    x = rng.normal(size=(B, H * W, d))
    wg, wv, wo = rng.normal(size=(h, d)), rng.normal(size=(h, d)), rng.normal(size=(d, h))
    cw = rng.normal(size=(h, 3, 3))  # every tap nonzero, no symmetry
    cb = rng.normal(size=h)
    want = swiglu_by_loops(x, wg, wv, wo, cw, cb, H, W)
    got = fn(x, wg, wv, wo, cw, cb, H=H, W=W)
    return np.allclose(got, want, rtol=1e-12, atol=1e-12)


def py_spatial_swiglu(x, wg, wv, wo, cw, cb, *, H, W, mistake=None):
    """A copy of the composition in which one mistake can be planted (the
    depthwise convolution itself is the pinned oracle routine)."""
    g = x @ wg.T
    v = x @ wv.T
    silu = lambda a: a / (1.0 + np.exp(-a))
    if mistake == "conv_on_gate":
        hid = silu(oracle.dwconv3x3(g, cw, cb, H=H, W=W)) * v
    elif mistake == "conv_after_gating":
        hid = oracle.dwconv3x3(silu(g) * v, cw, cb, H=H, W=W)
    elif mistake == "no_bias":
        hid = silu(g) * oracle.dwconv3x3(v, cw, None, H=H, W=W)
    else:
        hid = silu(g) * oracle.dwconv3x3(v, cw, cb, H=H, W=W)
    return hid @ wo.T


def test_spatial_swiglu_composition_matches_scalar_loops():
    assert swiglu_composition_pin(oracle.spatial_swiglu)


def test_spatial_swiglu_python_copy_passes_the_composition_pin():
    assert swiglu_composition_pin(lambda *a, **kw: py_spatial_swiglu(*a, **kw))


@pytest.mark.parametrize("mistake", ["conv_on_gate", "conv_after_gating", "no_bias"])
def test_spatial_swiglu_composition_pin_rejects_planted_mistakes(mistake):
    assert not swiglu_composition_pin(lambda *a, **kw: py_spatial_swiglu(*a, mistake=mistake, **kw))


# ---------------------------------------------------------------------------
# One GTR block (Sec. 3.1): layer normalisation and the block's composition
# ---------------------------------------------------------------------------
def layer_norm_pins(fn) -> bool:
    """True when ``fn(x, w, b, eps)`` behaves as a layer normalisation over the last axis."""
    rng = np.random.default_rng(21)
    x = rng.normal(size=(4, 6, 48)) * rng.uniform(0.1, 10.0, size=(4, 6, 1)) + rng.normal(size=(4, 6, 1)) * 5
    w = rng.uniform(0.5, 2.0, size=48)
    b = rng.normal(size=48)
    y = fn(x, None, None, 0.0)
    pins = [
        np.allclose(y.mean(axis=-1), 0.0, atol=1e-12),                        # zero mean per row
        np.allclose((y * y).mean(axis=-1), 1.0, rtol=1e-12),                  # unit (biased) variance per row
        np.allclose(fn(x, w, b, 0.0), y * w + b, rtol=1e-12, atol=1e-12),    # affine per channel
        np.allclose(fn(x * 3.0 + 7.0, None, None, 0.0), y, rtol=1e-10, atol=1e-10),  # shift / scale invariant
    ]
    # epsilon under the root: the row (-1, 1, -1, 1, ...) has variance 1 -> 1 / sqrt(1 + eps)
    alt = np.tile([-1.0, 1.0], 24)[None]
    pins.append(np.allclose(fn(alt, None, None, 3.0), alt / 2.0, rtol=1e-12))
    # a constant row maps to the bias
    pins.append(np.allclose(fn(np.full((1, 48), 4.0), w, b, 1e-6), b, rtol=1e-12))
    return all(pins)


def py_layer_norm(x, w, b, eps, mistake=None):
    w = np.ones(x.shape[-1]) if w is None else w
    b = np.zeros(x.shape[-1]) if b is None else b
    axis = -2 if mistake == "axis" else -1
    mean = 0.0 if mistake == "no_center" else np.mean(x, axis=axis, keepdims=True)
    var = np.var(x, axis=axis, keepdims=True, ddof=1 if mistake == "unbiased" else 0)
    den = np.sqrt(var) + eps if mistake == "eps_outside" else np.sqrt(var + eps)
    return (x - mean) / den * w + b


def test_layer_norm_oracle_passes_its_pins():
    assert layer_norm_pins(lambda x, w, b, eps: oracle.layer_norm(x, w, b, eps))


@pytest.mark.parametrize("mistake", ["axis", "no_center", "unbiased", "eps_outside"])
def test_layer_norm_pins_reject_planted_mistakes(mistake):
    assert not layer_norm_pins(lambda x, w, b, eps: py_layer_norm(x, w, b, eps, mistake))


def test_layer_norm_python_copy_passes_pins():
    assert layer_norm_pins(lambda x, w, b, eps: py_layer_norm(x, w, b, eps))


def _small_block(seed=5):
    """A GTR block at d = 16, 2 heads, hidden 64 on a 4 x 5 grid, float64 weights."""
    rng = np.random.default_rng(seed)
    d, heads, hidden, r = 16, 2, 64, 4
    n = lambda *s, std=1.0, mu=0.0: mu + std * rng.normal(size=s)
    p = {"ln1_w": n(d, std=0.1, mu=1.0), "ln1_b": n(d, std=0.1), "w_qkvr": n(4 * d, d, std=d ** -0.5),
         "w_a1": n(r, d, std=d ** -0.5), "w_a2": n(d, r, std=r ** -0.5), "b_a": n(d, mu=2.0, std=0.5),
         "norm_w": n(d // heads, mu=1.0, std=0.1), "w_o": n(d, d, std=d ** -0.5), "ln2_w": n(d, std=0.1, mu=1.0),
         "ln2_b": n(d, std=0.1), "w_g": n(hidden, d, std=d ** -0.5), "w_v": n(hidden, d, std=d ** -0.5),
         "w_out": n(d, hidden, std=hidden ** -0.5), "conv_w": n(hidden, 3, 3, std=1 / 3), "conv_b": n(hidden, std=0.1)}
    return n(2, 20, d), p, heads


@pytest.mark.parametrize("scan", ["row", "col_rev"])
def test_block_reduces_to_its_parts(scan):
    """Pins of the composition: with W_o = 0 and the Spatial SwiGLU's W_out = 0
    the block is the identity; with W_out = 0 alone it is x + the token mixer,
    which matches per-head scalar loops over the recurrence (gate from the
    logits, output gate); with zero query weights the mixer vanishes and the
    block is x + SpatialSwiGLU(LN2(x))."""
    x, p, heads = _small_block()
    H, W = 4, 5
    q = dict(p, w_o=np.zeros_like(p["w_o"]), w_out=np.zeros_like(p["w_out"]))
    assert np.array_equal(oracle.gtr_block(x, q, H=H, W=W, heads=heads, scan=scan), x)
    # the mixer by scalar loops, in scan order
    q = dict(p, w_out=np.zeros_like(p["w_out"]))
    got = oracle.gtr_block(x, q, H=H, W=W, heads=heads, scan=scan) - x
    d = x.shape[-1]
    dh = d // heads
    n1 = oracle.layer_norm(x, p["ln1_w"], p["ln1_b"], 1e-6)
    proj = n1 @ p["w_qkvr"].T
    a = n1 @ p["w_a1"].T @ p["w_a2"].T + p["b_a"]
    order = oracle.scan_order(H, W, scan)
    u = np.zeros_like(x)
    for bb in range(x.shape[0]):
        for h in range(heads):
            cols = slice(h * dh, (h + 1) * dh)
            S = np.zeros((dh, dh))
            for t in order:
                qt, kt, vt = proj[bb, t, cols], proj[bb, t, d:2 * d][cols], proj[bb, t, 2 * d:3 * d][cols]
                zt = proj[bb, t, 3 * d:][cols]
                gam = (1.0 / (1.0 + np.exp(-a[bb, t, cols]))) ** (1.0 / 16.0)
                S = gam[:, None] * S + np.outer(kt, vt)
                o = dh ** -0.5 * qt @ S
                rms = np.sqrt(np.mean(o * o) + 1e-5)
                u[bb, t, cols] = zt / (1.0 + np.exp(-zt)) * o / rms * p["norm_w"]
    assert np.allclose(got, u @ p["w_o"].T, rtol=1e-10, atol=1e-12)
    # zero query weights: the GLA output, hence the gated output, is zero
    wq = p["w_qkvr"].copy()
    wq[:d] = 0.0
    q = dict(p, w_qkvr=wq)
    want = x + oracle.spatial_swiglu(oracle.layer_norm(x, p["ln2_w"], p["ln2_b"], 1e-6), p["w_g"], p["w_v"],
                                     p["w_out"], p["conv_w"], p["conv_b"], H=H, W=W)
    assert np.allclose(oracle.gtr_block(x, q, H=H, W=W, heads=heads, scan=scan), want, rtol=1e-12, atol=1e-12)
