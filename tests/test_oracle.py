"""Pins of the CPU oracle against what the paper and mathematics fix.

Nothing here compares the oracle with itself: worked examples derived by hand
(tests/golden/worked_examples.json), brute-force pure-Python evaluation of the
definitions on tiny inputs (own fp32 / bf16 emulation through ``struct`` and
``math``), closed forms and invariants, and the LPT scheduling bound.
"""

import json
import math
import os
import struct

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import workloads as W

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))

# ---------------------------------------------------------------------------
# independent scalar helpers (pure Python)
# ---------------------------------------------------------------------------


def f32(x: float) -> float:
    """Round a Python float to the nearest fp32 value (ties to even)."""
    return struct.unpack("f", struct.pack("f", x))[0]


def bf16_round(x: float) -> float:
    if x == 0 or math.isinf(x):
        return x
    _, e = math.frexp(x)
    sp = 2.0 ** max(e - 8, -133)
    return round(x / sp) * sp          # round() is half-to-even


def f16_round(x: float) -> float:
    return struct.unpack("e", struct.pack("e", x))[0]


def bits_to_float_bf16(b: int) -> float:
    return struct.unpack("f", struct.pack("I", (int(b) & 0xFFFF) << 16))[0]


def py_act_quant(row, qmax):
    amax = max(abs(v) for v in row)
    if amax == 0:
        return [0] * len(row), 0.0
    inv = f32(qmax / amax)
    s = f32(amax / qmax)
    codes = [max(-qmax, min(qmax, round(f32(v * inv)))) for v in row]
    return codes, s


E2M1 = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def py_e2m1(code):
    v = E2M1[code & 7]
    return -v if code & 8 else v


def py_mx_quant(vals):
    """Brute-force MXFP4 encoding of one 32-block of Python floats: the
    exponent from frexp, then the grid value nearest to each scaled element
    (ties: the one with an even code), clamped to 6."""
    amax = max(abs(v) for v in vals)
    e = -127 if amax == 0 else max(-127, min(127, math.frexp(amax)[1] - 1 - 2))
    codes = []
    for v in vals:
        x = abs(v) / 2.0 ** e
        best = None
        for c, g in enumerate(E2M1):
            key = (abs(x - g), c % 2)          # nearer first, then the even code
            if best is None or key < best[0]:
                best = (key, c)
        c = 7 if x > 6 else best[1]
        codes.append(c | 8 if (v < 0 and c) else c)
    return codes, e


def py_e4m3(code):
    """Value of an OCP FP8 e4m3 byte from its bit fields (sign, 4-bit exponent
    of bias 7, 3-bit mantissa; exponent field 0 is subnormal)."""
    sgn = -1.0 if code & 0x80 else 1.0
    e, m = (code >> 3) & 15, code & 7
    assert not (e == 15 and m == 7), "NaN code"
    return sgn * (m / 8.0 * 2.0 ** -6 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7))


E4M3_GRID = sorted({py_e4m3(c) for c in range(127)})


def py_e4m3_encode(x):
    """Nearest e4m3 byte to the Python float x by scanning all 127 magnitudes
    (ties: the even code; beyond 448: 448); sign kept unless the magnitude is 0."""
    best = None
    for c in range(127):
        key = (abs(abs(x) - py_e4m3(c)), c % 2)
        if best is None or key < best[0]:
            best = (key, c)
    c = 126 if abs(x) >= 448 else best[1]
    return c | 0x80 if (x < 0 and c) else c


def py_fp8_quant(row):
    amax = max(abs(v) for v in row)
    if amax == 0:
        return [0] * len(row), 0.0
    inv = f32(448.0 / amax)
    s = f32(amax / 448.0)
    return [py_e4m3_encode(f32(v * inv)) for v in row], s


def py_weight(lin, act, n, c):
    s = lin.scheme
    if getattr(s, "fmt", 0) == 1:
        return py_e2m1(int(lin.codes[n, c])) * 2.0 ** (int(lin.scales[n, c // 32]) - 127)
    if getattr(s, "fmt", 0) == 2:
        return py_e4m3(int(lin.codes[n, c])) * float(lin.scales[n])
    if s.w_bits == 16:
        w = bits_to_float_bf16(lin.codes[n, c])
        return f16_round(w) if act == "fp16" else w
    if s.a_bits == 16:
        g = c // s.w_group
        return float(lin.scales[n, g]) * (int(lin.codes[n, c]) - float(lin.zeros[n, g]))
    if s.w_group > 0:
        return float(lin.scales[n, c // s.w_group]) * int(lin.codes[n, c])
    return float(lin.scales[n]) * int(lin.codes[n, c])


def py_linear(a_row, lin, act):
    s = lin.scheme
    if getattr(s, "fmt", 0) == 1:
        a_hat = []
        for b in range(lin.k // 32):
            codes, e = py_mx_quant([float(f32(v)) for v in a_row[32 * b: 32 * b + 32]])
            a_hat += [py_e2m1(cd) * 2.0 ** e for cd in codes]
        return [sum(a_hat[c] * py_weight(lin, act, n, c) for c in range(lin.k)) for n in range(lin.n)]
    if getattr(s, "fmt", 0) == 2:
        qa, sa = py_fp8_quant([float(f32(v)) for v in a_row])
        av = [py_e4m3(cd) for cd in qa]
        return [sum(av[c] * py_e4m3(int(lin.codes[n, c])) for c in range(lin.k)) * sa * float(lin.scales[n])
                for n in range(lin.n)]
    if s.a_bits < 16 and s.a_group > 0:
        # per 128-wide block: integer dot of the block's codes, times both block scales
        g, qmax = s.a_group, (1 << (s.a_bits - 1)) - 1
        out = [0.0] * lin.n
        for b in range(lin.k // g):
            qa, sa = py_act_quant(a_row[b * g:(b + 1) * g], qmax)
            for n in range(lin.n):
                acc = sum(qa[c] * int(lin.codes[n, b * g + c]) for c in range(g))
                out[n] += acc * sa * float(lin.scales[n, b])
        return out
    if s.a_bits < 16:
        qa, sa = py_act_quant(a_row, (1 << (s.a_bits - 1)) - 1)
        out = []
        for n in range(lin.n):
            acc = sum(qa[c] * int(lin.codes[n, c]) for c in range(lin.k))
            out.append(acc * sa * float(lin.scales[n]))
        return out
    return [sum(a_row[c] * py_weight(lin, act, n, c) for c in range(lin.k)) for n in range(lin.n)]


def py_round_act(x, act):
    return f16_round(x) if act == "fp16" else bf16_round(x)


def py_expert(a_row, lins, act):
    g = py_linear(a_row, lins[0], act)
    u = py_linear(a_row, lins[1], act)
    h = [py_round_act(gi / (1.0 + math.exp(-gi)) * ui, act) for gi, ui in zip(g, u)]
    return py_linear(h, lins[2], act)


def py_moe(block):
    cfg = block.cfg
    x = O.act_values(block.x, cfg.act)
    T, H = x.shape
    y = np.zeros((T, H))
    for t in range(T):
        row = [float(v) for v in x[t]]
        for s in range(cfg.k):
            e = int(block.topk_ids[t, s])
            if not (0 <= e < cfg.E):
                continue
            d = py_expert(row, block.linears[e], cfg.act)
            for h in range(H):
                y[t, h] += float(block.topk_w[t, s]) * d[h]
        for j in range(cfg.n_shared):
            d = py_expert(row, block.linears[cfg.E + j], cfg.act)
            for h in range(H):
                y[t, h] += d[h]
    return y


def _lin(scheme, codes, scales=None, zeros=None):
    codes = np.asarray(codes)
    return W.QLinear(scheme, codes.shape[0], codes.shape[1], codes, scales, zeros)

# ---------------------------------------------------------------------------
# worked examples
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("case", GOLDEN["act_quant"]["cases"])
def test_act_quant_worked(case):
    codes, s = O.act_quant(np.array([case["row"]], np.float32), case["qmax"])
    assert codes[0].tolist() == case["codes"]
    assert float(s[0]) == case["scale"]


def test_dequant_g128_worked():
    g = GOLDEN["dequant_g128"]
    codes = np.full((1, 128), g["fill_code"], np.uint8)
    codes[0, :3] = g["codes_first3"]
    lin = _lin(W.W4G128, codes, np.array([[g["scale"]]], np.float16), np.array([[g["zero"]]], np.float16))
    w = O.dequant(lin, "bf16")
    assert w[0, :3].tolist() == g["values_first3"]
    assert np.all(w[0, 3:] == g["fill_value"])


def test_linear_w8a8_worked():
    g = GOLDEN["linear_w8a8"]
    lin = _lin(W.W8A8, np.array([g["w_codes"]], np.int8), np.array([g["w_scale"]], np.float32))
    a = np.array([g["a"]])
    assert int(O.linear(a, lin, "bf16", return_int=True)[0, 0]) == g["acc"]
    assert float(O.linear(a, lin, "bf16")[0, 0]) == g["out"]


def test_moe_w16_worked():
    g = GOLDEN["moe_w16"]
    bf = lambda m: W.f32_to_bf16_bits(np.array(m, np.float32))
    zero = [_lin(W.W16, bf([[0.0, 0.0]])), _lin(W.W16, bf([[0.0, 0.0]])), _lin(W.W16, bf([[0.0], [0.0]]))]
    one = [_lin(W.W16, bf(g["w_gate"])), _lin(W.W16, bf(g["w_up"])), _lin(W.W16, bf(g["w_down"]))]
    x = bf([g["x"]])
    out = O.moe_forward(x, np.array([[g["topk_id"]]], np.int32), np.array([[g["topk_w"]]], np.float32),
                        [zero, one], 2, "bf16", return_h=True)
    assert out["h"][1][0, 0] == g["h"]
    assert out["y"][0].tolist() == g["y"]

# ---------------------------------------------------------------------------
# routing: brute force and invariants
# ---------------------------------------------------------------------------


def _py_route(ids, E):
    flat = [int(v) for v in np.asarray(ids).ravel()]
    sorted_pair, counts = [], [0] * E
    for e in range(E):
        for p, v in enumerate(flat):
            if v == e:
                sorted_pair.append(p)
                counts[e] += 1
    return counts, sorted_pair


@pytest.mark.parametrize("T,k,E,seed", [(1, 1, 1, 0), (7, 3, 5, 1), (33, 2, 4, 2), (64, 4, 4, 3),
                                         (100, 6, 64, 4), (0, 2, 3, 5), (50, 8, 8, 6)])
def test_route_brute_force(T, k, E, seed):
    rng = np.random.default_rng(seed)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]) if T else np.zeros((0, k), np.int64)
    r = O.route(ids, E)
    counts, sp = _py_route(ids, E)
    assert r["counts"].tolist() == counts
    assert r["sorted_pair"].tolist() == sp
    assert int(r["offsets"][-1]) == T * k == sum(counts)
    assert np.all(r["inv"][r["sorted_pair"]] == np.arange(T * k))
    assert sorted(r["sorted_pair"].tolist()) == list(range(T * k))


def test_route_special_cases():
    T, k = 9, 3
    # E = 1 with k = 1: identity order
    r = O.route(np.zeros((T, 1), np.int32), 1)
    assert r["sorted_pair"].tolist() == list(range(T))
    # k = E: every expert gets every token, in token order
    ids = np.array([np.random.default_rng(t).permutation(k) for t in range(T)])
    r = O.route(ids, k)
    assert r["counts"].tolist() == [T] * k
    for e in range(k):
        toks = r["sorted_pair"][r["offsets"][e]:r["offsets"][e + 1]] // k
        assert toks.tolist() == list(range(T))


def test_route_bad_ids_dropped():
    ids = np.array([[0, 5], [-1, 1], [2, 1]], np.int32)
    r = O.route(ids, 3)
    assert r["bad"].tolist() == [False, True, True, False, False, False]
    assert r["sorted_pair"].tolist() == [0, 3, 5, 4]
    assert r["inv"].tolist() == [0, -1, -1, 1, 3, 2]

# ---------------------------------------------------------------------------
# quantization: dequant against the original weights, act-quant properties
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("scheme", [W.W2G128, W.W3G128, W.W4G128, W.W8G128, W.W8A8, W.W4A4, W.W4A4G128])
def test_dequant_recovers_weights(scheme):
    w = W.draw_weight(11, 0, 0, 48, 384)
    lin = W.quantize_linear(w, scheme)
    deq = O.dequant(lin, "bf16")
    if scheme.a_bits == 16:
        s = np.repeat(lin.scales.astype(np.float64), 128, axis=1)
        qmax = (1 << scheme.w_bits) - 1
        inner = (lin.codes > 0) & (lin.codes < qmax)
        err = np.abs(deq - w.astype(np.float64))
        assert np.all(err[inner] <= 0.5 * s[inner] * (1 + 1e-12))
        # clamped codes sit at the ends of the range: error bounded by one step
        assert np.all(err <= 1.0 * s + 1e-12)
        assert inner.mean() > 0.5 if scheme.w_bits > 2 else True
    elif scheme.w_group > 0:
        # symmetric groups with an fp16 scale: the scale rounding can push the
        # group maximum just past qmax * s, where the clamp adds at most
        # qmax * |s - amax/qmax| <= qmax * 2^-11 * s
        qmax = (1 << (scheme.w_bits - 1)) - 1
        s = np.repeat(lin.scales.astype(np.float64), scheme.w_group, axis=1)
        assert np.all(np.abs(deq - w) <= (0.5 + qmax * 2.0 ** -11) * s * (1 + 1e-12))
        groups = np.abs(lin.codes.astype(np.int64)).reshape(lin.n, -1, scheme.w_group).max(axis=2)
        assert np.all(groups == qmax)
    else:
        s = lin.scales.astype(np.float64)[:, None]
        assert np.all(np.abs(deq - w) <= 0.5 * s * (1 + 1e-12))
        qmax = (1 << (scheme.w_bits - 1)) - 1
        assert np.all(np.abs(lin.codes).max(axis=1) == qmax)


def test_mxfp4_quantizer_pins():
    """OCP MX FP4: values on the e2m1 grid times a power of two; the error of
    an element is at most a quarter of max(|x|, 1) in units of its block scale
    (half the grid spacing in every binade, 2 at most above 6); a block of
    equal values encodes exactly; doubling the input adds one to every scale
    and keeps every code; brute force on a few blocks."""
    w = W.draw_weight(12, 0, 0, 48, 384)
    lin = W.quantize_linear(w, W.MXFP4)
    deq = O.dequant(lin, "bf16")
    sc = np.exp2(np.repeat(lin.scales.astype(np.float64) - 127, 32, axis=1))
    x = np.abs(w.astype(np.float64)) / sc
    assert np.all(np.abs(deq - w) <= 0.25 * np.maximum(x, 1.0) * sc * (1 + 1e-12))
    assert np.all(np.isin(np.abs(deq) / sc, O._E2M1))
    # every block reaches a code of 4 or 6 (its maximum lies in [4, 8) scaled)
    mags = (lin.codes & 7).reshape(48, -1, 32).max(axis=2)
    assert np.all(mags >= 6)
    # activations: the oracle's encoder on equal, doubled and brute-forced rows
    a = np.full((1, 64), 1.0, np.float32)
    q, e = O.mx_quant(a)
    assert np.all(O._mx_values(q, e, 32) == 1.0)
    rng = np.random.default_rng(3)
    r = rng.standard_normal((5, 128)).astype(np.float32)
    q1, e1 = O.mx_quant(r)
    q2, e2 = O.mx_quant(r * np.float32(2))
    assert np.array_equal(q1, q2) and np.array_equal(e2.astype(int), e1.astype(int) + 1)
    for i in range(5):
        for b in range(4):
            pc, pe = py_mx_quant([float(v) for v in r[i, 32 * b: 32 * b + 32]])
            assert q1[i, 32 * b: 32 * b + 32].tolist() == pc and int(e1[i, b]) - 127 == pe
    # the weight quantizer of the input generator agrees with the oracle's encoder
    cw, ew = W.quantize_mxfp4(w)
    co, eo = O.mx_quant(w)
    assert np.array_equal(cw, co) and np.array_equal(ew, eo)


def test_fp8_e4m3_pins():
    """OCP FP8 e4m3: the oracle's table against the bit-field definition for
    every byte, anchors (1.0 = 0x38, 448 = 0x7E the largest, 2^-6 the smallest
    normal, 2^-9 the smallest subnormal), nearest-value encoding with ties to
    the even code against a scan of all magnitudes, saturation at 448, the
    round-trip of every grid value, and a relative error of at most 2^-4 in
    the normal range."""
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], np.uint8)
    assert O.e4m3_values(codes).tolist() == [py_e4m3(int(c)) for c in codes]
    anchors = {0x38: 1.0, 0x7E: 448.0, 0x08: 2.0 ** -6, 0x01: 2.0 ** -9, 0x40: 2.0, 0xB8: -1.0, 0x07: 7 * 2.0 ** -9}
    for c, v in anchors.items():
        assert O.e4m3_values(np.array([c], np.uint8))[0] == v
    with pytest.raises(ValueError):
        O.e4m3_values(np.array([0x7F], np.uint8))
    grid = np.array(E4M3_GRID)
    assert np.array_equal(O.e4m3_code(grid), np.arange(127))                 # grid values round-trip
    mids = (grid[:-1] + grid[1:]) / 2
    assert O.e4m3_code(mids).tolist() == [i if i % 2 == 0 else i + 1 for i in range(126)]  # ties to even
    rng = np.random.default_rng(5)
    x = np.concatenate([np.exp2(rng.uniform(-12, 10, 400)), [0.0, 448.0, 460.0, 1e6, 2.0 ** -10, 2.0 ** -10 * 1.0001]])
    assert O.e4m3_code(x).tolist() == [py_e4m3_encode(float(v)) for v in x]
    nrm = (x >= 2.0 ** -6) & (x <= 448)
    assert np.all(np.abs(O._E4M3[O.e4m3_code(x[nrm])] - x[nrm]) <= 2.0 ** -4 * x[nrm])


def test_fp8_quantizer_pins():
    """Per-token FP8 activations: brute force of the fp32 recipe on random rows
    (the row maximum lands on 448), an all-zero row, sign symmetry, and a
    linear whose operands are exact scaled e4m3 values reproduces the plain
    product; the input generator's weight quantizer agrees with a scan of the
    grid."""
    rng = np.random.default_rng(6)
    a = (rng.standard_normal((6, 128)) * np.exp2(rng.uniform(-8, 8, (6, 1)))).astype(np.float32)
    a[3] = 0
    q, s = O.fp8_quant(a)
    for i in range(6):
        pc, ps = py_fp8_quant([float(v) for v in a[i]])
        assert q[i].tolist() == pc and float(s[i]) == ps
    nz = [i for i in range(6) if i != 3]
    assert np.all(O.e4m3_values(q[nz]).__abs__().max(axis=1) == 448.0)
    assert np.all(q[3] == 0) and s[3] == 0
    qn, sn = O.fp8_quant(-a)
    assert np.array_equal(O.e4m3_values(qn), -O.e4m3_values(q)) and np.array_equal(sn, s)
    # exact operands: activations 448 * grid / 448 and weights grid * 2^-3 per channel
    av = np.array([[1.0, -0.5, 448.0, 3.0] * 32], np.float64)
    wc = np.array([[0x38, 0xC0, 0x01, 0x7E] * 32, [0x30, 0x30, 0x30, 0x30] * 32], np.uint8)
    lin = W.QLinear(W.FP8, 2, 128, wc, np.array([0.125, 1.0], np.float32))
    exact = av @ (O.e4m3_values(wc) * np.array([[0.125], [1.0]])).T
    assert np.array_equal(O.linear(av, lin, "bf16"), exact)
    # weights: the input generator's e4m3 codes are the nearest grid values
    w = W.draw_weight(13, 0, 0, 16, 256)
    lq = W.quantize_linear(w, W.FP8)
    for n in range(0, 16, 5):
        sc = float(lq.scales[n])
        assert sc == f32(float(np.abs(w[n].astype(np.float64)).max()) / 448.0)
        assert lq.codes[n].tolist() == [py_e4m3_encode(float(v) / sc) for v in w[n].astype(np.float64)]


def test_w16_fp16_conversion():
    w = np.array([[1.0, -0.0078125, 3.0e-6, 60000.0, 1.0e-7]], np.float32)
    lin = W.quantize_linear(w, W.W16)
    assert O.dequant(lin, "bf16")[0].tolist() == [bf16_round(v) for v in w[0].tolist()]
    assert O.dequant(lin, "fp16")[0].tolist() == [f16_round(bf16_round(v)) for v in w[0].tolist()]


@pytest.mark.parametrize("qmax", [7, 127])
def test_act_quant_properties(qmax):
    rng = np.random.default_rng(qmax)
    a = rng.standard_normal((40, 300)).astype(np.float32)
    a[3] = 0
    q, s = O.act_quant(a, qmax)
    assert q.dtype == np.int8 and np.all(np.abs(q) <= qmax)
    assert s[3] == 0 and np.all(q[3] == 0)
    rows = [r for r in range(40) if r != 3]
    # the amax element maps to +-qmax
    am = np.abs(a).argmax(axis=1)
    assert np.all(np.abs(q[rows, am[rows]]) == qmax)
    # dequantization error within half a step (plus fp32 rounding)
    err = np.abs(q[rows].astype(np.float64) * s[rows, None] - a[rows])
    assert np.all(err <= 0.5 * s[rows, None] * (1 + 1e-5) + 1e-30)
    # scaling by a power of two keeps the codes and scales the step exactly
    q2, s2 = O.act_quant(a * np.float32(4.0), qmax)
    assert np.array_equal(q, q2) and np.array_equal(s2, s * np.float32(4.0))
    # brute force on a few rows
    for r in (0, 5, 17):
        pq, ps = py_act_quant([float(v) for v in a[r]], qmax)
        assert q[r].tolist() == pq and float(s[r]) == ps

# ---------------------------------------------------------------------------
# linear and block: brute force on tiny shapes
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("scheme", W.ALL_SCHEMES)
@pytest.mark.parametrize("act", ["bf16", "fp16"])
def test_linear_brute_force(scheme, act):
    m, n, k = 3, 5, 256
    lin = W.quantize_linear(W.draw_weight(3, 1, 2, n, k), scheme)
    x = W.f64_to_act(np.random.default_rng(4).standard_normal((m, k)), act)
    a = O.act_values(x, act)
    got = O.linear(a, lin, act)
    for i in range(m):
        ref = py_linear([float(v) for v in a[i]], lin, act)
        np.testing.assert_allclose(got[i], ref, rtol=1e-12, atol=1e-12)


def test_int_linear_doubling():
    lin = W.quantize_linear(W.draw_weight(5, 0, 0, 16, 256), W.W8A8)
    a = O.act_values(W.f64_to_act(np.random.default_rng(1).standard_normal((4, 256)), "bf16"), "bf16")
    assert np.array_equal(O.linear(2 * a, lin, "bf16"), 2 * O.linear(a, lin, "bf16"))
    assert np.array_equal(O.linear(2 * a, lin, "bf16", return_int=True),
                          O.linear(a, lin, "bf16", return_int=True))


def test_group_linear_blocks_add_up():
    """w4a4-g128: the linear over K = 384 is the sum of three independent
    w4a4-g128 linears over its 128-wide column blocks, each with its own slice
    of codes and scales (a misplaced block index or scale column fails this)."""
    lin = W.quantize_linear(W.draw_weight(8, 0, 1, 24, 384), W.W4A4G128)
    a = O.act_values(W.f64_to_act(np.random.default_rng(6).standard_normal((7, 384)), "bf16"), "bf16")
    whole = O.linear(a, lin, "bf16")
    parts = sum(O.linear(a[:, b * 128:(b + 1) * 128],
                         _lin(W.W4A4G128, lin.codes[:, b * 128:(b + 1) * 128], lin.scales[:, b:b + 1]), "bf16")
                for b in range(3))
    np.testing.assert_allclose(whole, parts, rtol=1e-13, atol=1e-15)
    # one block: w4a4-g128 is w4a4 per token / per channel with the fp16 scale
    one = _lin(W.W4A4G128, lin.codes[:, :128], lin.scales[:, :1])
    pc = _lin(W.W4A4, lin.codes[:, :128], lin.scales[:, 0].astype(np.float32))
    np.testing.assert_allclose(O.linear(a[:, :128], one, "bf16"), O.linear(a[:, :128], pc, "bf16"),
                               rtol=1e-13, atol=1e-15)
    # doubling the activations keeps every code and doubles every block scale
    assert np.array_equal(O.linear(2 * a, lin, "bf16"), 2 * whole)


MIXED = [(W.W4G128, W.W4G128, W.W2G128), (W.W8A8, W.W8A8, W.W4A4), (W.W16, W.W16, W.W8A8),
         (W.W3G128, W.W3G128, W.W16), (W.W4A4, W.W8G128, W.W4G128)]
MIXED_G = [(W.W4A4G128, W.W4A4G128, W.W2G128), (W.W8A8, W.W8A8, W.W4A4G128), (W.W4A4G128,) * 3,
           (W.W16, W.W16, W.W4A4G128), (W.W4A4G128, W.W4A4G128, W.W8A8)]
MIXED_MX = [(W.MXFP4,) * 3, (W.MXFP4, W.MXFP4, W.W3G128), (W.W8A8, W.W8A8, W.MXFP4), (W.W16, W.W16, W.MXFP4),
            (W.MXFP4, W.MXFP4, W.W4A4G128)]
MIXED_F8 = [(W.FP8,) * 3, (W.FP8, W.FP8, W.W2G128), (W.W8A8, W.W8A8, W.FP8), (W.W16, W.W16, W.FP8),
            (W.MXFP4, W.MXFP4, W.FP8)]


@pytest.mark.parametrize("act", ["bf16", "fp16"])
@pytest.mark.parametrize("mix,H,F", [(MIXED, 128, 128), (MIXED_G, 256, 256), (MIXED_MX, 128, 256),
                                     (MIXED_F8, 128, 128)])
def test_moe_brute_force(act, mix, H, F):
    blk = W.random_small_block(21, T=5, H=H, F=F, E=4, k=2, n_shared=1, F_shared=128, act=act,
                               schemes=mix)
    blk.topk_ids[2, 1] = 9          # an invalid expert id is skipped
    out = O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears, 4, act)
    np.testing.assert_allclose(out["y"], py_moe(blk), rtol=1e-9, atol=1e-12)


def test_moe_zero_input():
    blk = W.random_small_block(2, T=5, H=128, F=128, E=3, k=2, schemes=MIXED[:3])
    blk.x[:] = 0
    out = O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears, 3, "bf16")
    assert np.all(out["y"] == 0)


def test_moe_equivariance_and_relabel():
    blk = W.random_small_block(3, T=12, H=128, F=128, E=4, k=2, n_shared=1, F_shared=256,
                               schemes=MIXED)
    base = O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears, 4, "bf16")["y"]
    perm = np.random.default_rng(0).permutation(12)
    out = O.moe_forward(blk.x[perm], blk.topk_ids[perm], blk.topk_w[perm], blk.linears, 4, "bf16")["y"]
    assert np.array_equal(out, base[perm])
    relabel = np.array([2, 0, 3, 1])           # expert e becomes relabel[e]
    lin2 = [None] * 4
    for e in range(4):
        lin2[relabel[e]] = blk.linears[e]
    lin2 += blk.linears[4:]
    out = O.moe_forward(blk.x, relabel[blk.topk_ids].astype(np.int32), blk.topk_w, lin2, 4, "bf16")["y"]
    np.testing.assert_allclose(out, base, rtol=1e-12, atol=1e-14)


def test_uniform_bf16_is_dense_mlp():
    """E = 1, k = 1, w = 1 with 16-bit weights is a dense gated-SiLU MLP."""
    blk = W.random_small_block(4, T=7, H=128, F=24, E=1, k=1, schemes=[(W.W16, W.W16, W.W16)])
    blk.topk_w[:] = 1.0
    y = O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears, 1, "bf16")["y"]
    x = np.array([[bits_to_float_bf16(b) for b in row] for row in blk.x])
    wg, wu, wd = [np.array([[bits_to_float_bf16(b) for b in r] for r in l.codes]) for l in blk.linears[0]]
    g, u = x @ wg.T, x @ wu.T
    h = np.vectorize(bf16_round)(g * u / (1 + np.exp(-g)))
    np.testing.assert_allclose(y, h @ wd.T, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------------------
# tile scheduling: LPT against the exact optimum (Graham's bound)
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("seed", range(12))
def test_lpt_graham_bound(seed):
    rng = np.random.default_rng(seed)
    P = int(rng.integers(2, 4))
    costs = rng.integers(1, 20, size=int(rng.integers(P + 1, 9))).astype(float).tolist()
    opt = O.optimal_makespan(costs, P)
    lpt = O.lpt_makespan(costs, P)
    assert opt <= lpt <= (4.0 / 3.0 - 1.0 / (3 * P)) * opt + 1e-9
    assert opt >= max(max(costs), sum(costs) / P) - 1e-9


def test_lpt_tight_instance():
    # Graham's tight example for P = 2: {3,3,2,2,2} has OPT 6 and LPT 7 = (4/3 - 1/6) * 6
    assert O.optimal_makespan([3, 3, 2, 2, 2], 2) == 6
    assert O.lpt_makespan([3, 3, 2, 2, 2], 2) == 7


def test_runtime_model_many_tiles():
    """Sec. 4.2.2: with #tiles >> #processors, makespan ~ sum(c) / P."""
    rng = np.random.default_rng(0)
    P = 256
    errs = []
    for n in (512, 4096, 32768):
        c = rng.choice([1.0, 2.5, 7.0], size=n)
        errs.append(O.lpt_makespan(c, P) / (c.sum() / P) - 1)
    assert errs[-1] < 0.01 and errs[0] > errs[-1]


def _cost_table(which: str):
    from paper_2505_05799_amd import tile_cost as TC
    return TC.CostTable.load().device_table() if which == "profiled" else W.random_tile_costs(int(which[6:]))


def test_tile_cost_of_the_table():
    """The plan's tile cost against the profiled model it encodes: the table
    in ps prices every tile within the rounding of its coefficients (1 ps per
    term) of the continuous model c_t(K, mt) = a + K/128 (bs + bu / mt) in ns;
    a larger mt never costs more; a sliced tile pays the hand-off h once; the
    clamp holds at both ends."""
    from paper_2505_05799_amd import tile_cost as TC
    t = TC.CostTable.load()
    dev = t.device_table()
    for ph in (0, 1):
        for s in W.ALL_SCHEMES:
            i = O.scheme_index(s)
            assert W.ALL_SCHEMES[i] is s
            for c in range(4):
                e = dev[ph][i][c]
                for kb in (1, 8, 28, 160):
                    prev = None
                    for mt in (1, 2, 3, 8, 128):
                        got = O._tile_cost(e, kb, 1, mt)
                        want = t.tile_ns(ph, s, c, kb * 128, mt) * 1000.0
                        assert abs(got - min(max(want, 1.0), 2e9)) <= 2 + kb * 2, (ph, s.name, c, kb, mt)
                        assert prev is None or got <= prev
                        prev = got
                    c1, c2 = O._tile_cost(e, kb, 1, 1), O._tile_cost(e, kb, 2, 1)
                    if c1 > 1:    # (a tile priced at the lower clamp may gain less than h)
                        assert c2 - c1 == min(int(e[3]), 2 * 10**9 - c1)
                    else:
                        assert 0 <= c2 - c1 <= int(e[3])
    assert O._tile_cost((0, 0, 0, 0), 5, 1, 1) == 1
    assert O._tile_cost((2 * 10**9, 10**7, 0, 0), 500, 1, 1) == 2 * 10**9
    assert O._tile_cost((0, 0, 7, 0), 3, 1, 4) == 5        # floor(21 / 4)


@pytest.mark.parametrize("table", ["profiled", "random1", "random2"])
@pytest.mark.parametrize("nwg", [2, 64, 512])
def test_tile_plan_slices_minimal(nwg, table):
    """Slicing invariants: with an ample partial buffer a group takes the fewest
    slices whose tile cost is within the threshold, or if there are none the
    cheapest tile's slice count; a budget of zero floats slices nothing."""
    costs = _cost_table(table)
    blk = W.make_block("dsv2lite", with_weights=False)
    cfg = blk.cfg
    counts = np.bincount(blk.topk_ids.ravel(), minlength=cfg.E).tolist() + [cfg.T] * cfg.n_shared
    for phase, (n, k) in ((0, (cfg.F, cfg.H)), (1, (cfg.H, cfg.F))):
        lins = [W.QLinear(s[0 if phase == 0 else 2], n if e < cfg.E else
                          (cfg.F_shared if phase == 0 else cfg.H),
                          k if e < cfg.E else (cfg.H if phase == 0 else cfg.F_shared), None)
                for e, s in enumerate(W.schemes_of(cfg))]
        plan, _ = O.tile_plan(counts, lins, phase, costs, partial_floats=1 << 40, nwg=nwg)
        entry = lambda r, lin: costs[phase][O.scheme_index(lin.scheme)][r["cfg"]]
        work = sum(r["mtiles"] * r["ntiles"] * O._tile_cost(entry(r, lin), lin.k // 128, 1, r["mtiles"])
                   for r, lin in zip(plan, lins) if r["mtiles"] * r["ntiles"])
        theta = work // nwg // 2
        fb_groups = []
        for r, lin in zip(plan, lins):
            if r["mtiles"] * r["ntiles"] == 0:
                assert r["split"] == 1
                continue
            kb = lin.k // 128
            smax = max(1, min(8, kb // 6))
            cost = lambda sp: O._tile_cost(entry(r, lin), -(-kb // sp), sp, r["mtiles"])
            sp = r["split"]
            assert 1 <= sp <= smax
            assert r["cost"] == cost(sp)
            if cost(sp) <= theta:   # the fewest slices within the threshold
                assert sp == 1 or cost(sp - 1) > theta
            elif sp > 1:            # none within it: the cheapest tile
                assert all(cost(s) > theta for s in range(1, smax + 1))
                assert cost(sp) == min(cost(s) for s in range(1, smax + 1))
                assert all(cost(s) > cost(sp) for s in range(1, sp))
            else:                   # unsliced: S = 1 is the cheapest, or slicing would pass nwg tiles
                cheapest = min(range(1, smax + 1), key=lambda s: (cost(s), s))
                fb_groups.append((r, cheapest))
        # a fallback group left unsliced although slicing was cheaper: its added
        # tiles would have taken the phase past one tile per workgroup
        unsliced = sum(r["mtiles"] * r["ntiles"] for r in plan)
        added = 0
        for r in plan:
            if r["split"] > 1:
                added += r["mtiles"] * r["ntiles"] * (r["split"] - 1)
        refused = [r for r, cheapest in fb_groups if cheapest > 1]
        if refused:   # the first refused one would have passed nwg tiles
            r0 = refused[0]
            cheapest0 = dict((id(r), c) for r, c in fb_groups)[id(r0)]
            assert unsliced + added + r0["mtiles"] * r0["ntiles"] * (cheapest0 - 1) > nwg
        none, _ = O.tile_plan(counts, lins, phase, costs, partial_floats=0, nwg=nwg)
        assert all(r["split"] == 1 for r in none)
    # numpy int32 row counts (as routing returns them) plan like Python ints:
    # the phase's work sum exceeds 32 bits at full size
    big = [c * 64 for c in counts]
    assert O.tile_plan([np.int32(c) for c in big], lins, 1, costs, partial_floats=1 << 40)[0] == \
        O.tile_plan(big, lins, 1, costs, partial_floats=1 << 40)[0]
    # fewer workgroups -> a larger threshold -> never more slices
    a, _ = O.tile_plan(counts, lins, 1, costs, partial_floats=1 << 40, nwg=2)
    b, _ = O.tile_plan(counts, lins, 1, costs, partial_floats=1 << 40, nwg=512)
    assert all(x["split"] <= y["split"] for x, y in zip(a, b))


@pytest.mark.parametrize("table", ["profiled", "random3"])
@pytest.mark.parametrize("name", ["tiny", "dsv2lite", "qwen15_mixed", "qwen15_w5a5"])
def test_tile_plan_covers_every_output(name, table):
    blk = W.make_block(name, with_weights=False)
    cfg = blk.cfg
    counts = np.bincount(blk.topk_ids.ravel(), minlength=cfg.E).tolist() + [cfg.T] * cfg.n_shared
    for phase, (n, k) in ((0, (cfg.F, cfg.H)), (1, (cfg.H, cfg.F))):
        lins = [W.QLinear(s[0 if phase == 0 else 2], n if e < cfg.E else
                          (cfg.F_shared if phase == 0 else cfg.H),
                          k if e < cfg.E else (cfg.H if phase == 0 else cfg.F_shared), None)
                for e, s in enumerate(W.schemes_of(cfg))]
        plan, order = O.tile_plan(counts, lins, phase, _cost_table(table), partial_floats=1 << 26)
        for m, lin, r in zip(counts, lins, plan):
            bm = (16, 32, 64, 128)[r["cfg"]]
            bn = ((256, 256, 128, 128), (512, 512, 256, 256))[phase][r["cfg"]]
            assert r["mtiles"] * bm >= m > (r["mtiles"] - 1) * bm or m == r["mtiles"] == 0
            assert r["ntiles"] * bn >= lin.n > (r["ntiles"] - 1) * bn
        costs = [plan[g]["cost"] for g in order]
        assert costs == sorted(costs, reverse=True)
        assert sorted(order) == [g for g, m in enumerate(counts) if m > 0]
        # the per-XCD queues hold every tile of every group exactly once, the
        # queue totals match, and groups appear in rank order within a queue
        queues, totals = O.xcd_queues(plan, order)
        tiles = O.xcd_tiles(plan, order)
        assert [len(t) for t in tiles] == totals
        flat = [t for q in tiles for t in q]
        want = [(g, mi, ni) for g in order for mi in range(plan[g]["mtiles"])
                for ni in range(plan[g]["ntiles"] * plan[g]["split"])]
        for g, r in enumerate(plan):  # slices: at least 6 k blocks each, at most 8
            k = lins[g].k // 128
            assert 1 <= r["split"] <= 8 and (r["split"] == 1 or k // r["split"] >= 6)
        assert sorted(flat) == sorted(want) and len(flat) == len(set(flat))
        rank = {g: i for i, g in enumerate(order)}
        for q in tiles:
            ranks = [rank[g] for g, _, _ in q]
            assert ranks == sorted(ranks)


# ---------------------------------------------------------------------------
# router front-end (Eq. 2 gate weights from the router softmax)
# ---------------------------------------------------------------------------


def py_router(row, k, renorm):
    """Brute force: sort expert ids by (-logit, id), softmax with math.exp."""
    E = len(row)
    order = sorted(range(E), key=lambda e: (-row[e], e))[:k]
    m = max(row)
    ex = [math.exp(v - m) for v in row]
    den = sum(ex[e] for e in order) if renorm else sum(ex)
    return order, [ex[e] / den for e in order]


@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("T,E,k", [(5, 8, 2), (7, 60, 4), (3, 65, 8), (4, 64, 64)])
def test_router_brute_force(T, E, k, renorm):
    l, _ = W.router_logits(T, E, seed=E + k, zipf_s=1.0)
    l[0, :4] = l[0, 4]                       # ties go to the lower id
    ids, w = O.router_topk(l, k, renorm)
    for t in range(T):
        pi, pw = py_router([float(v) for v in l[t]], k, renorm)
        assert ids[t].tolist() == pi
        np.testing.assert_allclose(w[t], pw, rtol=1e-13)


def test_router_closed_forms():
    # equal logits: ids in order, weights 1/E, renormalised 1/k
    ids, w = O.router_topk(np.zeros((2, 8), np.float32), 3)
    assert ids.tolist() == [[0, 1, 2]] * 2 and np.all(w == 1 / 8)
    ids, w = O.router_topk(np.zeros((1, 8), np.float32), 3, renormalize=True)
    assert np.allclose(w, 1 / 3, rtol=1e-15)
    # [1, 3, 3, 2], k = 2: the tied 3s in id order, each e^3 / (e + 2 e^3 + e^2)
    ids, w = O.router_topk(np.array([[1, 3, 3, 2]], np.float32), 2)
    assert ids.tolist() == [[1, 2]]
    assert np.allclose(w, math.exp(3) / (math.exp(1) + 2 * math.exp(3) + math.exp(2)), rtol=1e-15)
    # k = E: a permutation sorted by logit, probabilities summing to 1
    l, _ = W.router_logits(9, 16, seed=3)
    ids, w = O.router_topk(l, 16)
    assert all(sorted(r) == list(range(16)) for r in ids.tolist())
    assert np.all(np.diff(np.take_along_axis(l, ids, axis=1), axis=1) <= 0)
    assert np.allclose(w.sum(axis=1), 1.0, rtol=1e-14)
    # a constant shift of the logits changes nothing (logits on a 2^-10 grid,
    # so the shift is exact in fp32)
    l = (np.rint(l * 1024) / 1024).astype(np.float32)
    ids, w = O.router_topk(l, 16)
    ids2, w2 = O.router_topk(l + np.float32(4.0), 16)
    assert np.array_equal(ids, ids2) and np.allclose(w, w2, rtol=1e-12)


def test_shared_gate_closed_forms():
    assert O.shared_gate(np.array([0.0], np.float32))[0] == 0.5
    x = np.linspace(-8, 8, 33).astype(np.float32)
    g = O.shared_gate(x)
    assert np.allclose(g + O.shared_gate(-x), 1.0, rtol=1e-15)
    assert np.allclose(g, [1 / (1 + math.exp(-float(v))) for v in x], rtol=1e-15)


def test_moe_shared_gate_is_linear_in_the_gate():
    blk = W.random_small_block(4, T=6, H=128, F=128, E=3, k=2, n_shared=2, F_shared=128,
                               schemes=MIXED[:3] + [MIXED[3], MIXED[4]])
    args = (blk.x, blk.topk_ids, blk.topk_w, blk.linears, 3, "bf16")
    base = O.moe_forward(*args)["y"]
    ones = O.moe_forward(*args, shared_w=np.ones((6, 2), np.float32))["y"]
    assert np.array_equal(base, ones)
    routed = O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears[:3], 3, "bf16")["y"]
    zero = O.moe_forward(*args, shared_w=np.zeros((6, 2), np.float32))["y"]
    assert np.array_equal(zero, routed)
    g = np.random.default_rng(1).random((6, 2)).astype(np.float32)
    y = O.moe_forward(*args, shared_w=g)["y"]
    s0 = O.moe_forward(*args, shared_w=np.array([[1, 0]] * 6, np.float32))["y"] - routed
    s1 = O.moe_forward(*args, shared_w=np.array([[0, 1]] * 6, np.float32))["y"] - routed
    np.testing.assert_allclose(y, routed + g[:, :1] * s0 + g[:, 1:] * s1, rtol=1e-12, atol=1e-14)
