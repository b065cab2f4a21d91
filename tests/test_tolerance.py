"""CPU pins of the error models behind the GPU parity tolerances
(tests/tolerance.py).  Each test emulates, in IEEE float32 with numpy, the
arithmetic the kernels perform in their order of operations (products exact,
one rounding per MFMA step into the fp32 accumulator, the per-group rescale
and bias removal of the weight-only kinds, split-K partial sums, the fp32
epilogue), and checks the emulated error against the bound with margin."""

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import workloads as W
from tests import tolerance as TL

f32 = np.float32


def _bf16(x):
    return W.bf16_bits_to_f32(W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32)))


def _mfma_steps(a, w, step=32):
    """fp32 accumulation of a[m, K] @ w[n, K]^T, one rounding per MFMA step of
    `step` products (the step's exact sum, then added to the accumulator)."""
    m, K = a.shape
    acc = np.zeros((m, w.shape[0]), f32)
    for j in range(0, K, step):
        blk = a[:, j:j + step].astype(np.float64) @ w[:, j:j + step].astype(np.float64).T
        acc = (acc.astype(np.float64) + blk).astype(f32)
    return acc


def _operands(kind, m, n, K, seed):
    rng = np.random.default_rng(seed)
    if kind == "positive":
        a = _bf16(np.abs(rng.standard_normal((m, K))))
        w = _bf16(np.abs(rng.standard_normal((n, K))) * 0.02)
    else:
        a = _bf16(rng.standard_normal((m, K)))
        w = _bf16(rng.standard_normal((n, K)) * 0.02)
    return a, w


@pytest.mark.parametrize("K", [256, 4096, 14336, 20480])
@pytest.mark.parametrize("kind", ["gaussian", "positive"])
def test_acc16_model_plain(K, kind):
    """16-bit MFMA GEMM (w16): emulated error <= ACC16_EPS / 4 * sum |a||w|,
    also with up to 8 split-K slices added in fp32 afterwards."""
    a, w = _operands(kind, 8, 16, K, K + len(kind))
    exact = a.astype(np.float64) @ w.astype(np.float64).T
    bound = TL.acc_bound(np.abs(a).astype(np.float64), np.abs(w).astype(np.float64))
    got = _mfma_steps(a, w).astype(np.float64)
    assert np.all(np.abs(got - exact) <= bound / 4), float((np.abs(got - exact) / bound).max())
    # split-K: slices accumulate separately, then are added in slice order
    S = 8 if K >= 8 * 768 else 2
    cut = np.linspace(0, K // 128, S + 1).astype(int) * 128
    parts = [_mfma_steps(a[:, cut[i]:cut[i + 1]], w[:, cut[i]:cut[i + 1]]) for i in range(S)]
    tot = parts[0]
    for p in parts[1:]:
        tot = (tot + p).astype(f32)
    assert np.all(np.abs(tot.astype(np.float64) - exact) <= bound / 4)


def _magic_gemm(a, q, act, rng):
    """The weight-only kernel's arithmetic on bf16 activations: per 128-group g
    the running sum is moved into units of s_g (times s_{g-1} * rcp(s_g), the
    reciprocal within one ulp), the bias c * rowsum_g(a) is removed with one
    FMA, then the MFMA steps add a * (c + q - z); the output is s_last * Q.
    fp16 activations: the operand is q - z itself (no bias)."""
    s = q.scales.astype(f32)
    z = q.zeros.astype(f32)
    b = (1 << q.scheme.w_bits) - 1
    c = f32(128 + b) if act == "bf16" else f32(0)
    m, K = a.shape
    n = q.n
    Q = np.zeros((m, n), f32)
    s_prev = None
    for g in range(K // 128):
        sl = slice(128 * g, 128 * g + 128)
        op = (c + q.codes[:, sl].astype(f32) - z[:, g:g + 1]).astype(f32)
        R = np.zeros(m, f32)
        for col in range(128):                      # fp32 row sum of the group, in order
            R = (R + a[:, 128 * g + col]).astype(f32)
        sg = s[:, g]
        if s_prev is None:
            r = np.zeros(n, f32)
        else:
            rcp = (f32(1) / sg).astype(f32)
            rcp = (rcp * (1 + rng.choice([-1, 0, 1], size=n) * 2.0 ** -23)).astype(f32)  # rcp within one ulp
            r = (s_prev * rcp).astype(f32)
        Q = (Q.astype(np.float64) * r[None, :] + (-c * R).astype(np.float64)[:, None]).astype(f32)  # one FMA
        for j in range(4):
            blk = a[:, sl][:, 32 * j:32 * j + 32].astype(np.float64) @ op[:, 32 * j:32 * j + 32].T.astype(np.float64)
            Q = (Q.astype(np.float64) + blk).astype(f32)
        s_prev = sg
    return (Q * s_prev[None, :]).astype(f32)


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("K", [1024, 14336])
@pytest.mark.parametrize("act", ["bf16", "fp16"])
def test_acc16_model_weight_only(bits, K, act):
    """Weight-only kinds: the emulated bias-and-rescale arithmetic errs by at
    most ACC16_EPS / 4 * sum |a| |s (q - z)|."""
    rng = np.random.default_rng(bits * 1000 + K)
    q = W.quantize_linear(W.draw_weight(5, bits, 0, 16, K), W.Scheme(bits, 16, 128, -1, 0))
    x = rng.standard_normal((8, K))
    a = _bf16(x) if act == "bf16" else x.astype(np.float16).astype(f32)
    wd = O.dequant(q, act)
    exact = a.astype(np.float64) @ wd.T
    got = _magic_gemm(a, q, act, rng).astype(np.float64)
    bound = TL.acc_bound(np.abs(a).astype(np.float64), np.abs(wd))
    assert np.all(np.abs(got - exact) <= bound / 4), float((np.abs(got - exact) / bound).max())


def _fp8_model_block(pa, pw, drop=18):
    """The FP8 block-sum model: exact products aligned to the largest one,
    bits more than `drop` places below its leading bit truncated toward zero,
    summed exactly, rounded to fp32."""
    p = pa.astype(np.float64) * pw.astype(np.float64)
    pm = np.abs(p).max()
    if pm == 0:
        return 0.0, 0.0
    e = np.floor(np.log2(pm))
    quantum = 2.0 ** (e - drop)
    t = np.trunc(p / quantum) * quantum
    return float(f32(t.sum())), float(p.sum())


def test_fp8_model_within_bound():
    """Under the FP8 model a 128-product block errs by less than
    127 * 2^(e - 18) <= 2^-11 of its largest product (2^e <= max|p|), a
    quarter of the per-block charge FP8_BLOCK_EPS * max|a| max|w|
    (max|p| <= max|a| max|w|); random, spiked, wide-range and adversarial
    (every product just below a truncation step, all of one sign) operands
    stay inside it, the adversarial ones within a factor 2 of the model's
    worst case, so the construction reaches it."""
    vals = O.e4m3_values(np.arange(0, 127, dtype=np.uint8))
    rng = np.random.default_rng(3)
    worst = 0.0
    for trial in range(400):
        kind = trial % 4
        if kind == 0:
            pa = rng.choice(vals, 128) * rng.choice([-1, 1], 128)
            pw = rng.choice(vals, 128) * rng.choice([-1, 1], 128)
        elif kind == 1:                               # one spike, many small
            pa = rng.choice(vals[:60], 128)
            pw = rng.choice(vals[:60], 128)
            pa[0], pw[0] = 448.0, 448.0
        elif kind == 2:                               # wide range, mixed signs
            pa = rng.choice(vals, 128) * rng.choice([-1, 1], 128)
            pw = rng.choice(vals[::7], 128)
        else:                                         # adversarial: residues just below the quantum
            pa = np.full(128, 0.9375)                 # 0.9375 * 0.25 = 15/64, just below the quantum
            pw = np.full(128, 0.25)
            pa[0], pw[0] = 256.0, 256.0               # max product 2^16: quantum 2^(16 - 18) = 1/4
        got, exact = _fp8_model_block(pa, pw)
        amax, wmax = np.abs(pa).max(), np.abs(pw).max()
        if amax * wmax == 0:
            continue
        err = abs(got - exact)
        assert err <= TL.FP8_BLOCK_EPS / 4 * amax * wmax * (1 + 2.0 ** -20)
        worst = max(worst, err / (np.abs(pa * pw).max()))
    assert worst <= 2.0 ** -11
    assert worst >= 2.0 ** -12            # the adversarial block gets close to the model's worst case


@pytest.mark.parametrize("kind", ["w16", "w4g128", "w8a8"])
@pytest.mark.parametrize("act", ["bf16", "fp16"])
def test_h_tolerance_covers_emulated_h(kind, act):
    """Stage A: h formed in fp32 from emulated fp32 g and u (SiLU in fp32
    with one extra rounding, the product rounded, then the rounding to the
    activation dtype) stays within ulp + H_ABS_REL / 4 * row max of the exact
    h64, on the shapes of the gate|up linears (K = 4096)."""
    rng = np.random.default_rng(len(kind) * 7 + len(act))
    sch = {"w16": W.W16, "w4g128": W.W4G128, "w8a8": W.W8A8}[kind]
    K, n, m = 4096, 32, 16
    gq = W.quantize_linear(W.draw_weight(11, 0, 0, n, K), sch)
    uq = W.quantize_linear(W.draw_weight(11, 0, 1, n, K), sch)
    x = rng.standard_normal((m, K))
    a = _bf16(x) if act == "bf16" else x.astype(np.float16).astype(f32)
    a64 = a.astype(np.float64)
    g64, u64 = O.linear(a64, gq, act), O.linear(a64, uq, act)
    if kind == "w8a8":
        qa, sa = O.act_quant(a, 127)
        g32 = ((O.linear(a64, gq, act, return_int=True).astype(f32) * sa[:, None]).astype(f32) * gq.scales).astype(f32)
        u32 = ((O.linear(a64, uq, act, return_int=True).astype(f32) * sa[:, None]).astype(f32) * uq.scales).astype(f32)
    elif kind == "w16":
        g32 = _mfma_steps(a, O.dequant(gq, act).astype(f32))
        u32 = _mfma_steps(a, O.dequant(uq, act).astype(f32))
    else:
        g32, u32 = _magic_gemm(a, gq, act, rng), _magic_gemm(a, uq, act, rng)
    sil = (g32.astype(np.float64) / (1 + np.exp(-g32.astype(np.float64)))).astype(f32)
    sil = (sil * (1 + rng.choice([-1, 1], size=sil.shape) * 2.0 ** -23)).astype(f32)   # a few-ulp SiLU
    h32 = (sil * u32).astype(f32)
    h_act = O.round_to_act(h32.astype(np.float64), act)
    h64 = O.silu(g64) * u64
    rowmax = np.abs(h64).max(axis=1, keepdims=True)
    tol = TL.ulp_act(h64, act) + TL.H_ABS_REL / 4 * rowmax
    assert np.all(np.abs(h_act - h64) <= tol), float((np.abs(h_act - h64) / tol).max())


def test_ulp_act_spacing():
    """ulp_act is the spacing of the dtype: 1 -> 2^-7 (bf16) / 2^-10 (fp16),
    just below 1 -> 2^-8 / 2^-11, subnormal floors 2^-133 / 2^-24."""
    assert TL.ulp_act(np.array([1.0]), "bf16")[0] == 2.0 ** -7
    assert TL.ulp_act(np.array([0.999]), "bf16")[0] == 2.0 ** -8
    assert TL.ulp_act(np.array([1.0]), "fp16")[0] == 2.0 ** -10
    assert TL.ulp_act(np.array([0.999]), "fp16")[0] == 2.0 ** -11
    assert TL.ulp_act(np.array([0.0]), "bf16")[0] == 2.0 ** -133
    assert TL.ulp_act(np.array([1e-7]), "fp16")[0] == 2.0 ** -24
    # every value of a dtype sits one spacing from the next larger value
    v = np.array([0.3, 1.7, 100.25, -3.0])
    for act, nxt in (("fp16", lambda t: np.nextafter(t.astype(np.float16), np.float16(np.inf)).astype(np.float64)),):
        r = O.round_to_act(v, act)
        assert np.all(nxt(np.abs(r)) - np.abs(r) == TL.ulp_act(r, act))


def test_f6_encoder_of_the_stagewise_check():
    """The FP6 byte layout the stage-wise check compares against: every int4
    value -7..7 decodes back from its 6-bit field by the e2m3 bit-field
    definition ((-1)^s (1 + m/8) 2^(e-1), e > 0; 0 for e = m = 0), fields sit at
    bits 6i..6i+5 of each 32-element group's 24 bytes, and the 8 bytes after
    them are zero."""
    from tests.stagewise import f6_bytes
    rng = np.random.default_rng(4)
    q = rng.integers(-7, 8, size=(3, 128))
    q[0, :15] = np.arange(-7, 8)
    b = f6_bytes(q)
    assert b.shape == q.shape and b.dtype == np.uint8
    for r in range(3):
        for g in range(4):
            grp = b[r, 32 * g:32 * g + 32]
            assert not grp[24:].any()
            bits = int.from_bytes(bytes(grp[:24]), "little")
            for i in range(32):
                f = (bits >> (6 * i)) & 63
                s, e, m = f >> 5, (f >> 3) & 3, f & 7
                v = 0.0 if e == 0 else (1 + m / 8) * 2.0 ** (e - 1)
                assert e != 0 or m == 0
                assert (-v if s else v) == q[r, 32 * g + i]


@pytest.mark.parametrize("act", ["bf16", "fp16"])
def test_slot_bound_covers_rounding_to_the_activation_dtype(act):
    """slot_bound: a value v within `bound` of ref, rounded to nearest in the
    activation dtype (here by the workloads' bf16 bit rounding of float32 and
    numpy's float16 cast, not the oracle's rounding), stays within
    slot_bound(ref, bound) of ref - on values straddling powers of two, near
    zero and at the largest v; the rounding part is used at least halfway."""
    rng = np.random.default_rng(11)
    ref = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-4, 3, 4000),
                          2.0 ** rng.integers(-10, 8, 2000) * (1 - 2.0 ** -20), [0.0, 1e-6, -1.0]])
    bound = np.abs(ref) * 2.0 ** -14 + 1e-9
    worst = 0.0
    for frac in (-1.0, -0.37, 0.0, 0.61, 1.0):
        v = (ref + frac * bound).astype(np.float32)
        r = _bf16(v).astype(np.float64) if act == "bf16" else v.astype(np.float16).astype(np.float64)
        b = TL.slot_bound(ref, bound, act)
        err = np.abs(r - ref)
        assert np.all(err <= b), float((err / b).max())
        worst = max(worst, float(((err - bound) / (b - bound)).max()))
    assert worst >= 0.5
