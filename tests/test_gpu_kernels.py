"""GPU parity of the individual steps against the CPU oracle: weight packing
(round trip), routing / permutation (bit-exact), per-token activation
quantization (bit-exact) and every micro-kernel as a single linear (exact
int32 accumulators for w8a8 / w4a4, fp32 within an accumulation bound else)."""

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W
from tests import tolerance as TL
from tests.gpuhelp import say, torch_mod

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- packing
@pytest.mark.parametrize("act", ["bf16", "fp16"])
@pytest.mark.parametrize("scheme", W.ALL_SCHEMES)
def test_pack_roundtrip(scheme, act):
    torch_mod()
    w = W.draw_weight(5, 0, 0, 48, 384)
    w[0, :4] = [3.0e-6, -1.0e-7, 60000.0, -0.0]        # fp16 subnormal / rounding corner cases
    q = W.quantize_linear(w, scheme)
    pl = M.PackedLinear(q, act)
    c, s, z = pl.unpack()
    if scheme.w_bits == 16:
        want = q.codes if act == "bf16" else \
            O.bf16_bits_to_f64(q.codes).astype(np.float16).view(np.uint16)
        assert np.array_equal(c, want)
    else:
        assert np.array_equal(c.astype(np.int64), q.codes.astype(np.int64))
        assert np.array_equal(s.view(np.uint8), q.scales.view(np.uint8))
        if z is not None:
            assert np.array_equal(z.view(np.uint8), q.zeros.view(np.uint8))


# ---------------------------------------------------------------- routing
# batches of up to 4096 pairs take the one-workgroup kernel, larger ones the
# chunked launches (1024 x 4 sits at the limit, 4097 x 1 just past it)
ROUTE_CASES = [(1, 1, 1, "uniform"), (64, 2, 4, "uniform"), (257, 6, 64, "uniform"),
               (2049, 8, 64, "uniform"), (1000, 4, 60, "skew"), (300, 2, 8, "one"),
               (0, 2, 4, "uniform"), (513, 3, 7, "bad"), (5000, 2, 1024, "uniform"),
               (16384, 8, 64, "zipf"), (1024, 4, 64, "zipf"), (4097, 1, 16, "uniform"),
               (6000, 3, 7, "bad")]


def _ids(T, k, E, kind, seed):
    rng = np.random.default_rng(seed)
    if kind == "one":
        ids = np.stack([np.r_[3, rng.permutation([e for e in range(E) if e != 3])[: k - 1]] for _ in range(T)])
    elif kind in ("skew", "zipf"):
        bias = -1.5 * np.log(np.arange(1, E + 1))
        logits = rng.standard_normal((T, E)) + bias
        ids = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    else:
        ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]) if T else np.zeros((0, k))
    ids = ids.astype(np.int32).reshape(T, k)
    if kind == "bad":
        ids[5, 1] = E + 3
        ids[400, 0] = -2
    return ids


@pytest.mark.parametrize("T,k,E,kind", ROUTE_CASES)
def test_route_permute(T, k, E, kind):
    torch = torch_mod()
    ids = _ids(T, k, E, kind, T * 31 + E)
    r = O.route(ids, E)
    g = M.route_permute(torch.from_numpy(ids).cuda(), E)
    torch.cuda.synchronize()
    assert np.array_equal(g["counts"].cpu().numpy(), r["counts"])
    assert np.array_equal(g["offsets"].cpu().numpy(), r["offsets"])
    nv = int(r["offsets"][-1])
    assert np.array_equal(g["sorted_pair"].cpu().numpy()[:nv], r["sorted_pair"])
    assert np.array_equal(g["inv"].cpu().numpy(), r["inv"])
    bad = np.nonzero(r["bad"])[0]
    assert int(g["status"].cpu().item()) == (int(bad[0]) + 1 if bad.size else 0)


# ------------------------------------------------------- activation quant
# row lengths that reach every kernel shape: one wavefront per row with 2, 4
# or 8 chunks per lane, one workgroup per row with 4 or 8, a streamed row
# read twice; ld_pad 3 misaligns the rows (element loads, one workgroup per row)
@pytest.mark.parametrize("act", ["bf16", "fp16"])
@pytest.mark.parametrize("qmax", [127, 7, 448])
@pytest.mark.parametrize("rows,cols,ld_pad", [(1, 128, 0), (37, 2048, 0), (300, 3584, 0), (5, 6144, 8),
                                              (9, 14336, 0), (3, 20480, 0), (6, 1000, 3), (4, 100, 0)])
def test_act_quant_bit_exact(act, qmax, rows, cols, ld_pad):
    torch = torch_mod()
    rng = np.random.default_rng(rows + cols + qmax)
    x64 = rng.standard_normal((rows, cols)) * np.exp(rng.uniform(-3, 3, size=(rows, 1)))
    x = W.f64_to_act(x64, act)
    if rows > 2:
        x[1] = 0                                       # zero row
        x[2, 5] = x[2, 0]                             # ties in amax
    wide = np.zeros((rows, cols + ld_pad), dtype=x.dtype)
    wide[:, :cols] = x
    a = M.act_tensor(wide, act)[:, :cols]
    assert a.stride(0) == cols + ld_pad
    codes, scales = M.act_quant(a, act, qmax)
    torch.cuda.synchronize()
    if qmax == 448:     # FP8 e4m3 bytes
        rc, rs = O.fp8_quant(O.act_values(x, act).astype(np.float32))
        assert np.array_equal(codes.cpu().numpy().view(np.uint8), rc)
        assert np.array_equal(scales.cpu().numpy().view(np.uint32), rs.view(np.uint32))
        return
    rc, rs = O.act_quant(O.act_values(x, act).astype(np.float32), qmax)
    assert np.array_equal(codes.cpu().numpy(), rc)
    assert np.array_equal(scales.cpu().numpy().view(np.uint32), rs.view(np.uint32))


# ------------------------------------------------------------- one linear
LIN_SHAPES = [(48, 384), (272, 256)]
LIN_M = [1, 5, 16, 17, 64, 65, 130, 300]


def _linear_case(scheme, act, m, n, k, seed):
    torch = torch_mod()
    q = W.quantize_linear(W.draw_weight(seed, 1, 0, n, k), scheme)
    x = W.f64_to_act(np.random.default_rng(seed).standard_normal((m, k)), act)
    pl = M.PackedLinear(q, act)
    out, ws = M.linear_forward(pl, M.act_tensor(x, act), return_ws=True)
    torch.cuda.synchronize()
    a = O.act_values(x, act)
    # slices the plan cut the reduction into (record of group 0, phase 0)
    split = int(ws[: 4 * PF_N].view(torch.int32)[PF_SPLIT].item())
    return q, a, out.cpu().numpy(), split


PF_N, PF_SPLIT = 12, 8   # int32 fields of a tile-plan group record; the slice count


def _check_linear(q, a, got, act):
    """Every scheme against the oracle's linear on the same operands:
    w8a8 / w4a4 exact int32; fp8 within the FP8 block model; the others
    within the fp32 accumulation model on the operands as the kernel
    multiplies them (tests/tolerance.py)."""
    s = q.scheme
    if s.a_bits < 16 and s.a_group < 0 and s.fmt in (0, 3):
        want = O.linear(a, q, act, return_int=True)
        assert np.array_equal(got.astype(np.int64), want)
        return 0.0
    want = O.linear(a, q, act)
    wd = O.dequant(q, act)
    if s.fmt == 2:
        qa, sa = O.fp8_quant(a.astype(np.float32))
        bound = TL.fp8_block_bound(O.e4m3_values(qa) * sa.astype(np.float64)[:, None], wd)
    elif s.fmt == 1:
        qa, ea = O.mx_quant(a.astype(np.float32), 32)
        bound = TL.acc_bound(np.abs(O._mx_values(qa, ea, 32)), np.abs(wd))
    elif s.a_group > 0:
        qa, sa = O.act_quant_groups(a.astype(np.float32), 2 ** (s.a_bits - 1) - 1, s.a_group)
        ad = (qa.astype(np.float64).reshape(a.shape[0], -1, s.a_group) * sa.astype(np.float64)[..., None]).reshape(a.shape)
        bound = TL.acc_bound(np.abs(ad), np.abs(wd))
    else:
        bound = TL.acc_bound(np.abs(a), np.abs(wd))
    bound = bound + 2 * TL.U32 * np.abs(want) + 1e-30
    err = np.abs(got - want)
    assert np.all(err <= bound), float((err / bound).max())
    return float((err / bound).max())


@pytest.mark.parametrize("scheme", W.ALL_SCHEMES)
@pytest.mark.parametrize("m", LIN_M)
@pytest.mark.parametrize("n,k", LIN_SHAPES)
def test_linear_bf16(scheme, m, n, k):
    q, a, got, _ = _linear_case(scheme, "bf16", m, n, k, m * 7 + n)
    _check_linear(q, a, got, "bf16")


@pytest.mark.parametrize("scheme", W.ALL_SCHEMES)
@pytest.mark.parametrize("m", [3, 33, 129])
def test_linear_fp16(scheme, m):
    q, a, got, _ = _linear_case(scheme, "fp16", m, 48, 256, m + 11)
    _check_linear(q, a, got, "fp16")


# Deep reductions: the plan slices K (split-K) once a tile has at least 12
# 128-wide k blocks; the slices store fp32 / int32 partial sums and the last
# one to arrive adds them in slice order.
@pytest.mark.parametrize("scheme", W.ALL_SCHEMES)
@pytest.mark.parametrize("m", [1, 17, 130, 300])
@pytest.mark.parametrize("k", [2048, 14336])
def test_linear_split_k(scheme, m, k):
    q, a, got, split = _linear_case(scheme, "bf16", m, 64, k, m * 13 + k)
    ratio = _check_linear(q, a, got, "bf16")
    if k == 14336 or m <= 17:
        assert split >= 2, f"the plan did not slice K = {k}"
    say(f"split-K {scheme.name} m={m} K={k}: {split} slices, worst err / bound {ratio:.4f}")


@pytest.mark.parametrize("scheme", W.ALL_SCHEMES)
def test_linear_split_k_fp16(scheme):
    q, a, got, split = _linear_case(scheme, "fp16", 65, 48, 14336, 41)
    ratio = _check_linear(q, a, got, "fp16")
    assert split >= 2
    say(f"split-K fp16 {scheme.name} m=65 K=14336: {split} slices, worst err / bound {ratio:.4f}")


def test_fp8_block_model_adversarial():
    """FP8 operands built to hit the block-sum model's worst case (one
    product 2^16, the other 127 just below the model's truncation step, all
    of one sign) stay within the FP8 bound; so do spiked and wide-range rows."""
    torch = torch_mod()
    n, k, m = 16, 2048, 4
    w = np.full((n, k), 0.25)
    w[:, ::128] = 256.0
    q = W.QLinear(W.FP8, n, k, *W.quantize_fp8(w))
    x = np.full((m, k), 0.9375)
    x[:, ::128] = 256.0
    x[1] = np.random.default_rng(1).standard_normal(k) * np.exp(np.random.default_rng(2).uniform(-6, 6, k))
    x[2, :] = 1e-3
    x[2, 5] = 300.0
    xa = W.f64_to_act(x, "bf16")
    pl = M.PackedLinear(q, "bf16")
    got = M.linear_forward(pl, M.act_tensor(xa, "bf16")).cpu().numpy()
    torch.cuda.synchronize()
    a = O.act_values(xa, "bf16")
    ratio = _check_linear(q, a, got, "bf16")
    say(f"fp8 adversarial: worst err / bound {ratio:.4f}")


def test_linear_deterministic():
    torch = torch_mod()
    q = W.quantize_linear(W.draw_weight(9, 0, 0, 256, 512), W.W4G128)
    x = W.f64_to_act(np.random.default_rng(1).standard_normal((100, 512)), "bf16")
    pl = M.PackedLinear(q, "bf16")
    a = M.act_tensor(x, "bf16")
    o1 = M.linear_forward(pl, a).cpu().numpy()
    o2 = M.linear_forward(pl, a).cpu().numpy()
    assert np.array_equal(o1.view(np.uint32), o2.view(np.uint32))


@pytest.mark.parametrize("scheme", [W.W2G128, W.W3G128, W.W4G128, W.W8G128, W.W4A4G128, W.W4A4, W.W4A4F6])
def test_pack_domain_of_codes_and_zeros(scheme):
    """Boundary zero points (0 and 2^N - 1, with the extreme codes) pack
    exactly and the linear matches the oracle in those channels; a zero
    point that is not an integer in [0, 2^N - 1], a weight-only code above
    2^N - 1 or a w4a4 code outside [-7, 7] stores that group's scale (the
    channel's for per-channel w4a4) as NaN, so its outputs are NaN instead of
    silently wrong, while the other channels stay exact."""
    torch = torch_mod()
    n, k, m = 48, 512, 5
    q = W.quantize_linear(W.draw_weight(77, 0, 0, n, k), scheme)
    codes, scales = q.codes.copy(), q.scales.copy()
    zeros = None if q.zeros is None else q.zeros.copy()
    poisoned = []
    if scheme.a_bits == 16:                        # weight-only: boundary zeros, then bad zeros / codes
        top = (1 << scheme.w_bits) - 1
        zeros[0, 0], codes[0, :128] = 0, np.arange(128) % (top + 1)
        zeros[1, 0], codes[1, :128] = top, np.arange(128) % (top + 1)
        zeros[2, 1] = 1.5                          # not an integer
        zeros[3, 2] = top + 1                      # above 2^N - 1
        poisoned += [(2, 1), (3, 2)]
        if scheme.w_bits < 8:
            codes[4, 300] = top + 1                # a code beyond N bits
            poisoned.append((4, 2))
    else:
        codes[2, 7] = 8
        codes[3, 130] = -8
        poisoned += [(2, 0), (3, 1)]
    bad = W.QLinear(scheme, n, k, codes, scales, zeros)
    pl = M.PackedLinear(bad, "bf16")
    _, sc, _ = pl.unpack()
    scf = sc.astype(np.float32)
    for ch, grp in poisoned:
        assert np.isnan(scf[ch] if scf.ndim == 1 else scf[ch, grp]), (ch, grp)
    rows = [c for c, _ in poisoned]
    good = [c for c in range(n) if c not in rows]
    assert not np.isnan(scf[good]).any()
    x = W.f64_to_act(np.random.default_rng(5).standard_normal((m, k)), "bf16")
    out = M.linear_forward(pl, M.act_tensor(x, "bf16")).cpu().numpy()
    torch.cuda.synchronize()
    a = O.act_values(x, "bf16")
    if scheme.a_bits < 16 and scheme.a_group < 0:      # per-channel w4a4: exact int32 in every channel
        want = O.linear(a, W.QLinear(scheme, n, k, np.clip(codes, -7, 7), scales), "bf16", return_int=True)
        assert np.array_equal(out[:, good].astype(np.int64), want[:, good])
    else:
        assert np.isnan(out[:, rows]).all()
        okq = W.QLinear(scheme, len(good), k, codes[good], scales[good], None if zeros is None else zeros[good])
        _check_linear(okq, a, out[:, good], "bf16")
    say(f"pack domain {scheme.name}: boundary zeros exact, {len(poisoned)} out-of-domain groups poisoned")
