"""GPU parity of the whole MoE block forward against the CPU oracle on small
blocks: the tiny workload (64 tokens, hidden 256, FFN 512, 4 experts, top-2,
fp16), random mixed-precision blocks with ragged tiles and shared experts,
edge cases (one token, empty experts, out-of-range ids), determinism and
token-permutation equivariance."""

import numpy as np
import pytest

from oracle import mxmoe_oracle as O
from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W
from tests.gpuhelp import say, torch_mod, upload_inputs
from tests.stagewise import check_forward

pytestmark = pytest.mark.gpu


def run_block(blk, **kw):
    torch = torch_mod()
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y = mb.forward(x, ids, w, **kw)
    torch.cuda.synchronize()
    return mb, y


def oracle(blk):
    return O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears, blk.cfg.E, blk.cfg.act)


def test_tiny_workload():
    torch = torch_mod()
    blk = W.make_block("tiny")
    mb, y = run_block(blk)
    rep = check_forward(mb, blk, y)
    say(f"tiny: {rep.line()}")
    ref = oracle(blk)
    T, k, E = blk.cfg.T, blk.cfg.k, blk.cfg.E
    r = ref["route"]
    cnt = mb.ws_view("counts", torch.int32, E, T).cpu().numpy()
    sp = mb.ws_view("sorted_pair", torch.int32, T * k, T).cpu().numpy()
    st = mb.ws_view("status", torch.int32, 1, T).cpu().numpy()
    assert np.array_equal(cnt, r["counts"]) and np.array_equal(sp, r["sorted_pair"]) and st[0] == 0
    # the gated intermediate h of every expert matches the oracle's rounded h
    h = mb.ws_view("h", torch.int16, T * k * blk.cfg.F, T).cpu().numpy().view(np.float16)
    h = h.reshape(T * k, blk.cfg.F).astype(np.float64)
    ref_h = O.moe_forward(blk.x, blk.topk_ids, blk.topk_w, blk.linears, E, "fp16", return_h=True)["h"]
    for e in range(E):
        lo, hi = int(r["offsets"][e]), int(r["offsets"][e + 1])
        d = np.abs(h[lo:hi] - ref_h[e])
        tol = 1e-2 * np.abs(ref_h[e]).max(axis=1, keepdims=True)
        assert np.all(d <= tol), (e, float(d.max()))


MIXES = [
    [(W.W4G128,) * 3, (W.W8A8, W.W8A8, W.W2G128), (W.W4A4,) * 3, (W.W16,) * 3, (W.W3G128,) * 3,
     (W.W8G128, W.W8G128, W.W4A4), (W.W2G128, W.W2G128, W.W8A8)],
    [(W.W8A8,) * 3] * 7,
    [(W.W4A4, W.W4A4, W.W16), (W.W16, W.W16, W.W4A4), (W.W3G128, W.W3G128, W.W8G128), (W.W4G128,) * 3,
     (W.W2G128,) * 3, (W.W8A8,) * 3, (W.W4A4,) * 3],
    # w4a4-g128 beside every neighbour: row sums of h for a magic-dequant down
    # behind a w4a4-g128 gate/up, group-quantized h for a w4a4-g128 down
    [(W.W4A4G128,) * 3, (W.W4A4G128, W.W4A4G128, W.W2G128), (W.W8A8, W.W8A8, W.W4A4G128),
     (W.W4A4G128, W.W4A4G128, W.W8A8), (W.W16, W.W16, W.W4A4G128), (W.W3G128, W.W3G128, W.W4A4G128),
     (W.W4A4G128, W.W4A4G128, W.W4A4)],
    # mxfp4 (FP4 e2m1 with E8M0 scales, on the scaled FP4 MFMA) beside the others
    [(W.MXFP4,) * 3, (W.MXFP4, W.MXFP4, W.W2G128), (W.W8A8, W.W8A8, W.MXFP4), (W.W16, W.W16, W.MXFP4),
     (W.MXFP4, W.MXFP4, W.W4A4G128), (W.W3G128, W.W3G128, W.MXFP4), (W.MXFP4, W.MXFP4, W.W8A8)],
    # fp8 (e4m3 with per-channel / per-token scales, on the FP8 MFMA) beside the others
    [(W.FP8,) * 3, (W.FP8, W.FP8, W.W2G128), (W.W8A8, W.W8A8, W.FP8), (W.W16, W.W16, W.FP8),
     (W.FP8, W.FP8, W.W4A4G128), (W.MXFP4, W.MXFP4, W.FP8), (W.FP8, W.FP8, W.W8A8)],
    # w4a4 on FP6 e2m3 operands beside the others (and beside int8-MFMA w4a4)
    [(W.W4A4F6,) * 3, (W.W4A4F6, W.W4A4F6, W.W2G128), (W.W8A8, W.W8A8, W.W4A4F6), (W.W16, W.W16, W.W4A4F6),
     (W.W4A4F6, W.W4A4F6, W.W4A4G128), (W.W4A4, W.W4A4, W.W4A4F6), (W.W4A4F6, W.W4A4F6, W.W4A4)],
]


def test_f8_activation_codes_bit_exact():
    """The forward's FP8 encoding of x and of the routed and shared h rows
    equals the oracle's encoder, byte for byte (h: the encoder applied to the
    GPU's own rounded h)."""
    torch = torch_mod()
    for act in ("bf16", "fp16"):
        T, H, F, Fs, k = 77, 256, 384, 256, 2
        blk = W.random_small_block(97, T=T, H=H, F=F, E=4, k=k, n_shared=1, F_shared=Fs, act=act,
                                   schemes=[(W.FP8,) * 3] * 5, skew=0.5)
        mb, _ = run_block(blk)
        qx, sx = O.fp8_quant(O.act_values(blk.x, act).astype(np.float32))
        assert np.array_equal(mb.ws_view("xqf8", torch.uint8, T * H, T).cpu().numpy().reshape(T, H), qx)
        assert np.array_equal(mb.ws_view("xsf8", torch.float32, T, T).cpu().numpy(), sx)
        P = int(mb.ws_view("offsets", torch.int32, 5, T).cpu().numpy()[4])

        def hvals(name, rows, cols):
            h = mb.ws_view(name, torch.int16, rows * cols, T).cpu().numpy().reshape(rows, cols)
            return O.act_values(h.view(np.float16) if act == "fp16" else h.view(np.uint16), act).astype(np.float32)

        qh, sh = O.fp8_quant(hvals("h", T * k, F)[:P])
        assert np.array_equal(mb.ws_view("hq", torch.uint8, T * k * F, T).cpu().numpy()[: P * F].reshape(P, F), qh)
        assert np.array_equal(mb.ws_view("hs", torch.float32, T * k, T).cpu().numpy()[:P], sh)
        qs, ss = O.fp8_quant(hvals("h_shared", T, Fs))
        assert np.array_equal(mb.ws_view("hq_shared", torch.uint8, T * Fs, T).cpu().numpy().reshape(T, Fs), qs)
        assert np.array_equal(mb.ws_view("hs_shared", torch.float32, T, T).cpu().numpy(), ss)
        say(f"fp8 codes {act}: x, {P} routed and {T} shared h rows bit-exact")


def test_mx_activation_codes_bit_exact():
    """The forward's MXFP4 encoding of x and of the routed and shared h rows
    equals the oracle's encoder, byte for byte."""
    torch = torch_mod()
    for act in ("bf16", "fp16"):
        blk = W.random_small_block(91, T=77, H=256, F=384, E=4, k=2, n_shared=1, F_shared=256, act=act,
                                   schemes=[(W.MXFP4,) * 3] * 5, skew=0.5)
        mb, _ = run_block(blk)
        T, H, F, k = 77, 256, 384, 2
        xq = mb.ws_view("xqmx", torch.uint8, T * H // 2, T).cpu().numpy().reshape(T, H // 2)
        xe = mb.ws_view("xsmx", torch.uint8, T * H // 32, T).cpu().numpy().reshape(T, H // 32)
        qx, ex = O.mx_quant(O.act_values(blk.x, act).astype(np.float32))
        assert np.array_equal(xq, (qx[:, 0::2] | (qx[:, 1::2] << 4)).astype(np.uint8))
        assert np.array_equal(xe, ex)
        # routed h rows, in sorted-pair order, against the encoder of the GPU's own h
        P = int(mb.ws_view("offsets", torch.int32, 5, T).cpu().numpy()[4])
        hdt = torch.int16
        h = mb.ws_view("h", hdt, T * k * F, T).cpu().numpy()[: P * F].reshape(P, F)
        hv = O.act_values(h.view(np.float16) if act == "fp16" else h.view(np.uint16), act)
        hq = mb.ws_view("hqmx", torch.uint8, T * k * F // 2, T).cpu().numpy()[: P * F // 2].reshape(P, F // 2)
        he = mb.ws_view("hsmx", torch.uint8, T * k * F // 32, T).cpu().numpy()[: P * F // 32].reshape(P, F // 32)
        qh, eh = O.mx_quant(hv.astype(np.float32))
        assert np.array_equal(hq, (qh[:, 0::2] | (qh[:, 1::2] << 4)).astype(np.uint8))
        assert np.array_equal(he, eh)
        say(f"mx codes {act}: x and {P} routed h rows bit-exact")


@pytest.mark.parametrize("H", [256, 4224])
def test_x_encodings_bit_exact(H):
    """Every encoding of x that the plan launch writes on its spare workgroups
    equals the oracle's encoders byte for byte: int8 and int4 codes per token,
    int4 codes per 128-group, MXFP4 codes and E8M0 bytes, FP8 codes and
    scales per token; the bf16 row sums
    per 128-block lie within the rounding of a 128-term fp32 sum.  H = 4224
    takes rows longer than the register-resident encoder holds."""
    torch = torch_mod()
    T = 300 if H == 256 else 37
    sch = [(W.W8A8, W.W8A8, W.W16), (W.W4A4,) * 3, (W.W2G128,) * 3, (W.W4A4G128,) * 3, (W.MXFP4,) * 3,
           (W.FP8,) * 3]
    blk = W.random_small_block(313 + H, T=T, H=H, F=128, E=6, k=2, act="bf16", schemes=sch, skew=0.3)
    mb, _ = run_block(blk)
    xv = O.act_values(blk.x, "bf16").astype(np.float32)

    def ws(name, dt, n, shape):
        return mb.ws_view(name, dt, n, T).cpu().numpy().reshape(shape)

    q8, s8 = O.act_quant(xv, 127)
    assert np.array_equal(ws("xq8", torch.int8, T * H, (T, H)), q8)
    assert np.array_equal(ws("xs8", torch.float32, T, (T,)), s8)
    q4, s4 = O.act_quant(xv, 7)
    assert np.array_equal(ws("xq4", torch.int8, T * H, (T, H)), q4)
    assert np.array_equal(ws("xs4", torch.float32, T, (T,)), s4)
    qg, sg = O.act_quant_groups(xv, 7, 128)
    assert np.array_equal(ws("xq4g", torch.int8, T * H, (T, H)), qg)
    assert np.array_equal(ws("xs4g", torch.float32, T * H // 128, (T, H // 128)), sg)
    qx, ex = O.mx_quant(xv)
    assert np.array_equal(ws("xqmx", torch.uint8, T * H // 2, (T, H // 2)),
                          (qx[:, 0::2] | (qx[:, 1::2] << 4)).astype(np.uint8))
    assert np.array_equal(ws("xsmx", torch.uint8, T * H // 32, (T, H // 32)), ex)
    qf, sf = O.fp8_quant(xv)
    assert np.array_equal(ws("xqf8", torch.uint8, T * H, (T, H)), qf)
    assert np.array_equal(ws("xsf8", torch.float32, T, (T,)), sf)
    rs = ws("rsx", torch.float32, T * H // 128, (T, H // 128)).astype(np.float64)
    blocks = xv.astype(np.float64).reshape(T, H // 128, 128)
    assert np.all(np.abs(rs - blocks.sum(-1)) <= 128 * 2.0 ** -24 * np.abs(blocks).sum(-1))
    say(f"x encodings H={H}: int8, int4, int4-g128, mxfp4, fp8 bit-exact; row sums within bound")


@pytest.mark.parametrize("act", ["bf16", "fp16"])
@pytest.mark.parametrize("mix", range(len(MIXES)))
@pytest.mark.parametrize("T", [1, 37, 300])
def test_random_blocks(act, mix, T):
    sch = MIXES[mix]
    blk = W.random_small_block(100 + mix * 7 + T, T=T, H=256, F=384, E=6, k=2, n_shared=1, F_shared=256,
                               act=act, schemes=sch, skew=1.2)
    mb, y = run_block(blk)
    rep = check_forward(mb, blk, y)
    say(f"mix{mix} T={T} {act}: {rep.line()}")


def test_many_cold_experts_and_bad_ids():
    torch = torch_mod()
    sch = [(W.W4A4,) * 3, (W.W3G128,) * 3, (W.W8A8,) * 3, (W.W2G128,) * 3] * 4
    blk = W.random_small_block(7, T=9, H=128, F=256, E=16, k=2, act="bf16", schemes=sch, skew=2.0)
    blk.topk_ids[3, 1] = 99
    blk.topk_ids[6, 0] = -1
    mb, y = run_block(blk)
    rep = check_forward(mb, blk, y)
    say(f"cold/bad ids: {rep.line()}")
    st = int(mb.ws_view("status", torch.int32, 1, 9).cpu().numpy()[0])
    assert st == 1 + 3 * 2 + 1


def test_determinism_and_permutation():
    torch = torch_mod()
    blk = W.random_small_block(55, T=200, H=256, F=256, E=5, k=2, n_shared=1, F_shared=128,
                               act="bf16", schemes=MIXES[2][:6], skew=1.0)
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y1 = M.act_numpy(mb.forward(x, ids, w), "bf16")
    y2 = M.act_numpy(mb.forward(x, ids, w), "bf16")
    assert np.array_equal(y1, y2)
    perm = np.random.default_rng(0).permutation(200)
    pt = torch.from_numpy(perm).cuda()
    y3 = M.act_numpy(mb.forward(x[pt].contiguous(), ids[pt].contiguous(), w[pt].contiguous()), "bf16")
    torch.cuda.synchronize()
    assert np.array_equal(y3, y1[perm])


def test_expert_mask_and_skip_combine():
    torch = torch_mod()
    blk = W.random_small_block(3, T=64, H=128, F=128, E=4, k=1, act="bf16",
                               schemes=[(W.W8A8,) * 3, (W.W4G128,) * 3, (W.W16,) * 3, (W.W4A4,) * 3])
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y = torch.zeros_like(x)
    mb.forward(x, ids, w, y=y, skip_combine=True)
    torch.cuda.synchronize()
    assert int((y.view(torch.int16) != 0).sum()) == 0
    # only expert 1 computes: its rows are right, the combine of other tokens is not checked
    mb.ws[:].zero_()
    y = mb.forward(x, ids, w, expert_mask=[0, 1, 0, 0])
    torch.cuda.synchronize()
    ref = oracle(blk)
    sel = blk.topk_ids[:, 0] == 1
    yv = O.act_values(M.act_numpy(y, "bf16"), "bf16")[sel]
    r = ref["y"][sel]
    assert np.all(np.abs(yv - r) <= 1e-2 * np.abs(r).max(axis=1, keepdims=True))


@pytest.mark.parametrize("act", ["bf16", "fp16"])
def test_fp32_slots_option(act):
    """fp32_slots keeps the weighted down rows in fp32: the stage-wise check
    then compares them bit for bit (integer kinds) or within the fp32 models,
    and the combine sums the fp32 rows; the default path rounds every slot
    row element once to the activation dtype (checked by every other test)."""
    torch = torch_mod()
    blk = W.random_small_block(911, T=200, H=256, F=384, E=6, k=2, n_shared=1, F_shared=256, act=act,
                               schemes=MIXES[0], skew=1.0)
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y32 = mb.forward(x, ids, w, fp32_slots=True)
    torch.cuda.synchronize()
    assert mb.slot_dtype() == torch.float32
    rep = check_forward(mb, blk, y32)
    y16 = mb.forward(x, ids, w)
    torch.cuda.synchronize()
    assert mb.slot_dtype() != torch.float32
    rep16 = check_forward(mb, blk, y16)
    say(f"fp32 slots {act}: {rep.line()}; 16-bit slots: {rep16.line()}")


@pytest.mark.parametrize("fp32_slots", [False, True])
def test_combine_of_more_than_ten_slots(fp32_slots):
    """k + n_shared = 11 slots per token: the combine takes its generic path
    (any slot count, one slot at a time) for 16-bit and fp32 slot rows; the
    stage-wise check emulates it bit for bit."""
    torch = torch_mod()
    sch = [(W.W8A8,) * 3, (W.W4G128,) * 3, (W.W16,) * 3, (W.W4A4,) * 3] * 3 + [(W.W8A8,) * 3, (W.W16,) * 3,
                                                                              (W.W4A4,) * 3]
    blk = W.random_small_block(1234, T=50, H=256, F=256, E=12, k=8, n_shared=3, F_shared=256, act="bf16",
                               schemes=sch, skew=0.5)
    mb = M.MoEBlock(blk)
    x, ids, w = upload_inputs(blk)
    y = mb.forward(x, ids, w, fp32_slots=fp32_slots)
    torch.cuda.synchronize()
    rep = check_forward(mb, blk, y)
    say(f"11 slots, fp32_slots={fp32_slots}: {rep.line()}")
