"""Host-side checks of the C ABI (no GPU work: only size queries and argument
validation, which return before anything is enqueued)."""

import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2505_05799_amd import mxmoe as M
from paper_2505_05799_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mxmoe.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(M.LIB_PATH):
        from paper_2505_05799_amd import build
        build.build()
    return M.load_library()


def header_functions():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"MXMOE_API\s+[\w\s\*]+?\b(mxmoe_\w+)\s*\(", txt)))


def test_header_declares_binding_exports():
    assert header_functions() == sorted(M.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", M.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT\s+(mxmoe_\w+)", out))
    assert set(header_functions()) <= exported
    # internals stay hidden
    assert not any("launch_" in l for l in out.splitlines())
    for f in header_functions():
        assert hasattr(lib, f)


def _L(s, n=256, k=512):
    return M.Linear_t(n, k, M.scheme_t(s))


@pytest.mark.parametrize("s", W.ALL_SCHEMES)
def test_packed_bytes_closed_form(lib, s):
    n, k = 272, 1408
    got = lib.mxmoe_packed_bytes(C.byref(_L(s, n, k)), M.BF16)
    if s.w_bits == 16:
        want = 2 * n * k
    elif s.fmt == 3:
        want = n * k * 6 // 8 + 4 * n                          # 4-bit codes held as 6-bit e2m3
    elif s.a_bits == 16:
        want = n * k * s.w_bits // 8 + (n * k // 128) * 4      # N + 0.25 bits per weight
    elif s.w_group > 0:
        want = n * k * s.w_bits // 8 + (n * k // 128) * 4      # fp16 group scale in a 4-byte slot
    else:
        want = n * k * s.w_bits // 8 + 4 * n
    assert got == want == W.QLinear(s, n, k, None).nbytes_packed


def test_packed_bits_per_weight_paper_accounting(lib):
    """Sec. 5.2: 3-bit and 2-bit g128 with 16-bit scale and zero are 3.25 and 2.25 bits."""
    for s, bits in ((W.W3G128, 3.25), (W.W2G128, 2.25)):
        n, k = 4096, 4096
        assert lib.mxmoe_packed_bytes(C.byref(_L(s, n, k)), M.BF16) * 8 / (n * k) == bits


@pytest.mark.parametrize("n,k,scheme", [(250, 512, W.W4G128), (256, 500, W.W8A8), (0, 128, W.W16),
                                        (16, 128, W.Scheme(5, 16, 128, -1, 0)),
                                        (16, 128, W.Scheme(4, 4, 128, -1, 1)),
                                        (16, 128, W.Scheme(8, 8, 128, 128, 1)),
                                        (16, 64, W.W4A4G128),
                                        (16, 128, W.Scheme(8, 8, -1, -1, 0))])
def test_packed_bytes_rejects(lib, n, k, scheme):
    assert lib.mxmoe_packed_bytes(C.byref(_L(scheme, n, k)), M.BF16) == 0


def test_pack_validation(lib):
    L = _L(W.W4G128)
    buf = C.c_void_p(4096 * 256)  # never dereferenced: validation fails first
    assert lib.mxmoe_pack_weights(C.byref(L), M.BF16, M.BF16, None, buf, buf, buf, 10 ** 6, None) == M.ERR_INVALID_ARG
    assert lib.mxmoe_pack_weights(C.byref(L), M.BF16, M.BF16, buf, None, buf, buf, 10 ** 6, None) == M.ERR_INVALID_ARG
    assert lib.mxmoe_pack_weights(C.byref(L), M.BF16, M.BF16, buf, buf, buf, C.c_void_p(4096 * 256 + 8), 10 ** 6,
                                  None) == M.ERR_INVALID_ARG
    assert lib.mxmoe_pack_weights(C.byref(L), M.BF16, M.BF16, buf, buf, buf, buf, 100, None) == M.ERR_WORKSPACE
    assert lib.mxmoe_pack_weights(C.byref(L), 7, M.BF16, buf, buf, buf, buf, 10 ** 6, None) == M.ERR_INVALID_ARG
    bad = _L(W.Scheme(6, 6, -1, -1, 1))
    assert lib.mxmoe_pack_weights(C.byref(bad), M.BF16, M.BF16, buf, buf, buf, buf, 10 ** 6, None) == M.ERR_UNSUPPORTED


def test_route_validation(lib):
    p = C.c_void_p(1 << 20)
    assert lib.mxmoe_route_permute(p, 4, 3, 2, p, p, p, p, p, p, 10 ** 6, None) == M.ERR_INVALID_ARG  # k > E
    assert lib.mxmoe_route_permute(p, 4, 1, 2000, p, p, p, p, p, p, 10 ** 6, None) == M.ERR_INVALID_ARG
    assert lib.mxmoe_route_permute(p, 4, 2, 8, p, p, p, p, p, p, 0, None) == M.ERR_WORKSPACE
    assert lib.mxmoe_route_workspace_bytes(131072 // 8, 8, 64) > 0


def test_act_quant_validation(lib):
    p = C.c_void_p(1 << 20)
    assert lib.mxmoe_act_quant(p, M.BF16, 4, 128, 128, 15, p, p, None) == M.ERR_UNSUPPORTED
    assert lib.mxmoe_act_quant(p, M.BF16, 4, 128, 64, 127, p, p, None) == M.ERR_INVALID_ARG


def _block(cfg_name, schemes=None, packed=None):
    cfg = W.CONFIGS[cfg_name]
    sch = schemes or W.schemes_of(cfg)
    G = cfg.E + cfg.n_shared
    arr = (M.Scheme_t * (3 * G))(*[M.scheme_t(s) for t in sch for s in t])
    ptrs = (C.c_void_p * (3 * G))(*([packed or 256 * 4096] * (3 * G)))
    B = M.Block_t(cfg.H, cfg.F, cfg.E, cfg.k, cfg.n_shared, cfg.F_shared, M.act_code(cfg.act),
                  C.cast(arr, C.POINTER(M.Scheme_t)), C.cast(ptrs, C.POINTER(C.c_void_p)))
    return B, (arr, ptrs)


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_workspace_layout(lib, name):
    cfg = W.CONFIGS[name]
    B, keep = _block(name)
    T = cfg.T
    total = lib.mxmoe_workspace_bytes(C.byref(B), T)
    lay = M.WsLayout_t()
    assert lib.mxmoe_workspace_layout(C.byref(B), T, C.byref(lay)) == M.OK
    assert lay.total == total
    none = (1 << 64) - 1
    P = T * cfg.k
    regions = [(lay.h, 2 * P * cfg.F), (lay.slots, 4 * T * (cfg.k + cfg.n_shared) * cfg.H),
               (lay.sorted_pair, 4 * P), (lay.inv, 4 * P)]
    for off, size in regions:
        assert off % 256 == 0 and off + size <= total
    # a8/a4 code buffers exist exactly when some linear needs them
    sch = W.schemes_of(cfg)
    assert (lay.xq8 != none) == any(t[0] == W.W8A8 for t in sch)
    assert (lay.xq4 != none) == any(t[0] == W.W4A4 for t in sch)
    # table: 3 linears x 32 bytes per expert
    assert lib.mxmoe_block_table_bytes(C.byref(B)) == 96 * (cfg.E + cfg.n_shared)
    host = (C.c_uint8 * (96 * (cfg.E + cfg.n_shared)))()
    assert lib.mxmoe_block_table_fill(C.byref(B), host, len(host)) == M.OK


def test_block_validation(lib):
    cfg = W.CONFIGS["tiny"]
    sch = W.schemes_of(cfg)
    mixed = [list(t) for t in sch]
    mixed[0][1] = W.W8A8                                 # gate != up
    B, keep = _block("tiny", [tuple(t) for t in mixed])
    assert lib.mxmoe_workspace_bytes(C.byref(B), 64) == 0
    B, keep = _block("tiny")
    B.top_k = 5                                          # k > E
    assert lib.mxmoe_workspace_bytes(C.byref(B), 64) == 0
    B, keep = _block("tiny")
    B.hidden = 200
    p = C.c_void_p(1 << 20)
    assert lib.mxmoe_moe_forward(C.byref(B), p, 64, p, p, p, p, p, 10 ** 9, None) == M.ERR_UNSUPPORTED
    B, keep = _block("tiny")
    assert lib.mxmoe_moe_forward(C.byref(B), p, 64, p, p, p, p, p, 16, None) == M.ERR_WORKSPACE
    assert lib.mxmoe_moe_forward(C.byref(B), p, 64, None, p, p, p, p, 10 ** 9, None) == M.ERR_INVALID_ARG
    assert lib.mxmoe_moe_forward(C.byref(B), p, 0, None, None, None, None, None, 0, None) == M.OK  # T = 0
    B, keep = _block("tiny", packed=256 * 4096 + 16)     # misaligned packed pointer
    host = (C.c_uint8 * 384)()
    assert lib.mxmoe_block_table_fill(C.byref(B), host, len(host)) == M.ERR_INVALID_ARG


def test_status_strings(lib):
    for s in range(5):
        assert lib.mxmoe_status_string(s)


def test_router_validation(lib):
    p = C.c_void_p(1 << 20)
    f = lib.mxmoe_router_topk
    assert f(p, 4, 8, 0, 0, None, 0, p, p, None, None) == M.ERR_INVALID_ARG     # k = 0
    assert f(p, 4, 8, 9, 0, None, 0, p, p, None, None) == M.ERR_INVALID_ARG     # k > E
    assert f(p, 4, 100, 65, 0, None, 0, p, p, None, None) == M.ERR_INVALID_ARG  # k > 64
    assert f(p, 4, 1025, 2, 0, None, 0, p, p, None, None) == M.ERR_INVALID_ARG  # E > 1024
    assert f(p, 4, 8, 2, 2, None, 0, p, p, None, None) == M.ERR_INVALID_ARG     # renormalize not 0/1
    assert f(p, 4, 8, 2, 0, p, 65, p, p, p, None) == M.ERR_INVALID_ARG          # n_shared > 64
    assert f(p, 4, 8, 2, 0, p, 1, p, p, None, None) == M.ERR_INVALID_ARG        # shared gates without output
    assert f(None, 4, 8, 2, 0, None, 0, p, p, None, None) == M.ERR_INVALID_ARG
    assert f(C.c_void_p((1 << 20) + 2), 4, 8, 2, 0, None, 0, p, p, None, None) == M.ERR_INVALID_ARG
    assert f(None, 0, 8, 2, 0, None, 0, None, None, None, None) == M.OK          # T = 0


def test_forward_router_mode_validation(lib):
    B, keep = _block("tiny")
    p = C.c_void_p(1 << 20)
    o = M.ForwardOpts_t()
    o.router_logits = p
    o.renormalize = 3
    assert lib.mxmoe_moe_forward_ex(C.byref(B), p, 64, p, None, None, p, p, 10 ** 9, C.byref(o), None) == \
        M.ERR_INVALID_ARG
    o.renormalize = 0
    o.shared_w = p                          # direct shared weights belong to the ids mode
    assert lib.mxmoe_moe_forward_ex(C.byref(B), p, 64, p, None, None, p, p, 10 ** 9, C.byref(o), None) == \
        M.ERR_INVALID_ARG
    o2 = M.ForwardOpts_t()
    o2.shared_logits = p                    # gate logits need router mode
    assert lib.mxmoe_moe_forward_ex(C.byref(B), p, 64, p, p, p, p, p, 10 ** 9, C.byref(o2), None) == \
        M.ERR_INVALID_ARG
    o3 = M.ForwardOpts_t()                  # ids mode without ids
    assert lib.mxmoe_moe_forward_ex(C.byref(B), p, 64, p, None, None, p, p, 10 ** 9, C.byref(o3), None) == \
        M.ERR_INVALID_ARG


@pytest.mark.parametrize("s", W.ALL_SCHEMES)
def test_pack_operand_extent_is_checked(s):
    """The binding refuses operands smaller than what the packer reads."""
    q = W.quantize_linear(W.draw_weight(2, 0, 0, 32, 256), s)
    M.check_operands(q)                                   # the generator's own operands fit
    if q.scales is not None:
        short = W.QLinear(s, q.n, q.k, q.codes, q.scales.reshape(-1)[: q.scales.size // 2], q.zeros)
        with pytest.raises(ValueError):
            M.check_operands(short)
    with pytest.raises(ValueError):
        M.check_operands(W.QLinear(s, q.n, q.k, q.codes.reshape(-1)[:10], q.scales, q.zeros))
    # the wrong format's scales (w4a4-g128's fp16 [n, k/128] for mxfp4) are refused
    if s == W.MXFP4:
        g = W.quantize_linear(W.draw_weight(2, 0, 0, 32, 256), W.W4A4G128)
        with pytest.raises(ValueError):
            M.check_operands(W.QLinear(s, q.n, q.k, q.codes, g.scales))


def test_activation_buffers_beyond_4gib_are_rejected(lib):
    """The Group-GEMM addresses activation rows with 32-bit byte offsets: a
    forward whose x, routed h or shared h would reach 4 GiB, and a single
    linear whose input would, return UNSUPPORTED before anything is enqueued
    (the pointers are never dereferenced)."""
    p = C.c_void_p(1 << 20)
    B, keep = _block("mixtral")
    T_ok, T_big = 65536, 81920                  # routed h: T * 2 * 14336 * 2 bytes
    assert 2 * T_ok * 2 * 14336 < 1 << 32 <= 2 * T_big * 2 * 14336
    assert lib.mxmoe_moe_forward(C.byref(B), p, T_big, p, p, p, p, p, 1 << 62, None) == M.ERR_UNSUPPORTED
    assert lib.mxmoe_moe_forward(C.byref(B), p, T_ok, p, p, p, p, p, 16, None) == M.ERR_WORKSPACE
    B2, keep2 = _block("qwen2")                 # shared h: T * 20480 * 2 bytes
    assert lib.mxmoe_moe_forward(C.byref(B2), p, 1 << 17, p, p, p, p, p, 1 << 62, None) == M.ERR_UNSUPPORTED
    L = _L(W.W8A8, 256, 16384)                  # linear input m * k * 2 bytes
    assert lib.mxmoe_linear_forward(C.byref(L), M.BF16, p, 1 << 17, p, p, p, 1 << 62, None) == M.ERR_UNSUPPORTED


def test_forward_reserved_options_must_be_zero(lib):
    B, keep = _block("tiny")
    p = C.c_void_p(1 << 20)
    for field in ("reserved0", "reserved1", "fp32_slots"):
        o = M.ForwardOpts_t()
        setattr(o, field, 2 if field == "fp32_slots" else 1)   # fp32_slots takes 0 or 1
        assert lib.mxmoe_moe_forward_ex(C.byref(B), p, 64, p, p, p, p, p, 10 ** 9, C.byref(o), None) == \
            M.ERR_INVALID_ARG


def test_noalloc_validation(lib):
    """mxmoe_moe_forward_noalloc validates on the host: a block whose
    workspace exceeds the scratch array gets WORKSPACE, T = 0 is a no-op."""
    B, keep = _block("qwen2")
    p = C.c_void_p(1 << 20)
    assert lib.mxmoe_workspace_bytes(C.byref(B), 4096) > M.NOALLOC_SCRATCH_BYTES
    assert lib.mxmoe_moe_forward_noalloc(C.byref(B), p, 4096, p, p, p, p, None) == M.ERR_WORKSPACE
    assert lib.mxmoe_moe_forward_noalloc(C.byref(B), p, 0, p, p, p, p, None) == M.OK
    assert lib.mxmoe_moe_forward_noalloc(C.byref(B), p, -1, p, p, p, p, None) == M.ERR_INVALID_ARG
