"""Stage-wise parity of one block forward against the CPU oracle (tests only).

A forward is checked in the order its stages run, each stage on the operands
it actually received (read back from the workspace):

  A  gate|up + SiLU gate: the GPU's h against the oracle's fp64
     h64 = SiLU(x Wg^T) (x Wu^T) of the same rows, element by element within
     tolerance.h_tolerance (one unit in the last place of the activation
     dtype plus 2^-12 of the row's largest |h|);
  B  down-projection activation encodings (a8 / a4 / per-128-group / FP8 /
     MXFP4): the oracle's encoder applied to the GPU's h, byte for byte;
  C  down projection: the oracle's down linear on the GPU's h (so on exactly
     the codes of B), times the router gate weight, against the GPU's slot
     rows (rounded to the activation dtype, or fp32 when the forward kept
     them so) - bit for bit for w8a8 / w4a4 (their fp32 epilogue products
     are evaluated here in IEEE float32 in the kernel's order, then rounded
     the same way), within the accumulation models of tolerance.py plus the
     slot rounding for the other kinds;
  D  combine: the GPU's slot rows widened to fp32, summed in fp32 in slot
     order (dropped pairs skipped) and rounded once to the activation dtype,
     evaluated here in IEEE float32: bit for bit;
  E  end to end, against the oracle alone (its own rounded h): every row
     within REL_TOL of its largest |y|, no slack.  Where h sits near a
     rounding midpoint, the GPU's fp32 h and the oracle's fp64 h can round
     to neighbouring values, and a down projection that quantizes its input
     can then see other codes (a scale moves when the row maximum is such an
     element).  Both are correct evaluations of the method, so a row outside
     the bar is accepted only if (i) the GPU's h passed A, (ii) its down
     codes differ from those of the oracle's rounded h in that token, and
     (iii) the row is within REL_TOL of the oracle evaluated on the GPU's h
     (the sum of the C references).  Such rows are counted and reported.
"""

from __future__ import annotations

import numpy as np

from oracle import mxmoe_oracle as O
from tests import tolerance as TL

REL_TOL = 1e-2


def _ws(mb, T, name, dtype, count):
    v = mb.ws_view(name, dtype, count, T)
    return None if v is None else v.cpu().numpy()


def _act16(raw, act):
    """int16 storage -> exact fp64 values."""
    return O.act_values(raw.view(np.float16) if act == "fp16" else raw.view(np.uint16), act)


def _down_kind(s):
    fmt = getattr(s, "fmt", 0)
    if fmt == 1:
        return "mx"
    if fmt == 2:
        return "fp8"
    if fmt == 3:
        return "f6"
    if s.a_bits < 16 and s.a_group > 0:
        return "g"
    if s.a_bits < 16:
        return "int"
    return "float"


# e2m3 codes of the integers -7..7 from the bit-field definition (sign bit 5,
# two exponent bits of bias 1, three mantissa bits): |v| = (1 + m/8) 2^(e-1)
_E2M3_OF = {}
for _e in range(1, 4):
    for _m in range(8):
        _v = (1 + _m / 8) * 2.0 ** (_e - 1)
        if _v == int(_v) and _v <= 7:
            _E2M3_OF[int(_v)] = (_e << 3) | _m
_E2M3_OF[0] = 0


def f6_bytes(q):
    """int4 codes [rows, cols] -> the FP6 byte layout of the workspace: per 32
    elements 24 bytes of 6-bit e2m3 codes (element i at bits 6i..6i+5, little
    endian) followed by 8 zero bytes."""
    q = np.asarray(q, dtype=np.int64)
    rows, cols = q.shape
    code = np.vectorize(lambda v: (0x20 if v < 0 else 0) | _E2M3_OF[abs(int(v))], otypes=[np.int64])(q)
    g = code.reshape(rows, cols // 32, 32)
    out = np.zeros((rows, cols // 32, 32), np.uint8)
    bits = np.zeros((rows, cols // 32), dtype=object)
    for i in range(32):
        bits = bits + (g[:, :, i].astype(object) << (6 * i))
    for b in range(24):
        out[:, :, b] = np.vectorize(lambda x: (x >> (8 * b)) & 0xFF, otypes=[np.uint8])(bits)
    return out.reshape(rows, cols)


def _codes(h32, s):
    """The oracle's encoding of h rows for a down linear of scheme s:
    (codes, scales) in the layout the workspace holds."""
    kind = _down_kind(s)
    if kind == "int":
        return O.act_quant(h32, (1 << (s.a_bits - 1)) - 1)
    if kind == "f6":
        q, sc = O.act_quant(h32, 7)
        return f6_bytes(q), sc
    if kind == "g":
        return O.act_quant_groups(h32, (1 << (s.a_bits - 1)) - 1, s.a_group)
    if kind == "fp8":
        return O.fp8_quant(h32)
    if kind == "mx":
        q, e = O.mx_quant(h32, s.a_group)
        return (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8), e
    return None, None


def _down_ref(hv, lin, act, gw):
    """C reference of one group: (fp64 value * gw, exact-emulation float32 or
    None, per-element bound or None)."""
    kind = _down_kind(lin.scheme)
    gw64 = gw.astype(np.float64)[:, None]
    if kind in ("int", "f6"):
        h32 = hv.astype(np.float32)
        qa, sa = O.act_quant(h32, (1 << (lin.scheme.a_bits - 1)) - 1)
        acc = O.linear(hv, lin, act, return_int=True)
        # the kernel's epilogue: ((float)acc * s_a) * s_w, then * gate weight
        f = ((acc.astype(np.float32) * sa[:, None]).astype(np.float32) * lin.scales[None, :]).astype(np.float32)
        f = (f * gw.astype(np.float32)[:, None]).astype(np.float32)
        val = acc.astype(np.float64) * sa.astype(np.float64)[:, None] * lin.scales.astype(np.float64)[None, :]
        return val * gw64, f, None
    val = O.linear(hv, lin, act)
    wd = O.dequant(lin, act)
    if kind == "fp8":
        qa, sa = O.fp8_quant(hv.astype(np.float32))
        bound = TL.fp8_block_bound(O.e4m3_values(qa) * sa.astype(np.float64)[:, None], wd)
    elif kind == "mx":
        qa, ea = O.mx_quant(hv.astype(np.float32), lin.scheme.a_group)
        bound = TL.acc_bound(np.abs(O._mx_values(qa, ea, lin.scheme.a_group)), np.abs(wd))
    elif kind == "g":
        qa, sa = O.act_quant_groups(hv.astype(np.float32), (1 << (lin.scheme.a_bits - 1)) - 1, lin.scheme.a_group)
        ad = (qa.astype(np.float64).reshape(qa.shape[0], -1, lin.scheme.a_group)
              * sa.astype(np.float64)[..., None]).reshape(qa.shape)
        bound = TL.acc_bound(np.abs(ad), np.abs(wd))
    else:
        bound = TL.acc_bound(np.abs(hv), np.abs(wd))
    # the epilogue's fp32 products (scales, gate weight) add a few roundings
    return val * gw64, None, (bound + 4 * TL.U32 * np.abs(val)) * np.abs(gw64) + 1e-30


class Report(dict):
    def line(self):
        return ", ".join(f"{k}={v}" for k, v in self.items())


def check_forward(mb, blk, y, shared_w=None, chunk=4096, log=None) -> Report:
    """Run every stage check on a finished forward (mb: MoEBlock, blk: its
    inputs, y: the output tensor).  Asserts; returns a report of the worst
    ratios and the rows accepted through (E)."""
    import torch
    cfg = blk.cfg
    act = cfg.act
    T, k, E, nsh, H = cfg.T, cfg.k, cfg.E, cfg.n_shared, cfg.H
    S = k + nsh
    r = O.route(blk.topk_ids, E)
    P = T * k
    xv = O.act_values(blk.x, act)
    ynp = y.detach().contiguous().view(torch.int16).cpu().numpy()
    y_gpu = _act16(ynp, act)
    slots = mb.slot_rows(T)                      # float32 (16-bit slots widen exactly)
    slot16 = mb.slot_dtype() != torch.float32
    h_r = _ws(mb, T, "h", torch.int16, P * cfg.F).reshape(P, cfg.F) if P else None
    h_s = _ws(mb, T, "h_shared", torch.int16, nsh * T * cfg.F_shared).reshape(nsh, T, cfg.F_shared) if nsh else None

    cache = {}

    def buf(name, dtype, rows, cols):
        """A workspace buffer [rows, cols], copied to the host once."""
        key = (name, str(dtype))
        if key not in cache:
            cache[key] = _ws(mb, T, name, dtype, rows * cols).reshape(rows, cols)
        return cache[key]

    def enc_buffers(s, shared, rows_lo, rows_hi, j, F):
        """The GPU's encoding of h rows [rows_lo, rows_hi) of a group."""
        kind = _down_kind(s)
        pre = "" if not shared else "_shared"
        nrows = P if not shared else nsh * T
        base = 0 if not shared else j * T
        lo, hi = base + rows_lo, base + rows_hi
        if kind in ("int", "fp8", "g", "f6"):
            q = buf("hq" + pre, torch.int8, nrows, F)[lo:hi]
            if kind in ("fp8", "f6"):
                q = q.view(np.uint8)
            if kind == "g":
                return q, buf("hsg" + pre, torch.float32, nrows, F // 128)[lo:hi]
            return q, buf("hs" + pre, torch.float32, nrows, 1)[lo:hi, 0]
        if kind == "mx":
            return (buf("hqmx" + pre, torch.uint8, nrows, F // 2)[lo:hi],
                    buf("hsmx" + pre, torch.uint8, nrows, F // 32)[lo:hi])
        return None, None

    y_pure = np.zeros((T, H))
    y_alt = np.zeros((T, H))
    codes_moved = np.zeros(T, dtype=bool)
    rep = Report(h_ratio=0.0, h_moved=0, slot_ratio=0.0, int_slots_exact=0, rows_via_E=0)
    topw = blk.topk_w

    def one_group(g, rows_x, lins, gw, slot_idx, h_gpu_rows, shared, j, tok, row_base):
        gate, up, down = lins
        F = gate.n
        wg = O.dequant(gate, act) if gate.scheme.a_bits == 16 else None
        wu = O.dequant(up, act) if up.scheme.a_bits == 16 else None
        for c0 in range(0, len(rows_x), chunk):
            c1 = min(len(rows_x), c0 + chunk)
            a = xv[rows_x[c0:c1]]
            h64 = O.silu(O.linear(a, gate, act, wg)) * O.linear(a, up, act, wu)
            hb = O.round_to_act(h64, act)
            hg = _act16(h_gpu_rows[c0:c1], act)
            # A
            tol = TL.h_tolerance(h64, act)
            d = np.abs(hg - h64)
            if d.size:
                rep["h_ratio"] = max(rep["h_ratio"], float((d / tol).max()))
            if not np.all(d <= tol):
                i, f = np.argwhere(d > tol)[0]
                raise AssertionError(f"stage A, group {g}: h[{c0 + i}, {f}] gpu={hg[i, f]!r} exact={h64[i, f]!r} "
                                     f"tol={tol[i, f]!r}")
            moved = (hg != hb).any(axis=1)
            rep["h_moved"] += int(moved.sum())
            # B
            qr, sr = _codes(hg.astype(np.float32), down.scheme)
            if qr is not None:
                qg, sg = enc_buffers(down.scheme, shared, row_base + c0, row_base + c1, j, F)
                qg = qg.view(qr.dtype) if qg.dtype != qr.dtype else qg
                if not np.array_equal(qg, qr):
                    bad = np.argwhere(qg != qr)
                    i, f = bad[0]
                    raise AssertionError(
                        f"stage B, group {g}: {len(bad)} down codes of the GPU's h differ from the oracle's "
                        f"encoder; first row {c0 + i} col {f}: gpu {int(qg[i, f])} oracle {int(qr[i, f])}, "
                        f"h {hg[i, f]!r}, gpu scale {np.asarray(sg)[i]!r} oracle scale {np.asarray(sr)[i]!r}, "
                        f"rows with a difference {len(np.unique(bad[:, 0]))} of {qr.shape[0]}")
                if sr.dtype == np.float32:
                    assert TL.f32_bits_equal(sg, sr), f"stage B, group {g}: down scales differ"
                else:
                    assert np.array_equal(sg, sr), f"stage B, group {g}: E8M0 bytes differ"
                # (E ii) does the oracle's own rounded h give other codes?
                if moved.any():
                    qb, sb = _codes(hb[moved].astype(np.float32), down.scheme)
                    diff = (qb != qr[moved]).reshape(int(moved.sum()), -1).any(axis=1)
                    diff |= (np.asarray(sb).reshape(int(moved.sum()), -1)
                             != np.asarray(sr[moved]).reshape(int(moved.sum()), -1)).any(axis=1)
                    codes_moved[tok[c0:c1][moved][diff]] = True
            # C
            gwc = gw[c0:c1]
            ref, exact32, bound = _down_ref(hg, down, act, gwc)
            got = slots[tok[c0:c1], slot_idx[c0:c1]]
            if exact32 is not None:
                if slot16:
                    exact32 = O.round_to_act(exact32.astype(np.float64), act).astype(np.float32)
                if not TL.f32_bits_equal(got, exact32):
                    i, n = np.argwhere(got.view(np.uint32) != exact32.view(np.uint32))[0]
                    raise AssertionError(f"stage C, group {g}: int slot [{c0 + i}, {n}] gpu={got[i, n]!r} "
                                         f"emulated={exact32[i, n]!r}")
                rep["int_slots_exact"] += int(got.size)
            else:
                if slot16:
                    bound = TL.slot_bound(ref, bound, act)
                e = np.abs(got.astype(np.float64) - ref)
                if e.size:
                    rep["slot_ratio"] = max(rep["slot_ratio"], float((e / bound).max()))
                if not np.all(e <= bound):
                    i, n = np.argwhere(e > bound)[0]
                    raise AssertionError(f"stage C, group {g}: slot [{c0 + i}, {n}] gpu={got[i, n]!r} "
                                         f"ref={ref[i, n]!r} bound={bound[i, n]!r}")
            np.add.at(y_alt, tok[c0:c1], ref)
            if moved.any():
                ref_b = ref.copy()
                ref_b[moved] = _down_ref(hb[moved], down, act, gwc[moved])[0]
                np.add.at(y_pure, tok[c0:c1], ref_b)
            else:
                np.add.at(y_pure, tok[c0:c1], ref)

    for e in range(E):
        lo, hi = int(r["offsets"][e]), int(r["offsets"][e + 1])
        if hi == lo:
            continue
        pairs = r["sorted_pair"][lo:hi].astype(np.int64)
        tok = pairs // k
        one_group(e, tok, blk.linears[e], topw.reshape(-1)[pairs], pairs % k, h_r[lo:hi], False, 0, tok, lo)
        if log:
            log(f"  group {e}: {hi - lo} rows checked")
    for j in range(nsh):
        tok = np.arange(T)
        gw = np.ones(T, np.float32) if shared_w is None else np.asarray(shared_w, np.float32)[:, j]
        one_group(E + j, tok, blk.linears[E + j], gw, np.full(T, k + j), h_s[j], True, j, tok, 0)
        if log:
            log(f"  shared {j}: {T} rows checked")

    # D: the combine, emulated in float32 in slot order
    acc = np.zeros((T, H), np.float32)
    valid = np.concatenate([(blk.topk_ids >= 0) & (blk.topk_ids < E), np.ones((T, nsh), bool)], axis=1)
    for s in range(S):
        # (rows of dropped pairs hold whatever the workspace held: never added)
        acc = np.where(valid[:, s:s + 1], (acc + np.where(valid[:, s:s + 1], slots[:, s], 0)).astype(np.float32), acc)
    want = O.round_to_act(acc.astype(np.float64), act)
    if not np.array_equal(want, y_gpu):
        t, h = np.argwhere(want != y_gpu)[0]
        raise AssertionError(f"stage D: y[{t}, {h}] gpu={y_gpu[t, h]!r} fp32 sum of slots rounds to {want[t, h]!r}")

    # E
    scale = np.abs(y_pure).max(axis=1, keepdims=True)
    err = np.abs(y_gpu - y_pure)
    rep["e2e_ratio"] = float((err / np.maximum(REL_TOL * scale, 1e-300)).max()) if err.size else 0.0
    bad = (err > REL_TOL * scale).any(axis=1)
    if bad.any():
        alt_scale = np.abs(y_alt).max(axis=1, keepdims=True)
        alt_ok = (np.abs(y_gpu - y_alt) <= REL_TOL * alt_scale).all(axis=1)
        unexplained = bad & ~(codes_moved & alt_ok)
        if unexplained.any():
            t = int(np.nonzero(unexplained)[0][0])
            raise AssertionError(f"stage E: token {t} off by {float(err[t].max() / scale[t, 0]):.4g} of its row max "
                                 f"(down codes moved: {bool(codes_moved[t])}, within the bar on the GPU's h: "
                                 f"{bool(alt_ok[t])})")
        rep["rows_via_E"] = int(bad.sum())
    rep["tokens"] = T
    rep["h_ratio"] = round(rep["h_ratio"], 4)
    rep["slot_ratio"] = round(rep["slot_ratio"], 4)
    rep["e2e_ratio"] = round(rep["e2e_ratio"], 4)
    return rep


def check_pure(y_np, ref_y, act, what=""):
    """End-to-end comparison of act-dtype outputs against an oracle output,
    REL_TOL of each row's largest |y|, no slack.  Returns the worst ratio."""
    yv = O.act_values(y_np, act)
    scale = np.abs(ref_y).max(axis=1, keepdims=True)
    err = np.abs(yv - ref_y)
    bad = err > REL_TOL * scale
    if bad.any():
        t, h = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} outputs out of tolerance; first t={t} h={h} "
                             f"gpu={yv[t, h]!r} ref={ref_y[t, h]!r} rowmax={scale[t, 0]!r}")
    return float((err / np.maximum(REL_TOL * scale, 1e-300)).max()) if err.size else 0.0
