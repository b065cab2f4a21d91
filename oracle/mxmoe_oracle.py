"""CPU oracle for the MxMoE mixed-precision MoE block forward (arXiv 2505.05799).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, links or runs
this module: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` use it.  It shares no code with the HIP path and imports
nothing but numpy.

What it computes is the plain definition of the MoE block, on the same quantized
operands the GPU receives (codes, scales, zeros - never the packed layout):

* Sec. 2.2, Eq. (1)-(2): each routed expert e maps its tokens X_e through
  W_down( SiLU(W_gate X_e) * W_up X_e ); the block output is the sum over the
  token's experts of that result times the router gate weight w_e.  Shared
  experts are dense experts over every token with weight 1.
* Sec. 2.1 min-max quantizer and the weight storage of Sec. 5.2: a wNg128 weight
  dequantizes to s * (q - z) per group of 128 along K; a per-channel symmetric
  weight (w8a8 / w4a4, Fig. 4 caption) to s_w[n] * q.
* Sec. 2.2, Eq. (2), router front-end: the gate weights are the router's
  softmax probabilities of the token's k largest logits (optionally
  renormalised over those k); a shared expert's output may be scaled by a
  per-token sigmoid gate (Qwen-MoE style shared experts).
* MXFP4 (the OCP Microscaling format the MI355X matrix cores take natively; the
  paper's scheme set S is whatever the hardware supports, Sec. 4.2.1): a value is
  an FP4 e2m1 element times a power-of-two scale shared by 32 consecutive
  values along K; activations get the same encoding at run time.
* FP8 (OCP e4m3, the 8-bit floating-point operand of the MI355X matrix cores;
  again a member of the hardware's scheme set, Sec. 4.2.1): a weight is an e4m3
  value times a per-channel fp32 scale, an activation an e4m3 value times a
  per-token fp32 scale that maps the row's largest magnitude onto 448.
* Sec. 4.2.2 (end): activations of w8a8 / w4a4 linears are quantized dynamically
  at run time, per token (a_gsize = -1 in the W5A5 allocation table), with the
  fp32 recipe of :func:`act_quant`.

Floating point runs in fp64; integer GEMMs are exact (fp64 BLAS on integer
values, every partial sum < 2^53).  Rounding points mirrored from the GPU
contract: the gated intermediate h is rounded once to the activation dtype
before the down projection; a8/a4 down projections quantize that rounded h.
The block output is returned unrounded in fp64.

Parity pins live in ``tests/test_oracle.py``.
"""

from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "bf16_bits_to_f64", "round_to_act", "act_values", "route", "router_topk", "shared_gate", "dequant",
    "act_quant", "fp8_quant", "e4m3_values", "e4m3_code", "linear", "moe_forward", "lpt_makespan", "optimal_makespan",
    "silu", "tile_plan", "scheme_index", "xcd_queues", "xcd_tiles",
]

# ----------------------------------------------------------------------------
# dtype handling (own implementation; the GPU path has its own)
# ----------------------------------------------------------------------------


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp64 values."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def act_values(a: np.ndarray, act: str) -> np.ndarray:
    """Activation-dtype storage (float16 array or bf16 bits) -> exact fp64 values."""
    if act == "fp16":
        return np.asarray(a, dtype=np.float16).astype(np.float64)
    if act == "bf16":
        return bf16_bits_to_f64(a)
    raise ValueError(act)


def round_to_act(x: np.ndarray, act: str) -> np.ndarray:
    """Round fp64 values to the nearest activation-dtype value (ties to even).

    Returns fp64 values that are exactly representable in the target dtype.
    fp16 uses numpy's correctly rounded float64 -> float16 cast.  bf16 keeps 8
    significant bits: the value is snapped to multiples of 2^(e-8) where
    x = m * 2^e with 0.5 <= |m| < 1 (subnormal spacing 2^-133).
    """
    x = np.asarray(x, dtype=np.float64)
    if act == "fp16":
        return x.astype(np.float16).astype(np.float64)
    if act != "bf16":
        raise ValueError(act)
    _, e = np.frexp(x)
    spacing = np.ldexp(1.0, np.maximum(e - 8, -133))
    r = np.rint(x / spacing) * spacing
    # values that round past the largest finite bf16 become inf (never hit here)
    big = np.abs(r) > 3.3895313892515355e38
    return np.where(big, np.copysign(np.inf, x), r)


# ----------------------------------------------------------------------------
# O1: routing / permutation (Eq. 2: which tokens form X_e)
# ----------------------------------------------------------------------------


def route(topk_ids: np.ndarray, E: int) -> Dict[str, np.ndarray]:
    """Stable grouping of the T*k (token, slot) pairs by expert.

    Pair id p = t*k + s.  Pairs are ordered by (expert, p); pairs whose expert
    id is outside [0, E) are dropped (they contribute nothing to the output).
    Returns counts [E], offsets [E+1], sorted_pair [#valid], inv [T*k]
    (position of pair p in sorted order, -1 if dropped), bad [#pairs] bool.
    """
    e = np.asarray(topk_ids, dtype=np.int64).ravel()
    P = e.size
    p = np.arange(P, dtype=np.int64)
    bad = (e < 0) | (e >= E)
    good = ~bad
    order = np.lexsort((p[good], e[good]))           # primary key: expert, then pair
    sorted_pair = p[good][order]
    counts = np.bincount(e[good], minlength=E)[:E]
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    inv = np.full(P, -1, dtype=np.int64)
    inv[sorted_pair] = np.arange(sorted_pair.size)
    return {
        "counts": counts.astype(np.int32),
        "offsets": offsets.astype(np.int32),
        "sorted_pair": sorted_pair.astype(np.int32),
        "inv": inv.astype(np.int32),
        "bad": bad,
    }


def router_topk(logits: np.ndarray, k: int, renormalize: bool = False) -> Tuple[np.ndarray, np.ndarray]:
    """Router front-end of Eq. (2) on fp32 logits [T, E].

    The chosen experts are the k largest logits, in decreasing order, ties to
    the lower expert id (softmax is increasing, so this is the top-k of the
    probabilities).  Weights: p_e = exp(l_e - max l) / sum exp(l - max l) in
    fp64, or with ``renormalize`` the chosen exp(l - max l) over their own sum.
    Returns ids int32 [T, k] and weights fp64 [T, k].
    """
    l = np.asarray(logits, dtype=np.float32).astype(np.float64)
    T, E = l.shape
    order = np.argsort(-l, axis=1, kind="stable")[:, :k]     # stable: equal logits keep id order
    ex = np.exp(l - l.max(axis=1, keepdims=True))
    sel = np.take_along_axis(ex, order, axis=1)
    den = sel.sum(axis=1, keepdims=True) if renormalize else ex.sum(axis=1, keepdims=True)
    return order.astype(np.int32), sel / den


def shared_gate(logits: np.ndarray) -> np.ndarray:
    """Sigmoid gate of the shared experts, 1 / (1 + exp(-l)), fp64."""
    l = np.asarray(logits, dtype=np.float32).astype(np.float64)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-l))


# ----------------------------------------------------------------------------
# O2: weight dequantization (Sec. 2.1 quantizer, Sec. 5.2 storage)
# ----------------------------------------------------------------------------


def _is_weight_only(s) -> bool:
    return s.w_bits < 16 and s.a_bits == 16


def dequant(lin, act: str) -> np.ndarray:
    """Exact fp64 value of every weight of a quantized linear, [n, k]."""
    s = lin.scheme
    if s.w_bits == 16:
        w = bf16_bits_to_f64(lin.codes)
        if act == "fp16":
            # the 16-bit weights feed an fp16 MFMA: they are converted to fp16 once
            w = w.astype(np.float16).astype(np.float64)
        return w
    if _is_weight_only(s):
        g = s.w_group
        q = lin.codes.astype(np.float64).reshape(lin.n, lin.k // g, g)
        sc = lin.scales.astype(np.float64)[..., None]
        z = lin.zeros.astype(np.float64)[..., None]
        return (sc * (q - z)).reshape(lin.n, lin.k)
    if getattr(s, "fmt", 0) == 1:  # MXFP4: e2m1 element times 2^(E8M0 - 127) of its 32-block
        return _mx_values(lin.codes, lin.scales, s.w_group)
    if getattr(s, "fmt", 0) == 2:  # FP8: e4m3 element times the channel's fp32 scale
        return e4m3_values(lin.codes) * lin.scales.astype(np.float64)[:, None]
    if s.w_group > 0:  # symmetric groups (w4a4-g128): code times its group's scale
        g = s.w_group
        q = lin.codes.astype(np.float64).reshape(lin.n, lin.k // g, g)
        return (q * lin.scales.astype(np.float64)[..., None]).reshape(lin.n, lin.k)
    return lin.codes.astype(np.float64) * lin.scales.astype(np.float64)[:, None]


# FP4 e2m1: sign bit 3, two exponent bits (bias 1), one mantissa bit
_E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def _mx_values(codes: np.ndarray, exps: np.ndarray, block: int) -> np.ndarray:
    c = np.asarray(codes, dtype=np.int64)
    v = _E2M1[c & 7] * np.where(c & 8, -1.0, 1.0)
    r, k = v.shape
    sc = np.exp2(np.asarray(exps, dtype=np.float64) - 127.0)
    return (v.reshape(r, k // block, block) * sc[..., None]).reshape(r, k)


def _mx_exponent(amax: np.ndarray) -> np.ndarray:
    """Shared exponent floor(log2(amax)) - 2 in [-127, 127]; -127 for amax = 0."""
    e = np.full(np.shape(amax), -127, dtype=np.int64)
    nz = amax > 0
    e[nz] = np.floor(np.log2(amax[nz])).astype(np.int64) - 2
    return np.clip(e, -127, 127)


def _e2m1_code(x: np.ndarray) -> np.ndarray:
    """Magnitude code (0..7) of the e2m1 value nearest to x >= 0; an exact tie
    takes the even code; beyond 6 the code of 6."""
    d = np.abs(np.asarray(x)[..., None] - _E2M1)
    cand = d == d.min(axis=-1, keepdims=True)
    even = cand & (np.arange(8) % 2 == 0)
    code = np.where(even.any(axis=-1), even.argmax(axis=-1), cand.argmax(axis=-1))
    return np.where(np.asarray(x) > 6.0, 7, code)


# FP8 e4m3 (OCP): sign bit 7, four exponent bits (bias 7), three mantissa bits.
# Exponent field 0 holds the subnormals m/8 * 2^-6; there are no infinities and
# the magnitude code 0x7F is NaN, so 0x7E = 448 is the largest finite value.
# Entry c of the table is the value of magnitude code c (0..126), increasing.
_E4M3 = np.array([(m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
                  for e in range(16) for m in range(8)][:127])
E4M3_MAX = 448.0


def e4m3_values(codes: np.ndarray) -> np.ndarray:
    """Exact value of e4m3 codes (uint8; NaN codes are not accepted)."""
    c = np.asarray(codes).astype(np.int64) & 0xFF
    mag = c & 0x7F
    if (mag == 0x7F).any():
        raise ValueError("e4m3 NaN code")
    return np.where(c & 0x80, -1.0, 1.0) * _E4M3[mag]


def e4m3_code(x: np.ndarray) -> np.ndarray:
    """Magnitude code (0..126) of the e4m3 value nearest to x >= 0; an exact
    tie takes the even code; at and beyond 448 the code of 448."""
    x = np.asarray(x, dtype=np.float64)
    hi = np.clip(np.searchsorted(_E4M3, x, side="left"), 1, 126)   # _E4M3[hi-1] < x <= _E4M3[hi]
    lo = hi - 1
    dl = x - _E4M3[lo]
    dh = _E4M3[hi] - x
    code = np.where(dl < dh, lo, np.where(dh < dl, hi, np.where(lo % 2 == 0, lo, hi)))
    return np.where(x >= E4M3_MAX, 126, code)


def fp8_quant(a: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-row FP8 e4m3 encoding of activations, evaluated in IEEE fp32 like
    :func:`act_quant` with 448 in place of qmax: amax = max |a_r|;
    inv = fl32(448 / amax), s = fl32(amax / 448); element = the e4m3 value
    nearest to fl32(a * inv) (ties to the even code, magnitudes past 448 give
    448), the sign kept unless the magnitude code is 0.  An all-zero row gets
    s = 0 and zero codes.  Returns codes uint8 [rows, cols], scales fp32 [rows]."""
    a = np.asarray(a, dtype=np.float32)
    m32 = np.float32(E4M3_MAX)
    amax = np.abs(a).max(axis=1) if a.shape[1] else np.zeros(a.shape[0], np.float32)
    zero = amax == 0
    safe = np.where(zero, np.float32(1), amax).astype(np.float32)
    inv = (m32 / safe).astype(np.float32)
    s = np.where(zero, np.float32(0), (safe / m32).astype(np.float32)).astype(np.float32)
    prod = (a * inv[:, None]).astype(np.float32)
    mag = np.where(zero[:, None], 0, e4m3_code(np.abs(prod)))
    code = np.where((prod < 0) & (mag > 0), mag | 0x80, mag)
    return code.astype(np.uint8), s


def mx_quant(a: np.ndarray, block: int = 32) -> Tuple[np.ndarray, np.ndarray]:
    """MXFP4 encoding of rows of fp32 values, per `block` along the row (OCP MX):
    shared exponent e = floor(log2(amax)) - 2 (2 = the largest e2m1 exponent),
    clamped to [-127, 127], -127 for an all-zero block; element = the e2m1
    value nearest to a / 2^e (ties to the even code; beyond 6 it is 6), sign
    kept unless the magnitude is 0.  Division by 2^e is exact.
    Returns codes uint8 [rows, cols] and E8M0 bytes uint8 [rows, cols/block]."""
    a = np.asarray(a, dtype=np.float32).astype(np.float64)
    r, k = a.shape
    v = a.reshape(r, k // block, block)
    e = _mx_exponent(np.abs(v).max(axis=2))
    code = _e2m1_code(np.abs(v) / np.exp2(e.astype(np.float64))[..., None])
    code = np.where((v < 0) & (code > 0), code | 8, code)
    return code.reshape(r, k).astype(np.uint8), (e + 127).astype(np.uint8)


# ----------------------------------------------------------------------------
# O3: dynamic per-token activation quantization (fp32 recipe)
# ----------------------------------------------------------------------------


def act_quant(a: np.ndarray, qmax: int) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric per-row quantization of activations, evaluated in IEEE fp32.

    amax = max |a_r| (exact).  amax == 0 gives scale 0 and all-zero codes.
    Otherwise inv = fl32(qmax / amax), s = fl32(amax / qmax) (correctly rounded
    divisions) and q = clamp(rne(fl32(a * inv)), -qmax, qmax).
    Returns codes int8 [rows, cols] and scales fp32 [rows].
    """
    a = np.asarray(a, dtype=np.float32)
    q32 = np.float32(qmax)
    amax = np.abs(a).max(axis=1) if a.shape[1] else np.zeros(a.shape[0], np.float32)
    zero = amax == 0
    safe = np.where(zero, np.float32(1), amax).astype(np.float32)
    inv = (q32 / safe).astype(np.float32)
    s = np.where(zero, np.float32(0), (safe / q32).astype(np.float32)).astype(np.float32)
    prod = (a * inv[:, None]).astype(np.float32)
    q = np.clip(np.rint(prod), -qmax, qmax)
    q = np.where(zero[:, None], 0, q)
    return q.astype(np.int8), s


def act_quant_groups(a: np.ndarray, qmax: int, group: int) -> Tuple[np.ndarray, np.ndarray]:
    """The recipe of :func:`act_quant` applied to every block of `group`
    consecutive columns of a row (activation group size of Sec. 4.2.2 and the
    a_gsize column of the W5A5 allocation table).  Returns codes int8
    [rows, cols] and scales fp32 [rows, cols / group]."""
    a = np.asarray(a, dtype=np.float32)
    m, k = a.shape
    q, sc = act_quant(a.reshape(m * (k // group), group), qmax)
    return q.reshape(m, k), sc.reshape(m, k // group)


def _qmax(a_bits: int) -> int:
    return (1 << (a_bits - 1)) - 1


# ----------------------------------------------------------------------------
# O4: one linear y = A W^T on identical operands
# ----------------------------------------------------------------------------


def linear(a: np.ndarray, lin, act: str, w_deq: Optional[np.ndarray] = None,
           return_int: bool = False):
    """A [m, k] holds activation-dtype values as fp64.  Returns fp64 [m, n].

    Weight-only and 16-bit linears: sum_c a[m,c] * w_hat[n,c] in fp64.
    w8a8 / w4a4: codes of A from :func:`act_quant`, exact integer GEMM
    acc = sum_c qa * qw, then acc * s_a[m] * s_w[n] in fp64.  With
    ``return_int`` the exact integer accumulators are returned instead.
    """
    s = lin.scheme
    if getattr(s, "fmt", 0) == 1:
        # MXFP4: both operands decoded exactly, the product summed in fp64
        qa, ea = mx_quant(a.astype(np.float32), s.a_group)
        return _mx_values(qa, ea, s.a_group) @ dequant(lin, act).T
    if getattr(s, "fmt", 0) == 2:
        # FP8: exact sum of the e4m3 products, times s_a[m] * s_w[n]
        qa, sa = fp8_quant(a.astype(np.float32))
        acc = e4m3_values(qa) @ e4m3_values(lin.codes).T
        return acc * sa.astype(np.float64)[:, None] * lin.scales.astype(np.float64)[None, :]
    if s.a_bits < 16 and s.a_group > 0:
        # w4a4-g128: per 128-wide block b, the exact integer dot of the block's
        # codes times s_a[m, b] * s_w[n, b], summed over the blocks in fp64
        g = s.a_group
        qa, sa = act_quant_groups(a.astype(np.float32), _qmax(s.a_bits), g)
        out = np.zeros((a.shape[0], lin.n))
        for b in range(lin.k // g):
            blk = qa[:, b * g:(b + 1) * g].astype(np.float64) @ lin.codes[:, b * g:(b + 1) * g].astype(np.float64).T
            out += blk * sa[:, b].astype(np.float64)[:, None] * lin.scales[:, b].astype(np.float64)[None, :]
        return out
    if s.a_bits < 16:
        qa, sa = act_quant(a.astype(np.float32), _qmax(s.a_bits))
        acc = qa.astype(np.float64) @ lin.codes.astype(np.float64).T
        if return_int:
            return acc.astype(np.int64)
        return acc * sa.astype(np.float64)[:, None] * lin.scales.astype(np.float64)[None, :]
    if w_deq is None:
        w_deq = dequant(lin, act)
    return a @ w_deq.T


def silu(g: np.ndarray) -> np.ndarray:
    """SiLU(g) = g * sigmoid(g) = g / (1 + exp(-g)) in fp64."""
    with np.errstate(over="ignore"):
        return g / (1.0 + np.exp(-g))


# ----------------------------------------------------------------------------
# O5-O7: expert MLP, gate-weighted combine (Eq. 1-2)
# ----------------------------------------------------------------------------

def _expert_mlp(a: np.ndarray, lins: Sequence, act: str):
    """Eq. (1) for one expert on rows a [m, H] (fp64 act values).

    Returns (down output fp64 [m, H], h rounded to act [m, F]).
    """
    gate, up, down = lins
    wg = dequant(gate, act) if gate.scheme.a_bits == 16 else None
    wu = dequant(up, act) if up.scheme.a_bits == 16 else None
    g = linear(a, gate, act, wg)
    u = linear(a, up, act, wu)
    hb = round_to_act(silu(g) * u, act)          # rounding point: h stored in act dtype
    return linear(hb, down, act), hb


def moe_forward(x: np.ndarray, topk_ids: np.ndarray, topk_w: np.ndarray,
                linears: Sequence[Sequence], E: int, act: str,
                return_h: bool = False, shared_w: Optional[np.ndarray] = None):
    """Eq. (2): y[t] = sum_s w[t,s] * Expert_{ids[t,s]}(x[t]) + sum_j g[t,j] * Shared_j(x[t]),
    with g = ``shared_w`` [T, n_shared] (fp32 values) or 1.

    x: [T, H] activations in act storage; topk_ids int32 [T, k]; topk_w fp32
    [T, k]; linears[e] = (gate, up, down) for e < E routed, then shared experts.
    Returns dict with y (fp64, unrounded), the routing and optionally
    per-expert h.
    """
    a_all = act_values(x, act)
    T, H = a_all.shape
    k = topk_ids.shape[1]
    r = route(topk_ids, E)
    w64 = np.asarray(topk_w, dtype=np.float64).ravel()
    y = np.zeros((T, H))
    hs = {}
    for e in range(E):
        lo, hi = int(r["offsets"][e]), int(r["offsets"][e + 1])
        if hi == lo:
            continue
        pairs = r["sorted_pair"][lo:hi].astype(np.int64)
        toks = pairs // k
        d, hb = _expert_mlp(a_all[toks], linears[e], act)
        # pairs of one expert belong to distinct tokens (top-k ids are distinct per token)
        np.add.at(y, toks, d * w64[pairs][:, None])
        if return_h:
            hs[e] = hb
    for j in range(len(linears) - E):
        d, hb = _expert_mlp(a_all, linears[E + j], act)
        gj = np.ones((T, 1)) if shared_w is None else np.asarray(shared_w, dtype=np.float64)[:, j:j + 1]
        y += d * gj
        if return_h:
            hs[E + j] = hb
    out = {"y": y, "route": r}
    if return_h:
        out["h"] = hs
    return out


# ----------------------------------------------------------------------------
# Tile scheduling (Sec. 4.3 "Tile Schedule"; Sec. 4.2.2 runtime model)
# ----------------------------------------------------------------------------


def lpt_makespan(costs: Sequence[float], P: int, presorted: bool = False) -> float:
    """Greedy list scheduling: tiles in queue order, each to the machine that frees first.

    With the queue sorted by decreasing cost this is the longest-processing-time
    rule the paper uses (computationally intensive tiles first).
    """
    c = list(costs) if presorted else sorted(costs, reverse=True)
    loads = [0.0] * P
    for x in c:
        i = min(range(P), key=lambda j: (loads[j], j))
        loads[i] += x
    return max(loads) if loads else 0.0


def optimal_makespan(costs: Sequence[float], P: int) -> float:
    """Exact minimum makespan by exhaustive assignment (tiny instances only)."""
    c = sorted(costs, reverse=True)
    best = [math.inf]
    loads = [0.0] * P

    def rec(i):
        if max(loads) >= best[0]:
            return
        if i == len(c):
            best[0] = max(loads)
            return
        seen = set()
        for j in range(P):
            if loads[j] in seen:
                continue
            seen.add(loads[j])
            loads[j] += c[i]
            rec(i + 1)
            loads[j] -= c[i]

    rec(0)
    return best[0] if c else 0.0


# ----------------------------------------------------------------------------
# Tile plan of the Group-GEMM (Sec. 4.3 tile configuration and tile schedule)
# ----------------------------------------------------------------------------
#
# The paper fixes tile configurations offline per linear (the y variables of its
# allocation problem, Eq. (7)) and orders tiles greedily, longest first.  This
# library picks the configuration at run time from the group's row count m and
# orders groups by a static per-tile cost.  The rule, restated here:
#   configuration S (m <= 16): 16 rows x (gate|up 256, down 512) channels
#   configuration T (m <= 32): 32 rows x (gate|up 256, down 512) channels
#   configuration M (m <= 64): 64 rows x (gate|up 128, down 256) channels
#   configuration L (m > 64) : 128 rows x (gate|up 128, down 256) channels,
#   except w4a4-g128 groups, which stay at configuration M
#   cost of a tile (ps) = min(max(bytes * 32, flops * 1000 / rate) + 2e6, 2e9),
#   truncated to an integer, with bytes = wbytes / mt + abytes / nt (the group's
#   mt row tiles share a weight tile, its nt channel tiles an activation tile),
#   wbytes = linears * BN * K * wbits / 8, abytes = BM * K * (1 or 2), plus
#   8 * BM * BN * linears for a sliced tile (its partial sums written and read
#   back); flops = 2 * linears * BM * BN * K, rate 39062 (FP4, and w4a4 on FP6
#   operands, whose weights count 6 bits), 19531 (int8) or 9766 (16-bit)
#   FLOP/ns - one CU's share of 8 TB/s and of 5.0 / 2.5 PFLOP/s - and 2e6 ps
#   (2 us) of fixed per-tile work;
#   queue order: decreasing cost, ties by lower expert index.
# Slicing of the reduction (split-K, the paper's slice-K tile parameter):
#   theta = (sum over the phase's tiles of the unsliced tile cost) // nwg // 2,
#   nwg the workgroups of the launch; a group takes the fewest slices S in
#   1 .. Smax = clamp(K/128 // 6, 1, 8) whose tile cost (reduction length
#   ceil(K/128 / S) k blocks) is at most theta, else the S of the cheapest tile
#   (the fewest slices among equals); groups without tiles are not sliced;
#   budgets, granted in group order: the slices' partial sums (tiles * S * BM *
#   BN * linears floats) fit the partial buffer and the tiles added by slicing
#   (tiles * (S - 1)) stay within 16384 per phase, and a group whose S is the
#   cheapest tile's (none within theta) is sliced only if the phase's unsliced
#   tiles plus every added tile granted so far plus its own stay within nwg
#   and no earlier such group failed that test; else S = 1;
#   a sliced group queues tiles * S tiles.
#
# Tile cost (Sec. 4.2.2: the cost c_t of a tile of each configuration is
# profiled ahead of time and given to the scheduler): `costs` is that table,
# an input like the weights, [phase][scheme][configuration] -> (a, bs, bu, h)
# in ps, schemes numbered w16, w8a8, w4a4, w2g128, w3g128, w4g128, w8g128,
# w4a4-g128, mxfp4, fp8, w4a4 on FP6.  A tile of kb k blocks whose group has
# mt row tiles (which share its weights) costs
#   a + kb * bs + floor(kb * bu / mt) + (h if the group is sliced),
# clamped to [1, 2 * 10^9].

_TILE_BM = (16, 32, 64, 128)
_TILE_BN = ((256, 256, 128, 128), (512, 512, 256, 256))   # [phase][config]
_SPLIT_EXTRA = 16384
_SPLIT_MAX = 8
_SPLIT_SHARE = 2
_SPLIT_MIN_KB = 6


def scheme_index(s) -> int:
    """Position of a scheme in the cost table's scheme axis."""
    fmt = getattr(s, "fmt", 0)
    if s.a_bits == 16:
        return 0 if s.w_bits == 16 else {2: 3, 3: 4, 4: 5, 8: 6}[s.w_bits]
    if fmt == 1:
        return 8
    if fmt == 2:
        return 9
    if fmt == 3:
        return 10
    if s.a_group > 0:
        return 7
    return 1 if s.w_bits == 8 else 2


def _tile_cost(entry, kb: int, split: int, mt: int) -> int:
    a, bs, bu, h = (int(v) for v in entry)
    c = a + kb * bs + (kb * bu) // max(mt, 1) + (h if split > 1 else 0)
    return min(max(c, 1), 2 * 10**9)


def _choose_split(entry, kblocks: int, mt: int, nt: int, theta: int):
    """(slices, True if no slice count is within theta)."""
    if mt * nt <= 0:
        return 1, False
    smax = max(1, min(_SPLIT_MAX, kblocks // _SPLIT_MIN_KB))
    best, cbest = 1, None
    for sp in range(1, smax + 1):
        c = _tile_cost(entry, -(-kblocks // sp), sp, mt)
        if c <= theta:
            return sp, False
        if cbest is None or c < cbest:
            best, cbest = sp, c
    return best, True


def tile_plan(ms: Sequence[int], lins: Sequence, phase: int, costs, partial_floats: int = 0, nwg: int = 512):
    """Tile configuration, tile counts, slices, cost and queue rank per group.

    ms[g]: rows of group g; lins[g]: its linear (gate for phase 0, down for 1);
    costs: the tile cost table (see above); partial_floats: size of the
    split-K partial buffer; nwg: workgroups of the launch.  Returns a list of
    dicts (cfg, mtiles, ntiles, split, tiles, cost, rank) and the queue order
    (group indices with tiles, longest tile first).
    """
    out = []
    geo = []
    work = 0
    unsliced = 0
    for m, lin in zip(ms, lins):
        m = int(m)  # Python integers: the sums below exceed 32 bits
        cfg = 0 if m <= 16 else (1 if m <= 32 else (2 if m <= 64 else 3))
        if cfg == 3 and lin.scheme.a_bits < 16 and (lin.scheme.a_group > 0
                                                     or (getattr(lin.scheme, "fmt", 0) == 2 and phase != 1)):
            cfg = 2   # w4a4-g128 and mxfp4 groups stop at 64-row tiles, fp8 outside the down phase
        bm, bn = _TILE_BM[cfg], _TILE_BN[phase][cfg]
        mt = -(-m // bm) if m > 0 else 0
        nt = -(-int(lin.n) // bn)
        entry = costs[phase][scheme_index(lin.scheme)][cfg]
        geo.append((cfg, mt, nt, entry))
        if mt * nt > 0:
            work += mt * nt * _tile_cost(entry, lin.k // 128, 1, mt)
            unsliced += mt * nt
    theta = work // nwg // _SPLIT_SHARE
    pused = eused = 0
    stopped = False
    for (cfg, mt, nt, entry), lin in zip(geo, lins):
        sp, fallback = _choose_split(entry, lin.k // 128, mt, nt, theta)
        if sp > 1:
            need = mt * nt * sp * _TILE_BM[cfg] * _TILE_BN[phase][cfg] * (2 if phase == 0 else 1)
            extra = mt * nt * (sp - 1)
            if fallback and unsliced + eused + extra > nwg:
                stopped = True
            if pused + need > partial_floats or eused + extra > _SPLIT_EXTRA or (fallback and stopped):
                sp = 1
            else:
                pused += need
                eused += extra
        out.append({"cfg": cfg, "mtiles": mt, "ntiles": nt, "split": sp})
    for r, lin, (_, _, _, entry) in zip(out, lins, geo):
        tiles = r["mtiles"] * r["ntiles"] * r["split"]
        r["tiles"] = tiles
        r["cost"] = _tile_cost(entry, -(-(lin.k // 128) // r["split"]), r["split"], r["mtiles"]) if tiles else 0
    live = [g for g, r in enumerate(out) if r["tiles"] > 0]
    order = sorted(live, key=lambda g: (-out[g]["cost"], g))
    for r in out:
        r["rank"] = -1
    start = 0
    for rank, g in enumerate(order):
        out[g]["rank"] = rank
        out[g]["start"] = start
        start += out[g]["tiles"]
    return out, order


# Super-tiles and per-XCD queues.  A group of mt x nt tiles (nt counting the
# slices of a sliced group as extra channel tiles) is cut into
# super-tiles of sm = min(mt, 8) row tiles by sn = min(nt, 64 // sm) channel
# tiles, numbered with the row index fastest; the super-tiles of all groups, in
# queue (rank) order, are dealt round-robin to 8 queues.  Each queue lists
# (group, super-tile, first tile) with first tiles as a running sum of the
# super-tiles' tile counts.


def _super_dims(mt: int, nt: int):
    sm = min(mt, 8)
    sn = min(nt, 64 // max(sm, 1))
    return sm, sn, -(-mt // sm), -(-nt // sn)


def xcd_queues(plan, order, n_queues: int = 8):
    """Expected queue entries [(group, super-tile, first tile)] and tile totals."""
    queues = [[] for _ in range(n_queues)]
    totals = [0] * n_queues
    u = 0
    for g in order:
        mt, nt = int(plan[g]["mtiles"]), int(plan[g]["ntiles"]) * int(plan[g].get("split", 1))
        sm, sn, nsm, nsn = _super_dims(mt, nt)
        for s in range(nsm * nsn):
            smi, sni = s % nsm, s // nsm
            size = min(sm, mt - smi * sm) * min(sn, nt - sni * sn)
            x = u % n_queues
            queues[x].append((g, s, totals[x]))
            totals[x] += size
            u += 1
    return queues, totals


def xcd_tiles(plan, order, n_queues: int = 8):
    """Per-queue tile lists [(group, row tile, channel tile)]: each queue entry
    expanded into its super-tile's tiles, row tile fastest.  Channel tiles of a
    sliced group count slice * ntiles + channel tile."""
    queues, _ = xcd_queues(plan, order, n_queues)
    out = []
    for q in queues:
        tiles = []
        for g, s, _first in q:
            mt, nt = int(plan[g]["mtiles"]), int(plan[g]["ntiles"]) * int(plan[g].get("split", 1))
            sm, sn, nsm, _nsn = _super_dims(mt, nt)
            smi, sni = s % nsm, s // nsm
            em, en = min(sm, mt - smi * sm), min(sn, nt - sni * sn)
            tiles += [(g, smi * sm + t % em, sni * sn + t // em) for t in range(em * en)]
        out.append(tiles)
    return out
