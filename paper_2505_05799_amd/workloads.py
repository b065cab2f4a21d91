"""Seeded synthetic inputs for the MoE-block workloads.

This module only *prepares inputs*: token activations, router top-k ids and
gate weights, and per-linear quantized weights (codes + scales + zeros).  It
contains none of the arithmetic of the forward pass itself (no GEMM, no
runtime activation quantizer, no SiLU-gate, no combine).  Both the CPU oracle
and the GPU path consume what it returns; neither imports the other.

Shapes follow the paper's evaluated models (Sec. 5.1, table ``tab:exp-model``)
and the two token counts of its throughput study (Sec. 5.3: 512-token
memory-bound and 8192-token compute-bound regimes).  The real WikiText-2 inputs,
trained routers and trained weights are not available, so seeded Gaussian data
with a Zipf-skewed router stands in for them:

* X ~ N(0, 1), rounded to the activation dtype (RNE).
* router logits ~ N(0, 1) plus a per-expert bias -s*ln(rank) (an unnormalised
  Zipf pmf in log space); softmax in fp64, top-k by probability (ties go to the
  lower expert id); gate weights are the fp32 softmax probabilities, not
  renormalised.
* weights ~ N(0, 0.02^2) drawn in fp32, rounded to bf16, then quantized offline
  with round-to-nearest min-max quantizers (Sec. 2.1).  GPTQ and the Hadamard
  rotation the paper applies offline need calibration data and trained weights;
  the packed kernel contract (codes + scale + zero) is identical either way.

Offline quantizers (input preparation, not part of the forward pass):

* ``wNg128`` asymmetric (Sec. 5.2: groups of 128 along K, 16-bit scale and zero):
  s = fp16((max - min) / (2^N - 1)), z = clamp(rne(-min / s), 0, 2^N - 1)
  stored as fp16, q = clamp(rne(w / s) + z, 0, 2^N - 1); the dequantized value
  is s * (q - z), the min-max quantizer with x_min snapped onto the grid.
* per-channel symmetric (``w8a8``/``w4a4``, Fig. 4 caption): qmax = 2^(b-1) - 1,
  s = fp32(amax_row / qmax), q = clamp(rne(w / s), -qmax, qmax).
* ``mxfp4`` (the OCP Microscaling MXFP4 format, one of the 4-bit schemes the
  MI355X matrix cores run natively): per 32 consecutive weights along K a
  shared power-of-two scale 2^e (E8M0 byte e + 127), e = floor(log2(amax)) - 2,
  and FP4 e2m1 elements rne(w / 2^e) on the grid {0, 0.5, 1, 1.5, 2, 3, 4, 6}
  (ties to the even code, magnitudes above 6 clamp to 6).
* ``fp8`` (OCP FP8 e4m3, the 8-bit floating-point operand of the MI355X matrix
  cores): per output channel s = fp32(amax_row / 448) and elements = the e4m3
  value nearest to w / s (ties to the even code), taken here from the binary
  exponent and a rounded 3-bit mantissa (below 2^-6: multiples of 2^-9).
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# Schemes (notation wXaY_gZ_{sym,asym} of the paper's Fig. 1 caption)
# ----------------------------------------------------------------------------


@dataclass(frozen=True)
class Scheme:
    w_bits: int      # 16, 8, 4, 3, 2
    a_bits: int      # 16 = weight-only, 8 or 4 = weight-activation
    w_group: int     # 128 for groups along K, -1 = per output channel
    a_group: int     # 128 for groups along K, -1 = per token
    symmetric: int   # 1 for w8a8 / w4a4 (per channel or g128), 0 for wNg128 asym and 16-bit
    fmt: int = 0     # 0 integer codes; 1 OCP MX floating point (e2m1 elements, E8M0 scale per 32);
                     # 2 FP8 e4m3 elements with per-channel / per-token fp32 scales;
                     # 3 w4a4 codes held as FP6 e2m3 operands (same quantization as fmt 0)

    @property
    def name(self) -> str:
        if self.fmt == 1:
            return "mxfp4"
        if self.fmt == 2:
            return "fp8"
        if self.fmt == 3:
            return "w4a4f6"
        if self.w_bits == 16:
            return "w16"
        if self.a_bits < 16:
            g = f"g{self.w_group}" if self.w_group > 0 else ""
            return f"w{self.w_bits}a{self.a_bits}{g}"
        return f"w{self.w_bits}g{self.w_group}"

    @property
    def weight_only(self) -> bool:
        return self.w_bits < 16 and self.a_bits == 16

    def bits_per_weight(self, k: int) -> float:
        """Stored bits per weight including scale/zero overhead."""
        if self.w_bits == 16:
            return 16.0
        if self.fmt == 1:
            return self.w_bits + 8.0 / self.w_group    # one E8M0 byte per 32
        if self.fmt == 3:
            return 6.0 + 32.0 / k                      # 4-bit codes stored as 6-bit e2m3, fp32 row scale
        if self.weight_only:
            return self.w_bits + 32.0 / self.w_group   # fp16 scale + fp16 zero
        if self.w_group > 0:
            return self.w_bits + 16.0 / self.w_group   # fp16 scale per group
        return self.w_bits + 32.0 / k                 # one fp32 scale per row


W16 = Scheme(16, 16, -1, -1, 0)
W8A8 = Scheme(8, 8, -1, -1, 1)
W4A4 = Scheme(4, 4, -1, -1, 1)
W2G128 = Scheme(2, 16, 128, -1, 0)
W3G128 = Scheme(3, 16, 128, -1, 0)
W4G128 = Scheme(4, 16, 128, -1, 0)
W8G128 = Scheme(8, 16, 128, -1, 0)
W4A4G128 = Scheme(4, 4, 128, 128, 1)   # 4-bit weights and activations, per-128 group scales
MXFP4 = Scheme(4, 4, 32, 32, 1, 1)     # FP4 e2m1 weights and activations, E8M0 scale per 32
FP8 = Scheme(8, 8, -1, -1, 1, 2)       # FP8 e4m3 weights (per channel) and activations (per token)
W4A4F6 = Scheme(4, 4, -1, -1, 1, 3)    # w4a4 whose int4 codes run as FP6 e2m3 operands (6 stored bits)
ALL_SCHEMES = (W16, W8A8, W4A4, W2G128, W3G128, W4G128, W8G128, W4A4G128, MXFP4, FP8, W4A4F6)
SCHEME_BY_NAME = {s.name: s for s in ALL_SCHEMES}

LINEAR_NAMES = ("gate", "up", "down")

# ----------------------------------------------------------------------------
# Block configurations
# ----------------------------------------------------------------------------

Alloc = Callable[[int, int], Tuple[Scheme, Scheme, Scheme]]  # (expert, rank) -> schemes


@dataclass
class BlockConfig:
    name: str
    T: int                      # tokens
    H: int                      # hidden
    F: int                      # routed-expert FFN
    E: int                      # routed experts
    k: int                      # top-k
    n_shared: int               # shared experts (dense over all tokens)
    F_shared: int               # shared-expert FFN
    act: str                    # "fp16" | "bf16"
    zipf_s: Optional[float]     # router skew; None = no bias
    alloc: Alloc                # routed-expert schemes
    shared_alloc: Tuple[Scheme, Scheme, Scheme] = (W16, W16, W16)
    description: str = ""

    def scaled(self, T: int) -> "BlockConfig":
        """Same block with another token count (used for bounded CPU samples)."""
        c = BlockConfig(**{**self.__dict__})
        c.T = T
        return c

    def flops(self, counts: Sequence[int]) -> float:
        """Algorithmic FLOPs of the forward: 2*m*N*K per linear, real rows only."""
        f = sum(6.0 * int(m) * self.H * self.F for m in counts)
        f += self.n_shared * 6.0 * self.T * self.H * self.F_shared
        return f


def _tiny_alloc(e: int, rank: int):
    return [
        (W4G128, W4G128, W4G128),
        (W8A8, W8A8, W2G128),
        (W4A4, W4A4, W4A4),
        (W16, W16, W16),
    ][e]


def _mixtral_alloc(e: int, rank: int):
    if rank == 1:
        return (W8A8, W8A8, W8A8)
    down = W4G128 if rank == 2 else (W3G128 if rank <= 7 else W2G128)
    return (W2G128, W2G128, down)


def _dsv2_alloc(e: int, rank: int):
    if rank <= 16:
        return (W8A8, W8A8, W8A8)
    if rank <= 48:
        return (W4G128, W4G128, W4G128)
    return (W2G128, W2G128, W2G128)


def _qwen15_uniform(e: int, rank: int):
    return (W4A4, W4A4, W4A4)


def _qwen15_mixed(e: int, rank: int):
    if rank <= 2:
        return (W8A8, W8A8, W8A8)
    if rank <= 28:
        return (W4A4, W4A4, W4A4)
    return (W3G128, W3G128, W3G128)


def _qwen15_float(e: int, rank: int):
    return (FP8, FP8, FP8) if rank <= 6 else (MXFP4, MXFP4, MXFP4)


# The W5A5 allocation the paper prints for layer 5 of Qwen1.5-MoE (appendix
# table of per-linear schemes): one character per expert, experts 0..59 then
# the shared expert.  g = w4a4 with 128-groups on both operands, c = w4a4 per
# channel / per token, 8 = w8a8 per channel / per token.  Gate and up carry the
# same scheme in every row of that table, so one string serves both.
_W5A5_GATE_UP = "ggggcggcggggggcggggggg8gggggggggggggggggggggcgggggggggcccgcgc"
_W5A5_DOWN = "g888gg8g88888gg88888g88g8g8g8gg8gg88888gg888g88g88gg8gggggg88"
_W5A5_CODE = {"g": W4A4G128, "c": W4A4, "8": W8A8}


def _qwen15_w5a5(e: int, rank: int):
    gu = _W5A5_CODE[_W5A5_GATE_UP[e]]
    return (gu, gu, _W5A5_CODE[_W5A5_DOWN[e]])


def _qwen2_alloc(e: int, rank: int):
    return (W8A8, W8A8, W8A8) if rank <= 10 else (W4A4, W4A4, W4A4)


def _qwen2_f6_alloc(e: int, rank: int):
    return (W8A8, W8A8, W8A8) if rank <= 10 else (W4A4F6, W4A4F6, W4A4F6)


CONFIGS: Dict[str, BlockConfig] = {
    "tiny": BlockConfig(
        "tiny", T=64, H=256, F=512, E=4, k=2, n_shared=0, F_shared=0, act="fp16",
        zipf_s=None, alloc=_tiny_alloc,
        description="tiny MoE block: 64 tokens, hidden 256, FFN 512, 4 experts, top-2, fp16"),
    "mixtral": BlockConfig(
        "mixtral", T=4096, H=4096, F=14336, E=8, k=2, n_shared=0, F_shared=0, act="bf16",
        zipf_s=1.0, alloc=_mixtral_alloc,
        description="Mixtral-8x7B-shaped prefill: 4096 tokens, hidden 4096, FFN 14336, "
                    "8 experts, top-2, 3.26 avg weight bits"),
    "dsv2lite": BlockConfig(
        "dsv2lite", T=2048, H=2048, F=1408, E=64, k=6, n_shared=2, F_shared=1408, act="bf16",
        zipf_s=1.2, alloc=_dsv2_alloc, shared_alloc=(W8A8, W8A8, W8A8),
        description="DeepSeek-V2-Lite-shaped: 2048 tokens, hidden 2048, 64 experts FFN 1408, "
                    "top-6, 2 shared experts"),
    "qwen15_uniform": BlockConfig(
        "qwen15_uniform", T=256, H=2048, F=1408, E=60, k=4, n_shared=1, F_shared=5632,
        act="bf16", zipf_s=1.5, alloc=_qwen15_uniform, shared_alloc=(W4A4, W4A4, W4A4),
        description="Qwen1.5-MoE-shaped decode batch: 256 tokens, 60 experts FFN 1408, top-4, "
                    "shared FFN 5632, uniform w4a4"),
    "qwen15_mixed": BlockConfig(
        "qwen15_mixed", T=256, H=2048, F=1408, E=60, k=4, n_shared=1, F_shared=5632,
        act="bf16", zipf_s=1.5, alloc=_qwen15_mixed, shared_alloc=(W8A8, W8A8, W8A8),
        description="Qwen1.5-MoE-shaped decode batch, mixed w8a8/w4a4/w3g128 at equal avg bits"),
    "qwen15_float": BlockConfig(
        "qwen15_float", T=8192, H=2048, F=1408, E=60, k=4, n_shared=1, F_shared=5632,
        act="bf16", zipf_s=1.5, alloc=_qwen15_float, shared_alloc=(FP8, FP8, FP8),
        description="Qwen1.5-MoE-shaped compute-bound batch (8192 tokens) on the MI355X floating-point "
                    "schemes: fp8 for the 6 hottest experts and the shared expert, mxfp4 for the rest"),
    "qwen15_w5a5": BlockConfig(
        "qwen15_w5a5", T=8192, H=2048, F=1408, E=60, k=4, n_shared=1, F_shared=5632,
        act="bf16", zipf_s=1.5, alloc=_qwen15_w5a5, shared_alloc=_qwen15_w5a5(60, 0),
        description="Qwen1.5-MoE-shaped compute-bound batch (8192 tokens) with the paper's "
                    "printed W5A5 allocation for layer 5 (w4a4-g128 / w4a4 / w8a8 per linear)"),
    "qwen2": BlockConfig(
        "qwen2", T=16384, H=3584, F=2560, E=64, k=8, n_shared=1, F_shared=20480, act="bf16",
        zipf_s=1.0, alloc=_qwen2_alloc, shared_alloc=(W8A8, W8A8, W8A8),
        description="Qwen2-57B-A14B-shaped prefill: 16384 tokens, hidden 3584, 64 experts FFN "
                    "2560, top-8, shared FFN 20480, w8a8/w4a4"),
    "qwen2_f6": BlockConfig(
        "qwen2_f6", T=16384, H=3584, F=2560, E=64, k=8, n_shared=1, F_shared=20480, act="bf16",
        zipf_s=1.0, alloc=_qwen2_f6_alloc, shared_alloc=(W8A8, W8A8, W8A8),
        description="Qwen2-57B-A14B-shaped prefill (16384 tokens, w8a8/w4a4) with the w4a4 experts' int4 codes "
                    "run as FP6 e2m3 operands"),
}

# ----------------------------------------------------------------------------
# dtype helpers (input preparation only)
# ----------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f64_to_act(x: np.ndarray, act: str) -> np.ndarray:
    """Round fp64 data to the activation dtype: float16 array or bf16 bits."""
    if act == "fp16":
        return x.astype(np.float16)
    # direct fp64 -> bf16 RNE: 8 significant bits, spacing 2^(e-8)
    m, e = np.frexp(x)
    spacing = np.ldexp(1.0, np.maximum(e - 8, -133))
    r = np.rint(x / spacing) * spacing
    return f32_to_bf16_bits(r.astype(np.float32))   # r is bf16-exact, conversion is exact


def act_to_f32(a: np.ndarray, act: str) -> np.ndarray:
    return a.astype(np.float32) if act == "fp16" else bf16_bits_to_f32(a)

# ----------------------------------------------------------------------------
# offline weight quantizers
# ----------------------------------------------------------------------------


def quantize_g128_asym(w: np.ndarray, bits: int, group: int = 128):
    """Min-max RTN per group along K; returns (codes uint8, scales fp16, zeros fp16)."""
    n, k = w.shape
    assert k % group == 0
    qmax = (1 << bits) - 1
    codes = np.empty((n, k), np.uint8)
    scales = np.empty((n, k // group), np.float16)
    zeros = np.empty((n, k // group), np.float16)
    rows = max(1, (1 << 22) // k)
    for r0 in range(0, n, rows):
        wg = w[r0:r0 + rows].astype(np.float64).reshape(-1, k // group, group)
        mx = wg.max(axis=2)
        mn = wg.min(axis=2)
        s = ((mx - mn) / qmax).astype(np.float16)
        degenerate = (mx == mn) | (s == 0)
        s = np.where(degenerate, np.float16(1.0), s)
        s64 = s.astype(np.float64)
        z = np.clip(np.rint(-mn / s64), 0, qmax)
        z = np.where(degenerate, 0.0, z)
        q = np.clip(np.rint(wg / s64[..., None]) + z[..., None], 0, qmax)
        codes[r0:r0 + rows] = q.reshape(-1, k).astype(np.uint8)
        scales[r0:r0 + rows] = s
        zeros[r0:r0 + rows] = z.astype(np.float16)
    return codes, scales, zeros


def quantize_sym_per_channel(w: np.ndarray, bits: int):
    """Symmetric per-output-channel RTN; returns (codes int8, scales fp32)."""
    qmax = (1 << (bits - 1)) - 1
    w64 = w.astype(np.float64)
    amax = np.abs(w64).max(axis=1)
    s = (amax / qmax).astype(np.float32)
    s64 = s.astype(np.float64)
    safe = np.where(s64 == 0, 1.0, s64)
    q = np.clip(np.rint(w64 / safe[:, None]), -qmax, qmax)
    q = np.where(s64[:, None] == 0, 0, q)
    return q.astype(np.int8), s


def quantize_sym_g128(w: np.ndarray, bits: int, group: int = 128):
    """Symmetric RTN per (output channel, group of `group` along K) with an fp16
    scale: s = fp16(amax / qmax), q = clamp(rne(w / s), -qmax, qmax); an all-zero
    group (or one whose scale rounds to 0) gets s = 0 and zero codes.
    Returns (codes int8 [n, k], scales fp16 [n, k/group])."""
    n, k = w.shape
    assert k % group == 0
    qmax = (1 << (bits - 1)) - 1
    wg = w.astype(np.float64).reshape(n, k // group, group)
    s = (np.abs(wg).max(axis=2) / qmax).astype(np.float16)
    s64 = s.astype(np.float64)
    safe = np.where(s64 == 0, 1.0, s64)
    q = np.clip(np.rint(wg / safe[..., None]), -qmax, qmax)
    q = np.where(s64[..., None] == 0, 0, q)
    return q.reshape(n, k).astype(np.int8), s


E2M1_VALUES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def quantize_mxfp4(w: np.ndarray, block: int = 32):
    """MXFP4 (OCP MX) quantizer of the weights: codes uint8 [n, k] (e2m1, sign
    in bit 3), E8M0 scales uint8 [n, k/32].  An all-zero block gets e = -127."""
    n, k = w.shape
    assert k % block == 0
    v = w.astype(np.float64).reshape(n, k // block, block)
    amax = np.abs(v).max(axis=2)
    _, ex = np.frexp(amax)                      # amax = f 2^ex, f in [0.5, 1): floor(log2) = ex - 1
    e = np.where(amax > 0, ex - 1 - 2, -127).clip(-127, 127)
    r = np.abs(v) / np.exp2(e)[..., None]
    # round to the e2m1 grid, ties to the even code: at the midpoint above an
    # even code stay, above an odd code go up
    mids = (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0)
    code = np.zeros(r.shape, np.int64)
    for c, mp in enumerate(mids):
        code += (r > mp) if c % 2 == 0 else (r >= mp)
    code = np.where((v < 0) & (code > 0), code | 8, code)
    return code.reshape(n, k).astype(np.uint8), (e + 127).astype(np.uint8)


def quantize_fp8(w: np.ndarray):
    """FP8 e4m3 per-channel quantizer: codes uint8 [n, k] (sign bit 7, four
    exponent bits of bias 7, three mantissa bits), scales fp32 [n] =
    fp32(amax / 448).  A row of zeros gets scale 0 and zero codes."""
    w64 = w.astype(np.float64)
    s = (np.abs(w64).max(axis=1) / 448.0).astype(np.float32)
    s64 = s.astype(np.float64)
    r = np.abs(w64) / np.where(s64 == 0, 1.0, s64)[:, None]
    r = np.where(s64[:, None] == 0, 0.0, np.minimum(r, 448.0))
    _, ex = np.frexp(r)                         # r = f 2^ex, f in [0.5, 1): exponent ex - 1
    e = np.maximum(ex - 1, -6)
    normal = r >= 2.0 ** -6
    # normal: mantissa steps of 2^(e-3); below 2^-6: steps of 2^-9 (code = count)
    m = np.rint(np.where(normal, (r / np.exp2(e) - 1.0) * 8.0, r * 512.0)).astype(np.int64)
    code = np.where(normal, ((e + 7) << 3) + m, m)   # a mantissa carry moves into the exponent
    code = np.minimum(code, 126)
    code = np.where((w64 < 0) & (code > 0), code | 0x80, code)
    return code.astype(np.uint8), s


@dataclass
class QLinear:
    """One quantized linear, W is [n, k] = [out, in] (nn.Linear layout)."""
    scheme: Scheme
    n: int
    k: int
    codes: np.ndarray                    # uint8 / int8 [n,k]; bf16 bits uint16 for w16
    scales: Optional[np.ndarray] = None  # fp16 [n, k/128] (groups) | fp32 [n] (per channel)
    zeros: Optional[np.ndarray] = None   # fp16 [n, k/128]

    @property
    def nbytes_packed(self) -> int:
        s = self.scheme
        if s.w_bits == 16:
            return 2 * self.n * self.k
        if s.weight_only:
            return self.n * self.k * s.w_bits // 8 + (self.n * self.k // 128) * 4
        if s.fmt == 1:      # e2m1 nibbles + one E8M0 byte per 32
            return self.n * self.k // 2 + self.n * self.k // 32
        if s.fmt == 3:      # 6-bit e2m3 codes + one fp32 scale per row
            return self.n * self.k * 6 // 8 + 4 * self.n
        if s.w_group > 0:   # packed with the same 4-byte metadata slot per group
            return self.n * self.k * s.w_bits // 8 + (self.n * self.k // 128) * 4
        return self.n * self.k * s.w_bits // 8 + 4 * self.n


def quantize_linear(w_bf16_f32: np.ndarray, scheme: Scheme) -> QLinear:
    n, k = w_bf16_f32.shape
    if scheme.w_bits == 16:
        return QLinear(scheme, n, k, f32_to_bf16_bits(w_bf16_f32))
    if scheme.weight_only:
        c, s, z = quantize_g128_asym(w_bf16_f32, scheme.w_bits, scheme.w_group)
        return QLinear(scheme, n, k, c, s, z)
    if scheme.fmt == 1:
        c, s = quantize_mxfp4(w_bf16_f32, scheme.w_group)
        return QLinear(scheme, n, k, c, s)
    if scheme.fmt == 2:
        c, s = quantize_fp8(w_bf16_f32)
        return QLinear(scheme, n, k, c, s)
    if scheme.w_group > 0:
        c, s = quantize_sym_g128(w_bf16_f32, scheme.w_bits, scheme.w_group)
        return QLinear(scheme, n, k, c, s)
    c, s = quantize_sym_per_channel(w_bf16_f32, scheme.w_bits)
    return QLinear(scheme, n, k, c, s)


def draw_weight(seed: int, expert: int, lin: int, n: int, k: int, std: float = 0.02):
    """bf16-valued fp32 weight [n,k]; one independent stream per (expert, linear)."""
    g = np.random.default_rng([seed, 2, expert, lin])
    w = g.standard_normal((n, k), dtype=np.float32) * np.float32(std)
    return bf16_bits_to_f32(f32_to_bf16_bits(w))

# ----------------------------------------------------------------------------
# routing and activations
# ----------------------------------------------------------------------------


def expert_ranks(cfg: BlockConfig, seed: int = 0) -> np.ndarray:
    """Zipf popularity rank of each routed expert (1 = hottest)."""
    if cfg.zipf_s is None:
        return np.arange(1, cfg.E + 1)
    return np.random.default_rng([seed, 3]).permutation(cfg.E) + 1


def make_routing(cfg: BlockConfig, seed: int = 0, T: Optional[int] = None):
    """Top-k ids int32 [T,k] and gate weights fp32 [T,k]."""
    T = cfg.T if T is None else T
    logits = np.random.default_rng([seed, 1]).standard_normal((cfg.T, cfg.E))[:T]
    if cfg.zipf_s is not None:
        logits = logits - cfg.zipf_s * np.log(expert_ranks(cfg, seed).astype(np.float64))
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    ids = np.argsort(-p, axis=1, kind="stable")[:, : cfg.k]
    w = np.take_along_axis(p, ids, axis=1).astype(np.float32)
    return np.ascontiguousarray(ids.astype(np.int32)), np.ascontiguousarray(w)


def router_logits(T: int, E: int, seed: int = 0, zipf_s: Optional[float] = None,
                  n_shared: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """fp32 router logits [T, E] (N(0,1) plus the Zipf bias of make_routing,
    expert ranks a seeded permutation) and fp32 shared-gate logits [T, n_shared]
    (N(0,1)), for the router front-end."""
    rng = np.random.default_rng([seed, 4])
    l = rng.standard_normal((T, E))
    if zipf_s is not None:
        ranks = np.random.default_rng([seed, 5]).permutation(E) + 1
        l = l - zipf_s * np.log(ranks.astype(np.float64))
    sh = np.random.default_rng([seed, 6]).standard_normal((T, n_shared))
    return np.ascontiguousarray(l.astype(np.float32)), np.ascontiguousarray(sh.astype(np.float32))


def make_x(cfg: BlockConfig, seed: int = 0, T: Optional[int] = None) -> np.ndarray:
    T = cfg.T if T is None else T
    x = np.random.default_rng([seed, 0]).standard_normal((cfg.T, cfg.H))[:T]
    return np.ascontiguousarray(f64_to_act(x, cfg.act))


def schemes_of(cfg: BlockConfig, seed: int = 0) -> List[Tuple[Scheme, Scheme, Scheme]]:
    ranks = expert_ranks(cfg, seed)
    out = [tuple(cfg.alloc(e, int(ranks[e]))) for e in range(cfg.E)]
    out += [tuple(cfg.shared_alloc)] * cfg.n_shared
    return out


def linear_shapes(cfg: BlockConfig, expert: int) -> List[Tuple[int, int]]:
    F = cfg.F if expert < cfg.E else cfg.F_shared
    return [(F, cfg.H), (F, cfg.H), (cfg.H, F)]


def avg_weight_bits(cfg: BlockConfig, seed: int = 0) -> float:
    tot_bits = tot = 0.0
    for e, sch in enumerate(schemes_of(cfg, seed)):
        for s, (n, k) in zip(sch, linear_shapes(cfg, e)):
            tot_bits += s.bits_per_weight(k) * n * k
            tot += n * k
    return tot_bits / tot


@dataclass
class Block:
    cfg: BlockConfig
    seed: int
    x: np.ndarray                        # [T,H] float16 or bf16 bits (uint16)
    topk_ids: np.ndarray                 # int32 [T,k]
    topk_w: np.ndarray                   # fp32 [T,k]
    linears: List[List[QLinear]] = field(default_factory=list)  # [E+n_sh][3]

    @property
    def schemes(self):
        return [tuple(l.scheme for l in ls) for ls in self.linears]


def make_linears(cfg: BlockConfig, seed: int = 0, threads: Optional[int] = None):
    sch = schemes_of(cfg, seed)
    jobs = []
    for e in range(cfg.E + cfg.n_shared):
        for j, (n, k) in enumerate(linear_shapes(cfg, e)):
            jobs.append((e, j, n, k, sch[e][j]))

    def run(job):
        e, j, n, k, s = job
        return quantize_linear(draw_weight(seed, e, j, n, k), s)

    threads = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(run, jobs))
    out = [[None] * 3 for _ in range(cfg.E + cfg.n_shared)]
    for (e, j, *_), q in zip(jobs, res):
        out[e][j] = q
    return out


def random_tile_costs(seed: int) -> np.ndarray:
    """A seeded tile cost table of the run-time plan's shape, int32
    [phase][scheme][configuration][a, bs, bu, h] in ps: a in [0.1, 10] us,
    bs and bu in [0, 10] us per k block (a quarter of the entries with bu = 0),
    h in [0, 10] us."""
    rng = np.random.default_rng(seed)
    t = np.zeros((2, len(ALL_SCHEMES), 4, 4), dtype=np.int64)
    t[..., 0] = rng.integers(100_000, 10_000_000, t.shape[:-1])
    t[..., 1] = rng.integers(0, 10_000_000, t.shape[:-1])
    t[..., 2] = rng.integers(0, 10_000_000, t.shape[:-1]) * (rng.random(t.shape[:-1]) > 0.25)
    t[..., 3] = rng.integers(0, 10_000_000, t.shape[:-1])
    return t.astype(np.int32)


def make_block(cfg: BlockConfig | str, seed: int = 0, T: Optional[int] = None,
               with_weights: bool = True) -> Block:
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    if T is not None and T != cfg.T:
        base = cfg
        cfg = cfg.scaled(T)
        ids, w = make_routing(base, seed, T)
        x = make_x(base, seed, T)
    else:
        ids, w = make_routing(cfg, seed)
        x = make_x(cfg, seed)
    lin = make_linears(cfg, seed) if with_weights else []
    return Block(cfg, seed, x, ids, w, lin)


def random_small_block(seed: int, T: int, H: int, F: int, E: int, k: int,
                       n_shared: int = 0, F_shared: int = 0, act: str = "bf16",
                       schemes: Optional[Sequence[Tuple[Scheme, Scheme, Scheme]]] = None,
                       skew: float = 0.0) -> Block:
    """Small random block for parity sweeps (shapes must keep K % 128 == 0 and N % 16 == 0
    for the GPU path; the oracle accepts any shape)."""
    rng = np.random.default_rng([seed, 7])
    if schemes is None:
        pool = list(ALL_SCHEMES)
        schemes = []
        for _ in range(E + n_shared):
            gu = pool[rng.integers(len(pool))]
            dn = pool[rng.integers(len(pool))]
            schemes.append((gu, gu, dn))
    alloc = lambda e, r: schemes[e]
    cfg = BlockConfig(f"rand{seed}", T, H, F, E, k, n_shared, F_shared, act,
                      skew if skew > 0 else None, alloc,
                      shared_alloc=schemes[E] if n_shared else (W16, W16, W16))
    ids, w = make_routing(cfg, seed)
    x = make_x(cfg, seed)
    lins = [[None] * 3 for _ in range(E + n_shared)]
    for e in range(E + n_shared):
        for j, (n, kk) in enumerate(linear_shapes(cfg, e)):
            lins[e][j] = quantize_linear(draw_weight(seed, e, j, n, kk), schemes[e][j])
    return Block(cfg, seed, x, ids, w, lins)
