// Per-row activation encoders shared by the row kernels and the plan launch
// (which runs them on its spare workgroups, next to the one that plans): a
// wavefront (W = 1) or a workgroup of 4 wavefronts (W = 4) takes one row of
// 16-bit values and writes, with fixed fp32 recipes,
//   * per-token int8 / int4 codes and scales (Sec. 4.2.2, a_gsize = -1),
//   * per-token FP8 e4m3 codes and scales (the same recipe with 448 for qmax),
//   * per-128-group int4 codes and scales (w4a4-g128),
//   * MXFP4 codes and E8M0 scales (OCP MX, blocks of 32),
//   * bf16 row sums per 128-wide block (bias-dequantized weight-only tiles).
// Every output element depends on its own inputs and on order-free maxima
// only, or (row sums) on a fixed summation order, so the results do not
// depend on which kernel ran them.
#pragma once
#include "mxmoe_internal.h"

namespace mxmoe {
namespace {

__device__ inline void unpack8(uint4 u, int act, float* f) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (act == MXMOE_BF16) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    } else {
      const uint16_t lo = (uint16_t)w[i], hi = (uint16_t)(w[i] >> 16);
      f[2 * i] = (float)__builtin_bit_cast(_Float16, lo);
      f[2 * i + 1] = (float)__builtin_bit_cast(_Float16, hi);
    }
  }
}

// Largest magnitude of 8 elements as 16-bit magnitude bits (sign cleared,
// NaNs as 0): for non-negative values the bit order is the value order, so the
// row maximum equals the fmaxf reduction of quant_row, which skips NaNs.
__device__ inline uint32_t amax8_bits(uint4 u, uint32_t nan_lo) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
  uint32_t m = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = w[i] & 0x7fffu, hi = (w[i] >> 16) & 0x7fffu;
    m = max(m, lo < nan_lo ? lo : 0u);
    m = max(m, hi < nan_lo ? hi : 0u);
  }
  return m;
}
__device__ inline float bits_to_f32(uint32_t b, int act) {
  if (act == MXMOE_BF16) return __uint_as_float(b << 16);
  return (float)__builtin_bit_cast(_Float16, (uint16_t)b);
}

// FP8 e4m3 byte (OCP: sign bit 7, exponent bias 7, 3 mantissa bits) of the
// e4m3 value nearest to v, ties to the even code, magnitudes past 448 to 448
// (the largest finite value; there are no infinities), sign kept unless the
// magnitude code is 0.  Below 2^-6 the grid is the multiples of 2^-9 (code =
// count, 8 being the smallest normal); above, the fp32 mantissa is rounded to
// 3 bits in integer arithmetic and the exponent rebiased (127 -> 7).
__device__ inline uint32_t e4m3_byte(float v) {
  const uint32_t sgn = (__float_as_uint(v) >> 24) & 0x80u;
  const float a = fminf(fabsf(v), 448.0f);
  uint32_t mag;
  if (a < 0.015625f) {
    mag = (uint32_t)__builtin_rintf(a * 512.0f);
  } else {
    const uint32_t b = __float_as_uint(a);
    mag = ((b + 0x7FFFFu + ((b >> 20) & 1u)) >> 20) - (120u << 3);
  }
  return mag ? (sgn | mag) : 0u;
}

// codes of 8 elements with the same fp32 recipe as quant_row; q = 448 gives
// FP8 e4m3 codes (the row maximum scaled onto 448), else int8 codes
__device__ inline uint2 codes8(uint4 u, int act, float inv, float q) {
  float f[8];
  unpack8(u, act, f);
  uint32_t w[2] = {0u, 0u};
  if (q == (float)kQmaxF8) {
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i >> 2] |= e4m3_byte(__fmul_rn(f[i], inv)) << (8 * (i & 3));
    return make_uint2(w[0], w[1]);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float r = __builtin_rintf(__fmul_rn(f[i], inv));
    r = fminf(fmaxf(r, -q), q);
    w[i >> 2] |= ((uint32_t)(uint8_t)(int8_t)(int)r) << (8 * (i & 3));
  }
  return make_uint2(w[0], w[1]);
}

// FP6 e2m3 code of an integer v in [-7, 7] (sign bit 5, two exponent bits of
// bias 1, three mantissa bits): magnitudes 0..7 have codes 0, 8, 16, 20, 24,
// 26, 28, 30.
__device__ inline uint32_t e2m3_of_int(int v) {
  const uint32_t m = (uint32_t)(v < 0 ? -v : v);
  const uint32_t mag = m == 0 ? 0u : (m == 1 ? 8u : (m < 4 ? 16u + 4u * (m - 2u) : 24u + 2u * (m - 4u)));
  return (v < 0 ? 0x20u : 0u) | mag;
}
// int4 codes of 8 elements (the per-token recipe with q = 7) as one 48-bit
// run of 6-bit e2m3 codes, element i at bits 6i..6i+5.
__device__ inline uint64_t codes8_f6(uint4 u, int act, float inv) {
  float f[8];
  unpack8(u, act, f);
  uint64_t w = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float r = __builtin_rintf(__fmul_rn(f[i], inv));
    r = fminf(fmaxf(r, -7.f), 7.f);
    w |= (uint64_t)e2m3_of_int((int)r) << (6 * i);
  }
  return w;
}
// Store of 8 elements' e2m3 codes (chunk c of the row, 8 elements per chunk):
// a group of 32 elements is 24 bytes of codes then 8 zero bytes, so chunk c
// lands at byte 32 (c / 4) + 6 (c % 4); the last chunk of a group also writes
// the group's 8 zero bytes.
__device__ inline void store_f6_chunk(uint8_t* row, int c, uint64_t w) {
  uint16_t* p = reinterpret_cast<uint16_t*>(row + 32 * (c >> 2) + 6 * (c & 3));
  p[0] = (uint16_t)w;
  p[1] = (uint16_t)(w >> 16);
  p[2] = (uint16_t)(w >> 32);
  if ((c & 3) == 3) *reinterpret_cast<uint2*>(row + 32 * (c >> 2) + 24) = make_uint2(0u, 0u);
}

// Quantizes one row of cols (a multiple of 8) elements with W wavefronts (1:
// each wavefront of the workgroup takes its own row, 4: the workgroup takes
// one row).  NC > 0: the row's 16-byte chunks stay in registers
// (cols <= 512 * W * NC); NC == 0: any length, the row is read twice.
template <int NC, int W, bool F6 = false>
__device__ inline float quant_row_vec(const uint4* __restrict__ row, int cols, int act, int qmax,
                                      uint2* __restrict__ codes, float* __restrict__ scale, uint32_t* red) {
  const int idx = W == 1 ? (threadIdx.x & 63) : threadIdx.x, nch = cols >> 3;
  constexpr int kStride = 64 * W;
  const uint32_t nan_lo = act == MXMOE_BF16 ? 0x7f81u : 0x7c01u;  // smallest NaN magnitude
  const float q = (float)qmax;
  uint32_t mb = 0u;
  uint4 v[NC > 0 ? NC : 1];
  if constexpr (NC > 0) {
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = idx + kStride * i;
      v[i] = c < nch ? row[c] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int i = 0; i < NC; ++i) mb = max(mb, amax8_bits(v[i], nan_lo));
  } else {
    for (int c = idx; c < nch; c += kStride) mb = max(mb, amax8_bits(row[c], nan_lo));
  }
  for (int d = 32; d > 0; d >>= 1) mb = max(mb, (uint32_t)__shfl_xor((int)mb, d, 64));
  if constexpr (W > 1) {
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mb;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < W; ++i) mb = max(mb, red[i]);
  }
  const float amax = bits_to_f32(mb, act);
  float inv = 0.f, s = 0.f;
  if (amax > 0.f) {
    inv = __fdiv_rn(q, amax);
    s = __fdiv_rn(amax, q);
  }
  uint8_t* cb = reinterpret_cast<uint8_t*>(codes);
  if constexpr (NC > 0) {
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = idx + kStride * i;
      if (c < nch) {
        if constexpr (F6) store_f6_chunk(cb, c, codes8_f6(v[i], act, inv));
        else codes[c] = codes8(v[i], act, inv, q);
      }
    }
  } else {
    for (int c = idx; c < nch; c += kStride) {
      if constexpr (F6) store_f6_chunk(cb, c, codes8_f6(row[c], act, inv));
      else codes[c] = codes8(row[c], act, inv, q);
    }
  }
  if (idx == 0) *scale = s;
  return s;  // on every lane
}

// Quantizes one row per block of 128 elements (w4a4-g128 activations), one
// wavefront: a block is 16 chunks of 8, one per lane of a 16-lane group, whose
// maximum the group shares; the fp32 recipe of quant_row per block.
__device__ inline void quant_row_groups(const uint4* __restrict__ row, int cols, int act, int qmax,
                                        uint2* __restrict__ codes, float* __restrict__ scales) {
  const int lane = threadIdx.x & 63, nch = cols >> 3;
  const uint32_t nan_lo = act == MXMOE_BF16 ? 0x7f81u : 0x7c01u;
  const float q = (float)qmax;
  for (int c0 = 0; c0 < nch; c0 += 64) {  // nch is a multiple of 16: groups stay whole
    const int c = c0 + lane;
    const bool ok = c < nch;
    const uint4 v = ok ? row[c] : make_uint4(0u, 0u, 0u, 0u);
    uint32_t mb = amax8_bits(v, nan_lo);
    for (int d = 1; d < 16; d <<= 1) mb = max(mb, (uint32_t)__shfl_xor((int)mb, d, 64));
    const float amax = bits_to_f32(mb, act);
    float inv = 0.f, sc = 0.f;
    if (amax > 0.f) {
      inv = __fdiv_rn(q, amax);
      sc = __fdiv_rn(amax, q);
    }
    if (ok) codes[c] = codes8(v, act, inv, q);
    if (ok && (lane & 15) == 0) scales[c >> 4] = sc;
  }
}

// MXFP4 encoding of one row (OCP MX: FP4 e2m1 elements, one E8M0 scale per 32
// consecutive values), one wavefront: a lane takes a whole 32-wide block (64
// bytes) per step.  Shared exponent e = floor(log2(amax)) - 2, clamped to
// [-127, 127] (-127 for an all-zero block); element = nearest e2m1 value to
// |a| 2^-e (an exact power-of-two scaling of a 16-bit value), ties to the even
// code, clamped to 6; the sign is kept unless the magnitude code is 0.
// Element i of the block is nibble i of its 16 output bytes.
__device__ inline uint32_t e2m1_mag(float x) {
  return (uint32_t)(x > 0.25f) + (uint32_t)(x >= 0.75f) + (uint32_t)(x > 1.25f) + (uint32_t)(x >= 1.75f) +
         (uint32_t)(x > 2.5f) + (uint32_t)(x >= 3.5f) + (uint32_t)(x > 5.0f);
}
__device__ inline void quant_row_mx(const uint4* __restrict__ row, int cols, int act, uint4* __restrict__ codes,
                                    uint8_t* __restrict__ exps) {
  const int lane = threadIdx.x & 63, nb = cols >> 5;
  for (int b = lane; b < nb; b += 64) {
    float v[32];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint4 u = row[4 * b + c];
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint16_t lo = (uint16_t)(w[i] & 0xFFFFu), hi = (uint16_t)(w[i] >> 16);
        v[8 * c + 2 * i] = act == MXMOE_BF16 ? __uint_as_float((uint32_t)lo << 16) : (float)__builtin_bit_cast(_Float16, lo);
        v[8 * c + 2 * i + 1] = act == MXMOE_BF16 ? __uint_as_float((uint32_t)hi << 16) : (float)__builtin_bit_cast(_Float16, hi);
      }
    }
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < 32; ++i) amax = fmaxf(amax, fabsf(v[i]));
    int e = amax > 0.f ? (int)((__float_as_uint(amax) >> 23) & 0xFFu) - 127 - 2 : -127;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    const float inv = __builtin_amdgcn_ldexpf(1.0f, -e);
    uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      uint32_t c = e2m1_mag(fabsf(v[i]) * inv);
      if (v[i] < 0.f && c) c |= 8u;
      o[i >> 3] |= c << (4 * (i & 7));
    }
    codes[b] = make_uint4(o[0], o[1], o[2], o[3]);
    exps[b] = (uint8_t)(e + 127);
  }
}

// Row sums of each 128-wide block of one bf16 row (one wavefront): a block is
// 16 chunks of 8 elements, one per lane of a 16-lane group; each lane adds its
// 8 values in order, then the group adds its lanes pairwise.
__device__ inline void rowsum_row(const uint4* __restrict__ row, int cols, float* __restrict__ out) {
  const int lane = threadIdx.x & 63, nch = cols >> 3;
  for (int c0 = 0; c0 < nch; c0 += 64) {  // nch is a multiple of 16: groups stay whole
    const int c = c0 + lane;
    float sum = 0.f;
    if (c < nch) {
      float f[8];
      unpack8(row[c], MXMOE_BF16, f);
#pragma unroll
      for (int i = 0; i < 8; ++i) sum += f[i];
    }
    for (int d = 1; d < 16; d <<= 1) sum += __shfl_xor(sum, d, 64);
    if ((lane & 15) == 0 && c < nch) out[c >> 4] = sum;
  }
}

// Every encoding of x row r that the block's gate/up linears read (one
// wavefront; the same recipes as the separate row kernels).
__device__ inline void x_prep_row(const XPrep& p, int64_t r) {
  const int cols = p.cols;
  const uint4* row = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(p.x) + r * cols);
  const int lane = threadIdx.x & 63;
  // the token's routed rows get their copy of a per-token scale
  auto to_rows = [&](float* dst, float v) {
    if (!p.inv || !dst) return;
    for (int sl = lane; sl < p.k; sl += 64) {
      const int32_t j = p.inv[r * p.k + sl];
      if (j >= 0) dst[j] = v;
    }
  };
  if (cols <= 4096 && (p.q8 || p.q4 || p.qf8 || p.qf6)) {
    // the per-token encodings share the row maximum: the row is loaded and
    // reduced once, then each encoding is formed from the registers (the
    // recipes of quant_row_vec, so the codes and scales are the same)
    const int nch = cols >> 3;
    const uint32_t nan_lo = p.act == MXMOE_BF16 ? 0x7f81u : 0x7c01u;
    uint4 v[8];
    uint32_t mb = 0u;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = lane + 64 * i;
      v[i] = c < nch ? row[c] : make_uint4(0u, 0u, 0u, 0u);
      mb = max(mb, amax8_bits(v[i], nan_lo));
    }
    for (int d = 32; d > 0; d >>= 1) mb = max(mb, (uint32_t)__shfl_xor((int)mb, d, 64));
    const float amax = bits_to_f32(mb, p.act);
    auto enc = [&](uint8_t* codes, float* scale, int qmax, bool f6) {
      const float q = (float)qmax;
      float inv = 0.f, sc = 0.f;
      if (amax > 0.f) {
        inv = __fdiv_rn(q, amax);
        sc = __fdiv_rn(amax, q);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int c = lane + 64 * i;
        if (c < nch) {
          if (f6) store_f6_chunk(codes, c, codes8_f6(v[i], p.act, inv));
          else reinterpret_cast<uint2*>(codes)[c] = codes8(v[i], p.act, inv, q);
        }
      }
      if (lane == 0) *scale = sc;
      return sc;
    };
    if (p.q8) to_rows(p.r8, enc(reinterpret_cast<uint8_t*>(p.q8 + r * cols), p.s8 + r, 127, false));
    if (p.q4) to_rows(p.r4, enc(reinterpret_cast<uint8_t*>(p.q4 + r * cols), p.s4 + r, 7, false));
    if (p.qf8) enc(p.qf8 + r * cols, p.sf8 + r, kQmaxF8, false);
    if (p.qf6) enc(p.qf6 + r * cols, p.sf6 + r, 7, true);
  } else {  // longer rows: each encoding streams the row
    if (p.q8)
      to_rows(p.r8, quant_row_vec<0, 1>(row, cols, p.act, 127, reinterpret_cast<uint2*>(p.q8 + r * cols), p.s8 + r,
                                        nullptr));
    if (p.q4)
      to_rows(p.r4, quant_row_vec<0, 1>(row, cols, p.act, 7, reinterpret_cast<uint2*>(p.q4 + r * cols), p.s4 + r,
                                        nullptr));
    if (p.qf8)
      quant_row_vec<0, 1>(row, cols, p.act, kQmaxF8, reinterpret_cast<uint2*>(p.qf8 + r * cols), p.sf8 + r, nullptr);
    if (p.qf6)
      quant_row_vec<0, 1, true>(row, cols, p.act, 7, reinterpret_cast<uint2*>(p.qf6 + r * cols), p.sf6 + r, nullptr);
  }
  if (p.rs) rowsum_row(row, cols, p.rs + r * (cols >> 7));
  if (p.q4g)
    quant_row_groups(row, cols, p.act, 7, reinterpret_cast<uint2*>(p.q4g + r * cols), p.s4g + r * (cols >> 7));
  if (p.qmx)
    quant_row_mx(row, cols, p.act, reinterpret_cast<uint4*>(p.qmx + r * (cols >> 1)), p.smx + r * (cols >> 5));
}

}  // namespace
}  // namespace mxmoe
