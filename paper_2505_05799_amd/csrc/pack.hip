// Weight packer: codes + scales (+ zeros) of one linear -> fragment blocks in
// MFMA lane order (the layout the Group-GEMM micro-kernels stream), and its
// inverse for inspection.
//
// Lane l of a 16 x 128 fragment block owns output channel n = 16*nb + l%16
// and the reduction quarter qd = l/16.  Its 32 values, in slot order
// v = 0..31, are
//   16-bit MFMA kinds (w16, wNg128): k = 128*kb + 32*(v/8) + 8*qd + v%8
//   int8 MFMA kinds  (w8a8, w4a4, w4a4-g128): k = 128*kb + 64*(v/16) + 16*qd + v%16
// so that one 16x16x32 bf16/fp16 MFMA (or one 16x16x64 int8 MFMA) consumes
// slots 8j..8j+7 (16j..16j+15) of every lane.  Slot encodings (j = v/8 is the
// MFMA step, p = (v%8)/2 the 16-bit pair, h = v%2 the half of the pair):
//   w16  : 32 x 16-bit values in slot order
//   w8g  : 32 x uint8 codes in slot order
//   w4g  : dword j; slot at bits 16h + 4p        (pair p = (D >> 4p) & 0x000F000F)
//   w2g  : dword j/2; slot at bits 16h + 2P with P = 4(j%2) + p
//   w3g  : low two bits as w2g; bit 2 of the slot in dword 2 at bit 16h + P'
//          with P' = 4j + p
//   w8a8 : 32 x int8 codes in slot order
//   w4a4 (and w4a4-g128): dword 2j+d holds slots 16j+8d..+7 as 4-bit two's complement
//          nibbles; nibble 2i is slot i, nibble 2i+1 is slot 4+i (i < 4) so
//          that (D << 4) & 0xF0F0F0F0 and D & 0xF0F0F0F0 are the int8 slots
//          (times 16) in order.
// Weight-only blocks end with 16 (scale, zero) fp16 pairs, one per channel.
// A group whose scale is zero dequantizes to zero whatever its codes: it is
// stored with scale 1 and every code equal to its zero point (same values).
// w4a4-g128 blocks end with 16 (scale, 0) pairs; a zero scale stays zero.
//   mxfp4: lane l holds k = 128*kb + 32*qd + v for v = 0..31, slot v in nibble
//          v (dword v/8, bits 4(v%8)): the operand layout of one 16x16x128 FP4
//          MFMA.  The block ends with 16 dwords, one per channel, whose byte b
//          is the E8M0 scale of the channel's 32-wide block b of this k block.
//   w4a4 on FP6 operands: lane l holds k = 128*kb + 32*qd + v, slot v as the
//          6-bit e2m3 code of the int4 value at bits 6v..6v+5 of the lane's 24
//          bytes (the operand layout of one 16x16x128 FP6 MFMA); per-channel
//          fp32 scales after the last block, as w4a4.
#include "mxmoe_internal.h"
#include "rowquant.h"

namespace mxmoe {
namespace {

__device__ inline int slot_k(int kd, int v, int qd) {
  if (kd == K_MXFP4 || kd == K_W4A4F6) return 32 * qd + v;
  if (kind_is_int(kd)) return 64 * (v >> 4) + 16 * qd + (v & 15);
  return 32 * (v >> 3) + 8 * qd + (v & 7);
}

// position of the (low) code field of slot v: dword index and bit offset
__device__ inline void slot_field(int kd, int v, int* dw, int* bit, uint32_t* mask) {
  const int j = v >> 3, i = v & 7, p = i >> 1, h = i & 1;
  switch (kd) {
    case K_W16: *dw = v >> 1; *bit = 16 * (v & 1); *mask = 0xFFFFu; break;
    case K_W8G:
    case K_W8A8:
    case K_F8A8: *dw = v >> 2; *bit = 8 * (v & 3); *mask = 0xFFu; break;
    case K_W4G: *dw = j; *bit = 16 * h + 4 * p; *mask = 0xFu; break;
    case K_W2G:
    case K_W3G: *dw = j >> 1; *bit = 16 * h + 2 * (4 * (j & 1) + p); *mask = 0x3u; break;
    case K_MXFP4: *dw = v >> 3; *bit = 4 * (v & 7); *mask = 0xFu; break;
    default: {  // K_W4A4
      const int jj = v >> 4, ii = v & 15, d = ii >> 3, i8 = ii & 7;
      *dw = 2 * jj + d;
      *bit = 4 * (i8 < 4 ? 2 * i8 : 2 * (i8 - 4) + 1);
      *mask = 0xFu;
    }
  }
}
__device__ inline int w3_hibit(int v) {
  const int j = v >> 3, i = v & 7;
  return 16 * (i & 1) + 4 * j + (i >> 1);
}

__device__ inline uint16_t cvt16(uint16_t bits, int src, int act) {
  if (src == act) return bits;
  if (src == MXMOE_BF16) {  // bf16 -> fp16, RNE
    float f = __uint_as_float(((uint32_t)bits) << 16);
    _Float16 h = (_Float16)f;
    return __builtin_bit_cast(uint16_t, h);
  }
  float f = (float)__builtin_bit_cast(_Float16, bits);  // fp16 -> bf16, RNE
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ void pack_kernel(int kd, int n, int k, int act, int w16_src,
                            const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                            const uint8_t* __restrict__ zeros, uint8_t* __restrict__ packed) {
  const int kblocks = k / 128;
  const int64_t nblk = (int64_t)(n / 16) * kblocks;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= nblk * 64) return;
  const int lane = (int)(gid & 63);
  const int64_t blk = gid >> 6;
  const int nb = (int)(blk / kblocks), kb = (int)(blk % kblocks);
  const int row = nb * 16 + (lane & 15), qd = lane >> 4;
  const int64_t rbase = (int64_t)row * k + (int64_t)kb * 128;
  uint8_t* out = packed + blk * block_bytes(kd) + lane * lane_bytes(kd);
  // group metadata (weight-only): zero-scale groups become scale 1, codes = zero
  uint16_t s16 = 0, z16 = 0;
  bool zero_group = false;
  if (kind_is_wonly(kd)) {
    const int64_t g = (int64_t)row * kblocks + kb;
    s16 = reinterpret_cast<const uint16_t*>(scales)[g];
    z16 = reinterpret_cast<const uint16_t*>(zeros)[g];
    zero_group = (s16 & 0x7FFFu) == 0;
    if (zero_group) s16 = 0x3C00u;  // 1.0
  } else if (kd == K_W4A4G) {
    s16 = reinterpret_cast<const uint16_t*>(scales)[(int64_t)row * kblocks + kb];
  }
  uint32_t mxs = 0;  // mxfp4: the four E8M0 bytes of the channel's 32-wide blocks of this k block
  if (kd == K_MXFP4) {
    const uint8_t* e = scales + (int64_t)row * (k / 32) + 4 * kb;
    mxs = (uint32_t)e[0] | ((uint32_t)e[1] << 8) | ((uint32_t)e[2] << 16) | ((uint32_t)e[3] << 24);
  }
  const uint32_t zcode = zero_group ? (uint32_t)(float)__builtin_bit_cast(_Float16, z16) : 0u;
  // Inputs outside the documented domain - a zero point that is not an
  // integer in [0, 2^N - 1], a weight-only code above 2^N - 1, a w4a4 code
  // outside [-7, 7] - cannot be represented exactly by the packed form; they
  // make the group's scale NaN, so every output that uses the group is NaN
  // rather than silently wrong (per-channel w4a4: poison_channels_kernel).
  const float qtop = (float)((1 << kind_wbits(kd)) - 1);
  bool bad = false;
  if (kind_is_wonly(kd)) {
    const float zf = (float)__builtin_bit_cast(_Float16, z16);
    bad = !(zf >= 0.f && zf <= qtop && zf == __builtin_rintf(zf));
  }
  uint32_t w[16];
  for (int i = 0; i < 16; ++i) w[i] = 0;
  for (int v = 0; v < 32; ++v) {
    const int64_t idx = rbase + slot_k(kd, v, qd);
    uint32_t c;
    if (kd == K_W16) c = cvt16(reinterpret_cast<const uint16_t*>(codes)[idx], w16_src, act);
    else c = zero_group ? zcode : (uint32_t)codes[idx];
    if (kind_is_wonly(kd) && !zero_group && (float)c > qtop) bad = true;
    if (kd == K_W4A4G) {
      const int sc = (int)(int8_t)codes[idx];
      bad |= sc < -7 || sc > 7;
    }
    if (kd == K_W4A4F6) {  // 6-bit e2m3 field at bit 6v, possibly across two dwords
      const uint32_t e = e2m3_of_int((int)(int8_t)c) & 63u;
      const int b = 6 * v;
      w[b >> 5] |= e << (b & 31);
      if ((b & 31) > 26) w[(b >> 5) + 1] |= e >> (32 - (b & 31));
      continue;
    }
    int dw, bit;
    uint32_t mask;
    slot_field(kd, v, &dw, &bit, &mask);
    w[dw] |= (c & mask) << bit;
    if (kd == K_W3G) w[2] |= ((c >> 2) & 1u) << w3_hibit(v);
  }
  uint32_t* o32 = reinterpret_cast<uint32_t*>(out);
  for (int i = 0; i < lane_bytes(kd) / 4; ++i) o32[i] = w[i];
  // the four lanes of a channel (lane % 16 + 16 qd, qd = 0..3) share its
  // group: an OR over lane ^ 16, then over lane ^ 32, by every lane
  int b = bad ? 1 : 0;
  b |= __shfl_xor(b, 16, 64);
  b |= __shfl_xor(b, 32, 64);
  if (b) s16 = 0x7E00u;  // fp16 NaN
  if (kind_has_gmeta(kd) && qd == 0) {
    const uint32_t sz = kd == K_MXFP4 ? mxs : ((uint32_t)s16 | ((uint32_t)z16 << 16));
    reinterpret_cast<uint32_t*>(packed + blk * block_bytes(kd) + 64 * lane_bytes(kd))[lane & 15] = sz;
  }
  if (kind_is_int(kd) && kd != K_W4A4G && kb == 0 && qd == 0) {
    float* ws = reinterpret_cast<float*>(packed + codes_bytes(kd, n, k));
    ws[row] = reinterpret_cast<const float*>(scales)[row];
  }
}

// Per-channel w4a4 (int8 or FP6 operands): a channel with a code outside
// [-7, 7] gets a NaN scale
// (after pack_kernel wrote the scales, same stream), one workgroup per channel.
__global__ void __launch_bounds__(256) poison_channels_kernel(int n, int k, const int8_t* __restrict__ codes,
                                                              float* __restrict__ wscale) {
  __shared__ int any;
  if (threadIdx.x == 0) any = 0;
  __syncthreads();
  const int64_t row = blockIdx.x;
  int bad = 0;
  for (int c = threadIdx.x; c < k; c += blockDim.x) {
    const int v = codes[row * k + c];
    bad |= v < -7 || v > 7;
  }
  if (bad) atomicOr(&any, 1);
  __syncthreads();
  if (threadIdx.x == 0 && any) wscale[row] = __builtin_nanf("");
}

__global__ void unpack_kernel(int kd, int n, int k, int act, const uint8_t* __restrict__ packed,
                              uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                              uint8_t* __restrict__ zeros) {
  const int kblocks = k / 128;
  const int64_t nblk = (int64_t)(n / 16) * kblocks;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= nblk * 64) return;
  const int lane = (int)(gid & 63);
  const int64_t blk = gid >> 6;
  const int nb = (int)(blk / kblocks), kb = (int)(blk % kblocks);
  const int row = nb * 16 + (lane & 15), qd = lane >> 4;
  const int64_t rbase = (int64_t)row * k + (int64_t)kb * 128;
  const uint32_t* w = reinterpret_cast<const uint32_t*>(packed + blk * block_bytes(kd) + lane * lane_bytes(kd));
  for (int v = 0; v < 32; ++v) {
    const int64_t idx = rbase + slot_k(kd, v, qd);
    if (kd == K_W4A4F6) {  // e2m3 field -> the integer it holds
      const int b = 6 * v;
      uint32_t e = w[b >> 5] >> (b & 31);
      if ((b & 31) > 26) e |= w[(b >> 5) + 1] << (32 - (b & 31));
      e &= 63u;
      const int ex = (int)((e >> 3) & 3u), mn = (int)(e & 7u);
      const int mag = ex == 0 ? 0 : ((8 + mn) << (ex - 1)) >> 3;  // (1 + m/8) 2^(ex-1) for the integer codes
      codes[idx] = (uint8_t)(int8_t)((e & 32u) ? -mag : mag);
      continue;
    }
    int dw, bit;
    uint32_t mask;
    slot_field(kd, v, &dw, &bit, &mask);
    uint32_t c = (w[dw] >> bit) & mask;
    if (kd == K_W3G) c |= ((w[2] >> w3_hibit(v)) & 1u) << 2;
    if (kd == K_W16) reinterpret_cast<uint16_t*>(codes)[idx] = (uint16_t)c;
    else if (kd == K_W4A4 || kd == K_W4A4G) codes[idx] = (uint8_t)(int8_t)((int32_t)(c << 28) >> 28);  // sign-extend
    else codes[idx] = (uint8_t)c;
  }
  if (kind_has_gmeta(kd) && qd == 0) {
    uint32_t sz = reinterpret_cast<const uint32_t*>(packed + blk * block_bytes(kd) + 64 * lane_bytes(kd))[lane & 15];
    if (kd == K_MXFP4) {
      uint8_t* e = scales + (int64_t)row * (k / 32) + 4 * kb;
      for (int b = 0; b < 4; ++b) e[b] = (uint8_t)(sz >> (8 * b));
      return;
    }
    int64_t g = (int64_t)row * kblocks + kb;
    reinterpret_cast<uint16_t*>(scales)[g] = (uint16_t)(sz & 0xFFFF);
    if (kind_is_wonly(kd)) reinterpret_cast<uint16_t*>(zeros)[g] = (uint16_t)(sz >> 16);
  }
  if (kind_is_int(kd) && kd != K_W4A4G && kb == 0 && qd == 0) {
    const float* ws = reinterpret_cast<const float*>(packed + codes_bytes(kd, n, k));
    reinterpret_cast<float*>(scales)[row] = ws[row];
  }
}

}  // namespace

hipError_t launch_pack(int kind, int n, int k, int act, int w16_src, const void* codes,
                       const void* scales, const void* zeros, uint8_t* packed, hipStream_t s) {
  int64_t threads = (int64_t)(n / 16) * (k / 128) * 64;
  int64_t blocks = (threads + 255) / 256;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(256), 0, s, kind, n, k, act, w16_src,
                     (const uint8_t*)codes, (const uint8_t*)scales, (const uint8_t*)zeros, packed);
  if (kind == K_W4A4 || kind == K_W4A4F6) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(poison_channels_kernel, dim3((unsigned)n), dim3(256), 0, s, n, k, (const int8_t*)codes,
                       reinterpret_cast<float*>(packed + codes_bytes(kind, n, k)));
  }
  return hipGetLastError();
}

hipError_t launch_unpack(int kind, int n, int k, int act, const uint8_t* packed, void* codes,
                         void* scales, void* zeros, hipStream_t s) {
  int64_t threads = (int64_t)(n / 16) * (k / 128) * 64;
  int64_t blocks = (threads + 255) / 256;
  hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)blocks), dim3(256), 0, s, kind, n, k, act, packed,
                     (uint8_t*)codes, (uint8_t*)scales, (uint8_t*)zeros);
  return hipGetLastError();
}

}  // namespace mxmoe
