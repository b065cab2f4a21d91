// Weight packer: codes + scales (+ zeros) of one linear -> fragment blocks in
// MFMA lane order (the layout the Group-GEMM micro-kernels stream), and its
// inverse for inspection.
//
// Lane l of a 16 x 128 fragment block owns output row n = 16*nb + l%16 and the
// reduction quarter qd = l/16.  Its 32 values, in slot order v = 0..31, are
//   16-bit MFMA kinds (w16, wNg128): k = 128*kb + 32*(v/8) + 8*qd + v%8
//   int8 MFMA kinds  (w8a8, w4a4):   k = 128*kb + 64*(v/16) + 16*qd + v%16
// so that one 16x16x32 bf16/fp16 MFMA (or one 16x16x64 int8 MFMA) consumes
// slots 8j..8j+7 (16j..16j+15) of every lane.  Encodings of the slots:
//   w16  : 32 x 16-bit values in slot order
//   w8g  : 32 x uint8 codes in slot order
//   w4g  : dword j holds slots 8j..8j+7 as nibbles (slot 8j+i at bits 4i)
//   w2g  : dword d holds slots 16d..16d+15 as 2-bit fields (bits 2i)
//   w3g  : dwords 0,1 = low two bits as w2g, dword 2 bit v = bit 2 of slot v
//   w8a8 : 32 x int8 codes in slot order
//   w4a4 : dword 2j+d holds slots 16j+8d..+7 as 4-bit two's complement
//          nibbles; nibble 2i is slot i, nibble 2i+1 is slot 4+i (i < 4) so
//          that (D << 4) & 0xF0F0F0F0 and D & 0xF0F0F0F0 are the int8 slots
//          (times 16) in order.
// Weight-only blocks end with 16 (scale, zero) fp16 pairs, one per row.
#include "mxmoe_internal.h"

namespace mxmoe {
namespace {

__device__ inline int slot_k(int kd, int v, int qd) {
  if (kind_is_int(kd)) return 64 * (v >> 4) + 16 * qd + (v & 15);
  return 32 * (v >> 3) + 8 * qd + (v & 7);
}

__device__ inline uint16_t cvt16(uint16_t bits, int src, int act) {
  if (src == act) return bits;
  if (src == MXMOE_BF16) {  // bf16 -> fp16, RNE
    float f = __uint_as_float(((uint32_t)bits) << 16);
    _Float16 h = (_Float16)f;
    return *reinterpret_cast<uint16_t*>(&h);
  }
  // fp16 -> bf16, RNE
  _Float16 h = *reinterpret_cast<_Float16*>(&bits);
  float f = (float)h;
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
  uint32_t w[16];
  for (int i = 0; i < 16; ++i) w[i] = 0;
  switch (kd) {
    case K_W16: {
      const uint16_t* c16 = reinterpret_cast<const uint16_t*>(codes);
      for (int v = 0; v < 32; ++v) {
        uint16_t b = cvt16(c16[rbase + slot_k(kd, v, qd)], w16_src, act);
        w[v >> 1] |= (uint32_t)b << (16 * (v & 1));
      }
      break;
    }
    case K_W8G:
    case K_W8A8:
      for (int v = 0; v < 32; ++v) w[v >> 2] |= (uint32_t)codes[rbase + slot_k(kd, v, qd)] << (8 * (v & 3));
      break;
    case K_W4G:
      for (int v = 0; v < 32; ++v) w[v >> 3] |= ((uint32_t)codes[rbase + slot_k(kd, v, qd)] & 15u) << (4 * (v & 7));
      break;
    case K_W2G:
      for (int v = 0; v < 32; ++v) w[v >> 4] |= ((uint32_t)codes[rbase + slot_k(kd, v, qd)] & 3u) << (2 * (v & 15));
      break;
    case K_W3G:
      for (int v = 0; v < 32; ++v) {
        uint32_t c = codes[rbase + slot_k(kd, v, qd)] & 7u;
        w[v >> 4] |= (c & 3u) << (2 * (v & 15));
        w[2] |= (c >> 2) << v;
      }
      break;
    case K_W4A4:
      for (int v = 0; v < 32; ++v) {
        uint32_t c = codes[rbase + slot_k(kd, v, qd)] & 15u;  // two's complement nibble
        int j = v >> 4, i = v & 15, d = i >> 3, ii = i & 7;
        int nib = ii < 4 ? 2 * ii : 2 * (ii - 4) + 1;
        w[2 * j + d] |= c << (4 * nib);
      }
      break;
  }
  uint32_t* o32 = reinterpret_cast<uint32_t*>(out);
  for (int i = 0; i < lane_bytes(kd) / 4; ++i) o32[i] = w[i];
  if (kind_is_wonly(kd) && qd == 0) {
    const uint16_t* s16 = reinterpret_cast<const uint16_t*>(scales);
    const uint16_t* z16 = reinterpret_cast<const uint16_t*>(zeros);
    int64_t g = (int64_t)row * kblocks + kb;
    uint32_t sz = (uint32_t)s16[g] | ((uint32_t)z16[g] << 16);
    reinterpret_cast<uint32_t*>(packed + blk * block_bytes(kd) + 64 * lane_bytes(kd))[lane & 15] = sz;
  }
  if (kind_is_int(kd) && kb == 0 && qd == 0) {
    float* ws = reinterpret_cast<float*>(packed + codes_bytes(kd, n, k));
    ws[row] = reinterpret_cast<const float*>(scales)[row];
  }
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
    int64_t idx = rbase + slot_k(kd, v, qd);
    switch (kd) {
      case K_W16:
        reinterpret_cast<uint16_t*>(codes)[idx] = (uint16_t)(w[v >> 1] >> (16 * (v & 1)));
        break;
      case K_W8G:
      case K_W8A8:
        codes[idx] = (uint8_t)(w[v >> 2] >> (8 * (v & 3)));
        break;
      case K_W4G:
        codes[idx] = (uint8_t)((w[v >> 3] >> (4 * (v & 7))) & 15u);
        break;
      case K_W2G:
        codes[idx] = (uint8_t)((w[v >> 4] >> (2 * (v & 15))) & 3u);
        break;
      case K_W3G:
        codes[idx] = (uint8_t)(((w[v >> 4] >> (2 * (v & 15))) & 3u) | (((w[2] >> v) & 1u) << 2));
        break;
      case K_W4A4: {
        int j = v >> 4, i = v & 15, d = i >> 3, ii = i & 7;
        int nib = ii < 4 ? 2 * ii : 2 * (ii - 4) + 1;
        uint32_t c = (w[2 * j + d] >> (4 * nib)) & 15u;
        codes[idx] = (uint8_t)(int8_t)((int32_t)(c << 28) >> 28);  // sign-extend
        break;
      }
    }
  }
  if (kind_is_wonly(kd) && qd == 0) {
    uint32_t sz = reinterpret_cast<const uint32_t*>(packed + blk * block_bytes(kd) + 64 * lane_bytes(kd))[lane & 15];
    int64_t g = (int64_t)row * kblocks + kb;
    reinterpret_cast<uint16_t*>(scales)[g] = (uint16_t)(sz & 0xFFFF);
    reinterpret_cast<uint16_t*>(zeros)[g] = (uint16_t)(sz >> 16);
  }
  if (kind_is_int(kd) && kb == 0 && qd == 0) {
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
