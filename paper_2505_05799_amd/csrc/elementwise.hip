// HBM-bound row kernels of the block forward:
//   * dynamic per-token activation quantization (Sec. 4.2.2; per-token
//     granularity a_gsize = -1 of the W5A5 allocation table) for x and for the
//     gated intermediate h of a8/a4 down projections;
//   * the weighted combine of Eq. (2): the per-slot down rows, already scaled
//     by their gate weight, are summed in a fixed order in fp32 and rounded
//     once to the activation dtype.
#include "mxmoe_internal.h"

namespace mxmoe {
namespace {

constexpr int kThreads = 256;

__device__ inline float load_act(const void* p, int64_t i, int act) {
  uint16_t b = reinterpret_cast<const uint16_t*>(p)[i];
  if (act == MXMOE_BF16) return __uint_as_float(((uint32_t)b) << 16);
  return (float)*reinterpret_cast<const _Float16*>(&b);
}

__device__ inline uint16_t f32_to_act(float f, int act) {
  if (act == MXMOE_BF16) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);  // quiet NaN
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
  }
  _Float16 h = (_Float16)f;
  return *reinterpret_cast<uint16_t*>(&h);
}

__device__ inline float block_max(float v, float* red) {
  for (int d = 32; d > 0; d >>= 1) v = fmaxf(v, __shfl_xor(v, d, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float m = red[0];
  for (int i = 1; i < kThreads / 64; ++i) m = fmaxf(m, red[i]);
  __syncthreads();
  return m;
}

// One row: amax, then codes with the fp32 recipe.
__device__ inline void quant_row(const void* a, int64_t row_off, int cols, int act, int qmax,
                                 int8_t* __restrict__ codes, float* __restrict__ scale, float* red) {
  float m = 0.f;
  for (int c = threadIdx.x; c < cols; c += kThreads) m = fmaxf(m, fabsf(load_act(a, row_off + c, act)));
  const float amax = block_max(m, red);
  const float q = (float)qmax;
  float inv = 0.f, s = 0.f;
  if (amax > 0.f) {
    inv = __fdiv_rn(q, amax);
    s = __fdiv_rn(amax, q);
  }
  for (int c = threadIdx.x; c < cols; c += kThreads) {
    float v = load_act(a, row_off + c, act);
    float r = __builtin_rintf(__fmul_rn(v, inv));
    r = fminf(fmaxf(r, -q), q);
    codes[c] = (int8_t)(int)r;
  }
  if (threadIdx.x == 0) *scale = s;
}

__global__ void __launch_bounds__(kThreads) act_quant_kernel(const void* a, int act, int cols, int64_t ld, int qmax,
                                                             int8_t* codes, float* scales) {
  __shared__ float red[kThreads / 64];
  const int64_t r = blockIdx.x;
  quant_row(a, r * ld, cols, act, qmax, codes + r * cols, scales + r, red);
}

__global__ void __launch_bounds__(kThreads) hquant_routed_kernel(const void* h, int act, int F,
                                                                 const int32_t* __restrict__ offsets, int E,
                                                                 const int32_t* __restrict__ down_qmax,
                                                                 int8_t* hq, float* hs) {
  __shared__ float red[kThreads / 64];
  const int r = blockIdx.x;
  if (r >= offsets[E]) return;
  int lo = 0, hi = E;  // largest e with offsets[e] <= r
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (offsets[mid] <= r) lo = mid; else hi = mid;
  }
  const int qmax = down_qmax[lo];
  if (qmax == 0) return;
  quant_row(h, (int64_t)r * F, F, act, qmax, hq + (int64_t)r * F, hs + r, red);
}

__global__ void __launch_bounds__(kThreads) combine_kernel(const float* __restrict__ slots,
                                                           const int32_t* __restrict__ ids, int T, int k, int E,
                                                           int nsh, int H, int act, uint16_t* __restrict__ y) {
  const int64_t i4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;  // index of 4 outputs
  const int q4 = H / 4;
  if (i4 >= (int64_t)T * q4) return;
  const int t = (int)(i4 / q4), h = (int)(i4 % q4) * 4;
  const int S = k + nsh;
  const float* base = slots + (int64_t)t * S * H + h;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < S; ++s) {
    if (s < k) {
      int e = ids[(int64_t)t * k + s];
      if (e < 0 || e >= E) continue;
    }
    float4 v = *reinterpret_cast<const float4*>(base + (int64_t)s * H);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  uint2 o;
  o.x = (uint32_t)f32_to_act(acc.x, act) | ((uint32_t)f32_to_act(acc.y, act) << 16);
  o.y = (uint32_t)f32_to_act(acc.z, act) | ((uint32_t)f32_to_act(acc.w, act) << 16);
  *reinterpret_cast<uint2*>(y + (int64_t)t * H + h) = o;
}

// Per-row data of the sorted (token, slot) pairs, read by every Group-GEMM
// tile with contiguous loads instead of gathers through the permutation.
__global__ void row_meta_kernel(const int32_t* __restrict__ sorted_pair, const int32_t* __restrict__ offsets, int E,
                                int k, int n_sh, const float* __restrict__ topk_w, const float* __restrict__ xs8,
                                const float* __restrict__ xs4, int32_t* __restrict__ rtok, int32_t* __restrict__ rslot,
                                float* __restrict__ rgw, float* __restrict__ rxs8, float* __restrict__ rxs4) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= offsets[E]) return;  // pairs dropped for an invalid expert id have no row
  const int p = sorted_pair[j];
  const int t = p / k, sl = p - t * k;
  rtok[j] = t;
  rslot[j] = t * (k + n_sh) + sl;
  rgw[j] = topk_w[p];
  if (xs8) rxs8[j] = xs8[t];
  if (xs4) rxs4[j] = xs4[t];
}

}  // namespace

hipError_t launch_row_meta(const int32_t* sorted_pair, const int32_t* offsets, int E, int P, int k, int n_sh,
                           const float* topk_w, const float* xs8, const float* xs4, int32_t* rtok, int32_t* rslot,
                           float* rgw, float* rxs8, float* rxs4, hipStream_t s) {
  if (P <= 0) return hipSuccess;
  hipLaunchKernelGGL(row_meta_kernel, dim3((P + kThreads - 1) / kThreads), dim3(kThreads), 0, s, sorted_pair, offsets,
                     E, k, n_sh, topk_w, xs8, xs4, rtok, rslot, rgw, rxs8, rxs4);
  return hipGetLastError();
}

hipError_t launch_act_quant(const void* a, int act, int rows, int cols, int64_t ld, int qmax, int8_t* codes,
                            float* scales, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(act_quant_kernel, dim3(rows), dim3(kThreads), 0, s, a, act, cols, ld, qmax, codes, scales);
  return hipGetLastError();
}

hipError_t launch_hquant_routed(const void* h, int act, int P, int F, const int32_t* offsets, int E,
                                const int32_t* down_qmax, int8_t* hq, float* hs, hipStream_t s) {
  if (P <= 0) return hipSuccess;
  hipLaunchKernelGGL(hquant_routed_kernel, dim3(P), dim3(kThreads), 0, s, h, act, F, offsets, E, down_qmax, hq, hs);
  return hipGetLastError();
}

hipError_t launch_combine(const float* slots, const int32_t* ids, int T, int k, int E, int nsh, int H, int act,
                          void* y, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  int64_t n4 = (int64_t)T * (H / 4);
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)((n4 + kThreads - 1) / kThreads)), dim3(kThreads), 0, s, slots,
                     ids, T, k, E, nsh, H, act, (uint16_t*)y);
  return hipGetLastError();
}

}  // namespace mxmoe
