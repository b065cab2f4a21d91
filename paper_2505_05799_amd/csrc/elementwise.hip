// HBM-bound row kernels of the block forward:
//   * dynamic per-token activation quantization (Sec. 4.2.2; per-token
//     granularity a_gsize = -1 of the W5A5 allocation table) of the gated
//     intermediate h of a8/a4 down projections, and of the input of a single
//     linear (the block forward encodes x inside the plan launch, with the
//     same row encoders);
//   * the weighted combine of Eq. (2): the per-slot down rows, already scaled
//     by their gate weight, are summed in a fixed order in fp32 and rounded
//     once to the activation dtype.
#include "mxmoe_internal.h"
#include "rowquant.h"

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
    if (qmax == kQmaxF8) {
      codes[c] = (int8_t)e4m3_byte(__fmul_rn(v, inv));
      continue;
    }
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

// ---- one wavefront per row, 16-byte loads (8 elements per lane and chunk)
constexpr int kRowsPerBlock = kThreads / 64;

__global__ void __launch_bounds__(kThreads) act_quant_mx_kernel(const void* a, int act, int rows, int cols,
                                                                int64_t ld, uint8_t* codes, uint8_t* exps) {
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= rows) return;
  quant_row_mx(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a) + r * ld), cols, act,
               reinterpret_cast<uint4*>(codes + r * (cols >> 1)), exps + r * (cols >> 5));
}

__global__ void __launch_bounds__(kThreads) act_quant_g128_kernel(const void* a, int act, int rows, int cols,
                                                                  int64_t ld, int qmax, int8_t* codes,
                                                                  float* scales) {
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= rows) return;
  quant_row_groups(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a) + r * ld), cols, act, qmax,
                   reinterpret_cast<uint2*>(codes + r * cols), scales + r * (cols >> 7));
}

// row handled by this thread: W == 1 one per wavefront, W == 4 one per workgroup
template <int W> __device__ inline int64_t my_row() {
  return W == 1 ? (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6) : (int64_t)blockIdx.x;
}

template <int NC, int W, bool F6 = false>
__global__ void __launch_bounds__(kThreads) act_quant_vec_kernel(const void* a, int act, int rows, int cols,
                                                                 int64_t ld, int qmax, int8_t* codes,
                                                                 float* scales) {
  __shared__ uint32_t red[kThreads / 64];
  const int64_t r = my_row<W>();
  if (r >= rows) return;
  quant_row_vec<NC, W, F6>(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a) + r * ld), cols, act,
                           qmax, reinterpret_cast<uint2*>(codes + r * cols), scales + r, red);
}

// Rows of the sorted (token, slot) pairs whose expert's down projection takes
// a8/a4 activations; the expert of a row is found in an LDS copy of offsets.
template <int NC, int W>
__global__ void __launch_bounds__(kThreads) hquant_routed_kernel(const void* h, int act, int P, int F,
                                                                 const int32_t* __restrict__ offsets, int E,
                                                                 const int32_t* __restrict__ down_qmax,
                                                                 int8_t* hq, float* hs, float* hsg, uint8_t* hqmx,
                                                                 uint8_t* hsmx) {
  __shared__ int32_t s_off[kMaxE + 1];
  __shared__ uint32_t red[kThreads / 64];
  for (int i = threadIdx.x; i <= E; i += kThreads) s_off[i] = offsets[i];
  __syncthreads();
  const int r = (int)my_row<W>();
  if (r >= P || r >= s_off[E]) return;
  int lo = 0, hi = E;  // largest e with offsets[e] <= r
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_off[mid] <= r) lo = mid; else hi = mid;
  }
  const int qm = down_qmax[lo];
  if (qm == 0) return;
  if (qm & kDownQMX) {  // MXFP4 down projection: one wavefront per row
    if (W == 1 || threadIdx.x < 64)
      quant_row_mx(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(h) + (int64_t)r * F), F, act,
                   reinterpret_cast<uint4*>(hqmx + (int64_t)r * (F >> 1)), hsmx + (int64_t)r * (F >> 5));
    return;
  }
  if (qm & kDownQGroup) {  // per-128-group scales: one wavefront per row
    if (W == 1 || threadIdx.x < 64)
      quant_row_groups(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(h) + (int64_t)r * F), F, act,
                       qm & 0xFF, reinterpret_cast<uint2*>(hq + (int64_t)r * F), hsg + (int64_t)r * (F >> 7));
    return;
  }
  if (qm & kDownQF6) {  // int4 codes as FP6 e2m3 groups
    quant_row_vec<NC, W, true>(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(h) + (int64_t)r * F), F,
                               act, 7, reinterpret_cast<uint2*>(hq + (int64_t)r * F), hs + r, red);
    return;
  }
  const int qmax = (qm & kDownQF8) ? kQmaxF8 : qm;
  quant_row_vec<NC, W>(reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(h) + (int64_t)r * F), F,
                       act, qmax, reinterpret_cast<uint2*>(hq + (int64_t)r * F), hs + r, red);
}

// Row sums of each 128-wide block of bf16 rows, one wavefront per row: a
// block is 16 chunks of 8 elements, one per lane of a 16-lane group; each lane
// adds its 8 values in order, then the group adds its lanes pairwise.
__global__ void __launch_bounds__(kThreads) rowsum_kernel(const uint16_t* __restrict__ a, int rows, int cols,
                                                          int64_t ld, float* __restrict__ out) {
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= rows) return;
  rowsum_row(reinterpret_cast<const uint4*>(a + r * ld), cols, out + r * (cols >> 7));
}

// 8 outputs per thread.  SC > 0 slots (compile time): every slot row is
// loaded before the expert ids are consulted (rows of dropped pairs are in
// bounds, their values unused); SC == 0: any slot count, one slot at a time.
// F32: fp32 slot rows (two 16-byte loads per slot), else rows in the
// activation dtype (one 16-byte load per slot, widened exactly to fp32).
template <int SC, bool F32>
__global__ void __launch_bounds__(kThreads) combine_kernel(const void* __restrict__ slots,
                                                           const int32_t* __restrict__ ids, int T, int k, int E,
                                                           int S, int H, int act, uint16_t* __restrict__ y) {
  const int64_t i8 = (int64_t)blockIdx.x * kThreads + threadIdx.x;  // index of 8 outputs
  const int q8 = H / 8;
  if (i8 >= (int64_t)T * q8) return;
  const int t = (int)(i8 / q8), h = (int)(i8 % q8) * 8;
  if constexpr (SC > 0) S = SC;
  const int64_t off = (int64_t)t * S * H + h;  // element offset of slot 0
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  typedef float f8v[8];
  auto load = [&](int s, f8v& v) {
    if constexpr (F32) {
      const float4* p = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(slots) + off + (int64_t)s * H);
      const float4 a = p[0], b = p[1];
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
      v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
      const uint4 u = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(slots) + off + (int64_t)s * H);
      unpack8(u, act, v);
    }
  };
  auto valid = [&](int s) {
    if (s >= k) return true;  // shared-expert slots
    const int e = ids[(int64_t)t * k + s];
    return e >= 0 && e < E;
  };
  if constexpr (SC > 0) {
    float v[SC][8];
#pragma unroll
    for (int s = 0; s < SC; ++s) load(s, v[s]);
#pragma unroll
    for (int s = 0; s < SC; ++s)
      if (valid(s)) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] += v[s][i];
      }
  } else {
    for (int s = 0; s < S; ++s)
      if (valid(s)) {
        float v[8];
        load(s, v);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] += v[i];
      }
  }
  uint4 o;
  o.x = (uint32_t)f32_to_act(acc[0], act) | ((uint32_t)f32_to_act(acc[1], act) << 16);
  o.y = (uint32_t)f32_to_act(acc[2], act) | ((uint32_t)f32_to_act(acc[3], act) << 16);
  o.z = (uint32_t)f32_to_act(acc[4], act) | ((uint32_t)f32_to_act(acc[5], act) << 16);
  o.w = (uint32_t)f32_to_act(acc[6], act) | ((uint32_t)f32_to_act(acc[7], act) << 16);
  *reinterpret_cast<uint4*>(y + (int64_t)t * H + h) = o;
}

// Register-resident shapes by row length: (chunks per lane, wavefronts per row).
enum RowShape { RS_1x2, RS_1x4, RS_1x8, RS_4x4, RS_4x8, RS_4x16, RS_STREAM };
RowShape row_shape(int cols) {
  const int nch = cols / 8, per = (nch + 63) / 64, per4 = (nch + 255) / 256;
  if (per <= 2) return RS_1x2;
  if (per <= 4) return RS_1x4;
  if (per <= 8) return RS_1x8;
  if (per4 <= 4) return RS_4x4;
  if (per4 <= 8) return RS_4x8;
  if (per4 <= 16) return RS_4x16;  // rows up to 32768 elements stay in registers (read once)
  return RS_STREAM;
}
template <template <int, int> class K, typename... Args>
hipError_t launch_rows(int rows, int cols, hipStream_t s, Args... args) {
  const RowShape rs = row_shape(cols);
  const dim3 g1((rows + kRowsPerBlock - 1) / kRowsPerBlock), g4(rows), b(kThreads);
  switch (rs) {
    case RS_1x2: hipLaunchKernelGGL((K<2, 1>::fn), g1, b, 0, s, args...); break;
    case RS_1x4: hipLaunchKernelGGL((K<4, 1>::fn), g1, b, 0, s, args...); break;
    case RS_1x8: hipLaunchKernelGGL((K<8, 1>::fn), g1, b, 0, s, args...); break;
    case RS_4x4: hipLaunchKernelGGL((K<4, 4>::fn), g4, b, 0, s, args...); break;
    case RS_4x8: hipLaunchKernelGGL((K<8, 4>::fn), g4, b, 0, s, args...); break;
    case RS_4x16: hipLaunchKernelGGL((K<16, 4>::fn), g4, b, 0, s, args...); break;
    default: hipLaunchKernelGGL((K<0, 1>::fn), g1, b, 0, s, args...); break;
  }
  return hipGetLastError();
}
template <int NC, int W> struct ActQuantK { static constexpr auto fn = act_quant_vec_kernel<NC, W>; };
template <int NC, int W> struct ActQuantF6K { static constexpr auto fn = act_quant_vec_kernel<NC, W, true>; };
template <int NC, int W> struct HQuantK { static constexpr auto fn = hquant_routed_kernel<NC, W>; };
}  // namespace

hipError_t launch_rowsum(const void* a, int rows, int cols, int64_t ld, float* out, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(a) & 15) || cols % 128 || ld % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rowsum_kernel, dim3((rows + kRowsPerBlock - 1) / kRowsPerBlock), dim3(kThreads), 0, s,
                     reinterpret_cast<const uint16_t*>(a), rows, cols, ld, out);
  return hipGetLastError();
}

hipError_t launch_act_quant(const void* a, int act, int rows, int cols, int64_t ld, int qmax, int8_t* codes,
                            float* scales, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const bool vec = (reinterpret_cast<uintptr_t>(a) & 15) == 0 && (reinterpret_cast<uintptr_t>(codes) & 7) == 0 &&
                   cols % 8 == 0 && ld % 8 == 0;
  if (!vec) {  // unaligned rows: one workgroup per row, element loads
    hipLaunchKernelGGL(act_quant_kernel, dim3(rows), dim3(kThreads), 0, s, a, act, cols, ld, qmax, codes, scales);
    return hipGetLastError();
  }
  return launch_rows<ActQuantK>(rows, cols, s, a, act, rows, cols, ld, qmax, codes, scales);
}

hipError_t launch_act_quant_f6(const void* a, int act, int rows, int cols, int64_t ld, uint8_t* codes, float* scales,
                               hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(a) & 15) || (reinterpret_cast<uintptr_t>(codes) & 31) || cols % 128 || ld % 8)
    return hipErrorInvalidValue;
  return launch_rows<ActQuantF6K>(rows, cols, s, a, act, rows, cols, ld, 7, reinterpret_cast<int8_t*>(codes), scales);
}

hipError_t launch_act_quant_g128(const void* a, int act, int rows, int cols, int64_t ld, int qmax, int8_t* codes,
                                 float* scales, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(a) & 15) || (reinterpret_cast<uintptr_t>(codes) & 7) || cols % 128 || ld % 8)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(act_quant_g128_kernel, dim3((rows + kRowsPerBlock - 1) / kRowsPerBlock), dim3(kThreads), 0, s, a,
                     act, rows, cols, ld, qmax, codes, scales);
  return hipGetLastError();
}

hipError_t launch_act_quant_mx(const void* a, int act, int rows, int cols, int64_t ld, uint8_t* codes, uint8_t* exps,
                               hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(a) & 15) || (reinterpret_cast<uintptr_t>(codes) & 15) || cols % 128 || ld % 8)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(act_quant_mx_kernel, dim3((rows + kRowsPerBlock - 1) / kRowsPerBlock), dim3(kThreads), 0, s, a,
                     act, rows, cols, ld, codes, exps);
  return hipGetLastError();
}

hipError_t launch_hquant_routed(const void* h, int act, int P, int F, const int32_t* offsets, int E,
                                const int32_t* down_qmax, int8_t* hq, float* hs, float* hsg, uint8_t* hqmx,
                                uint8_t* hsmx, hipStream_t s) {
  if (P <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(h) & 15) || (reinterpret_cast<uintptr_t>(hq) & 7) || F % 8 || E > kMaxE)
    return hipErrorInvalidValue;
  if (F % 128) return hipErrorInvalidValue;
  return launch_rows<HQuantK>(P, F, s, h, act, P, F, offsets, E, down_qmax, hq, hs, hsg, hqmx, hsmx);
}

hipError_t launch_combine(const void* slots, int slot16, const int32_t* ids, int T, int k, int E, int nsh, int H,
                          int act, void* y, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (H % 8 || (reinterpret_cast<uintptr_t>(y) & 15) || (reinterpret_cast<uintptr_t>(slots) & 15))
    return hipErrorInvalidValue;
  const int64_t n8 = (int64_t)T * (H / 8);
  const dim3 grid((unsigned)((n8 + kThreads - 1) / kThreads));
  const int S = k + nsh;
  auto run = [&](auto f32) {
    constexpr bool F = decltype(f32)::value;
    switch (S) {
#define MX_COMBINE(S_) \
  case S_:             \
    hipLaunchKernelGGL((combine_kernel<S_, F>), grid, dim3(kThreads), 0, s, slots, ids, T, k, E, S, H, act, (uint16_t*)y); \
    break;
      MX_COMBINE(1) MX_COMBINE(2) MX_COMBINE(3) MX_COMBINE(4) MX_COMBINE(5) MX_COMBINE(6) MX_COMBINE(7) MX_COMBINE(8)
      MX_COMBINE(9) MX_COMBINE(10)
#undef MX_COMBINE
      default:
        hipLaunchKernelGGL((combine_kernel<0, F>), grid, dim3(kThreads), 0, s, slots, ids, T, k, E, S, H, act,
                           (uint16_t*)y);
    }
  };
  if (slot16) run(std::false_type{});
  else run(std::true_type{});
  return hipGetLastError();
}

}  // namespace mxmoe
