// Tile plan of the mixed-precision Group-GEMM and the launch dispatch (the
// micro-kernels themselves are in group_gemm_impl.h, one translation unit per
// activation dtype and phase).
#include "group_gemm_impl.h"

namespace mxmoe {
namespace {

// ---------------------------------------------------------------- plan
struct MaskBits { uint32_t w[64]; };

__global__ void __launch_bounds__(1024) plan_kernel(const DevExpert* __restrict__ experts, int E, int G, int T,
                                                    const int32_t* __restrict__ counts, int raw_m,
                                                    DevLinear raw_lin, MaskBits mask, int32_t* __restrict__ plan,
                                                    int32_t* __restrict__ down_qmax) {
  __shared__ int32_t s_cost[2][2048];
  __shared__ int32_t s_tiles[2][2048];
  const int tid = threadIdx.x;
  const int nphase = raw_m >= 0 ? 1 : 2;
  for (int ph = 0; ph < nphase; ++ph) {
    for (int g = tid; g < G; g += blockDim.x) {
      int m = raw_m >= 0 ? raw_m : (g < E ? counts[g] : T);
      if (!((mask.w[g >> 5] >> (g & 31)) & 1u)) m = 0;
      const DevLinear& L = raw_m >= 0 ? raw_lin : experts[g].lin[ph == 0 ? 0 : 2];
      const int cfg = pick_cfg(m);
      const int phase_eff = raw_m >= 0 ? 1 : ph;  // raw mode: one linear
      const int bm = cfg_bm(cfg), bn = cfg_bn(cfg, phase_eff);
      const int mt = m > 0 ? (m + bm - 1) / bm : 0;
      const int nt = (L.n + bn - 1) / bn;
      const int tiles = mt * nt;
      const int nl = (raw_m < 0 && ph == 0) ? 2 : 1;
      const int kd = L.kind;
      const double wbytes = (double)nl * bn * L.k * kind_wbits(kd) / 8.0;
      const double abytes = (double)bm * L.k * (kind_is_int(kd) ? 1.0 : 2.0);
      const double flops = 2.0 * nl * bm * bn * L.k;
      // per-CU shares of MI355X peaks: 8 TB/s HBM, 2.5 PF 16-bit / 5 POPS int8 MFMA
      const double t_mem = (wbytes + abytes) * 32.0;  // ps
      const double t_mma = flops * 1000.0 / (kind_is_int(kd) ? 19531.0 : 9766.0);
      double c = t_mem > t_mma ? t_mem : t_mma;
      if (c > 2.0e9) c = 2.0e9;
      int32_t* r = plan + ((int64_t)ph * G + g) * PF_N;
      r[PF_EXPERT] = g;
      r[PF_M] = m;
      r[PF_CFG] = cfg;
      r[PF_MTILES] = mt;
      r[PF_NTILES] = nt;
      r[PF_COST] = tiles ? (int32_t)c : 0;
      s_cost[ph][g] = tiles ? (int32_t)c : 0;
      s_tiles[ph][g] = tiles;
      if (ph == 0 && raw_m < 0) down_qmax[g] = kind_qmax(experts[g].lin[2].kind);
    }
  }
  __syncthreads();
  int32_t* order = plan + 2LL * G * PF_N;
  for (int ph = 0; ph < nphase; ++ph) {
    for (int g = tid; g < G; g += blockDim.x) {
      int rank = -1;
      if (s_tiles[ph][g] > 0) {
        rank = 0;
        const int cg = s_cost[ph][g];
        for (int h = 0; h < G; ++h) {
          if (s_tiles[ph][h] <= 0) continue;
          const int ch = s_cost[ph][h];
          rank += (ch > cg) || (ch == cg && h < g);
        }
        order[(int64_t)ph * G + rank] = g;
      }
      plan[((int64_t)ph * G + g) * PF_N + PF_RANK] = rank;
    }
  }
  __syncthreads();
  if (tid < nphase) {
    const int ph = tid;
    int run = 0, ng = 0;
    for (int g = 0; g < G; ++g) ng += s_tiles[ph][g] > 0;
    for (int r = 0; r < ng; ++r) {
      const int g = order[(int64_t)ph * G + r];
      plan[((int64_t)ph * G + g) * PF_N + PF_START] = run;
      run += s_tiles[ph][g];
    }
    for (int r = ng; r < G; ++r) order[(int64_t)ph * G + r] = -1;
    int32_t* ctr = plan + 2LL * G * PF_N + 2LL * G;
    ctr[PC_HEAD0 + ph] = 0;
    ctr[PC_TOTAL0 + ph] = run;
    ctr[4 + ph] = ng;
  }
  if (nphase == 1 && tid == 1) {
    int32_t* ctr = plan + 2LL * G * PF_N + 2LL * G;
    ctr[PC_HEAD1] = 0;
    ctr[PC_TOTAL1] = 0;
    ctr[5] = 0;
  }
}

}  // namespace

hipError_t launch_plan(const DevExpert* experts, int E, int G, int T, const int32_t* counts, int raw_m,
                       const DevLinear& raw_lin, const uint32_t* mask_words, int32_t* plan, int32_t* down_qmax,
                       hipStream_t s) {
  MaskBits mb;
  for (int i = 0; i < 64; ++i) mb.w[i] = mask_words ? mask_words[i] : 0xffffffffu;
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, experts, E, G, T, counts, raw_m, raw_lin, mb, plan,
                     down_qmax);
  return hipGetLastError();
}

hipError_t launch_group_gemm(const GemmArgs& a, int phase, int grid, hipStream_t s) {
  if (a.act == MXMOE_BF16) return phase == 0 ? gg_bf16_p0(a, grid, s) : (phase == 1 ? gg_bf16_p1(a, grid, s) : gg_bf16_raw(a, grid, s));
  return phase == 0 ? gg_f16_p0(a, grid, s) : (phase == 1 ? gg_f16_p1(a, grid, s) : gg_f16_raw(a, grid, s));
}

int group_gemm_grid(int device) {
  static int cached[64] = {0};
  if (device < 0 || device >= 64) device = 0;
  if (!cached[device]) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || cus <= 0) cus = 256;
    cached[device] = cus * 2;
  }
  return cached[device];
}

}  // namespace mxmoe
