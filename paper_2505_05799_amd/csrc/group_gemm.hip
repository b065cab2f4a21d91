// Mixed-precision Group-GEMM of the MoE block (Sec. 4.3 of the paper:
// micro-kernel specialization, equal-resource tile configurations, and a
// greedy longest-tile-first schedule).
//
//   plan_kernel        one workgroup: per (phase, expert) group picks a tile
//                      configuration from the group's row count, counts its
//                      tiles, estimates a per-tile cost, and orders the groups
//                      by decreasing tile cost (ties: lower expert first).  The
//                      tile queue of a phase is the concatenation of the
//                      groups' tiles in that order: workgroups that free up
//                      take the next tile, i.e. list scheduling with the
//                      longest tiles first (the greedy rule of Sec. 4.3).
//   group_gemm_kernel  persistent: every workgroup pops tile indices from an
//                      atomic head counter and dispatches, outside the MAC loop,
//                      to the micro-kernel of the tile's (scheme, config).
//
// Phase 0 computes gate and up of an expert in the same tile (they share the
// activation rows) and applies the SiLU gate in registers: h = SiLU(g) * u,
// rounded once to the activation dtype.  Phase 1 computes the down projection,
// multiplies each row by its router gate weight and stores fp32 rows in the
// per-(token, slot) buffer that the combine sums in a fixed order.
//
// MFMA operand roles: the weight fragment is the "A" operand (16 output
// channels x 32/64 reduction) and the activation fragment the "B" operand
// (16 rows), so a lane's four accumulators are four consecutive output
// channels of one row - contiguous stores and one row scale per lane.
//
// Numerics per scheme:
//   w16   : 16-bit MFMA, fp32 accumulation.
//   wNg128: (q - z) is formed exactly as a 16-bit value (|q - z| <= 255), each
//           128-wide group is accumulated by MFMA in fp32 and scaled by its fp16
//           scale in fp32 before joining the running sum: the dequantized
//           weight s*(q - z) is used exactly.
//   w8a8  : int8 MFMA, exact int32 sums, then fp32 (acc * s_a) * s_w.
//   w4a4  : nibbles widened to int8 as 16*q, int8 MFMA, exact sum / 16.
#include "mxmoe_internal.h"

namespace mxmoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));

constexpr int kThreads = 256;
constexpr int kPhaseRaw = 2;

// ------------------------------------------------------------ tile configs
template <int CFG> struct CfgT;
template <> struct CfgT<CFG_S> { static constexpr int WM = 1, WN = 4, MB = 1; };
template <> struct CfgT<CFG_M> { static constexpr int WM = 2, WN = 2, MB = 2; };
template <> struct CfgT<CFG_L> { static constexpr int WM = 2, WN = 2, MB = 4; };

__host__ __device__ inline int cfg_wm(int c) { return c == CFG_S ? 1 : 2; }
__host__ __device__ inline int cfg_wn(int c) { return c == CFG_S ? 4 : 2; }
__host__ __device__ inline int cfg_mb(int c) { return c == CFG_S ? 1 : (c == CFG_M ? 2 : 4); }
// fragments (of 16 output channels) per wavefront and linear: 2 for the fused
// gate|up phase, 4 for the single-linear phases
__host__ __device__ inline int cfg_nb(int phase) { return phase == 0 ? 2 : 4; }
__host__ __device__ inline int cfg_bm(int c) { return 16 * cfg_mb(c) * cfg_wm(c); }
__host__ __device__ inline int cfg_bn(int c, int phase) { return 16 * cfg_nb(phase) * cfg_wn(c); }
__host__ __device__ inline int pick_cfg(int m) { return m <= 16 ? CFG_S : (m <= 64 ? CFG_M : CFG_L); }

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
      const int phase_eff = raw_m >= 0 ? 1 : ph;  // raw mode: one linear, wide tiles
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
      const double t_mem = (wbytes + abytes) * 32.0;                        // ps
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

// -------------------------------------------------------- helpers
__device__ inline uint32_t pack_bf16_exact(float lo, float hi) {
  // lo, hi are small integers: truncation to bf16 is exact
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}
__device__ inline uint32_t pack_f16_exact(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
}
template <int ACT> __device__ inline uint32_t pack2(float lo, float hi) {
  return ACT == MXMOE_BF16 ? pack_bf16_exact(lo, hi) : pack_f16_exact(lo, hi);
}

// 8 integer codes (slot order) minus the zero point -> one 16-bit MFMA operand
template <int ACT> __device__ inline u32x4 deq8(const uint32_t v[8], float z) {
  u32x4 r;
  r[0] = pack2<ACT>((float)v[0] - z, (float)v[1] - z);
  r[1] = pack2<ACT>((float)v[2] - z, (float)v[3] - z);
  r[2] = pack2<ACT>((float)v[4] - z, (float)v[5] - z);
  r[3] = pack2<ACT>((float)v[6] - z, (float)v[7] - z);
  return r;
}

// raw lane bytes of one fragment block
template <int KD> struct Raw;
template <> struct Raw<K_W16> { u32x4 d[4]; };
template <> struct Raw<K_W8G> { u32x4 d[2]; };
template <> struct Raw<K_W4G> { u32x4 d; };
template <> struct Raw<K_W3G> { u32x3 d; };
template <> struct Raw<K_W2G> { u32x2 d; };
template <> struct Raw<K_W8A8> { u32x4 d[2]; };
template <> struct Raw<K_W4A4> { u32x4 d; };

template <int KD> __device__ inline void load_raw(Raw<KD>& r, const uint8_t* p);
template <> __device__ inline void load_raw<K_W16>(Raw<K_W16>& r, const uint8_t* p) {
  const u32x4* q = reinterpret_cast<const u32x4*>(p);
  r.d[0] = q[0]; r.d[1] = q[1]; r.d[2] = q[2]; r.d[3] = q[3];
}
template <> __device__ inline void load_raw<K_W8G>(Raw<K_W8G>& r, const uint8_t* p) {
  const u32x4* q = reinterpret_cast<const u32x4*>(p);
  r.d[0] = q[0]; r.d[1] = q[1];
}
template <> __device__ inline void load_raw<K_W8A8>(Raw<K_W8A8>& r, const uint8_t* p) {
  const u32x4* q = reinterpret_cast<const u32x4*>(p);
  r.d[0] = q[0]; r.d[1] = q[1];
}
template <> __device__ inline void load_raw<K_W4G>(Raw<K_W4G>& r, const uint8_t* p) {
  r.d = *reinterpret_cast<const u32x4*>(p);
}
template <> __device__ inline void load_raw<K_W4A4>(Raw<K_W4A4>& r, const uint8_t* p) {
  r.d = *reinterpret_cast<const u32x4*>(p);
}
template <> __device__ inline void load_raw<K_W3G>(Raw<K_W3G>& r, const uint8_t* p) {
  const uint32_t* q = reinterpret_cast<const uint32_t*>(p);  // 4-byte aligned (12-byte lanes)
  r.d[0] = q[0]; r.d[1] = q[1]; r.d[2] = q[2];
}
template <> __device__ inline void load_raw<K_W2G>(Raw<K_W2G>& r, const uint8_t* p) {
  r.d = *reinterpret_cast<const u32x2*>(p);
}

// weight operand of MFMA step j (16-bit kinds): 8 values as u32x4
template <int KD, int ACT> __device__ inline u32x4 wfrag16(const Raw<KD>& r, int j, float z);
template <> __device__ inline u32x4 wfrag16<K_W16, MXMOE_BF16>(const Raw<K_W16>& r, int j, float) { return r.d[j]; }
template <> __device__ inline u32x4 wfrag16<K_W16, MXMOE_F16>(const Raw<K_W16>& r, int j, float) { return r.d[j]; }

template <int KD, int ACT> __device__ inline u32x4 wfrag16(const Raw<KD>& r, int j, float z) {
  uint32_t v[8];
  if constexpr (KD == K_W8G) {
    const uint32_t a = r.d[j >> 1][(j & 1) * 2], b = r.d[j >> 1][(j & 1) * 2 + 1];
#pragma unroll
    for (int i = 0; i < 4; ++i) { v[i] = (a >> (8 * i)) & 0xFFu; v[4 + i] = (b >> (8 * i)) & 0xFFu; }
  } else if constexpr (KD == K_W4G) {
    const uint32_t d = r.d[j];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (d >> (4 * i)) & 0xFu;
  } else if constexpr (KD == K_W2G) {
    const uint32_t d = r.d[j >> 1] >> (16 * (j & 1));
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (d >> (2 * i)) & 0x3u;
  } else {  // K_W3G
    const uint32_t d = r.d[j >> 1] >> (16 * (j & 1));
    const uint32_t h = r.d[2] >> (8 * j);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = ((d >> (2 * i)) & 0x3u) | (((h >> i) & 1u) << 2);
  }
  return deq8<ACT>(v, z);
}

// weight operand of int8 MFMA step j (int kinds)
template <int KD> __device__ inline i32x4 wfrag8(const Raw<KD>& r, int j);
template <> __device__ inline i32x4 wfrag8<K_W8A8>(const Raw<K_W8A8>& r, int j) {
  return __builtin_bit_cast(i32x4, r.d[j]);
}
template <> __device__ inline i32x4 wfrag8<K_W4A4>(const Raw<K_W4A4>& r, int j) {
  const uint32_t d0 = r.d[2 * j], d1 = r.d[2 * j + 1];
  i32x4 o;
  o[0] = (int)((d0 << 4) & 0xF0F0F0F0u);
  o[1] = (int)(d0 & 0xF0F0F0F0u);
  o[2] = (int)((d1 << 4) & 0xF0F0F0F0u);
  o[3] = (int)(d1 & 0xF0F0F0F0u);
  return o;
}

template <int ACT> __device__ inline f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (ACT == MXMOE_BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b),
                                                  c, 0, 0, 0);
}

__device__ inline float act_to_f32(uint16_t b, int act) {
  if (act == MXMOE_BF16) return __uint_as_float(((uint32_t)b) << 16);
  return (float)__builtin_bit_cast(_Float16, b);
}
template <int ACT> __device__ inline uint16_t f32_to_act(float f) {
  if constexpr (ACT == MXMOE_BF16) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
  } else {
    return __builtin_bit_cast(uint16_t, (_Float16)f);
  }
}

__device__ inline float silu_f32(float g) { return g / (1.0f + expf(-g)); }

// ---------------------------------------------------------- tile body
// One tile of one (expert, phase) group.  Wavefronts work independently (no
// LDS, no barriers): wave (wm, wn) owns rows [row0, row0 + 16*MB) and output
// channels [16*nb0, 16*(nb0 + NB)) of every linear of the phase.
template <int KD, int ACT, int CFG, int PHASE>
__device__ inline void run_tile(const GemmArgs& a, const DevExpert* ex, int g, int m_g, int mt, int nt) {
  using C = CfgT<CFG>;
  constexpr int MB = C::MB;
  constexpr int WN = C::WN;
  constexpr int NB = PHASE == 0 ? 2 : 4;
  constexpr int NL = PHASE == 0 ? 2 : 1;
  constexpr bool INT = kind_is_int(KD);
  constexpr bool WONLY = kind_is_wonly(KD);
  constexpr int J = INT ? 2 : 4;  // MFMA steps per 128-wide k block
  constexpr int BM = 16 * MB * C::WM;
  constexpr int BN = 16 * NB * WN;
  constexpr int LB = lane_bytes(KD);
  constexpr int BB = block_bytes(KD);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave / WN, wn = wave % WN;
  const int row0 = mt * BM + wm * MB * 16;
  if (row0 >= m_g) return;
  const int li = lane & 15, qd = lane >> 4;

  const bool shared = g >= a.E_routed;
  const DevLinear* lins[NL];
  if constexpr (PHASE == 0) { lins[0] = &ex->lin[0]; lins[1] = &ex->lin[1]; }
  else if constexpr (PHASE == 1) { lins[0] = &ex->lin[2]; }
  else { lins[0] = &a.raw_lin; }
  const int N = lins[0]->n, K = lins[0]->k;
  const int kblocks = K / 128;
  const int nb0 = (nt * BN + wn * NB * 16) / 16;
  int nvalid = N / 16 - nb0;
  if (nvalid <= 0) return;
  if (nvalid > NB) nvalid = NB;

  // ---- activation rows of this lane (one per row fragment)
  const int off_e = (!shared && PHASE != kPhaseRaw) ? a.offsets[g] : 0;
  const uint8_t* arow[MB];
  float a_scale[MB];
  int rows[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    int m = row0 + mb * 16 + li;
    rows[mb] = m;
    if (m >= m_g) m = m_g - 1;
    int64_t src;  // activation row index
    if constexpr (PHASE == 0) {
      src = shared ? m : a.sorted_pair[off_e + m] / a.k;
    } else if constexpr (PHASE == 1) {
      src = shared ? (int64_t)(g - a.E_routed) * a.T + m : off_e + m;
    } else {
      src = m;
    }
    a_scale[mb] = 1.f;
    if constexpr (INT) {
      const int8_t* q;
      const float* s;
      if constexpr (PHASE == 1) {
        q = shared ? a.hq_shared : a.hq;
        s = shared ? a.hs_shared : a.hs;
      } else {
        q = KD == K_W8A8 ? a.xq8 : a.xq4;
        s = KD == K_W8A8 ? a.xs8 : a.xs4;
      }
      arow[mb] = reinterpret_cast<const uint8_t*>(q) + src * K;
      a_scale[mb] = s[src];
    } else {
      const void* base = PHASE == 0 ? a.x : (PHASE == 1 ? (shared ? a.h_shared : a.h) : a.x);
      arow[mb] = reinterpret_cast<const uint8_t*>(base) + src * K * 2;
    }
  }

  // ---- accumulators
  typedef typename std::conditional<INT, i32x4, f32x4>::type AccT;
  AccT acc[NL][NB][MB];
#pragma unroll
  for (int l = 0; l < NL; ++l)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[l][nb][mb] = AccT{0, 0, 0, 0};

  const uint8_t* wbase[NL];
#pragma unroll
  for (int l = 0; l < NL; ++l) wbase[l] = lins[l]->packed + (int64_t)nb0 * kblocks * BB + lane * LB;

  for (int kb = 0; kb < kblocks; ++kb) {
    Raw<KD> raw[NL][NB];
    float zf[NL][NB];
    f32x4 sc[NL][NB];
#pragma unroll
    for (int l = 0; l < NL; ++l)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        if (nb < nvalid) {
          const uint8_t* blk = wbase[l] + ((int64_t)nb * kblocks + kb) * BB;
          load_raw<KD>(raw[l][nb], blk);
          if constexpr (WONLY) {
            const uint8_t* meta = blk - lane * LB + 64 * LB;
            const uint32_t zz = reinterpret_cast<const uint32_t*>(meta)[li];
            zf[l][nb] = (float)__builtin_bit_cast(_Float16, (uint16_t)(zz >> 16));
            const u32x4 ss = reinterpret_cast<const u32x4*>(meta)[qd];
#pragma unroll
            for (int r = 0; r < 4; ++r) sc[l][nb][r] = (float)__builtin_bit_cast(_Float16, (uint16_t)(ss[r] & 0xFFFF));
          }
        }
      }
    if constexpr (INT) {
#pragma unroll
      for (int j = 0; j < J; ++j) {
        i32x4 af[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          af[mb] = *reinterpret_cast<const i32x4*>(arow[mb] + kb * 128 + 64 * j + 16 * qd);
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            if (nb < nvalid) {
              const i32x4 wf = wfrag8<KD>(raw[l][nb], j);
#pragma unroll
              for (int mb = 0; mb < MB; ++mb)
                acc[l][nb][mb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wf, af[mb], acc[l][nb][mb], 0, 0, 0);
            }
          }
      }
    } else {
      f32x4 part[NL][NB][MB];
#pragma unroll
      for (int j = 0; j < J; ++j) {
        u32x4 af[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          af[mb] = *reinterpret_cast<const u32x4*>(arow[mb] + 2 * (kb * 128 + 32 * j + 8 * qd));
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            if (nb < nvalid) {
              const u32x4 wf = wfrag16<KD, ACT>(raw[l][nb], j, WONLY ? zf[l][nb] : 0.f);
#pragma unroll
              for (int mb = 0; mb < MB; ++mb) {
                if constexpr (WONLY)
                  part[l][nb][mb] = mfma16<ACT>(wf, af[mb], j == 0 ? f32x4{0, 0, 0, 0} : part[l][nb][mb]);
                else
                  acc[l][nb][mb] = mfma16<ACT>(wf, af[mb], acc[l][nb][mb]);
              }
            }
          }
      }
      if constexpr (WONLY) {
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            if (nb < nvalid)
#pragma unroll
              for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  acc[l][nb][mb][r] = __builtin_fmaf(sc[l][nb][r], part[l][nb][mb][r], acc[l][nb][mb][r]);
      }
    }
  }

  // ---- epilogue: lane holds channels n = 16*(nb0+nb) + 4*qd + r of row rows[mb]
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (nb >= nvalid) continue;
    const int n0 = 16 * (nb0 + nb) + 4 * qd;
    f32x4 wsc[NL];
#pragma unroll
    for (int l = 0; l < NL; ++l) {
      if constexpr (INT) wsc[l] = *reinterpret_cast<const f32x4*>(lins[l]->wscale + n0);
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = rows[mb];
      if (m >= m_g) continue;
      f32x4 v[NL];
#pragma unroll
      for (int l = 0; l < NL; ++l) {
        if constexpr (INT) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            int iv = acc[l][nb][mb][r];
            if constexpr (KD == K_W4A4) iv >>= 4;  // exact: every product is a multiple of 16
            v[l][r] = ((float)iv * a_scale[mb]) * wsc[l][r];
          }
        } else {
          v[l] = acc[l][nb][mb];
        }
      }
      if constexpr (PHASE == 0) {
        const int F = N;
        uint8_t* hb = reinterpret_cast<uint8_t*>(shared ? a.h_shared : a.h);
        const int64_t hrow = shared ? (int64_t)(g - a.E_routed) * a.T + m : (int64_t)off_e + m;
        uint32_t o[2];
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          const float h0 = silu_f32(v[0][r]) * v[1][r];
          const float h1 = silu_f32(v[0][r + 1]) * v[1][r + 1];
          o[r / 2] = (uint32_t)f32_to_act<ACT>(h0) | ((uint32_t)f32_to_act<ACT>(h1) << 16);
        }
        *reinterpret_cast<u32x2*>(hb + (hrow * F + n0) * 2) = u32x2{o[0], o[1]};
      } else if constexpr (PHASE == 1) {
        int64_t srow;
        float gw;
        if (shared) {
          srow = (int64_t)m * (a.k + a.n_shared) + a.k + (g - a.E_routed);
          gw = 1.f;
        } else {
          const int p = a.sorted_pair[off_e + m];
          srow = (int64_t)(p / a.k) * (a.k + a.n_shared) + (p % a.k);
          gw = a.topk_w[p];
        }
        f32x4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = v[0][r] * gw;
        *reinterpret_cast<f32x4*>(a.slots + srow * N + n0) = o;
      } else {
        if constexpr (INT) {
          *reinterpret_cast<i32x4*>(reinterpret_cast<int32_t*>(a.raw_out) + (int64_t)m * N + n0) =
              KD == K_W4A4 ? (acc[0][nb][mb] >> 4) : acc[0][nb][mb];
        } else {
          *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.raw_out) + (int64_t)m * N + n0) = v[0];
        }
      }
    }
  }
}

template <int ACT, int PHASE, int CFG>
__device__ inline void dispatch_kind(const GemmArgs& a, const DevExpert* ex, int g, int m_g, int mt, int nt, int kd) {
  switch (kd) {
    case K_W16: run_tile<K_W16, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    case K_W8A8: run_tile<K_W8A8, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    case K_W4A4: run_tile<K_W4A4, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    case K_W2G: run_tile<K_W2G, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    case K_W3G: run_tile<K_W3G, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    case K_W4G: run_tile<K_W4G, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    case K_W8G: run_tile<K_W8G, ACT, CFG, PHASE>(a, ex, g, m_g, mt, nt); break;
    default: break;
  }
}

template <int ACT, int PHASE>
__global__ void __launch_bounds__(kThreads) group_gemm_kernel(GemmArgs a) {
  __shared__ int s_tile;
  const int G = a.G;
  const int pidx = PHASE == kPhaseRaw ? 0 : PHASE;
  const int32_t* rec = a.plan + (int64_t)pidx * G * PF_N;
  const int32_t* order = a.plan + 2LL * G * PF_N + (int64_t)pidx * G;
  int32_t* ctr = a.plan + 2LL * G * PF_N + 2LL * G;
  const int total = ctr[PC_TOTAL0 + pidx];
  const int ng = ctr[4 + pidx];
  for (;;) {
    if (threadIdx.x == 0) s_tile = atomicAdd(&ctr[PC_HEAD0 + pidx], 1);
    __syncthreads();
    const int tile = s_tile;
    __syncthreads();
    if (tile >= total) break;
    int lo = 0, hi = ng;  // largest rank whose first tile <= tile
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (rec[(int64_t)order[mid] * PF_N + PF_START] <= tile) lo = mid; else hi = mid;
    }
    const int g = order[lo];
    const int32_t* r = rec + (int64_t)g * PF_N;
    const int local = tile - r[PF_START];
    const int mtiles = r[PF_MTILES];
    const int mt = local % mtiles, nt = local / mtiles;
    const DevExpert* ex = PHASE == kPhaseRaw ? nullptr : a.experts + g;
    const int kd = PHASE == kPhaseRaw ? a.raw_lin.kind : ex->lin[PHASE == 0 ? 0 : 2].kind;
    const int m_g = r[PF_M];
    switch (r[PF_CFG]) {
      case CFG_S: dispatch_kind<ACT, PHASE, CFG_S>(a, ex, g, m_g, mt, nt, kd); break;
      case CFG_M: dispatch_kind<ACT, PHASE, CFG_M>(a, ex, g, m_g, mt, nt, kd); break;
      default: dispatch_kind<ACT, PHASE, CFG_L>(a, ex, g, m_g, mt, nt, kd); break;
    }
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
  if (a.act == MXMOE_BF16) {
    if (phase == 0) hipLaunchKernelGGL((group_gemm_kernel<MXMOE_BF16, 0>), dim3(grid), dim3(kThreads), 0, s, a);
    else if (phase == 1) hipLaunchKernelGGL((group_gemm_kernel<MXMOE_BF16, 1>), dim3(grid), dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL((group_gemm_kernel<MXMOE_BF16, kPhaseRaw>), dim3(grid), dim3(kThreads), 0, s, a);
  } else {
    if (phase == 0) hipLaunchKernelGGL((group_gemm_kernel<MXMOE_F16, 0>), dim3(grid), dim3(kThreads), 0, s, a);
    else if (phase == 1) hipLaunchKernelGGL((group_gemm_kernel<MXMOE_F16, 1>), dim3(grid), dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL((group_gemm_kernel<MXMOE_F16, kPhaseRaw>), dim3(grid), dim3(kThreads), 0, s, a);
  }
  return hipGetLastError();
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
