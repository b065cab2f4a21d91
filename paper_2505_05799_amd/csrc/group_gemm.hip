// Tile plan of the mixed-precision Group-GEMM and the launch dispatch (the
// micro-kernels themselves are in group_gemm_impl.h, one translation unit per
// activation dtype and phase).
//
// plan_kernel (one workgroup, no host round trip):
//   1. per (phase, expert) group: rows m (routing counts, T for shared experts),
//      tile configuration from m, tile counts, a static per-tile cost;
//   2. rank the groups by decreasing tile cost (ties: lower expert first) - the
//      greedy longest-tile-first order of the paper's tile schedule;
//   3. cut every group into super-tiles (up to 64 tiles that share row and
//      channel blocks) and deal them round-robin, in rank order, to one queue
//      per XCD; per-queue prefix sums give each entry's first tile;
//   4. expand every queue into one 16-byte entry per tile (group, configuration,
//      kind, slices, tile coordinates, first sorted row and rows of the group),
//      so that a workgroup resolves a popped tile with a single load.
// Groups may be sliced along the reduction (split-K, see split_rule): their
// slices are queued as extra channel tiles, within fixed budgets of added
// tiles and of partial-sum storage.
#include "group_gemm_impl.h"

namespace mxmoe {
namespace {

struct MaskBits { uint32_t w[64]; };

// In-place exclusive scan of n ints v[0], v[stride], ... by one workgroup
// (chunk sums per thread, wavefront prefix sums, then wavefront totals);
// returns the sum.  red: LDS scratch of blockDim/64 + 1 ints.
__device__ int block_scan(int32_t* v, int n, int32_t* red, int stride = 1) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, w = tid >> 6, nw = nt >> 6;
  const int per = (n + nt - 1) / nt;
  const int lo = tid * per, hi = min(n, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += v[(int64_t)i * stride];
  int incl = s;
  for (int d = 1; d < 64; d <<= 1) {
    const int t = __shfl_up(incl, d, 64);
    if (lane >= d) incl += t;
  }
  if (lane == 63) red[w] = incl;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int i = 0; i < nw; ++i) {
      const int t = red[i];
      red[i] = run;
      run += t;
    }
    red[nw] = run;
  }
  __syncthreads();
  int run = red[w] + incl - s;
  for (int i = lo; i < hi; ++i) {
    const int t = v[(int64_t)i * stride];
    v[(int64_t)i * stride] = run;
    run += t;
  }
  const int total = red[nw];
  __syncthreads();
  return total;
}

__global__ void __launch_bounds__(1024) plan_kernel(const DevExpert* __restrict__ experts, int E, int G, int T,
                                                    const int32_t* __restrict__ counts,
                                                    const int32_t* __restrict__ offsets, int raw_m,
                                                    DevLinear raw_lin, MaskBits mask, int32_t* __restrict__ plan,
                                                    int qcap, int fcap, int64_t pfloats,
                                                    int32_t* __restrict__ down_qmax, int nwg) {
  __shared__ int32_t s_cost[2][2048];
  __shared__ int32_t s_tiles[2][2048];  // queued tiles (output tiles x slices)
  __shared__ int32_t s_red[1025];
  __shared__ int32_t s_ns[2048];
  __shared__ int8_t s_sp[2][2048];      // proposed slices of each group
  __shared__ int32_t s_used[2];         // output-tile counters used per phase
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nphase = raw_m >= 0 ? 1 : 2;
  const PlanLayout PL = plan_layout(G, qcap, fcap);
  int32_t* misc = plan + PL.misc;
  if (tid == 0) misc[4] = 0;
  // 1. per group: rows, configuration, output tiles; the phase's work (tiles
  //    times unsliced tile cost, summed exactly) sets the slicing threshold;
  //    then the proposed slices and, for the budget pass, the partial-sum
  //    floats (capped at pfloats + 1, which no budget admits) and the output
  //    tiles of every group that would be sliced
  struct Geom { int m, cfg, bm, bn, mt, nt, kb, kd, nl; };
  auto geom = [&](int ph, int g) {
    Geom q;
    q.m = raw_m >= 0 ? raw_m : (g < E ? counts[g] : T);
    if (!((mask.w[g >> 5] >> (g & 31)) & 1u)) q.m = 0;
    const DevLinear& L = raw_m >= 0 ? raw_lin : experts[g].lin[ph == 0 ? 0 : 2];
    q.cfg = pick_cfg(q.m);
    const int phase_eff = raw_m >= 0 ? 1 : ph;  // raw mode: one linear
    q.bm = cfg_bm(q.cfg);
    q.bn = cfg_bn(q.cfg, phase_eff);
    q.mt = q.m > 0 ? (q.m + q.bm - 1) / q.bm : 0;
    q.nt = (L.n + q.bn - 1) / q.bn;
    q.kb = L.k / 128;
    q.kd = L.kind;
    q.nl = (raw_m < 0 && ph == 0) ? 2 : 1;
    return q;
  };
  __shared__ int64_t s_work[2][1024 / 64];
  for (int ph = 0; ph < nphase; ++ph) {
    int64_t w = 0;
    for (int g = tid; g < G; g += blockDim.x) {
      const Geom q = geom(ph, g);
      const int tiles = q.mt * q.nt;
      if (tiles > 0) w += (int64_t)tiles * tile_cost(q.bm, q.bn, q.nl, q.kd, q.kb * 128, 1, q.mt, q.nt);
    }
    for (int d = 32; d > 0; d >>= 1) w += __shfl_xor(w, d, 64);
    if (lane == 0) s_work[ph][wave] = w;
  }
  __syncthreads();
  for (int ph = 0; ph < nphase; ++ph) {
    int64_t work = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) work += s_work[ph][i];
    const int64_t theta = work / nwg / kSplitShare;
    for (int g = tid; g < G; g += blockDim.x) {
      const Geom q = geom(ph, g);
      const int sp = choose_split(q.bm, q.bn, q.nl, q.kd, q.kb, q.mt, q.nt, theta);
      int32_t* r = plan + PL.rec + ((int64_t)ph * G + g) * PF_N;
      r[PF_EXPERT] = g;
      r[PF_M] = q.m;
      r[PF_CFG] = q.cfg;
      r[PF_MTILES] = q.mt;
      r[PF_NTILES] = q.nt;
      r[PF_START] = 0;
      if (ph == 0 && raw_m < 0) down_qmax[g] = kind_qmax(experts[g].lin[2].kind);
      const int64_t need = (int64_t)q.mt * q.nt * sp * q.bm * q.bn * q.nl;
      s_sp[ph][g] = (int8_t)sp;
      s_tiles[ph][g] = sp > 1 ? q.mt * q.nt : 0;
      s_cost[ph][g] = sp > 1 ? (int32_t)(need <= pfloats ? need : pfloats + 1) : 0;
    }
  }
  if (tid == 0) misc[8] = nwg;
  __syncthreads();
  // 2. slices within the budgets, greedily in group order: a group is sliced
  //    if its partial sums and added tiles still fit, else it runs unsliced.
  //    One wavefront per phase takes 64 groups at a time; a chunk that fits
  //    whole is accepted at once (what the greedy pass does with it), any
  //    other chunk is decided group by group.
  if (wave < nphase) {
    const int ph = wave;
    int64_t pused = 0;
    int eused = 0, cused = 0;
    for (int c0 = 0; c0 < G; c0 += 64) {
      const int g = c0 + lane;
      const int sp = g < G ? s_sp[ph][g] : 1;
      const int tl = g < G ? s_tiles[ph][g] : 0;  // 0 unless sliced
      const int64_t need = g < G ? s_cost[ph][g] : 0;
      const int extra = tl * (sp - 1) <= kSplitExtra ? tl * (sp - 1) : kSplitExtra + 1;
      int64_t pin = need;
      int ein = extra, cin = tl;
      for (int d = 1; d < 64; d <<= 1) {
        const int64_t tp = __shfl_up(pin, d, 64);
        const int te = __shfl_up(ein, d, 64), tc = __shfl_up(cin, d, 64);
        if (lane >= d) {
          pin += tp;
          ein += te;
          cin += tc;
        }
      }
      const int64_t ptot = __shfl(pin, 63, 64);
      const int etot = __shfl(ein, 63, 64), ctot = __shfl(cin, 63, 64);
      bool take = tl > 0;
      int64_t pbase = 0;
      int cbase = 0;
      if (pused + ptot <= pfloats && (int64_t)eused + etot <= kSplitExtra) {
        pbase = pused + pin - need;
        cbase = cused + cin - tl;
        pused += ptot;
        eused += etot;
        cused += ctot;
      } else {
        for (int j = 0; j < 64; ++j) {
          const int64_t nj = __shfl(need, j, 64);
          const int ej = __shfl(extra, j, 64), tj = __shfl(tl, j, 64);
          if (tj <= 0) continue;
          const bool ok = pused + nj <= pfloats && eused + ej <= kSplitExtra;
          if (lane == j) {
            take = ok;
            pbase = pused;
            cbase = cused;
          }
          if (ok) {
            pused += nj;
            eused += ej;
            cused += tj;
          }
        }
      }
      if (g < G) {
        int32_t* r = plan + PL.rec + ((int64_t)ph * G + g) * PF_N;
        r[PF_SPLIT] = take ? sp : 1;
        r[PF_PBASE] = take ? (int32_t)pbase : 0;
        r[PF_CBASE] = take ? cbase : 0;
      }
    }
    if (lane == 0) {
      s_used[ph] = cused;
      misc[6 + ph] = (int32_t)pused;
    }
  }
  __syncthreads();
  // 3. per-tile cost estimate with the final slices, arrival counters cleared
  for (int ph = 0; ph < nphase; ++ph) {
    for (int g = tid; g < G; g += blockDim.x) {
      int32_t* r = plan + PL.rec + ((int64_t)ph * G + g) * PF_N;
      const Geom q = geom(ph, g);
      const int sp = r[PF_SPLIT];
      const int tiles = q.mt * q.nt * sp;
      const int c = tiles ? tile_cost(q.bm, q.bn, q.nl, q.kd, (q.kb + sp - 1) / sp * 128, sp, q.mt, q.nt) : 0;
      r[PF_COST] = c;
      s_cost[ph][g] = c;
      s_tiles[ph][g] = tiles;
    }
    int32_t* cnt = plan + PL.cnt + (int64_t)ph * kSplitExtra;
    for (int i = tid; i < s_used[ph]; i += blockDim.x) cnt[i] = 0;
  }
  __syncthreads();
  // 4. rank the groups by decreasing tile cost (ties: lower group first)
  int32_t* order = plan + PL.order;
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
      plan[PL.rec + ((int64_t)ph * G + g) * PF_N + PF_RANK] = rank;
    }
  }
  __syncthreads();
  // 5. super-tiles dealt to the XCD queues, 6. expanded to tile entries
  for (int ph = 0; ph < nphase; ++ph) {
    int ng = 0;
    for (int g = 0; g < G; ++g) ng += s_tiles[ph][g] > 0;  // same value in every thread
    for (int r = ng + tid; r < G; r += blockDim.x) order[(int64_t)ph * G + r] = -1;
    for (int r = tid; r < ng; r += blockDim.x) {
      const int32_t* rec = plan + PL.rec + ((int64_t)ph * G + order[(int64_t)ph * G + r]) * PF_N;
      s_ns[r] = super_tiles(rec[PF_MTILES], rec[PF_NTILES] * rec[PF_SPLIT]);
    }
    __syncthreads();
    const int S = block_scan(s_ns, ng, s_red);  // s_ns[r]: first global super-tile of rank r
    int32_t* ent = plan + PL.ent + (int64_t)ph * kXcd * qcap * 3;
    // deal super-tile u to queue u % kXcd, position u / kXcd
    for (int u = tid; u < S; u += blockDim.x) {
      int lo = 0, hi = ng;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_ns[mid] <= u) lo = mid; else hi = mid;
      }
      const int g = order[(int64_t)ph * G + lo];
      const int s = u - s_ns[lo];
      const int32_t* rec = plan + PL.rec + ((int64_t)ph * G + g) * PF_N;
      if (u / kXcd >= qcap) {  // cannot happen with the host's capacity bound
        misc[4] = 1;
        continue;
      }
      int32_t* e = ent + ((int64_t)(u % kXcd) * qcap + u / kXcd) * 3;
      e[0] = g;
      e[1] = s;
      e[2] = super_tile_size(rec[PF_MTILES], rec[PF_NTILES] * rec[PF_SPLIT], s);
    }
    __syncthreads();
    // per-queue exclusive prefix sums of the entry sizes, one wavefront per queue
    int32_t* ctr = plan + PL.ctr + (int64_t)ph * kXcd * 4;
    if (wave < kXcd) {
      const int x = wave;
      int n = S / kXcd + (x < S % kXcd ? 1 : 0);
      n = n < qcap ? n : qcap;
      int32_t* q = ent + (int64_t)x * qcap * 3 + 2;
      int run = 0;
      for (int c0 = 0; c0 < n; c0 += 64) {
        const int i = c0 + lane;
        const int v = i < n ? q[(int64_t)i * 3] : 0;
        int incl = v;
        for (int d = 1; d < 64; d <<= 1) {
          const int t = __shfl_up(incl, d, 64);
          if (lane >= d) incl += t;
        }
        if (i < n) q[(int64_t)i * 3] = run + incl - v;
        run += __shfl(incl, 63, 64);
      }
      if (lane == 0) {
        ctr[x * 4 + 0] = 0;
        ctr[x * 4 + 1] = run;
        ctr[x * 4 + 2] = n;
      }
    }
    __syncthreads();
    // expand the queues: one thread per queue entry writes its tiles
    int32_t* flat = plan + PL.flat + (int64_t)ph * kXcd * fcap * 4;
    for (int u = tid; u < S; u += blockDim.x) {
      const int x = u % kXcd, pos = u / kXcd;
      if (pos >= qcap) continue;
      const int32_t* e = ent + ((int64_t)x * qcap + pos) * 3;
      const int g = e[0], st = e[1], first = e[2];
      const int32_t* rec = plan + PL.rec + ((int64_t)ph * G + g) * PF_N;
      const int sp = rec[PF_SPLIT];
      const int mt = rec[PF_MTILES], ntv = rec[PF_NTILES] * sp;
      const int size = super_tile_size(mt, ntv, st);
      if (first + size > fcap) {  // cannot happen with the host's capacity bound
        misc[4] = 1;
        continue;
      }
      const int kd = raw_m >= 0 ? raw_lin.kind : experts[g].lin[ph == 0 ? 0 : 2].kind;
      const int w0 = tile_word0(g, rec[PF_CFG], kd, sp);
      const int off_e = (raw_m < 0 && g < E) ? offsets[g] : 0;
      const int m_g = rec[PF_M];
      int32_t* f = flat + ((int64_t)x * fcap + first) * 4;
      for (int t = 0; t < size; ++t) {
        int mi, ni;
        super_tile_pos(mt, ntv, st, t, &mi, &ni);
        *reinterpret_cast<int4*>(f + 4 * t) = make_int4(w0, mi | (ni << 16), off_e, m_g);
      }
    }
    __syncthreads();
    if (tid == 0) misc[2 + ph] = ng;
    __syncthreads();
  }
  if (nphase == 1) {  // single-linear mode: the second phase is empty
    int32_t* ctr = plan + PL.ctr + (int64_t)kXcd * 4;
    if (tid < kXcd) {
      ctr[tid * 4 + 0] = 0;
      ctr[tid * 4 + 1] = 0;
      ctr[tid * 4 + 2] = 0;
    }
    if (tid == 0) misc[3] = 0;
  }
}

}  // namespace

hipError_t launch_plan(const DevExpert* experts, int E, int G, int T, const int32_t* counts,
                       const int32_t* offsets, int raw_m, const DevLinear& raw_lin, const uint32_t* mask_words,
                       int32_t* plan, int qcap, int fcap, int64_t pfloats, int32_t* down_qmax, int nwg,
                       hipStream_t s) {
  MaskBits mb;
  for (int i = 0; i < 64; ++i) mb.w[i] = mask_words ? mask_words[i] : 0xffffffffu;
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, experts, E, G, T, counts, offsets, raw_m, raw_lin, mb,
                     plan, qcap, fcap, pfloats, down_qmax, nwg < 1 ? 1 : nwg);
  return hipGetLastError();
}

hipError_t launch_group_gemm(const GemmArgs& a, int phase, int grid, hipStream_t s) {
  if (a.act == MXMOE_BF16)
    return phase == 0 ? gg_bf16_p0(a, grid, s) : (phase == 1 ? gg_bf16_p1(a, grid, s) : gg_bf16_raw(a, grid, s));
  return phase == 0 ? gg_f16_p0(a, grid, s) : (phase == 1 ? gg_f16_p1(a, grid, s) : gg_f16_raw(a, grid, s));
}

int group_gemm_grid(int device) {
  static int cached[64] = {0};
  if (device < 0 || device >= 64) device = 0;
  if (!cached[device]) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || cus <= 0) cus = 256;
    cached[device] = cus * 2;  // two resident workgroups per CU
  }
  return cached[device];
}

}  // namespace mxmoe
