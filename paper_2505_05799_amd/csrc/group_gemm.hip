// Tile plan of the mixed-precision Group-GEMM and the launch dispatch (the
// micro-kernels themselves are in group_gemm_impl.h, one translation unit per
// activation dtype and phase).
//
// plan_kernel (one workgroup, no host round trip):
//   1. per (phase, expert) group: rows m (routing counts, T for shared experts),
//      tile configuration from m, tile counts, the per-tile cost from the
//      cost table (tile_cost);
//   2. rank the groups by decreasing tile cost (ties: lower expert first) - the
//      greedy longest-tile-first order of the paper's tile schedule;
//   3. cut every group into super-tiles (up to 64 tiles that share row and
//      channel blocks) and deal them round-robin, in rank order, to one queue
//      per XCD; per-queue prefix sums give each entry's first tile;
//   4. expand every queue into one 16-byte entry per tile (group, configuration,
//      kind, slices, tile coordinates, first sorted row and rows of the group),
//      so that a workgroup resolves a popped tile with a single load.
// Groups may be sliced along the reduction (split-K, kSplitShare / kSplitMinKb): their
// slices are queued as extra channel tiles, within fixed budgets of added
// tiles and of partial-sum storage.
#include <mutex>

#include "group_gemm_impl.h"
#include "rowquant.h"

namespace mxmoe {
namespace {

struct MaskBits { uint32_t w[64]; };

// x / d for 0 <= x < 2^22 and 1 <= d < 2^22, exactly: a float reciprocal
// estimate (within one of the quotient there) and one correction step; a
// fraction of the cost of a general integer division, which the plan's
// per-tile loops would otherwise repeat thousands of times.
__device__ inline int div_small(int x, int d) {
  int q = (int)((float)x * __builtin_amdgcn_rcpf((float)d));
  q -= q * d > x;
  q += (q + 1) * d <= x;
  return q;
}
// Super-tile geometry (SuperDims), with div_small for the divisions
__device__ inline SuperDims plan_super_dims(int mt, int nt) {
  SuperDims d;
  d.sm = mt < 8 ? mt : 8;
  const int cap = div_small(kSuperTiles, d.sm > 0 ? d.sm : 1);
  d.sn = nt < cap ? nt : cap;
  d.nsm = d.sm ? div_small(mt + d.sm - 1, d.sm) : 0;
  d.nsn = d.sn ? div_small(nt + d.sn - 1, d.sn) : 0;
  return d;
}

__global__ void __launch_bounds__(1024) plan_kernel(const DevExpert* __restrict__ experts, int E, int G, int T,
                                                    const int32_t* __restrict__ counts,
                                                    const int32_t* __restrict__ offsets, int raw_m,
                                                    DevLinear raw_lin, MaskBits mask, int32_t* __restrict__ plan,
                                                    int qcap, int fcap, int64_t pfloats,
                                                    int32_t* __restrict__ down_qmax, int nwg, XPrep xp,
                                                    TileCosts tc) {
  // workgroups 1.. encode x, one row per wavefront (grid-stride); the plan
  // below runs on workgroup 0 alone
  if (blockIdx.x > 0) {
    const int64_t nw = (int64_t)(gridDim.x - 1) * (blockDim.x >> 6);
    for (int64_t r = (int64_t)(blockIdx.x - 1) * (blockDim.x >> 6) + (threadIdx.x >> 6); r < xp.rows; r += nw)
      x_prep_row(xp, r);
    return;
  }
  // Every per-group input is read from global memory once, into LDS; the steps
  // below work from LDS and only write the plan out, so their barriers wait
  // for LDS traffic only and the plan's stores drain in the background.
  __shared__ int32_t s_m[kMaxG];          // rows of each group (0 if masked)
  __shared__ int32_t s_off[kMaxG];        // first sorted row (routed groups)
  __shared__ int32_t s_n[2][kMaxG];       // output channels of the phase's linear
  __shared__ int32_t s_kb[2][kMaxG];      // its 128-wide k blocks
  __shared__ int8_t s_kd[2][kMaxG];       // its micro-kernel kind
  __shared__ int8_t s_sp[2][kMaxG];       // slices: proposed (| 16 if by the fallback), then final
  __shared__ int32_t s_cost[2][kMaxG];    // budget need, then tile cost
  __shared__ int32_t s_tiles[2][kMaxG];   // sliced output tiles, then queued tiles
  __shared__ int32_t s_order[2][kMaxG];   // group per rank
  __shared__ int32_t s_c1[2][kMaxG];      // unsliced tile cost
  __shared__ int32_t s_cs[2][kMaxG];      // tile cost with the proposed slices
  __shared__ int64_t s_work[2][1024 / 64];
  __shared__ int64_t s_theta[2];          // slicing threshold per phase
  __shared__ int32_t s_ut[2][1024 / 64];  // unsliced tiles per wavefront, then per phase in [p][0]
  __shared__ int32_t s_used[2];           // output-tile counters used per phase
  __shared__ int32_t s_tc[kCostEntries];  // tile cost table
  __shared__ int32_t s_ng[2];             // groups with tiles per phase
  __shared__ int32_t s_nst[2];            // super-tiles per phase
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nwave = blockDim.x >> 6;
  const int nphase = raw_m >= 0 ? 1 : 2;
  const PlanLayout PL = plan_layout(G, qcap, fcap);
  int32_t* misc = plan + PL.misc;
  int32_t* order = plan + PL.order;
  auto rec_of = [&](int ph, int g) { return plan + PL.rec + ((int64_t)ph * G + g) * PF_N; };

  // 0. inputs (and the cost table)
  for (int i = tid; i < kCostEntries; i += blockDim.x) s_tc[i] = tc.v[i];
  for (int g = tid; g < G; g += blockDim.x) {
    int m = raw_m >= 0 ? raw_m : (g < E ? counts[g] : T);
    if (!((mask.w[g >> 5] >> (g & 31)) & 1u)) m = 0;
    s_m[g] = m;
    s_off[g] = (raw_m < 0 && g < E) ? offsets[g] : 0;
    for (int ph = 0; ph < nphase; ++ph) {
      const DevLinear& L = raw_m >= 0 ? raw_lin : experts[g].lin[ph == 0 ? 0 : 2];
      s_n[ph][g] = L.n;
      s_kb[ph][g] = L.k / 128;
      s_kd[ph][g] = (int8_t)L.kind;
    }
    if (raw_m < 0) {
      const int dk = experts[g].lin[2].kind;
      down_qmax[g] = dk == K_MXFP4 ? kDownQMX
                    : (dk == K_F8A8 ? kDownQF8
                                    : (kind_qmax(dk) | (dk == K_W4A4G ? kDownQGroup : 0) | (dk == K_W4A4F6 ? kDownQF6 : 0)));
    }
  }
  if (tid < 2) s_ng[tid] = 0;
  if (tid == 0) {
    misc[4] = 0;
    misc[8] = nwg;
  }
  lds_barrier();
  struct Geom { int m, cfg, bm, bn, mt, nt, kb, kd, nl, ce; };
  auto geom = [&](int ph, int g) {
    Geom q;
    q.m = s_m[g];
    q.cfg = pick_cfg(q.m, s_kd[ph][g], raw_m >= 0 ? 0 : ph);
    q.bm = cfg_bm(q.cfg);
    q.bn = cfg_bn(q.cfg, raw_m >= 0 ? 1 : ph);  // raw mode: one linear
    q.mt = q.m > 0 ? div_small(q.m + q.bm - 1, q.bm) : 0;
    q.nt = div_small(s_n[ph][g] + q.bn - 1, q.bn);
    q.kb = s_kb[ph][g];
    q.kd = s_kd[ph][g];
    q.nl = (raw_m < 0 && ph == 0) ? 2 : 1;
    q.ce = cost_index(raw_m >= 0 ? 1 : ph, q.kd, q.cfg);  // raw mode: one linear
    return q;
  };

  // 1. per group the unsliced tile cost (kept for the steps below); the
  //    phase's work (tiles times that cost, summed exactly) sets the slicing
  //    threshold and its unsliced tiles the fallback budget; then per group
  //    the proposed slices and, for the budget pass, the partial-sum floats
  //    (capped at pfloats + 1, which no budget admits) and the output tiles
  //    of every group that would be sliced
  for (int ph = 0; ph < nphase; ++ph) {
    int64_t w = 0;
    int u = 0;
    for (int g = tid; g < G; g += blockDim.x) {
      const Geom q = geom(ph, g);
      const int tiles = q.mt * q.nt;
      const int32_t c = tiles > 0 ? tile_cost(s_tc + q.ce, q.kb, 1, q.mt) : 0;
      s_c1[ph][g] = c;
      w += (int64_t)tiles * c;
      u += tiles;
    }
    for (int d = 32; d > 0; d >>= 1) {
      w += __shfl_xor(w, d, 64);
      u += __shfl_xor(u, d, 64);
    }
    if (lane == 0) {
      s_work[ph][wave] = w;
      s_ut[ph][wave] = u;
    }
  }
  lds_barrier();
  if (wave < nphase) {  // wavefront p sums phase p's per-wavefront totals
    int64_t work = lane < nwave ? s_work[wave][lane] : 0;
    int ut = lane < nwave ? s_ut[wave][lane] : 0;
    for (int d = 32; d > 0; d >>= 1) {
      work += __shfl_xor(work, d, 64);
      ut += __shfl_xor(ut, d, 64);
    }
    if (lane == 0) {
      s_theta[wave] = work / nwg / kSplitShare;
      s_ut[wave][0] = ut;
    }
  }
  lds_barrier();
  // The slice rule (kSplitShare, kSplitMinKb), evaluated by eight lanes per group: lane
  // j prices j + 1 slices; the group takes the fewest slices whose tile cost
  // is within theta, else the cheapest (the fewest slices among equals).
  for (int base = 0; base < nphase * G; base += (int)blockDim.x / 8) {
    const int item = base + tid / 8, s = (tid & 7) + 1;
    const bool live = item < nphase * G;
    const int ph = live && item >= G ? 1 : 0, g = live ? item - ph * G : 0;
    const Geom q = geom(ph, g);
    const bool tiled = live && q.mt * q.nt > 0;
    int smax = q.kb / kSplitMinKb;
    smax = smax < 1 ? 1 : (smax > kSplitMax ? kSplitMax : smax);
    const bool ok = tiled && s <= smax;
    int32_t c = 0;
    if (ok) c = s == 1 ? s_c1[ph][g] : tile_cost(s_tc + q.ce, (q.kb + s - 1) / s, s, q.mt);
    int first = (ok && c <= s_theta[ph]) ? s : 64;
    int64_t key = ok ? (((int64_t)c << 8) | s) : INT64_MAX;
    for (int d = 1; d < 8; d <<= 1) {
      first = min(first, __shfl_xor(first, d, 64));
      const int64_t kk = __shfl_xor(key, d, 64);
      key = kk < key ? kk : key;
    }
    // the cost of `first` slices, from the lane that priced it (every lane
    // takes part in the shuffle)
    const int32_t c_first = __shfl(c, (lane & ~7) + (first <= kSplitMax ? first - 1 : 0), 64);
    if (live && s == 1) {
      int sp = 1;
      int32_t csp = s_c1[ph][g];
      if (tiled) {
        if (first <= kSplitMax) {
          sp = first;
          csp = c_first;
        } else {
          sp = (int)(key & 0xFF);
          csp = (int32_t)(key >> 8);
        }
      }
      int32_t* r = rec_of(ph, g);
      r[PF_EXPERT] = g;
      r[PF_M] = q.m;
      r[PF_CFG] = q.cfg;
      r[PF_MTILES] = q.mt;
      r[PF_NTILES] = q.nt;
      r[PF_START] = 0;
      const int64_t need = (int64_t)q.mt * q.nt * sp * q.bm * q.bn * q.nl;
      s_sp[ph][g] = (int8_t)(sp | (tiled && first > kSplitMax && sp > 1 ? 16 : 0));
      s_cs[ph][g] = csp;
      s_tiles[ph][g] = sp > 1 ? q.mt * q.nt : 0;
      s_cost[ph][g] = sp > 1 ? (int32_t)(need <= pfloats ? need : pfloats + 1) : 0;
    }
  }
  lds_barrier();
  // 2. slices within the budgets, greedily in group order: a group is sliced
  //    if its partial sums and added tiles still fit; a group whose slices
  //    come from the fallback (no slice count within theta) also needs the
  //    phase's tiles, with every slice granted so far and its own, to stay
  //    within one tile per workgroup, and once one such group is refused
  //    for that no later one is sliced.  (Slicing the long tiles of a launch
  //    with fewer tiles than workgroups shortens its one wave of tiles; past
  //    one tile per workgroup it adds a second wave.)  Groups not sliced run
  //    unsliced.  One wavefront per phase takes 64 groups at a time; in a
  //    chunk whose partial sums and added tiles fit whole the fallback rule
  //    is one prefix sum, any other chunk is decided group by group.
  if (wave < nphase) {
    const int ph = wave;
    const int64_t ut = s_ut[ph][0];
    int64_t pused = 0;
    int eused = 0, cused = 0;
    bool stopped = false;  // a fallback group was refused (wave-uniform)
    auto scan3 = [&](int64_t& p, int& e, int& c) {
      for (int d = 1; d < 64; d <<= 1) {
        const int64_t tp = __shfl_up(p, d, 64);
        const int te = __shfl_up(e, d, 64), tc = __shfl_up(c, d, 64);
        if (lane >= d) {
          p += tp;
          e += te;
          c += tc;
        }
      }
    };
    for (int c0 = 0; c0 < G; c0 += 64) {
      const int g = c0 + lane;
      const int spv = g < G ? s_sp[ph][g] : 1;
      const int sp = spv & 15;
      const bool fb = (spv & 16) != 0;
      const int tl = g < G ? s_tiles[ph][g] : 0;  // 0 unless sliced
      const int64_t need = g < G ? s_cost[ph][g] : 0;
      const int extra = tl * (sp - 1) <= kSplitExtra ? tl * (sp - 1) : kSplitExtra + 1;
      int64_t pin = need;
      int ein = extra, cin = tl;
      scan3(pin, ein, cin);
      const int64_t ptot = __shfl(pin, 63, 64);
      const int etot = __shfl(ein, 63, 64);
      bool take = tl > 0;
      int64_t pbase = 0;
      int cbase = 0;
      if (pused + ptot <= pfloats && (int64_t)eused + etot <= kSplitExtra) {
        // every group before the first refused fallback group is granted, so
        // the tiles a group sees are the prefix sum over all candidates
        const uint64_t fm = __ballot(fb && tl > 0 && (stopped || ut + eused + ein > nwg));
        const int f = fm ? __ffsll((unsigned long long)fm) - 1 : 64;
        take = tl > 0 && (!fb || lane < f);
        stopped = stopped || fm != 0;
        int64_t p2 = take ? need : 0;
        int e2 = take ? extra : 0, c2 = take ? tl : 0;
        scan3(p2, e2, c2);
        pbase = pused + p2 - (take ? need : 0);
        cbase = cused + c2 - (take ? tl : 0);
        pused += __shfl(p2, 63, 64);
        eused += __shfl(e2, 63, 64);
        cused += __shfl(c2, 63, 64);
      } else {
        // the chunk's candidates in group order (a wave-uniform lane index,
        // so each input is one lane read)
        uint64_t cand = __ballot(tl > 0);
        while (cand) {
          const int j = __ffsll((unsigned long long)cand) - 1;
          cand &= cand - 1;
          const int64_t nj = __builtin_amdgcn_readlane((int)need, j);
          const int ej = __builtin_amdgcn_readlane(extra, j);
          const int tj = __builtin_amdgcn_readlane(tl, j);
          const bool fj = __builtin_amdgcn_readlane((int)fb, j) != 0;
          if (fj && ut + eused + ej > nwg) stopped = true;
          const bool ok = pused + nj <= pfloats && eused + ej <= kSplitExtra && (!fj || !stopped);
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
        int32_t* r = rec_of(ph, g);
        r[PF_SPLIT] = take ? sp : 1;
        r[PF_PBASE] = take ? (int32_t)pbase : 0;
        r[PF_CBASE] = take ? cbase : 0;
        s_sp[ph][g] = (int8_t)(take ? sp : 1);
      }
    }
    if (lane == 0) {
      s_used[ph] = cused;
      misc[6 + ph] = (int32_t)pused;
    }
  }
  lds_barrier();
  // 3. per-tile cost with the final slices (priced in step 1), arrival
  //    counters cleared
  for (int ph = 0; ph < nphase; ++ph) {
    for (int g = tid; g < G; g += blockDim.x) {
      const Geom q = geom(ph, g);
      const int sp = s_sp[ph][g];
      const int tiles = q.mt * q.nt * sp;
      const int c = tiles ? (sp > 1 ? s_cs[ph][g] : s_c1[ph][g]) : 0;
      rec_of(ph, g)[PF_COST] = c;
      s_cost[ph][g] = c;
      s_tiles[ph][g] = tiles;
      if (tiles > 0) atomicAdd(&s_ng[ph], 1);
    }
    int32_t* cnt = plan + PL.cnt + (int64_t)ph * kSplitExtra;
    for (int i = tid; i < s_used[ph]; i += blockDim.x) cnt[i] = 0;
  }
  lds_barrier();
  // 4. rank the groups by decreasing tile cost (ties: lower group first):
  //    one wavefront per group, each lane tests the groups of one chunk of 64
  //    and a ballot counts those ahead; the first chunk's costs stay in
  //    registers across the wavefront's groups of a phase
  for (int ph = 0; ph < nphase; ++ph) {
    const int own_c = lane < G ? s_cost[ph][lane] : 0;
    const bool own_l = lane < G && s_tiles[ph][lane] > 0;
    for (int g = wave; g < G; g += nwave) {
      int rank = -1;
      if (s_tiles[ph][g] > 0) {
        const int cg = s_cost[ph][g];
        int ahead = 0;
        for (int c0 = 0; c0 < G; c0 += 64) {
          const int h = c0 + lane;
          const int ch = c0 == 0 ? own_c : (h < G ? s_cost[ph][h] : 0);
          const bool live = c0 == 0 ? own_l : (h < G && s_tiles[ph][h] > 0);
          ahead += __popcll(__ballot(live && (ch > cg || (ch == cg && h < g))));
        }
        rank = ahead;
        if (lane == 0) {
          s_order[ph][rank] = g;
          order[(int64_t)ph * G + rank] = g;
        }
      }
      if (lane == 0) rec_of(ph, g)[PF_RANK] = rank;
    }
  }
  lds_barrier();
  // 5. super-tiles dealt to the XCD queues, 6. expanded to tile entries;
  //    both phases at once (waves 8p .. 8p + 7 build the queues of phase p).
  //    s_cost is free from here on: s_cost[p][r] holds the super-tile count
  //    of rank r, then its exclusive prefix sum (first global super-tile).
  auto dims = [&](int ph, int g, int* mt, int* ntv) {  // row tiles, channel tiles x slices
    const Geom q = geom(ph, g);
    *mt = q.mt;
    *ntv = q.nt * s_sp[ph][g];
  };
  for (int ph = 0; ph < nphase; ++ph) {
    const int ng = s_ng[ph];
    for (int r = ng + tid; r < G; r += blockDim.x) order[(int64_t)ph * G + r] = -1;
    for (int r = tid; r < ng; r += blockDim.x) {
      int mt, ntv;
      dims(ph, s_order[ph][r], &mt, &ntv);
      const SuperDims dd = plan_super_dims(mt, ntv);
      s_cost[ph][r] = (mt > 0 && ntv > 0) ? dd.nsm * dd.nsn : 0;
    }
  }
  lds_barrier();
  // exclusive prefix sums of the super-tile counts in rank order, one
  //    wavefront per phase, 64 ranks at a time
  if (wave < nphase) {
    const int ph = wave, n = s_ng[ph];
    int run = 0;
    for (int c0 = 0; c0 < n; c0 += 64) {
      const int i = c0 + lane;
      const int v = i < n ? s_cost[ph][i] : 0;
      int incl = v;
      for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(incl, d, 64);
        if (lane >= d) incl += t;
      }
      if (i < n) s_cost[ph][i] = run + incl - v;
      run += __shfl(incl, 63, 64);
    }
    if (lane == 0) s_nst[ph] = run;
  }
  lds_barrier();
  int S_ph[2] = {0, 0};
  for (int ph = 0; ph < nphase; ++ph) S_ph[ph] = s_nst[ph];
  if (tid < nphase) {
    if ((S_ph[tid] + kXcd - 1) / kXcd > qcap) misc[4] = 1;  // cannot happen with the host's capacity bound
    misc[2 + tid] = s_ng[tid];
  }
  if (wave < nphase * kXcd) {
    const int ph = wave / kXcd, x = wave % kXcd;
    const int ng = s_ng[ph], S = S_ph[ph];
    const int32_t* s_ns = s_cost[ph];
    // super-tile u -> (rank, index within the group)
    auto locate = [&](int u, int* g, int* st) {
      int lo = 0, hi = ng;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_ns[mid] <= u) lo = mid; else hi = mid;
      }
      *g = s_order[ph][lo];
      *st = u - s_ns[lo];
    };
    int32_t* ent = plan + PL.ent + (int64_t)ph * kXcd * qcap * 3;
    int32_t* ctr = plan + PL.ctr + (int64_t)ph * kXcd * 4;
    // deal super-tile u to queue u % kXcd, position u / kXcd; the queue's
    // wavefront forms the exclusive prefix sums of the entry sizes (each
    // entry's first tile) and expands each entry into its tiles
    int32_t* flat = plan + PL.flat + (int64_t)ph * kXcd * fcap * 4;
    int n = S / kXcd + (x < S % kXcd ? 1 : 0);
    n = n < qcap ? n : qcap;
    int32_t* q = ent + (int64_t)x * qcap * 3;
    int run = 0;
    for (int c0 = 0; c0 < n; c0 += 64) {
      const int i = c0 + lane;
      int g = 0, st = 0, v = 0, mt = 0, ntv = 0;
      if (i < n) {
        locate(i * kXcd + x, &g, &st);
        dims(ph, g, &mt, &ntv);
        const SuperDims dd = plan_super_dims(mt, ntv);
        const int sni = div_small(st, dd.nsm), smi = st - sni * dd.nsm;
        v = min(dd.sm, mt - smi * dd.sm) * min(dd.sn, ntv - sni * dd.sn);
      }
      int incl = v;
      for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(incl, d, 64);
        if (lane >= d) incl += t;
      }
      const int first = run + incl - v;
      run += __shfl(incl, 63, 64);
      // this lane's entry: its record, and what expanding it takes
      int w0 = 0, off_e = 0, m_g = 0, mi0 = 0, ni0 = 0, em = 1, inv = 65536, size = 0;
      if (i < n) {
        q[(int64_t)i * 3 + 0] = g;
        q[(int64_t)i * 3 + 1] = st;
        q[(int64_t)i * 3 + 2] = first;
        if (first + v <= fcap) {
          const SuperDims dd = plan_super_dims(mt, ntv);
          const int sni = div_small(st, dd.nsm), smi = st - sni * dd.nsm;
          em = min(dd.sm, mt - smi * dd.sm);
          inv = div_small(65536 + em - 1, em);  // t / em = (t * inv) >> 16 for t < 64, em <= 8
          mi0 = smi * dd.sm;
          ni0 = sni * dd.sn;
          w0 = tile_word0(g, pick_cfg(s_m[g], s_kd[ph][g], raw_m >= 0 ? 0 : ph), s_kd[ph][g], s_sp[ph][g]);
          off_e = s_off[g];
          m_g = s_m[g];
          size = v;
        } else {
          misc[4] = 1;  // cannot happen with the host's capacity bound
        }
      }
      // The chunk's entries are expanded one at a time by the whole
      // wavefront (lane t writes the entry's tile t, row tile fastest, the
      // order of the SuperDims geometry), so that every store is contiguous; the
      // entry's fields come from its lane's registers.
      const int cnt = n - c0 < 64 ? n - c0 : 64;
      for (int j = 0; j < cnt; ++j) {
        const int sz = __builtin_amdgcn_readlane(size, j);
        if (sz == 0) continue;
        const int fj = __builtin_amdgcn_readlane(first, j);
        const int emj = __builtin_amdgcn_readlane(em, j), invj = __builtin_amdgcn_readlane(inv, j);
        const int w0j = __builtin_amdgcn_readlane(w0, j), offj = __builtin_amdgcn_readlane(off_e, j);
        const int mgj = __builtin_amdgcn_readlane(m_g, j);
        const int mi0j = __builtin_amdgcn_readlane(mi0, j), ni0j = __builtin_amdgcn_readlane(ni0, j);
        if (lane < sz) {
          const int b2 = (int)(((uint32_t)lane * (uint32_t)invj) >> 16), a2 = lane - b2 * emj;
          reinterpret_cast<int4*>(flat + ((int64_t)x * fcap + fj) * 4)[lane] =
              make_int4(w0j, (mi0j + a2) | ((ni0j + b2) << 16), offj, mgj);
        }
      }
    }
    if (lane == 0) {
      ctr[x * 4 + 0] = 0;
      ctr[x * 4 + 1] = run;
      ctr[x * 4 + 2] = n;
    }
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

// Roofline default of the tile cost table, in the table's additive form: a
// fixed 2 us per tile; bs the MFMA time of a k block at one CU's share of the
// MI355X dense peak of the kind's operands (10 PFLOP/s FP4 / FP6, 5 POPS int8
// and FP8, 2.5 PFLOP/s 16-bit); bu the time of the tile's weight bytes of a k
// block at one CU's share of 8 TB/s (32 ps per byte); h the time of writing
// and reading back the tile's fp32 partial sums (8 bytes per output) at that
// share.
void tile_costs_default(TileCosts* out) {
  for (int ph = 0; ph < 2; ++ph)
    for (int kd = 0; kd < K_COUNT; ++kd)
      for (int c = 0; c < kCostCfgs; ++c) {
        const int bm = cfg_bm(c), bn = cfg_bn(c, ph), nl = ph == 0 ? 2 : 1;
        const double rate = (kind_is_mx(kd) || kind_is_f6(kd)) ? 39062.0 : (kind_is_int(kd) ? 19531.0 : 9766.0);
        int32_t* e = out->v + cost_index(ph, kd, c);
        e[0] = 2000000;
        e[1] = (int32_t)(2.0 * nl * bm * bn * 128 * 1000.0 / rate);
        e[2] = (int32_t)((double)nl * bn * 128 * kind_wbits(kd) / 8.0 * 32.0);
        e[3] = (int32_t)(8.0 * bm * bn * nl * 32.0);
      }
}

namespace {
std::mutex g_cost_mu;
TileCosts g_costs;
bool g_costs_init = false;
}  // namespace

void tile_costs_set(const TileCosts* t) {
  std::lock_guard<std::mutex> lk(g_cost_mu);
  if (t)
    g_costs = *t;
  else
    tile_costs_default(&g_costs);
  g_costs_init = true;
}

void tile_costs_get(TileCosts* out) {
  std::lock_guard<std::mutex> lk(g_cost_mu);
  if (!g_costs_init) {
    tile_costs_default(&g_costs);
    g_costs_init = true;
  }
  *out = g_costs;
}

hipError_t launch_plan(const DevExpert* experts, int E, int G, int T, const int32_t* counts,
                       const int32_t* offsets, int raw_m, const DevLinear& raw_lin, const uint32_t* mask_words,
                       int32_t* plan, int qcap, int fcap, int64_t pfloats, int32_t* down_qmax, int nwg,
                       const XPrep& xp, hipStream_t s) {
  MaskBits mb;
  for (int i = 0; i < 64; ++i) mb.w[i] = mask_words ? mask_words[i] : 0xffffffffu;
  if (xp.rows > 0 && ((reinterpret_cast<uintptr_t>(xp.x) & 15) || xp.cols % 128)) return hipErrorInvalidValue;
  // 16 rows per encoding workgroup, at most 1024 of them (grid-stride beyond)
  int nxb = xp.rows > 0 ? (xp.rows + 15) / 16 : 0;
  nxb = nxb < 1024 ? nxb : 1024;
  TileCosts tc;
  tile_costs_get(&tc);
  hipLaunchKernelGGL(plan_kernel, dim3(1 + nxb), dim3(1024), 0, s, experts, E, G, T, counts, offsets, raw_m, raw_lin,
                     mb, plan, qcap, fcap, pfloats, down_qmax, nwg < 1 ? 1 : nwg, xp, tc);
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
