// Router front-end and routing.
//
// Routing / permutation: stable counting sort of the T*k (token, slot) pairs
// by expert id, which forms the per-expert row groups X_e of Eq. (2).
//
// Three launches (one workgroup for batches of at most kRouteSmall pairs), no
// atomics on anything order-dependent:
//   1. route_count   : one workgroup per chunk of kRouteChunk pairs builds the
//                      chunk's expert histogram (integer LDS atomics: the
//                      counts do not depend on their order) and the smallest
//                      out-of-range pair id of the chunk.
//   2. route_scan    : one workgroup scans chunk histograms in (expert, chunk)
//                      order -> counts, offsets and each chunk's base per expert.
//   3. route_scatter : each chunk walks its pairs in order, 256 at a time; a
//                      wavefront finds lanes with equal expert ids with one
//                      ballot per id bit, ranks them by lane, and wavefront
//                      totals are combined through LDS in wavefront order.
#include <cstring>

#include "mxmoe_internal.h"

namespace mxmoe {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxE = 1024;

__global__ void __launch_bounds__(kThreads) route_count(const int32_t* __restrict__ ids, int P, int E,
                                                         int32_t* __restrict__ chunk_counts,
                                                         int32_t* __restrict__ chunk_bad) {
  __shared__ int32_t hist[kMaxE];
  __shared__ int32_t bad;
  const int c = blockIdx.x;
  for (int e = threadIdx.x; e < E; e += kThreads) hist[e] = 0;
  if (threadIdx.x == 0) bad = 0x7fffffff;
  __syncthreads();
  const int p0 = c * kRouteChunk;
  const int p1 = min(P, p0 + kRouteChunk);
  for (int p = p0 + threadIdx.x; p < p1; p += kThreads) {
    int e = ids[p];
    if (e >= 0 && e < E) atomicAdd(&hist[e], 1);
    else atomicMin(&bad, p);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += kThreads) chunk_counts[(int64_t)c * E + e] = hist[e];
  if (threadIdx.x == 0) chunk_bad[c] = bad;
}

__global__ void __launch_bounds__(1024) route_scan(int nchunks, int E, int32_t* __restrict__ chunk_counts,
                                                   const int32_t* __restrict__ chunk_bad,
                                                   int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
                                                   int32_t* __restrict__ status) {
  __shared__ int32_t tot[kMaxE];
  __shared__ int32_t wsum[16];
  const int tid = threadIdx.x;  // blockDim = 1024 >= E
  // the chunk histograms are read kBatch chunks at a time (independent loads
  // in flight together; one at a time, the loop is a chain of memory round
  // trips: 26 us for 64 chunks)
  constexpr int kBatch = 16;
  int mine = 0;
  if (tid < E) {
    int c = 0;
    for (; c + kBatch <= nchunks; c += kBatch) {
      int v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) v[j] = chunk_counts[(int64_t)(c + j) * E + tid];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) mine += v[j];
    }
    for (; c < nchunks; ++c) mine += chunk_counts[(int64_t)c * E + tid];
  }
  // exclusive scan of per-expert totals across the workgroup
  const int lane = tid & 63, w = tid >> 6;
  int incl = mine;
  for (int d = 1; d < 64; d <<= 1) {
    int v = __shfl_up(incl, d, 64);
    if (lane >= d) incl += v;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int base = 0;
  for (int i = 0; i < w; ++i) base += wsum[i];
  const int excl = base + incl - mine;
  if (tid < E) {
    counts[tid] = mine;
    offsets[tid] = excl;
    tot[tid] = excl;
    // chunk bases, in place: chunk_counts[c][e] <- offset of chunk c's first pair of e
    int run = excl;
    int c = 0;
    for (; c + kBatch <= nchunks; c += kBatch) {
      int v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) v[j] = chunk_counts[(int64_t)(c + j) * E + tid];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        chunk_counts[(int64_t)(c + j) * E + tid] = run;
        run += v[j];
      }
    }
    for (; c < nchunks; ++c) {
      const int64_t i = (int64_t)c * E + tid;
      const int v = chunk_counts[i];
      chunk_counts[i] = run;
      run += v;
    }
  }
  if (tid == E - 1) offsets[E] = excl + mine;
  if (w == 0) {  // smallest out-of-range pair id over the chunks, one wavefront
    int b = 0x7fffffff;
    for (int c = lane; c < nchunks; c += 64) b = min(b, chunk_bad[c]);
    for (int d = 32; d > 0; d >>= 1) b = min(b, __shfl_xor(b, d, 64));
    if (lane == 0) status[0] = b == 0x7fffffff ? 0 : b + 1;
  }
}

__global__ void __launch_bounds__(kThreads) route_scatter(const int32_t* __restrict__ ids, int P, int E, int ebits,
                                                          const int32_t* __restrict__ chunk_base,
                                                          int32_t* __restrict__ sorted_pair,
                                                          int32_t* __restrict__ inv,
                                                          RowMeta rm) {
  __shared__ int32_t base[kMaxE];
  __shared__ int32_t wcnt[kThreads / 64][kMaxE];
  const int c = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int e = tid; e < E; e += kThreads) base[e] = chunk_base[(int64_t)c * E + e];
  const int p0 = c * kRouteChunk;
  const int p1 = min(P, p0 + kRouteChunk);
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  for (int s = p0; s < p1; s += kThreads) {
    for (int e = tid; e < E; e += kThreads)
      for (int i = 0; i < kThreads / 64; ++i) wcnt[i][e] = 0;
    __syncthreads();
    const int p = s + tid;
    int e = -1;
    if (p < p1) {
      e = ids[p];
      if (e < 0 || e >= E) e = -1;
    }
    // lanes holding the same valid expert id
    uint64_t same = __ballot(e >= 0);
    for (int b = 0; b < ebits; ++b) {
      const bool bit = e >= 0 && ((e >> b) & 1);
      const uint64_t m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    if (e < 0) same = 0;
    const int rank = __popcll(same & below);
    if (e >= 0 && rank == 0) wcnt[w][e] = __popcll(same);
    __syncthreads();
    if (e >= 0) {
      int pos = base[e] + rank;
      for (int i = 0; i < w; ++i) pos += wcnt[i][e];
      sorted_pair[pos] = p;
      inv[p] = pos;
      if (rm.rtok) {
        const int t = p / rm.k, sl = p - t * rm.k;
        rm.rtok[pos] = t;
        rm.rslot[pos] = t * (rm.k + rm.n_sh) + sl;
        rm.rgw[pos] = rm.topk_w[p];
      }
    } else if (p < p1) {
      inv[p] = -1;
    }
    __syncthreads();
    for (int ee = tid; ee < E; ee += kThreads) {
      int add = 0;
      for (int i = 0; i < kThreads / 64; ++i) add += wcnt[i][ee];
      base[ee] += add;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------- router front-end
// Eq. (2) weights its experts by the router's softmax.  One wavefront per
// token; lane l holds the logits of experts l, l + 64, ... in registers.  The
// k largest are found in k rounds of a wavefront arg-max under the strict
// order (larger logit, then lower id), which all lanes agree on, so the
// result is unique and every lane of the butterfly ends with the same value.
constexpr int kRouterJ = kMaxE / 64;

__device__ inline bool router_better(float va, int ea, float vb, int eb) {
  return va > vb || (va == vb && ea < eb);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int d = 32; d; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

struct RouterArgs {
  const float* logits;  // [T, E]
  int k, renorm;
  const float* shared_logits;  // [T, n_sh] or null
  int n_sh;
  int32_t* ids;  // [T, k]
  float* w;      // [T, k]
  float* shared_w;
};

// Token t by the calling wavefront.
__device__ void router_token_wave(const RouterArgs& ra, int t, int E, int lane) {
  const float* __restrict__ logits = ra.logits;
  const int k = ra.k, renorm = ra.renorm, n_sh = ra.n_sh;
  const float* __restrict__ shared_logits = ra.shared_logits;
  int32_t* __restrict__ ids = ra.ids;
  float* __restrict__ w = ra.w;
  float* __restrict__ shared_w = ra.shared_w;
  const float* row = logits + (int64_t)t * E;
  const int J = (E + 63) >> 6;
  float v[kRouterJ];
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < kRouterJ; ++j) {
    const int e = lane + 64 * j;
    v[j] = (j < J && e < E) ? row[e] : -INFINITY;
    m = fmaxf(m, v[j]);
  }
#pragma unroll
  for (int d = 32; d; d >>= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
  float se = 0.f;
#pragma unroll
  for (int j = 0; j < kRouterJ; ++j)
    if (j < J && lane + 64 * j < E) se += expf(v[j] - m);
  se = wave_sum(se);

  uint32_t taken = 0;  // bit j: this lane's v[j] is chosen
  int my_e = -1;
  float my_v = -INFINITY;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int be = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < kRouterJ; ++j) {
      const int e = lane + 64 * j;
      if (j < J && e < E && !((taken >> j) & 1u) && router_better(v[j], e, bv, be)) {
        bv = v[j];
        be = e;
      }
    }
#pragma unroll
    for (int d = 32; d; d >>= 1) {
      const float ov = __shfl_xor(bv, d, 64);
      const int oe = __shfl_xor(be, d, 64);
      if (router_better(ov, oe, bv, be)) {
        bv = ov;
        be = oe;
      }
    }
    if (be != 0x7fffffff && (be & 63) == lane) taken |= 1u << (be >> 6);
    if (lane == r) {
      my_e = be == 0x7fffffff ? -1 : be;
      my_v = bv;
    }
  }
  const float q = (lane < k && my_e >= 0) ? expf(my_v - m) : 0.f;
  const float den = renorm ? wave_sum(q) : se;
  if (lane < k) {
    ids[(int64_t)t * k + lane] = my_e;
    w[(int64_t)t * k + lane] = q / den;
  }
  if (shared_logits && lane < n_sh)
    shared_w[(int64_t)t * n_sh + lane] = 1.f / (1.f + expf(-shared_logits[(int64_t)t * n_sh + lane]));
}

// Token t by a group of 8 lanes (E <= 64, k <= 8): lane j of the group holds
// experts j, j + 8, ..., j + 56.  Each lane keeps its best k entries sorted;
// three butterfly steps (partner lane^1, ^2, ^4) merge two sorted lists into
// the best k of their union (a bitonic merge), so that every lane ends with
// the token's k best, sorted.  The maximum and the sum of exp(v - max) take
// the same butterfly, after the lane's own 8 values in expert order.  The
// best k under the strict order are unique, so the ids equal those of the
// wavefront form; the weights differ from it only in the order of the sum.
constexpr int kGroupMaxE = 64;
constexpr int kGroupMaxK = 8;
__host__ __device__ constexpr bool router_by_group(int E, int k) { return E <= kGroupMaxE && k <= kGroupMaxK; }

// the strict order without short-circuit evaluation, so that the compare-
// exchanges below compile to selects rather than branches
__device__ inline bool router_better_sel(float va, int ea, float vb, int eb) {
  return (va > vb) | ((va == vb) & (ea < eb));
}
__device__ inline void router_cmpx(float& va, int& ea, float& vb, int& eb) {  // (a, b) -> (better, worse)
  const bool sw = router_better_sel(vb, eb, va, ea);
  const float xa = sw ? vb : va, xb = sw ? va : vb;
  const int ya = sw ? eb : ea, yb = sw ? ea : eb;
  va = xa;
  vb = xb;
  ea = ya;
  eb = yb;
}

__device__ void router_token_group(const RouterArgs& ra, int t, bool live, int E, int j) {
  constexpr int K = kGroupMaxK;
  const float* row = ra.logits + (int64_t)(live ? t : 0) * E;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (live && j + 8 * i < E) ? row[j + 8 * i] : -INFINITY;
  const float shl = (live && ra.shared_logits && j < ra.n_sh) ? ra.shared_logits[(int64_t)t * ra.n_sh + j] : 0.f;
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = fmaxf(m, v[i]);
#pragma unroll
  for (int d = 1; d < 8; d <<= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
  float se = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
    if (j + 8 * i < E) se += expf(v[i] - m);
#pragma unroll
  for (int d = 1; d < 8; d <<= 1) se += __shfl_xor(se, d, 64);
  // the lane's own list: its 8 entries sorted by a bitonic network, past-E
  // entries and NaNs replaced by the sentinel (-inf, max int), which every
  // real entry beats (a NaN is never chosen)
  float tv[K];
  int te[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const bool ok = (j + 8 * i < E) & (v[i] == v[i]);
    tv[i] = ok ? v[i] : -INFINITY;
    te[i] = ok ? j + 8 * i : 0x7fffffff;
  }
#pragma unroll
  for (int kk = 2; kk <= K; kk <<= 1)
#pragma unroll
    for (int jj = kk >> 1; jj > 0; jj >>= 1)
#pragma unroll
      for (int i = 0; i < K; ++i) {
        const int l = i ^ jj;
        if (l > i) {
          if ((i & kk) == 0)
            router_cmpx(tv[i], te[i], tv[l], te[l]);  // better first
          else
            router_cmpx(tv[l], te[l], tv[i], te[i]);
        }
      }
  // butterfly merges
#pragma unroll
  for (int d = 1; d < 8; d <<= 1) {
    float ov[K];
    int oe[K];
#pragma unroll
    for (int r = 0; r < K; ++r) {
      ov[r] = __shfl_xor(tv[r], d, 64);
      oe[r] = __shfl_xor(te[r], d, 64);
    }
    // the better of tv[r] and ov[K-1-r]: the best K of the union, bitonic
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const bool b = router_better_sel(ov[K - 1 - r], oe[K - 1 - r], tv[r], te[r]);
      tv[r] = b ? ov[K - 1 - r] : tv[r];
      te[r] = b ? oe[K - 1 - r] : te[r];
    }
    // sort the bitonic sequence: half-cleaners of span 4, 2, 1
#pragma unroll
    for (int h = K / 2; h > 0; h >>= 1)
#pragma unroll
      for (int r = 0; r < K; ++r)
        if ((r & h) == 0) router_cmpx(tv[r], te[r], tv[r + h], te[r + h]);
  }
  if (!live) return;
  const int k = ra.k;
  float q = 0.f, den = 0.f;
  int my_e = -1;
#pragma unroll
  for (int r = 0; r < K; ++r) {
    const float qr = (r < k && te[r] != 0x7fffffff) ? expf(tv[r] - m) : 0.f;
    if (r < k) den += qr;
    if (r == j) {
      q = qr;
      my_e = te[r] == 0x7fffffff ? -1 : te[r];
    }
  }
  if (!ra.renorm) den = se;
  if (j < k) {
    ra.ids[(int64_t)t * k + j] = my_e;
    ra.w[(int64_t)t * k + j] = q / den;
  }
  if (ra.shared_logits)
    for (int s2 = j; s2 < ra.n_sh; s2 += 8)
      ra.shared_w[(int64_t)t * ra.n_sh + s2] =
          1.f / (1.f + expf(-(s2 == j ? shl : ra.shared_logits[(int64_t)t * ra.n_sh + s2])));
}

// One wavefront per token, or 8 tokens per wavefront where router_by_group
// (the launcher sizes the grid to match).
__global__ void __launch_bounds__(kThreads) router_topk_kernel(RouterArgs ra, int T, int E) {
  if (router_by_group(E, ra.k)) {
    const int t = blockIdx.x * (kThreads / 8) + (threadIdx.x >> 3);
    router_token_group(ra, t, t < T, E, threadIdx.x & 7);  // every lane takes part in the shuffles
    return;
  }
  const int t = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (t >= T) return;  // a whole wavefront leaves together
  router_token_wave(ra, t, E, threadIdx.x & 63);
}

// Batches of at most kRouteSmall pairs: the three steps in one workgroup of
// 1024 threads, with barriers where the launches were.  The pairs are ranked
// 1024 at a time by the same ballots; positions follow from the expert's base,
// the counts of earlier wavefronts of the step and the rank in the wavefront,
// so the order (expert, then pair id) is the one the chunked launches give.
constexpr int kRouteSmall = 4096;  // one step costs ~1 us: past 4096 pairs the chunked launches win
constexpr int kSmallThreads = 1024;
// With ra.logits set (and router_by_group(E, k)) the workgroup first runs the
// router front-end for the T = P / k tokens, 8 lanes per token, and routes the
// ids it wrote (ids == ra.ids; the barrier makes them visible to the
// workgroup).
__global__ void __launch_bounds__(kSmallThreads) route_small(const int32_t* ids, int P, int E, int ebits,
                                                             int32_t* __restrict__ counts,
                                                             int32_t* __restrict__ offsets,
                                                             int32_t* __restrict__ sorted_pair,
                                                             int32_t* __restrict__ inv, int32_t* __restrict__ status,
                                                             RouterArgs ra, RowMeta rm) {
  constexpr int NW = kSmallThreads / 64;
  __shared__ int32_t base[kMaxE];
  __shared__ int32_t wcnt[NW][kMaxE];
  __shared__ int32_t wsum[NW];
  __shared__ int32_t bad;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (ra.logits) {
    const int T = P / ra.k;
    for (int t0 = 0; t0 < T; t0 += kSmallThreads / 8) {  // uniform trip count: every lane shuffles
      const int t = t0 + (tid >> 3);
      router_token_group(ra, t, t < T, E, tid & 7);
    }
    __syncthreads();
  }
  for (int e = tid; e < E; e += kSmallThreads) base[e] = 0;
  if (tid == 0) bad = 0x7fffffff;
  __syncthreads();
  // 1. histogram (LDS atomics: the counts do not depend on their order)
  for (int p = tid; p < P; p += kSmallThreads) {
    const int e = ids[p];
    if (e >= 0 && e < E) atomicAdd(&base[e], 1);
    else atomicMin(&bad, p);
  }
  __syncthreads();
  // 2. exclusive scan of the counts (E <= 1024: one expert per thread)
  const int mine = tid < E ? base[tid] : 0;
  int incl = mine;
  for (int d = 1; d < 64; d <<= 1) {
    const int v = __shfl_up(incl, d, 64);
    if (lane >= d) incl += v;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int excl = incl - mine;
  for (int i = 0; i < w; ++i) excl += wsum[i];
  if (tid < E) {
    counts[tid] = mine;
    offsets[tid] = excl;
    base[tid] = excl;  // only this thread read base[tid]
  }
  if (tid == E - 1) offsets[E] = excl + mine;
  if (tid == 0) status[0] = bad == 0x7fffffff ? 0 : bad + 1;
  // 3. scatter, 1024 pairs per step
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  for (int s = 0; s < P; s += kSmallThreads) {
    for (int e = tid; e < E; e += kSmallThreads)
#pragma unroll
      for (int i = 0; i < NW; ++i) wcnt[i][e] = 0;
    __syncthreads();
    const int p = s + tid;
    int e = -1;
    if (p < P) {
      e = ids[p];
      if (e < 0 || e >= E) e = -1;
    }
    uint64_t same = __ballot(e >= 0);
    for (int b = 0; b < ebits; ++b) {
      const bool bit = e >= 0 && ((e >> b) & 1);
      const uint64_t m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    if (e < 0) same = 0;
    const int rank = __popcll(same & below);
    if (e >= 0 && rank == 0) wcnt[w][e] = __popcll(same);
    __syncthreads();
    if (e >= 0) {
      int pos = base[e] + rank;
      for (int i = 0; i < w; ++i) pos += wcnt[i][e];
      sorted_pair[pos] = p;
      inv[p] = pos;
      if (rm.rtok) {
        const int t = p / rm.k, sl = p - t * rm.k;
        rm.rtok[pos] = t;
        rm.rslot[pos] = t * (rm.k + rm.n_sh) + sl;
        rm.rgw[pos] = rm.topk_w[p];
      }
    } else if (p < P) {
      inv[p] = -1;
    }
    __syncthreads();
    for (int ee = tid; ee < E; ee += kSmallThreads) {
      int add = 0;
#pragma unroll
      for (int i = 0; i < NW; ++i) add += wcnt[i][ee];
      base[ee] += add;
    }
    // (no barrier here: thread t alone updates base[t], t + 1024, ... and
    // clears the same columns of wcnt at the next step, whose first barrier
    // orders both before any other thread reads them)
  }
}

}  // namespace

hipError_t launch_router_topk(const float* logits, int T, int E, int k, int renorm, const float* shared_logits,
                              int n_sh, int32_t* ids, float* w, float* shared_w, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int per = router_by_group(E, k) ? kThreads / 8 : kThreads / 64;
  const RouterArgs ra{logits, k, renorm, shared_logits, n_sh, ids, w, shared_w};
  hipLaunchKernelGGL(router_topk_kernel, dim3((T + per - 1) / per), dim3(kThreads), 0, s, ra, T, E);
  return hipGetLastError();
}

hipError_t launch_router_route(const float* logits, int T, int E, int k, int renorm, const float* shared_logits,
                               int n_sh, int32_t* ids, float* w, float* shared_w, int32_t* counts,
                               int32_t* offsets, int32_t* sorted_pair, int32_t* inv, int32_t* status,
                               int32_t* chunk_counts, int32_t* chunk_bad, const RowMeta* rm, hipStream_t s) {
  const int P = T * k;
  RowMeta rmv;
  memset(&rmv, 0, sizeof(rmv));
  if (rm) rmv = *rm;
  rmv.k = k;
  rmv.topk_w = w;
  if (P > 0 && P <= kRouteSmall && router_by_group(E, k)) {
    int ebits = 0;
    while ((1 << ebits) < E) ++ebits;
    const RouterArgs ra{logits, k, renorm, shared_logits, n_sh, ids, w, shared_w};
    hipLaunchKernelGGL(route_small, dim3(1), dim3(kSmallThreads), 0, s, ids, P, E, ebits, counts, offsets,
                       sorted_pair, inv, status, ra, rmv);
    return hipGetLastError();
  }
  hipError_t e = launch_router_topk(logits, T, E, k, renorm, shared_logits, n_sh, ids, w, shared_w, s);
  if (e != hipSuccess) return e;
  return launch_route(ids, T, k, E, counts, offsets, sorted_pair, inv, status, chunk_counts, chunk_bad, &rmv, s);
}

hipError_t launch_route(const int32_t* ids, int T, int k, int E, int32_t* counts, int32_t* offsets,
                        int32_t* sorted_pair, int32_t* inv, int32_t* status, int32_t* chunk_counts,
                        int32_t* chunk_bad, const RowMeta* rm, hipStream_t s) {
  const int P = T * k;
  RowMeta rmv;
  memset(&rmv, 0, sizeof(rmv));
  if (rm) rmv = *rm;
  rmv.k = k;
  const int nchunks = (P + kRouteChunk - 1) / kRouteChunk;
  int ebits = 0;
  while ((1 << ebits) < E) ++ebits;
  if (P <= kRouteSmall) {
    RouterArgs none;
    memset(&none, 0, sizeof(none));
    hipLaunchKernelGGL(route_small, dim3(1), dim3(kSmallThreads), 0, s, ids, P, E, ebits, counts, offsets,
                       sorted_pair, inv, status, none, rmv);
    return hipGetLastError();
  }
  if (nchunks > 0) {
    hipLaunchKernelGGL(route_count, dim3(nchunks), dim3(kThreads), 0, s, ids, P, E, chunk_counts, chunk_bad);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(route_scan, dim3(1), dim3(1024), 0, s, nchunks, E, chunk_counts, chunk_bad, counts,
                     offsets, status);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || nchunks == 0) return err;
  hipLaunchKernelGGL(route_scatter, dim3(nchunks), dim3(kThreads), 0, s, ids, P, E, ebits, chunk_counts,
                     sorted_pair, inv, rmv);
  return hipGetLastError();
}

}  // namespace mxmoe
