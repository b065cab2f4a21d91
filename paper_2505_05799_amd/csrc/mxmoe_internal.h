// Internal declarations shared by the HIP translation units of libmxmoe.
// Device layouts of the block table, the tile plan and the packed weights.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

#include "../../include/mxmoe.h"

namespace mxmoe {

// ---------------------------------------------------------------- schemes
// Kind ids of the micro-kernels (one per supported scheme).
enum Kind : int32_t {
  K_W16 = 0,   // 16-bit weights, 16-bit MFMA
  K_W8A8 = 1,  // int8 x int8 MFMA, per-channel / per-token scales
  K_W4A4 = 2,  // int4 codes widened to int8 (x16) on the fly, int8 MFMA
  K_W2G = 3,   // weight-only 2-bit, group 128
  K_W3G = 4,   // weight-only 3-bit (2+1 bit planes), group 128
  K_W4G = 5,   // weight-only 4-bit, group 128
  K_W8G = 6,   // weight-only 8-bit, group 128
  K_W4A4G = 7, // int4 weights and activations with per-128-group scales (w4a4-g128)
  K_MXFP4 = 8, // FP4 e2m1 weights and activations with E8M0 scales per 32 (scaled FP4 MFMA)
  K_F8A8 = 9,  // FP8 e4m3 weights (per-channel fp32 scale) and activations (per-token), FP8 MFMA
  K_W4A4F6 = 10,  // w4a4 (per channel / per token) with the int4 codes as FP6 e2m3 operands, FP6 MFMA
  K_COUNT = 11
};

// kinds whose activations arrive as one byte per element with a per-token
// (or per-group) fp32 scale and whose weights carry fp32 channel scales: the
// integer kinds and FP8, which shares their layouts
__host__ __device__ constexpr inline bool kind_is_int(int kd) {
  return kd == K_W8A8 || kd == K_W4A4 || kd == K_W4A4G || kd == K_F8A8 || kd == K_W4A4F6;
}
__host__ __device__ constexpr inline bool kind_is_f8(int kd) { return kd == K_F8A8; }
// w4a4 on FP6 operands: every int4 code in [-7, 7] is an e2m3 value, products
// are integers up to 49 and a 128-wide k block sums to at most 6272 in
// magnitude, so the FP6 MFMA's fp32 results are the exact integer sums.
// Activations: per 32 consecutive elements 24 bytes of 6-bit codes (element i
// at bits 6i..6i+5) and 8 zero bytes, one byte per element like int8 codes.
__host__ __device__ constexpr inline bool kind_is_f6(int kd) { return kd == K_W4A4F6; }
__host__ __device__ constexpr inline bool kind_is_wonly(int kd) { return kd >= K_W2G && kd <= K_W8G; }
// kinds whose scales come per 128-wide group along K (a 64-byte metadata tail
// per fragment block): the weight-only kinds and w4a4-g128
__host__ __device__ constexpr inline bool kind_has_gmeta(int kd) {
  return kind_is_wonly(kd) || kd == K_W4A4G || kd == K_MXFP4;
}
__host__ __device__ constexpr inline bool kind_is_mx(int kd) { return kd == K_MXFP4; }
// activations of the kind arrive quantized (integer codes or MX elements)
__host__ __device__ constexpr inline bool kind_quant_act(int kd) { return kind_is_int(kd) || kind_is_mx(kd); }
__host__ __device__ constexpr inline int kind_wbits(int kd) {
  switch (kd) {
    case K_W16: return 16;
    case K_W8A8: return 8;
    case K_F8A8: return 8;
    case K_W4A4F6: return 6;  // stored bits (4-bit codes held as e2m3)
    case K_W4A4: return 4;
    case K_W4A4G: return 4;
    case K_MXFP4: return 4;
    case K_W2G: return 2;
    case K_W3G: return 3;
    case K_W4G: return 4;
    default: return 8;
  }
}
// activation qmax of an integer scheme (0 for 16-bit activations)
// 2/3/4-bit group-wise kinds: dequantized through a bias whose product with
// the activations is removed through activation row sums (16-bit bf16 path)
__host__ __device__ constexpr inline bool kind_is_magic(int kd) { return kd == K_W2G || kd == K_W3G || kd == K_W4G; }
// FP8 activations are scaled so that the row maximum lands on 448, the
// largest finite e4m3 value, which takes the place of qmax in the recipe
constexpr int kQmaxF8 = 448;
__host__ __device__ constexpr inline int kind_qmax(int kd) {
  return kd == K_W8A8 ? 127 : ((kd == K_W4A4 || kd == K_W4A4G || kd == K_W4A4F6) ? 7 : (kd == K_F8A8 ? kQmaxF8 : 0));
}

// Packed layout: the weight matrix [n, k] is cut into fragment blocks of
// 16 output rows x 128 reduction columns, stored n-block major, k-block minor.
// A block holds 64 lanes x lane_bytes(kind) bytes in MFMA lane order (lane l
// owns output row l%16 and reduction quarter l/16); blocks of the group-scaled
// kinds are followed by 16 (scale, zero) fp16 pairs, one per output row of the
// block (zero 0 for w4a4-g128).  Per-channel fp32 scales of w8a8/w4a4 follow
// the last block.
__host__ __device__ constexpr inline int lane_bytes(int kd) {
  switch (kd) {
    case K_W16: return 64;
    case K_W8A8: return 32;
    case K_F8A8: return 32;
    case K_W4A4F6: return 24;  // 32 e2m3 codes
    case K_W4A4: return 16;
    case K_W4A4G: return 16;
    case K_MXFP4: return 16;
    case K_W2G: return 8;
    case K_W3G: return 12;
    case K_W4G: return 16;
    default: return 32;  // K_W8G
  }
}
__host__ __device__ constexpr inline int block_bytes(int kd) {
  return 64 * lane_bytes(kd) + (kind_has_gmeta(kd) ? 64 : 0);
}
__host__ __device__ inline int64_t codes_bytes(int kd, int n, int k) {
  return (int64_t)(n / 16) * (k / 128) * block_bytes(kd);
}

// ------------------------------------------------------------ block table
struct DevLinear {
  const uint8_t* packed;  // fragment blocks
  const float* wscale;    // per-channel scales (w8a8/w4a4) or nullptr
  int32_t n, k;
  int32_t kind;
  int32_t pad;
};
static_assert(sizeof(DevLinear) == 32, "DevLinear layout");

struct DevExpert {
  DevLinear lin[3];  // gate, up, down
};

struct DevHeader {
  int32_t hidden, ffn, E, topk, n_shared, ffn_shared, act, G;  // G = E + n_shared
};

// ------------------------------------------------------------- tile plan
// Tile configurations of the persistent Group-GEMM (16, 32, 64, 128 rows).
// All use 256 threads (4 wavefronts stacked along the output channels).
enum Cfg : int32_t { CFG_S = 0, CFG_T = 1, CFG_M = 2, CFG_L = 3, CFG_COUNT = 4 };

// Plan record per (phase, expert): int32 fields.  A group of mt x nt output
// tiles whose reduction is sliced S ways (split-K, the paper's slice-K tile
// parameter) is queued as mt x (S nt) tiles: channel tile index n' = s nt + n.
// Every slice writes its partial sums to the partial buffer (floats from
// PF_PBASE, BM x BN x linears per slice) and bumps the output tile's counter
// (PF_CBASE + tile); the last slice to arrive adds the partials in slice order
// and runs the epilogue.
enum PlanField : int32_t {
  PF_EXPERT = 0, PF_M = 1, PF_CFG = 2, PF_MTILES = 3, PF_NTILES = 4,
  PF_START = 5, PF_COST = 6, PF_RANK = 7, PF_SPLIT = 8, PF_PBASE = 9, PF_CBASE = 10, PF_N = 12
};
// Split-K budgets per phase: at most kSplitExtra tiles added by slicing (and
// as many output-tile counters); the partial buffer size comes from the host.
constexpr int kSplitExtra = 16384;
constexpr int kSplitMax = 8;

// Limits of a block: routed experts, shared experts, groups (routed + shared).
constexpr int kMaxE = 1024;
constexpr int kMaxShared = 64;
constexpr int kMaxG = 2048;

// Tiles are grouped into super-tiles of up to 64 tiles sharing row and channel
// blocks (min(mt, 8) x min(nt, 64 / that) tiles) and dealt round-robin to one
// queue per XCD, in decreasing tile-cost order of their groups; each queue is
// drained first by the workgroups resident on that XCD (L2 reuse of the shared
// weights and activation rows), then by any workgroup.
constexpr int kXcd = 8;
constexpr int kSuperTiles = 64;

// Plan region layout (int32), phases p = 0 (gate|up, or the single linear)
// and 1 (down):
//   rec   [2][G][PF_N]        group records
//   order [2][G]              group index per rank (-1 past the last group with tiles)
//   ent   [2][kXcd][cap][3]   queue entries: group, super-tile index, first tile
//   ctr   [2][kXcd][4]        per queue: head, total tiles, entries, -
//   misc  [16]                [2 + p]: number of groups with tiles in phase p,
//                             [4]: 1 if a queue overflowed its capacity,
//                             [6 + p]: partial-buffer floats used in phase p,
//                             [8]: workgroups the slicing threshold assumes
//   flat  [2][kXcd][fcap][4]  the queues expanded to one entry per tile
//   cnt   [2][kSplitExtra]    arrival counters of sliced output tiles
struct PlanLayout { int64_t rec, order, ent, ctr, misc, flat, cnt, total; };
__host__ __device__ inline PlanLayout plan_layout(int G, int cap, int fcap) {
  PlanLayout L;
  L.rec = 0;
  L.order = L.rec + 2LL * G * PF_N;
  L.ent = L.order + 2LL * G;
  L.ent = (L.ent + 3) & ~3LL;
  L.ctr = L.ent + 2LL * kXcd * cap * 3;
  L.misc = L.ctr + 2LL * kXcd * 4;
  L.flat = L.misc + 16;
  L.cnt = L.flat + 2LL * kXcd * fcap * 4;
  L.total = L.cnt + 2LL * kSplitExtra;
  return L;
}
// Per-queue capacity bound from the rows and channel counts (host side):
// super-tiles of a group <= (mt/8 + 1)(nt/8 + 1) with mt <= m/1024*8 + 1,
// nt <= N/64 + 1 (smallest tiles are 16 x 64 per linear), plus the super-tiles
// that slicing adds (at most one per added tile, dealt round-robin).
__host__ __device__ inline int plan_queue_cap(int64_t rows_total, int groups, int n_max) {
  const int64_t s = (rows_total / 1024 + 2LL * groups + 1) * ((int64_t)n_max / 512 + 2);
  return (int)(s / kXcd + 2 + kSplitExtra / kXcd + 1);
}
// Per-queue tile capacity: at most 64 tiles per unsliced queue entry, plus
// every tile that slicing adds.
__host__ __device__ inline int plan_flat_cap(int qcap) {
  return (qcap - kSplitExtra / kXcd - 1) * kSuperTiles + kSplitExtra;
}

// One tile of a queue, as the Group-GEMM pops it (int32 x 4):
//   [0] group | cfg << 16 | kind << 20 | (slices - 1) << 24
//   [1] row tile | channel tile n' << 16 (n' = slice * channel tiles + channel tile)
//   [2] first sorted row of the group (0 for shared experts and single linears)
//   [3] rows of the group
__host__ __device__ inline int32_t tile_word0(int g, int cfg, int kind, int split) {
  return g | (cfg << 16) | (kind << 20) | ((split - 1) << 24);
}
// Tile cost of the run-time plan: the paper's per-tile cost c_t, profiled
// ahead of time per tile configuration (Sec. 4.2.2), held as a table of four
// integers in ps per (phase, kind, configuration):
//   a   fixed cost of a tile (prologue, epilogue, queue pop; a fit's
//       intercept, so it may be negative)
//   bs  cost per 128-wide k block that no other tile shares (MFMA issue,
//       activation streaming)
//   bu  cost per k block of streaming the tile's weights; the group's mt row
//       tiles share each weight tile through L2, so a tile is charged bu / mt
//   h   hand-off cost of a sliced tile (partial sums written, then read back)
// A tile of kb k blocks (its slice's share when sliced) costs
//   c = a + kb * bs + floor(kb * bu / mt) + (slices > 1 ? h : 0)
// in exact integer arithmetic, clamped to [1, 2e9].  Phase 1 also serves the
// single-linear plan.  The table comes from the caller (mxmoe_set_tile_costs)
// or is the roofline default below.
constexpr int kCostCfgs = 4;
constexpr int kCostVals = 4;
constexpr int kCostEntries = 2 * K_COUNT * kCostCfgs * kCostVals;
struct TileCosts {
  int32_t v[kCostEntries];
};
__host__ __device__ constexpr inline int cost_index(int ph, int kd, int cfg) {
  return ((ph * K_COUNT + kd) * kCostCfgs + cfg) * kCostVals;
}
constexpr int64_t kCostMaxPs = 2000000000LL;
__host__ __device__ inline int32_t tile_cost(const int32_t* e, int kb, int split, int mt) {
  const int64_t wu = (int64_t)kb * e[2];  // >= 0; a 32-bit quotient where it fits
  const uint32_t d = mt > 0 ? (uint32_t)mt : 1u;
  const int64_t shared = wu < (1LL << 32) ? (int64_t)((uint32_t)wu / d) : wu / d;
  int64_t c = (int64_t)e[0] + (int64_t)kb * e[1] + shared + (split > 1 ? e[3] : 0);
  c = c < 1 ? 1 : (c > kCostMaxPs ? kCostMaxPs : c);
  return (int32_t)c;
}
// Slices of a group (split-K, the paper's slice-K tile parameter): the fewest
// slices whose tile cost is at most theta, with at least kSplitMinKb k blocks
// per slice and at most kSplitMax slices; if none is, the slice count of the
// cheapest tile (the fewest slices among equals).  theta is half of the
// phase's mean work per workgroup (unsliced tile costs summed over all tiles,
// over the grid), so that no tile is long next to the schedule it is part of.
// At a quarter of the mean work, or with 4 k blocks per slice, the launches
// measured slower (DeepSeek-V2-Lite-shaped forward 8% and Qwen1.5-MoE-shaped
// 12% slower).
constexpr int kSplitShare = 2;
constexpr int kSplitMinKb = 6;

// Workspace layout (byte offsets), shared by host code of the forward.
struct WsLayout {
  size_t status, counts, offsets, sorted_pair, inv, chunk_counts, chunk_bad, plan, down_qmax;
  size_t rtok, rslot, rgw, rxs8, rxs4;
  size_t xq8, xs8, xq4, xs4, h, h_shared, hq, hs, hq_shared, hs_shared, slots, total;
  size_t partial;  // fp32 split-K partial sums (both phases reuse it)
  size_t rsx, rsh, rsh_shared;  // fp32 row sums per 128-wide k block of x, h, h_shared
  size_t xq4g, xs4g, hsg, hsg_shared;  // w4a4-g128 codes and group scales
  size_t rids, rw, shw;  // router front-end outputs: ids, gate weights, shared-expert gates
  size_t xqmx, xsmx, hqmx, hsmx, hqmx_shared, hsmx_shared;  // mxfp4 activation codes and E8M0 bytes
  size_t xqf8, xsf8;  // FP8 e4m3 codes and per-token scales of x
  size_t xqf6, xsf6;  // FP6-encoded int4 codes and per-token scales of x
  int qcap;  // XCD queue capacity of the tile plan (super-tiles)
  int fcap;  // XCD queue capacity of the tile plan (tiles)
  int64_t pfloats;  // size of the partial buffer
};

constexpr int kRouteChunk = 512;  // pairs per routing workgroup
constexpr size_t kNone = (size_t)-1;

// ----------------------------------------------------------- launchers
// (defined in the .hip files; all return hipError_t of the launch)
hipError_t launch_pack(int kind, int n, int k, int act, int w16_src, const void* codes,
                       const void* scales, const void* zeros, uint8_t* packed, hipStream_t s);
hipError_t launch_unpack(int kind, int n, int k, int act, const uint8_t* packed, void* codes,
                         void* scales, void* zeros, hipStream_t s);

// Per sorted row j of the routed groups, written by the routing launch that
// places the pair p = sorted_pair[j] (token t = p / k, slot p % k): rtok[j] =
// t, rslot[j] = t * (k + n_sh) + p % k (its row of the down-projection slots),
// rgw[j] = topk_w[p].  The per-token activation scales of the row follow from
// the x encodings (XPrep::inv).
struct RowMeta {
  int k, n_sh;
  const float* topk_w;
  int32_t* rtok;
  int32_t* rslot;
  float* rgw;
};
// rm may be null (routing arrays only).
hipError_t launch_route(const int32_t* ids, int T, int k, int E, int32_t* counts,
                        int32_t* offsets, int32_t* sorted_pair, int32_t* inv, int32_t* status,
                        int32_t* chunk_counts, int32_t* chunk_bad, const RowMeta* rm, hipStream_t s);
// Router front-end, one wavefront per token: softmax top-k of fp32 logits
// [T,E] (E <= 1024, k <= 64) and, if shared_logits, sigmoid gates [T,n_sh].
constexpr int kRouterMaxK = 64;
hipError_t launch_router_topk(const float* logits, int T, int E, int k, int renorm, const float* shared_logits,
                              int n_sh, int32_t* ids, float* w, float* shared_w, hipStream_t s);
// The router front-end followed by routing of the ids it writes: one launch
// where the batch fits the one-workgroup routing kernel (E <= 64, k <= 8),
// else the two calls above.  Results equal those of the two calls.
// (rm->topk_w is ignored: the rows take the router's weights w.)
hipError_t launch_router_route(const float* logits, int T, int E, int k, int renorm, const float* shared_logits,
                               int n_sh, int32_t* ids, float* w, float* shared_w, int32_t* counts,
                               int32_t* offsets, int32_t* sorted_pair, int32_t* inv, int32_t* status,
                               int32_t* chunk_counts, int32_t* chunk_bad, const RowMeta* rm, hipStream_t s);

// Row sums of each 128-wide block of bf16 rows: out[r][b] = sum of a[r][128b ..
// 128b + 127] in fp32; cols a multiple of 128, rows 16-byte aligned.
hipError_t launch_rowsum(const void* a, int rows, int cols, int64_t ld, float* out, hipStream_t s);
// Per-(row, 128-wide block) quantization (w4a4-g128 activations): codes int8
// [rows, cols], scales fp32 [rows][cols/128]; cols a multiple of 128.
hipError_t launch_act_quant_g128(const void* a, int act, int rows, int cols, int64_t ld, int qmax, int8_t* codes,
                                 float* scales, hipStream_t s);
hipError_t launch_act_quant(const void* a, int act, int rows, int cols, int64_t ld, int qmax,
                            int8_t* codes, float* scales, hipStream_t s);

// Per sorted row j < offsets[E] (pair p = sorted_pair[j], token t = p / k,
// slot s = p % k): rtok[j] = t, rslot[j] = t (k + n_sh) + s, rgw[j] = topk_w[p],
// and rxs8[j] / rxs4[j] = the token's activation scale where those exist.


// Quantize routed h rows whose expert's down projection is a8/a4 (qmax from
// down_qmax[expert]); rows of other experts are skipped.
// Routed h rows of the experts whose down linear quantizes its activations:
// down_qmax[e] = qmax | kDownQGroup for per-128-group scales (into hsg
// [P][F/128]), else per-row scales (into hs); 0 = not quantized.
constexpr int kDownQGroup = 0x100;
constexpr int kDownQMX = 0x200;  // MXFP4 codes into hqmx [P][F/2], E8M0 bytes into hsmx [P][F/32]
constexpr int kDownQF8 = 0x400;  // FP8 e4m3 codes into hq, per-row scales into hs
constexpr int kDownQF6 = 0x800;  // int4 codes as FP6 e2m3 (32 per 24 + 8 zero bytes) into hq, scales into hs
hipError_t launch_hquant_routed(const void* h, int act, int P, int F, const int32_t* offsets,
                                int E, const int32_t* down_qmax, int8_t* hq, float* hs, float* hsg,
                                uint8_t* hqmx, uint8_t* hsmx, hipStream_t s);
// MXFP4 encoding of rows (cols a multiple of 128): codes [rows][cols/2] (two
// e2m1 nibbles a byte, element order), E8M0 bytes [rows][cols/32].
hipError_t launch_act_quant_mx(const void* a, int act, int rows, int cols, int64_t ld, uint8_t* codes, uint8_t* exps,
                               hipStream_t s);
// Per-row int4 quantization (qmax 7, the per-token recipe) written as FP6 e2m3
// groups: per 32 elements 24 bytes of 6-bit codes and 8 zero bytes, codes
// [rows, cols] bytes, scales [rows]; cols a multiple of 128.
hipError_t launch_act_quant_f6(const void* a, int act, int rows, int cols, int64_t ld, uint8_t* codes, float* scales,
                               hipStream_t s);

struct GemmArgs {
  const DevExpert* experts;  // device [G]
  int32_t* plan;             // device plan region
  const int32_t* sorted_pair;
  const int32_t* offsets;
  const float* topk_w;
  const void* x;             // [T,H] act
  const int8_t* xq8; const float* xs8;
  const int8_t* xq4; const float* xs4;
  // w4a4-g128: x codes [T,H] with scales [T][H/128]; group scales of h rows
  // (routed [P][F/128], shared [n_shared*T][F_sh/128]; codes in hq / hq_shared)
  const int8_t* xq4g; const float* xs4g;
  const float* hsg; const float* hsg_shared;
  // mxfp4: e2m1 codes [rows][K/2] and E8M0 bytes [rows][K/32] of x, routed h and shared h
  const uint8_t* xqmx; const uint8_t* xsmx;
  const uint8_t* hqmx; const uint8_t* hsmx;
  const uint8_t* hqmx_shared; const uint8_t* hsmx_shared;
  // FP8: e4m3 codes [T,H] and per-token scales [T] of x (h rows of an FP8 down
  // projection use hq / hs and hq_shared / hs_shared)
  const uint8_t* xqf8; const float* xsf8;
  // w4a4 on FP6 operands: x codes [T,H] (e2m3 groups of 32, one byte per
  // element) and per-token scales [T]; h rows of such a down projection use
  // hq / hs and hq_shared / hs_shared
  const uint8_t* xqf6; const float* xsf6;
  void* h; void* h_shared;
  const int8_t* hq; const float* hs;
  const int8_t* hq_shared; const float* hs_shared;
  void* slots;         // weighted down rows [T][k + n_shared][H]: activation dtype (slot16), else fp32
  int32_t slot16;
  const float* shared_w;     // [T][n_shared] weights of the shared experts' rows, or null (weight 1)
  const int32_t* down_qmax;
  int32_t T, k;
  int32_t act;
  int32_t G;          // experts incl. shared
  int32_t E_routed;
  int32_t n_shared;
  int32_t qcap;        // capacity of each XCD queue in the plan region (super-tiles)
  int32_t fcap;        // capacity of each XCD queue in the plan region (tiles)
  float* partial;      // split-K partial sums
  // per sorted row (RowMeta; rxs8 / rxs4 from the x encodings, XPrep::inv)
  const int32_t* rtok; const int32_t* rslot; const float* rgw; const float* rxs8; const float* rxs4;
  // Row sums of each 128-wide k block of the 16-bit activation rows that the
  // bias-dequantized weight kinds need (bf16): x [T][H/128] (the input in
  // single-linear mode), routed h [P][F/128] and shared h [n_shared*T][F_sh/128],
  // the latter two written by the gate|up epilogue.
  const float* rsx; float* rsh; float* rsh_shared;
  // single-linear mode (mxmoe_linear_forward): raw int32 / fp32 output
  DevLinear raw_lin;
  void* raw_out;
};

// Encodings of the block input x [rows, cols] (16-bit, rows 16-byte aligned,
// ld = cols, cols a multiple of 128) that the gate/up linears read; a null
// output pointer skips that encoding.  rows = 0: none.
struct XPrep {
  const void* x;
  int act, rows, cols;
  int8_t* q8;     // int8 codes [rows, cols], scales s8 [rows]
  float* s8;
  int8_t* q4;     // int4 codes (one per byte), scales s4 [rows]
  float* s4;
  float* rs;      // bf16 row sums per 128-wide block [rows, cols / 128]
  int8_t* q4g;    // int4 codes with per-128-group scales s4g [rows, cols / 128]
  float* s4g;
  uint8_t* qmx;   // MXFP4 codes [rows, cols / 2], E8M0 bytes smx [rows, cols / 32]
  uint8_t* smx;
  uint8_t* qf8;   // FP8 e4m3 codes [rows, cols], scales sf8 [rows]
  float* sf8;
  uint8_t* qf6;   // int4 codes as FP6 e2m3 groups [rows, cols] (one byte per element), scales sf6 [rows]
  float* sf6;
  // the routed rows' copies of the per-token scales s8 / s4: row inv[r * k +
  // s] (skipped where -1) of r8 / r4, for s < k (null: none)
  const int32_t* inv;
  int k;
  float* r8;
  float* r4;
};

// raw_m >= 0: single-linear plan (raw_lin, m = raw_m); else the block plan of
// both phases from counts.  mask_words: 64 words, bit g = expert g gets tiles.
// The same launch encodes xp on its other workgroups (they do not wait for
// the plan, nor it for them).
// The plan prices tiles with the process-wide cost table (tile_costs_get).
hipError_t launch_plan(const DevExpert* experts, int E, int G, int T, const int32_t* counts,
                       const int32_t* offsets, int raw_m, const DevLinear& raw_lin, const uint32_t* mask_words,
                       int32_t* plan, int qcap, int fcap, int64_t pfloats, int32_t* down_qmax, int nwg,
                       const XPrep& xp, hipStream_t s);
// Process-wide tile cost table: the roofline default until a caller sets one;
// set (nullptr restores the default) and get copy under a lock.
void tile_costs_default(TileCosts* out);
void tile_costs_set(const TileCosts* t);
void tile_costs_get(TileCosts* out);
hipError_t launch_group_gemm(const GemmArgs& a, int phase, int grid, hipStream_t s);
int group_gemm_grid(int device);

// slots in the activation dtype (slot16) or fp32
hipError_t launch_combine(const void* slots, int slot16, const int32_t* ids, int T, int k, int E, int n_sh,
                          int H, int act, void* y, hipStream_t s);

}  // namespace mxmoe
