// Host side of the C ABI: argument validation, workspace carving and launch
// sequencing.  Nothing here allocates device memory or synchronizes.
#include <string.h>

#include <algorithm>
#include <mutex>

#include "mxmoe_internal.h"

using namespace mxmoe;

// Workspace of mxmoe_moe_forward_noalloc: one file-scope device array, of
// which every GPU the library runs on holds its own copy until the process
// ends.  Host code never uses the array's name as an address: the copy of a
// device is found once with hipGetSymbolAddress (with that device current)
// and its address kept per device.
static __device__ __align__(256) uint8_t scratch[MXMOE_NOALLOC_SCRATCH_BYTES];

namespace {

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// scheme -> micro-kernel kind, -1 if unsupported
int scheme_kind(const mxmoe_scheme& s) {
  if (s.fmt == 1)  // OCP MX: FP4 e2m1 on both operands, E8M0 scale per 32
    return (s.w_bits == 4 && s.a_bits == 4 && s.w_group == 32 && s.a_group == 32 && s.symmetric == 1) ? K_MXFP4 : -1;
  if (s.fmt == 2)  // FP8 e4m3: per-channel weight scales, per-token activation scales
    return (s.w_bits == 8 && s.a_bits == 8 && s.w_group == -1 && s.a_group == -1 && s.symmetric == 1) ? K_F8A8 : -1;
  if (s.fmt == 3)  // w4a4 (per channel / per token) with its int4 codes held as FP6 e2m3 operands
    return (s.w_bits == 4 && s.a_bits == 4 && s.w_group == -1 && s.a_group == -1 && s.symmetric == 1) ? K_W4A4F6 : -1;
  if (s.fmt != 0) return -1;
  if (s.w_bits == 4 && s.a_bits == 4 && s.w_group == 128 && s.a_group == 128 && s.symmetric == 1) return K_W4A4G;
  if (s.a_group != -1) return -1;
  if (s.w_bits == 16 && s.a_bits == 16 && s.w_group == -1 && s.symmetric == 0) return K_W16;
  if (s.a_bits == 8 && s.w_bits == 8 && s.w_group == -1 && s.symmetric == 1) return K_W8A8;
  if (s.a_bits == 4 && s.w_bits == 4 && s.w_group == -1 && s.symmetric == 1) return K_W4A4;
  if (s.a_bits == 16 && s.w_group == 128 && s.symmetric == 0) {
    switch (s.w_bits) {
      case 2: return K_W2G;
      case 3: return K_W3G;
      case 4: return K_W4G;
      case 8: return K_W8G;
    }
  }
  return -1;
}

bool same_scheme(const mxmoe_scheme& a, const mxmoe_scheme& b) {
  return a.w_bits == b.w_bits && a.a_bits == b.a_bits && a.w_group == b.w_group && a.a_group == b.a_group &&
         a.symmetric == b.symmetric && a.fmt == b.fmt;
}

bool valid_dtype(int d) { return d == MXMOE_F16 || d == MXMOE_BF16; }

mxmoe_status check_linear(const mxmoe_linear* L, int* kind) {
  if (!L) return MXMOE_ERR_INVALID_ARG;
  if (L->n <= 0 || L->k <= 0) return MXMOE_ERR_INVALID_ARG;
  const int kd = scheme_kind(L->s);
  if (kd < 0) return MXMOE_ERR_UNSUPPORTED;
  if (L->n % 16 || L->k % 128) return MXMOE_ERR_UNSUPPORTED;
  if ((int64_t)L->n * L->k >= (1LL << 31)) return MXMOE_ERR_UNSUPPORTED;
  *kind = kd;
  return MXMOE_OK;
}

size_t packed_bytes_kind(int kd, int n, int k) {
  size_t b = (size_t)codes_bytes(kd, n, k);
  if (kind_is_int(kd) && kd != K_W4A4G) b += 4 * (size_t)n;  // per-channel fp32 scales
  return b;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

struct BlockInfo {
  int H, F, E, k, nsh, Fsh, act, G;
  bool any_x8 = false, any_x4 = false, any_hq = false, any_hq_sh = false;
  bool rs_x = false, rs_h = false, rs_hsh = false;  // row sums of x / h / h_shared needed (bf16)
  bool any_x4g = false, any_hg = false, any_hg_sh = false;  // w4a4-g128 gate|up, routed / shared down
  bool any_xmx = false, any_hmx = false, any_hmx_sh = false;  // mxfp4 gate|up, routed / shared down
  bool any_xf8 = false;  // FP8 gate|up
  bool any_xf6 = false;  // w4a4 on FP6 operands, gate|up
  int kinds[kMaxG][3];
};

mxmoe_status check_block(const mxmoe_block* B, BlockInfo* bi) {
  if (!B || !B->scheme) return MXMOE_ERR_INVALID_ARG;
  if (!valid_dtype(B->act)) return MXMOE_ERR_INVALID_ARG;
  if (B->hidden <= 0 || B->ffn <= 0 || B->n_experts <= 0 || B->top_k <= 0) return MXMOE_ERR_INVALID_ARG;
  if (B->n_experts > kMaxE || B->top_k > B->n_experts) return MXMOE_ERR_INVALID_ARG;
  if (B->n_shared < 0 || B->n_shared > kMaxShared) return MXMOE_ERR_INVALID_ARG;
  if (B->n_shared > 0 && B->ffn_shared <= 0) return MXMOE_ERR_INVALID_ARG;
  if (B->hidden % 128 || B->ffn % 128 || (B->n_shared > 0 && B->ffn_shared % 128)) return MXMOE_ERR_UNSUPPORTED;
  bi->H = B->hidden;
  bi->F = B->ffn;
  bi->E = B->n_experts;
  bi->k = B->top_k;
  bi->nsh = B->n_shared;
  bi->Fsh = B->n_shared > 0 ? B->ffn_shared : 0;
  bi->act = B->act;
  bi->G = bi->E + bi->nsh;
  bi->any_x8 = bi->any_x4 = bi->any_hq = bi->any_hq_sh = false;
  bi->rs_x = bi->rs_h = bi->rs_hsh = false;
  bi->any_x4g = bi->any_hg = bi->any_hg_sh = false;
  bi->any_xmx = bi->any_hmx = bi->any_hmx_sh = false;
  bi->any_xf8 = false;
  bi->any_xf6 = false;
  if (bi->G > kMaxG) return MXMOE_ERR_UNSUPPORTED;
  for (int g = 0; g < bi->G; ++g) {
    const mxmoe_scheme* s = B->scheme + 3 * g;
    for (int j = 0; j < 3; ++j) {
      const int kd = scheme_kind(s[j]);
      if (kd < 0) return MXMOE_ERR_UNSUPPORTED;
      bi->kinds[g][j] = kd;
    }
    if (!same_scheme(s[0], s[1])) return MXMOE_ERR_UNSUPPORTED;  // gate|up share one tile
    const bool sh = g >= bi->E;
    const int kg = bi->kinds[g][0];
    if (kg == K_W8A8) bi->any_x8 = true;
    if (kg == K_W4A4) bi->any_x4 = true;
    if (kg == K_W4A4G) bi->any_x4g = true;
    if (bi->kinds[g][2] == K_W4A4G) (sh ? bi->any_hg_sh : bi->any_hg) = true;
    if (kg == K_MXFP4) bi->any_xmx = true;
    if (kg == K_F8A8) bi->any_xf8 = true;
    if (kg == K_W4A4F6) bi->any_xf6 = true;
    if (bi->kinds[g][2] == K_MXFP4) (sh ? bi->any_hmx_sh : bi->any_hmx) = true;
    if (kind_is_int(bi->kinds[g][2])) (sh ? bi->any_hq_sh : bi->any_hq) = true;
    if (bi->act == MXMOE_BF16 && kind_is_magic(kg)) bi->rs_x = true;
    if (bi->act == MXMOE_BF16 && kind_is_magic(bi->kinds[g][2])) (sh ? bi->rs_hsh : bi->rs_h) = true;
  }
  return MXMOE_OK;
}

// The Group-GEMM addresses activation rows with 32-bit byte offsets from the
// start of their buffer: x, the routed h rows and the shared h rows (and their
// one-byte and half-byte encodings, which are smaller) stay below 4 GiB.
bool activations_fit(const BlockInfo& bi, int64_t T) {
  const int64_t lim = (int64_t)1 << 32;
  return T * bi.H * 2 < lim && T * bi.k * bi.F * 2 < lim && (int64_t)bi.nsh * T * bi.Fsh * 2 < lim;
}

WsLayout layout_of(const BlockInfo& bi, int T) {
  WsLayout L;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  const size_t P = (size_t)T * bi.k;
  const size_t nchunks = (P + kRouteChunk - 1) / kRouteChunk;
  L.status = take(16 * 4);
  L.counts = take(4 * (size_t)bi.E);
  L.offsets = take(4 * ((size_t)bi.E + 1));
  L.sorted_pair = take(4 * P);
  L.inv = take(4 * P);
  L.chunk_counts = take(4 * nchunks * bi.E);
  L.chunk_bad = take(4 * nchunks);
  L.qcap = plan_queue_cap((int64_t)T * bi.k + (int64_t)bi.nsh * T, bi.G, std::max(std::max(bi.F, bi.Fsh), bi.H));
  L.fcap = plan_flat_cap(L.qcap);
  L.plan = take(4 * (size_t)plan_layout(bi.G, L.qcap, L.fcap).total);
  L.down_qmax = take(4 * (size_t)bi.G);
  L.rtok = take(4 * P);
  L.rslot = take(4 * P);
  L.rgw = take(4 * P);
  L.rxs8 = bi.any_x8 ? take(4 * P) : kNone;
  L.rxs4 = bi.any_x4 ? take(4 * P) : kNone;
  // split-K partial sums: a few times the largest layer output, at most 512 MB
  L.pfloats = std::min<int64_t>((int64_t)1 << 27,
                                4 * ((int64_t)P + (int64_t)bi.nsh * T) * std::max(std::max(bi.F, bi.Fsh), bi.H));
  L.partial = take(4 * (size_t)L.pfloats);
  L.xq8 = L.xs8 = L.xq4 = L.xs4 = kNone;
  if (bi.any_x8) { L.xq8 = take((size_t)T * bi.H); L.xs8 = take(4 * (size_t)T); }
  if (bi.any_x4) { L.xq4 = take((size_t)T * bi.H); L.xs4 = take(4 * (size_t)T); }
  L.h = take(2 * P * bi.F);
  L.h_shared = bi.nsh ? take(2 * (size_t)bi.nsh * T * bi.Fsh) : kNone;
  L.hq = L.hs = L.hq_shared = L.hs_shared = kNone;
  if (bi.any_hq) { L.hq = take(P * bi.F); L.hs = take(4 * P); }
  if (bi.any_hq_sh) { L.hq_shared = take((size_t)bi.nsh * T * bi.Fsh); L.hs_shared = take(4 * (size_t)bi.nsh * T); }
  L.slots = take(4 * (size_t)T * (bi.k + bi.nsh) * bi.H);
  L.rsx = bi.rs_x ? take(4 * (size_t)T * (bi.H / 128)) : kNone;
  L.rsh = bi.rs_h ? take(4 * P * (bi.F / 128)) : kNone;
  L.rsh_shared = bi.rs_hsh ? take(4 * (size_t)bi.nsh * T * (bi.Fsh / 128)) : kNone;
  L.xq4g = bi.any_x4g ? take((size_t)T * bi.H) : kNone;
  L.xs4g = bi.any_x4g ? take(4 * (size_t)T * (bi.H / 128)) : kNone;
  L.hsg = bi.any_hg ? take(4 * P * (bi.F / 128)) : kNone;
  L.hsg_shared = bi.any_hg_sh ? take(4 * (size_t)bi.nsh * T * (bi.Fsh / 128)) : kNone;
  L.xqmx = bi.any_xmx ? take((size_t)T * bi.H / 2) : kNone;
  L.xsmx = bi.any_xmx ? take((size_t)T * bi.H / 32) : kNone;
  L.hqmx = bi.any_hmx ? take(P * bi.F / 2) : kNone;
  L.hsmx = bi.any_hmx ? take(P * bi.F / 32) : kNone;
  L.hqmx_shared = bi.any_hmx_sh ? take((size_t)bi.nsh * T * bi.Fsh / 2) : kNone;
  L.hsmx_shared = bi.any_hmx_sh ? take((size_t)bi.nsh * T * bi.Fsh / 32) : kNone;
  L.xqf8 = bi.any_xf8 ? take((size_t)T * bi.H) : kNone;
  L.xsf8 = bi.any_xf8 ? take(4 * (size_t)T) : kNone;
  L.xqf6 = bi.any_xf6 ? take((size_t)T * bi.H) : kNone;
  L.xsf6 = bi.any_xf6 ? take(4 * (size_t)T) : kNone;
  L.rids = take(4 * P);
  L.rw = take(4 * P);
  L.shw = bi.nsh ? take(4 * (size_t)T * bi.nsh) : kNone;
  L.total = o;
  return L;
}

template <typename TT> TT* at(void* ws, size_t off) {
  return off == kNone ? nullptr : reinterpret_cast<TT*>(reinterpret_cast<uint8_t*>(ws) + off);
}

mxmoe_status hip_status(hipError_t e) { return e == hipSuccess ? MXMOE_OK : MXMOE_ERR_HIP; }

int current_device() {
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess) d = 0;
  return d;
}

}  // namespace

extern "C" {

int32_t mxmoe_version(void) { return (0 << 16) | 1; }

mxmoe_status mxmoe_set_tile_costs(const int32_t* table, int32_t n_entries) {
  static_assert(MXMOE_TILE_COST_ENTRIES == mxmoe::kCostEntries, "cost table size");
  if (!table) {
    mxmoe::tile_costs_set(nullptr);
    return MXMOE_OK;
  }
  if (n_entries != MXMOE_TILE_COST_ENTRIES) return MXMOE_ERR_INVALID_ARG;
  mxmoe::TileCosts t;
  for (int i = 0; i < MXMOE_TILE_COST_ENTRIES; ++i) {
    if (table[i] < 0 && i % 4 != 0) return MXMOE_ERR_INVALID_ARG;  // a may be negative
    t.v[i] = table[i];
  }
  mxmoe::tile_costs_set(&t);
  return MXMOE_OK;
}

mxmoe_status mxmoe_get_tile_costs(int32_t* out, int32_t n_entries) {
  if (!out || n_entries != MXMOE_TILE_COST_ENTRIES) return MXMOE_ERR_INVALID_ARG;
  mxmoe::TileCosts t;
  mxmoe::tile_costs_get(&t);
  for (int i = 0; i < MXMOE_TILE_COST_ENTRIES; ++i) out[i] = t.v[i];
  return MXMOE_OK;
}

const char* mxmoe_status_string(mxmoe_status s) {
  switch (s) {
    case MXMOE_OK: return "ok";
    case MXMOE_ERR_INVALID_ARG: return "invalid argument";
    case MXMOE_ERR_UNSUPPORTED: return "unsupported scheme or shape";
    case MXMOE_ERR_WORKSPACE: return "workspace or buffer too small";
    case MXMOE_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

size_t mxmoe_packed_bytes(const mxmoe_linear* L, mxmoe_dtype act) {
  int kd;
  if (!valid_dtype(act) || check_linear(L, &kd) != MXMOE_OK) return 0;
  return packed_bytes_kind(kd, L->n, L->k);
}

mxmoe_status mxmoe_pack_weights(const mxmoe_linear* L, mxmoe_dtype act, mxmoe_dtype w16_src, const void* codes,
                                const void* scales, const void* zeros, void* packed, size_t packed_bytes,
                                hipStream_t stream) {
  int kd;
  mxmoe_status st = check_linear(L, &kd);
  if (st != MXMOE_OK) return st;
  if (!valid_dtype(act) || !valid_dtype(w16_src)) return MXMOE_ERR_INVALID_ARG;
  if (!codes || !packed || !aligned(packed, 256) || !aligned(codes, 4)) return MXMOE_ERR_INVALID_ARG;
  if (kd != K_W16 && (!scales || !aligned(scales, 4))) return MXMOE_ERR_INVALID_ARG;
  if (kind_is_wonly(kd) && (!zeros || !aligned(zeros, 4))) return MXMOE_ERR_INVALID_ARG;
  if (packed_bytes < packed_bytes_kind(kd, L->n, L->k)) return MXMOE_ERR_WORKSPACE;
  return hip_status(launch_pack(kd, L->n, L->k, act, w16_src, codes, scales, zeros, (uint8_t*)packed, stream));
}

mxmoe_status mxmoe_unpack_weights(const mxmoe_linear* L, mxmoe_dtype act, const void* packed, void* codes,
                                  void* scales, void* zeros, hipStream_t stream) {
  int kd;
  mxmoe_status st = check_linear(L, &kd);
  if (st != MXMOE_OK) return st;
  if (!valid_dtype(act) || !codes || !packed || !aligned(packed, 256)) return MXMOE_ERR_INVALID_ARG;
  if (kd != K_W16 && !scales) return MXMOE_ERR_INVALID_ARG;
  if (kind_is_wonly(kd) && !zeros) return MXMOE_ERR_INVALID_ARG;
  return hip_status(launch_unpack(kd, L->n, L->k, act, (const uint8_t*)packed, codes, scales, zeros, stream));
}

size_t mxmoe_route_workspace_bytes(int32_t T, int32_t k, int32_t E) {
  if (T < 0 || k <= 0 || E <= 0) return 0;
  const size_t P = (size_t)T * k;
  const size_t nchunks = (P + kRouteChunk - 1) / kRouteChunk;
  return align256(4 * nchunks * E) + align256(4 * nchunks) + 256;
}

mxmoe_status mxmoe_route_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                                 int32_t* offsets, int32_t* sorted_pair, int32_t* inv, int32_t* status,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (T < 0 || k <= 0 || E <= 0 || k > E || E > kMaxE) return MXMOE_ERR_INVALID_ARG;
  if ((int64_t)T * k >= (1LL << 31)) return MXMOE_ERR_INVALID_ARG;
  if (!counts || !offsets || !status || !workspace) return MXMOE_ERR_INVALID_ARG;
  if (T > 0 && (!topk_ids || !sorted_pair || !inv)) return MXMOE_ERR_INVALID_ARG;
  if (!aligned(workspace, 256)) return MXMOE_ERR_INVALID_ARG;
  if (workspace_bytes < mxmoe_route_workspace_bytes(T, k, E)) return MXMOE_ERR_WORKSPACE;
  const size_t P = (size_t)T * k;
  const size_t nchunks = (P + kRouteChunk - 1) / kRouteChunk;
  int32_t* cc = reinterpret_cast<int32_t*>(workspace);
  int32_t* cb = reinterpret_cast<int32_t*>(reinterpret_cast<uint8_t*>(workspace) + align256(4 * nchunks * E));
  return hip_status(launch_route(topk_ids, T, k, E, counts, offsets, sorted_pair, inv, status, cc, cb, nullptr, stream));
}

mxmoe_status mxmoe_router_topk(const float* logits, int32_t T, int32_t E, int32_t k, int32_t renormalize,
                               const float* shared_logits, int32_t n_shared, int32_t* topk_ids, float* topk_w,
                               float* shared_w, hipStream_t stream) {
  if (T < 0 || E <= 0 || E > kMaxE || k <= 0 || k > E || k > kRouterMaxK) return MXMOE_ERR_INVALID_ARG;
  if (n_shared < 0 || n_shared > kMaxShared || (renormalize != 0 && renormalize != 1)) return MXMOE_ERR_INVALID_ARG;
  if ((int64_t)T * E >= (1LL << 31)) return MXMOE_ERR_INVALID_ARG;
  if (T == 0) return MXMOE_OK;
  if (!logits || !topk_ids || !topk_w) return MXMOE_ERR_INVALID_ARG;
  if (shared_logits && n_shared > 0 && !shared_w) return MXMOE_ERR_INVALID_ARG;
  if (!aligned(logits, 4) || !aligned(topk_ids, 4) || !aligned(topk_w, 4) || !aligned(shared_logits, 4) ||
      !aligned(shared_w, 4))
    return MXMOE_ERR_INVALID_ARG;
  return hip_status(launch_router_topk(logits, T, E, k, renormalize, n_shared > 0 ? shared_logits : nullptr, n_shared,
                                       topk_ids, topk_w, shared_w, stream));
}

mxmoe_status mxmoe_act_quant(const void* a, mxmoe_dtype act, int32_t rows, int32_t cols, int64_t ld, int32_t qmax,
                             int8_t* codes, float* scales, hipStream_t stream) {
  if (!valid_dtype(act) || rows < 0 || cols <= 0 || ld < cols) return MXMOE_ERR_INVALID_ARG;
  if (qmax != 127 && qmax != 7 && qmax != kQmaxF8) return MXMOE_ERR_UNSUPPORTED;
  if (rows > 0 && (!a || !codes || !scales)) return MXMOE_ERR_INVALID_ARG;
  return hip_status(launch_act_quant(a, act, rows, cols, ld, qmax, codes, scales, stream));
}

// -------------------------------------------------------- single linear
namespace {
struct LinWs { size_t plan, partial, aq, as, rsa, total; int qcap, fcap; int64_t pfloats; };
LinWs lin_layout(int kd, int m, int n, int k) {
  LinWs w;
  size_t o = 0;
  w.qcap = plan_queue_cap(m, 1, n);
  w.fcap = plan_flat_cap(w.qcap);
  w.plan = o; o = align256(o + 4 * (size_t)plan_layout(1, w.qcap, w.fcap).total);
  // split-K partial sums: room for every tile of the linear in up to 8 slices
  // (at most m + 128 rows by n + 512 channels of tiles), at most 64 MB
  w.pfloats = std::min<int64_t>((int64_t)1 << 24, 8 * ((int64_t)m + 128) * ((int64_t)n + 512));
  w.partial = o; o = align256(o + 4 * (size_t)w.pfloats);
  w.aq = w.as = w.rsa = kNone;
  if (kind_is_int(kd)) {
    w.aq = o; o = align256(o + (size_t)m * k);
    w.as = o; o = align256(o + 4 * (size_t)m * (kd == K_W4A4G ? k / 128 : 1));
  }
  if (kind_is_mx(kd)) {  // e2m1 codes and E8M0 bytes of the input
    w.aq = o; o = align256(o + (size_t)m * k / 2);
    w.as = o; o = align256(o + (size_t)m * k / 32);
  }
  // row sums of the input per 128-wide k block (used with bf16 activations)
  if (kind_is_magic(kd)) { w.rsa = o; o = align256(o + 4 * (size_t)m * (k / 128)); }
  w.total = o;
  return w;
}
}  // namespace

size_t mxmoe_linear_workspace_bytes(const mxmoe_linear* L, int32_t m) {
  int kd;
  if (m < 0 || check_linear(L, &kd) != MXMOE_OK) return 0;
  return lin_layout(kd, m, L->n, L->k).total;
}

mxmoe_status mxmoe_linear_forward(const mxmoe_linear* L, mxmoe_dtype act, const void* packed, int32_t m,
                                  const void* a, void* out, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
  int kd;
  mxmoe_status st = check_linear(L, &kd);
  if (st != MXMOE_OK) return st;
  if (!valid_dtype(act) || m < 0) return MXMOE_ERR_INVALID_ARG;
  if ((int64_t)m * L->k * 2 >= ((int64_t)1 << 32)) return MXMOE_ERR_UNSUPPORTED;  // 32-bit row offsets
  if (m == 0) return MXMOE_OK;
  if (!packed || !a || !out || !workspace) return MXMOE_ERR_INVALID_ARG;
  if (!aligned(packed, 256) || !aligned(a, 16) || !aligned(out, 16) || !aligned(workspace, 256))
    return MXMOE_ERR_INVALID_ARG;
  const LinWs w = lin_layout(kd, m, L->n, L->k);
  if (workspace_bytes < w.total) return MXMOE_ERR_WORKSPACE;
  DevLinear dl;
  dl.packed = reinterpret_cast<const uint8_t*>(packed);
  dl.wscale = (kind_is_int(kd) && kd != K_W4A4G)
                  ? reinterpret_cast<const float*>(dl.packed + codes_bytes(kd, L->n, L->k)) : nullptr;
  dl.n = L->n;
  dl.k = L->k;
  dl.kind = kd;
  dl.pad = 0;
  GemmArgs ga;
  memset(&ga, 0, sizeof(ga));
  ga.plan = at<int32_t>(workspace, w.plan);
  ga.x = a;
  ga.T = m;
  ga.k = 1;
  ga.act = act;
  ga.G = 1;
  ga.E_routed = 1;
  ga.raw_lin = dl;
  ga.raw_out = out;
  ga.qcap = w.qcap;
  ga.fcap = w.fcap;
  ga.partial = at<float>(workspace, w.partial);
  if (kind_is_int(kd)) {
    int8_t* aq = at<int8_t>(workspace, w.aq);
    float* as = at<float>(workspace, w.as);
    hipError_t e = kd == K_W4A4G ? launch_act_quant_g128(a, act, m, L->k, L->k, kind_qmax(kd), aq, as, stream)
                   : (kd == K_W4A4F6 ? launch_act_quant_f6(a, act, m, L->k, L->k, reinterpret_cast<uint8_t*>(aq), as, stream)
                                     : launch_act_quant(a, act, m, L->k, L->k, kind_qmax(kd), aq, as, stream));
    if (e != hipSuccess) return MXMOE_ERR_HIP;
    if (kd == K_W8A8) { ga.xq8 = aq; ga.xs8 = as; }
    else if (kd == K_F8A8) { ga.xqf8 = reinterpret_cast<const uint8_t*>(aq); ga.xsf8 = as; }
    else if (kd == K_W4A4F6) { ga.xqf6 = reinterpret_cast<const uint8_t*>(aq); ga.xsf6 = as; }
    else if (kd == K_W4A4G) { ga.xq4g = aq; ga.xs4g = as; }
    else { ga.xq4 = aq; ga.xs4 = as; }
  }
  if (kind_is_mx(kd)) {
    uint8_t* aq = at<uint8_t>(workspace, w.aq);
    uint8_t* ae = at<uint8_t>(workspace, w.as);
    if (launch_act_quant_mx(a, act, m, L->k, L->k, aq, ae, stream) != hipSuccess) return MXMOE_ERR_HIP;
    ga.xqmx = aq;
    ga.xsmx = ae;
  }
  if (act == MXMOE_BF16 && kind_is_magic(kd)) {
    float* rs = at<float>(workspace, w.rsa);
    if (launch_rowsum(a, m, L->k, L->k, rs, stream) != hipSuccess) return MXMOE_ERR_HIP;
    ga.rsx = rs;
  }
  const int grid = group_gemm_grid(current_device());
  XPrep nox;
  memset(&nox, 0, sizeof(nox));
  hipError_t e = launch_plan(nullptr, 1, 1, m, nullptr, nullptr, m, dl, nullptr, ga.plan, w.qcap, w.fcap, w.pfloats,
                             nullptr, grid, nox, stream);
  if (e != hipSuccess) return MXMOE_ERR_HIP;
  return hip_status(launch_group_gemm(ga, 2, grid, stream));
}

// -------------------------------------------------------- MoE block
size_t mxmoe_block_table_bytes(const mxmoe_block* B) {
  static thread_local BlockInfo bi;
  if (check_block(B, &bi) != MXMOE_OK) return 0;
  return sizeof(DevExpert) * (size_t)bi.G;
}

mxmoe_status mxmoe_block_table_fill(const mxmoe_block* B, void* host_buf, size_t host_bytes) {
  static thread_local BlockInfo bi;
  mxmoe_status st = check_block(B, &bi);
  if (st != MXMOE_OK) return st;
  if (!host_buf || !B->packed) return MXMOE_ERR_INVALID_ARG;
  if (host_bytes < sizeof(DevExpert) * (size_t)bi.G) return MXMOE_ERR_WORKSPACE;
  DevExpert* ex = reinterpret_cast<DevExpert*>(host_buf);
  for (int g = 0; g < bi.G; ++g) {
    const bool sh = g >= bi.E;
    const int F = sh ? bi.Fsh : bi.F;
    for (int j = 0; j < 3; ++j) {
      const void* p = B->packed[3 * g + j];
      if (!p || !aligned(p, 256)) return MXMOE_ERR_INVALID_ARG;
      DevLinear& d = ex[g].lin[j];
      d.kind = bi.kinds[g][j];
      d.n = j < 2 ? F : bi.H;
      d.k = j < 2 ? bi.H : F;
      d.packed = reinterpret_cast<const uint8_t*>(p);
      d.wscale = (kind_is_int(d.kind) && d.kind != K_W4A4G)
                     ? reinterpret_cast<const float*>(d.packed + codes_bytes(d.kind, d.n, d.k))
                                     : nullptr;
      d.pad = 0;
    }
  }
  return MXMOE_OK;
}

size_t mxmoe_workspace_bytes(const mxmoe_block* B, int32_t T) {
  static thread_local BlockInfo bi;
  if (T < 0 || check_block(B, &bi) != MXMOE_OK) return 0;
  return layout_of(bi, T).total;
}

mxmoe_status mxmoe_workspace_layout(const mxmoe_block* B, int32_t T, mxmoe_ws_layout* out) {
  static thread_local BlockInfo bi;
  if (!out || T < 0) return MXMOE_ERR_INVALID_ARG;
  mxmoe_status st = check_block(B, &bi);
  if (st != MXMOE_OK) return st;
  const WsLayout L = layout_of(bi, T);
  out->status = L.status;
  out->counts = L.counts;
  out->offsets = L.offsets;
  out->sorted_pair = L.sorted_pair;
  out->inv = L.inv;
  out->plan = L.plan;
  out->xq8 = L.xq8;
  out->xs8 = L.xs8;
  out->xq4 = L.xq4;
  out->xs4 = L.xs4;
  out->h = L.h;
  out->h_shared = L.h_shared;
  out->hq = L.hq;
  out->hs = L.hs;
  out->hq_shared = L.hq_shared;
  out->hs_shared = L.hs_shared;
  out->slots = L.slots;
  out->total = L.total;
  out->plan_queue_cap = (size_t)L.qcap;
  out->plan_flat_cap = (size_t)L.fcap;
  out->partial = L.partial;
  out->partial_floats = (size_t)L.pfloats;
  out->rsx = L.rsx;
  out->rsh = L.rsh;
  out->rsh_shared = L.rsh_shared;
  out->xq4g = L.xq4g;
  out->xs4g = L.xs4g;
  out->hsg = L.hsg;
  out->hsg_shared = L.hsg_shared;
  out->xqmx = L.xqmx;
  out->xsmx = L.xsmx;
  out->hqmx = L.hqmx;
  out->hsmx = L.hsmx;
  out->hqmx_shared = L.hqmx_shared;
  out->hsmx_shared = L.hsmx_shared;
  out->xqf8 = L.xqf8;
  out->xsf8 = L.xsf8;
  out->xqf6 = L.xqf6;
  out->xsf6 = L.xsf6;
  out->router_ids = L.rids;
  out->router_w = L.rw;
  out->shared_w = L.shw;
  return MXMOE_OK;
}

mxmoe_status mxmoe_moe_forward_ex(const mxmoe_block* B, const void* block_table, int32_t T, const void* x,
                                  const int32_t* topk_ids, const float* topk_w, void* y, void* workspace,
                                  size_t workspace_bytes, const mxmoe_forward_opts* opts, hipStream_t stream) {
  static thread_local BlockInfo bi;
  mxmoe_status st = check_block(B, &bi);
  if (st != MXMOE_OK) return st;
  if (T < 0) return MXMOE_ERR_INVALID_ARG;
  if ((int64_t)T * bi.k >= (1LL << 31)) return MXMOE_ERR_UNSUPPORTED;
  if (!activations_fit(bi, T)) return MXMOE_ERR_UNSUPPORTED;
  const bool router = opts && opts->router_logits;
  if (opts && (opts->reserved0 != 0 || (opts->fp32_slots != 0 && opts->fp32_slots != 1) || opts->reserved1 != 0))
    return MXMOE_ERR_INVALID_ARG;
  if (router) {
    if (opts->renormalize != 0 && opts->renormalize != 1) return MXMOE_ERR_INVALID_ARG;
    if (opts->shared_w || !aligned(opts->router_logits, 4) || !aligned(opts->shared_logits, 4))
      return MXMOE_ERR_INVALID_ARG;
    if (bi.k > kRouterMaxK) return MXMOE_ERR_UNSUPPORTED;
  } else {
    if (opts && opts->shared_logits) return MXMOE_ERR_INVALID_ARG;
    if (opts && !aligned(opts->shared_w, 4)) return MXMOE_ERR_INVALID_ARG;
  }
  if (T == 0) return MXMOE_OK;
  if (!block_table || !x || !y || !workspace) return MXMOE_ERR_INVALID_ARG;
  if (!router && (!topk_ids || !topk_w)) return MXMOE_ERR_INVALID_ARG;
  if (!aligned(block_table, 16) || !aligned(x, 16) || !aligned(y, 16) || !aligned(workspace, 256) ||
      !aligned(topk_ids, 4) || !aligned(topk_w, 4))
    return MXMOE_ERR_INVALID_ARG;
  const WsLayout L = layout_of(bi, T);
  if (workspace_bytes < L.total) return MXMOE_ERR_WORKSPACE;

  uint32_t mask_words[64];
  const uint32_t* mask = nullptr;
  if (opts && opts->expert_mask) {
    memset(mask_words, 0, sizeof(mask_words));
    for (int g = 0; g < bi.G; ++g)
      if (opts->expert_mask[g]) mask_words[g >> 5] |= 1u << (g & 31);
    mask = mask_words;
  }
  const DevExpert* experts = reinterpret_cast<const DevExpert*>(block_table);
  hipError_t e;
#define MX_CHECK(call)                       \
  do {                                       \
    e = (call);                              \
    if (e != hipSuccess) return MXMOE_ERR_HIP; \
  } while (0)

  hipEvent_t* ev = (opts && opts->events) ? opts->events : nullptr;
#define MX_EVENT(i)                                          \
  do {                                                       \
    if (ev && hipEventRecord(ev[i], stream) != hipSuccess) return MXMOE_ERR_HIP; \
  } while (0)

  int32_t* counts = at<int32_t>(workspace, L.counts);
  int32_t* offsets = at<int32_t>(workspace, L.offsets);
  int32_t* sorted_pair = at<int32_t>(workspace, L.sorted_pair);
  int32_t* plan = at<int32_t>(workspace, L.plan);
  int32_t* down_qmax = at<int32_t>(workspace, L.down_qmax);
  MX_EVENT(0);
  // router front-end: ids and gate weights come from the logits, into the workspace
  const int32_t* ids = topk_ids;
  const float* tw = topk_w;
  const float* shw = opts ? opts->shared_w : nullptr;
  // the routing launch also writes each sorted row's token, slot row and
  // gate weight
  RowMeta rm;
  rm.k = bi.k;
  rm.n_sh = bi.nsh;
  rm.topk_w = tw;
  rm.rtok = at<int32_t>(workspace, L.rtok);
  rm.rslot = at<int32_t>(workspace, L.rslot);
  rm.rgw = at<float>(workspace, L.rgw);
  if (router) {  // in the routing launch where the batch allows
    int32_t* rids = at<int32_t>(workspace, L.rids);
    float* rw = at<float>(workspace, L.rw);
    float* rshw = (bi.nsh && opts->shared_logits) ? at<float>(workspace, L.shw) : nullptr;
    MX_CHECK(launch_router_route(opts->router_logits, T, bi.E, bi.k, opts->renormalize,
                                 rshw ? opts->shared_logits : nullptr, bi.nsh, rids, rw, rshw, counts, offsets,
                                 sorted_pair, at<int32_t>(workspace, L.inv), at<int32_t>(workspace, L.status),
                                 at<int32_t>(workspace, L.chunk_counts), at<int32_t>(workspace, L.chunk_bad), &rm,
                                 stream));
    ids = rids;
    tw = rw;
    shw = rshw;
  } else {
    MX_CHECK(launch_route(ids, T, bi.k, bi.E, counts, offsets, sorted_pair, at<int32_t>(workspace, L.inv),
                          at<int32_t>(workspace, L.status), at<int32_t>(workspace, L.chunk_counts),
                          at<int32_t>(workspace, L.chunk_bad), &rm, stream));
  }
  DevLinear none;
  memset(&none, 0, sizeof(none));
  const int grid = group_gemm_grid(current_device());
  // the encodings of x ride on the plan launch (its spare workgroups; x is
  // 16-byte aligned, checked above)
  XPrep xp;
  memset(&xp, 0, sizeof(xp));
  xp.x = x;
  xp.act = bi.act;
  xp.rows = T;
  xp.cols = bi.H;
  if (bi.any_x8) {
    xp.q8 = at<int8_t>(workspace, L.xq8);
    xp.s8 = at<float>(workspace, L.xs8);
  }
  if (bi.any_x4) {
    xp.q4 = at<int8_t>(workspace, L.xq4);
    xp.s4 = at<float>(workspace, L.xs4);
  }
  if (bi.rs_x) xp.rs = at<float>(workspace, L.rsx);
  if (bi.any_x4g) {
    xp.q4g = at<int8_t>(workspace, L.xq4g);
    xp.s4g = at<float>(workspace, L.xs4g);
  }
  if (bi.any_xmx) {
    xp.qmx = at<uint8_t>(workspace, L.xqmx);
    xp.smx = at<uint8_t>(workspace, L.xsmx);
  }
  if (bi.any_xf8) {
    xp.qf8 = at<uint8_t>(workspace, L.xqf8);
    xp.sf8 = at<float>(workspace, L.xsf8);
  }
  if (bi.any_xf6) {
    xp.qf6 = at<uint8_t>(workspace, L.xqf6);
    xp.sf6 = at<float>(workspace, L.xsf6);
  }
  // the x encodings also copy the per-token scales to the token's sorted rows
  xp.inv = at<int32_t>(workspace, L.inv);
  xp.k = bi.k;
  if (xp.q8) xp.r8 = at<float>(workspace, L.rxs8);
  if (xp.q4) xp.r4 = at<float>(workspace, L.rxs4);
  MX_CHECK(launch_plan(experts, bi.E, bi.G, T, counts, offsets, -1, none, mask, plan, L.qcap, L.fcap, L.pfloats,
                       down_qmax, grid, xp, stream));
  GemmArgs ga;
  memset(&ga, 0, sizeof(ga));
  ga.experts = experts;
  ga.plan = plan;
  ga.sorted_pair = sorted_pair;
  ga.offsets = offsets;
  ga.topk_w = tw;
  ga.shared_w = shw;
  ga.x = x;
  ga.xq8 = at<int8_t>(workspace, L.xq8);
  ga.xs8 = at<float>(workspace, L.xs8);
  ga.xq4 = at<int8_t>(workspace, L.xq4);
  ga.xs4 = at<float>(workspace, L.xs4);
  ga.h = at<void>(workspace, L.h);
  ga.h_shared = at<void>(workspace, L.h_shared);
  ga.hq = at<int8_t>(workspace, L.hq);
  ga.hs = at<float>(workspace, L.hs);
  ga.hq_shared = at<int8_t>(workspace, L.hq_shared);
  ga.hs_shared = at<float>(workspace, L.hs_shared);
  ga.slots = at<void>(workspace, L.slots);
  ga.slot16 = (opts && opts->fp32_slots) ? 0 : 1;
  ga.down_qmax = down_qmax;
  ga.T = T;
  ga.k = bi.k;
  ga.act = bi.act;
  ga.G = bi.G;
  ga.E_routed = bi.E;
  ga.n_shared = bi.nsh;
  ga.qcap = L.qcap;
  ga.fcap = L.fcap;
  ga.rtok = at<int32_t>(workspace, L.rtok);
  ga.rslot = at<int32_t>(workspace, L.rslot);
  ga.rgw = at<float>(workspace, L.rgw);
  ga.rxs8 = at<float>(workspace, L.rxs8);
  ga.rxs4 = at<float>(workspace, L.rxs4);
  ga.partial = at<float>(workspace, L.partial);
  ga.rsx = at<float>(workspace, L.rsx);
  ga.xq4g = at<int8_t>(workspace, L.xq4g);
  ga.xs4g = at<float>(workspace, L.xs4g);
  ga.hsg = at<float>(workspace, L.hsg);
  ga.hsg_shared = at<float>(workspace, L.hsg_shared);
  ga.rsh = at<float>(workspace, L.rsh);
  ga.rsh_shared = at<float>(workspace, L.rsh_shared);
  ga.xqmx = at<uint8_t>(workspace, L.xqmx);
  ga.xsmx = at<uint8_t>(workspace, L.xsmx);
  ga.hqmx = at<uint8_t>(workspace, L.hqmx);
  ga.hsmx = at<uint8_t>(workspace, L.hsmx);
  ga.hqmx_shared = at<uint8_t>(workspace, L.hqmx_shared);
  ga.hsmx_shared = at<uint8_t>(workspace, L.hsmx_shared);
  ga.xqf8 = at<uint8_t>(workspace, L.xqf8);
  ga.xsf8 = at<float>(workspace, L.xsf8);
  ga.xqf6 = at<uint8_t>(workspace, L.xqf6);
  ga.xsf6 = at<float>(workspace, L.xsf6);
  MX_EVENT(1);
  MX_EVENT(2);
  MX_CHECK(launch_group_gemm(ga, 0, grid, stream));
  MX_EVENT(3);
  MX_EVENT(4);
  if (bi.any_hq || bi.any_hmx)
    MX_CHECK(launch_hquant_routed(ga.h, bi.act, T * bi.k, bi.F, offsets, bi.E, down_qmax, at<int8_t>(workspace, L.hq),
                                  at<float>(workspace, L.hs), at<float>(workspace, L.hsg), at<uint8_t>(workspace, L.hqmx),
                                  at<uint8_t>(workspace, L.hsmx), stream));
  for (int j = 0; j < bi.nsh; ++j) {
    const size_t rows = (size_t)j * T;
    const void* hsrc = reinterpret_cast<const uint8_t*>(ga.h_shared) + rows * bi.Fsh * 2;
    if (bi.kinds[bi.E + j][2] == K_MXFP4) {
      MX_CHECK(launch_act_quant_mx(hsrc, bi.act, T, bi.Fsh, bi.Fsh, at<uint8_t>(workspace, L.hqmx_shared) + rows * bi.Fsh / 2,
                                   at<uint8_t>(workspace, L.hsmx_shared) + rows * bi.Fsh / 32, stream));
      continue;
    }
    const int qm = kind_qmax(bi.kinds[bi.E + j][2]);
    if (!qm) continue;
    int8_t* hq = at<int8_t>(workspace, L.hq_shared) + rows * bi.Fsh;
    if (bi.kinds[bi.E + j][2] == K_W4A4F6) {
      MX_CHECK(launch_act_quant_f6(hsrc, bi.act, T, bi.Fsh, bi.Fsh, reinterpret_cast<uint8_t*>(hq),
                                   at<float>(workspace, L.hs_shared) + rows, stream));
      continue;
    }
    if (bi.kinds[bi.E + j][2] == K_W4A4G)
      MX_CHECK(launch_act_quant_g128(hsrc, bi.act, T, bi.Fsh, bi.Fsh, qm, hq,
                                     at<float>(workspace, L.hsg_shared) + rows * (bi.Fsh / 128), stream));
    else
      MX_CHECK(launch_act_quant(hsrc, bi.act, T, bi.Fsh, bi.Fsh, qm, hq, at<float>(workspace, L.hs_shared) + rows,
                                stream));
  }
  MX_EVENT(5);
  MX_EVENT(6);
  MX_CHECK(launch_group_gemm(ga, 1, grid, stream));
  MX_EVENT(7);
  MX_EVENT(8);
  if (!(opts && opts->skip_combine))
    MX_CHECK(launch_combine(ga.slots, ga.slot16, ids, T, bi.k, bi.E, bi.nsh, bi.H, bi.act, y, stream));
  MX_EVENT(9);
#undef MX_EVENT
#undef MX_CHECK
  return MXMOE_OK;
}

}  // extern "C"

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Address of the current device's copy of `scratch` (looked up on the first
// call on that device, then cached).
mxmoe_status scratch_of_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MXMOE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MXMOE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MXMOE_OK;
}
}  // namespace

extern "C" {

mxmoe_status mxmoe_moe_forward_noalloc(const mxmoe_block* B, const void* block_table, int32_t T, const void* x,
                                       const int32_t* topk_ids, const float* topk_w, void* y, hipStream_t stream) {
  static thread_local BlockInfo bi;
  mxmoe_status st = check_block(B, &bi);
  if (st != MXMOE_OK) return st;
  if (T < 0) return MXMOE_ERR_INVALID_ARG;
  if ((int64_t)T * bi.k >= (1LL << 31)) return MXMOE_ERR_UNSUPPORTED;
  if (layout_of(bi, T).total > (size_t)MXMOE_NOALLOC_SCRATCH_BYTES) return MXMOE_ERR_WORKSPACE;
  if (T == 0) return MXMOE_OK;
  void* ws = nullptr;
  st = scratch_of_current_device(&ws);
  if (st != MXMOE_OK) return st;
  return mxmoe_moe_forward_ex(B, block_table, T, x, topk_ids, topk_w, y, ws, (size_t)MXMOE_NOALLOC_SCRATCH_BYTES,
                              nullptr, stream);
}

mxmoe_status mxmoe_moe_forward(const mxmoe_block* B, const void* block_table, int32_t T, const void* x,
                               const int32_t* topk_ids, const float* topk_w, void* y, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  return mxmoe_moe_forward_ex(B, block_table, T, x, topk_ids, topk_w, y, workspace, workspace_bytes, nullptr, stream);
}

}  // extern "C"
