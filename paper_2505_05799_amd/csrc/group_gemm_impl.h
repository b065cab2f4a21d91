// Mixed-precision Group-GEMM of the MoE block (Sec. 4.3 of the paper:
// micro-kernel specialization, equal-resource tile configurations, and a
// greedy longest-tile-first schedule), written for gfx950.
//
//   plan_kernel        one workgroup: per (phase, expert) group picks a tile
//                      configuration from the group's row count, counts its
//                      tiles, estimates a per-tile cost and orders the groups by
//                      decreasing tile cost (ties: lower expert first).  The tile
//                      queue of a phase is the concatenation of the groups'
//                      tiles in that order: workgroups that free up take the next
//                      tile, i.e. list scheduling with the longest tiles first.
//   group_gemm_kernel  persistent: every workgroup pops tile indices from an
//                      atomic head counter and dispatches, outside the MAC loop,
//                      to the micro-kernel of the tile's (scheme, configuration).
//
// Every configuration uses 4 wavefronts (equal resources for all micro-kernels,
// as the paper requires for horizontal fusion) stacked along the output
// channels: a tile is BM rows x BN channels (per linear) and wavefront w owns
// channels [w*BN/4, (w+1)*BN/4).  Activation rows of the tile are staged per
// 128-wide k block into LDS with direct global->LDS loads (16-byte chunks,
// XOR-swizzled so that MFMA fragment reads are bank-conflict free), double
// buffered; weights stream from HBM straight into registers in the packed
// fragment order (each weight is read once per tile, by one wavefront).
//
// MFMA roles: activations are the A operand (16 rows x 32/64 k), weights the B
// operand (32/64 k x 16 channels).  A lane's four accumulators are four rows of
// one output channel, so a lane needs one (scale, zero) pair per fragment.
//
// Numerics per scheme (every result is exact up to fp32 accumulation):
//   w16   : 16-bit MFMA, fp32 accumulation.
//   mxfp4 : scaled FP4 MFMA (e2m1 x e2m1 with an E8M0 scale per 32 on both
//           operands), fp32 accumulation.
//   w8a8  : int8 MFMA, exact int32 sums, then fp32 (acc * s_a) * s_w.
//   w4a4  : nibbles widened to int8 as 16*q, int8 MFMA, exact sum / 16.
//   w4a4 on FP6 operands: the int4 codes of both operands stored as e2m3
//           values, scaled FP6 MFMA (twice the int8 rate); every product is an
//           integer and every fp32 sum stays below 2^24, so the sums are the
//           exact integer ones; then fp32 (acc * s_a) * s_w as w8a8.
//   wNg128: the 16-bit operand is formed exactly.  bf16 activations: a packed
//           integer add turns the codes of two slots into bf16 values
//           c + (q - z), c = 128 + 2^N - 1, and the row sums R of the staged
//           activations (computed by an MFMA against ones) remove c * R.  fp16
//           activations: the same bit pattern in fp16 minus 1024 + 2^N - 1 gives
//           q - z exactly.  8-bit codes are converted through fp32.  Each
//           128-wide group has its own fp16 scale s_g: the running sum Q is kept
//           in units of the current group's scale, Q_g = Q_{g-1} * s_{g-1}/s_g +
//           sum_g a*(q - z) (the correction -c*R folded into the same FMA), and
//           the output is s_last * Q_last.
//
// Phase 0 computes gate and up of an expert in the same tile and applies the
// SiLU gate in registers: h = SiLU(g) * u, rounded once to the activation
// dtype.  Phase 1 computes the down projection, multiplies each row by its
// router gate weight and stores fp32 rows in the per-(token, slot) buffer that
// the combine sums in a fixed order.
#pragma once
#include "mxmoe_internal.h"

namespace mxmoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kPhaseRaw = 2;
constexpr int KC = 128;        // k per stage = one weight group
constexpr int BM_MAX = 128;
constexpr int STAGE_BYTES = BM_MAX * 256;

// ------------------------------------------------------------ tile configs
// MF: 16-row fragments per tile (BM = 16 MF); NF: 16-channel fragments per
// wavefront and linear.  Accumulator registers per lane = 4 * MF * NF * NL.
__host__ __device__ constexpr int cfg_mf(int c) { return c == CFG_S ? 1 : (c == CFG_T ? 2 : (c == CFG_M ? 4 : 8)); }
__host__ __device__ constexpr int cfg_nf(int c, int phase) {
  return phase == 0 ? ((c == CFG_S || c == CFG_T) ? 4 : 2) : ((c == CFG_S || c == CFG_T) ? 8 : 4);
}
__host__ __device__ constexpr int cfg_bm(int c) { return 16 * cfg_mf(c); }
__host__ __device__ constexpr int cfg_bn(int c, int phase) { return 64 * cfg_nf(c, phase); }
// Tile configuration of a group from its rows; w4a4-g128 and mxfp4 groups stop
// at 64-row tiles (the per-group rescale keeps a partial sum next to every
// accumulator; the scaled FP4 MFMA adds its scale registers), and so do fp8
// groups outside the down phase (its two linears' 32-byte operands do not fit
// next to 128-row accumulators), which keeps every kernel within its register
// budget.  phase: 0 gate|up (and single linears), 1 down.
__host__ __device__ inline int pick_cfg(int m, int kind, int phase) {
  const int c = m <= 16 ? CFG_S : (m <= 32 ? CFG_T : (m <= 64 ? CFG_M : CFG_L));
  const bool cap = kind == K_W4A4G || kind == K_MXFP4 || (kind == K_F8A8 && phase != 1);
  return (cap && c == CFG_L) ? CFG_M : c;
}

// Super-tile geometry of a group of mt x nt tiles: sm x sn tiles per super-tile
// (sm = min(mt, 8), sn = min(nt, 64 / sm)), nsm x nsn super-tiles, super-tile
// s at (s % nsm, s / nsm); inside, tile t at (t % em, t / em) with em the
// super-tile's row tiles (the plan expands the queues in this order).
struct SuperDims { int sm, sn, nsm, nsn; };

// ---------------------------------------------------------- MFMA helpers
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
// fp32 -> activation dtype, round to nearest even (NaN stays NaN)
template <int ACT> __device__ inline uint16_t f32_to_act(float f) {
  if constexpr (ACT == MXMOE_BF16)
    return __builtin_bit_cast(uint16_t, (__bf16)f);
  else
    return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// SiLU(g) = g / (1 + e^-g), formed as g * rcp(1 + e^-g) with e^-g = 2^t,
// t = -g log2(e) rounded to fp32 and capped at 126 (a large negative g then
// yields a tiny finite value instead of inf * 0).  The rounding of t moves
// e^-g by at most |t| 2^-24 relatively, which with the exp2 and reciprocal
// instructions (about one ulp each) keeps the result within 2^-16 of the exact
// value for |g| < 64: far below the one rounding of h to the 16-bit
// activation dtype that follows.  silu_exp(g) = e^-g.
__device__ inline float silu_exp(float g) {
  return __builtin_amdgcn_exp2f(fminf(g * -1.44269502162933349609375f, 126.0f));
}

// ------------------------------------------------------- weight operands
// Low-bit kinds and w8a8 prefetch a whole 128-wide k block (8-32 bytes per
// lane); the 16-bit-operand wide kinds (w16, w8g: 32-64 bytes per lane) stream
// one MFMA step at a time.
template <int KD> constexpr bool streamed() { return KD == K_W16 || KD == K_W8G; }
template <int KD> struct Raw { u32x4 d[1]; };
template <> struct Raw<K_W2G> { u32x2 d; };
template <> struct Raw<K_W3G> { uint32_t d[3]; };
template <> struct Raw<K_W8A8> { u32x4 d[2]; };
template <> struct Raw<K_F8A8> { u32x4 d[2]; };
template <> struct Raw<K_W4A4F6> { u32x4 d0; u32x2 d1; };  // 24 bytes: 32 e2m3 codes

// loads through the global address space (the pointers come from the block
// table, so the compiler cannot infer it and would emit flat loads)
template <typename V> __device__ inline V gload(const void* p) {
  typedef __attribute__((address_space(1))) const V GV;
  return *(GV*)p;
}

template <int KD> __device__ inline void load_raw(Raw<KD>& r, const uint8_t* p) {
  if constexpr (KD == K_W2G) {
    r.d = gload<u32x2>(p);
  } else if constexpr (KD == K_W3G) {  // 12-byte lanes: 4-byte aligned
    r.d[0] = gload<uint32_t>(p);
    r.d[1] = gload<uint32_t>(p + 4);
    r.d[2] = gload<uint32_t>(p + 8);
  } else if constexpr (KD == K_W8A8 || KD == K_F8A8) {
    r.d[0] = gload<u32x4>(p);
    r.d[1] = gload<u32x4>(p + 16);
  } else if constexpr (KD == K_W4A4F6) {  // 24-byte lanes: 8-byte aligned
    r.d0 = gload<u32x4>(p);
    r.d1 = gload<u32x2>(p + 16);
  } else if constexpr (!streamed<KD>()) {
    r.d[0] = gload<u32x4>(p);
  }
}

// streamed kinds: the lane's bytes of MFMA step j
template <int KD> __device__ inline u32x4 load_step(const uint8_t* p, int j) {
  if constexpr (KD == K_W8G) {
    const u32x2 v = gload<u32x2>(p + 8 * j);
    return u32x4{v[0], v[1], 0u, 0u};
  } else {
    return gload<u32x4>(p + 16 * j);
  }
}

// Wait until at most N vector-memory loads of this wavefront are outstanding
// (loads complete in issue order), leaving LDS and export counters alone.
// An empty statement that reads a value: the compiler waits for the loads of
// its registers before it.
__device__ inline void touch(uint32_t v) { asm volatile("" ::"v"(v)); }
__device__ inline void touch(const u32x2& v) { asm volatile("" ::"v"(v)); }
__device__ inline void touch(const u32x4& v) { asm volatile("" ::"v"(v)); }
template <int KD> __device__ inline void touch_raw(const Raw<KD>& r) {
  if constexpr (KD == K_W2G) touch(r.d);
  else if constexpr (KD == K_W3G) { touch(r.d[0]); touch(r.d[1]); touch(r.d[2]); }
  else if constexpr (KD == K_W4A4F6) { touch(r.d0); touch(r.d1); }
  else if constexpr (KD == K_W8A8 || KD == K_F8A8) { touch(r.d[0]); touch(r.d[1]); }
  else touch(r.d[0]);
}

template <int N> __device__ inline void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for LDS hand-offs inside the k loop: waits for this
// wavefront's LDS operations only.  __syncthreads() carries a fence that also
// drains every outstanding global load, which would stall the weight prefetch;
// the direct-to-LDS stage loads are covered by wait_vmem before this barrier.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Device-scope coherent 16-byte store and load (scope bit sc1), used for
// partial sums that another XCD reads within the same launch.  The store is
// followed by wait states: the compiler, which does not look into the asm,
// may overwrite the data registers in the next instruction, and a store wider
// than 8 bytes still reads them then.  The load is asynchronous: wait_loaded()
// must run before its result is used.
__device__ inline void store_coherent(float* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" ::"v"(p), "v"(v) : "memory");
}
__device__ inline u32x4 load_coherent(const float* p) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// Wait for every outstanding vector-memory load; the registers of v are tied
// to the wait so that no use of them is scheduled before it.
template <int N> __device__ inline void wait_loaded(u32x4 (&v)[N]) {
  if constexpr (N == 1) asm volatile("s_waitcnt vmcnt(0)" : "+v"(v[0])::"memory");
  else if constexpr (N == 2) asm volatile("s_waitcnt vmcnt(0)" : "+v"(v[0]), "+v"(v[1])::"memory");
  else if constexpr (N == 4)
    asm volatile("s_waitcnt vmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3])::"memory");
  else {
    static_assert(N == 8, "fragment count");
    asm volatile("s_waitcnt vmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7])::"memory");
  }
}

// bias constant b = 2^N - 1 of the exact magic-number dequantization
template <int KD> constexpr int wbias() { return KD == K_W2G ? 3 : (KD == K_W3G ? 7 : 15); }

template <int ACT> __device__ inline uint32_t pack_exact(float lo, float hi) {
  if constexpr (ACT == MXMOE_BF16)  // small integers: truncation to bf16 is exact
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
  else
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
}

// 16-bit weight operand of MFMA step j (8 slots) for the lane's channel.
// bz: per-group constant (bias pair for 2/3/4-bit codes, zero point for 8-bit).
template <int KD, int ACT>
__device__ inline u32x4 wfrag16(const Raw<KD>& r, u32x4 step, int j, uint32_t bz, float zf) {
  u32x4 o;
  if constexpr (KD == K_W16) {
    o = step;
  } else if constexpr (KD == K_W8G) {
    const uint32_t a = step[0], b = step[1];
    o[0] = pack_exact<ACT>((float)(a & 0xFFu) - zf, (float)((a >> 8) & 0xFFu) - zf);
    o[1] = pack_exact<ACT>((float)((a >> 16) & 0xFFu) - zf, (float)(a >> 24) - zf);
    o[2] = pack_exact<ACT>((float)(b & 0xFFu) - zf, (float)((b >> 8) & 0xFFu) - zf);
    o[3] = pack_exact<ACT>((float)((b >> 16) & 0xFFu) - zf, (float)(b >> 24) - zf);
  } else {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t v;
      if constexpr (KD == K_W4G) {
        v = (r.d[0][j] >> (4 * p)) & 0x000F000Fu;
      } else if constexpr (KD == K_W2G) {
        const int P = 4 * (j & 1) + p;
        v = (r.d[j >> 1] >> (2 * P)) & 0x00030003u;
      } else {  // K_W3G
        const int P = 4 * (j & 1) + p, P3 = 4 * j + p;
        const uint32_t hi = (P3 >= 2 ? (r.d[2] >> (P3 - 2)) : (r.d[2] << (2 - P3))) & 0x00040004u;
        v = ((r.d[j >> 1] >> (2 * P)) & 0x00030003u) | hi;
      }
      v += bz;
      if constexpr (ACT == MXMOE_F16) {
        // fp16 1024 + b + (q - z)  ->  q - z, exact
        const f16x2 off = {(_Float16)(-(1024 + wbias<KD>())), (_Float16)(-(1024 + wbias<KD>()))};
        v = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, v) + off);
      }
      o[p] = v;
    }
  }
  return o;
}

// int8 weight operand of MFMA step j (16 slots)
template <int KD> __device__ inline i32x4 wfrag8(const Raw<KD>& r, u32x4 step, int j) {
  if constexpr (KD == K_W8A8) {
    return __builtin_bit_cast(i32x4, r.d[j]);
  } else {
    const uint32_t d0 = r.d[0][2 * j], d1 = r.d[0][2 * j + 1];
    i32x4 o;
    o[0] = (int)((d0 << 4) & 0xF0F0F0F0u);
    o[1] = (int)(d0 & 0xF0F0F0F0u);
    o[2] = (int)((d1 << 4) & 0xF0F0F0F0u);
    o[3] = (int)(d1 & 0xF0F0F0F0u);
    return o;
  }
}

// ------------------------------------------------------------- LDS stage
struct __align__(16) Smem {
  uint8_t act[2][STAGE_BYTES];   // activation rows of the tile, one 128-wide k block per stage
  float rsum[2][BM_MAX];         // per-row sums of a stage (bf16 weight-only kinds)
  int32_t rowsrc[BM_MAX];        // activation row index of every tile row
  int32_t rowout[BM_MAX];        // output row index of every tile row, -1 past the group's rows
  float rowscale[BM_MAX];        // per-token activation scale (a8/a4), else 1
  float rowgw[BM_MAX];           // router gate weight of the row's (token, slot) (down phase), else 1
  int4 entry;                    // the next tile (plan tile entry; group -1: none left)
  int32_t qtotal[kXcd];          // tiles per XCD queue
  int32_t qi;                    // queues tried so far by this workgroup
  int32_t last;                  // split-K: this workgroup finishes the output tile
  int32_t spec;                  // index claimed ahead on queue qi, or -1
  int32_t cur_idx;               // queue index of the tile in progress
  float wsc[512];                // per-channel weight scales of the tile's channels (a8/a4, FP8, FP6)
};

// Tile queues of one phase, rebuilt from the kernel arguments where needed so
// that no queue state stays in registers across a tile.  Thread 0 of a
// workgroup claims tiles: first from the queue of its own XCD, then from the
// others in turn once that is empty (sm.qi counts the queues tried).
struct TileQueue {
  int32_t* ctr;       // [kXcd][4] head counters (field 0)
  const int4* flat;   // [kXcd][fcap] tile entries
  int fcap;
  int x0;             // queue of this workgroup's XCD
};
__device__ inline TileQueue tile_queue(const GemmArgs& a, int pidx) {
  int32_t* plan = a.plan;
  asm volatile("" : "+s"(plan));  // recomputed here, not kept live from an earlier use
  const PlanLayout PL = plan_layout(a.G, a.qcap, a.fcap);
  TileQueue Q;
  Q.ctr = plan + PL.ctr + (int64_t)pidx * kXcd * 4;
  Q.flat = reinterpret_cast<const int4*>(plan + PL.flat) + (int64_t)pidx * kXcd * a.fcap;
  Q.fcap = a.fcap;
  Q.x0 = blockIdx.x % kXcd;  // workgroups are dealt round-robin over the XCDs
  return Q;
}
// claim the next index of the current queue (thread 0).  A queue whose head
// has already passed its tile count is skipped after a plain load: once the
// tiles run out, every workgroup would otherwise add to every head counter,
// and those same-address atomics serialize in L2 (hundreds per counter).
// Heads only grow, so a stale read can only cost one extra atomic.
__device__ inline int pop_start(const TileQueue& Q, const Smem& sm, int qi) {
  if (qi >= kXcd) return 0;
  const int x = (Q.x0 + qi) % kXcd;
  int32_t* c = &Q.ctr[x * 4];
  if (__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= sm.qtotal[x]) return 0x7fffffff;
  return atomicAdd(c, 1);
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Stage one k block of BM rows into act[buf] with direct global->LDS loads.
// A row's k block is RB bytes: 256 for 16-bit rows (16 chunks, chunk c stored
// at c ^ (r & 15)), 128 for int8 codes (8 chunks, at c ^ ((r >> 1) & 7)), 64
// for FP4 codes (4 chunks, at c ^ ((r >> 2) & 3)), so that the 16 rows one
// fragment read touches hit distinct banks.  One wavefront instruction fills
// 1 KB (4, 8 or 16 rows).  Wavefront w fills blocks w, w + 4, ...; its lanes'
// source offsets (row start + swizzled chunk, at k block 0) are computed once
// per tile.
template <int KD> constexpr int stage_rb() { return kind_is_mx(KD) ? 64 : (kind_is_int(KD) ? 128 : 256); }
template <int RB> __device__ constexpr int stage_swz(int c, int r) {
  return RB == 256 ? (c ^ (r & 15)) : (RB == 128 ? (c ^ ((r >> 1) & 7)) : (c ^ ((r >> 2) & 3)));
}
template <int RB_, int BM> struct StageOffs {
  static constexpr int RB = RB_;
  static constexpr int NBLK = BM * RB / 1024;
  static constexpr int PER_WAVE = (NBLK + 3) / 4;
  uint32_t off[PER_WAVE];
};

template <int RB, int BM>
__device__ inline void stage_offsets(StageOffs<RB, BM>& so, const Smem& sm, int64_t row_bytes, int wave, int lane) {
  using S = StageOffs<RB, BM>;
#pragma unroll
  for (int i = 0; i < S::PER_WAVE; ++i) {
    const int blk = wave + 4 * i;
    const int r = (blk < S::NBLK ? blk : 0) * (1024 / RB) + lane / (RB / 16);
    const int p = lane % (RB / 16);
    const int cc = stage_swz<RB>(p, r);
    so.off[i] = (uint32_t)((int64_t)sm.rowsrc[r] * row_bytes + cc * 16);
  }
}

// One direct global->LDS load of 16 bytes per lane: lane l's bytes at
// base + voff land at LDS address m0 + 16 l.  Issued through inline assembly
// so that the compiler's wait-counter pass does not treat every later LDS read
// as a possible reader of this stage (it would drain all outstanding global
// loads, weight prefetch included, before the first one); completion is
// waited for explicitly (wait_vmem) before the barrier that publishes the
// stage.
// The base address is uniform by construction.  With UP it passes through
// readfirstlane, so that the scalar operand does not depend on the compiler
// proving that; the mxfp4 tiles need it (without it the compiler keeps the
// base in a VGPR there), the others do without (the extra copies would cost
// registers across the whole kernel).
__device__ inline const uint8_t* uniform_ptr(const uint8_t* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}
template <bool UP = false> __device__ inline void lds_dma16(const uint8_t* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(UP ? uniform_ptr(base) : base), "s"(lds_addr)
               : "memory", "m0");
}

// The same load with device scope (sc1: past this XCD's L2), for partial sums
// that other XCDs stored with store_coherent (base made wave-uniform).
__device__ inline void lds_dma16_coherent(const uint8_t* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 sc1"
               :
               : "v"(voff), "s"(uniform_ptr(base)), "s"(lds_addr)
               : "memory", "m0");
}

// Claim the next tile and load its entry straight into sm.entry (thread 0;
// the caller waits for the load with its vector-memory count), or mark the
// end with group -1.  The first claim of a workgroup uses a plain load.
template <bool DMA> __device__ inline void claim_from(const TileQueue& Q, Smem& sm, int idx) {
  int qi = sm.qi;
  while (qi < kXcd) {
    const int x = (Q.x0 + qi) % kXcd;
    if (idx < sm.qtotal[x]) {
      sm.qi = qi;
      sm.cur_idx = idx;
      if constexpr (DMA) {
        const uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>((lds_ptr_t)&sm.entry);
        lds_dma16(reinterpret_cast<const uint8_t*>(Q.flat), (uint32_t)(((int64_t)x * Q.fcap + idx) * 16),
                  __builtin_amdgcn_readfirstlane(lds));
      } else {
        sm.entry = Q.flat[(int64_t)x * Q.fcap + idx];
      }
      return;
    }
    ++qi;
    idx = pop_start(Q, sm, qi);
  }
  sm.qi = qi;
  sm.entry.x = -1;  // only the group field is read when no tile is left
}
template <bool DMA> __device__ inline void claim_next(const TileQueue& Q, Smem& sm) {
  claim_from<DMA>(Q, sm, pop_start(Q, sm, sm.qi));
}
// A tile started while its queue still holds more than this many unclaimed
// tiles claims the next one at its start (the claim's round trips then hide
// behind the tile); near a queue's end the claim waits for the tile's end, so
// that no tile sits reserved by a busy workgroup while others run out.
constexpr int kClaimAheadMargin = 256;

// sub: sub-stage of the buffer (tiles that stage two k blocks per step put
// the second one's BM rows after the first one's)
template <int RB, int BM>
__device__ inline void stage_load(Smem& sm, int buf, const uint8_t* base, const StageOffs<RB, BM>& so, int kb,
                                  int wave, int sub = 0) {
  using S = StageOffs<RB, BM>;
  const uint8_t* bk = base + (int64_t)kb * S::RB;  // uniform
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>((lds_ptr_t)sm.act[buf]) + sub * BM * RB;
#pragma unroll
  for (int i = 0; i < S::PER_WAVE; ++i) {
    const int blk = wave + 4 * i;
    if (blk < S::NBLK) lds_dma16<RB == 64>(bk, so.off[i], __builtin_amdgcn_readfirstlane(lds0 + blk * 1024));
  }
}

template <int RB> __device__ inline u32x4 act_frag(const Smem& sm, int buf, int r, int cc) {
  return *reinterpret_cast<const u32x4*>(sm.act[buf] + r * RB + stage_swz<RB>(cc, r) * 16);
}

// Row sums of a stage (bias-dequantized kinds with bf16 activations): one
// direct global->LDS load of 4 bytes per lane brings the precomputed sums of
// rows 64w .. 64w + 63 of k block kb into sm.rsum[buf] (wavefronts
// w < ceil(BM / 64)); rsoff: the lane's row offset (bytes) at k block 0.
template <bool UP = false> __device__ inline void lds_dma4(const uint8_t* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(UP ? uniform_ptr(base) : base), "s"(lds_addr)
               : "memory", "m0");
}
// (sub-stage s of a tile of at most 64 rows takes rsum[buf][64 s ..])
template <int BM, bool UP = false>
__device__ inline void rowsum_load(Smem& sm, int buf, const float* rsbase, uint32_t rsoff, int kb, int wave,
                                   int sub = 0) {
  if (wave * 64 < BM) {
    const uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>((lds_ptr_t)&sm.rsum[buf][sub * 64 + wave * 64]);
    lds_dma4<UP>(reinterpret_cast<const uint8_t*>(rsbase + kb), rsoff, __builtin_amdgcn_readfirstlane(lds));
  }
}

// ---------------------------------------------------------- tile body
template <int KD, int ACT, int CFG, int PHASE>
__device__ __attribute__((always_inline)) inline void run_tile(Smem& sm, const GemmArgs& a, const DevExpert* ex, int g, int m_g, int mt, int ntv,
                                int off_e, int split) {
  constexpr int MF = cfg_mf(CFG);
  constexpr int NF = cfg_nf(CFG, PHASE == 0 ? 0 : 1);
  constexpr int NL = PHASE == 0 ? 2 : 1;
  constexpr bool INT = kind_is_int(KD);
  constexpr bool WONLY = kind_is_wonly(KD);
  constexpr bool MAGIC = WONLY && KD != K_W8G;          // 2/3/4-bit codes
  constexpr bool RSUM = MAGIC && ACT == MXMOE_BF16;     // bias removed through row sums
  constexpr bool GSC = KD == K_W4A4G;                   // per-128-group activation and weight scales
  constexpr bool MX = kind_is_mx(KD);                   // FP4 e2m1 operands with E8M0 scales per 32
  constexpr bool F8 = kind_is_f8(KD);                   // FP8 e4m3 operands, fp32 accumulation
  constexpr bool F6 = kind_is_f6(KD);                   // int4 codes as FP6 e2m3 operands, exact fp32 sums
  constexpr bool GMETA = kind_has_gmeta(KD);            // group metadata after each fragment block
  constexpr bool RSLOAD = RSUM || GSC || MX;            // a per-row value per k block rides with the stage
  constexpr int RB = stage_rb<KD>();                    // activation bytes per row and k block
  constexpr int BM = 16 * MF;
  constexpr int BN = 64 * NF;
  constexpr int LB = lane_bytes(KD);
  constexpr int BB = block_bytes(KD);
  constexpr float CB = (float)(128 + (MAGIC ? wbias<KD>() : 0));

  // Opaque thread id: keeps lane-derived values inside the tile body instead of
  // letting the persistent loop hoist them for every micro-kernel at once.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;  // wave index is uniform
  const int li = lane & 15, q = lane >> 4;
  const bool shared = g >= a.E_routed;
  const DevLinear* lins[NL];
  if constexpr (PHASE == 0) { lins[0] = &ex->lin[0]; lins[1] = &ex->lin[1]; }
  else if constexpr (PHASE == 1) { lins[0] = &ex->lin[2]; }
  else { lins[0] = &a.raw_lin; }
  const int N = lins[0]->n, K = lins[0]->k;
  const int kblocks = K / 128;
  // split-K: queued channel tile ntv = slice * (channel tiles) + channel tile;
  // the slice reduces k blocks [kb0, kb1), balanced so that every slice is
  // non-empty (the plan only slices when there are >= 6 k blocks per slice)
  const int ntr = (N + BN - 1) / BN;
  const int slice = split > 1 ? ntv / ntr : 0;
  const int nt = ntv - slice * ntr;
  const int kb0 = slice * kblocks / split;
  const int kb1 = (slice + 1) * kblocks / split;
  const int row0 = mt * BM;
  const int nb0 = (nt * BN) / 16 + wave * NF;   // first 16-channel block of this wavefront
  int nvalid = N / 16 - nb0;
  nvalid = nvalid < 0 ? 0 : (nvalid > NF ? NF : nvalid);

  const uint8_t* abase;
  const float* ascale = nullptr;
  if constexpr (MX) {
    abase = PHASE == 1 ? (shared ? a.hqmx_shared : a.hqmx) : a.xqmx;
  } else if constexpr (INT) {
    const int8_t* qb;
    if constexpr (PHASE == 1) { qb = shared ? a.hq_shared : a.hq; ascale = shared ? a.hs_shared : a.hs; }
    else {
      qb = F8 ? reinterpret_cast<const int8_t*>(a.xqf8)
              : (F6 ? reinterpret_cast<const int8_t*>(a.xqf6) : (KD == K_W8A8 ? a.xq8 : (GSC ? a.xq4g : a.xq4)));
      ascale = F8 ? a.xsf8 : (F6 ? a.xsf6 : (KD == K_W8A8 ? a.xs8 : a.xs4));
    }
    abase = reinterpret_cast<const uint8_t*>(qb);
  } else {
    abase = reinterpret_cast<const uint8_t*>(PHASE == 1 ? (shared ? a.h_shared : a.h) : a.x);
  }

  // ---- per-row data: activation source row (rows past the group repeat its
  // last row), output row, activation scale, router gate weight
  int spec = -1;
  if (tid == 0 && sm.qi < kXcd) {
    const TileQueue Q = tile_queue(a, PHASE == kPhaseRaw ? 0 : PHASE);
    const int x = (Q.x0 + sm.qi) % kXcd;
    if (sm.qtotal[x] - sm.cur_idx > kClaimAheadMargin) spec = atomicAdd(&Q.ctr[x * 4], 1);
  }
  if (tid < BM) {
    const int m0 = row0 + tid;
    const int m = m0 < m_g ? m0 : m_g - 1;
    int src, out;
    float gw = 1.f;
    float sc = 1.f;
    if constexpr (PHASE == 0) {
      src = shared ? m : a.rtok[off_e + m];
      out = shared ? (g - a.E_routed) * a.T + m : off_e + m;
      if constexpr (F8 || F6) sc = ascale[src];
      else if constexpr (INT && !GSC) sc = shared ? ascale[m] : (KD == K_W8A8 ? a.rxs8 : a.rxs4)[off_e + m];
    } else if constexpr (PHASE == 1) {
      src = shared ? (g - a.E_routed) * a.T + m : off_e + m;
      if (shared) {
        out = m * (a.k + a.n_shared) + a.k + (g - a.E_routed);
        if (a.shared_w) gw = a.shared_w[(int64_t)m * a.n_shared + (g - a.E_routed)];
      } else {
        out = a.rslot[off_e + m];
        gw = a.rgw[off_e + m];
      }
      if constexpr (INT && !GSC) sc = ascale[src];
    } else {
      src = m;
      out = m;
      if constexpr (INT && !GSC) sc = ascale[m];
    }
    sm.rowsrc[tid] = src;
    sm.rowout[tid] = m0 < m_g ? out : -1;
    sm.rowgw[tid] = gw;
    sm.rowscale[tid] = sc;
  }
  if constexpr (INT && !GSC) {  // the channels' weight scales, for the epilogue
    for (int i = tid; i < NL * BN; i += kThreads) {
      const int l = i / BN, c = i - l * BN;
      const int n = nt * BN + c;
      sm.wsc[i] = n < N ? lins[l]->wscale[n] : 0.f;
    }
  }
  const int64_t row_bytes = MX ? (int64_t)K / 2 : (int64_t)K * (INT ? 1 : 2);
  if (tid == 0) sm.spec = spec;
  __syncthreads();
  // the tile after this one, claimed ahead: its entry comes into LDS now (every
  // thread has read this tile's entry before the barrier above)
  if (tid == 0 && spec >= 0) claim_from<true>(tile_queue(a, PHASE == kPhaseRaw ? 0 : PHASE), sm, spec);
  StageOffs<RB, BM> soffs;
  stage_offsets<RB, BM>(soffs, sm, row_bytes, wave, lane);
  // row sums of the tile's activation rows per k block (bias-dequantized
  // kinds, bf16): x rows in the gate|up phase, h rows in the down phase
  const float* rsbase = nullptr;
  uint32_t rsoff = 0;
  if constexpr (RSLOAD) {
    // row sums (bias-dequantized kinds), activation group scales (w4a4-g128)
    // or the four E8M0 bytes of a row's k block (mxfp4)
    if constexpr (MX)
      rsbase = reinterpret_cast<const float*>(PHASE == 1 ? (shared ? a.hsmx_shared : a.hsmx) : a.xsmx);
    else if constexpr (GSC) rsbase = PHASE == 1 ? (shared ? a.hsg_shared : a.hsg) : a.xs4g;
    else rsbase = PHASE == 1 ? (shared ? a.rsh_shared : a.rsh) : a.rsx;
    const int r = wave * 64 + lane;
    rsoff = (uint32_t)sm.rowsrc[r < BM ? r : 0] * (uint32_t)kblocks * 4u;
  }

  // ---- accumulators and weight streams
  typedef typename std::conditional<INT && !GSC && !F8 && !F6, i32x4, f32x4>::type AccT;
  typedef typename std::conditional<INT, i32x4, u32x4>::type OpT;
  constexpr int J = MX ? 1 : (INT ? 2 : 4);      // MFMA steps per 128-wide k block
  constexpr bool HOLD_W = NL * NF <= MF;         // hold the smaller operand set in registers
  AccT acc[NL][NF][MF];
#pragma unroll
  for (int l = 0; l < NL; ++l)
#pragma unroll
    for (int nf = 0; nf < NF; ++nf)
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) acc[l][nf][mf] = AccT{0, 0, 0, 0};

  // Uniform base of every fragment's block stream (fragments past the last
  // channel block read block 0 and are never stored) and the lane's offset.
  const uint8_t* wp[NL][NF];
#pragma unroll
  for (int l = 0; l < NL; ++l)
#pragma unroll
    for (int nf = 0; nf < NF; ++nf)
      wp[l][nf] = lins[l]->packed + (int64_t)(nf < nvalid ? nb0 + nf : 0) * kblocks * BB;
  const uint32_t loff = (uint32_t)lane * LB;
  const uint32_t moff = 64u * LB + 4u * li;  // this lane's channel in the group metadata

  // Some tiles take two k blocks per step: both blocks' stages and weights
  // are in flight together, which doubles the prefetch distance and halves
  // the barriers per block.  Tiles of at most 32 rows with at most 16 weight
  // bytes per lane and block gain most (their MFMA work per block is too
  // small to hide one memory round trip); down tiles and integer / FP8
  // gate|up tiles gain a little at any size whose two-block stage fits one
  // stage buffer (1.5% on the gate|up launch of the Qwen2-shaped block);
  // 16-bit-activation gate/up tiles of more rows lose a little (their two
  // weight sets already fill the registers).
  // Slot s of the weight registers serves k block kb + s and is refilled
  // right after its MFMAs, for the next step (no register copy).  The per-row values of the
  // second block sit at rsum[buf][64..], so tiles with them stop at 64 rows.
  constexpr bool KBI_FITS = !streamed<KD>() && BM * RB * 2 <= STAGE_BYTES && (!RSLOAD || BM <= 64);
  constexpr int KBI = (KBI_FITS && (PHASE == 1 || (BM <= 32 && LB <= 16) || INT)) ? 2 : 1;
  static_assert(KBI == 1 || KBI_FITS, "two-block stage layout");
  Raw<KD> raw[KBI][NL][NF];   // low-bit kinds: next group(s), prefetched a step ahead
  u32x4 st[J][NL][NF];   // streamed kinds: step j of the k block, reloaded one block ahead
  uint32_t meta[KBI][NL][NF];
  float s_prev[NL][NF];
  // The prefetch of block kn is issued unconditionally: past the last block
  // (last = true) every lane reads the first 16 bytes of the fragment's block 0
  // instead (one cache line, result unused), so no register keeps two possible
  // values across the loop and no copy has to wait for an outstanding load.
  auto load_group = [&](auto S, int kn, bool last) {
    constexpr int SL = decltype(S)::value;
    const uint32_t lo = last ? 0u : loff, mo = last ? 0u : moff;
#pragma unroll
    for (int l = 0; l < NL; ++l)
#pragma unroll
      for (int nf = 0; nf < NF; ++nf) {
        const uint8_t* blk = wp[l][nf] + (last ? 0 : (int64_t)kn * BB);  // uniform
        if constexpr (!streamed<KD>()) load_raw<KD>(raw[SL][l][nf], blk + lo);
        if constexpr (GMETA) meta[SL][l][nf] = gload<uint32_t>(blk + mo);
      }
  };
  auto load_steps = [&](int kn, bool last, int j) {
    const uint32_t lo = last ? 0u : loff;
#pragma unroll
    for (int l = 0; l < NL; ++l)
#pragma unroll
      for (int nf = 0; nf < NF; ++nf)
        st[j][l][nf] = load_step<KD>(wp[l][nf] + (last ? 0 : (int64_t)kn * BB) + lo, j);
  };
  // Vector-memory loads issued after the activation stage (and its row sums) of
  // the next k block,
  // at least: one per fragment and step (streamed), one per fragment (group
  // prefetch; two 16-byte loads for w8a8), plus one metadata dword per fragment
  // (weight-only).  Waiting for
  // this many leaves the weight prefetch in flight across the barrier.
  constexpr int kLoadsAfterStage =
      NL * NF * (streamed<KD>() ? J : ((KD == K_W8A8 || KD == K_F8A8 || KD == K_W4A4F6) ? 2 : 1)) + (GMETA ? NL * NF : 0);

  stage_load<RB, BM>(sm, 0, abase, soffs, kb0, wave);
  if constexpr (RSLOAD) rowsum_load<BM, MX>(sm, 0, rsbase, rsoff, kb0, wave);
  if constexpr (KBI == 2) {
    if (kb0 + 1 < kb1) {
      stage_load<RB, BM>(sm, 0, abase, soffs, kb0 + 1, wave, 1);
      if constexpr (RSLOAD) rowsum_load<BM, MX>(sm, 0, rsbase, rsoff, kb0 + 1, wave, 1);
    }
  }
  load_group(std::integral_constant<int, 0>{}, kb0, false);
  if constexpr (KBI == 2) load_group(std::integral_constant<int, 1>{}, kb0 + 1, kb0 + 1 >= kb1);
  if constexpr (streamed<KD>()) {
#pragma unroll
    for (int j = 0; j < J; ++j) load_steps(kb0, false, j);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int kb = kb0, it = 0; kb < kb1; kb += KBI, ++it) {
    const int cur = it & 1;
    const bool more = kb + KBI < kb1;
    // The weights of the step (prefetched during the previous one) are waited
    // for here, before the stage loads below go out: the compiler does not
    // count those direct loads, so a wait it placed after them for an older
    // load would wait for them too (vector-memory loads complete in order).
    if constexpr (!streamed<KD>()) {
#pragma unroll
      for (int l = 0; l < NL; ++l)
#pragma unroll
        for (int nf = 0; nf < NF; ++nf) {
          touch_raw<KD>(raw[0][l][nf]);
          if constexpr (GMETA) touch(meta[0][l][nf]);
          if constexpr (KBI == 2) {
            touch_raw<KD>(raw[KBI - 1][l][nf]);
            if constexpr (GMETA) touch(meta[KBI - 1][l][nf]);
          }
        }
    }
#pragma unroll
    for (int sb = 0; sb < KBI; ++sb) {
      if (kb + KBI + sb < kb1) {
        stage_load<RB, BM>(sm, cur ^ 1, abase, soffs, kb + KBI + sb, wave, sb);
        if constexpr (RSLOAD) rowsum_load<BM, MX>(sm, cur ^ 1, rsbase, rsoff, kb + KBI + sb, wave, sb);
      }
    }
    // every weight load below is issued after the stage (see wait_vmem)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    // one k block (kbs = kb + SL) of the step; an inactive block (the second
    // one past the last k block) issues only what every path through the step
    // issues, so the compiler's wait counts need no drain where paths join
    auto kstep = [&](auto S, bool active) {
    constexpr int SL = decltype(S)::value;
    const int kbs = kb + SL;
    const int ra = SL * BM;   // first staged row of this k block
    const int rs0 = SL * 64;  // its per-row values
    if (active) {
    Raw<KD> rw[NL][NF];
    uint32_t bz[NL][NF];
    float zf[NL][NF];
    float wsc[NL][NF];  // w4a4-g128: the channel's weight scale of this group / 16
    uint32_t wsx[NL][NF];  // mxfp4: the E8M0 byte of this lane's 32-wide block
#pragma unroll
    for (int l = 0; l < NL; ++l)
#pragma unroll
      for (int nf = 0; nf < NF; ++nf) {
        if constexpr (!GSC && KBI == 1) rw[l][nf] = raw[0][l][nf];
        bz[l][nf] = 0;
        zf[l][nf] = 0.f;
        wsc[l][nf] = 0.f;
        wsx[l][nf] = 0u;
        if constexpr (MX) wsx[l][nf] = (meta[SL][l][nf] >> (8 * q)) & 0xFFu;
        if constexpr (GSC)  // (the 1/16 undoes the x16 of the widened nibbles, exactly)
          wsc[l][nf] = (float)__builtin_bit_cast(_Float16, (uint16_t)(meta[SL][l][nf] & 0xFFFFu)) * 0.0625f;
        if constexpr (WONLY) {
          const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(meta[SL][l][nf] & 0xFFFFu));
          const float z = (float)__builtin_bit_cast(_Float16, (uint16_t)(meta[SL][l][nf] >> 16));
          zf[l][nf] = z;
          if constexpr (MAGIC) {
            const uint32_t base = ACT == MXMOE_BF16 ? 0x43004300u : 0x64006400u;
            bz[l][nf] = base + (uint32_t)(wbias<KD>() - (int)z) * 0x00010001u;
          }
          // move the running sum into units of this group's scale
          const float r = kbs != kb0 ? s_prev[l][nf] * __builtin_amdgcn_rcpf(s) : 0.f;
          s_prev[l][nf] = s;
#pragma unroll
          for (int mf = 0; mf < MF; ++mf) {
            f32x4 cr = {0, 0, 0, 0};
            if constexpr (RSUM) cr = *reinterpret_cast<const f32x4*>(&sm.rsum[cur][rs0 + mf * 16 + 4 * q]) * (-CB);
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[l][nf][mf][i] = __builtin_fmaf(acc[l][nf][mf][i], r, cr[i]);
          }
        }
      }
    // w4a4-g128 decodes the whole k block's weight fragments here, before the
    // prefetch reuses their registers
    OpT gwf[GSC ? J : 1][NL][NF];
    if constexpr (GSC) {
#pragma unroll
      for (int j = 0; j < J; ++j)
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) gwf[j][l][nf] = wfrag8<KD>(raw[SL][l][nf], u32x4{0u, 0u, 0u, 0u}, j);
    }
    if constexpr (KBI == 1) {
      load_group(S, kb + 1, !more);
      // keep the prefetch here: the scheduler would otherwise sink it below the
      // MFMAs, next to its first use
      __builtin_amdgcn_sched_barrier(0);
    }
    // the weight operands of this k block: the copy (one step per block), or
    // the slot itself, refilled only after the MFMAs below
    auto& wr = [&]() -> Raw<KD>(&)[NL][NF] {
      if constexpr (KBI == 1) return rw;
      else return raw[SL];
    }();

    if constexpr (MX) {
      // mxfp4: one scaled FP4 MFMA per (row fragment, channel fragment) covers
      // the whole k block; lane l's operands are 32 consecutive elements of its
      // row (channel) with the E8M0 scale of that 32-wide block
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        const u32x4 af = act_frag<RB>(sm, cur, ra + mf * 16 + li, q);
        const int sa = (int)((__float_as_uint(sm.rsum[cur][rs0 + mf * 16 + li]) >> (8 * q)) & 0xFFu);
        const i32x8 A = {(int)af[0], (int)af[1], (int)af[2], (int)af[3], 0, 0, 0, 0};
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) {
            const u32x4 w = wr[l][nf].d[0];
            const i32x8 B = {(int)w[0], (int)w[1], (int)w[2], (int)w[3], 0, 0, 0, 0};
            acc[l][nf][mf] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(A, B, acc[l][nf][mf], 4, 4, 0, sa, 0,
                                                                             (int)wsx[l][nf]);
          }
      }
    } else if constexpr (F8) {
      // FP8: one 16x16x128 FP8 MFMA per (row fragment, channel fragment)
      // covers the k block.  A lane's 32 bytes are the two 16-byte pieces of
      // the int8 lane layout (k = 16q.. and 64 + 16q..) on both operands, so
      // both name the same k for every byte position and the dot product is
      // that of the k block.  Unit scales (E8M0 127) on both operands.
      i32x8 A[MF];
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        const u32x4 a0 = act_frag<RB>(sm, cur, ra + mf * 16 + li, q);
        const u32x4 a1 = act_frag<RB>(sm, cur, ra + mf * 16 + li, 4 + q);
        A[mf] = i32x8{(int)a0[0], (int)a0[1], (int)a0[2], (int)a0[3], (int)a1[0], (int)a1[1], (int)a1[2], (int)a1[3]};
      }
#pragma unroll
      for (int mf = 0; mf < MF; ++mf)
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) {
            const u32x4 w0 = wr[l][nf].d[0], w1 = wr[l][nf].d[1];
            const i32x8 B = {(int)w0[0], (int)w0[1], (int)w0[2], (int)w0[3], (int)w1[0], (int)w1[1], (int)w1[2], (int)w1[3]};
            acc[l][nf][mf] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(A[mf], B, acc[l][nf][mf], 0, 0, 0, 127, 0, 127);
          }
      // the activation fragments two row fragments ahead of the MFMAs (two
      // LDS reads each), so that few of them are live at once
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        __builtin_amdgcn_sched_group_barrier(0x008, NL * NF, 0);
        if (mf + 2 < MF) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
    } else if constexpr (F6) {
      // w4a4 on FP6 operands: one 16x16x128 FP6 MFMA per (row fragment,
      // channel fragment) covers the k block.  Lane (li, q) holds k = 32q ..
      // 32q + 31: for its row the first 24 bytes of the staged row's 32-byte
      // group q (chunk 2q and the low half of chunk 2q + 1), for its channel
      // the packed lane's 24 bytes.  Unit scales (E8M0 127) on both operands.
      i32x8 A[MF];
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        const u32x4 a0 = act_frag<RB>(sm, cur, ra + mf * 16 + li, 2 * q);
        const u32x4 a1 = act_frag<RB>(sm, cur, ra + mf * 16 + li, 2 * q + 1);
        A[mf] = i32x8{(int)a0[0], (int)a0[1], (int)a0[2], (int)a0[3], (int)a1[0], (int)a1[1], 0, 0};
      }
#pragma unroll
      for (int mf = 0; mf < MF; ++mf)
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) {
            const u32x4 w0 = wr[l][nf].d0;
            const u32x2 w1 = wr[l][nf].d1;
            const i32x8 B = {(int)w0[0], (int)w0[1], (int)w0[2], (int)w0[3], (int)w1[0], (int)w1[1], 0, 0};
            acc[l][nf][mf] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(A[mf], B, acc[l][nf][mf], 2, 2, 0, 127, 0, 127);
          }
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        __builtin_amdgcn_sched_group_barrier(0x008, NL * NF, 0);
        if (mf + 2 < MF) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
    } else if constexpr (GSC) {
      // w4a4-g128: per row fragment, the two MFMA steps of this k block give an
      // exact int32 block sum, which enters the fp32 accumulator scaled by the
      // row's activation scale and the channel's weight scale of the block
      auto& wf = gwf;
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        OpT af[J];
#pragma unroll
        for (int j = 0; j < J; ++j)
          af[j] = __builtin_bit_cast(OpT, act_frag<RB>(sm, cur, ra + mf * 16 + li, 4 * j + q));
        const f32x4 sa = *reinterpret_cast<const f32x4*>(&sm.rsum[cur][rs0 + mf * 16 + 4 * q]);
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) {
            i32x4 p = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[0], wf[0][l][nf], i32x4{0, 0, 0, 0}, 0, 0, 0);
#pragma unroll
            for (int j = 1; j < J; ++j) p = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[j], wf[j][l][nf], p, 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
              acc[l][nf][mf][i] = __builtin_fmaf((float)p[i], sa[i] * wsc[l][nf], acc[l][nf][mf][i]);
          }
      }
    } else {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      auto wop = [&](int l, int nf) -> OpT {
        const u32x4 sv = streamed<KD>() ? st[j][l][nf] : u32x4{0u, 0u, 0u, 0u};
        if constexpr (INT) return wfrag8<KD>(wr[l][nf], sv, j);
        else return wfrag16<KD, ACT>(wr[l][nf], sv, j, bz[l][nf], zf[l][nf]);
      };
      auto aop = [&](int mf) -> OpT {
        return __builtin_bit_cast(OpT, act_frag<RB>(sm, cur, ra + mf * 16 + li, 4 * j + q));
      };
      auto mma = [&](const OpT& af, const OpT& wf, AccT c) -> AccT {
        if constexpr (INT) return __builtin_amdgcn_mfma_i32_16x16x64_i8(af, wf, c, 0, 0, 0);
        else return mfma16<ACT>(af, wf, c);
      };
      if constexpr (HOLD_W) {
        OpT wf[NL][NF];
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) wf[l][nf] = wop(l, nf);
        OpT af[MF];
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) af[mf] = aop(mf);
#pragma unroll
        for (int mf = 0; mf < MF; ++mf)
#pragma unroll
          for (int l = 0; l < NL; ++l)
#pragma unroll
            for (int nf = 0; nf < NF; ++nf) acc[l][nf][mf] = mma(af[mf], wf[l][nf], acc[l][nf][mf]);
        // Software pipeline of the activation fragments: two LDS reads ahead,
        // then the MFMAs of one fragment and the read of the fragment two
        // places further, so an MFMA group never waits for a read issued just
        // before it (16-bit MFMA kinds: per MFMA step; the integer kinds over
        // all steps of the k block, below).
        if constexpr (!INT) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
          for (int mf = 0; mf < MF; ++mf) {
            __builtin_amdgcn_sched_group_barrier(0x008, NL * NF, 0);
            if (mf + 2 < MF) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
        }
      } else {
        OpT af[MF];
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) af[mf] = aop(mf);
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) {
            const OpT wf = wop(l, nf);
#pragma unroll
            for (int mf = 0; mf < MF; ++mf) acc[l][nf][mf] = mma(af[mf], wf, acc[l][nf][mf]);
          }
      }
      if constexpr (streamed<KD>()) {
        // step j's registers are free: refill them with step j of the next block
        load_steps(kb + 1, !more, j);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if constexpr (HOLD_W && INT) {
      // the activation fragments of all MFMA steps of the k block in one
      // pipeline, three reads ahead, with no drain between steps (with the
      // weight decode of 16-bit MFMA kinds in flight too, the fp16 kernel spilled)
      constexpr int T = J * MF, LA = 3;
      __builtin_amdgcn_sched_group_barrier(0x100, LA, 0);
#pragma unroll
      for (int t = 0; t < T; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, NL * NF, 0);
        if (t + LA < T) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    }
    }
    }  // active
    if constexpr (KBI == 2) {
      // this slot's registers are free: prefetch its block of the next step
      load_group(S, kbs + KBI, kbs + KBI >= kb1);
      __builtin_amdgcn_sched_barrier(0);
    }
    };  // kstep
    kstep(std::integral_constant<int, 0>{}, true);
    if constexpr (KBI == 2) kstep(std::integral_constant<int, 1>{}, kb + 1 < kb1);
    // The next stages have landed once no more than the weight prefetch is
    // outstanding (vector-memory loads complete in issue order; when more
    // steps follow, every k block of this one issued its prefetch).
    if (more) wait_vmem<kLoadsAfterStage * KBI>();
    else wait_vmem<0>();
    lds_barrier();
  }

  // Claim the next tile, unless it was claimed ahead at the start of this one,
  // and bring its entry into LDS (read at the top of the tile loop, after the
  // final barrier).  Its loads are waited for before the next barrier of the
  // split-K hand-off or the epilogue.  Claiming here and not inside the k loop
  // keeps the claim's pending loads out of the loop: the compiler would
  // otherwise drain every outstanding load, the prefetch of the next k blocks
  // included, at the top of each step.
  if (tid == 0 && sm.spec < 0) claim_next<true>(tile_queue(a, PHASE == kPhaseRaw ? 0 : PHASE), sm);

  // ---- split-K: partial sums of this slice; the last slice to arrive adds
  // all slices' partials in slice order and runs the epilogue
  bool finish = true;
  if (split > 1) {
    if constexpr (WONLY) {  // partials carry their last group's scale
#pragma unroll
      for (int l = 0; l < NL; ++l)
#pragma unroll
        for (int nf = 0; nf < NF; ++nf) {
#pragma unroll
          for (int mf = 0; mf < MF; ++mf) acc[l][nf][mf] = acc[l][nf][mf] * s_prev[l][nf];
          s_prev[l][nf] = 1.f;
        }
    }
    constexpr int AREA = BM * BN * NL;  // floats per slice of one output tile
    const int pidx = PHASE == kPhaseRaw ? 0 : PHASE;
    const PlanLayout PL = plan_layout(a.G, a.qcap, a.fcap);
    const int32_t* rec = a.plan + PL.rec + ((int64_t)pidx * a.G + g) * PF_N;
    const int otile = mt * ntr + nt;
    int32_t* cnt = a.plan + PL.cnt + (int64_t)pidx * kSplitExtra + rec[PF_CBASE] + otile;
    float* part = a.partial + rec[PF_PBASE] + (int64_t)otile * split * AREA;
    auto at_of = [&](int l, int nf, int mf) {  // this lane's 16 bytes of a fragment
      return ((((wave * NL + l) * NF + nf) * MF + mf) * 64 + lane) * 4;
    };
    // The partials are stored and loaded with device-scope coherent accesses
    // (write-through past this XCD's L2, and re-fetched on the reading side),
    // so that slices run on different XCDs see each other's sums without
    // writing back or invalidating whole L2 caches.
#pragma unroll
    for (int l = 0; l < NL; ++l)
#pragma unroll
      for (int nf = 0; nf < NF; ++nf)
#pragma unroll
        for (int mf = 0; mf < MF; ++mf)
          store_coherent(part + (int64_t)slice * AREA + at_of(l, nf, mf), __builtin_bit_cast(u32x4, acc[l][nf][mf]));
    wait_vmem<0>();  // this wavefront's partials are written
    __syncthreads();
    if (tid == 0) sm.last = atomicAdd(cnt, 1) == split - 1;
    __syncthreads();
    finish = sm.last;
    if (finish) {
      // every slice (this one included) is read back and summed in slice
      // order, so the result does not depend on which slice finished last.
      if constexpr (PHASE == 1) {
        // Down tiles (the deep reductions that get many slices) read through
        // the stage buffers (free after the k loop), 16 KB per wavefront: a
        // unit is one slice of one fragment column (MF loads of 1 KB, straight
        // into LDS), and QU units are in flight while the oldest is added from
        // LDS, so that their memory round trips overlap.  (In the gate|up
        // kernels the extra code measured 0.5% slower on unsliced tiles.)
        constexpr int QU = (16 / MF) < 4 ? (16 / MF) : 4;
        const uint32_t ldsw = (uint32_t)reinterpret_cast<uintptr_t>((lds_ptr_t)sm.act[0]) + wave * 16384;
        const uint8_t* pbase = reinterpret_cast<const uint8_t*>(part);
        const int nunits = NL * NF * split;
        auto issue = [&](int u) {  // unit u = (column, slice) into slot u % QU
          const int col = u / split, sl = u - col * split;
          const int l = col / NF, nf = col - l * NF;
          const uint32_t slot = ldsw + (uint32_t)((u % QU) * MF) * 1024u;
#pragma unroll
          for (int mf = 0; mf < MF; ++mf)
            lds_dma16_coherent(pbase, (uint32_t)(((int64_t)sl * AREA + at_of(l, nf, mf)) * 4),
                               __builtin_amdgcn_readfirstlane(slot + mf * 1024u));
        };
        for (int u = 0; u < QU && u < nunits; ++u) issue(u);
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf)
            for (int sl = 0; sl < split; ++sl) {
              const int u = (l * NF + nf) * split + sl;
              const int newer = (u + QU < nunits ? u + QU : nunits) - u - 1;  // units issued after u
              if (newer >= 3) wait_vmem<3 * MF>();
              else if (newer == 2) wait_vmem<2 * MF>();
              else if (newer == 1) wait_vmem<MF>();
              else wait_vmem<0>();
              const uint8_t* src = reinterpret_cast<const uint8_t*>(sm.act[0]) + wave * 16384 + (u % QU) * MF * 1024;
#pragma unroll
              for (int mf = 0; mf < MF; ++mf) {
                const u32x4 v = *reinterpret_cast<const u32x4*>(src + mf * 1024 + lane * 16);
                acc[l][nf][mf] = sl == 0 ? __builtin_bit_cast(AccT, v) : acc[l][nf][mf] + __builtin_bit_cast(AccT, v);
              }
              // the slot's LDS reads are done (their values are in acc) before
              // the next unit's loads overwrite it
              asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
              if (u + QU < nunits) issue(u + QU);
            }
        __syncthreads();  // every wavefront is done with the stage buffers before the epilogue uses them
      } else {
#pragma unroll
        for (int l = 0; l < NL; ++l)
#pragma unroll
          for (int nf = 0; nf < NF; ++nf)
            for (int sl = 0; sl < split; ++sl) {
              u32x4 v[MF];
#pragma unroll
              for (int mf = 0; mf < MF; ++mf) v[mf] = load_coherent(part + (int64_t)sl * AREA + at_of(l, nf, mf));
              wait_loaded<MF>(v);
#pragma unroll
              for (int mf = 0; mf < MF; ++mf)
                acc[l][nf][mf] = sl == 0 ? __builtin_bit_cast(AccT, v[mf]) : acc[l][nf][mf] + __builtin_bit_cast(AccT, v[mf]);
            }
      }
      if (tid == 0) *cnt = 0;  // ready for the next forward
    }
  }

  // ---- epilogue: lane holds rows 4q + i of fragment mf, channel li of fragment nf
  // (the per-row data is re-read from LDS for every row fragment: holding it
  // for all fragments would cost 64-96 registers next to the accumulators)
  const bool full = row0 + BM <= m_g;  // uniform: no row of the tile lies past the group
  // gate|up with a bias-dequantized down projection (bf16): the tile also
  // writes the row sums of its h values per 128-wide block, which the down
  // phase subtracts (the tile's channels are whole blocks: BN is 128 or 256)
  float* rsh_out = nullptr;
  if constexpr (PHASE == 0 && ACT == MXMOE_BF16) {
    // (the kind is read as a wave-uniform value: the branch around the barrier
    // below must not look divergent to the compiler)
    if (kind_is_magic(__builtin_amdgcn_readfirstlane(ex->lin[2].kind))) rsh_out = shared ? a.rsh_shared : a.rsh;
  }
  auto epilogue = [&](auto guard) {
    constexpr bool GUARD = decltype(guard)::value;
    float cs[NL][NF];
#pragma unroll
    for (int nf = 0; nf < NF; ++nf)
#pragma unroll
      for (int l = 0; l < NL; ++l) {
        cs[l][nf] = 1.f;
        if constexpr (INT && !GSC) cs[l][nf] = sm.wsc[l * BN + (wave * NF + nf) * 16 + li];
        if constexpr (WONLY) cs[l][nf] = s_prev[l][nf];
      }
    // value of accumulator (l, nf, mf, i) after the scheme's scales
    auto outv = [&](int l, int nf, int mf, int i, const f32x4& rs) -> float {
      if constexpr (F8 || F6) {
        return (acc[l][nf][mf][i] * rs[i]) * cs[l][nf];
      } else if constexpr (INT && !GSC) {
        int iv = acc[l][nf][mf][i];
        if constexpr (KD == K_W4A4) iv >>= 4;  // exact: every product is a multiple of 16
        return ((float)iv * rs[i]) * cs[l][nf];
      } else {
        return acc[l][nf][mf][i] * cs[l][nf];
      }
    };
    if constexpr (PHASE == 0) {
      // h = SiLU(g) u of the tile goes to LDS first (rows of BN values, the
      // idle stage buffers), then out in 16-byte row pieces; the h row sums of
      // a bias-dequantized down projection are added from the same LDS rows
      constexpr int HP = BN + 8;  // row pitch in elements (16-byte pad: reads of 16 rows hit distinct banks)
      static_assert(BM * HP * 2 <= 2 * STAGE_BYTES, "h tile fits the stage buffers");
      uint16_t* hl = reinterpret_cast<uint16_t*>(&sm.act[0][0]);
      // (channels past N are computed too, without a branch per fragment,
      // and never stored; each fragment's four values go through the SiLU in
      // step, so that four independent chains hide each other's latencies)
#pragma unroll
      for (int mf = 0; mf < MF; ++mf) {
        const int r = mf * 16 + 4 * q;
        const f32x4 rs = *reinterpret_cast<const f32x4*>(&sm.rowscale[r]);
#pragma unroll
        for (int nf = 0; nf < NF; ++nf) {
          const int c = (wave * NF + nf) * 16 + li;
          float gv[4], uv[4], ev[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            gv[i] = outv(0, nf, mf, i, rs);
            uv[i] = outv(1, nf, mf, i, rs);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) ev[i] = silu_exp(gv[i]);
#pragma unroll
          for (int i = 0; i < 4; ++i) ev[i] = __builtin_amdgcn_rcpf(1.0f + ev[i]);
#pragma unroll
          for (int i = 0; i < 4; ++i) hl[(r + i) * HP + c] = f32_to_act<ACT>((gv[i] * ev[i]) * uv[i]);
        }
      }
      wait_vmem<0>();  // the next tile's entry has landed
      lds_barrier();
      constexpr int CH = BN / 8;  // 16-byte pieces of a tile row
      int nch = (N - nt * BN) / 8;
      nch = nch > CH ? CH : nch;
      uint16_t* hout = reinterpret_cast<uint16_t*>(shared ? a.h_shared : a.h);
      for (int idx = tid; idx < BM * CH; idx += kThreads) {
        const int r = idx / CH, c = idx % CH;
        const int ro = sm.rowout[r];
        if (ro >= 0 && c < nch)
          *reinterpret_cast<u32x4*>(hout + (int64_t)ro * N + nt * BN + 8 * c) =
              *reinterpret_cast<const u32x4*>(hl + r * HP + 8 * c);
      }
      if (rsh_out) {  // one thread per (row, 128-wide block): its 128 bf16 values in order
        constexpr int KBT = BN / 128;
        const int nkb = N / 128;
        for (int idx = tid; idx < BM * KBT; idx += kThreads) {
          const int r = idx % BM, j = idx / BM;
          const int kbg = nt * KBT + j;
          const int ro = sm.rowout[r];
          if (ro < 0 || kbg >= nkb) continue;
          float t = 0.f;
#pragma unroll
          for (int c8 = 0; c8 < 16; ++c8) {
            const u32x4 p = *reinterpret_cast<const u32x4*>(hl + r * HP + 128 * j + 8 * c8);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              t += __uint_as_float(p[e] << 16);
              t += __uint_as_float(p[e] & 0xFFFF0000u);
            }
          }
          rsh_out[(int64_t)ro * nkb + kbg] = t;
        }
      }
    } else if constexpr (PHASE == 1) {
      // The tile's slot rows (value x router gate weight) go through LDS (the
      // idle stage buffers), RP rows at a time, and leave as 16-byte pieces of
      // whole rows: a store instruction writes 64 x 16 contiguous bytes
      // instead of 16-lane segments of four rows.  Slot rows are rounded once
      // to the activation dtype (a.slot16, the default), or kept in fp32.
      if (a.slot16) {
        constexpr int HP = BN + 8;                  // row pitch in elements (16-byte pad against bank conflicts)
        constexpr int RP = (BM >= 64 && 64 * HP * 2 <= 2 * STAGE_BYTES) ? 64 : BM;  // rows per pass
        static_assert(RP * HP * 2 <= 2 * STAGE_BYTES, "slot rows fit the stage buffers");
        uint16_t* hl = reinterpret_cast<uint16_t*>(&sm.act[0][0]);
        constexpr int CH = BN / 8;                  // 16-byte pieces of a tile row
        int nch = (N - nt * BN) / 8;
        nch = nch > CH ? CH : nch;
        uint16_t* sout = reinterpret_cast<uint16_t*>(a.slots);
#pragma unroll
        for (int pass = 0; pass < BM / RP; ++pass) {
#pragma unroll
          for (int mf = 0; mf < MF; ++mf) {
            if ((mf * 16) / RP != pass) continue;
            const int r = mf * 16 + 4 * q;
            const f32x4 rs = *reinterpret_cast<const f32x4*>(&sm.rowscale[r]);
            const f32x4 gwv = *reinterpret_cast<const f32x4*>(&sm.rowgw[r]);
#pragma unroll
            for (int nf = 0; nf < NF; ++nf) {  // (channels past N: written, never stored)
              const int c = (wave * NF + nf) * 16 + li;
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                // the fp32 product is rounded first, then converted: the
                // barrier keeps the compiler from fusing the multiply into a
                // mixed-precision instruction that rounds once to fp16
                float v = outv(0, nf, mf, i, rs) * gwv[i];
                asm volatile("" : "+v"(v));
                hl[(r + i - pass * RP) * HP + c] = f32_to_act<ACT>(v);
              }
            }
          }
          if (pass == 0) wait_vmem<0>();  // the next tile's entry has landed
          lds_barrier();
          for (int idx = tid; idx < RP * CH; idx += kThreads) {
            const int r = idx / CH, c = idx % CH;
            const int ro = sm.rowout[pass * RP + r];
            if (ro >= 0 && c < nch)
              *reinterpret_cast<u32x4*>(sout + (int64_t)ro * N + nt * BN + 8 * c) =
                  *reinterpret_cast<const u32x4*>(hl + r * HP + 8 * c);
          }
          lds_barrier();
        }
      } else {
      constexpr int FP = BN + 4;                  // row pitch in floats (16-byte pad against bank conflicts)
      constexpr int RP = (BM >= 32 && 32 * FP * 4 <= 2 * STAGE_BYTES) ? 32 : 16;  // rows per pass
      static_assert(RP * FP * 4 <= 2 * STAGE_BYTES, "slot rows fit the stage buffers");
      float* fl = reinterpret_cast<float*>(&sm.act[0][0]);
      constexpr int CH = BN / 4;                  // 16-byte pieces of a tile row
      int nch = (N - nt * BN) / 4;
      nch = nch > CH ? CH : nch;
#pragma unroll
      for (int pass = 0; pass < BM / RP; ++pass) {
#pragma unroll
        for (int mf = 0; mf < MF; ++mf) {
          if ((mf * 16) / RP != pass) continue;
          const int r = mf * 16 + 4 * q;
          const f32x4 rs = *reinterpret_cast<const f32x4*>(&sm.rowscale[r]);
          const f32x4 gwv = *reinterpret_cast<const f32x4*>(&sm.rowgw[r]);
#pragma unroll
          for (int nf = 0; nf < NF; ++nf) {  // (channels past N: written, never stored)
            const int c = (wave * NF + nf) * 16 + li;
#pragma unroll
            for (int i = 0; i < 4; ++i) fl[(r + i - pass * RP) * FP + c] = outv(0, nf, mf, i, rs) * gwv[i];
          }
        }
        if (pass == 0) wait_vmem<0>();  // the next tile's entry has landed
        lds_barrier();
        for (int idx = tid; idx < RP * CH; idx += kThreads) {
          const int r = idx / CH, c = idx % CH;
          const int ro = sm.rowout[pass * RP + r];
          if (ro >= 0 && c < nch)
            *reinterpret_cast<u32x4*>(reinterpret_cast<float*>(a.slots) + (int64_t)ro * N + nt * BN + 4 * c) =
                *reinterpret_cast<const u32x4*>(fl + r * FP + 4 * c);
        }
        lds_barrier();
      }
      }
    } else {
#pragma unroll
    for (int mf = 0; mf < MF; ++mf) {
      const int r = mf * 16 + 4 * q;
      const f32x4 rs = *reinterpret_cast<const f32x4*>(&sm.rowscale[r]);
      const i32x4 ro = *reinterpret_cast<const i32x4*>(&sm.rowout[r]);
#pragma unroll
      for (int nf = 0; nf < NF; ++nf) {
        if (nf >= nvalid) continue;
        const int n = 16 * (nb0 + nf) + li;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t orow = (int64_t)ro[i] * N + n;
          if (GUARD && ro[i] < 0) continue;
          if constexpr (F6) {  // the exact integer sum, held in fp32
            reinterpret_cast<int32_t*>(a.raw_out)[orow] = (int32_t)acc[0][nf][mf][i];
          } else if constexpr (INT && !GSC && !F8) {
            int iv = acc[0][nf][mf][i];
            if constexpr (KD == K_W4A4) iv >>= 4;
            reinterpret_cast<int32_t*>(a.raw_out)[orow] = iv;
          } else {
            reinterpret_cast<float*>(a.raw_out)[orow] = outv(0, nf, mf, i, rs);
          }
        }
      }
    }
    }
  };
  if (finish) {
    if (full) epilogue(std::false_type{});
    else epilogue(std::true_type{});
  }
  if constexpr (PHASE == kPhaseRaw) wait_vmem<0>();  // the next tile's entry (no barrier in this epilogue)
  __syncthreads();  // the next tile rewrites rowsrc and the stages
}

template <int ACT, int PHASE, int CFG>
__device__ __attribute__((always_inline)) inline void dispatch_kind(Smem& sm, const GemmArgs& a, const DevExpert* ex, int g, int m_g, int mt, int nt,
                                     int off_e, int kd, int split) {
  switch (kd) {
    case K_W16: run_tile<K_W16, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W8A8: run_tile<K_W8A8, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_F8A8:  // planned in 128-row tiles in the down phase only
      if constexpr (CFG != CFG_L || PHASE == 1) run_tile<K_F8A8, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split);
      break;
    case K_W4A4: run_tile<K_W4A4, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W4A4F6: run_tile<K_W4A4F6, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W2G: run_tile<K_W2G, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W3G: run_tile<K_W3G, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W4G: run_tile<K_W4G, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W8G: run_tile<K_W8G, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split); break;
    case K_W4A4G:  // never planned in 128-row tiles
      if constexpr (CFG != CFG_L) run_tile<K_W4A4G, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split);
      break;
    case K_MXFP4:  // never planned in 128-row tiles
      if constexpr (CFG != CFG_L) run_tile<K_MXFP4, ACT, CFG, PHASE>(sm, a, ex, g, m_g, mt, nt, off_e, split);
      break;
    default: break;
  }
}

template <int ACT, int PHASE>
__global__ void __launch_bounds__(kThreads, 2) group_gemm_kernel(GemmArgs a) {
  __shared__ Smem sm;
  {
    const TileQueue Q = tile_queue(a, PHASE == kPhaseRaw ? 0 : PHASE);
    if (threadIdx.x < kXcd) sm.qtotal[threadIdx.x] = min(Q.ctr[threadIdx.x * 4 + 1], a.fcap);
    if (threadIdx.x == 0) { sm.qi = 0; sm.cur_idx = 0; }
    __syncthreads();
    if (threadIdx.x == 0) claim_next<false>(Q, sm);
    __syncthreads();
  }
  for (;;) {
    // wave-uniform from here on: tile bookkeeping and weight pointers live in SGPRs
    const int w0 = __builtin_amdgcn_readfirstlane(sm.entry.x);
    if (w0 < 0) break;
    const int w1 = __builtin_amdgcn_readfirstlane(sm.entry.y);
    const int off_e = __builtin_amdgcn_readfirstlane(sm.entry.z);
    const int m_g = __builtin_amdgcn_readfirstlane(sm.entry.w);
    const int g = w0 & 0xFFFF, cfg = (w0 >> 16) & 15, kd = (w0 >> 20) & 15, split = ((w0 >> 24) & 7) + 1;
    const int mt = w1 & 0xFFFF, nt = w1 >> 16;
    const DevExpert* ex = PHASE == kPhaseRaw ? nullptr : a.experts + g;
    // (every thread has read the entry: run_tile passes a barrier before
    // thread 0 claims the next tile into it)
    switch (cfg) {
      case CFG_S: dispatch_kind<ACT, PHASE, CFG_S>(sm, a, ex, g, m_g, mt, nt, off_e, kd, split); break;
      case CFG_T: dispatch_kind<ACT, PHASE, CFG_T>(sm, a, ex, g, m_g, mt, nt, off_e, kd, split); break;
      case CFG_M: dispatch_kind<ACT, PHASE, CFG_M>(sm, a, ex, g, m_g, mt, nt, off_e, kd, split); break;
      default: dispatch_kind<ACT, PHASE, CFG_L>(sm, a, ex, g, m_g, mt, nt, off_e, kd, split); break;
    }
  }
}

}  // namespace

// Per-(activation dtype, phase) launchers, one translation unit each.
#define MXMOE_GG_LAUNCHER(NAME, ACT, PHASE)                                                   \
  hipError_t NAME(const GemmArgs& a, int grid, hipStream_t s) {                               \
    hipLaunchKernelGGL((group_gemm_kernel<ACT, PHASE>), dim3(grid), dim3(kThreads), 0, s, a); \
    return hipGetLastError();                                                                 \
  }

hipError_t gg_bf16_p0(const GemmArgs& a, int grid, hipStream_t s);
hipError_t gg_bf16_p1(const GemmArgs& a, int grid, hipStream_t s);
hipError_t gg_bf16_raw(const GemmArgs& a, int grid, hipStream_t s);
hipError_t gg_f16_p0(const GemmArgs& a, int grid, hipStream_t s);
hipError_t gg_f16_p1(const GemmArgs& a, int grid, hipStream_t s);
hipError_t gg_f16_raw(const GemmArgs& a, int grid, hipStream_t s);

}  // namespace mxmoe
