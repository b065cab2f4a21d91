/*
 * mxmoe.h - C ABI of the MI355X (gfx950) mixed-precision MoE block.
 *
 * The library evaluates one MoE block forward (MxMoE, arXiv 2505.05799,
 * Sec. 2.2 Eq. (1)-(2)):
 *
 *     y[t] = sum_{s<k} w[t,s] * Expert_{ids[t,s]}(x[t]) + sum_j Shared_j(x[t])
 *     Expert(x) = W_down( SiLU(W_gate x) * (W_up x) )
 *
 * where every linear block (gate, up, down) of every expert carries its own
 * quantization scheme (linear-block granularity, Sec. 3.1).  Supported schemes
 * (notation wXaY_gZ of the Fig. 1 caption):
 *
 *   w16      16-bit weights (bf16, or fp16 when activations are fp16)
 *   wNg128   weight-only, N in {2,3,4,8}, asymmetric, fp16 scale and fp16 zero
 *            per group of 128 along K (Sec. 5.2): w = s * (q - z)
 *   w8a8     8-bit per-output-channel symmetric weights (fp32 scale, codes in
 *            [-127,127]) and 8-bit per-token symmetric activations
 *   w4a4     same with 4 bits (codes in [-7,7])
 *   fp8      OCP FP8 e4m3 weights with an fp32 scale per output channel and
 *            e4m3 activations with an fp32 scale per token (the 8-bit
 *            floating-point operand of the MI355X matrix cores)
 *
 * Activations of w8a8 / w4a4 linears are quantized at run time, per token
 * (Sec. 4.2.2): amax = max|a|, inv = fl32(qmax/amax), s = fl32(amax/qmax),
 * q = clamp(rne(fl32(a*inv)), -qmax, qmax); an all-zero row gets s = 0.
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers unless marked (host).
 *   - The caller owns every buffer.  No call allocates device memory, frees,
 *     or synchronizes the stream; work is enqueued on `stream` (0 = null
 *     stream) and completes asynchronously.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     failed validation returns a status and enqueues nothing.
 *   - MXMOE_ERR_HIP means a launch failed; the stream state is then undefined.
 *   - Calls on different streams with separate workspaces may run concurrently.
 *   - Identical inputs give bitwise identical outputs (no floating-point
 *     atomics; routing order is fixed).
 */
#ifndef MXMOE_H
#define MXMOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__)
#define MXMOE_API __attribute__((visibility("default")))
#else
#define MXMOE_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MXMOE_OK = 0,
  MXMOE_ERR_INVALID_ARG = 1,  /* null / misaligned pointer, bad size or count   */
  MXMOE_ERR_UNSUPPORTED = 2,  /* scheme or shape outside the supported set      */
  MXMOE_ERR_WORKSPACE = 3,    /* workspace or packed buffer too small           */
  MXMOE_ERR_HIP = 4           /* a HIP launch failed                            */
} mxmoe_status;

typedef enum { MXMOE_F16 = 0, MXMOE_BF16 = 1 } mxmoe_dtype;

/* Quantization scheme of one linear block: w{w_bits}a{a_bits}_g{w_group}
 * (notation of Fig. 1; a_gsize of the W5A5 allocation table).
 * Accepted combinations:
 *   {16,16,-1,-1,0}  {8,8,-1,-1,1}  {4,4,-1,-1,1}  {N,16,128,-1,0} N=2,3,4,8
 *   {4,4,128,128,1}  w4a4-g128: symmetric 4-bit weights and activations with
 *                    one scale per 128 consecutive k of a channel / a token
 *   {4,4,32,32,1} with fmt = 1: mxfp4, the OCP Microscaling FP4 format the
 *                    MI355X matrix cores take natively (the paper's scheme set
 *                    is whatever the hardware supports, Sec. 4.2.1): FP4 e2m1
 *                    elements on both operands with one E8M0 power-of-two
 *                    scale per 32 consecutive k; activations are encoded at
 *                    run time (e = floor(log2 amax) - 2, elements rounded to
 *                    nearest, ties to even, clamped to 6)
 *   {4,4,-1,-1,1} with fmt = 3: w4a4 (per channel / per token, the same
 *                    quantization and results as fmt = 0) whose int4 codes are
 *                    held as FP6 e2m3 values, so that the MI355X FP6 matrix
 *                    cores (twice the int8 rate) compute the exact integer
 *                    sums; weights take 6 bits per code (24 bytes per 32)
 *   {8,8,-1,-1,1} with fmt = 2: fp8, OCP FP8 e4m3 elements (sign bit 7,
 *                    exponent bias 7, no infinities, 448 the largest finite
 *                    value) on both operands; fp32 scale per output channel
 *                    (weights) and per token (activations, encoded at run
 *                    time with the recipe above and 448 in place of qmax:
 *                    element = nearest e4m3 value of fl32(a*inv), ties to the
 *                    even code, magnitudes past 448 give 448)
 * All other combinations have fmt = 0.                                       */
typedef struct {
  int32_t w_bits;
  int32_t a_bits;     /* 16 = weight-only                                       */
  int32_t w_group;    /* 128 or 32 (mxfp4), or -1 = per output channel          */
  int32_t a_group;    /* 128 or 32 (mxfp4), or -1 = per token                   */
  int32_t symmetric;  /* 1 for w8a8 / w4a4 (per channel or g128) and mxfp4      */
  int32_t fmt;        /* 0: integer codes; 1: OCP MX floating point (mxfp4);
                         2: FP8 e4m3 with per-channel / per-token scales;
                         3: w4a4 codes held as FP6 e2m3 operands             */
} mxmoe_scheme;

/* One linear block y = x W^T with W of shape [n, k] = [out, in].
 * Requirements: n % 16 == 0, k % 128 == 0, n,k > 0.                          */
typedef struct {
  int32_t n;
  int32_t k;
  mxmoe_scheme s;
} mxmoe_linear;

/* ---------------------------------------------------------------- packing */

/* Bytes of the packed form of linear *L (host) for activations `act`:
 *   wNg128: n*k*N/8 + (n*k/128)*4   (N + 0.25 bits per weight, Sec. 5.2)
 *   w8a8/w4a4/fp8: n*k*b/8 + 4*n
 *   w4a4 on FP6 operands: n*k*6/8 + 4*n
 *   w4a4-g128: n*k/2 + (n*k/128)*4   (fp16 group scale, 4-byte slot per group)
 *   mxfp4: n*k/2 + n*k/32            (4.25 bits per weight)
 *   w16: 2*n*k
 * Returns 0 if *L is not supported.                                          */
MXMOE_API size_t mxmoe_packed_bytes(const mxmoe_linear* L, mxmoe_dtype act);

/* Pack the quantized operands of one linear into the tile-major layout the
 * Group-GEMM streams (weight fragments in MFMA lane order, group metadata next
 * to its codes).  Runs once per weight load.
 *   codes  : wNg128 uint8 [n,k] in [0, 2^N-1]; w8a8/w4a4/w4a4-g128 int8
 *            [n,k] in [-qmax, qmax] (w4a4 on FP6 operands too); mxfp4 uint8 [n,k] e2m1 codes 0..15
 *            (sign in bit 3); fp8 uint8 [n,k] e4m3 bytes (no NaN code);
 *            w16: 16-bit weights [n,k] of `w16_src`.
 *   scales : wNg128 and w4a4-g128 fp16 [n, k/128]; w8a8/w4a4/fp8 fp32 [n];
 *            mxfp4 uint8 E8M0 [n, k/32]; NULL for w16.
 *   zeros  : wNg128 fp16 [n, k/128] holding integers in [0, 2^N-1]; else NULL.
 * Codes and zero points outside these ranges (a zero point that is not an
 * integer in [0, 2^N-1], a wNg128 code above 2^N-1, a w4a4 / w4a4-g128 code
 * outside [-7, 7]) are not representable in the packed form: the group's
 * scale (per-channel w4a4: the channel's scale) is stored as NaN instead, so
 * every output that uses it is NaN.
 *   w16_src: dtype of 16-bit source weights; converted (RNE) to `act`.
 *   packed : output, mxmoe_packed_bytes(L, act) bytes, 256-byte aligned.
 * All inputs 4-byte aligned.  Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE
 * (packed_bytes too small), HIP.                                             */
MXMOE_API mxmoe_status mxmoe_pack_weights(const mxmoe_linear* L, mxmoe_dtype act, mxmoe_dtype w16_src,
                                const void* codes, const void* scales, const void* zeros,
                                void* packed, size_t packed_bytes, hipStream_t stream);

/* Inverse of mxmoe_pack_weights (testing and inspection): writes codes,
 * scales and zeros in the input formats above (w16: `act` dtype values).    */
MXMOE_API mxmoe_status mxmoe_unpack_weights(const mxmoe_linear* L, mxmoe_dtype act, const void* packed,
                                  void* codes, void* scales, void* zeros, hipStream_t stream);

/* ---------------------------------------------------------------- routing */

/* Scratch bytes mxmoe_route_permute needs for T tokens, top-k, E experts.   */
MXMOE_API size_t mxmoe_route_workspace_bytes(int32_t T, int32_t k, int32_t E);

/* Group the T*k (token, slot) pairs by expert (the X_e of Eq. (2)).  Pair id
 * p = t*k + s.  Pairs are ordered by (expert, p): stable, so the result is
 * unique.  Pairs whose id lies outside [0, E) are dropped.
 *   topk_ids   : int32 [T,k]
 *   counts     : int32 [E]       pairs per expert
 *   offsets    : int32 [E+1]     exclusive prefix of counts
 *   sorted_pair: int32 [T*k]     pair ids in sorted order (first offsets[E])
 *   inv        : int32 [T*k]     position of pair p, -1 if dropped
 *   status     : int32 [1]       0, or 1 + the smallest dropped pair id
 * Limits: 1 <= k <= E <= 1024, T >= 0, T*k < 2^31.                           */
MXMOE_API mxmoe_status mxmoe_route_permute(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                 int32_t* counts, int32_t* offsets, int32_t* sorted_pair,
                                 int32_t* inv, int32_t* status, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Router front-end (Eq. (2): the gate weights w_e come from a softmax over
 * the router's logits).  Per token t, one wavefront:
 *   p_e = exp(l_e - max l) / sum_e' exp(l_e' - max l)      (fp32)
 *   topk_ids[t, 0..k-1]: the k largest logits in decreasing order, ties to
 *            the lower expert id (the same order as the probabilities);
 *   topk_w[t, s] = p of that expert, or, with renormalize = 1,
 *            exp(l - max l) / (sum of it over the k chosen experts);
 *   shared_w[t, j] = 1 / (1 + exp(-shared_logits[t, j])): the sigmoid gate a
 *            shared expert's output is multiplied by (Qwen-MoE style), only
 *            if shared_logits is not NULL.
 *   logits       : fp32 [T, E], finite values (a NaN is never chosen; a token
 *                  left with only NaN candidates gets id -1 in its last slots)
 *   shared_logits: fp32 [T, n_shared] or NULL
 *   topk_ids: int32 [T, k], topk_w: fp32 [T, k], shared_w: fp32 [T, n_shared]
 * Limits: 1 <= k <= min(E, 64), E <= 1024, 0 <= n_shared <= 64.  All device
 * pointers, 4-byte aligned.  Errors: INVALID_ARG, HIP.                      */
MXMOE_API mxmoe_status mxmoe_router_topk(const float* logits, int32_t T, int32_t E, int32_t k,
                               int32_t renormalize, const float* shared_logits, int32_t n_shared,
                               int32_t* topk_ids, float* topk_w, float* shared_w,
                               hipStream_t stream);

/* ------------------------------------------------------ activation quant */

/* Per-row symmetric quantization of a [rows, cols] activation matrix (row
 * stride `ld` elements) with the fp32 recipe in the header comment.
 *   codes: int8 [rows, cols] (dense), scales: fp32 [rows].  qmax = 127 or 7;
 *   qmax = 448 writes FP8 e4m3 bytes (the fp8 scheme's activation encoding). */
MXMOE_API mxmoe_status mxmoe_act_quant(const void* a, mxmoe_dtype act, int32_t rows, int32_t cols,
                             int64_t ld, int32_t qmax, int8_t* codes, float* scales,
                             hipStream_t stream);

/* --------------------------------------------------------- one linear */

MXMOE_API size_t mxmoe_linear_workspace_bytes(const mxmoe_linear* L, int32_t m);

/* out = a W^T for one packed linear, through the same micro-kernels the block
 * uses (testing and single-GEMM measurement).
 *   a  : [m, k] `act` activations (dense)
 *   out: w8a8 / w4a4 (int8 or FP6 operands) -> int32 [m, n] exact integer
 *        accumulators sum_c qa[m,c]*qw[n,c] (qa from the per-token quantizer);
 *        w4a4-g128 -> fp32 [m, n]: per 128-wide block the exact integer sum
 *        times s_a[m,b]*s_w[n,b], added over the blocks in fp32;
 *        mxfp4 -> fp32 [m, n]: a encoded as mxfp4 at run time, products of
 *        the decoded operands accumulated in fp32 by the scaled FP4 MFMA;
 *        fp8 -> fp32 [m, n]: a encoded as e4m3 per token at run time, the
 *        e4m3 products accumulated in fp32 by the FP8 MFMA, times
 *        s_a[m]*s_w[n];
 *        other schemes -> fp32 [m, n] with fp32 accumulation.
 * Limits: m*k*2 bytes below 4 GiB (UNSUPPORTED beyond).                      */
MXMOE_API mxmoe_status mxmoe_linear_forward(const mxmoe_linear* L, mxmoe_dtype act, const void* packed,
                                  int32_t m, const void* a, void* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------- MoE block */

typedef struct {
  int32_t hidden;        /* H: multiple of 128                                 */
  int32_t ffn;           /* F of routed experts: multiple of 128               */
  int32_t n_experts;     /* E routed experts, 1..1024                          */
  int32_t top_k;         /* k, 1..E                                            */
  int32_t n_shared;      /* shared experts run densely over all tokens, 0..64  */
  int32_t ffn_shared;    /* F of shared experts (multiple of 128 if n_shared)  */
  mxmoe_dtype act;       /* dtype of x, y and the gated intermediate h         */
  /* host [(n_experts + n_shared) * 3]: gate, up, down of expert 0, 1, ...,
   * routed experts first.  Gate and up of one expert must share a scheme.    */
  const mxmoe_scheme* scheme;
  /* host array of device pointers to the packed linears, same order          */
  const void* const* packed;
} mxmoe_block;

/* Size of, and host-side fill for, the device block table: the caller copies
 * the filled host buffer to device memory once (e.g. hipMemcpy) and passes
 * it to every forward.  It holds the packed pointers, so it must be refilled
 * when weights move.                                                        */
MXMOE_API size_t mxmoe_block_table_bytes(const mxmoe_block* B);
MXMOE_API mxmoe_status mxmoe_block_table_fill(const mxmoe_block* B, void* host_buf, size_t host_bytes);

/* Workspace bytes mxmoe_moe_forward needs for T tokens (256-byte aligned
 * buffer).  Holds routing arrays, the tile plan, activation codes, the gated
 * intermediate h, and fp32 per-slot down-projection rows.                   */
MXMOE_API size_t mxmoe_workspace_bytes(const mxmoe_block* B, int32_t T);

/* The MoE block forward.
 *   x       : [T, hidden] act            topk_ids: int32 [T, k]
 *   topk_w  : fp32 [T, k] gate weights   y       : [T, hidden] act (output)
 * Out-of-range expert ids contribute nothing; the workspace status word
 * (see mxmoe_workspace_layout) records 1 + the first such pair id.
 * Limits (UNSUPPORTED beyond them): T*k < 2^31, and x (T*hidden*2 bytes), the
 * routed h rows (T*k*ffn*2) and the shared h rows (n_shared*T*ffn_shared*2)
 * each below 4 GiB.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, HIP.                          */
MXMOE_API mxmoe_status mxmoe_moe_forward(const mxmoe_block* B, const void* block_table, int32_t T,
                               const void* x, const int32_t* topk_ids, const float* topk_w,
                               void* y, void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/* Largest workspace mxmoe_moe_forward_noalloc can use (bytes).             */
#define MXMOE_NOALLOC_SCRATCH_BYTES (128u << 20)

/* mxmoe_moe_forward for callers that cannot allocate device memory or pass a
 * workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments and result as mxmoe_moe_forward,
 * minus the workspace: the library's own device array of
 * MXMOE_NOALLOC_SCRATCH_BYTES bytes serves as the workspace.  Each GPU holds
 * its own copy from the first call on it (made with that device current)
 * until the process ends; nothing is allocated, freed or synchronized.
 * Blocks whose workspace (mxmoe_workspace_bytes(B, T)) exceeds the array
 * return MXMOE_ERR_WORKSPACE and enqueue nothing (about 200 tokens of a
 * Mixtral- or Qwen1.5-MoE-shaped block, 32 of a Qwen2-57B-shaped one).
 * All calls on one GPU share the array: calls that may overlap on a GPU (on
 * different streams, or from several threads) race and give undefined
 * results; serialize them.  Intermediates of the last call stay readable
 * at the offsets of mxmoe_workspace_layout until the next call.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, HIP.                          */
MXMOE_API mxmoe_status mxmoe_moe_forward_noalloc(const mxmoe_block* B, const void* block_table, int32_t T,
                                       const void* x, const int32_t* topk_ids, const float* topk_w,
                                       void* y, hipStream_t stream);

/* Options of mxmoe_moe_forward_ex (measurement and testing).                 */
typedef struct {
  /* host [(n_experts + n_shared)] or NULL: experts with mask 0 get no tiles
   * (their rows keep whatever the workspace held); used to time subsets.   */
  const uint8_t* expert_mask;
  /* Must be 0.  (The forward always runs its phases as separate launches:
   * routing + plan + x encodings, the gate/up Group-GEMM, h quantization,
   * the down Group-GEMM and the combine; each Group-GEMM launch is one
   * persistent grid over all experts and schemes of its phase.)             */
  int32_t reserved0;
  /* 1: skip the combine (y untouched) - to time the Group-GEMM alone.       */
  int32_t skip_combine;
  /* host array of 2*MXMOE_N_PHASES caller-created events, or NULL: event 2i
   * is recorded on `stream` before phase i and event 2i+1 after it (phases:
   * 0 routing + plan + x quantization, 1 gate/up Group-GEMM, 2 h quantization,
   * 3 down Group-GEMM, 4 combine).                                          */
  hipEvent_t* events;
  /* fp32 [T, E] router logits, or NULL.  When set, the forward starts with
   * the router front-end of mxmoe_router_topk (same results; inside the
   * routing launch when T*k <= 4096, E <= 64 and k <= 8): topk_ids / topk_w
   * may then be NULL and are not read; the chosen ids and weights land in the
   * workspace (router_ids / router_w of mxmoe_ws_layout).                    */
  const float* router_logits;
  int32_t renormalize;           /* with router_logits: as in mxmoe_router_topk */
  /* With router_logits: fp32 [T, n_shared] shared-expert gate logits or NULL;
   * their sigmoid multiplies each shared expert's output.                    */
  const float* shared_logits;
  /* Without router_logits: fp32 [T, n_shared] weights of the shared experts'
   * outputs, or NULL for weight 1.                                           */
  const float* shared_w;
  /* 1: keep the down projection's weighted rows (the slot rows the combine
   * sums) in fp32, for callers that difference them (the allocator's error
   * probe); 0 (default): each slot row element is rounded once to the
   * activation dtype before the combine, which halves their traffic (with
   * fp16 activations an element beyond the fp16 range then becomes inf).    */
  int32_t fp32_slots;
  int32_t reserved1;             /* must be 0 */
} mxmoe_forward_opts;

#define MXMOE_N_PHASES 5

MXMOE_API mxmoe_status mxmoe_moe_forward_ex(const mxmoe_block* B, const void* block_table, int32_t T,
                                  const void* x, const int32_t* topk_ids, const float* topk_w,
                                  void* y, void* workspace, size_t workspace_bytes,
                                  const mxmoe_forward_opts* opts, hipStream_t stream);

/* Byte offsets of the intermediates inside the forward workspace (testing).
 * An offset of SIZE_MAX means the buffer is not present for this block.    */
typedef struct {
  size_t status;        /* int32 [4]: [0] = 0 or 1 + first dropped pair      */
  size_t counts;        /* int32 [E]                                         */
  size_t offsets;       /* int32 [E+1]                                       */
  size_t sorted_pair;   /* int32 [T*k]                                       */
  size_t inv;           /* int32 [T*k]                                       */
  size_t plan;          /* int32 tile plan: group records [2][G][12], order [2][G],
                           XCD queues [2][8][plan_queue_cap][3] (16-byte aligned),
                           queue counters [2][8][4], misc [16], the queues
                           expanded to tiles [2][8][plan_flat_cap][4], and
                           split-K arrival counters [2][16384]; misc[8] is
                           the workgroup count the slicing assumed            */
  size_t xq8, xs8;      /* int8 [T,H], fp32 [T]: x codes for a8 gate/up      */
  size_t xq4, xs4;      /* int8 [T,H], fp32 [T]: x codes for a4 gate/up      */
  size_t h;             /* act [T*k, F]: routed h rows, sorted-pair order    */
  size_t h_shared;      /* act [n_shared, T, F_shared]                       */
  size_t hq, hs;        /* int8 [T*k, F], fp32 [T*k]: routed h codes         */
  size_t hq_shared, hs_shared; /* int8 [n_shared,T,F_shared], fp32 [n_shared,T] */
  size_t slots;         /* [T, k + n_shared, H]: weighted down rows, in the
                           activation dtype (fp32 with opts.fp32_slots; the
                           buffer is sized for fp32)                          */
  size_t total;         /* = mxmoe_workspace_bytes                           */
  size_t plan_queue_cap;/* entries per XCD queue in the tile plan            */
  size_t plan_flat_cap; /* tiles per XCD queue in the tile plan              */
  size_t partial;       /* fp32 split-K partial sums                         */
  size_t partial_floats;/* size of that buffer (floats)                      */
  size_t rsx;           /* fp32 [T, H/128]: row sums of x per 128-wide block
                           (bf16 blocks with 2/3/4-bit gate|up), else -1    */
  size_t rsh;           /* fp32 [T*k, F/128]: same for routed h, else -1     */
  size_t rsh_shared;    /* fp32 [n_shared*T, F_shared/128], else -1          */
  size_t xq4g, xs4g;    /* int8 [T,H], fp32 [T, H/128]: x codes for w4a4-g128
                           gate|up (else -1)                                  */
  size_t hsg;           /* fp32 [T*k, F/128]: group scales of routed h rows
                           for w4a4-g128 down (codes in hq), else -1         */
  size_t hsg_shared;    /* fp32 [n_shared*T, F_shared/128], else -1          */
  size_t xqmx, xsmx;    /* uint8 [T, H/2] e2m1 codes, uint8 [T, H/32] E8M0: x
                           for mxfp4 gate|up (else -1)                      */
  size_t hqmx, hsmx;    /* uint8 [T*k, F/2], [T*k, F/32]: routed h for mxfp4
                           down (else -1)                                   */
  size_t hqmx_shared, hsmx_shared; /* the same for shared h (else -1)        */
  size_t router_ids;    /* int32 [T, k]: ids chosen by the router front-end  */
  size_t router_w;      /* fp32 [T, k]: their gate weights                   */
  size_t shared_w;      /* fp32 [T, n_shared]: sigmoid shared gates (-1 if no
                           shared experts)                                   */
  size_t xqf8, xsf8;    /* uint8 [T, H] e4m3 codes, fp32 [T] scales: x for fp8
                           gate|up (else -1); h rows of an fp8 down projection
                           use hq / hs and hq_shared / hs_shared             */
  size_t xqf6, xsf6;    /* uint8 [T, H] FP6-encoded int4 codes (per 32 elements
                           24 bytes of e2m3 codes, 8 zero bytes), fp32 [T]
                           scales: x for w4a4 gate|up on FP6 operands (else
                           -1); h rows of such a down projection use hq / hs
                           and hq_shared / hs_shared in the same encoding    */
} mxmoe_ws_layout;

MXMOE_API mxmoe_status mxmoe_workspace_layout(const mxmoe_block* B, int32_t T, mxmoe_ws_layout* out);

/* ------------------------------------------------------- tile cost model */

/* The run-time tile plan (one per forward, built on the GPU) prices every
 * output tile with the per-tile cost c_t that the paper profiles ahead of
 * time for each tile configuration (Sec. 4.2.2, runtime cost modelling), and
 * uses the costs to order tiles longest first and to choose how many slices
 * along K a group's tiles take.  The costs do not change any result, only
 * the schedule.
 *
 * Table (host, int32, MXMOE_TILE_COST_ENTRIES values), indexed
 *   [phase][scheme][configuration][value]
 *   phase          0: gate|up (both linears of a tile), 1: down, and the
 *                  single linear of mxmoe_linear_forward
 *   scheme         0 w16, 1 w8a8, 2 w4a4, 3 w2g128, 4 w3g128, 5 w4g128,
 *                  6 w8g128, 7 w4a4-g128, 8 mxfp4, 9 fp8, 10 w4a4 on FP6
 *   configuration  0..3: tiles of 16, 32, 64, 128 rows (the kernel picks
 *                  the smallest that holds the group's rows, up to 64 rows
 *                  for w4a4-g128 and mxfp4, and for fp8 outside the down
 *                  phase)
 *   value          a, bs, bu, h in picoseconds (bs, bu, h >= 0):
 *                  a  fixed cost of a tile (the intercept of a fit over K,
 *                     so it may be negative),
 *                  bs cost per 128-wide k block not shared with other tiles,
 *                  bu cost per k block of the weight stream, which the
 *                     group's mt row tiles share (charged bu / mt),
 *                  h  hand-off cost of a tile sliced along K.
 * A tile of kb k blocks costs a + kb*bs + floor(kb*bu/mt) + (sliced ? h : 0)
 * in exact integer arithmetic, clamped to [1, 2e9].
 *
 * mxmoe_set_tile_costs copies the table into a process-wide setting used by
 * every later forward on any device (table NULL restores the built-in
 * roofline default).  A forward reads the setting when it is enqueued; the
 * calls are thread-safe.  mxmoe_get_tile_costs copies the current table out.
 * Errors: INVALID_ARG (n_entries wrong, a negative bs, bu or h, out NULL).  */
#define MXMOE_TILE_COST_ENTRIES (2 * 11 * 4 * 4)
MXMOE_API mxmoe_status mxmoe_set_tile_costs(const int32_t* table, int32_t n_entries);
MXMOE_API mxmoe_status mxmoe_get_tile_costs(int32_t* out, int32_t n_entries);

MXMOE_API const char* mxmoe_status_string(mxmoe_status s);

/* Library version, (major << 16) | minor.                                    */
MXMOE_API int32_t mxmoe_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MXMOE_H */
