/*
 * archead.h -- C ABI of the ARCHead packed LM-head forward for AMD Instinct
 * MI355X (gfx950).
 *
 * The packed head (ARCHead, arXiv 2608.02703, Section 3.2 and the appendix
 * table "Logical contents of the packed ARCHead state dictionary") holds
 *
 *   W_d   = Q5(A_c) Q8(B_c) + Q_SC4(W - A_c B_c)   quantized core
 *   W_hat = W_d + A_w B_w                          core plus correction
 *
 * and the forward (Section 3.2, inference equation; appendix "Expanded
 * Construction Procedure") is Y_hat = H W_d^T + (H B_w^T) A_w^T.  In the
 * names of this library's buffers, for a token x (bf16 [d]) and vocabulary
 * row v:
 *
 *   logit[v] = sum_j s_res[v,j] * sum_{i in group j} c[v,i] x[i]     residual
 *            + s_U[v] * sum_k cU[v,k] * t_c[k]                       core
 *            + s_A[v] * sum_k cA[v,k] * t_w[k]                       correction
 *   t_c[k] = sum_i (s_V[k, i/g_v] cV[k,i]) x[i],
 *   t_w[k] = sum_i (s_B[k, i/g_b] cB[k,i]) x[i]
 *
 * No dense head is ever formed: the residual is unpacked in registers and the
 * two low-rank products are evaluated through t_c and t_w (the paper's
 * bracketing H B_w^T first).  All arithmetic is fp32.
 *
 * Buffer layouts (all row-major, rows back to back, no padding):
 *
 *   res_codes     uint8   [V, d/2]     INT4 residual codes, ARCHEAD_INT4_V1
 *   res_scales    fp16    [V, d/g]     residual group scales (groups of g
 *                                      consecutive elements along d)
 *   core_u        int8    [V, r_c]     core left codes (A_c side; any code
 *                                      range that fits int8, e.g. 5-bit), or
 *                 uint32  [V, ceil(r_c/6)]  the same codes bit-packed in
 *                                      ARCHEAD_I5 (desc.core_u_dtype)
 *   core_u_scale  fp16    [V]          per-row scales of core_u
 *   core_v        int8    [r_c, d]     core right codes (B_c side)
 *   core_v_scale  fp16    [r_c, d/g_v] group scales of core_v (g_v = d: one
 *                                      scale per row)
 *   corr_a        int8    [V, r_r]     correction left codes (A_w, row-wise)
 *   corr_a_scale  fp16    [V]
 *   corr_b        int8    [r_r, d]     correction right codes (B_w)
 *   corr_b_scale  fp16    [r_r, d/g_b] group scales of corr_b
 *
 * ARCHEAD_INT4_V1: bytes 4w..4w+3 of a row, read as a little-endian 32-bit
 * word q, hold elements 8w..8w+7 of that row.  Element 8w+2k (k = 0..3) is
 * the nibble in bits [4k, 4k+4) of q, element 8w+2k+1 the nibble in bits
 * [16+4k, 20+4k).  A nibble u stores the signed code c = u - 8 (c in
 * [-8, 7]).  With this order, (q >> 4k) & 0x000F000F places elements
 * (8w+2k, 8w+2k+1) in the two 16-bit halves of a register, ready to become
 * a bf16 pair.
 *
 * Memory ownership: every device pointer is borrowed.  The caller allocates
 * the head buffers, activations, outputs and the workspace, and keeps the
 * head buffers alive and unchanged for the lifetime of the handle.  The
 * library allocates no device memory.
 *
 * Errors: every call returns an archead_status; no C++ exception crosses the
 * ABI.  Argument checks happen on the host before any launch.  A failed HIP
 * launch returns ARCHEAD_E_HIP; archead_last_error() then gives a message
 * (thread-local).  Kernel faults surface, as usual for HIP, at the caller's
 * next synchronisation.  The compute calls are asynchronous on the given
 * stream and never synchronise.
 */
#ifndef ARCHEAD_H_
#define ARCHEAD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARCHEAD_ABI_VERSION 3u

typedef enum archead_status {
  ARCHEAD_OK = 0,
  ARCHEAD_E_INVALID_ARG = 1, /* null pointer, bad shape, bad enum value     */
  ARCHEAD_E_MISALIGNED = 2,  /* a pointer or stride breaks its alignment    */
  ARCHEAD_E_UNSUPPORTED = 3, /* no gfx950 device, or a shape outside limits */
  ARCHEAD_E_WORKSPACE = 4,   /* workspace smaller than archead_workspace_bytes */
  ARCHEAD_E_HIP = 5          /* a HIP runtime call failed                   */
} archead_status;

typedef enum archead_dtype {
  ARCHEAD_F32 = 0,
  ARCHEAD_BF16 = 1,
  ARCHEAD_F16 = 2,
  ARCHEAD_I32 = 3,
  ARCHEAD_I64 = 4,
  ARCHEAD_I8 = 5,
  ARCHEAD_U8 = 6,
  ARCHEAD_I5 = 7   /* signed 5-bit codes, six per little-endian 32-bit word */
} archead_dtype;

typedef enum archead_int4_encoding { ARCHEAD_INT4_V1 = 1 } archead_int4_encoding;

typedef enum archead_op {
  ARCHEAD_OP_LOGITS = 0,    /* archead_logits    */
  ARCHEAD_OP_LOGITS_CE = 1, /* archead_logits_ce */
  ARCHEAD_OP_ARGMAX = 2,    /* archead_logits_argmax */
  ARCHEAD_OP_TOPK = 3,      /* archead_logits_topk */
  ARCHEAD_OP_FIDELITY = 4   /* archead_logit_fidelity_head */
} archead_op;

/* Shape and encoding of a packed head (the "integer shapes/groups" metadata
 * of the paper's packed state dictionary).
 *   0 < V < 2^31, 0 < d <= 16384, d % g == 0, g % 32 == 0;
 *   r_c >= 0, r_r >= 0 (0 = component absent: r_c = r_r = 0 is plain group
 *   INT4, r_r = 0 is the "core only" ablation);
 *   g_v, g_b: group length along d of the core_v / corr_b scales, dividing d
 *   and a multiple of 32 (d = one scale per row);
 *   int4_encoding = ARCHEAD_INT4_V1, factor_dtype = ARCHEAD_I8;
 *   scale_dtype: the residual group scales s[v, j] (the "quantized group
 *   scales" of the paper's packed state dictionary, Section 3.3 and its
 *   packed-buffer appendix, which leave their format open):
 *     ARCHEAD_F16: res_scales holds s as fp16 [V, d/g];
 *     ARCHEAD_U8:  res_scales holds 8-bit codes q [V, d/g] (uint8) and
 *                  res_row_scales one fp16 scale rs per vocabulary row [V],
 *                  s[v, j] = rs[v] * q[v, j] (exact in fp32).  One byte of
 *                  scale per group is the storage the paper's reported head
 *                  sizes imply.  Served by every kernel (see
 *                  archead_logits).
 *   core_u_dtype: the core left factor's codes (the paper stores Q5(A_c),
 *   5-bit codes, Section 3.2 and the packed state-dictionary table):
 *     ARCHEAD_I8: int8 [V, r_c], one code per byte;
 *     ARCHEAD_I5: bit-packed, ARCHEAD_I5 layout: row v of core_u is
 *                 W5 = ceil(r_c / 6) little-endian 32-bit words (4 * W5
 *                 bytes, rows back to back); code k of the row is bits
 *                 [5 (k % 6), 5 (k % 6) + 5) of word k / 6, a 5-bit two's
 *                 complement value in [-16, 15]; bits 30-31 of every word and
 *                 the fields past r_c are zero.  core_u must then be 4-byte
 *                 aligned.  Every kernel reads this layout directly.
 *   Ranks need not be multiples of 4 on any kernel (the several-token and
 *   MFMA decode kernels read factor codes in pieces that need no alignment
 *   when a rank is not). */
typedef struct archead_desc {
  uint32_t abi_version; /* ARCHEAD_ABI_VERSION */
  int64_t V, d, g;
  int64_t r_c, r_r;
  int64_t g_v, g_b;
  int32_t int4_encoding;
  int32_t scale_dtype;
  int32_t factor_dtype;
  int32_t core_u_dtype;  /* ARCHEAD_I8 or ARCHEAD_I5 (ABI 3) */
} archead_desc;

/* Device pointers to the packed buffers (layouts above).  res_codes must
 * be 16-byte aligned, fp16 buffers 2-byte aligned.  Pointers of an absent
 * component (rank 0) may be NULL; res_row_scales is required with
 * ARCHEAD_U8 scales and ignored otherwise. */
typedef struct archead_ptrs {
  const void* res_codes;
  const void* res_scales;
  const void* core_u;
  const void* core_u_scale;
  const void* core_v;
  const void* core_v_scale;
  const void* corr_a;
  const void* corr_a_scale;
  const void* corr_b;
  const void* corr_b_scale;
  const void* res_row_scales;
} archead_ptrs;

typedef struct archead_handle archead_handle;

/* Check a descriptor on the host (no HIP call).  ARCHEAD_OK or
 * ARCHEAD_E_INVALID_ARG / ARCHEAD_E_UNSUPPORTED with a message. */
archead_status archead_validate_desc(const archead_desc* desc);

/* Create a handle for the head described by desc whose buffers are at ptrs
 * on the current HIP device.  The handle is host memory, immutable after
 * creation apart from the archead_set_* tuning calls, and may be used from several
 * threads and streams at once (each call with its own workspace).  Fails
 * with ARCHEAD_E_UNSUPPORTED if the current device is not gfx950 or there is
 * no device.  *out is set to NULL on failure. */
archead_status archead_create(const archead_desc* desc, const archead_ptrs* ptrs,
                              archead_handle** out);

/* Release a handle (NULL is a no-op).  Does not touch the borrowed buffers;
 * the caller must make sure no call using the handle is still queued on a
 * stream whose completion it has not awaited. */
void archead_destroy(archead_handle* h);

/* Bytes of workspace the call `op` needs for M tokens (0 for M == 0).  The
 * workspace holds the low-rank projections t (fp32 [M, r_c + r_r]; on the
 * decode and several-token paths with a 32-bit call stamp beside each value; on the tiled
 * MFMA path split into three bf16 parts), on the tiled path also per-call
 * tables derived from the head (group-scale ratios, the per-group sums of x,
 * the factor codes as bf16 and the U_c / A_w codes side by side: about
 * V * (r_c + r_r + 4 * (d/g + 3)) bytes, used only while the head has no
 * prepared buffer, see archead_prepare), and for the CE call the
 * per-vocabulary-tile softmax partials.  Returns 0 for a NULL handle or
 * M < 0. */
size_t archead_workspace_bytes(const archead_handle* h, int64_t M, archead_op op);

/* logits[m, v] for m < M, v < V.
 *   x        bf16 [M, ldx] device, 16-byte aligned, ldx >= d, ldx % 8 == 0
 *   out      [M, ldo] device, out_dtype ARCHEAD_F32 (4-byte aligned) or
 *            ARCHEAD_BF16 (2-byte aligned, fp32 result rounded to nearest
 *            even), ldo >= V
 *   ws       device workspace of ws_bytes >= archead_workspace_bytes(h, M,
 *            ARCHEAD_OP_LOGITS), 256-byte aligned; its contents on entry do
 *            not matter
 *   stream   hipStream_t to launch on (NULL = the default stream)
 * M == 0 returns ARCHEAD_OK without launching.  Four kernels serve the
 * call, chosen by M and the head shape:
 *   - M in the range of archead_set_dec_range (default from 2 to 32, or
 *     to the tokens it holds per pass where the several-token kernel
 *     applies: 16 at d = 4096, 8 at d = 8192) with g in {32, 64, 128},
 *     (d/g) % 4 == 0,
 *     d/g <= 64, r_c and r_r at most 128 each, and V * d / 2 < 2^31: the
 *     MFMA decode kernel, which streams the head once per pass of up to 16
 *     tokens (fewer when 16 rows of x do not fit in LDS);
 *   - otherwise M in the range of archead_set_mid_range (default: from one
 *     past the decode kernel's range to 32, one pass; to 24 at d >= 8192)
 *     with g in {64, 128},
 *     d % 512 == 0, d/g <= 64, r_c and r_r at most 128 each: the
 *     several-token kernel, which streams the head once per tile of up to
 *     32 tokens (x held in LDS in windows of 256 elements of d);
 *   - otherwise M <= archead_get_gemv_max_m (default 15), or g % 64 != 0:
 *     the decode GEMV (VALU dot products), one pass per 4 tokens;
 * These three kernels compute t = x V_c^T, x B_w^T inside the same launch
 * (a few leading workgroups publish t with a per-call stamp in the
 * workspace; the others wait for it a bounded time and otherwise compute it
 * themselves), so a decode step is a single kernel launch;
 *   - otherwise the tiled bf16 MFMA kernel (tiles of 64 tokens x 256
 *     vocabulary rows, three workgroups per CU, up to M = 64; 128 x 256,
 *     two workgroups per CU, up to M = 1024; 256 x 256 tiles above; its head-derived tables are built per call unless
 *     archead_prepare keeps them).
 * All produce fp32 logits from fp32 accumulation.  The tiled kernel carries
 * its accumulator in units of the current scale group's scale and feeds the
 * rank-r expansion t as three bf16 parts (t to fp32 precision), so its
 * logits differ from the others' in the last bits. */
archead_status archead_logits(const archead_handle* h, const void* x, int64_t M,
                              int64_t ldx, void* out, archead_dtype out_dtype,
                              int64_t ldo, void* ws, size_t ws_bytes,
                              void* stream);

/* Fused log-softmax and cross-entropy: ce[m] = logsumexp_v(logit[m, :]) -
 * logit[m, y_m] (natural log), and *mean_ce = (1/M) sum_m ce[m] when
 * mean_ce is not NULL.  This is the paper's CE / perplexity evaluation
 * (Section 4, "Data and metrics"; PPL = exp(mean CE)).  The [M, V] logits are
 * never written to memory: each vocabulary tile leaves a (max, sum of exp)
 * pair per token in the workspace and a merge kernel combines them in a fixed
 * order, so results are bitwise reproducible.
 *   targets  device int32 or int64 [M] (tgt_dtype ARCHEAD_I32 / ARCHEAD_I64)
 *   ce       device fp32 [M];  mean_ce  device fp32 scalar or NULL
 * A target outside [0, V) gives ce[m] = NaN (and a NaN mean); this is
 * detected on the device, the host does not synchronise. */
archead_status archead_logits_ce(const archead_handle* h, const void* x,
                                 int64_t M, int64_t ldx, const void* targets,
                                 archead_dtype tgt_dtype, float* ce,
                                 float* mean_ce, void* ws, size_t ws_bytes,
                                 void* stream);

/* Greedy decoding over the packed head: idx[m] = the smallest v attaining
 * max_v logit[m, v] and, when max_logit is not NULL, max_logit[m] = that
 * logit, for m < M.  The logits are the fp32 ones archead_logits computes
 * (the same kernel for the same M), so idx equals the first-index argmax of
 * its output, ties included.  This is the next-token choice of the
 * generation runs the paper times with the packed head in place ("Efficiency
 * and Calibration" and its throughput appendix), fused into the head pass,
 * and its top-1 agreement metric ("Logit Fidelity"): the [M, V]
 * logits are never written; each kernel leaves per-partial (max, smallest
 * index at the max) pairs in the workspace and a merge kernel combines them.
 *   idx        device int64 [M], 8-byte aligned
 *   max_logit  device fp32 [M] or NULL
 *   ws         archead_workspace_bytes(h, M, ARCHEAD_OP_ARGMAX) bytes
 * Other arguments and errors as archead_logits.  A token whose logits are
 * all NaN gets idx -1. */
archead_status archead_logits_argmax(const archead_handle* h, const void* x, int64_t M,
                                     int64_t ldx, int64_t* idx, float* max_logit, void* ws,
                                     size_t ws_bytes, void* stream);

/* Logit fidelity of the packed head against a dense bf16 head on the same
 * tokens, computed in the packed head's vocabulary-tile pass (Section 4,
 * "Logit Fidelity", and Table 8: KL, top-k agreement and logit MSE of a
 * compressed head against the dense one).  Per token m < M, with a = the
 * dense head's logits x W_dense^T and b = the packed head's logits (those of
 * archead_logits): kl[m] = KL(softmax(a) || softmax(b)), sq[m] = sum_v
 * (a_v - b_v)^2 (the MSE of Table 8 is its mean over tokens), ref_idx[m] =
 * the first v attaining max a, rank[m] = the number of v whose b is larger
 * than b at ref_idx[m], or equal at a smaller index (so the dense top-1 is
 * in the packed head's top k exactly when rank < k).  The tiled kernel
 * streams the dense head's rows through the same stages as the packed
 * codes and accumulates both products per tile (64 tokens x 256 rows); each
 * tile leaves per-token statistics, a merge kernel combines them in tile
 * order (fp64), and a second pass of the packed head counts the rank.  No
 * [M, V] array is written.  The same quantities as archead_logit_fidelity,
 * there from two logit arrays.
 *   dense      bf16 [V, ldw] device, 16-byte aligned, ldw >= d, ldw % 8 == 0
 *              (row v: the dense head's weights of vocabulary entry v)
 *   kl, sq     device fp32 [M];  ref_idx, rank  device int64 [M]
 *   ws         archead_workspace_bytes(h, M, ARCHEAD_OP_FIDELITY) bytes
 * The dense head is read once per 64 tokens (4 bytes per weight per 128
 * tokens); this is an evaluation pass.  ARCHEAD_E_UNSUPPORTED for heads
 * without the tiled kernel (g % 64 != 0) or ldw * 512 >= 2^31; other errors
 * as archead_logits. */
archead_status archead_logit_fidelity_head(const archead_handle* h, const void* x, int64_t M,
                                           int64_t ldx, const void* dense, int64_t ldw,
                                           float* kl, float* sq, int64_t* ref_idx,
                                           int64_t* rank, void* ws, size_t ws_bytes,
                                           void* stream);

/* Largest k of archead_logits_topk. */
#define ARCHEAD_TOPK_MAX 64

/* Top-k selection over the packed head: for m < M and j < k, idx[m * ldk +
 * j] is the j-th vocabulary index when the fp32 logits of token m (those
 * archead_logits computes for the same M) are sorted by decreasing value,
 * equal values by increasing index; vals[m * ldk + j] is its logit.  j = 0
 * is archead_logits_argmax's index.  This is the candidate set of top-k
 * decoding and of the top-k agreement metric ("Logit Fidelity", Section 4 and
 * its Table 8: top-1, top-5, top-10).  A single token on the decode GEMV
 * (M = 1 at the default ranges) selects inside the head pass: the [V]
 * logits are never written, each workgroup leaves its k best pairs in the
 * workspace and a merge kernel combines them.  Otherwise the logits of up to
 * 256 tokens at a time go to the workspace in fp32 (about 256 * V * 4
 * bytes) and a selection kernel reads them back.
 *   k          1 <= k <= min(ARCHEAD_TOPK_MAX, V)
 *   vals       device fp32 [M, ldk], 4-byte aligned, or NULL
 *   idx        device int64 [M, ldk], 8-byte aligned; ldk >= k
 *   ws         archead_workspace_bytes(h, M, ARCHEAD_OP_TOPK) bytes (it
 *              holds lists of ARCHEAD_TOPK_MAX entries, so any k fits)
 * NaN logits are never selected; slots that fewer than k non-NaN logits
 * leave empty get (-inf, -1).  Other arguments and errors as
 * archead_logits, plus ARCHEAD_E_INVALID_ARG for k out of range or
 * ldk < k. */
archead_status archead_logits_topk(const archead_handle* h, const void* x, int64_t M,
                                   int64_t ldx, int32_t k, float* vals, int64_t* idx,
                                   int64_t ldk, void* ws, size_t ws_bytes, void* stream);

/* Bytes of the static workspace of archead_logits_noalloc, one array per
 * device the library runs on (kept until the process ends). */
#define ARCHEAD_NOALLOC_SCRATCH_BYTES (4u << 20)

/* archead_logits without a caller workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  Same arguments, results and
 * kernels as archead_logits (bit-identical logits), except that the
 * workspace is a static device array of ARCHEAD_NOALLOC_SCRATCH_BYTES bytes
 * inside the library, whose device address archead_create takes once per
 * device.  The call allocates nothing (no hipMalloc, no allocating library
 * routine).
 *   Limit: M whose archead_workspace_bytes(h, M, ARCHEAD_OP_LOGITS) exceeds
 *   ARCHEAD_NOALLOC_SCRATCH_BYTES is rejected with ARCHEAD_E_WORKSPACE (the
 *   decode-shaped paths fit: at the Qwen3-8B shape, r_c + r_r = 96, every M
 *   up to 32; the many-token path's per-call tables do not).
 *   All calls on one GPU share that GPU's array, which keeps the last call's
 *   contents (no call needs it cleared): calls that overlap on one GPU, on
 *   different streams or from different threads, race and give undefined
 *   results; serialise them.
 * Errors as archead_logits, plus ARCHEAD_E_HIP when the array's address
 * could not be taken at create time. */
archead_status archead_logits_noalloc(const archead_handle* h, const void* x, int64_t M,
                                      int64_t ldx, void* out, archead_dtype out_dtype,
                                      int64_t ldo, void* stream);

/* Logit fidelity of `test` logits to reference logits `ref` (the paper's
 * "Logit Fidelity" metrics, Section 4 and its Table 8: the packed head
 * against the dense head on the same positions), per position m < M:
 *   kl[m]      = KL(p || q) = sum_v p_v (log p_v - log q_v), p = softmax(ref[m]),
 *                q = softmax(test[m]);
 *   sq[m]      = sum_v (ref[m, v] - test[m, v])^2 (its mean over positions is
 *                the logit MSE, the activation objective of Eq. (1));
 *   ref_idx[m] = the smallest v attaining max_v ref[m, v];
 *   rank[m]    = the number of v with test[m, v] > test[m, ref_idx[m]], plus
 *                those equal to it at a smaller index: the reference's top-1
 *                token is in the test top k exactly when rank < k (top-1
 *                agreement: rank == 0).
 *   ref, test  device fp32 [M, ld_ref] / [M, ld_test] row-major, ld >= V
 *   kl, sq     device fp32 [M];  ref_idx, rank  device int64 [M] (8-byte aligned)
 *   ws         device scratch of archead_fidelity_workspace_bytes(M, V)
 *              bytes, 256-byte aligned, caller-owned (per-chunk partials)
 *   stream     hipStream_t (NULL = the default stream); asynchronous
 * Sums are taken in fp64 over fp32 exponentials in a fixed order (the
 * result is reproducible).  Inputs must be finite.  M = 0 is a no-op.
 * ARCHEAD_E_INVALID_ARG for a null pointer, M < 0 or M > 65535, V < 1 or
 * V >= 2^31, or ld < V; ARCHEAD_E_MISALIGNED for a misaligned pointer;
 * ARCHEAD_E_WORKSPACE for a short workspace; ARCHEAD_E_HIP when a launch
 * fails. */
/* Bytes of workspace archead_logit_fidelity needs for M positions of V
 * logits (0 for M < 1 or V < 1). */
size_t archead_fidelity_workspace_bytes(int64_t M, int64_t V);
archead_status archead_logit_fidelity(const float* ref, int64_t ld_ref, const float* test,
                                      int64_t ld_test, int64_t M, int64_t V, float* kl,
                                      float* sq, int64_t* ref_idx, int64_t* rank, void* ws,
                                      size_t ws_bytes, void* stream);

/* Largest M served by the decode GEMV kernel when the MFMA decode kernel
 * does not take the call; larger M use the tiled MFMA kernel (unless
 * g % 64 != 0, which always takes the GEMV).
 * -1 restores the built-in threshold.  Not thread-safe with concurrent calls
 * on the same handle (set it once, after create). */
archead_status archead_set_gemv_max_m(archead_handle* h, int64_t m);
int64_t archead_get_gemv_max_m(const archead_handle* h);

/* Range of M served by the MFMA decode kernel, min_m <= M <= max_m (an
 * empty range, e.g. max_m = 0, never uses it; -1 restores the built-in
 * bound for the head shape, see archead_logits).  Same threading rule as archead_set_gemv_max_m.  get
 * returns ARCHEAD_E_INVALID_ARG for a NULL argument. */
archead_status archead_set_dec_range(archead_handle* h, int64_t min_m, int64_t max_m);
archead_status archead_get_dec_range(const archead_handle* h, int64_t* min_m, int64_t* max_m);

/* Range of M served by the several-token kernel when the MFMA decode kernel
 * does not take the call (-1 restores the built-in bound for the head
 * shape, see archead_logits; an empty range never uses it).  Same threading rule as
 * archead_set_gemv_max_m; get returns ARCHEAD_E_INVALID_ARG for a NULL
 * argument. */
archead_status archead_set_mid_range(archead_handle* h, int64_t min_m, int64_t max_m);
archead_status archead_get_mid_range(const archead_handle* h, int64_t* min_m, int64_t* max_m);

/* Head-derived tables of the many-token kernel (the path of archead_logits
 * and archead_logits_ce at large M) kept across calls.  Every call on that
 * path otherwise rebuilds, in its workspace and before stage 1, tables that
 * depend on the head alone: the ratios of consecutive residual group scales
 * and of the core and correction row scales, s_U and s_A (Section 3.2: the
 * three summands of the factorized head, accumulated in one fp32 register
 * chain), the V_c / B_w codes as bf16, and the U_c / A_w codes of each row
 * side by side.  archead_prepare builds them once into a caller-owned
 * buffer buf of bytes >= archead_prepared_bytes(h) bytes (device memory,
 * 256-byte aligned), asynchronously on `stream`; later calls read them from
 * there.  The caller keeps buf alive and unmodified, and the head's buffers
 * unchanged, until it detaches it (buf = NULL, bytes = 0) or destroys the
 * handle; calls on other streams must be ordered after `stream`'s work.
 * The workspace size of a call does not change.  Results are bit-identical
 * with and without a prepared buffer.  Same threading rule as
 * archead_set_gemv_max_m.
 * archead_prepared_bytes returns 0 for a NULL handle or a head with no
 * many-token kernel (g % 64 != 0).  archead_prepare: ARCHEAD_E_INVALID_ARG
 * for a NULL handle or buf = NULL with bytes > 0; ARCHEAD_E_UNSUPPORTED when
 * the head has no many-token kernel; ARCHEAD_E_MISALIGNED;
 * ARCHEAD_E_WORKSPACE for a short buffer; ARCHEAD_E_HIP when the launch
 * fails (the head is then left without a prepared buffer). */
size_t archead_prepared_bytes(const archead_handle* h);
archead_status archead_prepare(archead_handle* h, void* buf, size_t bytes, void* stream);

/* Launch settings of a handle, for tuning runs and tests; the library
 * reads no environment variables.  knob is one of:
 *   ARCHEAD_LAUNCH_GEMV_BLOCKS_PER_CU  resident decode-GEMV workgroups per CU
 *                                      (at most what the occupancy allows)
 *   ARCHEAD_LAUNCH_GEMV_GRID           decode-GEMV head-streaming workgroups
 *   ARCHEAD_LAUNCH_DEC_BLOCKS          consumer workgroups of the MFMA decode
 *                                      kernel (cap)
 *   ARCHEAD_LAUNCH_MID_BLOCKS          consumer workgroups of the
 *                                      several-token kernel (cap)
 *   ARCHEAD_LAUNCH_TILE_WAVES          waves per workgroup of the tiled
 *                                      kernel: 4 or 8
 *   ARCHEAD_LAUNCH_TILE_ROWS           token rows per tile of the 4-wave
 *                                      layout: 64 or 128
 *   ARCHEAD_LAUNCH_T_SPIN_LIMIT        polls of the in-launch stage-1
 *                                      exchange before a wave computes t
 *                                      itself (0: always computes it)
 * value 0 (the spin limit: -1) restores the built-in choice, which the
 * library otherwise makes per call from the head shape and M.  Every value
 * accepted keeps every kernel correct: the grids are persistent with
 * bounded indexes, and a consumer wave that outruns the producers computes
 * t itself after the bounded wait.  ARCHEAD_E_INVALID_ARG for a NULL handle
 * or pointer, an unknown knob, a negative size, a tile shape other than
 * those above, or a spin limit below -1.  Same threading rule as
 * archead_set_gemv_max_m; get returns the stored value (0 or -1 when
 * built-in). */
#define ARCHEAD_LAUNCH_GEMV_BLOCKS_PER_CU 0
#define ARCHEAD_LAUNCH_GEMV_GRID 1
#define ARCHEAD_LAUNCH_DEC_BLOCKS 2
#define ARCHEAD_LAUNCH_MID_BLOCKS 3
#define ARCHEAD_LAUNCH_TILE_WAVES 4
#define ARCHEAD_LAUNCH_TILE_ROWS 5
#define ARCHEAD_LAUNCH_T_SPIN_LIMIT 6
#define ARCHEAD_LAUNCH_KNOBS 7
archead_status archead_set_launch(archead_handle* h, int knob, int64_t value);
archead_status archead_get_launch(const archead_handle* h, int knob, int64_t* value);

/* Profiling hook: when start and stop are non-NULL hipEvent_t handles
 * (created by the caller on the handle's device), every later compute call
 * attaches `start` to the dispatch of the kernel that streams the packed head
 * and `stop` to its completion (the first and last dispatch when M needs
 * several), so hipEventElapsedTime gives that kernel's execution time alone.  NULL, NULL turns it off.  Same threading rule as
 * archead_set_gemv_max_m. */
archead_status archead_set_timing_events(archead_handle* h, void* start, void* stop);

/* ------------------------------------------------------------------------
 * Construction of a packed head from a dense head and calibration hidden
 * states (the paper's Algorithm 1 "ARCHead compression" and Algorithm 2
 * "Expanded packed-head construction"; Section 3.1 for the activation
 * metric, Section 3.2 for QuantizeCore and the correction):
 *   C_lambda = H^T H / N + lambda cbar I  (cbar = mean diagonal of H^T H / N)
 *   T_p = Q Lambda^p Q^T from C_lambda = Q Lambda Q^T, and T_p^-1
 *   A_c B_c = rank-r_c truncated SVD of W (A_c = U Sigma, B_c = V^T)
 *   QuantizeCore: core_u = Q5(A_c) (5-bit codes in [-15, 15] stored in the
 *     int8 container, one fp16 scale per row), core_v = Q8(B_c) (one scale
 *     per row), residual = Q_SC4(W - A_c B_c) in groups of g (the residual
 *     against the unquantized core)
 *   E = W - W_d (the realized error of the quantized core)
 *   E T_p ~ U_r Sigma_r V_r^T by a randomized SVD with the caller's
 *     Gaussian sketch omega and power_iters subspace iterations;
 *     A_w = U_r Sigma_r, B_w = V_r^T T_p^-1
 *   QuantizeINT8: corr_a per row, corr_b in groups of g_b along d.
 * Every quantizer: scale = fp16(absmax / qmax) (nearest even, from fp64),
 * code = clip(rint(value / scale), -qmax, qmax), qmax = 7 / 15 / 127; an
 * all-zero group gets scale 0 and codes 0.  All arithmetic is fp64 (rocBLAS
 * GEMMs, rocSOLVER eigen- and singular-value solvers, and this library's
 * kernels).  The randomized SVD's result is the truncated SVD of E T_p only
 * approximately (its error is bounded below by the exact tail).
 *
 * The written head has g_v = d and the descriptor
 * {V, d, g, r_c, r_r, g_v = d, g_b, ARCHEAD_INT4_V1, ARCHEAD_F16, ARCHEAD_I8}.
 */
typedef struct archead_build_desc {
  uint32_t abi_version;     /* ARCHEAD_ABI_VERSION */
  int64_t V, d, N;          /* dense head rows, hidden size, calibration tokens */
  int64_t g;                /* residual group along d (g % 32 == 0, d % g == 0) */
  int64_t r_c, r_r;         /* core and correction ranks (0 = component absent) */
  int64_t g_b;              /* group of the corr_b scales along d (d = one per row) */
  double p, lambda;         /* metric exponent, damping */
  int64_t oversample;       /* extra sketch columns of the randomized SVD */
  int64_t power_iters;      /* its subspace iterations */
} archead_build_desc;

/* Device workspace bytes archead_build_head needs (0 for an invalid
 * descriptor): about 17 V d + 8 N d + 56 d^2 bytes plus the factor-sized
 * buffers (fp64 copies of W, the residual / realized error, H, and the d x d
 * metric matrices). */
size_t archead_build_workspace_bytes(const archead_build_desc* b);

/* Build a packed head on the current device.
 *   W      fp32 [V, ldw] device, the dense head (ldw >= d)
 *   H      fp32 [N, ldh] device, calibration hidden states (ldh >= d)
 *   omega  fp64 [r_r + oversample, d] device, row-major: the sketch of the
 *          randomized SVD (i.i.d. standard normal draws; ignored when r_r = 0)
 *   out    device buffers to fill, in the layouts of archead_ptrs with the
 *          descriptor above (res_codes 4-byte aligned; res_row_scales unused)
 *   a_w, b_w  optional fp64 device outputs of the unquantized correction
 *          factors, [V, r_r] and [r_r, d] row-major (NULL to skip)
 *   ws     device workspace of archead_build_workspace_bytes(b) bytes,
 *          256-byte aligned
 *   stream hipStream_t (NULL = the default stream)
 * Synchronous: returns after the work on `stream` has finished.  The dense
 * library calls run through a rocBLAS handle created for the call, whose own
 * device workspace rocBLAS manages; the forward entry points never do this.
 * ARCHEAD_E_INVALID_ARG for a bad descriptor, a NULL buffer of a present
 * component, or a damped covariance that is not positive definite;
 * ARCHEAD_E_MISALIGNED; ARCHEAD_E_WORKSPACE; ARCHEAD_E_UNSUPPORTED for
 * shapes beyond 32-bit library sizes; ARCHEAD_E_HIP when a launch fails or
 * a solver does not converge. */
archead_status archead_build_head(const archead_build_desc* b, const float* W, int64_t ldw,
                                  const float* H, int64_t ldh, const double* omega,
                                  const archead_ptrs* out, double* a_w, double* b_w, void* ws,
                                  size_t ws_bytes, void* stream);

/* Persistent bytes of the packed head: the sum over its buffers of element
 * count times element size (the paper's bytes(ARCHead), Section 3.3).
 * 0 for an invalid descriptor. */
uint64_t archead_packed_bytes(const archead_desc* desc);

/* Host-side 5-bit packing to / from ARCHEAD_I5 (no HIP call).
 * codes: int8 [rows, r] with values in [-16, 15]; packed: uint32
 * [rows, ceil(r / 6)].  pack returns ARCHEAD_E_INVALID_ARG for a code out of
 * range, r < 1 or rows < 0. */
archead_status archead_pack_int5(const int8_t* codes, int64_t rows, int64_t r, uint32_t* packed);
archead_status archead_unpack_int5(const uint32_t* packed, int64_t rows, int64_t r,
                                   int8_t* codes);

/* Host-side INT4 packing to / from ARCHEAD_INT4_V1 (no HIP call).
 * codes: int8 [rows, d] with values in [-8, 7]; packed: uint8 [rows, d/2];
 * d % 8 == 0.  pack returns ARCHEAD_E_INVALID_ARG for a code out of range. */
archead_status archead_pack_int4(const int8_t* codes, int64_t rows, int64_t d,
                                 uint8_t* packed);
archead_status archead_unpack_int4(const uint8_t* packed, int64_t rows, int64_t d,
                                   int8_t* codes);

const char* archead_status_str(archead_status s);
/* Message of the last failing call on this thread ("" if none). */
const char* archead_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ARCHEAD_H_ */
