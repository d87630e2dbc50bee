/*
 * viscache.h -- C ABI of libviscache, a gfx950 (MI355X) implementation of
 * PruneKV, the visual KV-cache compression step of VisCache (Sec. 3.2,
 * "PruneKV: Layer-Aware Visual KV Cache Compression", and Appendix B,
 * Algorithm 1), plus decode attention over the compressed cache (Sec. 2,
 * "VLLM Decoding").
 *
 * Conventions for every entry point
 *   - Plain C types only.  Device pointers are addresses returned by the HIP
 *     allocator (or by a framework that uses it); host pointers are ordinary
 *     process memory.  Each argument says which one it is.
 *   - The caller owns every buffer.  The library never allocates or frees
 *     device memory, never synchronises a stream and keeps no mutable global
 *     state shared between threads: calls on different streams with
 *     different buffers may overlap.  Each calling thread keeps a host copy
 *     of its last plan (budgets, offsets, fusion job lists) and reuses it
 *     while the shape, the lengths n_vis[] and the parameters compare equal
 *     by value, so repeated calls of one shape plan once.
 *   - Sizes of outputs and of the workspace come from the host-only query
 *     functions below, so the device path needs no device-to-host copy.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Device work is enqueued asynchronously on it.
 *   - Every argument and shape check runs on the host before anything is
 *     enqueued; on error nothing is enqueued and the status says why.
 *     VC_ERR_HIP reports a failed launch.  Faults inside kernels surface at
 *     the caller's next synchronisation, as for any HIP kernel.
 *   - Inputs must be finite; non-finite values give unspecified results.
 *   - bf16 means IEEE binary32 truncated to its upper 16 bits (bfloat16),
 *     stored as 2-byte values.
 */
#ifndef VISCACHE_H
#define VISCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  VC_OK = 0,
  VC_ERR_ARG = 1,         /* null pointer, bad enum or out-of-range scalar */
  VC_ERR_SHAPE = 2,       /* inconsistent or unsupported shape */
  VC_ERR_BUDGET = 3,      /* retention / h / m give no valid budget (e.g. q > 1) */
  VC_ERR_WORKSPACE = 4,   /* workspace missing or smaller than required */
  VC_ERR_UNSUPPORTED = 5, /* shape outside what the kernels are built for */
  VC_ERR_HIP = 6          /* a HIP runtime call or launch failed */
} vc_status;

/* Which score ranks the tokens of a layer (Sec. "Ablation on Shared vs.
 * Layer-Specific Visual Token Ranking").
 *   LAYER_HEAD: every (layer, kv head) ranks by its own window score.
 *   GLOBAL:     one shared score per token, summed over all L layers and all
 *               kv heads; every layer and head keeps the top-k_l of it. */
typedef enum { VC_RANK_LAYER_HEAD = 0, VC_RANK_GLOBAL = 1 } vc_rank_mode;

/* Layer budget schedule: the proportions b_l, l = 1..h, before they are
 * normalised to h*m.  PARABOLIC is PruneKV's Eq. (parabolic); the others are
 * the alternatives of the budget ablation (Sec. 5, Table "Ablation study on
 * budget allocation strategy"), whose constants the paper leaves open:
 *   FIXED:      b_l = 1 (uniform);
 *   ARITHMETIC: linear from b_1 = 1 to b_h = 1/2 (the raw parabola's
 *               endpoints), b_l = 1 - (l-1) / (2 (h-1));
 *   GEOMETRIC:  layers 1..h in four equal depth blocks, block j (0-based,
 *               j = floor(4 (l-1) / h)) gets b_l = 2^-j. */
typedef enum {
  VC_SCHED_PARABOLIC = 0,
  VC_SCHED_FIXED = 1,
  VC_SCHED_ARITHMETIC = 2,
  VC_SCHED_GEOMETRIC = 3
} vc_schedule;

/* Which queries score the visual tokens (Eq. (token_score): the attention a
 * token receives, summed over queries).
 *   WINDOW:  the W trailing text queries of the prefill attend the n_b visual
 *            keys, softmax over those keys only (the observation-window
 *            reading; the default).
 *   PREFILL: every token of the prefill is a query, as the equation is
 *            written (its sum runs over all N tokens): the sequence is the
 *            n_b visual tokens followed by the W text tokens, token i attends
 *            tokens 0..i (causal self-attention, visual then text keys), and a
 *            visual token's score sums its attention weight over all heads of
 *            the group and all tokens i at or after it. */
typedef enum { VC_SCORE_WINDOW = 0, VC_SCORE_PREFILL = 1 } vc_score_queries;

/* Method parameters.  Defaults (viscache_default_params) are the paper's fixed
 * hyper-parameters from Sec. 4, Implementation Details: h = 3/4 L, m = 0.75,
 * tau = 1.0, mu = 0.7, the parabolic schedule, fusion of the top-q
 * survivors. */
typedef struct {
  double retention; /* overall retention ratio RR in (0, 1]; RR = q*(h/L)*m, so
                       the token-level ratio is q = RR / ((h/L) m), and q > 1 is
                       VC_ERR_BUDGET.  The totals satisfy
                       sum_l k_l = floor(RR*L*n + 0.5) per sequence. */
  int32_t h;        /* truncation layer in [2, L]; layers past h are evicted.
                       0 selects floor(0.75 L + 0.5). */
  double m;         /* mean layer budget in (0, 1] (normalisation target h*m
                       of Eq. (parabolic)). */
  float tau;        /* temperature of Eq. (redistribution), > 0 */
  float mu;         /* fusion weight of Eq. (weight_fusion), in [0, 1] */
  int32_t rank_mode;  /* vc_rank_mode */
  int32_t v_out_fp32; /* 0: fused values stored as bf16; 1: stored as fp32 */
  int32_t schedule;   /* vc_schedule */
  int32_t drop_all;   /* 0: the dropped tokens whose values are fused are the
                         survivors of the top-q cut outside the kept set
                         (Algorithm 1, n_surv = min(n, max(round(q n), k_1)));
                         1: every token outside the kept set (n_surv = n),
                         the reading of Eq. (redistribution) alone. */
  int32_t score_queries; /* vc_score_queries; default VC_SCORE_WINDOW */
} vc_params;

/* Problem shape.  L layers, Hq query heads, Hkv kv heads (Hq % Hkv == 0;
 * query head hq reads kv head hq / (Hq/Hkv)), head dim d in {64, 128},
 * W window queries per head (with VC_SCORE_PREFILL: W text tokens per
 * sequence), B sequences with n_vis[b] visual tokens each.
 * VC_ERR_UNSUPPORTED beyond the kernels' limits: d, (Hq/Hkv)*W > 1024 with
 * window scores, (Hq/Hkv)*(n_vis[b] + W) > 2^26 with prefill scores,
 * n_vis[b] > 32768, 64*L + 12*B + 16 > 30720 (the layer table and the
 * per-sequence offsets must fit the first 30 KB of the launch plan), a score
 * grid of 2^24 or more workgroups (Ls*B*Hkv units, Ls = h or L, times the
 * workgroups per unit), or 2^23 or more units (layer < h, sequence, kv head)
 * with kept tokens (the fusion job code holds a unit's rank in 23 bits). */
typedef struct {
  int32_t B, L, Hq, Hkv, d, W;
  const int32_t *n_vis; /* HOST array [B]; each entry in [0, 32768] */
} vc_shape;

/* Fill *p with the defaults above and the given retention. */
void viscache_default_params(vc_params *p, double retention);

/* Host only.  Layer budgets (the schedule normalised to h*m; Eq.
 * (parabolic) by default) and the survivor count of Algorithm 1 Step 1:
 *   k[b*L + l]      tokens kept in layer l of sequence b (0 for l >= h),
 *   n_surv[b*L + l] tokens that survive the top-q cut (same for every l),
 *   *h_out          the truncation layer used (may be NULL).
 * Returns VC_ERR_BUDGET for parameters without a valid budget. */
vc_status viscache_budget(const vc_shape *shape, const vc_params *params, int32_t *k,
                          int32_t *n_surv, int32_t *h_out);

/* Host only.  Output row offsets: rows[l*(B+1) + b] = sum_{b' < b} Hkv*k[b'*L+l]
 * for b = 0..B, so layer l's outputs hold rows[l*(B+1)+B] rows.  `rows` is a
 * HOST array of L*(B+1) entries. */
vc_status viscache_out_rows(const vc_shape *shape, const vc_params *params, int64_t *rows);

/* Host only.  Bytes of device workspace viscache_prune needs (0 on error). */
size_t viscache_prune_workspace_bytes(const vc_shape *shape, const vc_params *params);

/* Host only, diagnostic.  Byte offsets inside the prune workspace where
 * viscache_prune leaves its fp32 window scores once the call has completed:
 *   *scores_off: [Ls][sum_b Hkv*n_b], Ls = h (LAYER_HEAD) or L (GLOBAL), the
 *                score of token v of (layer l, sequence b, kv head g) at
 *                l*(sum_b Hkv*n_b) + off_b*Hkv + g*n_b + v;
 *   *shared_off: [sum_b n_b] shared scores (GLOBAL), token v of b at off_b + v;
 *                set to (size_t)-1 in LAYER_HEAD mode.
 * The contents stay valid until the workspace is reused. */
vc_status viscache_prune_score_offsets(const vc_shape *shape, const vc_params *params,
                                       size_t *scores_off, size_t *shared_off);

/* Buffers of one viscache_prune call.  Every member is a HOST array of L
 * DEVICE pointers, one per layer l.
 *   k_in[l], v_in[l]: bf16 visual keys / values of layer l, packed over
 *       sequences: row (b, g, v) at off_b*Hkv + g*n_b + v with
 *       off_b = sum_{b'<b} n_{b'}; each row holds d values.
 *   q_win[l]: fp32 window queries [B][Hq][W][d].  They enter the score
 *       contraction rounded to bf16 (round to nearest even).
 *   k_out[l]: bf16 kept keys, bit copies of the input rows; v_out[l]: fused
 *       values, bf16 or fp32 (vc_params.v_out_fp32); idx_out[l]: int32 token
 *       index (0..n_b-1) of every kept row.  Output row (b, g, j) sits at
 *       rows[l*(B+1)+b] + g*k[b*L+l] + j, rows ascending in token index.
 *       Layers l >= h have no rows; their pointers may be NULL.
 *   k_text (read with VC_SCORE_PREFILL only; may be NULL otherwise):
 *       k_text[l] holds the bf16 keys of the W text tokens of layer l,
 *       [B][Hkv][W][d].  With VC_SCORE_PREFILL, q_win[l] holds the fp32
 *       queries of every token instead of the window: row (b, hq, i) at
 *       (qoff_b*Hq + hq*(n_b + W) + i)*d, qoff_b = sum_{b'<b} (n_b' + W),
 *       tokens i < n_b visual, then the W text tokens.
 *   drop_out: may be NULL.  Otherwise drop_out[l] receives, per (b, g), the
 *       r = n_surv - k token indices whose values were fused (ascending),
 *       at dropped-row offset sum_{b'<b} Hkv*r_{b',l} + g*r_{b,l}.
 * Input buffers are read only; outputs must not overlap inputs. */
typedef struct {
  const void *const *k_in;
  const void *const *v_in;
  const float *const *q_win;
  void *const *k_out;
  void *const *v_out;
  int32_t *const *idx_out;
  int32_t *const *drop_out;
  const void *const *k_text;
} vc_prune_io;

/* Device, asynchronous.  PruneKV over all layers and sequences (Algorithm 1):
 * window scores (Eq. (token_score), read as the attention of the W window
 * queries, softmax over the n_b visual keys with scale 1/sqrt(d), summed over
 * the Hq/Hkv query heads of each kv head; or, with VC_SCORE_PREFILL, the
 * causal attention of every prefill token as described at vc_score_queries),
 * budgets as viscache_budget, the
 * keep set (top-k_l) and drop set (ranks k_l+1..n_surv) from one ranking
 * ordered by (score descending, token index ascending), key pruning, and
 * value fusion V_new = mu V_k + (1-mu) softmax(V_k V_d^T / tau) V_d
 * (Eq. (redistribution), Eq. (weight_fusion)); with no dropped or no kept
 * rows the kept values are copied unchanged.
 * `workspace` is a DEVICE buffer of at least viscache_prune_workspace_bytes
 * bytes, 256-byte aligned; its contents on entry do not matter. */
vc_status viscache_prune(const vc_shape *shape, const vc_params *params, const vc_prune_io *io,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Number of events viscache_prune_staged records. */
#define VC_PRUNE_EVENTS 7

/* Device, asynchronous.  viscache_prune with stage timing: `events` is a HOST
 * array of VC_PRUNE_EVENTS hipEvent_t handles (passed as void*) created by the
 * caller; event i is recorded on `stream` before stage i and the last one
 * after the final stage.  Stages: 0 plan upload past its first 30 KB
 * (empty for most shapes: the first 30 KB travel with stage 1), 1 score row
 * statistics, 2 score column sums, 3 shared-score reduction (empty in
 * LAYER_HEAD mode), 4 keep/drop selection, 5 key gather and value fusion.
 * events == NULL behaves exactly as viscache_prune. */
vc_status viscache_prune_staged(const vc_shape *shape, const vc_params *params,
                                const vc_prune_io *io, void *workspace, size_t workspace_bytes,
                                void *stream, void *const *events);

/* ---- decode over a (compressed) cache ------------------------------------ */

/* Decode shape: L layers, B sequences, Hq query heads, Hkv kv heads, head dim
 * d in {64, 128}, Hq/Hkv <= 16. */
typedef struct {
  int32_t B, L, Hq, Hkv, d;
} vc_decode_shape;

/* Cache pool for decode.  All layers' caches live in one pair of DEVICE bf16
 * row pools k_pool / v_pool (d values per row).  Unit u = (l*B + b)*Hkv + g
 * (layer l, sequence b, kv head g) owns the contiguous rows
 * [row_off[u], row_off[u] + cap[u]) of both pools and currently holds len[u]
 * rows.  row_off (int64), cap and len (int32) are DEVICE arrays of L*B*Hkv
 * entries; the blocks of different units must not overlap. */
typedef struct {
  void *k_pool;
  void *v_pool;
  const int64_t *row_off;
  const int32_t *cap;
  int32_t *len;
} vc_cache;

/* Host only.  Workspace bytes viscache_decode_attn needs for caches of at most
 * max_rows rows per (layer, sequence, kv head); 0 if the shape is invalid or
 * max_rows is negative or so large that L*B*Hkv*ceil(max_rows/32) reaches
 * 2^31. */
size_t viscache_decode_workspace_bytes(const vc_decode_shape *shape, int64_t max_rows);

/* Device, asynchronous.  Appends one key and one value row per unit
 * (Sec. 2, decoding: K <- concat[K, h_t W_K], V <- concat[V, h_t W_V]) at
 * row row_off[u] + len[u] and then increments len[u].  k_new, v_new: DEVICE bf16
 * [L][B][Hkv][d].  A full cache (len == cap) is left unchanged and its length
 * is not incremented. */
vc_status viscache_append_kv(const vc_decode_shape *shape, const vc_cache *cache,
                             const void *k_new, const void *v_new, void *stream);

/* Device, asynchronous.  Decode attention of one new token per sequence and
 * layer: out[l][b][hq] = softmax_t(scale * q[l][b][hq] . K_t) V_t over the
 * len rows of (l, b, hq / (Hq/Hkv)).  q: DEVICE bf16 [L][B][Hq][d]; out:
 * DEVICE fp32 [L][B][Hq][d]; a cache of length 0 gives zeros.  `workspace`:
 * DEVICE, at least viscache_decode_workspace_bytes(shape, max_rows) bytes,
 * where max_rows bounds every len (rows past max_rows are not attended;
 * VC_ERR_UNSUPPORTED where the workspace size is 0); 256-byte aligned.  Work
 * is balanced over capacities: each unit's cap rows (at most max_rows) are
 * cut into pieces of nearly equal size, their number in proportion to cap,
 * one workgroup each, so a cache whose units differ widely in length
 * still fills the chip when cap tracks len.  Where a unit's rows are cut
 * changes its result only by rounding. */
vc_status viscache_decode_attn(const vc_decode_shape *shape, const vc_cache *cache, const void *q,
                               float *out, float scale, int64_t max_rows, void *workspace,
                               size_t workspace_bytes, void *stream);

/* Host only.  Workspace bytes viscache_decode_step needs (the decode
 * workspace plus one arrival counter per unit); 0 where
 * viscache_decode_workspace_bytes is 0. */
size_t viscache_decode_step_workspace_bytes(const vc_decode_shape *shape, int64_t max_rows);

/* Device, asynchronous.  One decode step in a single launch, with the result
 * of viscache_append_kv followed by viscache_decode_attn (Sec. 2, decoding):
 * the new K/V row of every unit (k_new, v_new: DEVICE bf16 [L][B][Hkv][d]) is
 * appended where there is room and attended together with the cached rows;
 * q, out, scale and max_rows as for viscache_decode_attn (max_rows also
 * bounds the length after the append).  `workspace`: DEVICE, at least
 * viscache_decode_step_workspace_bytes(shape, max_rows) bytes, 256-byte
 * aligned, zero-filled before its first use and not modified by the caller
 * between calls (the call leaves its counters at zero).  Calls sharing a
 * workspace must be ordered on one stream. */
vc_status viscache_decode_step(const vc_decode_shape *shape, const vc_cache *cache, const void *k_new,
                               const void *v_new, const void *q, float *out, float scale,
                               int64_t max_rows, void *workspace, size_t workspace_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * library keeps one scratch array of VC_DECODE_NOALLOC_BYTES per device in
 * its code object, held from load until the process ends, with room for the
 * arrival counters of VC_DECODE_NOALLOC_UNITS units and the partial results
 * of the launch's pieces. */
#define VC_DECODE_NOALLOC_BYTES (16u << 20)
#define VC_DECODE_NOALLOC_UNITS 65536

/* Device, asynchronous.  viscache_decode_step without a workspace argument:
 * the same append, attention and merge, the same results bit for bit, with
 * the partial results and arrival counters in the library's scratch array of
 * the current device (which must be the device of `stream` and of every
 * pointer).  Allocates nothing: no hipMalloc, hipFree or allocating library
 * call.  The first call on a device looks the array up and enqueues a clear
 * of its counters on `stream`; every call leaves the counters at zero.
 * Calls that overlap on one device race on the array: order them on one
 * stream (calls on different devices are independent).  Every other
 * argument and error as for viscache_decode_step, plus VC_ERR_WORKSPACE
 * when L*B*Hkv > VC_DECODE_NOALLOC_UNITS or the partial results of the
 * launch (16 (d + 2) floats per workgroup, workgroups as for
 * viscache_decode_step_workspace_bytes) do not fit beside the counters. */
vc_status viscache_decode_step_noalloc(const vc_decode_shape *shape, const vc_cache *cache, const void *k_new,
                                       const void *v_new, const void *q, float *out, float scale,
                                       int64_t max_rows, void *stream);

/* ---- 4-bit cache rows ----------------------------------------------------
 * The quantisation experiments combine the pruned cache with 4-bit KV-cache
 * quantisation but do not define the quantiser.  The reading taken here: each
 * row's d channels form d/32 groups of 32; a group keeps lo = min and
 * scale = (max - min) / 15 as fp32 and its channels the 4-bit codes
 * clamp(rint((x - lo) / scale), 0, 15) (0 when scale = 0), all in IEEE fp32;
 * a row is read back as bf16(fma(code, scale, lo)).  Keys and values alike,
 * per row, so a tile of rows reads back without any other rows' data.
 * codes: uint8 [rows][d/2], channel 2j in the low nibble of byte j, 2j+1 in
 * the high one; meta: fp32 [rows][d/32][2] = (scale, lo). */

/* Device, asynchronous.  Quantises `rows` contiguous bf16 rows of d values
 * (src, DEVICE [rows][d]) into codes and meta (DEVICE, laid out as above;
 * the caller owns all three).  src and codes must be 16-byte aligned, meta
 * 8-byte aligned.  VC_ERR_UNSUPPORTED unless d is 64 or 128; VC_ERR_ARG for
 * rows < 0 or, with rows > 0, a null or misaligned pointer.  rows = 0 does
 * nothing. */
vc_status viscache_quantize_rows(int32_t d, int64_t rows, const void *src, void *codes, void *meta, void *stream);

/* A 4-bit prefix of a decode cache: rows [0, nq[u]) of unit u are read from
 * the quantised pools at rows qrow_off[u] + i (codes and meta as above, for
 * keys and values), rows [nq[u], len[u]) from the bf16 pools of the vc_cache
 * as usual (appended rows always go there).  nq[u] must be a multiple of 32
 * and at most len[u]; the kernel rounds it down to a multiple of 32 and
 * clamps it to len[u].  qrow_off (int64) and nq (int32): DEVICE arrays of
 * L*B*Hkv entries.  All pointers DEVICE. */
typedef struct {
  const void *k_codes;
  const void *k_meta;
  const void *v_codes;
  const void *v_meta;
  const int64_t *qrow_off;
  const int32_t *nq;
} vc_qcache;

/* Device, asynchronous.  viscache_decode_step over a cache whose leading rows
 * are 4-bit (read back as described above before they enter the products);
 * every other argument, the workspace (viscache_decode_step_workspace_bytes)
 * and the errors as for viscache_decode_step, plus VC_ERR_ARG for a null
 * qcache member, code arrays not 4-byte aligned or meta arrays not 8-byte
 * aligned. */
vc_status viscache_decode_step_q4(const vc_decode_shape *shape, const vc_cache *cache, const vc_qcache *qcache,
                                  const void *k_new, const void *v_new, const void *q, float *out, float scale,
                                  int64_t max_rows, void *workspace, size_t workspace_bytes, void *stream);

/* ---- decode with a piece table built once per cache ----------------------
 * The decode calls above cut every unit's rows into workgroup pieces on the
 * device, in every step, from the capacities.  Capacities do not change
 * between steps, so the cut can be made once, on the host, from host copies
 * of cap and row_off (Sec. 2, decoding: the cache of each step is the
 * previous one plus one row). */

/* Host only.  Bytes of the piece table for decode steps of this shape and row
 * bound (a 32-byte header and 32 bytes per workgroup of the launch); 0 where
 * viscache_decode_step_workspace_bytes is 0. */
size_t viscache_decode_plan_bytes(const vc_decode_shape *shape, int64_t max_rows);

/* Host only.  Builds the piece table of the caches whose capacities and first
 * pool rows are cap and row_off (HOST arrays of L*B*Hkv entries, the same
 * values as the vc_cache's device arrays) into `plan` (HOST, 4-byte aligned,
 * at least viscache_decode_plan_bytes bytes), for steps with this max_rows.
 * len_hint (HOST, L*B*Hkv entries, or NULL) are the units' lengths now: the
 * step requests each wave's first rows before it has read the unit's length,
 * and with the hint it does so only up to 64 rows past it (rows beyond are
 * read once the length is known), which keeps it from reading the unused
 * end of a cache whose capacity reaches far past its length; a stale hint
 * costs time, never correctness.
 * The caller copies the table to device memory and passes it to
 * viscache_decode_step_planned.  Each unit's min(cap, max_rows) rows are cut
 * into whole 32-row tiles; a workgroup's piece is shared by its four waves in
 * runs of consecutive tiles, and the table takes the smallest per-wave share
 * (at least two tiles) for which the pieces fit the launch.  VC_ERR_ARG for
 * a null cap, row_off or plan, a negative capacity, offset or length,
 * negative max_rows, or units whose blocks overlap; VC_ERR_UNSUPPORTED for a
 * capacity above 2^31 - 65 or a size viscache_decode_plan_bytes refuses;
 * VC_ERR_WORKSPACE if plan_bytes
 * is too small.  The table stays valid while cap and row_off do not change;
 * after a change, build it again (a stale table attends the wrong rows and
 * may read outside the caches' blocks). */
vc_status viscache_decode_plan(const vc_decode_shape *shape, const int32_t *cap, const int64_t *row_off,
                               const int32_t *len_hint, int64_t max_rows, void *plan, size_t plan_bytes);

/* Device, asynchronous.  viscache_decode_step (qcache NULL) or
 * viscache_decode_step_q4 (qcache non-NULL, as there) over the cut of a piece
 * table: the same append, attention and merge, equal to those calls up to
 * rounding (the pieces differ).  plan: DEVICE copy of a table from
 * viscache_decode_plan for this cache, shape and max_rows, 16-byte aligned,
 * plan_bytes at least viscache_decode_plan_bytes; a table built for another
 * shape or max_rows fills `out` with NaN.  The workspace is that of
 * viscache_decode_step (viscache_decode_step_workspace_bytes, zero-filled
 * before its first use, left at zero by every call); calls sharing it must be
 * ordered on one stream.  Every other argument and error as for
 * viscache_decode_step and viscache_decode_step_q4, plus VC_ERR_ARG for a
 * null or misaligned plan or a too small plan_bytes. */
vc_status viscache_decode_step_planned(const vc_decode_shape *shape, const vc_cache *cache, const vc_qcache *qcache,
                                       const void *plan, size_t plan_bytes, const void *k_new, const void *v_new,
                                       const void *q, float *out, float scale, int64_t max_rows, void *workspace,
                                       size_t workspace_bytes, void *stream);

/* Static text for a status code. */
const char *viscache_strerror(vc_status s);

#ifdef __cplusplus
}
#endif
#endif /* VISCACHE_H */
