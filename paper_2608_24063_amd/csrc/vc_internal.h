// vc_internal.h -- plan passed by value to the PruneKV kernels, and the host
// launchers each kernel file exports to the C ABI layer.  Internal.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace vc {

// Indices into the per-layer pointer table.
enum { LP_K_IN = 0, LP_V_IN, LP_Q, LP_K_OUT, LP_V_OUT, LP_IDX, LP_DROP, LP_K_TEXT, LP_COUNT };

// Tile sizes shared by host-side grid sizing and the kernels.
constexpr int kStatsRows = 256;   // query rows per stats workgroup (4 waves x 64)
constexpr int kKeyTile = 64;      // keys staged per LDS tile
constexpr int kColKeys = 256;     // keys per column-sum workgroup (4 waves x 64)
constexpr int kScoreSlots = 512;  // resident stats workgroups (256 CUs x 2)
constexpr int kMaxSplits = 8;     // key splits of the stats pass
constexpr int kFuseRows = 128;    // kept rows per fusion workgroup (4 waves x 32)
constexpr int kDropTile = 64;     // dropped rows staged per LDS tile
constexpr int kSelectThreads = 1024;
constexpr int kSelectPerThread = 32;  // => n <= 32768 tokens per sequence
constexpr int kMaxTokens = kSelectThreads * kSelectPerThread;
constexpr int kXcdsHost = 8;      // MI355X accelerator dies (host-side grid planning)

// One fusion unit (layer, sequence, kv head) with kept rows, as the fusion
// kernel reads it: absolute addresses of the unit's first rows and its sizes.
struct FuseUnit {
  uint64_t k_in, v_in;     // bf16 [n][d] input keys / values of the unit
  uint64_t k_out, v_out;   // bf16 [k][d] pruned keys; bf16 or fp32 [k][d] fused values
  uint64_t kept, drop;     // int32 [k] kept / [r] dropped token indices
  int32_t k, r, n, pad;
};
static_assert(sizeof(FuseUnit) == 64, "fusion unit record is four 16-byte words");

// The plan travels to the device as kernel arguments, in chunks of at most
// kChunkWords words: the first with the score statistics launch (which
// copies it into the workspace and reads its own tables from it), any
// further ones with upload launches.
constexpr uint32_t kChunkWordsSmall = 480, kChunkWordsMid = 2040, kChunkWords = 7680;  // 1.9 / 8 / 30 KB
template <uint32_t W>
struct UploadChunk {
  uint32_t words;
  uint32_t pad;
  uint32_t data[W];
};

// Everything the prune kernels need, by value (a few hundred bytes).  Array
// members point into the device workspace, filled from the plan chunks.
struct PrunePlan {
  int32_t B, L, Hq, Hkv, d, W, G, R;
  int32_t h;          // truncation layer: layers [0, h) keep tokens
  int32_t Ls;         // scored layers: h (layer/head ranking) or L (global)
  int32_t mode;       // 0 layer/head, 1 global
  int32_t v_fp32;     // fused values stored as fp32
  int32_t nqg, nks;   // stats grid: query groups x key splits per unit
  int32_t ncol;       // column-sum chunks per unit (max over sequences)
  int32_t nfunits;    // units with kept rows
  int32_t nfwg;       // fusion workgroups (persistent; a multiple of 8, the same number per XCD)
  int32_t nmax;       // max n_b
  int32_t pwg;        // prefill: workgroups per unit (each owns every pwg-th 256-row group)
  float sc;           // log2(e) / sqrt(d)
  float tc;           // log2(e) / tau
  float mu;
  int64_t Ntot;       // sum_b n_b
  int32_t w_lp, w_toff, w_nb;  // word offsets of those tables in the plan (first chunk)
  const uint64_t *lp;   // [LP_COUNT][L] per-layer device pointers
  const int32_t *nb;    // [B]
  const int64_t *toff;  // [B+1] token offsets
  const int32_t *kk;    // [B*L] kept per (b, l)
  const int32_t *ns;    // [B*L] survivors per (b, l)
  const int64_t *orow;  // [L*(B+1)] output row offsets per layer
  const int64_t *drow;  // [L*(B+1)] dropped-row offsets per layer
  const FuseUnit *funit; // [nfunits] fusion units, most dropped rows first
  const int32_t *fwoff;  // [9] job queue offsets per XCD
  const int32_t *fwjob;  // fusion jobs: unit rank << 8 | 128-row tile, each queue longest first
  int32_t *fcnt;         // [8] jobs handed out per queue (reset by every plan upload)
  uint16_t *qbf;        // [Ls][B][Hq][W][d] window queries in bf16
  float2 *part;         // [U][nks][R] partial row statistics (max*sc, sum)
  float *pcol;          // prefill: [U][pwg][nmax] column partials of each workgroup
  float *S;             // [Ls][Ntot*Hkv] window scores
  float *gs;            // [Ntot] shared (global) scores
};

// Host-side launchers (each returns hipSuccess or the launch error).
hipError_t launch_upload(uint8_t *dst, const uint8_t *src, size_t bytes, hipStream_t st);
// Score statistics; also writes the plan's first chunk (src, words <=
// kChunkWords) to dst.
hipError_t launch_score_stats(const PrunePlan &p, uint32_t *dst, const uint8_t *src, uint32_t words,
                              hipStream_t st);
hipError_t launch_score_colsum(const PrunePlan &p, hipStream_t st);
hipError_t launch_score_global(const PrunePlan &p, hipStream_t st);
// Prefill scores (every prefill token a query, causal): column partials per
// workgroup, carrying the plan's first chunk like launch_score_stats, then
// their fixed-order sum into S.
hipError_t launch_pscore(const PrunePlan &p, uint32_t *dst, const uint8_t *src, uint32_t words, hipStream_t st);
hipError_t launch_pscore_reduce(const PrunePlan &p, hipStream_t st);
hipError_t launch_select(const PrunePlan &p, hipStream_t st);
hipError_t launch_fuse(const PrunePlan &p, hipStream_t st);

// Decode work is dealt out in 32-row tiles: the tiles of each unit's capacity
// are split into pieces, one workgroup per piece (the device picks the piece
// size).
constexpr int kDecodeTileRows = 32;
constexpr int kDecodeSlots = 512;  // resident decode workgroups (256 CUs x 2)
constexpr int kDecodeMinPiece = 8; // smallest piece bound in tiles (a multiple of 4)

// Workgroups of a decode launch over `units` caches of at most max_rows rows:
// the resident slots (more for many units: each unit takes at least one
// piece), at most the pieces of kDecodeMinPiece tiles the rows can form, and
// always more than `units`, which the device's fallback piece size relies
// on.  0 if the tile count of the bound does not fit 31 bits.
inline int32_t decode_grid(int64_t units, int64_t max_rows) {
  if (units < 1 || max_rows < 0 || max_rows > (int64_t(1) << 40)) return 0;
  const int64_t per = max_rows == 0 ? 1 : (max_rows + kDecodeTileRows - 1) / kDecodeTileRows;
  if (per > ((int64_t(1) << 31) - 1) / units) return 0;
  int64_t n = units + kDecodeSlots / 2;
  if (n < kDecodeSlots) n = kDecodeSlots;
  const int64_t most = units * ((per + kDecodeMinPiece - 1) / kDecodeMinPiece);
  if (n > most) n = most;
  if (n < units + 1) n = units + 1;
  return n > INT32_MAX ? 0 : (int32_t)n;
}

struct DecodePlan {
  int32_t B, L, Hq, Hkv, d, G;
  int32_t units;     // L * B * Hkv
  int32_t max_rows;  // rows past this index are not attended
  int32_t nwg;       // workgroups of the launch (decode_grid)
  float sc;          // scale * log2(e)
  const uint16_t *k_pool, *v_pool;
  const int64_t *row_off;
  const int32_t *cap;
  const int32_t *len;
  const uint16_t *q;
  float *out;
  // Partial results of split units, one slot per piece (workgroup):
  // [nwg][16][d] and [nwg][16] (max, sum).
  float *part_o;
  float2 *part_ml;
  int2 *pinfo;       // [U] (first slot, pieces) of each unit (two-call path)
  // Fused step only: the row to append per unit ([U][d] each), the arrival
  // counters of the split units ([U], zero between calls) and the writable
  // views of pools and lengths.
  const uint16_t *k_new, *v_new;
  uint32_t *arrive;
  uint16_t *k_pool_w, *v_pool_w;
  int32_t *len_w;
  // 4-bit prefix (decode_step_q4 only): codes [rows][d/2], meta [rows][d/32]
  // (scale, lo) for keys and values, and per unit its first quantised row and
  // its quantised row count.
  const uint8_t *qk, *qv;
  const float2 *qkm, *qvm;
  const int64_t *qoff;
  const int32_t *nq;
  // Host-built piece table (decode_step_planned only): header, then one
  // record per workgroup.
  const int32_t *plan;
};

// Piece table of a planned decode step.  Header words: magic, units, nwg, d,
// max_rows, pieces, then zeros.  Record of workgroup i: unit u (-1: no
// piece), piece j and the unit's piece count np (j | np << 16; np <= 512),
// the unit's first piece's slot p0 (its partials use slot p0 + j), rows
// [r0, r1) of the unit's capacity, the bound rs <= r1 below which rows may be
// read before the unit's length is known, and the unit's first pool row (low
// word, high word).
constexpr int32_t kDecodePlanMagic = 0x50444356;  // "VCDP"
constexpr int kDecodePlanHdrWords = 8;
constexpr int kDecodePlanRecWords = 8;
// Host: bytes of the piece table of a launch of nwg workgroups.
inline size_t decode_plan_table_bytes(int64_t nwg) {
  return sizeof(int32_t) * (size_t)(kDecodePlanHdrWords + kDecodePlanRecWords * nwg);
}
// Host: builds the piece table of `units` caches with capacities cap[] and
// first pool rows row_off[] (host arrays) for a launch of nwg workgroups
// (decode_grid) at head dim d and row bound max_rows; len_hint[] (host, may
// be null) are the units' lengths when the table is built, which bound the
// rows read early.  Returns VC_OK or VC_ERR_ARG (a negative capacity, offset
// or length, overlapping blocks) or VC_ERR_UNSUPPORTED.
int decode_plan_build(int32_t units, const int32_t *cap, const int64_t *row_off, const int32_t *len_hint,
                      int64_t max_rows, int32_t nwg, int32_t d, int32_t *out);

// Scratch of the allocation-free decode step (viscache_decode_step_noalloc):
// a file-scope device array of kNoAllocBytes per device.  The arrival
// counters of at most kNoAllocUnits units sit at its front; the partial
// results of the pieces fill the rest.
constexpr size_t kNoAllocBytes = size_t(16) << 20;
constexpr int32_t kNoAllocUnits = 65536;
constexpr size_t kNoAllocCounterBytes = sizeof(uint32_t) * (size_t)kNoAllocUnits;
// The current device's scratch (device address); the first call on a device
// also enqueues, on `st`, the clear of the counters.
hipError_t noalloc_scratch(uint8_t **out, hipStream_t st);

hipError_t launch_append(int32_t units, int32_t d, uint16_t *k_pool, uint16_t *v_pool,
                         const int64_t *row_off, const int32_t *cap, int32_t *len,
                         const uint16_t *k_new, const uint16_t *v_new, hipStream_t st);
hipError_t launch_decode(const DecodePlan &p, hipStream_t st);
hipError_t launch_decode_step(const DecodePlan &p, hipStream_t st);
hipError_t launch_decode_step_q4(const DecodePlan &p, hipStream_t st);
hipError_t launch_decode_planned(const DecodePlan &p, bool q4, hipStream_t st);
// 4-bit rows: `rows` bf16 rows of d values -> codes [rows][d/2], meta [rows][d/32].
hipError_t launch_quant_rows(int32_t d, int64_t rows, const uint16_t *src, uint8_t *codes, float2 *meta,
                             hipStream_t st);

}  // namespace vc
