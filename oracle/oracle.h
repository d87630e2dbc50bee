/*
 * oracle.h -- CPU oracle for PruneKV (VisCache, "PruneKV: Layer-Aware Visual KV
 * Cache Compression", Sec. 3.2 and Appendix B, Algorithm 1).
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, single-threaded C
 * implementation in double precision, used to check the GPU library.  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load it;
 * the product path never calls it, and it shares no source with the GPU path.
 *
 * bf16 values are passed as uint16 bit patterns.  All functions are reentrant
 * (no global state) so callers may run independent units on several threads.
 */
#ifndef PRUNEKV_ORACLE_H
#define PRUNEKV_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Layer budgets: Eq. (parabolic) with the normalisation to sum h*m that
 * follows it, the retention-ratio composition RR = p*q*(h/L)*m of the
 * implementation details (p = 1), and Alg. 1 Step 1 (the top-q cut).
 * Inputs: L layers, n visual tokens, overall retention rr in (0,1], h_param
 * (0 selects round(0.75 L)), mean budget m in (0,1], schedule (0 parabola,
 * 1 fixed, 2 arithmetic, 3 geometric: the budget ablation's alternatives to
 * Eq. (parabolic)), drop_all (1: every token survives, so every non-kept
 * token is fused).
 * Outputs: k[L] kept tokens per layer (0 beyond h), *n_surv (tokens that
 * survive the top-q cut), *h_out, b_out[L] (normalised proportions, may be
 * NULL), *q_out (may be NULL).  Returns 0, or -1 on invalid parameters. */
int orc_budget(int32_t L, int32_t n, double rr, int32_t h_param, double m, int32_t schedule, int32_t drop_all,
               int32_t *k, int32_t *n_surv, int32_t *h_out, double *b_out, double *q_out);

/* Window score of one (sequence, layer, kv head) unit, Eq. (token_score) read
 * as: for every query row r of the G*W window rows, the softmax over the n
 * visual keys of (bf16(q_r) . k_v) / sqrt(d); S[v] = sum over rows.
 * K: bf16 [n][d]; Q: fp32 [G*W][d] (rounded to bf16 first).  S: fp64 [n]. */
void orc_scores_unit(int32_t n, int32_t d, int32_t rows, const uint16_t *K, const float *Q,
                     double *S);

/* Prefill score of one (sequence, layer, kv head) unit, Eq. (token_score)
 * with every token of the prefill as a query (N = n + T, the sum over
 * i = 1..N): the sequence is the n visual tokens followed by the T text tokens
 * (H = concat[H_v, H_q]); query i of each of the G query heads of the group
 * attends keys 0..i (causal self-attention), visual keys K[j] for j < n and
 * text keys Kt[j - n]; A_{i,j} = softmax over those keys of
 * (bf16(q_i) . k_j) / sqrt(d).  S[v] = sum over heads and queries of A_{i,v}
 * for the visual keys; St[t] (may be NULL) the same for the text keys, so
 * that sum(S) + sum(St) = G*N.
 * K: bf16 [n][d]; Kt: bf16 [T][d]; Q: fp32 [G][N][d] (rounded to bf16 first).
 * S: fp64 [n]; St: fp64 [T]. */
void orc_scores_unit_prefill(int32_t n, int32_t T, int32_t d, int32_t G, const uint16_t *K,
                             const uint16_t *Kt, const float *Q, double *S, double *St);

/* Keep / drop partition (Alg. 1 Step 1 and Step 3): order tokens by
 * (score descending, index ascending); kept = the first k, drop = the next
 * n_surv - k; the rest are discarded.  Both lists are written ascending. */
void orc_select(int32_t n, const float *score, int32_t k, int32_t n_surv,
                int32_t *kept, int32_t *drop);

/* Key pruning: K_out[j] = K[kept[j]] (bit copy of d bf16 values). */
void orc_gather(int32_t d, int32_t k, const int32_t *kept, const uint16_t *K, uint16_t *K_out);

/* Value fusion, Eq. (redistribution) and Eq. (weight_fusion):
 * Phi = row-softmax(V_k V_d^T / tau); V_new = mu V_k + (1 - mu) Phi V_d.
 * V: bf16 [n][d] rows of the unit; kept[k], drop[r] index it.
 * With k == 0 nothing is written; with r == 0, V_new = V_k.
 * out: fp64 [k][d]. */
void orc_fuse(int32_t d, int32_t k, int32_t r, const uint16_t *V, const int32_t *kept,
              const int32_t *drop, double tau, double mu, double *out);

/* Decode attention of one query over one cache (Sec. 2, decoding):
 * out = sum_t softmax_t(scale * q . K_t) V_t.  q: bf16 [d]; K, V: bf16 [rows][d];
 * out: fp64 [d]. */
void orc_attend(int32_t d, int32_t rows, const uint16_t *q, const uint16_t *K, const uint16_t *V,
                double scale, double *out);

/* 4-bit cache rows (the combination with 4-bit KV-cache quantisation of the
 * quantisation experiments; the paper names the quantisers but does not define
 * them, so this is a reading): every row of a bf16 [n][d] block is split into
 * d/32 groups of 32 consecutive channels; group g of row r keeps
 *   lo = min, hi = max of its 32 values (fp32),
 *   scale = fp32(hi - lo) / 15            (fp32, IEEE rounding),
 *   code_c = clamp(rint(fp32(x_c - lo) / scale), 0, 15), 0 when scale = 0,
 * and the row's value is read back as bf16(fma(code_c, scale, lo)).  Every
 * step is fp32 arithmetic, so the integer codes are fixed bit for bit.
 * codes: [n][d/2] bytes, channel 2j in the low nibble of byte j, 2j+1 in the
 * high nibble; meta: [n][d/32][2] fp32 (scale, lo).  d must be a multiple of 32. */
void orc_quant_rows(int32_t n, int32_t d, const uint16_t *x, uint8_t *codes, float *meta);
void orc_dequant_rows(int32_t n, int32_t d, const uint8_t *codes, const float *meta, uint16_t *out);

/* One LAYER_HEAD unit end to end: score -> select -> gather -> fuse.
 * S32 (may be NULL) receives the fp32 scores used for the ranking. */
void orc_prune_unit(int32_t n, int32_t d, int32_t rows, const uint16_t *K, const uint16_t *V,
                    const float *Q, int32_t k, int32_t n_surv, double tau, double mu,
                    int32_t *kept, int32_t *drop, uint16_t *K_out, double *V_out, float *S32);

#ifdef __cplusplus
}
#endif
#endif
