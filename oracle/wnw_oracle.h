/*
 * WnW decode-step oracle: plain CPU reference, TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the package smoke check and the benchmark's CPU-baseline leg call this
 * code.  It shares nothing with the HIP library: not this header, not a helper, not a table.
 *
 * Paper: "WnW: Waxing-and-Waning KV Cache for Long-Form Speech LLMs" (arXiv 2608.22704),
 * Method section (head triage, retention equation, prefill compression, Eq. 2 decode-step
 * score aggregation, dynamic chunk selection).
 *
 * Arrays are row-major.  bf16 values are uint16 bit patterns.  Every function returns 0 on
 * success and a negative number on invalid arguments.
 */
#ifndef WNW_ORACLE_H
#define WNW_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t batch, layers, q_heads, kv_heads, head_dim;
    int32_t audio_len, text_len;   /* T_a audio rows first, then T_t text rows            */
    int32_t chunk_len;             /* audio positions per chunk                            */
    int32_t budget_bp;             /* on-GPU audio retention in basis points               */
    int32_t top_k;                 /* 0: floor(budget_bp * T_a / (10000 * chunk_len))      */
    int32_t evict_lag;             /* delta; 0 means 3                                     */
    int32_t next_step;             /* 1: tidal heads use the previous step's resident set  */
    int32_t chunk_span;            /* segments per chunk: 0 or 1 disjoint chunks (one segment
                                      each); 2 the paper's chunks of two consecutive segments
                                      of chunk_len / 2 positions, one chunk per segment start  */
    int32_t prefill_global;        /* 1: prefill keeps the same number of positions, ranked over
                                      the whole audio of a head instead of per segment          */
    int32_t max_new;               /* tokens that wnwo_append may add (0: none; the oracle then
                                      references the caller's cache, else it keeps a copy)     */
} wnwo_config;

typedef struct wnwo wnwo;

/* Derived sizes: number of chunks (the selection's candidates), k, kept audio rows per
 * non-anchor head. */
int wnwo_geometry(const wnwo_config *cfg, int32_t *n_chunks, int32_t *k, int32_t *keep_total);

/* Number of segments (the unit of prefill keep sets, chunk mass and residency). */
int wnwo_segments(const wnwo_config *cfg, int32_t *n_segments);

/* k, v: [B][L][H_kv][T_a+T_t][d] bf16, referenced (not copied) for the oracle's lifetime.
 * roles: [L][H_kv] (0 anchor, 1 tidal, 2 fixed).  prefill: [B][L][H_kv][T_a] fp32. */
wnwo *wnwo_create(const wnwo_config *cfg, const uint16_t *k, const uint16_t *v,
                  const uint8_t *roles, const float *prefill);
/* As wnwo_create, with the per-head audio retention of Eq. 1: retention = min(importance *
 * lambda, 1) for every tidal and fixed head (importance [L][H_kv] fp32 in [0, 1], lambda >= 0
 * finite; anchors keep all audio).  importance NULL means the uniform budget. */
wnwo *wnwo_create_retention(const wnwo_config *cfg, const uint16_t *k, const uint16_t *v,
                            const uint8_t *roles, const float *prefill, const float *importance,
                            float lambda);
void wnwo_destroy(wnwo *o);

/* Audio positions kept at prefill by head (b, l, kv): mask[T_a] of 0/1 (all 1 for anchors). */
int wnwo_keep_mask(const wnwo *o, int32_t b, int32_t l, int32_t kv, uint8_t *mask);

/* Prefill scores of Prefill Compression: p [B][L][H_kv][T_a] (double) = the attention weight
 * that the text tokens put on each audio position, summed over the text tokens and over the
 * q-heads of the KV-head; text token t attends to every audio row and to text rows 0..t.
 *   k       [B][L][H_kv][T_a+T_t][d] bf16
 *   q_text  [B][L][H_q][T_t][d] bf16, the text tokens' queries at prefill */
int wnwo_prefill_scores(const wnwo_config *cfg, const uint16_t *k, const uint16_t *q_text, double *p);

/* Append the K and V rows [B][L][H_kv][d] bf16 of the token generated at this step: from the
 * next wnwo_step on they are part of every head's key set, after the text rows.  At most
 * max_new times. */
int wnwo_append(wnwo *o, const uint16_t *k_new, const uint16_t *v_new);

/* One decode step.
 *   q         [B][L][H_q][d] bf16
 *   forced    [B][k] chunk ids replacing this step's top-k (-1 = no chunk), or NULL
 *   head_mask [L][H_kv]: outputs of non-anchor heads are computed only where non-zero
 *             (NULL = all); anchor outputs are always computed
 *   out       [B][L][H_q][d]         attention outputs (rows of skipped heads are zeroed)
 *   scores    [B][n_chunks]          chunk scores (double)
 *   selected  [B][k]                 selected chunk ids, ascending (-1 pads a forced set)
 *   mass      [B][n_anchor*g][n_segments] or NULL: per anchor q-head segment mass
 *   resident  [B][n_segments] or NULL: 1 where the segment's complement was attended this step
 * With disjoint chunks a segment is a chunk.
 */
int wnwo_step(wnwo *o, const uint16_t *q, const int32_t *forced, const uint8_t *head_mask,
              double *out, double *scores, int32_t *selected, double *mass, uint8_t *resident);

/* Head triage arithmetic (Method, "Head Functional Triage via Offline Calibration"; the
 * calibration score details of the appendix), on given inputs (no model, alignment or autograd).
 *
 * Voice-score hits of answer token t and q-head (l, h): how many of the K audio positions with
 * the largest logit q.k / sqrt(d) (ties to the lower position) lie in [span[t][0], span[t][1]).
 *   k     [L][H_kv][T][d] bf16 of one calibration sample (audio rows first)
 *   q     [n_tok][L][H_q][d] bf16 answer-token queries;  span [n_tok][2] int32
 *   hits  [n_tok][L][H_q] int32 in 0..K */
int wnwo_voice_hits(int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int32_t T, int32_t Ta, int32_t n_tok,
                    const uint16_t *k, const uint16_t *q, const int32_t *span, int32_t K, int32_t *hits);

/* Key sensitivity: sens[t][l][kv] = mean over audio positions of the L2 norm of the loss
 * gradient grad [n_tok][L][H_kv][T_a][d] (fp32) at that position's key. */
int wnwo_key_sensitivity(int32_t L, int32_t Hkv, int32_t d, int32_t Ta, int32_t n_tok, const float *grad, double *sens);

/* Roles from n answer-token rows (sample[i] = calibration sample of row i): VS = mean over
 * samples of the per-sample mean of hits / K, then over the g q-heads of a KV-head; HS = mean
 * over samples of the per-sample mean of sens; VS * HS ranked descending (ties to the lower
 * head index): the first n_anchor heads are anchors, the next up to n_voice tidal, the rest
 * fixed; importance_norm = VS * HS / max (0 if the max is 0).  Outputs [L][H_kv]. */
int wnwo_triage(int32_t L, int32_t Hkv, int32_t g, int32_t n, const int32_t *sample, const int32_t *hits, int32_t K,
                const double *sens, int32_t n_voice, int32_t n_anchor, uint8_t *roles, double *vs, double *hs,
                double *importance_norm);

/* Top-k of n scores ordered by (score descending, id ascending); ids returned ascending. */
int wnwo_topk(const float *scores, int32_t n, int32_t k, int32_t *sel);

/* Tokens covered by a window of `seconds` at `rate` tokens per second: ceil(seconds * rate). */
int32_t wnwo_tokens_for_window(double seconds, double rate);

/* Threads used by the parallel loops from now on (n <= 0: unchanged); returns the count in use.
 * Timing only: every result is independent of it. */
int wnwo_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
