/*
 * wnw.h - C ABI of the WnW per-token decode step on one MI355X (gfx950).
 *
 * WnW (Waxing-and-Waning KV cache, arXiv 2608.22704) splits the KV-heads of a speech LLM into
 * three roles (Method, "Three-Way Classification"):
 *   anchor - keeps all of its audio KV on the GPU; its decode-time attention is the signal;
 *   tidal  - keeps a per-segment prefill subset on the GPU and its complement in host memory,
 *            from which chunks are recalled on demand;
 *   fixed  - keeps the prefill subset only.
 * Text (non-audio) KV is always kept in full (the remark under the retention equation, Eq. 1).
 *
 * One decode step (Method, "Decode-Step Score Aggregation", Eq. 2, and "Dynamic Chunk
 * Selection") does, for every sequence of the batch:
 *   1. attention of every anchor head over its full audio + text KV, which also yields the
 *      softmax mass each anchor q-head puts on every audio chunk (Eq. 2, reset every step);
 *   2. chunk scores = the mean over the chunk's positions of the mass summed over all anchor
 *      (layer, q-head) pairs, and a top-k chunk selection;
 *   3. recall of the complement of newly resident chunks from pinned host memory into tidal-head
 *      slots; a chunk left unselected for delta consecutive steps is dropped from the GPU (its
 *      host copy persists);
 *   4. attention of tidal heads over kept rows + resident complements + text, and of fixed heads
 *      over kept rows + text.
 *
 * Layout conventions (all row-major, bf16 = 16-bit brain float):
 *   K/V cache  [B][L][H_kv][T_a + T_t][d]  audio rows first, then text rows
 *   q          [B][L][H_q][d]              q-head hq belongs to KV-head hq / (H_q / H_kv)
 *   out        [B][L][H_q][d]              fp32
 *   scores     [B][n_chunks]               fp32
 *   selected   [B][k]                      int32 chunk ids, ascending
 *   resident   [B][n_segments]             flags (wnw_debug_read_resident)
 *
 * Segments are runs of chunk_len audio positions (chunk_len / 2 with WNW_F_OVERLAP_CHUNKS); the
 * last one may be shorter.  By default a chunk is one segment.  k defaults to
 * floor(budget * T_a / chunk_len); each tidal/fixed head keeps floor(budget * len) positions of
 * every segment, chosen by the caller's prefill scores (Method, "Prefill Compression"); ties
 * prefer the lower position.  Chunk ranking breaks ties by the lower chunk id.  A chunk is
 * resident at step s iff it was selected at one of the last delta steps (s - delta + 1 .. s); a
 * segment is resident iff a resident chunk covers it.
 *
 * Errors: every call returns a wnw_status; no C++ exception crosses the ABI.  A failing HIP call
 * turns the context sticky: every later call on it returns WNW_ERR_STATE.  wnw_last_error gives
 * the message (per context, or per thread when ctx is NULL).
 *
 * Threading: a context is not thread-safe.  Calls on one GPU that share a context must be
 * serialised by the caller.
 *
 * Environment: WNW_LOG=1 prints one trace line per decode step on stderr (what the call
 * enqueued; with WNW_F_RECALL_MEMCPY the segments it copied and the host's wait).
 * WNW_TEST_PINNED_LIMIT=<bytes> makes pinned allocations above that size fail with WNW_ERR_OOM
 * (a test hook for the failure path of wnw_set_roles).
 */
#ifndef WNW_H
#define WNW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    WNW_OK = 0,
    WNW_ERR_INVALID = -1,      /* bad argument or configuration                               */
    WNW_ERR_OOM = -2,          /* device or pinned host allocation failed                     */
    WNW_ERR_HIP = -3,          /* a HIP runtime call failed (context is now sticky)           */
    WNW_ERR_STATE = -4,        /* call out of order, or context in the sticky error state     */
    WNW_ERR_UNSUPPORTED = -5   /* configuration outside what this library implements         */
} wnw_status;

typedef enum { WNW_ANCHOR = 0, WNW_TIDAL = 1, WNW_FIXED = 2 } wnw_role;

enum {
    /* Tidal heads of step s attend over the resident set left by step s-1 (the paper's timing,
     * Method, "Dynamic Chunk Selection": the selection made after a step serves the next one);
     * default is the same step.  The chunks that become resident at step s are recalled on a
     * side stream, overlapped with the rest of step s and the anchor attention of step s+1;
     * a dropped chunk keeps its slot one step longer.  With both timings n_slots =
     * (delta + 1) * k (per segment: times the chunk's segments): the slots beyond the resident
     * set keep recently dropped complements, which are revived without a copy. */
    WNW_F_SELECT_NEXT_STEP = 1u,
    /* Recall with copy-engine transfers (hipMemcpyAsync from the pinned complement, spread over
     * four internal streams) that the host issues as soon as the step's selection has run: with
     * same-step timing the call polls for that point, so it returns only after the selection;
     * with WNW_F_SELECT_NEXT_STEP a library thread polls and issues them, and the call returns
     * once its own work is enqueued (see wnw_decode_step).  Without this flag
     * work-groups read the complements from mapped pinned memory (same-step timing: in the
     * tidal/fixed launch, which also attends to them; next-step timing: a copy kernel on a side
     * stream) and the call never waits.  The transfers occupy no compute units: with next-step
     * timing they disturb the attention launch beside them far less than work-groups holding
     * host reads, and they keep the link as busy. */
    WNW_F_RECALL_MEMCPY = 2u,
    /* Record HIP events around the kernels of every step; wnw_get_stats reports the times. */
    WNW_F_TIMING = 4u,
    /* The paper's chunk structure (Method, "Chunk Structure"): a chunk is two consecutive
     * segments of chunk_len / 2 positions and a chunk starts at every segment (stride one
     * segment), so there is one chunk fewer than segments.  Selection and eviction streaks are
     * per chunk; keep sets, masses, residency, slots and recall are per segment (a resident
     * chunk makes both its segments resident).  chunk_len must be even.  Default: disjoint
     * chunks of chunk_len positions, each its own segment. */
    WNW_F_OVERLAP_CHUNKS = 8u,
    /* Prefill compression without the per-segment quota: a head keeps the same number of audio
     * positions (the sum of its per-segment counts), the best over its whole audio; a segment
     * may then be kept whole or not at all, and complements differ in size from segment to
     * segment.  Default: per segment. */
    WNW_F_PREFILL_GLOBAL = 16u,
    /* wnw_decode_step writes out_dev as bf16 (each fp32 result rounded to nearest, ties to
     * even) instead of fp32; the arithmetic is unchanged. */
    WNW_F_OUT_BF16 = 32u
};

typedef struct wnw_ctx wnw_ctx;

typedef struct {
    int32_t batch;        /* B >= 1                                                  */
    int32_t layers;       /* L >= 1                                                  */
    int32_t q_heads;      /* H_q, a multiple of kv_heads; H_q / H_kv in {1,2,3,4,6,8} */
    int32_t kv_heads;     /* H_kv >= 1                                               */
    int32_t head_dim;     /* d; must be 128                                          */
    int32_t audio_len;    /* T_a >= 0 audio positions (same for every sequence)      */
    int32_t text_len;     /* T_t >= 0 text positions                                 */
    int32_t chunk_len;    /* 1 .. 256 audio positions per chunk                      */
    int32_t budget_bp;    /* on-GPU audio retention in basis points, 0 .. 10000      */
    int32_t top_k;        /* chunks selected per step; 0 = budget-derived            */
    int32_t evict_lag;    /* delta >= 1; 0 = 3                                       */
    uint32_t flags;       /* WNW_F_* bits                                            */
    int32_t max_new_tokens; /* generated tokens wnw_append_kv may add, >= 0 (device rows
                               are reserved for them in every head at set-up)           */
} wnw_config;

typedef struct {
    int64_t steps;             /* decode steps run                                       */
    int64_t recalled_chunks;   /* (sequence, chunk) complements copied host -> device    */
    int64_t revived_chunks;    /* newly resident complements whose bytes were still in a
                                  freed slot, so no copy was needed                        */
    int64_t recalled_bytes;    /* bytes copied host -> device                            */
    int64_t dropped_chunks;    /* (sequence, chunk) complements dropped from the device  */
    int64_t resident_chunks;   /* sum over steps and sequences of resident chunks        */
    int32_t peak_resident;     /* largest resident set of one sequence                   */
    int32_t n_slots;           /* recall slots per sequence                              */
    double r_gpu;              /* paper's r_GPU: device-resident audio KV / full audio KV,
                                  with the mean resident set over the steps run           */
    double r_gpu_cpu;          /* paper's r_GPU+CPU: adds the host-resident complement   */
    int64_t anchor_bytes;      /* algorithmic HBM bytes of one anchor-attention launch   */
    int64_t static_bytes;      /* algorithmic HBM bytes of the fixed heads + tidal kept rows    */
    int64_t slot_rows;         /* complement rows attended, summed over steps, sequences
                                  and tidal heads                                         */
    /* WNW_F_TIMING only: summed times (ms) between HIP events recorded on the caller's stream
     * around the step's launches, and the number of timed steps. */
    int64_t timed_steps;
    double t_anchor_ms;        /* the first launch: anchor attention + chunk mass (with
                                  WNW_F_SELECT_NEXT_STEP also the fixed heads and the tidal kept
                                  rows)                                                         */
    double t_select_ms;        /* anchor merge, chunk scores, top-k, residency, slots (up to the
                                  end of the select kernel).  Near zero in steps that run them
                                  inside the tidal/fixed launch (WNW_F_SELECT_NEXT_STEP with
                                  WNW_F_RECALL_MEMCPY, after a previous-step recall of at most
                                  4 MiB): t_tidal_fixed_ms holds them then                      */
    double t_tidal_fixed_ms;   /* the tidal/fixed launch after the selection.  Same-step timing:
                                  fixed heads, tidal kept rows, complements already on the
                                  device (default recall: also the recall and the attention over
                                  the recalled complements).  WNW_F_SELECT_NEXT_STEP: every
                                  resident complement (after the wait for the previous step's
                                  recall)                                                       */
    double t_new_ms;           /* WNW_F_RECALL_MEMCPY with same-step timing: attention over the
                                  complements copied this step                                  */
    double t_combine_ms;       /* merge of the tidal/fixed partial results                      */
    double t_step_ms;          /* whole step on the caller's stream                             */
    double t_recall_ms;        /* the recall: the launch that carries it (same-step timing), the
                                  copy kernel on the side stream (next-step timing) or the
                                  host-issued copies (WNW_F_RECALL_MEMCPY: from the first copy
                                  stream's start to the last copy's end, less the part spent
                                  behind the previous step's copies)                            */
    int64_t slot_exhausted;    /* steps that found no free recall slot; never expected (the
                                  slot count bounds the resident set).  When it happens the
                                  context fails: wnw_get_stats and the next wnw_decode_step
                                  return WNW_ERR_STATE with a message                            */
    double t_host_wait_ms;     /* WNW_F_RECALL_MEMCPY: host time spent polling for the step's
                                  selection before issuing the copies, summed over steps         */
    double t_recall_wait_ms;   /* WNW_F_TIMING: on the caller's stream, from the end of the
                                  select kernel (of the first launch when the selection runs
                                  inside the tidal/fixed launch) to the start of the tidal/fixed
                                  launch: with WNW_F_SELECT_NEXT_STEP the wait for the previous
                                  step's recall                                                  */
    int64_t kept_rows;         /* complement rows of the kept lists (segments whose bytes were
                                  on the device before the step's recall), summed over steps,
                                  sequences and tidal heads; the rest of slot_rows were recalled
                                  by the step before (WNW_F_SELECT_NEXT_STEP) or the step itself */
    int64_t selections_in_tidal; /* steps whose anchor mass merge and selection ran inside the
                                  tidal/fixed launch (WNW_F_SELECT_NEXT_STEP with
                                  WNW_F_RECALL_MEMCPY, after a previous-step recall of at most
                                  4 MiB); the other steps ran the two kernels before it         */
} wnw_stats;

/* Create a context for one batch of caches: the full KV cache as prefill leaves it, before any
 * compression (the starting point of Method, "Prefill Compression and Decode-Time Chunk Swap").
 *   cfg        copied; validated here (WNW_ERR_INVALID / WNW_ERR_UNSUPPORTED).
 *   k_dev/v_dev  device bf16 [B][L][H_kv][T_a+T_t][d], owned by the caller, read only by
 *              wnw_set_roles; they may be freed once it has returned.
 *   hip_stream stream for the set-up work (NULL = the null stream).
 *   out        receives the context; NULL on failure.
 * Allocates nothing until wnw_set_roles. */
wnw_status wnw_init_cache(const wnw_config *cfg, const void *k_dev, const void *v_dev,
                          void *hip_stream, wnw_ctx **out);

/* Per-head audio retention of Eq. 1 (Method, "Three-Way Classification"): every tidal and
 * fixed head keeps the fraction retention = min(importance * lambda, 1) of the audio positions
 * of each segment (taken in double: floor(retention * len)); anchors keep everything and text
 * is always kept.  Without this call the retention is budget_bp / 10000 for every head.
 *   importance  host fp32 [L][H_kv], each in [0, 1] (entries of anchor heads are ignored);
 *               copied.  NULL restores the uniform budget.
 *   lambda      finite, >= 0.
 * Only before wnw_set_roles (WNW_ERR_STATE after it); WNW_ERR_INVALID for values outside
 * those ranges.  k still comes from top_k or budget_bp. */
wnw_status wnw_set_retention(wnw_ctx *ctx, const float *importance, float lambda);

/* Assign roles and run prefill compression (Method, "Prefill Compression"): every tidal and
 * fixed head keeps floor(retention * len) positions of each segment with the highest prefill
 * score.
 *   roles           host uint8 [L][H_kv] of wnw_role, shared by the batch.
 *   prefill_scores  host fp32 [B][L][H_kv][T_a]; entries of anchor heads are ignored.
 * Builds the device tiers (anchor rows, kept rows, recall slots) and the pinned host
 * complement, then waits for the copies.  Exactly once per context, after wnw_init_cache. */
wnw_status wnw_set_roles(wnw_ctx *ctx, const uint8_t *roles, const float *prefill_scores);

/* Prefill scores of Prefill Compression, on the device: p [B][L][H_kv][T_a] fp32, for every
 * KV-head, the softmax weight that the text tokens put on each audio position, summed over the
 * text tokens and over the g q-heads of the KV-head.  Text token t (cache row T_a + t) attends
 * to every audio row and to text rows 0..t; logit scale 1 / sqrt(d); bf16 products summed in
 * fp32.
 *   q_text_dev  device bf16 [B][L][H_q][T_t][d]: the text tokens' queries at prefill (may be
 *               NULL when T_t = 0, then p = 0)
 *   scores_dev  device fp32 [B][L][H_kv][T_a], written
 * Reads the full cache given to wnw_init_cache, so only before wnw_set_roles / _device
 * (WNW_ERR_STATE after).  Runs on the stream given to wnw_init_cache and waits for it; uses a
 * temporary device buffer of B * L * H_q * T_t * 4 bytes. */
wnw_status wnw_prefill_scores(wnw_ctx *ctx, const void *q_text_dev, float *scores_dev);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc): wnw_prefill_scores without its temporary buffer.  The same
 * kernels compute the same scores (bit for bit); their per-row statistics go to a fixed device
 * array of the library (32 MiB, one per GPU, held until the process ends) instead of a
 * temporary allocation, and the call only enqueues work on hip_stream (NULL = null stream) and
 * returns: scores_dev is valid once that stream has completed.  Calls whose work overlaps on
 * one GPU (any context, any stream) share that array and race: the caller orders them.
 *   q_text_dev, scores_dev  as wnw_prefill_scores.
 * WNW_ERR_UNSUPPORTED when batch * layers * q_heads * text_len exceeds 8 388 608 rows (use
 * wnw_prefill_scores); WNW_ERR_STATE after wnw_set_roles.  Allocates nothing (no hipMalloc,
 * hipFree or allocating library call). */
wnw_status wnw_prefill_scores_static(wnw_ctx *ctx, const void *q_text_dev, float *scores_dev, void *hip_stream);

/* As wnw_set_roles, with the prefill scores in device memory (e.g. from wnw_prefill_scores):
 * the per-segment ranking (same rule and ties) runs on the device and the tiers are built from
 * its keep flags.  The same scores give the same tiers as wnw_set_roles.  On failure (or a
 * failure of wnw_set_roles) the context is in the error state and can only be destroyed. */
wnw_status wnw_set_roles_device(wnw_ctx *ctx, const uint8_t *roles, const float *prefill_scores_dev);

/* Decode-time append: the K and V rows of the token generated at this step join the key set of
 * every head from the next wnw_decode_step on, after the text rows; a generated token is not
 * audio, so every role keeps it in full (the remark under Eq. 1).
 *   k_new_dev, v_new_dev  device bf16 [B][L][H_kv][d]; read by a kernel enqueued on hip_stream
 *                         (valid until it has run).
 * Call it before the wnw_decode_step of the token it belongs to, on the same stream.
 * WNW_ERR_STATE before wnw_set_roles or once max_new_tokens rows have been appended. */
wnw_status wnw_append_kv(wnw_ctx *ctx, const void *k_new_dev, const void *v_new_dev, void *hip_stream);

/* One decode step (Eq. 2 and "Dynamic Chunk Selection"), enqueued on hip_stream (with
 * WNW_F_SELECT_NEXT_STEP or WNW_F_RECALL_MEMCPY the recall runs on internal streams, joined by
 * events; with both, a library thread issues each step's copies once its selection is done).
 *   q_dev             device bf16 [B][L][H_q][d]
 *   out_dev           device fp32 [B][L][H_q][d]     attention output of every q-head
 *                     (bf16, same layout, with WNW_F_OUT_BF16)
 *   chunk_scores_dev  device fp32 [B][n_chunks]      this step's chunk scores
 *   selected_dev      device int32 [B][k]            selected chunk ids, ascending
 *   hip_stream        caller's stream (NULL = null stream); outputs are valid once it has
 *                     completed.  Buffers and the stream must stay valid until then.
 * The default recall path does not block the host.  With WNW_F_RECALL_MEMCPY and same-step
 * timing the call waits once, mid-step (busy polling), for the selection before issuing the
 * copies.  With WNW_F_RECALL_MEMCPY and WNW_F_SELECT_NEXT_STEP the call returns once its work is
 * enqueued; before enqueueing the launch that reads the previous step's recall it waits until
 * the library's recall thread has issued that recall (that is, until the previous step's
 * selection has run on the device), so the caller runs at most about one step ahead. */
wnw_status wnw_decode_step(wnw_ctx *ctx, const void *q_dev, void *out_dev,
                           float *chunk_scores_dev, int32_t *selected_dev, void *hip_stream);

/* Derived sizes (Method, "Chunk Structure" and "Dynamic Chunk Selection"; k as the budget
 * gives it, see the file header): chunks (the selection's candidates), k, kept audio rows per tidal/fixed head
 * (-1 after wnw_set_retention: see wnw_query_head_keep), recall slots per sequence, and bytes of
 * one recalled segment of one sequence (all tidal heads; a segment is a chunk unless
 * WNW_F_OVERLAP_CHUNKS; known after wnw_set_roles).  Any pointer may be NULL. */
wnw_status wnw_query_geometry(const wnw_ctx *ctx, int32_t *n_chunks, int32_t *k,
                              int32_t *keep_total, int32_t *n_slots, int64_t *chunk_bytes);

/* Number of segments (Method, "Chunk Structure"; the unit of residency and recall; equal to n_chunks unless
 * WNW_F_OVERLAP_CHUNKS, then n_chunks + 1).  The pointer may be NULL. */
wnw_status wnw_query_segments(const wnw_ctx *ctx, int32_t *n_segments);

/* Kept audio rows of every head (Method, "Prefill Compression"; Eq. 1 with per-head retention),
 * host int32 [L][H_kv] (T_a for anchors).  After wnw_set_roles. */
wnw_status wnw_query_head_keep(const wnw_ctx *ctx, int32_t *keep);

/* Counters and (with WNW_F_TIMING) kernel times; waits for the device.  r_gpu and r_gpu_cpu are
 * the paper's audio KV retention ratios (Experiments, "Audio KV Retention and WnW Configuration");
 * recalled_bytes is the CPU-to-GPU volume of the runtime table (Experiments, "Efficiency and
 * Runtime Analysis"); the other fields are instrumentation with no passage behind them.
 * WNW_ERR_STATE (context failed) if a step ran out of recall slots. */
wnw_status wnw_get_stats(wnw_ctx *ctx, wnw_stats *out);

/* Test and benchmark support, no passage behind it.
 * Replace the top-k of the following steps by the ids in sel_dev (device int32 [B][k], read
 * when each step runs; -1 = no chunk; ids distinct, < n_chunks).  NULL restores the top-k.
 * Scores are still computed.  Used to keep two implementations on one trajectory and to force
 * a recall load. */
wnw_status wnw_set_selection_override(wnw_ctx *ctx, const int32_t *sel_dev);

/* Test support (the byte identity of a recalled chunk with its host copy), no passage behind it.
 * Copy the device slot holding the recalled complement of (b, segment) to host_dst (waits for
 * the device).  Valid for segments resident after the last step (with WNW_F_SELECT_NEXT_STEP,
 * also those recalled during it).  Layout: per tidal head in role order (roles scanned in
 * [L][H_kv] order), its complement K rows then V rows, c rows each, where c is that head's
 * complement of a full segment (zero rows pad a shorter last segment); bf16 [..][d]; `bytes` must
 * equal chunk_bytes.  WNW_ERR_INVALID if that segment is not resident. */
wnw_status wnw_debug_read_slot(wnw_ctx *ctx, int32_t b, int32_t chunk, void *host_dst, size_t bytes);

/* Test support, no passage behind it.
 * Copy the host (pinned) complement of (b, segment) in the same layout as wnw_debug_read_slot. */
wnw_status wnw_debug_read_host_chunk(wnw_ctx *ctx, int32_t b, int32_t chunk, void *host_dst, size_t bytes);

/* Test support, no passage behind it (the resident set is the one "Dynamic Chunk Selection"
 * defines).  Flags [B][n_segments] (uint8) of the segment complements the last step's tidal heads
 * attended: the resident set of that step, or of the step before it with
 * WNW_F_SELECT_NEXT_STEP (waits for the device). */
wnw_status wnw_debug_read_resident(wnw_ctx *ctx, uint8_t *host_dst);

/* Test support, no passage behind it (the stream ordering of the recall, which the paper leaves
 * to future work).  From the next recall on, every recall is delayed by `us` microseconds: the
 * host waits that long before issuing host-issued copies, and a host function sleeping as long is
 * queued ahead of the copies on each copy stream (ahead of the copy kernel on the side stream
 * without WNW_F_RECALL_MEMCPY).  Results must not change: every reader of a recalled slot waits
 * for the recall.  0 = no delay (default); WNW_ERR_INVALID outside 0..1000000. */
wnw_status wnw_debug_set_recall_delay(wnw_ctx *ctx, int32_t us);

/* Test support, no passage behind it.
 * Slot groups of a sequence whose slot region (n_slots * chunk_bytes) has `bytes` or more read
 * their rows through per-row pointers instead of 32-bit buffer offsets.  The default,
 * 4294967295, is the largest region buffer offsets can address; 0 forces the pointer path
 * everywhere.  Both paths compute the same results.  Takes effect from the next step;
 * WNW_ERR_INVALID for a negative value. */
wnw_status wnw_debug_set_slot_offset_limit(wnw_ctx *ctx, int64_t bytes);

/* Error reporting, no passage behind it.
 * Message of the last failure on ctx (or of this thread when ctx is NULL).  Never NULL. */
const char *wnw_last_error(const wnw_ctx *ctx);

/* Resource management, no passage behind it.
 * Free every device, pinned and stream resource of ctx (waits for its work).  NULL is a no-op. */
void wnw_destroy(wnw_ctx *ctx);

/* ---- head triage arithmetic (Method, "Head Functional Triage via Offline Calibration"; the
 * calibration score details of the appendix).  These calls need no context: they turn the
 * calibration inputs (answer-token queries and a sample's keys, aligned audio intervals, key
 * gradients) into the roles and normalised importance that wnw_set_roles / wnw_set_retention
 * take.  Producing those inputs (model, forced alignment, autograd) is outside the library.
 * Errors: WNW_ERR_INVALID / _UNSUPPORTED / _HIP, message from wnw_triage_last_error(). */

/* Voice-score hits.  For every answer token t and q-head (l, h): the top_k audio positions with
 * the largest logit q . k (the softmax keeps that order; ties to the lower position), and how
 * many lie in [span[t][0], span[t][1]).  Logits are exact bf16 products summed in double.
 *   k_dev     device bf16 [L][H_kv][rows][d] of one calibration sample, audio rows first
 *   q_dev     device bf16 [n_tok][L][H_q][d], the answer tokens' queries
 *   span_dev  device int32 [n_tok][2], audio-token interval [a, b) of each answer token
 *   hits_dev  device int32 [n_tok][L][H_q], written (0..top_k)
 * top_k in 1..8 and <= audio_len; d = 128.  Enqueued on hip_stream. */
wnw_status wnw_voice_hits(int32_t layers, int32_t q_heads, int32_t kv_heads, int32_t rows, int32_t audio_len,
                          int32_t n_tok, const void *k_dev, const void *q_dev, const int32_t *span_dev, int32_t top_k,
                          int32_t *hits_dev, void *hip_stream);

/* Key sensitivity.  sens[t][l][kv] = mean over the audio positions of the L2 norm of the loss
 * gradient at that position's key.
 *   grad_dev  device fp32 [n_tok][L][H_kv][audio_len][d]
 *   sens_dev  device fp32 [n_tok][L][H_kv], written
 * Enqueued on hip_stream. */
wnw_status wnw_key_sensitivity(int32_t layers, int32_t kv_heads, int32_t audio_len, int32_t n_tok, const float *grad_dev,
                               float *sens_dev, void *hip_stream);

/* Three-way classification (host).  Rows i = 0..n-1 are answer tokens of calibration samples
 * sample[i] >= 0.  VS = per-sample mean of hits / top_k, averaged over the samples, then over the
 * group q-heads of each KV-head; HS = per-sample mean of sens averaged over the samples.  Heads
 * are ranked by VS * HS (ties to the lower index l * H_kv + kv): the first n_anchor are anchors,
 * the next ones up to n_voice tidal, the rest fixed.  importance = VS * HS / its maximum (all 0
 * when the maximum is 0), the normalised importance of the retention equation (Eq. 1).
 *   hits [n][L][H_kv * group], sens [n][L][H_kv]; outputs [L][H_kv]: roles (wnw_role),
 *   importance; vs_out, hs_out (may be NULL). */
wnw_status wnw_triage(int32_t layers, int32_t kv_heads, int32_t group, int32_t n, const int32_t *sample,
                      const int32_t *hits, int32_t top_k, const float *sens, int32_t n_voice, int32_t n_anchor,
                      uint8_t *roles, float *importance, double *vs_out, double *hs_out);

/* Error reporting, no passage behind it.  Message of the last failed triage call of this thread. */
const char *wnw_triage_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* WNW_H */
