/*
 * WnW decode-step oracle: plain CPU reference, TEST INFRASTRUCTURE ONLY.
 *
 * Written from the Method section of "WnW: Waxing-and-Waning KV Cache for Long-Form Speech
 * LLMs" (arXiv 2608.22704).  It takes the method's steps in the paper's order, in the most
 * direct form, accumulating in double over the exact bf16 inputs:
 *
 *   1. Roles (Method, "Three-Way Classification"): anchor KV-heads keep all audio KV; tidal
 *      heads keep a prefill subset on the device and a recallable complement on the host; fixed
 *      heads keep the subset only.  Non-audio (text) KV is always kept in full (the remark under
 *      the retention equation, Eq. 1).
 *   2. Prefill compression (Method, "Prefill Compression"): inside each segment, keep the top
 *      floor(retention * segment length) audio positions by prefill score.
 *   3. Decode-step score aggregation (Eq. 2): A_tau is the sum, over every anchor (layer,
 *      q-head) pair, of that head's softmax weight at audio position tau; it is rebuilt from
 *      zero at every step.
 *   4. Dynamic chunk selection (Method, "Dynamic Chunk Selection"): a chunk's score is the mean
 *      of A over its positions; the top-k chunks are selected; for tidal heads the complement of
 *      a selected chunk becomes resident and is dropped after delta consecutive steps without
 *      selection.
 *   5. Attention of every head over what it holds: anchors over all rows, tidal heads over
 *      kept rows + resident complements + text, fixed heads over kept rows + text.
 *
 * Readings taken where the paper leaves a choice (all listed in the design notes):
 *   - by default chunks are disjoint runs of chunk_len audio positions, one segment per chunk;
 *     with chunk_span = 2 a chunk is two consecutive segments of chunk_len / 2 positions and a
 *     chunk starts at every segment (Method, "Chunk Structure"); the last segment may be
 *     shorter and a chunk's score is the mean over the positions it has; a selected chunk makes
 *     both of its segments resident;
 *   - retention is one uniform fraction budget_bp / 10000 for every tidal and fixed head, or,
 *     given per-head importance and lambda, min(importance * lambda, 1) per head (Eq. 1);
 *   - k = floor(budget_bp * T_a / (10000 * chunk_len)) unless given;
 *   - the softmax of Eq. 2 runs over the anchor head's whole key set (audio and text); only the
 *     audio weights enter A; the logit scale is 1 / sqrt(d);
 *   - ties: prefill ranking prefers the lower position, chunk ranking the lower chunk id; the
 *     ranking compares chunk scores rounded to fp32, the precision the scores are reported in;
 *   - residency: a chunk is resident at step s iff it was selected at one of the steps
 *     s - delta + 1 .. s, so a chunk selected once stays for delta steps;
 *   - by default the selection of step s already serves the tidal heads of step s; with
 *     next_step set they use the resident set left by step s - 1 (empty at the first step);
 *   - a head whose key set is empty outputs zeros.
 */
#include "wnw_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

struct wnwo {
    wnwo_config c;
    int32_t n_chunks, n_seg, span, k, keep_total, delta;
    int32_t n_gen, tcap;   /* tokens appended so far; rows per head in kc / vc          */
    const uint16_t *kc, *vc;
    uint16_t *kown, *vown; /* the oracle's copy of the cache when tokens may be appended */
    uint8_t *roles;        /* [L][Hkv]                                               */
    uint8_t *keep;         /* [B][L][Hkv][T_a] prefill keep flags of non-anchor heads */
    int32_t *streak;       /* [B][n_chunks] steps since last selection, capped at delta */
    uint8_t *res_prev;     /* [B][n_seg] resident segments after the previous step     */
};

static double bf16(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int32_t wnwo_tokens_for_window(double seconds, double rate)
{
    /* Method, "Chunk Structure": n = ceil(W * r_tok). */
    return (int32_t)ceil(seconds * rate);
}

/* Segments: runs of chunk_len / span audio positions, the last one possibly shorter. */
static int32_t span_of(const wnwo_config *c) { return c->chunk_span == 2 ? 2 : 1; }
static int32_t seg_len(const wnwo_config *c) { return c->chunk_len / span_of(c); }
static int32_t seg_count(const wnwo_config *c) { return (c->audio_len + seg_len(c) - 1) / seg_len(c); }
static int32_t seg_begin(const wnwo_config *c, int32_t j) { return j * seg_len(c); }
static int32_t seg_end(const wnwo_config *c, int32_t j)
{
    int32_t e = (j + 1) * seg_len(c);
    return e < c->audio_len ? e : c->audio_len;
}
/* Chunks: one per segment start; with span 2, chunk c = segments c and c + 1, so there is one
 * chunk fewer than segments (a single segment forms a chunk on its own). */
static int32_t chunk_count(const wnwo_config *c)
{
    int32_t ns = seg_count(c);
    return (span_of(c) == 2 && ns >= 2) ? ns - 1 : ns;
}
static int32_t chunk_last_seg(const wnwo_config *c, int32_t ch)
{
    int32_t last = ch + span_of(c) - 1, ns = seg_count(c);
    return last < ns ? last : ns - 1;
}

/* Positions kept at prefill inside a segment of `len` positions: floor(retention * len), with
 * the uniform retention budget_bp / 10000. */
static int32_t keep_count(const wnwo_config *c, int32_t len)
{
    return (int32_t)(((int64_t)c->budget_bp * len) / 10000);
}

/* Eq. 1: the audio retention of a non-anchor head is its normalised importance times lambda,
 * clipped at 1 (taken in double: the product of the two fp32 inputs is exact there).  Its keep
 * count in a segment of `len` positions is floor(retention * len).  Without per-head importance
 * the uniform budget applies. */
static int32_t keep_count_head(const wnwo_config *c, const float *importance, float lambda, size_t h, int32_t len)
{
    if (!importance) return keep_count(c, len);
    double r = (double)importance[h] * (double)lambda;
    if (r > 1.0) r = 1.0;
    return (int32_t)floor(r * (double)len);
}

int wnwo_geometry(const wnwo_config *c, int32_t *n_chunks, int32_t *k, int32_t *keep_total)
{
    if (!c || c->batch < 1 || c->layers < 1 || c->kv_heads < 1 || c->head_dim < 1 ||
        c->q_heads < c->kv_heads || c->q_heads % c->kv_heads || c->audio_len < 0 ||
        c->text_len < 0 || c->chunk_len < 1 || c->budget_bp < 0 || c->budget_bp > 10000 ||
        c->top_k < 0 || c->evict_lag < 0 || c->chunk_span < 0 || c->chunk_span > 2 || c->max_new < 0 ||
        (c->chunk_span == 2 && c->chunk_len % 2))
        return -1;
    int32_t nc = chunk_count(c), ns = seg_count(c);
    int32_t kk = c->top_k ? c->top_k
                          : (int32_t)(((int64_t)c->budget_bp * c->audio_len) / (10000LL * c->chunk_len));
    if (kk > nc) return -1;
    int32_t kt = 0;
    for (int32_t j = 0; j < ns; ++j) kt += keep_count(c, seg_end(c, j) - seg_begin(c, j));
    if (n_chunks) *n_chunks = nc;
    if (k) *k = kk;
    if (keep_total) *keep_total = kt;
    return 0;
}

int wnwo_segments(const wnwo_config *c, int32_t *n_segments)
{
    if (wnwo_geometry(c, NULL, NULL, NULL)) return -1;
    if (n_segments) *n_segments = seg_count(c);
    return 0;
}

/* ---- prefill compression: per-segment top floor(retention * len) by prefill score ---------- */

typedef struct { float s; int32_t pos; } ranked;

static int by_score_then_pos(const void *a, const void *b)
{
    const ranked *x = a, *y = b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

static void prefill_keep(const wnwo_config *c, const float *importance, float lambda, size_t h,
                         const float *score, uint8_t *keep, ranked *tmp)
{
    memset(keep, 0, (size_t)c->audio_len);
    int32_t ns = seg_count(c);
    if (c->prefill_global) {
        /* Global variant (ablation of per-segment selection): the same number of positions,
         * the sum of the per-segment counts, ranked over the whole audio of the head. */
        int32_t total = 0;
        for (int32_t j = 0; j < ns; ++j) total += keep_count_head(c, importance, lambda, h, seg_end(c, j) - seg_begin(c, j));
        for (int32_t i = 0; i < c->audio_len; ++i) { tmp[i].s = score[i]; tmp[i].pos = i; }
        qsort(tmp, (size_t)c->audio_len, sizeof *tmp, by_score_then_pos);
        for (int32_t i = 0; i < total; ++i) keep[tmp[i].pos] = 1;
        return;
    }
    for (int32_t j = 0; j < ns; ++j) {
        int32_t b0 = seg_begin(c, j), e0 = seg_end(c, j), n = e0 - b0;
        for (int32_t i = 0; i < n; ++i) { tmp[i].s = score[b0 + i]; tmp[i].pos = b0 + i; }
        qsort(tmp, (size_t)n, sizeof *tmp, by_score_then_pos);
        int32_t kc = keep_count_head(c, importance, lambda, h, n);
        for (int32_t i = 0; i < kc; ++i) keep[tmp[i].pos] = 1;
    }
}

wnwo *wnwo_create(const wnwo_config *cfg, const uint16_t *k, const uint16_t *v,
                  const uint8_t *roles, const float *prefill)
{
    return wnwo_create_retention(cfg, k, v, roles, prefill, NULL, 0.0f);
}

wnwo *wnwo_create_retention(const wnwo_config *cfg, const uint16_t *k, const uint16_t *v,
                            const uint8_t *roles, const float *prefill, const float *importance,
                            float lambda)
{
    int32_t nc, kk, kt;
    if (!cfg || !k || !v || !roles || !prefill) return NULL;
    if (wnwo_geometry(cfg, &nc, &kk, &kt)) return NULL;
    for (int32_t i = 0; i < cfg->layers * cfg->kv_heads; ++i)
        if (roles[i] > 2) return NULL;
    if (importance) {
        if (!(lambda >= 0.0f) || isinf(lambda)) return NULL;
        for (int32_t i = 0; i < cfg->layers * cfg->kv_heads; ++i)
            if (!(importance[i] >= 0.0f && importance[i] <= 1.0f)) return NULL;
    }
    wnwo *o = calloc(1, sizeof *o);
    if (!o) return NULL;
    o->c = *cfg;
    o->n_chunks = nc;
    o->n_seg = seg_count(cfg);
    o->span = span_of(cfg);
    o->k = kk;
    o->keep_total = kt;
    o->delta = cfg->evict_lag ? cfg->evict_lag : 3;
    o->kc = k;
    o->vc = v;
    o->tcap = cfg->audio_len + cfg->text_len;
    size_t nh = (size_t)cfg->layers * cfg->kv_heads, B = (size_t)cfg->batch;
    o->roles = malloc(nh);
    o->keep = malloc(B * nh * (size_t)(cfg->audio_len ? cfg->audio_len : 1));
    o->streak = malloc(B * (size_t)(nc ? nc : 1) * sizeof(int32_t));
    o->res_prev = calloc(B * (size_t)(o->n_seg ? o->n_seg : 1), 1);
    ranked *tmp = malloc((size_t)(cfg->prefill_global ? (cfg->audio_len ? cfg->audio_len : 1) : cfg->chunk_len) * sizeof *tmp);
    if (!o->roles || !o->keep || !o->streak || !o->res_prev || !tmp) {
        free(tmp);
        wnwo_destroy(o);
        return NULL;
    }
    memcpy(o->roles, roles, nh);
    if (cfg->max_new > 0) {
        /* room for max_new appended rows after each head's prompt rows */
        const int32_t T = cfg->audio_len + cfg->text_len, D = cfg->head_dim;
        o->tcap = T + cfg->max_new;
        size_t n = B * nh * (size_t)o->tcap * D;
        o->kown = calloc(n, sizeof(uint16_t));
        o->vown = calloc(n, sizeof(uint16_t));
        if (!o->kown || !o->vown) {
            free(tmp);
            wnwo_destroy(o);
            return NULL;
        }
        for (size_t i = 0; i < B * nh; ++i) {
            memcpy(o->kown + i * o->tcap * D, k + i * T * D, (size_t)T * D * sizeof(uint16_t));
            memcpy(o->vown + i * o->tcap * D, v + i * T * D, (size_t)T * D * sizeof(uint16_t));
        }
        o->kc = o->kown;
        o->vc = o->vown;
    }
    for (size_t b = 0; b < B; ++b)
        for (size_t h = 0; h < nh; ++h) {
            uint8_t *kp = o->keep + (b * nh + h) * (size_t)cfg->audio_len;
            if (roles[h] == 0)
                memset(kp, 1, (size_t)cfg->audio_len);         /* anchors keep all audio */
            else
                prefill_keep(cfg, importance, lambda, h, prefill + (b * nh + h) * (size_t)cfg->audio_len,
                             kp, tmp);
        }
    free(tmp);
    /* No chunk has been selected yet: every streak starts at delta (not resident). */
    for (size_t i = 0; i < B * (size_t)nc; ++i) o->streak[i] = o->delta;
    return o;
}

void wnwo_destroy(wnwo *o)
{
    if (!o) return;
    free(o->roles);
    free(o->keep);
    free(o->streak);
    free(o->res_prev);
    free(o->kown);
    free(o->vown);
    free(o);
}

int wnwo_keep_mask(const wnwo *o, int32_t b, int32_t l, int32_t kv, uint8_t *mask)
{
    if (!o || !mask) return -1;
    const wnwo_config *c = &o->c;
    if (b < 0 || b >= c->batch || l < 0 || l >= c->layers || kv < 0 || kv >= c->kv_heads)
        return -1;
    size_t nh = (size_t)c->layers * c->kv_heads;
    memcpy(mask, o->keep + ((size_t)b * nh + (size_t)l * c->kv_heads + kv) * (size_t)c->audio_len,
           (size_t)c->audio_len);
    return 0;
}

/* ---- top-k by (score descending, id ascending) --------------------------------------------- */

typedef struct { float s; int32_t id; } scored;

static int by_score_then_id(const void *a, const void *b)
{
    const scored *x = a, *y = b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->id > y->id) - (x->id < y->id);
}

static int by_int(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

int wnwo_topk(const float *scores, int32_t n, int32_t k, int32_t *sel)
{
    if (n < 0 || k < 0 || k > n || (k && (!scores || !sel))) return -1;
    if (!k) return 0;
    scored *t = malloc((size_t)n * sizeof *t);
    if (!t) return -2;
    for (int32_t i = 0; i < n; ++i) { t[i].s = scores[i]; t[i].id = i; }
    qsort(t, (size_t)n, sizeof *t, by_score_then_id);
    for (int32_t i = 0; i < k; ++i) sel[i] = t[i].id;
    free(t);
    qsort(sel, (size_t)k, sizeof *sel, by_int);
    return 0;
}

/* ---- softmax attention of one query over a listed key set ---------------------------------- */

/* x_i = q . K[rows[i]] / sqrt(d); p = softmax(x); out = sum_i p_i V[rows[i]].  p may be NULL. */
static void attend(const uint16_t *q, const uint16_t *K, const uint16_t *V, const int32_t *rows,
                   int32_t n, int32_t d, double *x, double *out, double *p)
{
    for (int32_t j = 0; j < d; ++j) out[j] = 0.0;
    if (n == 0) return;
    double scale = 1.0 / sqrt((double)d), m = -INFINITY, s = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        const uint16_t *kr = K + (size_t)rows[i] * d;
        double acc = 0.0;
        for (int32_t j = 0; j < d; ++j) acc += bf16(q[j]) * bf16(kr[j]);
        x[i] = acc * scale;
        if (x[i] > m) m = x[i];
    }
    for (int32_t i = 0; i < n; ++i) { x[i] = exp(x[i] - m); s += x[i]; }
    for (int32_t i = 0; i < n; ++i) {
        double pi = x[i] / s;
        const uint16_t *vr = V + (size_t)rows[i] * d;
        for (int32_t j = 0; j < d; ++j) out[j] += pi * bf16(vr[j]);
        if (p) p[i] = pi;
    }
}

/* ---- prefill scores (Method, "Prefill Compression") ------------------------------------------- */

/* p[b][l][kv][tau] = sum over the text tokens t and over the q-heads of KV-head kv of the
 * softmax weight that text token t puts on audio position tau.  Text token t (row T_a + t)
 * attends causally: to every audio row and to text rows up to its own. */
int wnwo_prefill_scores(const wnwo_config *c, const uint16_t *k, const uint16_t *q_text, double *p)
{
    if (!c || !k || !p || (c->text_len && !q_text) || wnwo_geometry(c, NULL, NULL, NULL)) return -1;
    const int32_t B = c->batch, L = c->layers, H = c->kv_heads, Hq = c->q_heads, g = Hq / H, D = c->head_dim;
    const int32_t Ta = c->audio_len, Tt = c->text_len, T = Ta + Tt;
    const int64_t n = (int64_t)B * L * H;
#pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < n; ++i) {
        const int32_t b = (int32_t)(i / ((int64_t)L * H)), l = (int32_t)(i / H % L), kv = (int32_t)(i % H);
        const uint16_t *K = k + (size_t)i * T * D;
        double *ph = p + (size_t)i * Ta;
        double *x = malloc((size_t)(T ? T : 1) * sizeof(double));
        int32_t *rows = malloc((size_t)(T ? T : 1) * sizeof(int32_t));
        double *o = malloc((size_t)D * sizeof(double)), *w = malloc((size_t)(T ? T : 1) * sizeof(double));
        for (int32_t r = 0; r < T; ++r) rows[r] = r;
        for (int32_t t = 0; t < Ta; ++t) ph[t] = 0.0;
        for (int32_t j = 0; j < g; ++j)
            for (int32_t t = 0; t < Tt; ++t) {
                const uint16_t *qv = q_text + ((((size_t)b * L + l) * Hq + (size_t)kv * g + j) * Tt + t) * D;
                attend(qv, K, K, rows, Ta + t + 1, D, x, o, w);
                for (int32_t tau = 0; tau < Ta; ++tau) ph[tau] += w[tau];
            }
        free(x); free(rows); free(o); free(w);
    }
    return 0;
}

/* ---- decode-time append ----------------------------------------------------------------------- */

/* The K and V rows of the token generated at this step, k_new / v_new [B][L][H_kv][d], join every
 * head's key set after the prompt text; generated tokens are not audio, so every role keeps them
 * in full (the remark under Eq. 1). */
int wnwo_append(wnwo *o, const uint16_t *k_new, const uint16_t *v_new)
{
    if (!o || !k_new || !v_new || o->n_gen >= o->c.max_new) return -1;
    const wnwo_config *c = &o->c;
    const size_t nh = (size_t)c->layers * c->kv_heads, D = (size_t)c->head_dim;
    const size_t row = (size_t)c->audio_len + c->text_len + o->n_gen;
    for (size_t i = 0; i < (size_t)c->batch * nh; ++i) {
        memcpy(o->kown + (i * o->tcap + row) * D, k_new + i * D, D * sizeof(uint16_t));
        memcpy(o->vown + (i * o->tcap + row) * D, v_new + i * D, D * sizeof(uint16_t));
    }
    o->n_gen++;
    return 0;
}

/* ---- one decode step -------------------------------------------------------------------------- */

int wnwo_step(wnwo *o, const uint16_t *q, const int32_t *forced, const uint8_t *head_mask,
              double *out, double *scores, int32_t *selected, double *mass, uint8_t *resident)
{
    if (!o || !q || !out || !scores || (o->k && !selected)) return -1;
    const wnwo_config *c = &o->c;
    const int32_t L = c->layers, H = c->kv_heads, Hq = c->q_heads, g = Hq / H, D = c->head_dim;
    /* rows of every key set: audio, prompt text, then the tokens appended so far (kept in full
     * by every head, like text); a head's rows sit at stride tcap */
    const int32_t Ta = c->audio_len, T = Ta + c->text_len + o->n_gen, nc = o->n_chunks, ns = o->n_seg, k = o->k,
                  B = c->batch;
    const size_t nh = (size_t)L * H, TS = (size_t)o->tcap;

    int32_t n_anchor = 0;
    for (size_t h = 0; h < nh; ++h) n_anchor += o->roles[h] == 0;
    const int32_t naq = n_anchor * g;

    /* Anchor KV-heads in (layer, kv) order; their q-heads j = 0..g-1 follow in that order. */
    int32_t *anchor_of = malloc((nh ? nh : 1) * sizeof(int32_t));
    double *m = calloc((size_t)B * (naq ? naq : 1) * (ns ? ns : 1), sizeof(double));
    uint8_t *res_now = calloc((size_t)B * (ns ? ns : 1), 1);
    uint8_t *res_use = calloc((size_t)B * (ns ? ns : 1), 1);
    if (!anchor_of || !m || !res_now || !res_use) {
        free(anchor_of); free(m); free(res_now); free(res_use);
        return -2;
    }
    for (size_t h = 0, a = 0; h < nh; ++h) anchor_of[h] = o->roles[h] == 0 ? (int32_t)a++ : -1;

    memset(out, 0, (size_t)B * L * Hq * D * sizeof(double));
    int status = 0;

    /* Step 1: anchor attention over all audio and text rows, and Eq. 2's mass per segment. */
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int32_t b = 0; b < B; ++b)
        for (int32_t hh = 0; hh < (int32_t)nh; ++hh) {
            if (o->roles[hh] != 0) continue;
            int32_t l = hh / H, kv = hh % H;
            int32_t *rows = malloc((size_t)(T ? T : 1) * sizeof(int32_t));
            double *x = malloc((size_t)(T ? T : 1) * sizeof(double));
            double *p = malloc((size_t)(T ? T : 1) * sizeof(double));
            if (!rows || !x || !p) {
                #pragma omp atomic write
                status = -2;
                free(rows); free(x); free(p);
                continue;
            }
            for (int32_t t = 0; t < T; ++t) rows[t] = t;
            size_t hoff = (((size_t)b * L + l) * H + kv) * TS * D;
            for (int32_t j = 0; j < g; ++j) {
                int32_t hq = kv * g + j;
                const uint16_t *qh = q + (((size_t)b * L + l) * Hq + hq) * D;
                double *oh = out + (((size_t)b * L + l) * Hq + hq) * D;
                attend(qh, o->kc + hoff, o->vc + hoff, rows, T, D, x, oh, p);
                double *mh = m + ((size_t)b * naq + (size_t)anchor_of[hh] * g + j) * ns;
                for (int32_t sg = 0; sg < ns; ++sg) {
                    double acc = 0.0;
                    for (int32_t t = seg_begin(c, sg); t < seg_end(c, sg); ++t) acc += p[t];
                    mh[sg] = acc;
                }
            }
            free(rows); free(x); free(p);
        }
    if (status) goto done;

    /* A forced selection must hold distinct chunk ids (or -1) before any state changes. */
    if (forced)
        for (int32_t b = 0; b < B && !status; ++b)
            for (int32_t i = 0; i < k; ++i) {
                int32_t id = forced[(size_t)b * k + i];
                if (id < -1 || id >= nc) status = -1;
                for (int32_t j = 0; j < i; ++j)
                    if (id >= 0 && forced[(size_t)b * k + j] == id) status = -1;
            }
    if (status) goto done;

    /* Steps 2-4 per sequence: chunk scores, top-k, residency. */
    for (int32_t b = 0; b < B; ++b) {
        float *sf = malloc((size_t)(nc ? nc : 1) * sizeof(float));
        int32_t *sel = malloc((size_t)(k ? k : 1) * sizeof(int32_t));
        if (!sf || !sel) { free(sf); free(sel); status = -2; goto done; }
        for (int32_t ch = 0; ch < nc; ++ch) {
            /* A summed over the chunk's positions (its segments), divided by their number */
            double a = 0.0;
            const int32_t s1 = chunk_last_seg(c, ch);
            for (int32_t h = 0; h < naq; ++h)
                for (int32_t sg = ch; sg <= s1; ++sg) a += m[((size_t)b * naq + h) * ns + sg];
            double sc = a / (double)(seg_end(c, s1) - seg_begin(c, ch));   /* mean over the chunk */
            scores[(size_t)b * nc + ch] = sc;
            sf[ch] = (float)sc;
        }
        if (forced) {
            for (int32_t i = 0; i < k; ++i) sel[i] = forced[(size_t)b * k + i];
            qsort(sel, (size_t)k, sizeof *sel, by_int);
        } else if (wnwo_topk(sf, nc, k, sel)) {
            status = -2;
        }
        if (status) { free(sf); free(sel); goto done; }
        for (int32_t i = 0; i < k; ++i) selected[(size_t)b * k + i] = sel[i];

        int32_t *st = o->streak + (size_t)b * nc;
        uint8_t *now = res_now + (size_t)b * ns;
        for (int32_t ch = 0; ch < nc; ++ch)
            if (st[ch] < o->delta) st[ch] += 1;            /* one more step without selection */
        for (int32_t i = 0; i < k; ++i)
            if (sel[i] >= 0) st[sel[i]] = 0;                /* selected this step             */
        /* resident chunks, and the segments they cover */
        for (int32_t ch = 0; ch < nc; ++ch)
            if (st[ch] < o->delta)
                for (int32_t sg = ch; sg <= chunk_last_seg(c, ch); ++sg) now[sg] = 1;
        memcpy(res_use + (size_t)b * ns, c->next_step ? o->res_prev + (size_t)b * ns : now, (size_t)ns);
        free(sf);
        free(sel);
    }

    /* Step 5: tidal heads (kept + resident complements + text) and fixed heads (kept + text). */
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int32_t b = 0; b < B; ++b)
        for (int32_t hh = 0; hh < (int32_t)nh; ++hh) {
            if (o->roles[hh] == 0 || (head_mask && !head_mask[hh])) continue;
            int32_t l = hh / H, kv = hh % H;
            int32_t *rows = malloc((size_t)(T ? T : 1) * sizeof(int32_t));
            double *x = malloc((size_t)(T ? T : 1) * sizeof(double));
            if (!rows || !x) {
                #pragma omp atomic write
                status = -2;
                free(rows); free(x);
                continue;
            }
            const uint8_t *kp = o->keep + ((size_t)b * nh + hh) * (size_t)Ta;
            const uint8_t *ru = res_use + (size_t)b * ns;
            int32_t n = 0;
            for (int32_t t = 0; t < Ta; ++t) {
                int32_t sg = t / seg_len(c);
                if (kp[t] || (o->roles[hh] == 1 && ru[sg])) rows[n++] = t;
            }
            for (int32_t t = Ta; t < T; ++t) rows[n++] = t;
            size_t hoff = (((size_t)b * L + l) * H + kv) * TS * D;
            for (int32_t j = 0; j < g; ++j) {
                int32_t hq = kv * g + j;
                attend(q + (((size_t)b * L + l) * Hq + hq) * D, o->kc + hoff, o->vc + hoff, rows, n, D, x,
                       out + (((size_t)b * L + l) * Hq + hq) * D, NULL);
            }
            free(rows);
            free(x);
        }
    if (status) goto done;

    memcpy(o->res_prev, res_now, (size_t)B * ns);
    if (mass) memcpy(mass, m, (size_t)B * naq * ns * sizeof(double));
    if (resident) memcpy(resident, res_use, (size_t)B * ns);
done:
    free(anchor_of);
    free(m);
    free(res_now);
    free(res_use);
    return status;
}

/* Threads of the parallel loops (timing only; results do not depend on it). */
int wnwo_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* ---- head triage arithmetic (Method, "Head Functional Triage via Offline Calibration" and the
 * calibration score details of the appendix) ------------------------------------------------------ */

typedef struct { double s; int32_t pos; } scored_d;

static int by_logit_then_pos(const void *a, const void *b)
{
    const scored_d *x = a, *y = b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

/* Voice-score hits: the K audio positions that answer token t's q-head (l, h) attends to most
 * (softmax keeps the order of the logits q.k / sqrt(d); ties to the lower position), counted
 * when inside the token's aligned audio interval [a_t, b_t). */
int wnwo_voice_hits(int32_t L, int32_t Hq, int32_t Hkv, int32_t d, int32_t T, int32_t Ta, int32_t n_tok,
                    const uint16_t *k, const uint16_t *q, const int32_t *span, int32_t K, int32_t *hits)
{
    if (L < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || d < 1 || Ta < 0 || T < Ta || n_tok < 0 || K < 1 || K > Ta ||
        !k || !q || !span || !hits)
        return -1;
    const int32_t g = Hq / Hkv;
    const int64_t n = (int64_t)n_tok * L * Hq;
    int status = 0;
#pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < n; ++i) {
        const int32_t t = (int32_t)(i / ((int64_t)L * Hq)), l = (int32_t)(i / Hq % L), h = (int32_t)(i % Hq);
        const uint16_t *qv = q + (size_t)i * d;
        const uint16_t *K0 = k + ((size_t)l * Hkv + h / g) * (size_t)T * d;
        scored_d *x = malloc((size_t)Ta * sizeof *x);
        if (!x) {
#pragma omp atomic write
            status = -2;
            continue;
        }
        for (int32_t tau = 0; tau < Ta; ++tau) {
            double acc = 0.0;
            for (int32_t j = 0; j < d; ++j) acc += bf16(qv[j]) * bf16(K0[(size_t)tau * d + j]);
            x[tau].s = acc / sqrt((double)d);
            x[tau].pos = tau;
        }
        qsort(x, (size_t)Ta, sizeof *x, by_logit_then_pos);
        int32_t c = 0;
        for (int32_t r = 0; r < K; ++r) c += x[r].pos >= span[2 * t] && x[r].pos < span[2 * t + 1];
        hits[i] = c;
        free(x);
    }
    return status;
}

/* Key sensitivity of each answer token and KV-head: the mean over audio positions of the L2
 * norm of the loss gradient with respect to the position's key vector. */
int wnwo_key_sensitivity(int32_t L, int32_t Hkv, int32_t d, int32_t Ta, int32_t n_tok, const float *grad, double *sens)
{
    if (L < 1 || Hkv < 1 || d < 1 || Ta < 1 || n_tok < 0 || !grad || !sens) return -1;
    const int64_t n = (int64_t)n_tok * L * Hkv;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int32_t tau = 0; tau < Ta; ++tau) {
            const float *gv = grad + ((size_t)i * Ta + tau) * d;
            double s2 = 0.0;
            for (int32_t j = 0; j < d; ++j) s2 += (double)gv[j] * (double)gv[j];
            acc += sqrt(s2);
        }
        sens[i] = acc / Ta;
    }
    return 0;
}

/* Mean over calibration samples of the per-sample mean over its rows of v[row][m] (m < M). */
static void sample_mean(int32_t n, const int32_t *sample, int32_t M, const double *v, double *out)
{
    int32_t ns = 0;
    for (int32_t i = 0; i < n; ++i) if (sample[i] + 1 > ns) ns = sample[i] + 1;
    double *sum = calloc((size_t)(ns ? ns : 1) * M, sizeof(double));
    int32_t *cnt = calloc((size_t)(ns ? ns : 1), sizeof(int32_t));
    for (int32_t i = 0; i < n; ++i) {
        cnt[sample[i]]++;
        for (int32_t m = 0; m < M; ++m) sum[(size_t)sample[i] * M + m] += v[(size_t)i * M + m];
    }
    int32_t used = 0;
    for (int32_t m = 0; m < M; ++m) out[m] = 0.0;
    for (int32_t s = 0; s < ns; ++s) {
        if (!cnt[s]) continue;
        ++used;
        for (int32_t m = 0; m < M; ++m) out[m] += sum[(size_t)s * M + m] / cnt[s];
    }
    for (int32_t m = 0; m < M; ++m) out[m] = used ? out[m] / used : 0.0;
    free(sum);
    free(cnt);
}

typedef struct { double s; int32_t id; } ranked_h;

static int by_importance_then_head(const void *a, const void *b)
{
    const ranked_h *x = a, *y = b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->id > y->id) - (x->id < y->id);
}

/* Three-way classification from the scores of n answer tokens (sample[i] >= 0 names the
 * calibration sample of row i): VS is the per-sample mean of hits / K, averaged over samples and
 * then over the g q-heads of each KV-head; HS the per-sample mean of sens averaged over samples;
 * the importance VS * HS ranks the heads (ties to the lower head index l * H_kv + kv).  The
 * first n_voice are voice heads: their first n_anchor are anchors, the rest tidal; the others are
 * fixed.  The normalised importance divides by the largest importance (all zero if it is 0). */
int wnwo_triage(int32_t L, int32_t Hkv, int32_t g, int32_t n, const int32_t *sample, const int32_t *hits, int32_t K,
                const double *sens, int32_t n_voice, int32_t n_anchor, uint8_t *roles, double *vs, double *hs,
                double *importance_norm)
{
    const int32_t nh = L * Hkv, nq = nh * g;
    if (L < 1 || Hkv < 1 || g < 1 || n < 1 || K < 1 || n_voice < 0 || n_voice > nh || n_anchor < 0 ||
        n_anchor > n_voice || !sample || !hits || !sens || !roles || !vs || !hs || !importance_norm)
        return -1;
    for (int32_t i = 0; i < n; ++i) if (sample[i] < 0) return -1;
    double *hr = malloc((size_t)n * nq * sizeof(double)), *hq = malloc((size_t)nq * sizeof(double));
    ranked_h *rk = malloc((size_t)nh * sizeof *rk);
    for (size_t i = 0; i < (size_t)n * nq; ++i) hr[i] = (double)hits[i] / K;
    sample_mean(n, sample, nq, hr, hq);
    sample_mean(n, sample, nh, sens, hs);
    double mx = 0.0;
    for (int32_t h = 0; h < nh; ++h) {
        double a = 0.0;
        for (int32_t j = 0; j < g; ++j) a += hq[(size_t)h * g + j];
        vs[h] = a / g;
        rk[h].s = vs[h] * hs[h];
        rk[h].id = h;
        if (rk[h].s > mx) mx = rk[h].s;
    }
    for (int32_t h = 0; h < nh; ++h) importance_norm[h] = mx > 0.0 ? rk[h].s / mx : 0.0;
    qsort(rk, (size_t)nh, sizeof *rk, by_importance_then_head);
    for (int32_t r = 0; r < nh; ++r) roles[rk[r].id] = r < n_anchor ? 0 : r < n_voice ? 1 : 2;
    free(hr);
    free(hq);
    free(rk);
    return 0;
}
