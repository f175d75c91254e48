// Internal declarations shared by the WnW host orchestrator and its HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wnw {

constexpr int D = 128;          // head dimension handled by the kernels
constexpr int TILE = 256;       // key rows per attention work-group
constexpr int NT = 256;         // threads per attention work-group (4 wavefronts)
constexpr int SEL_THREADS = 1024;

// Everything the kernels need to know about the cache and the step, fixed at set-up.
struct Geometry {
    int B, L, Hq, Hkv, G;
    int Ta, Tt, T;              // audio, text and total rows of an anchor head
    int cl, budget_bp;          // chunk length, retention in basis points
    int nc, k, delta;           // chunks, selected per step, eviction lag
    int keep_total, Rs;         // kept audio rows per non-anchor head; static rows = keep + text
    int comp_max;               // complement rows of a full chunk (chunk_len - keep(chunk_len))
    int n_slots;                // recall slots per sequence (delta * k)
    int nA, nT, nF;             // anchor / tidal / fixed KV-heads over all layers
    int n_tiles_a, maxc;        // anchor tiles per head, chunk entries per anchor tile
    int n_tiles_s;              // static tiles per tidal/fixed head
    int sg;                     // slots per slot-group work-group
    int ng_kept, ng_new;        // slot groups for kept / newly recalled complements
    int np;                     // partial entries per tidal/fixed head
    int64_t chunk_elems;        // bf16 elements of one recalled chunk of one sequence
};

// Keep count of a chunk of `len` positions: floor(retention * len).
__host__ __device__ inline int keep_of_len(int budget_bp, int len)
{
    return (int)(((int64_t)budget_bp * len) / 10000);
}
__host__ __device__ inline int chunk_len_of(const Geometry &g, int c)
{
    int e = (c + 1) * g.cl;
    return (e < g.Ta ? e : g.Ta) - c * g.cl;
}
__host__ __device__ inline int comp_of(const Geometry &g, int c)
{
    int len = chunk_len_of(g, c);
    return len - keep_of_len(g.budget_bp, len);
}

struct Tiers {
    const uint16_t *aK, *aV;    // [B][nA][T][D]
    const uint16_t *tK, *tV;    // [B][nT][Rs][D]
    const uint16_t *fK, *fV;    // [B][nF][Rs][D]
    uint16_t *slots;            // [B][n_slots][nT][2][comp_max][D]
    const uint16_t *host_comp;  // device view of pinned [B][nc][nT][2][comp_max][D]
    const int32_t *anchor_lk, *tidal_lk, *fixed_lk;  // l * Hkv + kv of each role's heads
};

struct StepBuffers {
    // anchor partials
    double *pa_m, *pa_l;        // [B][nA][n_tiles_a][G]
    float *pa_o;                // [B][nA][n_tiles_a][G][D]
    double *pa_mass;            // [B][nA][n_tiles_a][G][maxc]
    double *mass;               // [B][nA*G][nc]
    // tidal/fixed partials, head index = tidal 0..nT-1 then fixed nT..nT+nF-1
    float *ps_m, *ps_l;         // [B][nT+nF][np][G]
    float *ps_o;                // [B][nT+nF][np][G][D]
    // selection state
    int32_t *streak;            // [B][nc]
    int32_t *slot_of;           // [B][nc]  slot holding the chunk's complement or -1
    int32_t *slot_chunk;        // [B][n_slots] chunk held by the slot or -1
    int32_t *kept_list;         // [B][n_slots][2] (chunk, slot) resident before and now
    int32_t *new_list;          // [B][k][2]       (chunk, slot) newly resident this step
    int32_t *counts;            // [B][2] kept, new
    unsigned long long *stats;  // [8] recalled, dropped, resident, slot_rows, peak
};

// Launchers (wnw_kernels.hip).  Each returns the launch status.
hipError_t launch_anchor(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q,
                         hipStream_t st);
hipError_t launch_anchor_combine(const Geometry &g, const Tiers &t, const StepBuffers &s, float *out,
                                 hipStream_t st);
hipError_t launch_scores(const Geometry &g, const StepBuffers &s, float *scores, hipStream_t st);
hipError_t launch_select(const Geometry &g, const StepBuffers &s, const float *scores, const int32_t *override_sel,
                         int32_t *selected, hipStream_t st);
hipError_t launch_recall(const Geometry &g, const Tiers &t, const StepBuffers &s, hipStream_t st);
hipError_t launch_subset_static(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q,
                                hipStream_t st);
hipError_t launch_subset_slots(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q,
                               bool new_list, hipStream_t st);
hipError_t launch_subset_combine(const Geometry &g, const Tiers &t, const StepBuffers &s, float *out,
                                 hipStream_t st);
// Set-up: dst[i] = row idx[i] of src_k (idx >= 0), row -idx[i]-2 of src_v (idx <= -2), or zeros
// (idx == -1); a row is D bf16.
hipError_t launch_gather_rows(uint16_t *dst, const uint16_t *src_k, const uint16_t *src_v, const int32_t *idx,
                              int64_t n_rows, hipStream_t st);

}  // namespace wnw
