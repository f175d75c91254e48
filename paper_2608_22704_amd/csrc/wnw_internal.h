// Internal declarations shared by the WnW host orchestrator and its HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wnw {

constexpr int D = 128;          // head dimension handled by the kernels
constexpr int NT = 256;         // threads per attention work-group (4 wavefronts)
constexpr int TILE_A = 128;     // anchor key rows per work-group
constexpr int TILE_S = 128;     // tidal/fixed kept rows per work-group (slot groups: 128 or 256)
constexpr int MAX_CHUNK = 256;  // longest chunk the slot kernels handle
constexpr int SEL_THREADS = 1024;
constexpr int SCORE_PARTS = 4;   // fixed ranges of anchor KV-heads summed per segment mass

// Everything the kernels need to know about the cache and the step, fixed at set-up.
struct Geometry {
    int B, L, Hq, Hkv, G;
    int Ta, Tt, T;              // audio, prompt text and current rows of an anchor head (T grows by
                                // one per appended token)
    int Tcap, max_new, n_gen;   // anchor row stride (prompt rows + max_new), tokens appended so far
    int cl, budget_bp;          // segment length (the unit of keep sets, masses, residency,
                                // slots and recall), retention in basis points
    int span;                   // segments per chunk: 1 disjoint chunks, 2 overlapping chunks
    int nc;                     // segments
    int nchk;                   // chunks (the selection's candidates): segments - span + 1
    int k, knew, delta;         // chunks selected per step, segments newly resident per step at
                                // most (span * k), eviction lag
    int next_step;              // 1: tidal heads of step s attend over the resident set of step s-1
    int keep_total;             // kept audio rows per non-anchor head with the uniform budget
                                // (-1 with per-head retention)
    int n_slots;                // recall slots per sequence
    int nA, nT, nF;             // anchor / tidal / fixed KV-heads over all layers
    int n_tiles_a, maxc;        // anchor tiles per head (current rows), chunk entries per anchor tile
    int n_tiles_a_cap;          // anchor tiles per head at full capacity (partials are sized for it)
    // Set with the roles (per-head rows, see HeadRows):
    int RsT, RsF;               // rows of a sequence's tidal / fixed static tier
    int n_static;               // static tiles of one sequence (all tidal and fixed heads)
    int P, np_max;              // partial entries of one sequence; most of one head
    int comp_max;               // largest complement of one segment of one tidal head
    int blk_rows;               // rows of one segment's complement block (every tidal head, K and V)
    int64_t keep_sum;           // kept audio rows over all non-anchor heads
    int slot_tile;              // rows of one recall unit's work-group (TILE_S, or 2 * TILE_S when a
                                // complement exceeds TILE_S rows)
    int ng_kept;                // kept items (TILE_S rows of resident complements) of the head with
                                // the most
    int ng_new;                 // partial entries for newly resident complements of the head with
                                // the most (same-step timing: one per entry or TILE_S-row pieces)
    int n_cu;                   // compute units of the device (grid-stride launches)
    int64_t chunk_elems;        // bf16 elements of one segment's complement block (blk_rows * D)
    int64_t slot_off_max;       // slot regions below this many bytes use buffer offsets
    int out_bf16;               // decode-step output written as bf16
};

// Rows of one non-anchor head (tidal heads 0..nT-1, then fixed heads), whose audio retention
// may differ from head to head (Eq. 1).  Partials of a head: its static tiles, then (tidal) its
// kept-list items, then (same-step timing) one per newly resident segment.
struct HeadRows {
    int srow;    // first row of the head in its sequence's static tier (tidal or fixed)
    int rs;      // static rows at set-up: kept audio rows (ascending) + text rows; appended tokens
                 // follow them (rs + n_gen rows, room for max_new)
    int nts;     // static tiles (room included)
    int tile0;   // first static tile of the head among its sequence's static tiles
    int pbase;   // first partial entry of the head among its sequence's partials
    // tidal heads (0 for fixed heads)
    int cfull;   // block stride: the head's largest complement of one segment over the batch
    int coff;    // first row of the head in a segment's complement block: cfull K rows, cfull V rows
    int ngk;     // kept items: TILE_S-row pieces of the head's listed complements at most
    int ngn;     // same-step timing: partials for newly resident complements, one per entry or
                 // TILE_S-row pieces, whichever is more (next-step timing: 0, the kept list holds
                 // them)
    int kfull;   // kept positions of a full segment (set-up)
    int klast;   // kept positions of the last segment (set-up)
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

struct Tiers {
    const uint16_t *aK, *aV;    // [B][nA][T][D]
    const uint16_t *tK, *tV;    // [B][RsT][D]: tidal heads one after the other (HeadRows::srow, rs + max_new)
    const uint16_t *fK, *fV;    // [B][RsF][D]: fixed heads likewise
    uint16_t *slots;            // [B][n_slots][blk_rows][D]
    const uint16_t *host_comp;  // device view of pinned [B][nc][blk_rows][D]
    const int32_t *anchor_lk, *tidal_lk, *fixed_lk;  // l * Hkv + kv of each role's heads
    const HeadRows *hr;         // [nT + nF]
    const int32_t *tile_head;   // [n_static] head of each static tile of a sequence
    const int32_t *comp_rows;   // [B][nc][nT] complement rows of each (sequence, segment, tidal head)
};

struct StepBuffers {
    // anchor partials
    double *pa_m, *pa_l;        // [B][nA][n_tiles_a][G]
    float *pa_o;                // [B][nA][n_tiles_a][G][D]
    double *pa_mass;            // [B][nA][n_tiles_a][G][maxc]
    double *mass;               // [B][nA][nc] normalised chunk mass, summed over the head's q-heads
    double *a_stat;             // [B][nA][G][2] log-sum-exp maximum and 1 / sum of each anchor q-head
    // tidal/fixed partials, head index = tidal 0..nT-1 then fixed nT..nT+nF-1
    float *ps_m, *ps_l;         // [B][P][G]    (HeadRows::pbase + entry)
    float *ps_o;                // [B][P][G][D]
    // selection state (chunks for the selection and streaks; segments for everything else)
    int32_t *streak;            // [B][nchk] steps since the chunk's last selection, capped at delta
    int32_t *slot_of;           // [B][nc]  slot holding the segment's complement or -1
    int32_t *slot_last;         // [B][nc]  slot that last received the segment's bytes or -1
    int32_t *slot_data;         // [B][n_slots] segment whose bytes the slot holds or -1
    int32_t *slot_busy;         // [B][n_slots] 0 free, 1 owned, 2 freed once this step has read it
    int32_t *slot_since;        // [B][n_slots] step at which the slot was last freed
    int32_t *step;              // [B] steps run
    int32_t *att;               // [B][nc]  segment complements attended by the last step
    // Lists of a step (two of each, alternating by step; see wnw_decode_step for which step
    // reads which): kept = resident segments whose bytes are on the device already, new =
    // segments to recall.
    int32_t *kept_list;         // [B][n_slots][2] (segment, slot | full-stride bit 30)
    int32_t *new_list;          // [B][knew][2]    (segment, slot)
    int32_t *counts;            // [B][2] kept-list entries (next-step timing: kept + new), new
    int32_t *arrive;            // [B] the selection in the tidal/fixed launch: anchor heads whose chunk
                                // masses are merged, per sequence (zero between launches); else null
    int32_t *pub;               // host-issued recall: mapped pinned mirror of counts [B][2], new
                                // lists [B][knew][2] and publication tags [B], written by the select
                                // kernel; else null
    int32_t pub_tag;            // the tag the selection stores for each sequence once that
                                // sequence's mirror is visible to the host (nonzero, new each step)
    unsigned long long *stats;  // [8] recalled, dropped, resident, slot_rows, peak, exhausted, revived,
                                // kept-list rows
    int32_t *exhausted;         // mapped pinned flag, set to 1 by a step that found no free slot for a
                                // newly resident segment (the host fails the context on it)
    const int32_t *seg_rows;    // [B][nc] complement rows of a segment over the tidal heads
};

// The selection as part of the next-step tidal/fixed launch: the select kernel's arguments, s
// with the lists the selection writes and the arrival counters.
struct SelectArgs {
    StepBuffers s;
    float *scores;
    const int32_t *ovr;
    int32_t *selected;
    int n_mass;                 // work-groups that merge chunk masses (set by the launcher)
};

// Launchers (wnw_kernels.hip).  Each returns the launch status.  Where a launcher takes two
// events (either may be null), they are bound to the kernel's own dispatch and carry its start
// and end times (hipExtLaunchKernel), or are recorded back to back when there is nothing to launch.
hipError_t launch_anchor(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q,
                         hipStream_t st, hipEvent_t e0, hipEvent_t e1);
// Anchor normalisers and chunk masses (the selection's input); the anchor output rows are merged
// by launch_subset_combine at the end of the step.
hipError_t launch_anchor_mass(const Geometry &g, const StepBuffers &s, hipStream_t st);
// Scores, selection, residency and slot bookkeeping (writes scores[B][nc] and selected[B][k]).
hipError_t launch_select(const Geometry &g, const StepBuffers &s, float *scores, const int32_t *override_sel,
                         int32_t *selected, hipStream_t st);
// Shared memory of the select kernel (bounded at set-up).
inline size_t select_shared_bytes(const Geometry &g)
{
    return (size_t)g.nc * (3 * 8 + 4 + 11 * 4) + (size_t)g.n_slots * 6 * 4 + 3 * (size_t)((g.nc + 63) / 64) * 4;
}
// Fixed heads (with `with_static`), tidal kept rows and the tidal complements already in their
// slots; with `recall`
// (same-step timing), also the copy of the complements listed for recall from mapped pinned
// memory into their slots and the attention over them.
// The slot tiles are the kept list's items (after the static tiles when with_static); `items`:
// the most items of any head this step when the host knows it (the kernel's own count from the
// list counts then agrees), else -1.
// With sel (next-step timing, no recall in the launch), the launch also merges the anchor heads'
// chunk masses and runs the selection, in place of launch_anchor_mass and launch_select (which
// needs tidal_select_fits(g)).
hipError_t launch_tidal_fixed(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, bool recall,
                              bool with_static, long long items, hipStream_t st, hipEvent_t e0 = nullptr,
                              hipEvent_t e1 = nullptr, const SelectArgs *sel = nullptr);
// Whether the tidal/fixed launch's shared memory holds the mass merge and the selection of g.
bool tidal_select_fits(const Geometry &g);
// Anchor attention + chunk mass together with the static tidal/fixed tiles (next-step timing).
hipError_t launch_attention(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st,
                            hipEvent_t e0, hipEvent_t e1);
// Next-step timing: copy of the complements listed for recall from mapped pinned memory into
// their slots, no attention (they are attended from the next step on).
hipError_t launch_recall(const Geometry &g, const Tiers &t, const StepBuffers &s, hipStream_t st);
// Complements already copied to their slots by the host-waited recall path.
hipError_t launch_new_slots(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st);
// Final merge: tidal/fixed heads' partials and anchor heads' tiles into the output rows.
hipError_t launch_subset_combine(const Geometry &g, const Tiers &t, const StepBuffers &s, void *out,
                                 hipStream_t st);
// Prefill scores (wnw_prefill.hip): p [B][L][Hkv][Ta] fp32 from the full K cache
// [B][L][Hkv][T][D] and the text queries [B][L][Hq][Tt][D]; lse [B][L][Hq][Tt] is scratch.
hipError_t launch_prefill_scores(const Geometry &g, const uint16_t *K, const uint16_t *q_text, float *lse,
                                 float *p, hipStream_t st);
// Per-segment keep flags [B][n_sub][Ta] of the non-anchor heads sub_lk[n_sub] (l * Hkv + kv),
// keeping seg_keep[h].x positions of a full segment and .y of the last one.
// With `global`, the same total is ranked over the whole audio of the head instead.  A NaN
// score is marked 2.
hipError_t launch_prefill_keep(const Geometry &g, int n_sub, const int32_t *sub_lk, const int2 *seg_keep, bool global,
                               const float *p, uint8_t *keep, hipStream_t st);
// Decode-time append of one token's K and V rows [B][L][Hkv][D] to every head's tier at row
// T (anchors) or rs + n_gen (tidal, fixed); place[l * Hkv + kv] = anchor index, or -(1 + index
// among the tidal then fixed heads).
hipError_t launch_append_kv(const Geometry &g, const HeadRows *hr, const int32_t *place, uint16_t *aK, uint16_t *aV,
                            uint16_t *tK, uint16_t *tV, uint16_t *fK, uint16_t *fV, const uint16_t *k_new,
                            const uint16_t *v_new, hipStream_t st);
// Set-up: dst[i] = row idx[i] of src_k (idx >= 0), row -idx[i]-2 of src_v (idx <= -2), or zeros
// (idx == -1); a row is D bf16.
hipError_t launch_gather_rows(uint16_t *dst, const uint16_t *src_k, const uint16_t *src_v, const int32_t *idx,
                              int64_t n_rows, hipStream_t st);

}  // namespace wnw
