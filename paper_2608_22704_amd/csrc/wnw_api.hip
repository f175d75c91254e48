// Host orchestrator of the WnW decode step: the C ABI of include/wnw.h.
//
// Set-up (wnw_set_roles) performs the paper's prefill compression on the host (per segment,
// keep the floor(retention * len) positions with the highest prefill score, retention uniform
// or per head by Eq. 1) and lays the cache out in device tiers:
//   anchor tier   [B][nA][T][d]       every row of every anchor head
//   tidal tier    [B][RsT][d]         per tidal head in turn: kept audio rows (ascending) + text
//   fixed tier    [B][RsF][d]         same for fixed heads (their complement is dropped)
//   slots         [B][n_slots][blk_rows][d]   recalled segment blocks, n_slots from delta, k and
//                 the chunk span (one more k's worth with next-step timing)
//   host complement (pinned) [B][n_segments][blk_rows][d]: segment-major; the block of one
//                 segment holds, per tidal head in turn, its complement K rows then V rows
//                 (cfull of that head each, zero-padded in a short last segment), so the
//                 complement of one segment for every tidal head of a sequence is contiguous.
// A decode step is a fixed sequence of kernels on the caller's stream; recall runs on a side
// stream joined by events (see wnw_decode_step below for the ordering argument).
#include "wnw.h"
#include "wnw_internal.h"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdlib>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <condition_variable>
#include <deque>
#include <functional>
#include <mutex>
#include <numeric>
#include <string>
#include <thread>
#include <vector>

using namespace wnw;

namespace {

thread_local std::string t_err = "no error";

enum State { CREATED = 0, READY = 1, FAILED = 2 };

// Timing events of one step.  e[] on the caller's stream: 0 and 1 the first launch's own start
// and end, 6 after the anchor merge and the selection, 2 before the tidal/fixed launch (after any
// wait for the previous step's recall), 3 after it, 4 once the complements copied this step have
// been attended to (copy-engine recall with same-step timing only: has_new), 5 after the final
// merge.  r[] on the side stream around the recall.
// Streams that share the host-issued copies of one step: copy-engine transfers queued on one
// stream leave a gap between transfers (3 MB copies reach ~49 of ~57 GB/s on one stream, ~56
// on four).
constexpr int N_COPY_STREAMS = 4;
// Next-step timing with host-issued copies: the largest previous-step recall behind which the
// selection still joins the tidal/fixed launch.  4 MiB take ~80 us over the host link (~50 GB/s
// measured), less than the attention launch that precedes the wait for them on the headline
// cache (~96 us), so the selection does not wait.
constexpr int64_t SEL_IN_TIDAL_BYTES = 4ll << 20;

struct StepEvents {
    hipEvent_t e[7];
    bool has_new;
    hipEvent_t r[2];
    // next-step timing with host-issued copies: the end of each copy stream's share (the recall
    // ends with the last of them; joining the streams for one end marker would stall the next
    // step's copies behind the slowest stream)
    hipEvent_t rc[N_COPY_STREAMS];
    bool split;
};

}  // namespace

struct wnw_ctx {
    wnw_config cfg{};
    Geometry g{};
    State state = CREATED;
    std::string err = "no error";
    int device = 0;
    hipStream_t setup_stream = nullptr;
    const uint16_t *full_k = nullptr, *full_v = nullptr;
    std::vector<int32_t> anchor_lk, tidal_lk, fixed_lk;
    std::vector<float> importance;     // [L][Hkv] per-head importance (Eq. 1), empty: uniform budget
    float lambda = 0.f;
    std::vector<HeadRows> hrows;       // [nT + nF]
    std::vector<int32_t> head_keep;    // [nT + nF] kept audio rows
    int64_t keep_sum_t = 0;            // kept audio rows over the tidal heads
    int64_t static_rows = 0;           // static rows over the tidal and fixed heads at set-up
    std::vector<int32_t> comp_rows;    // [B][nc][nT] complement rows of each unit
    std::vector<int32_t> seg_rows;     // [B][nc] their sum over the tidal heads

    Tiers t{};
    StepBuffers s{};
    uint16_t *aK = nullptr, *aV = nullptr, *tK = nullptr, *tV = nullptr, *fK = nullptr, *fV = nullptr;
    uint16_t *slots = nullptr, *host_comp = nullptr;
    int32_t *d_lk = nullptr, *d_tile_head = nullptr, *d_comp_rows = nullptr, *d_seg_rows = nullptr, *d_place = nullptr;
    HeadRows *d_hr = nullptr;
    float *scores_int = nullptr;
    int32_t *sel_int = nullptr;
    const int32_t *override_sel = nullptr;

    hipStream_t side = nullptr;
    // host-issued recall: the copies of one step go round-robin to `side` and these streams,
    // which are joined back into `side` (one stream queues copies with a gap between them)
    hipStream_t copy_st[N_COPY_STREAMS - 1] = {};
    // by step parity: the end of each copy stream's share of that step's host-issued recall, and
    // the end of that step's select kernel (next-step timing with the copy kernel, which never
    // runs the selection inside the tidal launch)
    hipEvent_t ev_copy[2][N_COPY_STREAMS] = {};
    hipEvent_t ev_sel[2] = {}, ev_rec = nullptr;
    bool rec_pending = false;          // next-step timing: a recall issued on `side` not yet joined
    int32_t *h_newinfo = nullptr;      // pinned, two mirrors by step parity: counts [B][2], new
                                       // lists [B][knew][2], publication tags [B]
    int32_t *d_newinfo = nullptr;      // the same memory as the device addresses it
    size_t mirror_ints = 0;            // int32 entries of one mirror
    unsigned copy_mask[2] = {0, 0};    // by step parity: copy streams that received a copy
    unsigned copy_rr = 0;              // copy stream of the next recall's first run

    // Recall thread (next-step timing with host-issued copies): for each step it waits for the
    // step's selection, then issues the step's copies and records their end events, so that
    // wnw_decode_step returns once it has enqueued its own work.  A step waits (on the host) for
    // the previous step's copies to be issued before it enqueues the launch that reads them.
    struct RecallJob {
        int64_t step;
        hipStream_t stream;            // the caller's stream of the step
        bool timed;
        hipEvent_t r0, rc[N_COPY_STREAMS];
    };
    std::thread rthread;
    std::mutex rmu;
    std::condition_variable rcv;
    std::deque<RecallJob> rjobs;
    int64_t rissued = -1;              // last step whose copies are issued
    bool rstop = false;
    hipError_t rerr = hipSuccess;      // first failure of the recall thread
    std::string rerr_msg;
    int32_t delay_us = 0;              // test hook: delay before every recall (wnw_debug_set_recall_delay)
    int32_t *h_flag = nullptr;         // pinned, mapped: [0] slot exhaustion seen by a selection
    int32_t *d_flag = nullptr;         // the same memory as the device addresses it
    double host_wait_ms = 0.0;         // host time spent waiting for selections (copy-engine recall)
    int64_t sel_in_tidal = 0;          // steps whose selection ran inside the tidal launch
    bool log = false;                  // WNW_LOG set: one trace line per step on stderr

    std::vector<StepEvents> pending, spare;
    int n_gen = 0;                     // tokens appended (wnw_append_kv)
    double t_acc[8] = {0};             // anchor, select, tidal/fixed, new, combine, step, recall, recall wait
    int64_t timed_steps = 0, steps = 0;
};

namespace {

// ---- statistics buffer of the allocation-free prefill scores ------------------------------
// wnw_prefill_scores_static keeps the per-row log-sum-exp of the text queries (one fp32 per
// sequence, layer, q-head and text token) in this fixed device array instead of a temporary
// allocation.  Every GPU the library runs on holds its own copy until the process ends; its
// address on a device comes from hipGetSymbolAddress once per device (the array's name is a
// host-side stand-in and is never handed to a kernel).
constexpr size_t STATIC_PREFILL_ROWS = (size_t)8 << 20;   // 32 MiB of fp32
constexpr int MAX_DEVICES = 64;
static __device__ __align__(256) float scratch[STATIC_PREFILL_ROWS];
std::mutex g_scratch_mu;
float *g_scratch_dev[MAX_DEVICES] = {};

wnw_status fail(wnw_ctx *c, wnw_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    if (c) {
        c->err = buf;
        if (st == WNW_ERR_HIP) c->state = FAILED;
    }
    return st;
}

// Device address of the static statistics buffer on device `dev` (which must be current),
// taken once per device; null (with the message in t_err) on failure.
float *scratch_on_device(int dev)
{
    if (dev < 0 || dev >= MAX_DEVICES) {
        fail(nullptr, WNW_ERR_UNSUPPORTED, "device %d: the static prefill buffer is set up for devices 0..%d", dev,
             MAX_DEVICES - 1);
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) {
            (void)hipGetLastError();
            fail(nullptr, WNW_ERR_HIP, "hipGetSymbolAddress of the static prefill buffer on device %d: %s", dev,
                 hipGetErrorString(e));
            return nullptr;
        }
        g_scratch_dev[dev] = (float *)ptr;
    }
    return g_scratch_dev[dev];
}

#define HIPCHECK(ctx, call)                                                                       \
    do {                                                                                          \
        hipError_t e_ = (call);                                                                   \
        if (e_ != hipSuccess)                                                                     \
            return fail(ctx, WNW_ERR_HIP, "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), \
                        __FILE__, __LINE__);                                                      \
    } while (0)

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceGuard()
    {
        int cur;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

template <typename T>
wnw_status dalloc(wnw_ctx *c, T **p, size_t n, const char *what)
{
    *p = nullptr;
    if (n == 0) return WNW_OK;
    hipError_t e = hipMalloc((void **)p, n * sizeof(T));
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *p = nullptr;
        return fail(c, e == hipErrorOutOfMemory ? WNW_ERR_OOM : WNW_ERR_HIP, "hipMalloc of %s (%zu bytes): %s", what,
                    n * sizeof(T), hipGetErrorString(e));
    }
    return WNW_OK;
}

// Pinned host memory (hipHostMalloc).  WNW_TEST_PINNED_LIMIT=<bytes> makes every request above
// that size fail as if the host were out of pinned memory (a test hook for the failure path).
wnw_status palloc(wnw_ctx *c, void **p, size_t bytes, const char *what, unsigned flags = hipHostMallocDefault)
{
    *p = nullptr;
    if (const char *lim = std::getenv("WNW_TEST_PINNED_LIMIT")) {
        const long long cap = std::atoll(lim);
        if (cap >= 0 && bytes > (size_t)cap)
            return fail(c, WNW_ERR_OOM, "pinned %s of %zu bytes: above WNW_TEST_PINNED_LIMIT (%lld)", what, bytes, cap);
    }
    hipError_t e = hipHostMalloc(p, bytes, flags);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *p = nullptr;
        return fail(c, WNW_ERR_OOM, "pinned %s of %zu bytes: %s", what, bytes, hipGetErrorString(e));
    }
    return WNW_OK;
}

// Geometry that depends on the configuration only (roles fill nA/nT/nF later).
wnw_status derive(wnw_ctx *c, const wnw_config &cfg, Geometry &g)
{
    if (cfg.batch < 1 || cfg.layers < 1 || cfg.kv_heads < 1 || cfg.q_heads < 1 || cfg.q_heads % cfg.kv_heads)
        return fail(c, WNW_ERR_INVALID, "batch, layers, heads must be >= 1 and q_heads a multiple of kv_heads");
    if (cfg.audio_len < 0 || cfg.text_len < 0 || cfg.audio_len + (int64_t)cfg.text_len < 1)
        return fail(c, WNW_ERR_INVALID, "need audio_len, text_len >= 0 and at least one row");
    if (cfg.chunk_len < 1) return fail(c, WNW_ERR_INVALID, "chunk_len must be >= 1");
    if (cfg.budget_bp < 0 || cfg.budget_bp > 10000) return fail(c, WNW_ERR_INVALID, "budget_bp must be in 0..10000");
    if (cfg.top_k < 0 || cfg.evict_lag < 0) return fail(c, WNW_ERR_INVALID, "top_k and evict_lag must be >= 0");
    if (cfg.flags & ~(uint32_t)(WNW_F_SELECT_NEXT_STEP | WNW_F_RECALL_MEMCPY | WNW_F_TIMING | WNW_F_OVERLAP_CHUNKS |
                                WNW_F_PREFILL_GLOBAL | WNW_F_OUT_BF16))
        return fail(c, WNW_ERR_INVALID, "unknown flag bits 0x%x", cfg.flags);
    const int span = (cfg.flags & WNW_F_OVERLAP_CHUNKS) ? 2 : 1;
    if (span == 2 && cfg.chunk_len % 2)
        return fail(c, WNW_ERR_INVALID, "overlapping chunks need an even chunk_len (two segments), got %d", cfg.chunk_len);
    if (cfg.head_dim != D) return fail(c, WNW_ERR_UNSUPPORTED, "head_dim %d: only 128 is implemented", cfg.head_dim);
    const int G = cfg.q_heads / cfg.kv_heads;
    if (G != 1 && G != 2 && G != 3 && G != 4 && G != 6 && G != 8)
        return fail(c, WNW_ERR_UNSUPPORTED, "GQA group %d: implemented for 1, 2, 3, 4, 6, 8", G);
    if (cfg.chunk_len / span > MAX_CHUNK)
        return fail(c, WNW_ERR_UNSUPPORTED, "segments of %d positions > %d", cfg.chunk_len / span, MAX_CHUNK);

    g = Geometry{};
    g.slot_off_max = 0xffffffffll;
    g.B = cfg.batch;
    g.L = cfg.layers;
    g.Hq = cfg.q_heads;
    g.Hkv = cfg.kv_heads;
    g.G = G;
    g.Ta = cfg.audio_len;
    g.Tt = cfg.text_len;
    g.T = g.Ta + g.Tt;
    if (cfg.max_new_tokens < 0) return fail(c, WNW_ERR_INVALID, "max_new_tokens must be >= 0");
    g.max_new = cfg.max_new_tokens;
    g.Tcap = g.T + g.max_new;
    g.n_gen = 0;
    g.span = span;
    g.cl = cfg.chunk_len / span;   // segment length
    g.budget_bp = cfg.budget_bp;
    g.nc = (g.Ta + g.cl - 1) / g.cl;
    g.nchk = (span == 2 && g.nc >= 2) ? g.nc - 1 : g.nc;
    g.k = cfg.top_k ? cfg.top_k : (int)(((int64_t)cfg.budget_bp * g.Ta) / (10000LL * cfg.chunk_len));
    if (g.k > g.nchk) return fail(c, WNW_ERR_INVALID, "top_k %d exceeds the %d chunks", g.k, g.nchk);
    g.knew = std::min(g.nc, span * g.k);
    g.delta = cfg.evict_lag ? cfg.evict_lag : 3;
    g.next_step = (cfg.flags & WNW_F_SELECT_NEXT_STEP) ? 1 : 0;
    g.out_bf16 = (cfg.flags & WNW_F_OUT_BF16) ? 1 : 0;
    g.keep_total = 0;
    for (int ch = 0; ch < g.nc; ++ch) g.keep_total += keep_of_len(g.budget_bp, chunk_len_of(g, ch));
    // Slots: the resident set holds at most delta * k chunks, i.e. span * delta * k segments, and
    // the pool holds span * k more.  With next-step timing the segments dropped at a step keep
    // their slots until that step's attention has read them, which needs them; with both timings
    // the free slots keep their last bytes until reused, so a dropped segment that is selected
    // again soon is revived without a copy (the extra slots halve the recalled bytes on the
    // headline workload).  Never more than one per segment.
    const int64_t ns = std::min<int64_t>(g.nc, ((int64_t)g.delta + 1) * span * g.k);
    if (ns > 4096) return fail(c, WNW_ERR_UNSUPPORTED, "%lld recall slots > 4096", (long long)ns);
    g.n_slots = (int)ns;
    if (select_shared_bytes(g) > 150 * 1024)
        return fail(c, WNW_ERR_UNSUPPORTED, "%d chunks with %d slots exceed the selection kernel's shared memory", g.nc,
                    g.n_slots);
    g.n_tiles_a = (g.T + TILE_A - 1) / TILE_A;
    g.n_tiles_a_cap = (g.Tcap + TILE_A - 1) / TILE_A;
    if ((int64_t)g.n_tiles_a_cap * G * 8 > 65536)
        return fail(c, WNW_ERR_UNSUPPORTED, "cache of %d rows (with room for appended tokens) too long", g.Tcap);
    g.maxc = (TILE_A - 1) / g.cl + 2;
    if (g.B > 65535 || (int64_t)g.L * g.Hkv > 65535) return fail(c, WNW_ERR_UNSUPPORTED, "batch or head count too large");
    return WNW_OK;
}

// Keep count of a segment of `len` positions of the head at l * Hkv + kv: floor(retention *
// len), with the uniform budget or with Eq. 1's per-head retention min(importance * lambda, 1)
// (taken in double, where the product of the two fp32 inputs is exact).
int head_keep_of_len(const wnw_ctx *c, int lkh, int len)
{
    if (c->importance.empty()) return keep_of_len(c->g.budget_bp, len);
    double r = (double)c->importance[lkh] * (double)c->lambda;
    if (r > 1.0) r = 1.0;
    return (int)std::floor(r * (double)len);
}

// Keep counts and static rows of the tidal and fixed heads, once the roles are known: kept
// positions per segment, static tier rows and tiles (HeadRows).  The complement layout follows
// from the keep flags (plan_comp).
wnw_status plan_keep(wnw_ctx *c)
{
    Geometry &g = c->g;
    const int nsub = g.nT + g.nF;
    c->hrows.assign(nsub, HeadRows{});
    c->head_keep.assign(nsub, 0);
    const int len0 = g.nc ? chunk_len_of(g, 0) : 0, lenl = g.nc ? chunk_len_of(g, g.nc - 1) : 0;
    int64_t rowT = 0, rowF = 0, tiles = 0;
    g.keep_sum = 0;
    c->static_rows = 0;
    c->keep_sum_t = 0;
    for (int hi = 0; hi < nsub; ++hi) {
        const bool tidal = hi < g.nT;
        const int lkh = tidal ? c->tidal_lk[hi] : c->fixed_lk[hi - g.nT];
        const int k0 = head_keep_of_len(c, lkh, len0), kl = head_keep_of_len(c, lkh, lenl);
        const int keep = g.nc ? (g.nc - 1) * k0 + kl : 0;
        HeadRows &h = c->hrows[hi];
        h.kfull = k0;
        h.klast = kl;
        h.rs = keep + g.Tt;
        h.nts = (h.rs + g.max_new + TILE_S - 1) / TILE_S;   // room for the appended tokens
        h.tile0 = (int)tiles;
        tiles += h.nts;
        h.srow = (int)(tidal ? rowT : rowF);
        (tidal ? rowT : rowF) += h.rs + g.max_new;
        c->static_rows += h.rs;
        if (tidal) c->keep_sum_t += keep;
        c->head_keep[hi] = keep;
        g.keep_sum += keep;
    }
    if (rowT > INT32_MAX / 2 || rowF > INT32_MAX / 2 || tiles * g.B > INT32_MAX / 2)
        return fail(c, WNW_ERR_UNSUPPORTED, "static tiers too large");
    g.RsT = (int)rowT;
    g.RsF = (int)rowF;
    g.n_static = (int)tiles;
    return WNW_OK;
}

// Complement layout from the keep flags [B][nT + nF][T_a]: rows of every (sequence, segment,
// tidal head) complement (comp_rows) and their sum per (sequence, segment) (seg_rows); per
// tidal head the largest over the batch is its block stride (cfull); block offsets, kept-list
// items and partial entries follow.
wnw_status plan_comp(wnw_ctx *c, const uint8_t *flags)
{
    Geometry &g = c->g;
    const int nsub = g.nT + g.nF;
    c->comp_rows.assign((size_t)g.B * g.nc * g.nT, 0);
    c->seg_rows.assign((size_t)g.B * g.nc, 0);
    for (int b = 0; b < g.B; ++b)
        for (int ti = 0; ti < g.nT; ++ti) {
            const uint8_t *f = flags + ((size_t)b * nsub + ti) * g.Ta;
            for (int ch = 0; ch < g.nc; ++ch) {
                const int b0 = ch * g.cl, e0 = b0 + chunk_len_of(g, ch);
                int n = 0;
                for (int t = b0; t < e0; ++t) n += f[t] == 0;
                c->comp_rows[((size_t)b * g.nc + ch) * g.nT + ti] = n;
                c->seg_rows[(size_t)b * g.nc + ch] += n;
                c->hrows[ti].cfull = std::max(c->hrows[ti].cfull, n);
            }
        }
    int64_t coff = 0;
    g.comp_max = 0;
    for (int ti = 0; ti < g.nT; ++ti) {
        c->hrows[ti].coff = (int)coff;
        coff += 2 * c->hrows[ti].cfull;
        g.comp_max = std::max(g.comp_max, c->hrows[ti].cfull);
    }
    if (coff * D > INT32_MAX) return fail(c, WNW_ERR_UNSUPPORTED, "complement blocks too large");
    g.blk_rows = (int)coff;
    g.chunk_elems = coff * D;
    g.slot_tile = g.comp_max <= TILE_S ? TILE_S : 2 * TILE_S;
    // the kept list holds at most the resident segments (span * delta * k) in both timings; a
    // head's kept items cut the run of its kept complements into TILE_S-row pieces
    const int kept_max = (int)std::min<int64_t>(g.nc, (int64_t)g.delta * g.span * g.k);
    int64_t P = 0;
    g.ng_kept = g.ng_new = g.np_max = 0;
    for (int hi = 0; hi < nsub; ++hi) {
        HeadRows &h = c->hrows[hi];
        if (h.cfull > 0) {
            h.ngk = (int)(((int64_t)kept_max * h.cfull + TILE_S - 1) / TILE_S);
            // next-step timing: the new segments join the kept list (no partials of their own);
            // same-step timing: one partial per new entry, or TILE_S-row pieces
            h.ngn = g.next_step ? 0 : (int)std::max<int64_t>(g.knew, ((int64_t)g.knew * h.cfull + TILE_S - 1) / TILE_S);
        }
        g.ng_kept = std::max(g.ng_kept, h.ngk);
        g.ng_new = std::max(g.ng_new, h.ngn);
        h.pbase = (int)P;
        const int np = h.nts + (h.cfull > 0 ? h.ngk + h.ngn : 0);
        P += np;
        g.np_max = std::max(g.np_max, np);
    }
    if ((int64_t)g.np_max * g.G * 4 > 65536) return fail(c, WNW_ERR_UNSUPPORTED, "too many partial tiles per head");
    if (P * g.B > INT32_MAX / 2) return fail(c, WNW_ERR_UNSUPPORTED, "too many partial tiles");
    const int64_t grid_max = (int64_t)g.n_tiles_a_cap * g.nA * g.B + (int64_t)g.n_static * g.B +
                             (int64_t)g.ng_kept * g.nT * g.B;
    if (grid_max > INT32_MAX) return fail(c, WNW_ERR_UNSUPPORTED, "launch grid too large");
    g.P = (int)P;
    return WNW_OK;
}

// Prefill keep selection of one head on the host (Method, "Prefill Compression"), positions
// ranked by (score descending, position ascending): per segment, the kfull (klast for the last
// segment) best; or, globally, the same total over the whole audio.  flags[T_a] = 1 for kept
// positions.  False if a score is NaN.
bool keep_flags_host(const Geometry &g, const HeadRows &hr, bool global, const float *score, uint8_t *flags)
{
    for (int t = 0; t < g.Ta; ++t)
        if (std::isnan(score[t])) return false;
    auto better = [&](int32_t a, int32_t b) {
        if (score[a] != score[b]) return score[a] > score[b];
        return a < b;
    };
    std::vector<int32_t> pos;
    if (global) {
        const int keep = g.nc ? (g.nc - 1) * hr.kfull + hr.klast : 0;
        pos.resize(g.Ta);
        std::iota(pos.begin(), pos.end(), 0);
        std::sort(pos.begin(), pos.end(), better);
        for (int i = 0; i < g.Ta; ++i) flags[pos[i]] = i < keep;
        return true;
    }
    for (int ch = 0; ch < g.nc; ++ch) {
        const int b0 = ch * g.cl, len = chunk_len_of(g, ch), kc = ch == g.nc - 1 ? hr.klast : hr.kfull;
        pos.resize(len);
        std::iota(pos.begin(), pos.end(), b0);
        std::sort(pos.begin(), pos.end(), better);
        for (int i = 0; i < len; ++i) flags[pos[i]] = i < kc;
    }
    return true;
}

// Kept positions (ascending) and, per segment, the complement (ascending) into
// comp_by_seg[ch * cfull ..] (tidal heads; fixed heads drop theirs).  False if the flags do not
// hold `keep` kept positions or a complement exceeds the stride (the layout was sized for them).
bool rows_from_flags(const Geometry &g, const HeadRows &hr, int keep, bool tidal, const uint8_t *flags,
                     std::vector<int32_t> &kept, std::vector<int32_t> &comp_by_seg)
{
    kept.clear();
    comp_by_seg.assign((size_t)g.nc * hr.cfull, -1);
    for (int ch = 0; ch < g.nc; ++ch) {
        const int b0 = ch * g.cl, e0 = b0 + chunk_len_of(g, ch);
        int nd = 0;
        for (int t = b0; t < e0; ++t) {
            if (flags[t]) {
                kept.push_back(t);
            } else if (tidal) {
                if (nd >= hr.cfull) return false;
                comp_by_seg[(size_t)ch * hr.cfull + nd++] = t;
            }
        }
    }
    return (int)kept.size() == keep;
}

void parallel_for(int n, const std::function<void(int)> &fn)
{
    int nt = (int)std::min<unsigned>(16, std::max(1u, std::thread::hardware_concurrency()));
    nt = std::min(nt, std::max(n, 1));
    std::vector<std::thread> th;
    for (int w = 0; w < nt; ++w)
        th.emplace_back([&, w] {
            for (int i = w; i < n; i += nt) fn(i);
        });
    for (auto &x : th) x.join();
}

// Tag the selection of `step` publishes with the mirror (nonzero; steps two apart, which
// share a mirror, differ).
int32_t pub_tag(int64_t step)
{
    return (int32_t)(step % 0x7ffffffe) + 1;
}

// Waits (busy polling: a sleeping wait wakes tens to hundreds of microseconds late) until the
// selection of `step`, enqueued on `st`, has published the mirror of parity step & 1 for
// every sequence.  Every millisecond it also asks whether `st` has failed, or has completed
// without the tags (which would be a defect): either is returned as an error.
hipError_t wait_published(const wnw_ctx *c, int64_t step, hipStream_t st)
{
    const int B = c->g.B;
    const int32_t *tags = c->h_newinfo + (step & 1) * c->mirror_ints + B * 2 + (size_t)B * c->g.knew * 2;
    const int32_t want = pub_tag(step);
    auto published = [&] {
        for (int b = 0; b < B; ++b)
            if (__atomic_load_n(tags + b, __ATOMIC_ACQUIRE) != want) return false;
        return true;
    };
    auto next_check = std::chrono::steady_clock::now() + std::chrono::milliseconds(1);
    bool drained = false;
    for (;;) {
        for (int i = 0; i < 256; ++i)
            if (published()) return hipSuccess;
        const auto now = std::chrono::steady_clock::now();
        if (now < next_check) continue;
        if (drained) return hipErrorUnknown;   // the stream completed 1 ms ago, no tag since
        const hipError_t e = hipStreamQuery(st);
        if (e != hipSuccess && e != hipErrorNotReady) return e;
        drained = e == hipSuccess;
        next_check = now + std::chrono::milliseconds(1);
    }
}

// Test hook: a host function that sleeps `us` microseconds, queued ahead of a recall on its
// streams (the recall's readers must still see its bytes: tests compare against an undelayed run).
void delay_fn(void *us)
{
    std::this_thread::sleep_for(std::chrono::microseconds(*(const int32_t *)us));
}

// Host-issued recall of the step of parity `par`: one hipMemcpyAsync per run of consecutive
// chunks landing in consecutive slots, from the counts and new lists that step's selection
// mirrored to pinned memory (already complete on the host).  The runs go round-robin to `st` and
// the extra copy streams; ev_copy[par][i] marks the end of each stream's share.  The caller has
// seen the step's selection complete on the host, so every earlier reader of the target slots
// has finished and the copies need no device-side wait.  Returns the first failing call's status.
hipError_t issue_copies_raw(wnw_ctx *c, int par, hipStream_t st, const char **what)
{
    const Geometry &g = c->g;
    const int32_t *cnt = c->h_newinfo + par * c->mirror_ints, *nl = cnt + g.B * 2;
    const size_t cb = (size_t)g.chunk_elems * sizeof(uint16_t);
    hipError_t e = hipSuccess;
    unsigned mask = 0;
    if (c->delay_us > 0) {
        for (int i = 0; i < N_COPY_STREAMS && e == hipSuccess; ++i)
            e = hipLaunchHostFunc(i == 0 ? st : c->copy_st[i - 1], delay_fn, &c->delay_us);
        mask = (1u << N_COPY_STREAMS) - 1;   // every stream holds a delay
    }
    // the round-robin continues from the previous step's last stream, so that over the steps
    // every copy stream carries the same share (restarting at the first stream each step would
    // give the first ones one run more per step)
    unsigned n_runs = c->copy_rr;
    for (int b = 0; b < g.B && cb && e == hipSuccess; ++b) {
        const int n = cnt[b * 2 + 1];
        for (int i = 0; i < n && e == hipSuccess;) {
            int j = i + 1;
            const int32_t *e0 = nl + ((size_t)b * g.knew + i) * 2;
            while (j < n) {
                const int32_t *ej = nl + ((size_t)b * g.knew + j) * 2;
                if (ej[0] != e0[0] + (j - i) || ej[1] != e0[1] + (j - i)) break;
                ++j;
            }
            const int w = (int)(n_runs++ % N_COPY_STREAMS);
            mask |= 1u << w;
            e = hipMemcpyAsync(c->slots + ((size_t)b * g.n_slots + e0[1]) * g.chunk_elems,
                               c->host_comp + ((size_t)b * g.nc + e0[0]) * g.chunk_elems, cb * (j - i),
                               hipMemcpyHostToDevice, w == 0 ? st : c->copy_st[w - 1]);
            i = j;
        }
    }
    if (e != hipSuccess) {
        *what = "hipMemcpyAsync of a recall";
        return e;
    }
    // the readers wait only for the streams that received work (an empty wait still costs a
    // cross-stream synchronisation on the device)
    for (int i = 0; i < N_COPY_STREAMS; ++i) {
        if (!(mask >> i & 1)) continue;
        e = hipEventRecord(c->ev_copy[par][i], i == 0 ? st : c->copy_st[i - 1]);
        if (e != hipSuccess) {
            *what = "hipEventRecord after a recall";
            return e;
        }
    }
    c->copy_mask[par] = mask;
    c->copy_rr = n_runs % N_COPY_STREAMS;
    return hipSuccess;
}

wnw_status issue_copies(wnw_ctx *c, int par, hipStream_t st)
{
    const char *what = "";
    const hipError_t e = issue_copies_raw(c, par, st, &what);
    if (e != hipSuccess) return fail(c, WNW_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
    return WNW_OK;
}

// `s` waits for every copy of the host-issued recall of the step of parity `par` (one hop per
// copy stream).
wnw_status wait_copies(wnw_ctx *c, int par, hipStream_t s)
{
    for (int i = 0; i < N_COPY_STREAMS; ++i)
        if (c->copy_mask[par] >> i & 1) HIPCHECK(c, hipStreamWaitEvent(s, c->ev_copy[par][i], 0));
    return WNW_OK;
}

// The recall thread's loop (see wnw_ctx::RecallJob).
void recall_thread(wnw_ctx *c)
{
    (void)hipSetDevice(c->device);
    for (;;) {
        wnw_ctx::RecallJob job;
        {
            std::unique_lock<std::mutex> lk(c->rmu);
            c->rcv.wait(lk, [&] { return c->rstop || !c->rjobs.empty(); });
            if (c->rjobs.empty()) return;   // stopping, nothing left
            job = c->rjobs.front();
        }
        const int par = (int)(job.step & 1);
        hipError_t e = hipSuccess;
        const char *what = "";
        if (c->rerr == hipSuccess) {
            const auto w0 = std::chrono::steady_clock::now();
            e = wait_published(c, job.step, job.stream);
            const double waited = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - w0).count();
            if (e != hipSuccess) what = "the wait for a selection";
            if (e == hipSuccess && c->delay_us > 0) std::this_thread::sleep_for(std::chrono::microseconds(c->delay_us));
            if (e == hipSuccess && job.timed) {
                e = hipEventRecord(job.r0, c->side);
                if (e != hipSuccess) what = "hipEventRecord of a recall start";
            }
            if (e == hipSuccess) e = issue_copies_raw(c, par, c->side, &what);
            for (int i = 0; i < N_COPY_STREAMS && e == hipSuccess && job.timed; ++i) {
                e = hipEventRecord(job.rc[i], i == 0 ? c->side : c->copy_st[i - 1]);
                if (e != hipSuccess) what = "hipEventRecord of a recall end";
            }
            std::lock_guard<std::mutex> lk(c->rmu);
            c->host_wait_ms += waited;
        }
        {
            // a failure is kept for the caller's thread; the step still counts as issued so that
            // no one waits for it
            std::lock_guard<std::mutex> lk(c->rmu);
            if (e != hipSuccess && c->rerr == hipSuccess) {
                c->rerr = e;
                c->rerr_msg = std::string(what) + " failed: " + hipGetErrorString(e);
            }
            c->rjobs.pop_front();
            c->rissued = job.step;
        }
        c->rcv.notify_all();
    }
}

// Waits until the recall thread has issued the copies of every step up to `step` (all queued
// ones when step < 0); a failure of the thread fails the context.
wnw_status recall_wait_issued(wnw_ctx *c, int64_t step)
{
    if (!c->rthread.joinable()) return WNW_OK;
    std::unique_lock<std::mutex> lk(c->rmu);
    c->rcv.wait(lk, [&] { return step < 0 ? c->rjobs.empty() : c->rissued >= step; });
    if (c->rerr != hipSuccess) {
        c->state = FAILED;
        return fail(c, WNW_ERR_HIP, "recall thread: %s", c->rerr_msg.c_str());
    }
    return WNW_OK;
}

void recall_stop(wnw_ctx *c)
{
    if (!c->rthread.joinable()) return;
    {
        std::lock_guard<std::mutex> lk(c->rmu);
        c->rstop = true;
    }
    c->rcv.notify_all();
    c->rthread.join();
}

// Slot exhaustion reported by a selection (mapped pinned flag): the context fails, since
// tidal heads of that step missed a resident segment.  Reads host memory only (no wait).
wnw_status check_exhaustion(wnw_ctx *c)
{
    if (c->h_flag && *(volatile int32_t *)c->h_flag) {
        c->state = FAILED;
        return fail(c, WNW_ERR_STATE, "a decode step found no free recall slot for a newly resident segment "
                                      "(slot pool of %d per sequence exhausted)", c->g.n_slots);
    }
    return WNW_OK;
}

wnw_status harvest_timing(wnw_ctx *c)
{
    const StepEvents *prev = nullptr;
    int prev_last = 0;
    for (auto &ev : c->pending) {
        float ms;
        HIPCHECK(c, hipEventSynchronize(ev.e[5]));
        // anchor, select, tidal/fixed, new, combine, step, -, recall wait
        const int m = ev.has_new ? 4 : 3;
        const int from[8] = {0, 1, 2, 3, m, 0, -1, 6}, to[8] = {1, 6, 3, 4, 5, 5, -1, 2};
        for (int i = 0; i < 8; ++i) {
            if (from[i] < 0 || (i == 3 && !ev.has_new)) continue;
            HIPCHECK(c, hipEventElapsedTime(&ms, ev.e[from[i]], ev.e[to[i]]));
            c->t_acc[i] += ms;
        }
        if (ev.split) {
            float t = 0.f;
            int last = 0;
            for (int i = 0; i < N_COPY_STREAMS; ++i) {
                HIPCHECK(c, hipEventSynchronize(ev.rc[i]));
                HIPCHECK(c, hipEventElapsedTime(&ms, ev.r[0], ev.rc[i]));
                if (i == 0 || ms > t) t = ms, last = i;
            }
            // this step's copies queue behind the previous step's on each stream: the time
            // before the previous step's last copy ended is counted there
            if (prev && prev->split) {
                HIPCHECK(c, hipEventElapsedTime(&ms, ev.r[0], prev->rc[prev_last]));
                if (ms > 0.f) t -= ms;
            }
            c->t_acc[6] += t > 0.f ? t : 0.f;
            prev_last = last;
        } else {
            HIPCHECK(c, hipEventSynchronize(ev.r[1]));
            HIPCHECK(c, hipEventElapsedTime(&ms, ev.r[0], ev.r[1]));
            c->t_acc[6] += ms;
        }
        prev = &ev;
        c->timed_steps++;
        c->spare.push_back(ev);
    }
    c->pending.clear();
    return WNW_OK;
}

void free_all(wnw_ctx *c)
{
    void *ptrs[] = {c->aK, c->aV, c->tK, c->tV, c->fK, c->fV, c->slots, c->d_lk, c->d_tile_head, c->d_hr,
                    c->d_comp_rows, c->d_seg_rows, c->d_place,
                    c->scores_int, c->sel_int,
                    c->s.pa_m, c->s.pa_l, c->s.pa_o, c->s.pa_mass, c->s.mass, c->s.a_stat, c->s.ps_m, c->s.ps_l, c->s.ps_o,
                    c->s.streak, c->s.slot_of, c->s.slot_last, c->s.att, c->s.slot_data, c->s.slot_busy, c->s.slot_since,
                    c->s.step, c->s.kept_list, c->s.new_list, c->s.counts, c->s.arrive, c->s.stats};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);
    if (c->host_comp) (void)hipHostFree(c->host_comp);
    if (c->h_newinfo) (void)hipHostFree(c->h_newinfo);
    if (c->h_flag) (void)hipHostFree(c->h_flag);
    for (auto e : c->ev_sel)
        if (e) (void)hipEventDestroy(e);
    if (c->ev_rec) (void)hipEventDestroy(c->ev_rec);
    for (auto *v : {&c->pending, &c->spare})
        for (auto &ev : *v) {
            for (auto e : ev.e) (void)hipEventDestroy(e);
            for (auto e : ev.r) (void)hipEventDestroy(e);
            for (auto e : ev.rc) (void)hipEventDestroy(e);
        }
    if (c->side) (void)hipStreamDestroy(c->side);
    for (int i = 0; i < N_COPY_STREAMS - 1; ++i)
        if (c->copy_st[i]) (void)hipStreamDestroy(c->copy_st[i]);
    for (auto &par : c->ev_copy)
        for (auto e : par)
            if (e) (void)hipEventDestroy(e);
}

}  // namespace

extern "C" {

const char *wnw_last_error(const wnw_ctx *ctx)
{
    return ctx ? ctx->err.c_str() : t_err.c_str();
}

wnw_status wnw_init_cache(const wnw_config *cfg, const void *k_dev, const void *v_dev, void *hip_stream, wnw_ctx **out)
{
    if (!out) return fail(nullptr, WNW_ERR_INVALID, "out is NULL");
    *out = nullptr;
    if (!cfg || !k_dev || !v_dev) return fail(nullptr, WNW_ERR_INVALID, "cfg, k_dev and v_dev must not be NULL");
    Geometry g;
    wnw_status st = derive(nullptr, *cfg, g);
    if (st != WNW_OK) return st;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(nullptr, WNW_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    wnw_ctx *c = new (std::nothrow) wnw_ctx();
    if (!c) return fail(nullptr, WNW_ERR_OOM, "context allocation failed");
    c->cfg = *cfg;
    c->g = g;
    if (hipDeviceGetAttribute(&c->g.n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c->g.n_cu < 1) {
        (void)hipGetLastError();
        c->g.n_cu = 1;
    }
    c->device = dev;
    c->setup_stream = (hipStream_t)hip_stream;
    c->full_k = (const uint16_t *)k_dev;
    c->full_v = (const uint16_t *)v_dev;
    const char *lg = std::getenv("WNW_LOG");
    c->log = lg && *lg && strcmp(lg, "0") != 0;
    // the static prefill buffer's address on this device (once per device; the current device)
    if (!scratch_on_device(dev)) {
        delete c;
        return WNW_ERR_HIP;
    }
    *out = c;
    return WNW_OK;
}

}  // extern "C"

namespace {

// Roles and per-head rows; nothing allocated.
wnw_status assign_roles(wnw_ctx *c, const uint8_t *roles)
{
    Geometry &g = c->g;
    const int nh = g.L * g.Hkv;
    for (int i = 0; i < nh; ++i)
        if (roles[i] > WNW_FIXED) return fail(c, WNW_ERR_INVALID, "role %d of head %d is not a wnw_role", roles[i], i);
    c->anchor_lk.clear();
    c->tidal_lk.clear();
    c->fixed_lk.clear();
    for (int i = 0; i < nh; ++i)
        (roles[i] == WNW_ANCHOR ? c->anchor_lk : roles[i] == WNW_TIDAL ? c->tidal_lk : c->fixed_lk).push_back(i);
    g.nA = (int)c->anchor_lk.size();
    g.nT = (int)c->tidal_lk.size();
    g.nF = (int)c->fixed_lk.size();
    return plan_keep(c);
}

// Complement layout, allocations and tier construction from the keep flags [B][nT + nF][T_a]
// (ranked on the host or on the device).
wnw_status build_tiers(wnw_ctx *c, const uint8_t *keep_all)
{
    Geometry &g = c->g;
    const int nh = g.L * g.Hkv;
    DeviceGuard dg(c->device);
    hipStream_t st = c->setup_stream;
    const size_t B = g.B, Dz = D;
    wnw_status r = plan_comp(c, keep_all);
    if (r != WNW_OK) return r;

    // ---- allocations ------------------------------------------------------------------
#define ALLOC(p, n, what) \
    if ((r = dalloc(c, &(p), (size_t)(n), what)) != WNW_OK) return r
    // K/V tiers, each with one zeroed tile of padding rows at the end (the tiles' buffer loads)
    const size_t pad = (size_t)std::max(TILE_A, TILE_S) * Dz;
    ALLOC(c->aK, B * g.nA * g.Tcap * Dz + pad, "anchor K");
    ALLOC(c->aV, B * g.nA * g.Tcap * Dz + pad, "anchor V");
    ALLOC(c->tK, B * g.RsT * Dz + pad, "tidal K");
    ALLOC(c->tV, B * g.RsT * Dz + pad, "tidal V");
    ALLOC(c->fK, B * g.RsF * Dz + pad, "fixed K");
    ALLOC(c->fV, B * g.RsF * Dz + pad, "fixed V");
    // anchor rows reserved for appended tokens and every padding tile start out zero
    HIPCHECK(c, hipMemsetAsync(c->aK, 0, (B * g.nA * g.Tcap * Dz + pad) * sizeof(uint16_t), st));
    HIPCHECK(c, hipMemsetAsync(c->aV, 0, (B * g.nA * g.Tcap * Dz + pad) * sizeof(uint16_t), st));
    HIPCHECK(c, hipMemsetAsync(c->tK + B * g.RsT * Dz, 0, pad * sizeof(uint16_t), st));
    HIPCHECK(c, hipMemsetAsync(c->tV + B * g.RsT * Dz, 0, pad * sizeof(uint16_t), st));
    HIPCHECK(c, hipMemsetAsync(c->fK + B * g.RsF * Dz, 0, pad * sizeof(uint16_t), st));
    HIPCHECK(c, hipMemsetAsync(c->fV + B * g.RsF * Dz, 0, pad * sizeof(uint16_t), st));
    ALLOC(c->slots, B * g.n_slots * g.chunk_elems, "recall slots");
    ALLOC(c->d_lk, (size_t)nh, "role tables");
    ALLOC(c->d_hr, c->hrows.size(), "head rows");
    ALLOC(c->d_tile_head, (size_t)g.n_static, "static tile table");
    ALLOC(c->d_place, (size_t)nh, "append table");
    ALLOC(c->d_comp_rows, c->comp_rows.size(), "complement rows");
    ALLOC(c->d_seg_rows, c->seg_rows.size(), "segment rows");
    ALLOC(c->scores_int, B * g.nchk, "scores");
    ALLOC(c->sel_int, B * g.k, "selection");
    StepBuffers &s = c->s;
    ALLOC(s.pa_m, B * g.nA * g.n_tiles_a_cap * g.G, "anchor partial max");
    ALLOC(s.pa_l, B * g.nA * g.n_tiles_a_cap * g.G, "anchor partial sum");
    ALLOC(s.pa_o, B * g.nA * g.n_tiles_a_cap * g.G * Dz, "anchor partial out");
    ALLOC(s.pa_mass, B * g.nA * g.n_tiles_a_cap * g.G * g.maxc, "anchor partial mass");
    ALLOC(s.mass, B * g.nA * g.nc, "chunk mass");
    ALLOC(s.a_stat, B * g.nA * g.G * 2, "anchor normalisers");
    ALLOC(s.ps_m, B * g.P * g.G, "partial max");
    ALLOC(s.ps_l, B * g.P * g.G, "partial sum");
    ALLOC(s.ps_o, B * g.P * g.G * Dz, "partial out");
    ALLOC(s.streak, B * g.nchk, "streaks");
    ALLOC(s.slot_of, B * g.nc, "slot map");
    ALLOC(s.slot_last, B * g.nc, "slot history");
    ALLOC(s.att, B * g.nc, "attended complements");
    ALLOC(s.slot_data, B * g.n_slots, "slot contents");
    ALLOC(s.slot_busy, B * g.n_slots, "slot owners");
    ALLOC(s.slot_since, B * g.n_slots, "slot ages");
    ALLOC(s.step, B, "step counters");
    ALLOC(s.kept_list, 2 * B * g.n_slots * 2, "kept lists");   // two of each, alternating by step
    ALLOC(s.new_list, 2 * B * g.knew * 2, "new lists");
    ALLOC(s.counts, 2 * B * 2, "counts");
    ALLOC(s.arrive, B, "arrival counters");
    ALLOC(s.stats, 8, "stats");
#undef ALLOC
    const size_t host_bytes = B * g.nc * (size_t)g.chunk_elems * sizeof(uint16_t);
    if (host_bytes) {
        if ((r = palloc(c, (void **)&c->host_comp, host_bytes, "complement")) != WNW_OK) return r;
        void *dp = nullptr;
        HIPCHECK(c, hipHostGetDevicePointer(&dp, c->host_comp, 0));
        c->t.host_comp = (const uint16_t *)dp;
    }
    // coherent: the selection's stores reach host memory without a cache write-back
    c->mirror_ints = B * 2 + B * g.knew * 2 + B;
    if ((r = palloc(c, (void **)&c->h_newinfo, 2 * c->mirror_ints * sizeof(int32_t), "recall lists",
                    hipHostMallocCoherent)) != WNW_OK)
        return r;
    {
        memset(c->h_newinfo, 0, 2 * c->mirror_ints * sizeof(int32_t));   // no tag published yet
        void *dp = nullptr;
        HIPCHECK(c, hipHostGetDevicePointer(&dp, c->h_newinfo, 0));
        c->d_newinfo = (int32_t *)dp;
    }
    if ((r = palloc(c, (void **)&c->h_flag, 4 * sizeof(int32_t), "status flags")) != WNW_OK) return r;
    {
        memset(c->h_flag, 0, 4 * sizeof(int32_t));
        void *dp = nullptr;
        HIPCHECK(c, hipHostGetDevicePointer(&dp, c->h_flag, 0));
        c->d_flag = (int32_t *)dp;
        c->s.exhausted = c->d_flag;
    }
    HIPCHECK(c, hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking));
    if (c->cfg.flags & WNW_F_RECALL_MEMCPY) {
        for (int i = 0; i < N_COPY_STREAMS - 1; ++i)
            HIPCHECK(c, hipStreamCreateWithFlags(&c->copy_st[i], hipStreamNonBlocking));
        for (auto &par : c->ev_copy)
            for (auto &e : par) HIPCHECK(c, hipEventCreateWithFlags(&e, hipEventDisableTiming));
    }
    for (auto &e : c->ev_sel) HIPCHECK(c, hipEventCreateWithFlags(&e, hipEventDisableTiming));
    HIPCHECK(c, hipEventCreateWithFlags(&c->ev_rec, hipEventDisableTiming));

    std::vector<int32_t> lk;
    lk.insert(lk.end(), c->anchor_lk.begin(), c->anchor_lk.end());
    lk.insert(lk.end(), c->tidal_lk.begin(), c->tidal_lk.end());
    lk.insert(lk.end(), c->fixed_lk.begin(), c->fixed_lk.end());
    if (nh) HIPCHECK(c, hipMemcpy(c->d_lk, lk.data(), nh * sizeof(int32_t), hipMemcpyHostToDevice));
    if (!c->hrows.empty())
        HIPCHECK(c, hipMemcpy(c->d_hr, c->hrows.data(), c->hrows.size() * sizeof(HeadRows), hipMemcpyHostToDevice));
    {
        std::vector<int32_t> th((size_t)g.n_static);
        for (int hi = 0; hi < (int)c->hrows.size(); ++hi)
            for (int j = 0; j < c->hrows[hi].nts; ++j) th[(size_t)c->hrows[hi].tile0 + j] = hi;
        if (!th.empty())
            HIPCHECK(c, hipMemcpy(c->d_tile_head, th.data(), th.size() * sizeof(int32_t), hipMemcpyHostToDevice));
    }
    if (!c->comp_rows.empty())
        HIPCHECK(c, hipMemcpy(c->d_comp_rows, c->comp_rows.data(), c->comp_rows.size() * sizeof(int32_t), hipMemcpyHostToDevice));
    if (!c->seg_rows.empty())
        HIPCHECK(c, hipMemcpy(c->d_seg_rows, c->seg_rows.data(), c->seg_rows.size() * sizeof(int32_t), hipMemcpyHostToDevice));
    c->t.comp_rows = c->d_comp_rows;
    c->s.seg_rows = c->d_seg_rows;
    {
        std::vector<int32_t> place(nh);
        for (int a = 0; a < g.nA; ++a) place[c->anchor_lk[a]] = a;
        for (int i = 0; i < g.nT; ++i) place[c->tidal_lk[i]] = -(1 + i);
        for (int i = 0; i < g.nF; ++i) place[c->fixed_lk[i]] = -(1 + g.nT + i);
        if (nh) HIPCHECK(c, hipMemcpy(c->d_place, place.data(), nh * sizeof(int32_t), hipMemcpyHostToDevice));
    }
    c->t.hr = c->d_hr;
    c->t.tile_head = c->d_tile_head;
    c->t.anchor_lk = c->d_lk;
    c->t.tidal_lk = c->d_lk + g.nA;
    c->t.fixed_lk = c->d_lk + g.nA + g.nT;
    c->t.aK = c->aK; c->t.aV = c->aV;
    c->t.tK = c->tK; c->t.tV = c->tV;
    c->t.fK = c->fK; c->t.fV = c->fV;
    c->t.slots = c->slots;

    // ---- per-sequence tier construction ------------------------------------------------------
    const int nsub = g.nT + g.nF;
    const size_t seq_rows = (size_t)g.L * g.Hkv * g.T;
    // rows reserved for appended tokens stay zero (index -1) until an append writes them
    std::vector<int32_t> static_idx((size_t)g.RsT + g.RsF, -1), comp_idx((size_t)g.nc * g.blk_rows);
    int32_t *d_idx = nullptr;
    uint16_t *staging = nullptr;
    const size_t idx_n = std::max(static_idx.size(), comp_idx.size());
    if ((r = dalloc(c, &d_idx, idx_n, "set-up index")) != WNW_OK) return r;
    if ((r = dalloc(c, &staging, (size_t)g.nc * g.chunk_elems, "complement staging")) != WNW_OK) {
        (void)hipFree(d_idx);
        return r;
    }
    auto cleanup = [&] {
        (void)hipStreamSynchronize(st);
        if (d_idx) (void)hipFree(d_idx);
        if (staging) (void)hipFree(staging);
    };
    for (int b = 0; b < g.B; ++b) {
        const uint16_t *fk = c->full_k + b * seq_rows * D, *fv = c->full_v + b * seq_rows * D;
        // anchors: every row, one contiguous copy per head
        for (int a = 0; a < g.nA; ++a) {
            const size_t src = (size_t)c->anchor_lk[a] * g.T * D, dst = (((size_t)b * g.nA + a) * g.Tcap) * D;
            const size_t bytes = (size_t)g.T * D * sizeof(uint16_t);
            hipError_t e1 = hipMemcpyAsync(c->aK + dst, fk + src, bytes, hipMemcpyDeviceToDevice, st);
            hipError_t e2 = hipMemcpyAsync(c->aV + dst, fv + src, bytes, hipMemcpyDeviceToDevice, st);
            if (e1 != hipSuccess || e2 != hipSuccess) {
                cleanup();
                return fail(c, WNW_ERR_HIP, "anchor tier copy failed: %s", hipGetErrorString(e1 != hipSuccess ? e1 : e2));
            }
        }
        // row lists from the keep flags, threaded over heads
        std::vector<uint8_t> bad(nsub, 0);
        parallel_for(nsub, [&](int hi) {
            const bool tidal = hi < g.nT;
            const int lkh = tidal ? c->tidal_lk[hi] : c->fixed_lk[hi - g.nT];
            const HeadRows &hr = c->hrows[hi];
            const int keep = c->head_keep[hi];
            const uint8_t *flags = keep_all + ((size_t)b * nsub + hi) * g.Ta;
            std::vector<int32_t> kept, comp;
            if (!rows_from_flags(g, hr, keep, tidal, flags, kept, comp)) {
                bad[hi] = 1;
                return;
            }
            const int32_t base = (int32_t)((size_t)lkh * g.T);
            int32_t *si = static_idx.data() + (tidal ? 0 : (size_t)g.RsT) + hr.srow;
            for (int i = 0; i < keep; ++i) si[i] = base + kept[i];
            for (int i = 0; i < g.Tt; ++i) si[keep + i] = base + g.Ta + i;
            if (tidal)
                for (int ch = 0; ch < g.nc; ++ch)
                    for (int half = 0; half < 2; ++half)
                        for (int rr = 0; rr < hr.cfull; ++rr) {
                            const int32_t p = comp[(size_t)ch * hr.cfull + rr];
                            // K rows index the K cache (>= 0), V rows are encoded as -(row + 2)
                            comp_idx[(size_t)ch * g.blk_rows + hr.coff + (size_t)half * hr.cfull + rr] =
                                p < 0 ? -1 : (half == 0 ? base + p : -(base + p) - 2);
                        }
        });
        for (int hi = 0; hi < nsub; ++hi)
            if (bad[hi]) {
                cleanup();
                return fail(c, WNW_ERR_HIP, "keep flags of sequence %d, head %d do not match the keep counts", b, hi);
            }
        // static rows of tidal and fixed heads
        hipError_t e = hipMemcpyAsync(d_idx, static_idx.data(), static_idx.size() * sizeof(int32_t), hipMemcpyHostToDevice, st);
        if (e == hipSuccess && g.RsT)
            e = launch_gather_rows(c->tK + (size_t)b * g.RsT * D, fk, fv, d_idx, g.RsT, st);
        if (e == hipSuccess && g.RsT)
            e = launch_gather_rows(c->tV + (size_t)b * g.RsT * D, fv, fv, d_idx, g.RsT, st);
        if (e == hipSuccess && g.RsF)
            e = launch_gather_rows(c->fK + (size_t)b * g.RsF * D, fk, fv, d_idx + (size_t)g.RsT, g.RsF, st);
        if (e == hipSuccess && g.RsF)
            e = launch_gather_rows(c->fV + (size_t)b * g.RsF * D, fv, fv, d_idx + (size_t)g.RsT, g.RsF, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);   // static_idx is rewritten next
        // tidal complement, chunk-major, then to pinned host memory
        if (e == hipSuccess && g.chunk_elems) {
            e = hipMemcpyAsync(d_idx, comp_idx.data(), comp_idx.size() * sizeof(int32_t), hipMemcpyHostToDevice, st);
            if (e == hipSuccess) e = launch_gather_rows(staging, fk, fv, d_idx, (int64_t)comp_idx.size(), st);
            if (e == hipSuccess)
                e = hipMemcpyAsync(c->host_comp + (size_t)b * g.nc * g.chunk_elems, staging,
                                   (size_t)g.nc * g.chunk_elems * sizeof(uint16_t), hipMemcpyDeviceToHost, st);
            if (e == hipSuccess) e = hipStreamSynchronize(st);
        }
        if (e != hipSuccess) {
            cleanup();
            return fail(c, WNW_ERR_HIP, "tier construction failed: %s", hipGetErrorString(e));
        }
    }
    cleanup();

    // ---- selection state -----------------------------------------------------------------------
    std::vector<int32_t> init(B * g.nchk, g.delta);   // never selected: not resident
    if (!init.empty()) HIPCHECK(c, hipMemcpy(s.streak, init.data(), init.size() * sizeof(int32_t), hipMemcpyHostToDevice));
    if (g.nc) HIPCHECK(c, hipMemset(s.slot_of, 0xff, B * g.nc * sizeof(int32_t)));
    if (g.nc) HIPCHECK(c, hipMemset(s.slot_last, 0xff, B * g.nc * sizeof(int32_t)));
    if (g.nc) HIPCHECK(c, hipMemset(s.att, 0, B * g.nc * sizeof(int32_t)));
    if (g.n_slots) {
        HIPCHECK(c, hipMemset(s.slot_data, 0xff, B * g.n_slots * sizeof(int32_t)));
        HIPCHECK(c, hipMemset(s.slot_busy, 0, B * g.n_slots * sizeof(int32_t)));
        HIPCHECK(c, hipMemset(s.slot_since, 0, B * g.n_slots * sizeof(int32_t)));
    }
    HIPCHECK(c, hipMemset(s.step, 0, B * sizeof(int32_t)));
    HIPCHECK(c, hipMemset(s.counts, 0, 2 * B * 2 * sizeof(int32_t)));
    HIPCHECK(c, hipMemset(s.arrive, 0, B * sizeof(int32_t)));
    HIPCHECK(c, hipMemset(s.stats, 0, 8 * sizeof(unsigned long long)));
    HIPCHECK(c, hipDeviceSynchronize());
    c->full_k = c->full_v = nullptr;
    if (g.next_step && (c->cfg.flags & WNW_F_RECALL_MEMCPY)) {
        try {
            c->rthread = std::thread(recall_thread, c);
        } catch (...) {
            return fail(c, WNW_ERR_OOM, "could not start the recall thread");
        }
    }
    c->state = READY;
    return WNW_OK;
}

}  // namespace

extern "C" {

wnw_status wnw_set_roles(wnw_ctx *c, const uint8_t *roles, const float *prefill)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != CREATED) return fail(c, WNW_ERR_STATE, "wnw_set_roles must be called once, right after wnw_init_cache");
    if (!roles || !prefill) return fail(c, WNW_ERR_INVALID, "roles and prefill_scores must not be NULL");
    wnw_status r = assign_roles(c, roles);
    if (r != WNW_OK) return r;
    const Geometry &g = c->g;
    const int nsub = g.nT + g.nF, nh = g.L * g.Hkv;
    const bool global = c->cfg.flags & WNW_F_PREFILL_GLOBAL;
    std::vector<uint8_t> flags((size_t)g.B * nsub * g.Ta), ok((size_t)g.B * nsub, 1);
    parallel_for(g.B * nsub, [&](int i) {
        const int b = i / nsub, hi = i - b * nsub;
        const int lkh = hi < g.nT ? c->tidal_lk[hi] : c->fixed_lk[hi - g.nT];
        ok[i] = keep_flags_host(g, c->hrows[hi], global, prefill + ((size_t)b * nh + lkh) * g.Ta,
                                flags.data() + (size_t)i * g.Ta);
    });
    for (size_t i = 0; i < ok.size(); ++i)
        if (!ok[i]) return fail(c, WNW_ERR_INVALID, "prefill scores of sequence %zu hold NaN", i / nsub);
    r = build_tiers(c, flags.data());
    if (r != WNW_OK) c->state = FAILED;
    return r;
}

wnw_status wnw_set_roles_device(wnw_ctx *c, const uint8_t *roles, const float *prefill_dev)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != CREATED)
        return fail(c, WNW_ERR_STATE, "wnw_set_roles_device must be called once, right after wnw_init_cache");
    if (!roles || !prefill_dev) return fail(c, WNW_ERR_INVALID, "roles and prefill_scores_dev must not be NULL");
    wnw_status r = assign_roles(c, roles);
    if (r != WNW_OK) return r;
    const Geometry &g = c->g;
    const int nsub = g.nT + g.nF;
    DeviceGuard dg(c->device);
    std::vector<uint8_t> flags((size_t)g.B * nsub * g.Ta);
    if (!flags.empty()) {
        // per-segment ranking on the device; the flags come back for the index construction
        std::vector<int32_t> sub_lk(c->tidal_lk);
        sub_lk.insert(sub_lk.end(), c->fixed_lk.begin(), c->fixed_lk.end());
        std::vector<int2> sk(nsub);
        for (int hi = 0; hi < nsub; ++hi) sk[hi] = make_int2(c->hrows[hi].kfull, c->hrows[hi].klast);
        int32_t *d_sub = nullptr;
        int2 *d_sk = nullptr;
        uint8_t *d_flags = nullptr;
        hipError_t e = hipMalloc((void **)&d_sub, nsub * sizeof(int32_t));
        if (e == hipSuccess) e = hipMalloc((void **)&d_sk, nsub * sizeof(int2));
        if (e == hipSuccess) e = hipMalloc((void **)&d_flags, flags.size());
        hipStream_t st = c->setup_stream;
        if (e == hipSuccess) e = hipMemcpyAsync(d_sub, sub_lk.data(), nsub * sizeof(int32_t), hipMemcpyHostToDevice, st);
        if (e == hipSuccess) e = hipMemcpyAsync(d_sk, sk.data(), nsub * sizeof(int2), hipMemcpyHostToDevice, st);
        if (e == hipSuccess)
            e = launch_prefill_keep(g, nsub, d_sub, d_sk, (c->cfg.flags & WNW_F_PREFILL_GLOBAL) != 0, prefill_dev, d_flags,
                                    st);
        if (e == hipSuccess) e = hipMemcpyAsync(flags.data(), d_flags, flags.size(), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        (void)hipFree(d_sub);
        (void)hipFree(d_sk);
        (void)hipFree(d_flags);
        if (e != hipSuccess) {
            c->state = FAILED;
            return fail(c, WNW_ERR_HIP, "device keep selection failed: %s", hipGetErrorString(e));
        }
        // the ranking marks a NaN score with 2
        for (size_t i = 0; i < flags.size(); ++i)
            if (flags[i] > 1) return fail(c, WNW_ERR_INVALID, "prefill scores of sequence %zu hold NaN", i / ((size_t)nsub * g.Ta));
    }
    r = build_tiers(c, flags.data());
    if (r != WNW_OK) c->state = FAILED;
    return r;
}

wnw_status wnw_append_kv(wnw_ctx *c, const void *k_new_dev, const void *v_new_dev, void *hip_stream)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != READY) return fail(c, WNW_ERR_STATE, "wnw_append_kv needs a context after wnw_set_roles");
    if (!k_new_dev || !v_new_dev) return fail(c, WNW_ERR_INVALID, "k_new_dev and v_new_dev must not be NULL");
    if (c->n_gen >= c->g.max_new)
        return fail(c, WNW_ERR_STATE, "all %d rows reserved for appended tokens are used", c->g.max_new);
    DeviceGuard dg(c->device);
    Geometry g = c->g;
    g.n_gen = c->n_gen;
    g.T += c->n_gen;
    HIPCHECK(c, launch_append_kv(g, c->d_hr, c->d_place, c->aK, c->aV, c->tK, c->tV, c->fK, c->fV,
                                 (const uint16_t *)k_new_dev, (const uint16_t *)v_new_dev, (hipStream_t)hip_stream));
    c->n_gen++;
    return WNW_OK;
}

wnw_status wnw_prefill_scores(wnw_ctx *c, const void *q_text_dev, float *scores_dev)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != CREATED) return fail(c, WNW_ERR_STATE, "wnw_prefill_scores needs the full cache: call it before wnw_set_roles");
    const Geometry &g = c->g;
    if (!scores_dev || (g.Tt > 0 && !q_text_dev))
        return fail(c, WNW_ERR_INVALID, "scores_dev (and q_text_dev when text_len > 0) must not be NULL");
    DeviceGuard dg(c->device);
    float *stats = nullptr;
    const size_t ns = (size_t)g.B * g.L * g.Hq * g.Tt;
    if (ns) {
        hipError_t e = hipMalloc((void **)&stats, ns * sizeof(float));
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(c, e == hipErrorOutOfMemory ? WNW_ERR_OOM : WNW_ERR_HIP, "prefill statistics: %s", hipGetErrorString(e));
        }
    }
    hipStream_t st = c->setup_stream;
    hipError_t e = launch_prefill_scores(g, c->full_k, (const uint16_t *)q_text_dev, stats, scores_dev, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (stats) (void)hipFree(stats);
    if (e != hipSuccess) return fail(c, WNW_ERR_HIP, "prefill scores failed: %s", hipGetErrorString(e));
    return WNW_OK;
}

wnw_status wnw_prefill_scores_static(wnw_ctx *c, const void *q_text_dev, float *scores_dev, void *hip_stream)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != CREATED)
        return fail(c, WNW_ERR_STATE, "wnw_prefill_scores_static needs the full cache: call it before wnw_set_roles");
    const Geometry &g = c->g;
    if (!scores_dev || (g.Tt > 0 && !q_text_dev))
        return fail(c, WNW_ERR_INVALID, "scores_dev (and q_text_dev when text_len > 0) must not be NULL");
    const size_t ns = (size_t)g.B * g.L * g.Hq * g.Tt;
    if (ns > STATIC_PREFILL_ROWS)
        return fail(c, WNW_ERR_UNSUPPORTED,
                    "batch * layers * q_heads * text_len = %zu statistics rows exceed the static buffer's %zu "
                    "(use wnw_prefill_scores)", ns, STATIC_PREFILL_ROWS);
    DeviceGuard dg(c->device);
    float *stats = scratch_on_device(c->device);
    if (!stats) return fail(c, WNW_ERR_HIP, "%s", t_err.c_str());
    const hipError_t e = launch_prefill_scores(g, c->full_k, (const uint16_t *)q_text_dev, stats, scores_dev,
                                               (hipStream_t)hip_stream);
    if (e != hipSuccess) return fail(c, WNW_ERR_HIP, "prefill scores failed: %s", hipGetErrorString(e));
    return WNW_OK;
}

wnw_status wnw_decode_step(wnw_ctx *c, const void *q_dev, void *out, float *scores, int32_t *selected, void *hip_stream)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != READY)
        return fail(c, WNW_ERR_STATE, c->state == FAILED ? "context is in the error state: %s" : "%s",
                    c->state == FAILED ? c->err.c_str() : "wnw_set_roles has not run");
    if (!q_dev || !out) return fail(c, WNW_ERR_INVALID, "q_dev and out_dev must not be NULL");
    {
        wnw_status r = check_exhaustion(c);
        if (r != WNW_OK) return r;
        std::lock_guard<std::mutex> lk(c->rmu);
        if (c->rerr != hipSuccess) {
            c->state = FAILED;
            return fail(c, WNW_ERR_HIP, "recall thread: %s", c->rerr_msg.c_str());
        }
    }
    DeviceGuard dg(c->device);
    // this step's geometry: the prompt rows plus the tokens appended so far
    Geometry g = c->g;
    g.n_gen = c->n_gen;
    g.T += c->n_gen;
    g.n_tiles_a = (g.T + TILE_A - 1) / TILE_A;
    hipStream_t s0 = (hipStream_t)hip_stream;
    const uint16_t *q = (const uint16_t *)q_dev;
    float *sc = scores ? scores : c->scores_int;
    int32_t *sel = selected ? selected : c->sel_int;
    const bool timing = c->cfg.flags & WNW_F_TIMING;
    StepEvents ev{};
    if (timing) {
        if (!c->spare.empty()) {
            ev = c->spare.back();
            c->spare.pop_back();
        } else {
            // timing only: no system-scope fence (cache write-back and invalidation) on record,
            // which would slow the kernels that follow and blur the measurement
            for (auto &e : ev.e) HIPCHECK(c, hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
            for (auto &e : ev.r) HIPCHECK(c, hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
            for (auto &e : ev.rc) HIPCHECK(c, hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
        }
        ev.split = false;
        ev.has_new = false;
    }
#define MARK(i) \
    if (timing) HIPCHECK(c, hipEventRecord(ev.e[i], s0))

    // Lists (kept, new and their counts) alternate between two buffers by step.
    // Same-step timing: the selection of step s fills buffer s & 1 and step s reads it.
    // Next-step timing: the selection of step s fills buffer (s + 1) & 1 for step s + 1, and
    // step s reads buffer s & 1, filled by step s - 1: its tidal launch streams the kept list,
    // which then holds every resident complement (those on the device before step s - 1's
    // recall, then those step s - 1 recalled, once their copies have landed).  Neither select
    // kernel ever rewrites a list a launch or a recall still reads.  (The complements already
    // on the device could join the attention launch, which runs before the wait for the copies;
    // measured, that launch then streams slower than the two launches apart.)
    const int par = (int)(c->steps & 1), nxt = (int)((c->steps + 1) & 1);
    auto lists_of = [&](StepBuffers b, int i) {
        b.counts += (size_t)i * g.B * 2;
        b.new_list += (size_t)i * g.B * g.knew * 2;
        b.kept_list += (size_t)i * g.B * g.n_slots * 2;
        b.arrive = nullptr;
        return b;
    };
    StepBuffers sb = lists_of(c->s, par);                         // what this step reads
    StepBuffers sn = g.next_step ? lists_of(c->s, nxt) : sb;      // what its selection writes

    // (1) anchor attention + chunk mass, (2) scores, top-k and residency.  With next-step
    // timing the static tidal/fixed tiles (kept rows + text) join the anchor launch.
    // markers 0 and 1 are the first launch's own start and end (its dispatch excluded)
    hipEvent_t e0 = timing ? ev.e[0] : nullptr, e1 = timing ? ev.e[1] : nullptr;
    const bool memcpy_path = c->cfg.flags & WNW_F_RECALL_MEMCPY;
    // host-issued copies: the selection also writes the counts and new lists to mapped pinned
    // memory (one mirror per step parity) and then publishes a tag there, so the host reads them
    // once the selection is done, never behind copies still running on the side streams
    sn.pub = memcpy_path ? c->d_newinfo + (size_t)par * c->mirror_ints : nullptr;
    sn.pub_tag = pub_tag(c->steps);
    if (g.next_step)
        HIPCHECK(c, launch_attention(g, c->t, sb, q, s0, e0, e1));
    else
        HIPCHECK(c, launch_anchor(g, c->t, sb, q, s0, e0, e1));
    // Next-step timing with host-issued copies: the chunk-mass merge and the selection run inside
    // the tidal/fixed launch (its first work-groups, beside the slot items) when the previous
    // step recalled little.  That launch waits for the previous step's copies, and so would the
    // selection; a small recall has landed by then (SEL_IN_TIDAL_BYTES), while a large one keeps
    // the selection ahead of the wait, so that this step's copies queue behind the previous
    // step's and the link stays busy.  The host reads the previous step's recall size from its
    // mirror once the recall thread has issued it (the attention launch runs meanwhile).
    bool sel_in_tidal = false;
    if (g.next_step && memcpy_path && tidal_select_fits(g)) {
        int64_t prev_bytes = 0;
        if (c->rec_pending) {
            wnw_status r = recall_wait_issued(c, (int64_t)c->steps - 1);
            if (r != WNW_OK) return r;
            const int32_t *cnt = c->h_newinfo + (size_t)nxt * c->mirror_ints;
            for (int b = 0; b < g.B; ++b) prev_bytes += (int64_t)cnt[b * 2 + 1] * g.chunk_elems * (int64_t)sizeof(uint16_t);
        }
        sel_in_tidal = prev_bytes <= SEL_IN_TIDAL_BYTES;
    }
    c->sel_in_tidal += sel_in_tidal ? 1 : 0;
    if (!sel_in_tidal) {
        HIPCHECK(c, launch_anchor_mass(g, sb, s0));
        HIPCHECK(c, launch_select(g, sn, sc, c->override_sel, sel, s0));
    }
    MARK(6);
    // the copy kernel of the next-step recall follows the selection on the device (an event; the
    // host-issued copies follow the published tag instead)
    if (g.next_step && !memcpy_path) HIPCHECK(c, hipEventRecord(c->ev_sel[par], s0));
    bool combined = false;
    if (g.next_step) {
        // Next-step timing: the chunks that became resident now are copied on the side stream
        // (host-issued: by the recall thread, over the copy streams, of which the side stream is
        // the first), back to back with the previous step's copies.  The target slots were free
        // at this step's selection, which follows on s0 every reader of them (up to the previous
        // step's last tidal launch; a slot dropped now stays busy until the next selection, since
        // this step's last launch may still read it).
        if (!memcpy_path) {
            HIPCHECK(c, hipStreamWaitEvent(c->side, c->ev_sel[par], 0));
            if (timing) HIPCHECK(c, hipEventRecord(ev.r[0], c->side));
            if (c->delay_us > 0) HIPCHECK(c, hipLaunchHostFunc(c->side, delay_fn, &c->delay_us));
            HIPCHECK(c, launch_recall(g, c->t, sn, c->side));
        }
        // this step's last tidal launch reads the complements the previous step recalled
        if (c->rec_pending) {
            if (memcpy_path) {
                wnw_status r = recall_wait_issued(c, (int64_t)c->steps - 1);
                if (r == WNW_OK) r = wait_copies(c, nxt, s0);
                if (r != WNW_OK) return r;
            } else {
                HIPCHECK(c, hipStreamWaitEvent(s0, c->ev_rec, 0));
            }
        }
        // with host-issued copies the host has read the previous step's mirror (its copies are
        // issued), so it knows the length of the list this launch streams
        long long items = -1;
        if (memcpy_path && c->rec_pending) {
            const int32_t *cnt = c->h_newinfo + (size_t)nxt * c->mirror_ints;
            int nmax = 0;
            for (int b = 0; b < g.B; ++b) nmax = std::max(nmax, cnt[b * 2]);
            items = ((long long)nmax * g.comp_max + TILE_S - 1) / TILE_S;
        }
        // markers 2 and 3: the launch's own start and end
        SelectArgs sa{};
        if (sel_in_tidal) {
            sa.s = sn;
            sa.s.arrive = c->s.arrive;
            sa.scores = sc;
            sa.ovr = c->override_sel;
            sa.selected = sel;
        }
        HIPCHECK(c, launch_tidal_fixed(g, c->t, sb, q, false, false, items, s0, timing ? ev.e[2] : nullptr,
                                       timing ? ev.e[3] : nullptr, sel_in_tidal ? &sa : nullptr));
        // the final merge is queued before the host waits for the selection below, so that the
        // device never idles behind that wait
        HIPCHECK(c, launch_subset_combine(g, c->t, sb, out, s0));
        MARK(5);
        combined = true;
        if (memcpy_path && g.nc > 0) {
            // the recall thread issues this step's copies once its selection is done; the copy
            // engines queue them behind the previous step's copies, so the link stays busy
            wnw_ctx::RecallJob job{(int64_t)c->steps, s0, timing, timing ? ev.r[0] : nullptr, {}};
            if (timing)
                for (int i = 0; i < N_COPY_STREAMS; ++i) job.rc[i] = ev.rc[i];
            ev.split = timing;
            {
                std::lock_guard<std::mutex> lk(c->rmu);
                c->rjobs.push_back(job);
            }
            c->rcv.notify_all();
        }
        if (!memcpy_path) {
            if (timing) HIPCHECK(c, hipEventRecord(ev.r[1], c->side));
            HIPCHECK(c, hipEventRecord(c->ev_rec, c->side));   // host-issued copies: ev_copy[] instead
        } else if (g.nc == 0 && timing) {
            // no recall: an empty interval on the side stream
            HIPCHECK(c, hipEventRecord(ev.r[0], c->side));
            HIPCHECK(c, hipEventRecord(ev.r[1], c->side));
        }
        // with no chunks (no audio) no selection runs, and the recall thread gets no job
        c->rec_pending = !memcpy_path || g.nc > 0;
    } else if (!memcpy_path) {
        MARK(2);
        // (3) + (4) in one launch: its first work-groups copy the complements listed for recall
        // from mapped pinned memory into their slots and attend to them, the others run the fixed
        // heads and the tidal rows already on the device.  The slots being written were freed by
        // this step's select kernel; every kernel that could still read them (the previous
        // step's) precedes it on this stream.
        if (timing) HIPCHECK(c, hipEventRecord(ev.r[0], s0));
        HIPCHECK(c, launch_tidal_fixed(g, c->t, sb, q, true, true, -1, s0));
        if (timing) HIPCHECK(c, hipEventRecord(ev.r[1], s0));
        MARK(3);
    } else {
        MARK(2);
        // (4a) device-resident rows while the host waits for the selection and issues the copies
        HIPCHECK(c, launch_tidal_fixed(g, c->t, sb, q, false, true, -1, s0));
        MARK(3);
        // (3) copies on the side stream.  The target slots were freed by this step's select
        // kernel, which follows every earlier reader on s0: once it has published its tag, no
        // reader of them is left and the copies need no device-side wait.
        wnw_status r = WNW_OK;
        if (g.nc > 0) {
            const auto w0 = std::chrono::steady_clock::now();
            HIPCHECK(c, wait_published(c, (int64_t)c->steps, s0));
            c->host_wait_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - w0).count();
            if (timing) HIPCHECK(c, hipEventRecord(ev.r[0], c->side));
            r = check_exhaustion(c);
            if (r != WNW_OK) return r;
            r = issue_copies(c, par, c->side);
            if (r != WNW_OK) return r;
        } else {
            // no chunks (no audio): no selection ran, so no tag comes, and nothing is recalled
            c->copy_mask[par] = 0;
            if (timing) HIPCHECK(c, hipEventRecord(ev.r[0], c->side));
        }
        if (timing) {
            r = wait_copies(c, par, c->side);
            if (r != WNW_OK) return r;
            HIPCHECK(c, hipEventRecord(ev.r[1], c->side));
        }
        r = wait_copies(c, par, s0);
        if (r != WNW_OK) return r;
        // (4b) the complements copied this step
        HIPCHECK(c, launch_new_slots(g, c->t, sb, q, s0));
        MARK(4);
        ev.has_new = timing;
    }
    if (!combined) {
        HIPCHECK(c, launch_subset_combine(g, c->t, sb, out, s0));
        MARK(5);
    }
#undef MARK
    if (timing) c->pending.push_back(ev);
    if (c->log) {
        // host-side trace: what this call enqueued and, with host-issued copies, what it copied
        int n_new = -1;
        if (memcpy_path && !g.next_step)
            for (int b = n_new = 0; b < g.B; ++b) n_new += c->h_newinfo[par * c->mirror_ints + b * 2 + 1];
        fprintf(stderr, "[wnw] step %lld: %s timing, %s recall, %d sequences, new segments copied %d, host wait %.3f ms "
                        "total, selection %s\n",
                (long long)c->steps, g.next_step ? "next-step" : "same-step",
                memcpy_path ? "copy-engine" : "work-group", g.B, n_new, c->host_wait_ms,
                sel_in_tidal ? "inside the tidal launch" : "before the tidal launch");
    }
    c->steps++;
    return WNW_OK;
}

wnw_status wnw_query_geometry(const wnw_ctx *c, int32_t *n_chunks, int32_t *k, int32_t *keep_total, int32_t *n_slots,
                              int64_t *chunk_bytes)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (n_chunks) *n_chunks = c->g.nchk;
    if (k) *k = c->g.k;
    if (keep_total) *keep_total = c->importance.empty() ? c->g.keep_total : -1;
    if (n_slots) *n_slots = c->g.n_slots;
    if (chunk_bytes) {
        if (c->state == CREATED) return fail(const_cast<wnw_ctx *>(c), WNW_ERR_STATE, "chunk size is known after wnw_set_roles");
        *chunk_bytes = c->g.chunk_elems * (int64_t)sizeof(uint16_t);
    }
    return WNW_OK;
}

wnw_status wnw_set_retention(wnw_ctx *c, const float *importance, float lambda)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (c->state != CREATED) return fail(c, WNW_ERR_STATE, "wnw_set_retention must come before wnw_set_roles");
    const size_t nh = (size_t)c->g.L * c->g.Hkv;
    if (!importance) {
        c->importance.clear();
        return WNW_OK;
    }
    if (!(lambda >= 0.f) || std::isinf(lambda)) return fail(c, WNW_ERR_INVALID, "lambda must be finite and >= 0");
    for (size_t i = 0; i < nh; ++i)
        if (!(importance[i] >= 0.f && importance[i] <= 1.f))
            return fail(c, WNW_ERR_INVALID, "importance of head %zu is not in [0, 1]", i);
    c->importance.assign(importance, importance + nh);
    c->lambda = lambda;
    return WNW_OK;
}

wnw_status wnw_query_head_keep(const wnw_ctx *c, int32_t *keep)
{
    if (!c || !keep) return fail(const_cast<wnw_ctx *>(c), WNW_ERR_INVALID, "ctx and keep must not be NULL");
    if (c->state == CREATED) return fail(const_cast<wnw_ctx *>(c), WNW_ERR_STATE, "keep counts are known after wnw_set_roles");
    const Geometry &g = c->g;
    for (int a : c->anchor_lk) keep[a] = g.Ta;
    for (int i = 0; i < g.nT; ++i) keep[c->tidal_lk[i]] = c->head_keep[i];
    for (int i = 0; i < g.nF; ++i) keep[c->fixed_lk[i]] = c->head_keep[g.nT + i];
    return WNW_OK;
}

wnw_status wnw_query_segments(const wnw_ctx *c, int32_t *n_segments)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (n_segments) *n_segments = c->g.nc;
    return WNW_OK;
}

wnw_status wnw_get_stats(wnw_ctx *c, wnw_stats *o)
{
    if (!c || !o) return fail(c, WNW_ERR_INVALID, "ctx and out must not be NULL");
    if (c->state != READY) return fail(c, WNW_ERR_STATE, "context not ready");
    DeviceGuard dg(c->device);
    wnw_status r = recall_wait_issued(c, -1);
    if (r != WNW_OK) return r;
    HIPCHECK(c, hipDeviceSynchronize());
    r = harvest_timing(c);
    if (r != WNW_OK) return r;
    unsigned long long st[8];
    HIPCHECK(c, hipMemcpy(st, c->s.stats, sizeof st, hipMemcpyDeviceToHost));
    if (st[5]) {
        c->state = FAILED;
        return fail(c, WNW_ERR_STATE, "%llu decode step(s) found no free recall slot (slot pool of %d per sequence)",
                    st[5], c->g.n_slots);
    }
    const Geometry &g = c->g;
    *o = wnw_stats{};
    o->steps = c->steps;
    o->recalled_chunks = (int64_t)st[0];
    o->recalled_bytes = (int64_t)st[0] * g.chunk_elems * (int64_t)sizeof(uint16_t);
    o->dropped_chunks = (int64_t)st[1];
    o->resident_chunks = (int64_t)st[2];
    o->peak_resident = (int32_t)st[4];
    o->n_slots = g.n_slots;
    o->slot_rows = (int64_t)st[3];
    const double full = (double)g.L * g.Hkv * g.Ta;
    const double res_rows = c->steps ? (double)st[3] / ((double)c->steps * g.B) : 0.0;
    if (full > 0) {
        // slot_rows sums the attended complement rows over the tidal heads
        o->r_gpu = ((double)g.nA * g.Ta + (double)g.keep_sum + res_rows) / full;
        o->r_gpu_cpu = o->r_gpu + ((double)g.nT * g.Ta - (double)c->keep_sum_t) / full;
    }
    o->anchor_bytes = (int64_t)g.B * g.nA * (g.T + c->n_gen) * 2 * D * 2;
    o->static_bytes = (int64_t)g.B * (c->static_rows + (int64_t)c->n_gen * (g.nT + g.nF)) * 2 * D * 2;
    o->revived_chunks = (int64_t)st[6];
    o->timed_steps = c->timed_steps;
    o->t_anchor_ms = c->t_acc[0];
    o->t_select_ms = c->t_acc[1];
    o->t_tidal_fixed_ms = c->t_acc[2];
    o->t_new_ms = c->t_acc[3];
    o->t_combine_ms = c->t_acc[4];
    o->t_step_ms = c->t_acc[5];
    o->t_recall_ms = c->t_acc[6];
    o->slot_exhausted = (int64_t)st[5];
    {
        std::lock_guard<std::mutex> lk(c->rmu);
        o->t_host_wait_ms = c->host_wait_ms;
    }
    o->t_recall_wait_ms = c->t_acc[7];
    o->kept_rows = (int64_t)st[7];
    o->selections_in_tidal = c->sel_in_tidal;
    return WNW_OK;
}

wnw_status wnw_set_selection_override(wnw_ctx *c, const int32_t *sel_dev)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    c->override_sel = sel_dev;
    return WNW_OK;
}

wnw_status wnw_debug_set_recall_delay(wnw_ctx *c, int32_t us)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (us < 0 || us > 1000000) return fail(c, WNW_ERR_INVALID, "recall delay must be in 0..1000000 us");
    wnw_status r = recall_wait_issued(c, -1);   // no recall in flight reads the old value
    if (r != WNW_OK) return r;
    c->delay_us = us;
    return WNW_OK;
}

wnw_status wnw_debug_set_slot_offset_limit(wnw_ctx *c, int64_t bytes)
{
    if (!c) return fail(nullptr, WNW_ERR_INVALID, "ctx is NULL");
    if (bytes < 0) return fail(c, WNW_ERR_INVALID, "slot offset limit must be >= 0");
    c->g.slot_off_max = std::min<int64_t>(bytes, 0xffffffffll);
    return WNW_OK;
}

wnw_status wnw_debug_read_slot(wnw_ctx *c, int32_t b, int32_t chunk, void *dst, size_t bytes)
{
    if (!c || !dst) return fail(c, WNW_ERR_INVALID, "ctx and host_dst must not be NULL");
    if (c->state != READY) return fail(c, WNW_ERR_STATE, "context not ready");
    const Geometry &g = c->g;
    if (b < 0 || b >= g.B || chunk < 0 || chunk >= g.nc) return fail(c, WNW_ERR_INVALID, "(b, segment) out of range");
    if (bytes != (size_t)g.chunk_elems * sizeof(uint16_t)) return fail(c, WNW_ERR_INVALID, "bytes must equal chunk_bytes");
    DeviceGuard dg(c->device);
    wnw_status r = recall_wait_issued(c, -1);
    if (r != WNW_OK) return r;
    HIPCHECK(c, hipDeviceSynchronize());
    int32_t slot = -1;
    HIPCHECK(c, hipMemcpy(&slot, c->s.slot_of + (size_t)b * g.nc + chunk, sizeof slot, hipMemcpyDeviceToHost));
    if (slot < 0) return fail(c, WNW_ERR_INVALID, "chunk %d of sequence %d is not resident", chunk, b);
    HIPCHECK(c, hipMemcpy(dst, c->slots + ((size_t)b * g.n_slots + slot) * g.chunk_elems, bytes, hipMemcpyDeviceToHost));
    return WNW_OK;
}

wnw_status wnw_debug_read_host_chunk(wnw_ctx *c, int32_t b, int32_t chunk, void *dst, size_t bytes)
{
    if (!c || !dst) return fail(c, WNW_ERR_INVALID, "ctx and host_dst must not be NULL");
    if (c->state != READY) return fail(c, WNW_ERR_STATE, "context not ready");
    const Geometry &g = c->g;
    if (b < 0 || b >= g.B || chunk < 0 || chunk >= g.nc) return fail(c, WNW_ERR_INVALID, "(b, segment) out of range");
    if (bytes != (size_t)g.chunk_elems * sizeof(uint16_t)) return fail(c, WNW_ERR_INVALID, "bytes must equal chunk_bytes");
    if (bytes) memcpy(dst, c->host_comp + ((size_t)b * g.nc + chunk) * g.chunk_elems, bytes);
    return WNW_OK;
}

wnw_status wnw_debug_read_resident(wnw_ctx *c, uint8_t *dst)
{
    if (!c || !dst) return fail(c, WNW_ERR_INVALID, "ctx and host_dst must not be NULL");
    if (c->state != READY) return fail(c, WNW_ERR_STATE, "context not ready");
    const Geometry &g = c->g;
    DeviceGuard dg(c->device);
    wnw_status r = recall_wait_issued(c, -1);
    if (r != WNW_OK) return r;
    HIPCHECK(c, hipDeviceSynchronize());
    std::vector<int32_t> att((size_t)g.B * g.nc);
    if (!att.empty()) HIPCHECK(c, hipMemcpy(att.data(), c->s.att, att.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
    for (size_t i = 0; i < att.size(); ++i) dst[i] = att[i] != 0;
    return WNW_OK;
}

void wnw_destroy(wnw_ctx *c)
{
    if (!c) return;
    DeviceGuard dg(c->device);
    recall_stop(c);   // issues every queued recall first
    (void)hipDeviceSynchronize();
    free_all(c);
    delete c;
}

}  // extern "C"
