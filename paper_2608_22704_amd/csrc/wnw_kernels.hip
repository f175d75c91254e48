// HIP kernels of the WnW decode step for CDNA4 (gfx950).
//
// Work decomposition (all kernels are launched by wnw_api.hip on the caller's stream, the
// recall on a side stream):
//   anchor_attn     one work-group per (sequence, anchor KV-head, tile of TILE key rows): the
//                   g q-heads' logits, the tile max, exp, the per-chunk softmax mass (Eq. 2) and
//                   the unnormalised P.V partial.  Logits and masses are kept in double: the
//                   chunk ranking must agree with an fp64 reference to well under 1e-6.
//   anchor_combine  log-sum-exp merge of the tiles of one anchor head -> its outputs and its
//                   normalised chunk masses.
//   scores          per chunk: fixed-order sum over anchor q-heads / chunk length (mean).
//   select          one work-group per sequence: top-k by (score desc, id asc), streaks,
//                   residency, slot assignment, kept/new lists.
//   recall          copies newly resident complements from mapped pinned host memory.
//   subset_static   tidal and fixed heads over their kept rows + text (fp32 logits).
//   subset_slots    tidal heads over resident complements (kept list, then new list).
//   subset_combine  merge of a tidal/fixed head's partials.
//
// Layout inside a tile: 16 lanes share one 256-byte key row (8 bf16 = 16 bytes each), so one
// wavefront load moves 4 rows (1 KiB) fully coalesced; a work-group of 4 wavefronts covers 256
// rows in 16 steps.  Dot products are reduced across the 16 lanes with cross-lane shuffles.
#include "wnw_internal.h"

#include <math.h>

namespace wnw {

namespace {

constexpr int WAVES = NT / 64;
constexpr int ROWS_PER_WAVE = TILE / WAVES;   // 64
constexpr int STEPS = ROWS_PER_WAVE / 4;      // 16 steps of 4 rows
constexpr double SCALE_D = 0.088388347648318440550;   // 1 / sqrt(128)
constexpr float SCALE_F = 0.08838834764831845f;

__device__ inline void unpack8(const uint4 u, float f[8])
{
    f[0] = __uint_as_float(u.x << 16); f[1] = __uint_as_float(u.x & 0xffff0000u);
    f[2] = __uint_as_float(u.y << 16); f[3] = __uint_as_float(u.y & 0xffff0000u);
    f[4] = __uint_as_float(u.z << 16); f[5] = __uint_as_float(u.z & 0xffff0000u);
    f[6] = __uint_as_float(u.w << 16); f[7] = __uint_as_float(u.w & 0xffff0000u);
}

template <typename T>
__device__ inline T sum16(T v)
{
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

template <typename T>
__device__ inline T wave_max(T v)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

template <typename T>
__device__ inline T wave_sum(T v)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

// Block-wide max / sum of G values per thread (NT threads).  red: [WAVES][G] shared.
template <int G, typename T>
__device__ inline void block_max(T v[G], T *red)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int h = 0; h < G; ++h) v[h] = wave_max(v[h]);
    if (lane == 0)
#pragma unroll
        for (int h = 0; h < G; ++h) red[wave * G + h] = v[h];
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
        T m = red[h];
        for (int w = 1; w < WAVES; ++w) m = fmax(m, red[w * G + h]);
        v[h] = m;
    }
    __syncthreads();
}

template <int G, typename T>
__device__ inline void block_sum(T v[G], T *red)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int h = 0; h < G; ++h) v[h] = wave_sum(v[h]);
    if (lane == 0)
#pragma unroll
        for (int h = 0; h < G; ++h) red[wave * G + h] = v[h];
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
        T m = red[h];
        for (int w = 1; w < WAVES; ++w) m += red[w * G + h];
        v[h] = m;
    }
    __syncthreads();
}

// -------------------------------------------------------------------------------------------
// Anchor attention + chunk mass (double logits)
// -------------------------------------------------------------------------------------------
template <int G>
__global__ __launch_bounds__(NT) void anchor_attn_kernel(Geometry g, Tiers t, StepBuffers s,
                                                         const uint16_t *__restrict__ q)
{
    const int tile = blockIdx.x, ai = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, sub = lane & 15, rg = lane >> 4;
    const int lk = t.anchor_lk[ai], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const size_t hrow = ((size_t)b * g.nA + ai) * (size_t)g.T;
    const uint16_t *__restrict__ K = t.aK + hrow * D;
    const uint16_t *__restrict__ V = t.aV + hrow * D;
    const uint16_t *__restrict__ qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;

    __shared__ double xs[G * TILE];      // logits -> probabilities -> (as float) wave partials
    __shared__ double red[WAVES * G];

    double qd[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        float f[8];
        unpack8(*(const uint4 *)(qh + h * D + sub * 8), f);
#pragma unroll
        for (int e = 0; e < 8; ++e) qd[h][e] = (double)f[e];
    }

    const int t0 = tile * TILE;
    // Pass 1: x = q.k / sqrt(d), exact products, double accumulation.
    for (int i0 = 0; i0 < STEPS; i0 += 4) {
        uint4 kr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int row = t0 + wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            kr[u] = row < g.T ? *(const uint4 *)(K + (size_t)row * D + sub * 8) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            float f[8];
            unpack8(kr[u], f);
            double acc[G];
#pragma unroll
            for (int h = 0; h < G; ++h) {
                acc[h] = 0.0;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h] = fma(qd[h][e], (double)f[e], acc[h]);
                acc[h] = sum16(acc[h]);
            }
            if (sub == 0) {
                const bool ok = t0 + r < g.T;
#pragma unroll
                for (int h = 0; h < G; ++h) xs[h * TILE + r] = ok ? acc[h] * SCALE_D : -INFINITY;
            }
        }
    }
    __syncthreads();

    // Tile max, probabilities relative to it, and their sum.
    double m[G], p[G];
#pragma unroll
    for (int h = 0; h < G; ++h) m[h] = xs[h * TILE + tid];
    block_max<G>(m, red);
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const double x = xs[h * TILE + tid];
        p[h] = (m[h] == -INFINITY) ? 0.0 : exp(x - m[h]);
        xs[h * TILE + tid] = p[h];
    }
    block_sum<G>(p, red);     // p[h] now holds the tile sum l; also a barrier for xs

    const size_t pidx = ((size_t)b * g.nA + ai) * g.n_tiles_a + tile;
    if (tid == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            s.pa_m[pidx * G + h] = m[h];
            s.pa_l[pidx * G + h] = p[h];
        }
    }
    // Per-chunk mass of this tile (Eq. 2 restricted to the tile), fixed summation order.
    const int c_first = t0 / g.cl;
    for (int idx = tid; idx < G * g.maxc; idx += NT) {
        const int h = idx / g.maxc, c = c_first + (idx - h * g.maxc);
        const int r0 = max(c * g.cl, t0), r1 = min(min((c + 1) * g.cl, t0 + TILE), g.Ta);
        double acc = 0.0;
        for (int r = r0; r < r1; ++r) acc += xs[h * TILE + (r - t0)];
        s.pa_mass[pidx * G * g.maxc + idx] = acc;
    }

    // Pass 2: unnormalised P.V in fp32.
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    for (int i0 = 0; i0 < STEPS; i0 += 4) {
        uint4 vr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int row = t0 + wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            vr[u] = row < g.T ? *(const uint4 *)(V + (size_t)row * D + sub * 8) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            float f[8];
            unpack8(vr[u], f);
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float ph = (float)xs[h * TILE + r];
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(ph, f[e], acc[h][e]);
            }
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[h][e] += __shfl_xor(acc[h][e], 16);
            acc[h][e] += __shfl_xor(acc[h][e], 32);
        }
    __syncthreads();                     // every read of xs is done
    float *ored = (float *)xs;           // [WAVES][G][D]
    if (rg == 0)
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) ored[(wave * G + h) * D + sub * 8 + e] = acc[h][e];
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += NT) {
        float o = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) o += ored[w * G * D + idx];
        s.pa_o[pidx * G * D + idx] = o;
    }
}

template <int G>
__global__ __launch_bounds__(NT) void anchor_combine_kernel(Geometry g, Tiers t, StepBuffers s, float *out)
{
    const int ai = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    extern __shared__ double fac[];      // [n_tiles_a][G]
    __shared__ double Mh[G], Lh[G];
    const size_t base = ((size_t)b * g.nA + ai) * g.n_tiles_a;
    const int nt = g.n_tiles_a;
    if (tid < G) {
        double M = -INFINITY;
        for (int i = 0; i < nt; ++i) M = fmax(M, s.pa_m[(base + i) * G + tid]);
        double L = 0.0;
        if (M > -INFINITY)
            for (int i = 0; i < nt; ++i) {
                const double mi = s.pa_m[(base + i) * G + tid];
                if (mi > -INFINITY) L += s.pa_l[(base + i) * G + tid] * exp(mi - M);
            }
        Mh[tid] = M;
        Lh[tid] = L;
    }
    __syncthreads();
    for (int idx = tid; idx < nt * G; idx += NT) {
        const int h = idx % G;
        const double mi = s.pa_m[base * G + idx];
        fac[idx] = (Lh[h] > 0.0 && mi > -INFINITY) ? exp(mi - Mh[h]) / Lh[h] : 0.0;
    }
    __syncthreads();
    const int lk = t.anchor_lk[ai], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    float *oh = out + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    for (int idx = tid; idx < G * D; idx += NT) {
        const int h = idx / D;
        double acc = 0.0;
        for (int i = 0; i < nt; ++i) acc += (double)s.pa_o[(base + i) * G * D + idx] * fac[i * G + h];
        oh[idx] = (float)acc;
    }
    double *mass = s.mass + ((size_t)b * g.nA + ai) * G * (size_t)g.nc;
    for (int idx = tid; idx < G * g.nc; idx += NT) {
        const int h = idx / g.nc, c = idx - h * g.nc;
        const int t_lo = (c * g.cl) / TILE, t_hi = (min((c + 1) * g.cl, g.Ta) - 1) / TILE;
        double acc = 0.0;
        for (int i = t_lo; i <= t_hi; ++i) {
            const int j = c - (i * TILE) / g.cl;
            acc += s.pa_mass[((base + i) * G + h) * g.maxc + j] * fac[i * G + h];
        }
        mass[idx] = acc;
    }
}

__global__ void scores_kernel(Geometry g, StepBuffers s, float *scores)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= g.B * g.nc) return;
    const int b = i / g.nc, c = i - b * g.nc, naq = g.nA * g.G;
    const double *m = s.mass + (size_t)b * naq * g.nc + c;
    double acc = 0.0;
    for (int a = 0; a < naq; ++a) acc += m[(size_t)a * g.nc];
    scores[i] = (float)(acc / (double)chunk_len_of(g, c));
}

// -------------------------------------------------------------------------------------------
// Selection, residency and slot bookkeeping: one work-group per sequence.
// -------------------------------------------------------------------------------------------
__device__ int block_scan_excl(int *a, int n, int *wsum)
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
    int carry = 0;
    for (int base = 0; base < n; base += blockDim.x) {
        const int i = base + tid;
        const int v = i < n ? a[i] : 0;
        int x = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (lane == 63) wsum[wave] = x;
        __syncthreads();
        if (tid == 0) {
            int acc = 0;
            for (int w = 0; w < nw; ++w) {
                const int tt = wsum[w];
                wsum[w] = acc;
                acc += tt;
            }
            wsum[nw] = acc;
        }
        __syncthreads();
        if (i < n) a[i] = carry + wsum[wave] + x - v;
        carry += wsum[nw];
        __syncthreads();
    }
    return carry;
}

__global__ __launch_bounds__(SEL_THREADS) void select_kernel(Geometry g, StepBuffers s, const float *__restrict__ scores,
                                                             const int32_t *__restrict__ ovr, int32_t *__restrict__ selected)
{
    const int b = blockIdx.x, tid = threadIdx.x, nthr = blockDim.x;
    const int nc = g.nc, k = g.k, ns = g.n_slots;
    extern __shared__ int smem[];
    float *sc = (float *)smem;           // [nc]
    int *fsel = smem + nc;               // [nc] selected flag
    int *fnew = fsel + nc;               // [nc] newly resident flag
    int *fkept = fnew + nc;              // [nc] resident before and now
    int *rank = fkept + nc;              // [nc] scan scratch
    int *ffree = rank + nc;              // [ns] free slot flag
    int *freelist = ffree + ns;          // [ns] free slots ascending
    __shared__ int wsum[SEL_THREADS / 64 + 1];
    __shared__ int ndrop, nrows;

    for (int c = tid; c < nc; c += nthr) {
        sc[c] = scores[(size_t)b * nc + c];
        fsel[c] = 0;
    }
    if (tid == 0) ndrop = nrows = 0;
    __syncthreads();
    if (ovr) {
        for (int i = tid; i < k; i += nthr) {
            const int c = ovr[(size_t)b * k + i];
            if (c >= 0 && c < nc) fsel[c] = 1;
        }
    } else {
        // rank of chunk c under (score desc, id asc); selected iff rank < k
        for (int c = tid; c < nc; c += nthr) {
            const float v = sc[c];
            int cnt = 0;
            for (int j = 0; j < nc; ++j) {
                const float u = sc[j];
                cnt += (u > v) || (u == v && j < c);
            }
            fsel[c] = cnt < k;
        }
    }
    __syncthreads();

    int32_t *streak = s.streak + (size_t)b * nc, *slot_of = s.slot_of + (size_t)b * nc;
    int32_t *slot_chunk = s.slot_chunk + (size_t)b * ns;
    for (int c = tid; c < nc; c += nthr) {
        int st = streak[c];
        st = fsel[c] ? 0 : min(st + 1, g.delta);
        streak[c] = st;
        const bool now = st < g.delta;
        const int slot = slot_of[c];
        const bool was = slot >= 0;
        if (was && !now) {
            slot_chunk[slot] = -1;
            slot_of[c] = -1;
            atomicAdd(&ndrop, 1);
        }
        fnew[c] = now && !was;
        fkept[c] = now && was;
        if (now) atomicAdd(&nrows, comp_of(g, c));
    }
    __syncthreads();

    // selected ids, ascending
    for (int c = tid; c < nc; c += nthr) rank[c] = fsel[c];
    __syncthreads();
    const int nsel = block_scan_excl(rank, nc, wsum);
    if (selected) {
        for (int c = tid; c < nc; c += nthr)
            if (fsel[c]) selected[(size_t)b * k + rank[c]] = c;
        for (int i = nsel + tid; i < k; i += nthr) selected[(size_t)b * k + i] = -1;
    }
    __syncthreads();

    // free slots, ascending
    for (int i = tid; i < ns; i += nthr) ffree[i] = slot_chunk[i] < 0;
    __syncthreads();
    for (int i = tid; i < ns; i += nthr) freelist[i] = ffree[i];
    __syncthreads();
    const int nfree = block_scan_excl(freelist, ns, wsum);   // freelist holds ranks now
    for (int i = tid; i < ns; i += nthr) ffree[i] = ffree[i] ? freelist[i] : -1;
    __syncthreads();
    for (int i = tid; i < ns; i += nthr)
        if (ffree[i] >= 0) freelist[ffree[i]] = i;
    __syncthreads();

    // newly resident chunks take the free slots in order (lowest id -> lowest slot)
    for (int c = tid; c < nc; c += nthr) rank[c] = fnew[c];
    __syncthreads();
    const int nnew = block_scan_excl(rank, nc, wsum);
    int32_t *nl = s.new_list + (size_t)b * k * 2;
    for (int c = tid; c < nc; c += nthr)
        if (fnew[c] && rank[c] < nfree && rank[c] < k) {
            const int slot = freelist[rank[c]];
            slot_of[c] = slot;
            slot_chunk[slot] = c;
            nl[rank[c] * 2] = c;
            nl[rank[c] * 2 + 1] = slot;
        }
    __syncthreads();

    for (int c = tid; c < nc; c += nthr) rank[c] = fkept[c];
    __syncthreads();
    const int nkept = block_scan_excl(rank, nc, wsum);
    int32_t *kl = s.kept_list + (size_t)b * ns * 2;
    for (int c = tid; c < nc; c += nthr)
        if (fkept[c]) {
            kl[rank[c] * 2] = c;
            kl[rank[c] * 2 + 1] = slot_of[c];
        }
    if (tid == 0) {
        const int nn = min(nnew, min(nfree, k));
        s.counts[b * 2] = nkept;
        s.counts[b * 2 + 1] = nn;
        atomicAdd(&s.stats[0], (unsigned long long)nn);
        atomicAdd(&s.stats[1], (unsigned long long)ndrop);
        atomicAdd(&s.stats[2], (unsigned long long)(nkept + nn));
        atomicAdd(&s.stats[3], (unsigned long long)nrows);
        atomicMax(&s.stats[4], (unsigned long long)(nkept + nn));
        if (nnew > nn) atomicAdd(&s.stats[5], 1ull);   // slot exhaustion (never expected)
    }
}

// -------------------------------------------------------------------------------------------
// Recall: newly resident complements, mapped pinned host memory -> device slots.
// -------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void recall_kernel(Geometry g, Tiers t, StepBuffers s)
{
    const int i = blockIdx.y, b = blockIdx.z;
    if (i >= s.counts[b * 2 + 1]) return;
    const int c = s.new_list[((size_t)b * g.k + i) * 2], slot = s.new_list[((size_t)b * g.k + i) * 2 + 1];
    const uint4 *src = (const uint4 *)(t.host_comp + ((size_t)b * g.nc + c) * g.chunk_elems);
    uint4 *dst = (uint4 *)(t.slots + ((size_t)b * g.n_slots + slot) * g.chunk_elems);
    const size_t n16 = (size_t)g.chunk_elems * 2 / 16;
    for (size_t j = (size_t)blockIdx.x * blockDim.x + threadIdx.x; j < n16; j += (size_t)gridDim.x * blockDim.x)
        dst[j] = src[j];
}

// -------------------------------------------------------------------------------------------
// Tidal / fixed attention (fp32 logits): one tile of up to TILE rows given by a row map.
// -------------------------------------------------------------------------------------------
template <int G, class RowMap>
__device__ inline void subset_tile(const uint16_t *__restrict__ qh, RowMap map, float *pm, float *pl, float *po)
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, sub = lane & 15, rg = lane >> 4;
    __shared__ float xs[WAVES * G * D];  // logits (G*TILE) -> probabilities -> wave partials
    __shared__ float red[WAVES * G];
    static_assert(WAVES * D >= TILE, "partial buffer must hold the logits");

    float qf[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) unpack8(*(const uint4 *)(qh + h * D + sub * 8), qf[h]);

    for (int i0 = 0; i0 < STEPS; i0 += 4) {
        uint4 kr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            const uint16_t *kp = map.k(r);
            kr[u] = kp ? *(const uint4 *)(kp + sub * 8) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            float f[8];
            unpack8(kr[u], f);
            float acc[G];
#pragma unroll
            for (int h = 0; h < G; ++h) {
                acc[h] = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h] = fmaf(qf[h][e], f[e], acc[h]);
                acc[h] = sum16(acc[h]);
            }
            if (sub == 0) {
                const bool ok = map.valid(r);
#pragma unroll
                for (int h = 0; h < G; ++h) xs[h * TILE + r] = ok ? acc[h] * SCALE_F : -INFINITY;
            }
        }
    }
    __syncthreads();
    float m[G], p[G];
#pragma unroll
    for (int h = 0; h < G; ++h) m[h] = xs[h * TILE + tid];
    block_max<G>(m, red);
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float x = xs[h * TILE + tid];
        p[h] = (m[h] == -INFINITY) ? 0.f : __expf(x - m[h]);
        xs[h * TILE + tid] = p[h];
    }
    block_sum<G>(p, red);
    if (tid == 0)
#pragma unroll
        for (int h = 0; h < G; ++h) {
            pm[h] = m[h];
            pl[h] = p[h];
        }

    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    for (int i0 = 0; i0 < STEPS; i0 += 4) {
        uint4 vr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            const uint16_t *vp = map.v(r);
            vr[u] = vp ? *(const uint4 *)(vp + sub * 8) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave * ROWS_PER_WAVE + (i0 + u) * 4 + rg;
            float f[8];
            unpack8(vr[u], f);
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float ph = xs[h * TILE + r];
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(ph, f[e], acc[h][e]);
            }
        }
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[h][e] += __shfl_xor(acc[h][e], 16);
            acc[h][e] += __shfl_xor(acc[h][e], 32);
        }
    __syncthreads();
    if (rg == 0)
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) xs[(wave * G + h) * D + sub * 8 + e] = acc[h][e];
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += NT) {
        float o = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) o += xs[w * G * D + idx];
        po[idx] = o;
    }
}

struct StaticRows {
    const uint16_t *K, *V;
    int t0, R;
    __device__ bool valid(int r) const { return t0 + r < R; }
    __device__ const uint16_t *k(int r) const { return valid(r) ? K + (size_t)(t0 + r) * D : nullptr; }
    __device__ const uint16_t *v(int r) const { return valid(r) ? V + (size_t)(t0 + r) * D : nullptr; }
};

struct SlotRows {
    const uint16_t *slots;   // base of this sequence's slots
    const int32_t *list;     // (chunk, slot) entries of this group
    int n_entries, ti, comp_max, nT, Ta, cl, budget_bp;
    __device__ const uint16_t *row(int r, int half) const
    {
        const int e = r / comp_max, rr = r - e * comp_max;
        if (e >= n_entries) return nullptr;
        const int c = list[e * 2], slot = list[e * 2 + 1];
        const int len = min((c + 1) * cl, Ta) - c * cl;
        if (rr >= len - keep_of_len(budget_bp, len)) return nullptr;
        return slots + ((((size_t)slot * nT + ti) * 2 + half) * comp_max + rr) * D;
    }
    __device__ bool valid(int r) const { return row(r, 0) != nullptr; }
    __device__ const uint16_t *k(int r) const { return row(r, 0); }
    __device__ const uint16_t *v(int r) const { return row(r, 1); }
};

template <int G>
__global__ __launch_bounds__(NT) void subset_static_kernel(Geometry g, Tiers t, StepBuffers s, const uint16_t *__restrict__ q)
{
    const int tile = blockIdx.x, hi = blockIdx.y, b = blockIdx.z;
    const bool tidal = hi < g.nT;
    const int idx = tidal ? hi : hi - g.nT;
    const int lk = tidal ? t.tidal_lk[idx] : t.fixed_lk[idx], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const size_t hb = ((size_t)b * (tidal ? g.nT : g.nF) + idx) * (size_t)g.Rs * D;
    StaticRows map{(tidal ? t.tK : t.fK) + hb, (tidal ? t.tV : t.fV) + hb, tile * TILE, g.Rs};
    const uint16_t *qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    const size_t p = ((size_t)b * (g.nT + g.nF) + hi) * g.np + tile;
    subset_tile<G>(qh, map, s.ps_m + p * G, s.ps_l + p * G, s.ps_o + p * G * D);
}

template <int G>
__global__ __launch_bounds__(NT) void subset_slots_kernel(Geometry g, Tiers t, StepBuffers s, const uint16_t *__restrict__ q,
                                                          int which)
{
    const int grp = blockIdx.x, ti = blockIdx.y, b = blockIdx.z;
    const int cnt = s.counts[b * 2 + which];
    if (grp * g.sg >= cnt) return;
    const int32_t *list = which ? s.new_list + (size_t)b * g.k * 2 : s.kept_list + (size_t)b * g.n_slots * 2;
    const int lk = t.tidal_lk[ti], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    SlotRows map{t.slots + (size_t)b * g.n_slots * g.chunk_elems, list + grp * g.sg * 2,
                 min(g.sg, cnt - grp * g.sg), ti, g.comp_max, g.nT, g.Ta, g.cl, g.budget_bp};
    const uint16_t *qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    const size_t p = ((size_t)b * (g.nT + g.nF) + ti) * g.np + g.n_tiles_s + (which ? g.ng_kept : 0) + grp;
    subset_tile<G>(qh, map, s.ps_m + p * G, s.ps_l + p * G, s.ps_o + p * G * D);
}

template <int G>
__global__ __launch_bounds__(NT) void subset_combine_kernel(Geometry g, Tiers t, StepBuffers s, float *out)
{
    const int hi = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const bool tidal = hi < g.nT;
    extern __shared__ float sfac[];      // [np][G]
    __shared__ float Mh[G], Lh[G];
    const int nk = tidal ? min((s.counts[b * 2] + g.sg - 1) / g.sg, g.ng_kept) : 0;
    const int nn = tidal ? min((s.counts[b * 2 + 1] + g.sg - 1) / g.sg, g.ng_new) : 0;
    const int nvalid = g.n_tiles_s + nk + nn;
    // valid partial j -> its slot in the per-head partial array
    auto slot_of_valid = [&](int j) {
        if (j < g.n_tiles_s) return j;
        j -= g.n_tiles_s;
        if (j < nk) return g.n_tiles_s + j;
        return g.n_tiles_s + g.ng_kept + (j - nk);
    };
    const size_t base = ((size_t)b * (g.nT + g.nF) + hi) * g.np;
    if (tid < G) {
        float M = -INFINITY;
        for (int j = 0; j < nvalid; ++j) M = fmaxf(M, s.ps_m[(base + slot_of_valid(j)) * G + tid]);
        float L = 0.f;
        if (M > -INFINITY)
            for (int j = 0; j < nvalid; ++j) {
                const float mj = s.ps_m[(base + slot_of_valid(j)) * G + tid];
                if (mj > -INFINITY) L += s.ps_l[(base + slot_of_valid(j)) * G + tid] * __expf(mj - M);
            }
        Mh[tid] = M;
        Lh[tid] = L;
    }
    __syncthreads();
    for (int idx = tid; idx < nvalid * G; idx += NT) {
        const int j = idx / G, h = idx - j * G;
        const float mj = s.ps_m[(base + slot_of_valid(j)) * G + h];
        sfac[idx] = (Lh[h] > 0.f && mj > -INFINITY) ? __expf(mj - Mh[h]) / Lh[h] : 0.f;
    }
    __syncthreads();
    const int lk = tidal ? t.tidal_lk[hi] : t.fixed_lk[hi - g.nT], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    float *oh = out + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    for (int idx = tid; idx < G * D; idx += NT) {
        const int h = idx / D;
        float acc = 0.f;
        for (int j = 0; j < nvalid; ++j) acc += s.ps_o[(base + slot_of_valid(j)) * G * D + idx] * sfac[j * G + h];
        oh[idx] = acc;
    }
}

// Row gather for set-up: idx >= 0 reads row idx of src_k, idx <= -2 reads row -idx-2 of src_v,
// idx == -1 writes zeros.  One thread moves 16 bytes; 16 threads move one row.
__global__ void gather_rows_kernel(uint16_t *__restrict__ dst, const uint16_t *__restrict__ src_k,
                                   const uint16_t *__restrict__ src_v, const int32_t *__restrict__ idx, int64_t n_rows)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t row = i >> 4;
    const int part = (int)(i & 15);
    if (row >= n_rows) return;
    const int32_t sidx = idx[row];
    uint4 v = make_uint4(0, 0, 0, 0);
    if (sidx >= 0)
        v = ((const uint4 *)(src_k + (int64_t)sidx * D))[part];
    else if (sidx <= -2)
        v = ((const uint4 *)(src_v + (int64_t)(-(int64_t)sidx - 2) * D))[part];
    ((uint4 *)(dst + row * D))[part] = v;
}

template <template <int> class F, typename... A>
hipError_t dispatch_g(int G, A... args)
{
    switch (G) {
    case 1: return F<1>::run(args...);
    case 2: return F<2>::run(args...);
    case 3: return F<3>::run(args...);
    case 4: return F<4>::run(args...);
    case 6: return F<6>::run(args...);
    case 8: return F<8>::run(args...);
    default: return hipErrorInvalidValue;
    }
}

template <int G>
struct AnchorL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st)
    {
        if (g.nA == 0 || g.n_tiles_a == 0) return hipSuccess;
        hipLaunchKernelGGL(anchor_attn_kernel<G>, dim3(g.n_tiles_a, g.nA, g.B), dim3(NT), 0, st, g, t, s, q);
        return hipGetLastError();
    }
};
template <int G>
struct AnchorCombineL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, float *out, hipStream_t st)
    {
        if (g.nA == 0) return hipSuccess;
        const size_t shm = (size_t)(g.n_tiles_a ? g.n_tiles_a : 1) * G * sizeof(double);
        hipLaunchKernelGGL(anchor_combine_kernel<G>, dim3(g.nA, g.B), dim3(NT), shm, st, g, t, s, out);
        return hipGetLastError();
    }
};
template <int G>
struct StaticL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st)
    {
        if (g.nT + g.nF == 0 || g.n_tiles_s == 0) return hipSuccess;
        hipLaunchKernelGGL(subset_static_kernel<G>, dim3(g.n_tiles_s, g.nT + g.nF, g.B), dim3(NT), 0, st, g, t, s, q);
        return hipGetLastError();
    }
};
template <int G>
struct SlotsL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, bool nl,
                          hipStream_t st)
    {
        const int ng = nl ? g.ng_new : g.ng_kept;
        if (g.nT == 0 || ng == 0) return hipSuccess;
        hipLaunchKernelGGL(subset_slots_kernel<G>, dim3(ng, g.nT, g.B), dim3(NT), 0, st, g, t, s, q, nl ? 1 : 0);
        return hipGetLastError();
    }
};
template <int G>
struct CombineL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, float *out, hipStream_t st)
    {
        if (g.nT + g.nF == 0) return hipSuccess;
        const size_t shm = (size_t)(g.np ? g.np : 1) * G * sizeof(float);
        hipLaunchKernelGGL(subset_combine_kernel<G>, dim3(g.nT + g.nF, g.B), dim3(NT), shm, st, g, t, s, out);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_anchor(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st)
{
    return dispatch_g<AnchorL>(g.G, g, t, s, q, st);
}

hipError_t launch_anchor_combine(const Geometry &g, const Tiers &t, const StepBuffers &s, float *out, hipStream_t st)
{
    return dispatch_g<AnchorCombineL>(g.G, g, t, s, out, st);
}

hipError_t launch_scores(const Geometry &g, const StepBuffers &s, float *scores, hipStream_t st)
{
    const int n = g.B * g.nc;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(scores_kernel, dim3((n + 255) / 256), dim3(256), 0, st, g, s, scores);
    return hipGetLastError();
}

hipError_t launch_select(const Geometry &g, const StepBuffers &s, const float *scores, const int32_t *ovr,
                         int32_t *selected, hipStream_t st)
{
    if (g.nc == 0) return hipSuccess;
    const size_t shm = (size_t)(5 * g.nc + 2 * g.n_slots) * sizeof(int);
    hipLaunchKernelGGL(select_kernel, dim3(g.B), dim3(SEL_THREADS), shm, st, g, s, scores, ovr, selected);
    return hipGetLastError();
}

hipError_t launch_recall(const Geometry &g, const Tiers &t, const StepBuffers &s, hipStream_t st)
{
    if (g.k == 0 || g.chunk_elems == 0 || g.nT == 0) return hipSuccess;
    hipLaunchKernelGGL(recall_kernel, dim3(16, g.k, g.B), dim3(256), 0, st, g, t, s);
    return hipGetLastError();
}

hipError_t launch_subset_static(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st)
{
    return dispatch_g<StaticL>(g.G, g, t, s, q, st);
}

hipError_t launch_subset_slots(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, bool new_list,
                               hipStream_t st)
{
    return dispatch_g<SlotsL>(g.G, g, t, s, q, new_list, st);
}

hipError_t launch_subset_combine(const Geometry &g, const Tiers &t, const StepBuffers &s, float *out, hipStream_t st)
{
    return dispatch_g<CombineL>(g.G, g, t, s, out, st);
}

hipError_t launch_gather_rows(uint16_t *dst, const uint16_t *src_k, const uint16_t *src_v, const int32_t *idx,
                              int64_t n_rows, hipStream_t st)
{
    if (n_rows == 0) return hipSuccess;
    const int64_t threads = n_rows * 16;
    hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, dst, src_k,
                       src_v, idx, n_rows);
    return hipGetLastError();
}

}  // namespace wnw
