// Prefill compression on the device (Method, "Prefill Compression"): the text-to-audio attention
// sums that rank a head's audio positions, and the keep selection from them (per segment, or
// over the whole audio of a head for the global variant).
//
// p[b][l][kv][tau] = sum over the text tokens t and the g q-heads of KV-head kv of the softmax
// weight that text token t puts on audio position tau; text token t attends to every audio row
// and to text rows 0..t.  Per KV-head this is S = Q K^T with Q the g * T_t text query rows and K
// the T_a + T_t key rows, a dense contraction, so both passes run on
// v_mfma_f32_16x16x32_bf16 (bf16 operands, fp32 accumulation):
//   pass 1 (prefill_rowstats_kernel): per query row, the log-sum-exp of its logits over its
//           causal key set (base 2);
//   pass 2 (prefill_colsum_kernel): per audio key, the sum over all query rows of
//           exp(s - lse).  Audio keys are visible to every text row, so pass 2 needs no mask.
// Operand layout of v_mfma_f32_16x16x32_bf16 (wave64): lane l holds A row l % 16 and B column
// l % 16, each at k = 8 * (l / 16) .. + 8 (of 32); the 16x16 fp32 result holds column l % 16 of
// rows 4 * (l / 16) + i in element i.
#include "wnw_internal.h"

#include <algorithm>

#include <math.h>

namespace wnw {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float LOG2E = 1.4426950408889634f;
constexpr float C2 = 0.08838834764831845f * LOG2E;   // logit scale 1 / sqrt(128), base 2
constexpr int RS_ROWS = 128;                          // query rows per pass-1 work-group (32 per wave)
constexpr int CS_KB = 3;                              // 16-key blocks per pass-2 wavefront
constexpr int CS_KEYS = 4 * 16 * CS_KB;               // audio keys per pass-2 work-group (48 per wave)
constexpr int TILE = 64;                              // rows staged in LDS per iteration
constexpr int PADU = D / 8 + 1;                       // uint4 per staged row: 16 + 1 of padding

// 2^x by the hardware instruction alone: outputs below 2^-126 flush to zero (exp2f adds a
// range fix-up of ~3 instructions per call for them).
__device__ inline float exp2_hw(float x)
{
    return __builtin_amdgcn_exp2f(x);
}

__device__ inline bf16x8_t as_bf8(uint4 u)
{
    return __builtin_bit_cast(bf16x8_t, u);
}

__device__ inline f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// A tile of TILE rows of D bf16 goes global -> registers (load, rows >= n read as zero) ->
// padded LDS rows (store), so the next tile's loads overlap the current tile's arithmetic.
constexpr int SPT = TILE * (D / 8) / NT;   // 16-byte pieces per thread
__device__ inline void tile_load(uint4 v[SPT], const uint16_t *src, int r0, int n)
{
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int i = threadIdx.x + j * NT, r = r0 + (i >> 4);
        v[j] = r < n ? *(const uint4 *)(src + (size_t)r * D + (i & 15) * 8) : make_uint4(0, 0, 0, 0);
    }
}
__device__ inline void tile_store(uint4 *dst, const uint4 v[SPT])
{
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int i = threadIdx.x + j * NT;
        dst[(i >> 4) * PADU + (i & 15)] = v[j];
    }
}

// Work-group w is dispatched to accelerator die (XCD) w % 8, each with its own L2.  The
// returned order gives the work-groups of one die consecutive logical indices, so the blocks
// of one KV-head (which share its K or Q rows) run on one die and share its L2.
__device__ inline int xcd_order(int w, int n)
{
    const int q = n / 8, r = n % 8, x = w % 8;
    return x * q + min(x, r) + w / 8;
}

// Merge of two (max, sum) pairs of base-2 softmax statistics.
__device__ inline void merge_ms(float &m, float &l, float m2, float l2)
{
    const float mm = fmaxf(m, m2);
    const float a = m == -INFINITY ? 0.f : l * exp2f(m - mm);
    const float b = m2 == -INFINITY ? 0.f : l2 * exp2f(m2 - mm);
    m = mm;
    l = a + b;
}

// Pass 1.  Grid: ceil(g * T_t / RS_ROWS) row blocks for each of the B * L * H_kv KV-heads,
// in XCD order.  Wave w owns query rows
// r0 + 32 w .. + 32 (two 16-row blocks) of KV-head (b, lk); rows r = j * T_t + t (q-head j of
// the group, text token t).  Each lane keeps an online (max, sum) for the four rows it holds in
// the result layout, over the keys of its column; the 16 columns are merged at the end.
__global__ __launch_bounds__(NT) void prefill_rowstats_kernel(Geometry g, const uint16_t *__restrict__ K,
                                                             const uint16_t *__restrict__ qt, float *__restrict__ lse)
{
    const int R = g.G * g.Tt, nrb = (R + RS_ROWS - 1) / RS_ROWS;
    const int v = xcd_order(blockIdx.x, gridDim.x), hd = v / nrb, rblk = v - hd * nrb;
    const int b = hd / (g.L * g.Hkv), lk = hd - b * g.L * g.Hkv, l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, grp = lane >> 4;
    const uint16_t *Kh = K + (size_t)hd * g.T * D;
    const size_t qbase = (((size_t)b * g.L + l) * g.Hq + (size_t)kv * g.G) * g.Tt;
    const uint16_t *Qh = qt + qbase * D;
    const int rw = rblk * RS_ROWS + wave * 32;

    bf16x8_t qf[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        const int r = rw + rb * 16 + col;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
            qf[rb][kk] = as_bf8(r < R ? *(const uint4 *)(Qh + (size_t)r * D + grp * 8 + 32 * kk) : make_uint4(0, 0, 0, 0));
    }
    // causal limit (last visible key) of the rows this lane holds in the result layout
    int lim[2][4];
    float nm[2][4], s[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = rw + rb * 16 + 4 * grp + i;
            lim[rb][i] = r < R ? g.Ta + r % g.Tt : -1;
            nm[rb][i] = INFINITY;
            s[rb][i] = 0.f;
        }

    __shared__ uint4 kbuf[2][TILE * PADU];
    uint4 pre[SPT];
    tile_load(pre, Kh, 0, g.T);
    tile_store(kbuf[0], pre);
    __syncthreads();
    for (int k0 = 0, it = 0; k0 < g.T; k0 += TILE, ++it) {
        const uint4 *ks = kbuf[it & 1];
        const bool more = k0 + TILE < g.T;
        if (more) tile_load(pre, Kh, k0 + TILE, g.T);
        // logits of the tile: x[rb][kb][i] for row 4 * grp + i of block rb, key k0 + 16 kb + col
        f32x4_t x[2][TILE / 16];
#pragma unroll
        for (int kb = 0; kb < TILE / 16; ++kb) {
            bf16x8_t kf[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) kf[kk] = as_bf8(ks[(kb * 16 + col) * PADU + grp + 4 * kk]);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
                f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) acc = mfma16(qf[rb][kk], kf[kk], acc);
                x[rb][kb] = acc;   // unscaled; the scale folds into the exponent's FMA
            }
        }
        // Statistics are base 2 and scaled, the running maximum kept negated (nm = -m) for the
        // exponent's FMA.  Every row sum holds a term of at least 2^0, so exponentials that flush
        // below 2^-126 change nothing.
        if (k0 + TILE <= g.Ta) {
            // audio tile: every key visible to every row, no mask.  The terms are first taken
            // against the running maximum as it stands; only when a row's terms add up to more
            // than 2^20 (or its maximum is still -inf, which gives +inf) does the wavefront raise
            // the maxima and take the tile again.  Sums stay far inside fp32's range either way.
            float t[2][4], tall = 0.f;
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float acc = exp2_hw(fmaf(x[rb][0][i], C2, nm[rb][i]));
#pragma unroll
                    for (int kb = 1; kb < TILE / 16; ++kb) acc += exp2_hw(fmaf(x[rb][kb][i], C2, nm[rb][i]));
                    t[rb][i] = acc;
                    tall += acc;
                }
            if (__any(tall > 0x1p20f)) {
#pragma unroll
                for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float mt = fmaxf(fmaxf(x[rb][0][i], x[rb][1][i]), fmaxf(x[rb][2][i], x[rb][3][i]));
                        const float mn = fmaxf(-nm[rb][i], mt * C2);
                        float acc = s[rb][i] * exp2_hw(-nm[rb][i] - mn);   // 0 before the first tile
#pragma unroll
                        for (int kb = 0; kb < TILE / 16; ++kb) acc += exp2_hw(fmaf(x[rb][kb][i], C2, -mn));
                        s[rb][i] = acc;
                        nm[rb][i] = -mn;
                    }
            } else {
#pragma unroll
                for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) s[rb][i] += t[rb][i];
            }
        } else {
            // keys past a row's causal limit (text rows after its token, rows past the end, keys
            // past the cache) drop out
#pragma unroll
            for (int kb = 0; kb < TILE / 16; ++kb) {
                const int key = k0 + kb * 16 + col;
#pragma unroll
                for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (key > lim[rb][i]) x[rb][kb][i] = -INFINITY;
            }
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float mt = x[rb][0][i];
#pragma unroll
                    for (int kb = 1; kb < TILE / 16; ++kb) mt = fmaxf(mt, x[rb][kb][i]);
                    if (mt == -INFINITY) continue;   // every key of the tile masked for this row
                    const float mn = fmaxf(-nm[rb][i], mt * C2);
                    float acc = s[rb][i] * exp2_hw(-nm[rb][i] - mn);   // exp2(-inf) = 0 for an empty row
#pragma unroll
                    for (int kb = 0; kb < TILE / 16; ++kb) acc += exp2_hw(fmaf(x[rb][kb][i], C2, -mn));
                    s[rb][i] = acc;
                    nm[rb][i] = -mn;
                }
        }
        if (more) tile_store(kbuf[(it + 1) & 1], pre);
        __syncthreads();
    }
    // merge the 16 columns of each row (lanes of one group), in a fixed order
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float m = -nm[rb][i], l = s[rb][i];
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) {
                const float m2 = __shfl_xor(m, o), l2 = __shfl_xor(l, o);
                merge_ms(m, l, m2, l2);
            }
            const int r = rw + rb * 16 + 4 * grp + i;
            if (col == 0 && r < R) lse[qbase + r] = m + log2f(l);
        }
}

// Pass 2.  Grid: ceil(T_a / CS_KEYS) key blocks for each of the B * L * H_kv KV-heads, in XCD
// order.  Wave w owns audio keys k0 + 48 w .. + 48 (three 16-key blocks, their K fragments held
// in registers, so each query fragment read from LDS feeds three MFMA chains); the work-group
// walks every query row of the KV-head in tiles of TILE rows staged in LDS with their
// log-sum-exp, and each lane adds exp2(s * C2 - lse) over the rows it holds for its key column.
__global__ __launch_bounds__(NT, 3) void prefill_colsum_kernel(Geometry g, const uint16_t *__restrict__ K,
                                                           const uint16_t *__restrict__ qt,
                                                           const float *__restrict__ lse, float *__restrict__ p)
{
    const int R = g.G * g.Tt, nkb = (g.Ta + CS_KEYS - 1) / CS_KEYS;
    const int v = xcd_order(blockIdx.x, gridDim.x), hd = v / nkb, kblk = v - hd * nkb;
    const int b = hd / (g.L * g.Hkv), lk = hd - b * g.L * g.Hkv, l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, grp = lane >> 4;
    const uint16_t *Kh = K + (size_t)hd * g.T * D;
    const size_t qbase = (((size_t)b * g.L + l) * g.Hq + (size_t)kv * g.G) * g.Tt;
    const uint16_t *Qh = qt + qbase * D;
    const int kw = kblk * CS_KEYS + wave * 16 * CS_KB;

    bf16x8_t kf[CS_KB][4];
#pragma unroll
    for (int kb = 0; kb < CS_KB; ++kb) {
        const int key = kw + kb * 16 + col;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
            kf[kb][kk] = as_bf8(key < g.Ta ? *(const uint4 *)(Kh + (size_t)key * D + grp * 8 + 32 * kk)
                                           : make_uint4(0, 0, 0, 0));
    }
    float acc[CS_KB] = {};
    __shared__ uint4 qbuf[2][TILE * PADU];
    __shared__ float sbuf[2][TILE];
    uint4 pre[SPT];
    float pl = 0.f;
    // Terms are taken as 2^(x - lse + 64) and the sum scaled by 2^-64 at the end, so that terms
    // below 2^-126 still count without the exponential's range fix-up (terms are at most 1 and
    // sums of at most R of them stay far below the fp32 range).  sbuf holds 64 - lse; a padding
    // row holds -inf and adds 0.
    auto lse_of = [&](int r) { return r < R ? 64.f - lse[qbase + r] : -INFINITY; };
    tile_load(pre, Qh, 0, R);
    tile_store(qbuf[0], pre);
    if (threadIdx.x < TILE) sbuf[0][threadIdx.x] = lse_of(threadIdx.x);
    __syncthreads();
    for (int r0 = 0, it = 0; r0 < R; r0 += TILE, ++it) {
        const uint4 *qs = qbuf[it & 1];
        const float *sst = sbuf[it & 1];
        const bool more = r0 + TILE < R;
        if (more) {
            tile_load(pre, Qh, r0 + TILE, R);
            if (threadIdx.x < TILE) pl = lse_of(r0 + TILE + threadIdx.x);
        }
#pragma unroll
        for (int rb = 0; rb < TILE / 16; ++rb) {
            bf16x8_t qf[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) qf[kk] = as_bf8(qs[(rb * 16 + col) * PADU + grp + 4 * kk]);
            float st[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) st[i] = sst[rb * 16 + 4 * grp + i];
#pragma unroll
            for (int kb = 0; kb < CS_KB; ++kb) {
                f32x4_t sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) sc = mfma16(qf[kk], kf[kb][kk], sc);
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[kb] += exp2_hw(fmaf(sc[i], C2, st[i]));
            }
        }
        if (more) {
            tile_store(qbuf[(it + 1) & 1], pre);
            if (threadIdx.x < TILE) sbuf[(it + 1) & 1][threadIdx.x] = pl;
        }
        __syncthreads();
    }
#pragma unroll
    for (int kb = 0; kb < CS_KB; ++kb) {
        acc[kb] += __shfl_xor(acc[kb], 16);
        acc[kb] += __shfl_xor(acc[kb], 32);
    }
    if (grp == 0)
#pragma unroll
        for (int kb = 0; kb < CS_KB; ++kb) {
            const int key = kw + kb * 16 + col;
            if (key < g.Ta) p[(size_t)hd * g.Ta + key] = ldexpf(acc[kb], -64);
        }
}

// Per-segment keep selection.  Grid (n_sub, B), one work-group per non-anchor head: position
// tau of segment j is kept iff fewer than keep(j) positions of the segment outrank it, by
// (score descending, position ascending); keep(j) is kfull, or klast for the last segment.
__global__ __launch_bounds__(NT) void prefill_keep_kernel(Geometry g, const int32_t *__restrict__ sub_lk,
                                                         const int2 *__restrict__ seg_keep,
                                                         const float *__restrict__ p, uint8_t *__restrict__ keep)
{
    const int hi = blockIdx.x, b = blockIdx.y, nsub = gridDim.x;
    const int lkh = sub_lk[hi];
    const int2 kc = seg_keep[hi];
    const float *ph = p + ((size_t)b * g.L * g.Hkv + lkh) * g.Ta;
    uint8_t *kh = keep + ((size_t)b * nsub + hi) * g.Ta;
    for (int tau = threadIdx.x; tau < g.Ta; tau += NT) {
        const int j = tau / g.cl, b0 = j * g.cl, e0 = min(b0 + g.cl, g.Ta);
        const int k = j == g.nc - 1 ? kc.y : kc.x;
        const float v = ph[tau];
        int rank = 0;
        for (int u = b0; u < e0; ++u) {
            const float w = ph[u];
            rank += (w > v) || (w == v && u < tau);
        }
        kh[tau] = isnan(v) ? 2 : rank < k;
    }
}

// Order-preserving key of a score: larger score, larger key; -0 and +0 are one key (they compare
// equal, so they tie and the lower position wins, as in the per-segment ranking).
__device__ inline uint32_t score_key(float v)
{
    uint32_t u = __float_as_uint(v);
    if (u == 0x80000000u) u = 0;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Global variant: one work-group per non-anchor head keeps the total of its per-segment counts,
// ranked over the whole audio.  A radix selection (four 8-bit digits, most significant first)
// finds the key v of the k-th best score and how many positions holding exactly v are kept;
// those go to the lowest positions (a block-wide prefix count in position order).
__global__ __launch_bounds__(NT) void prefill_keep_global_kernel(Geometry g, const int32_t *__restrict__ sub_lk,
                                                                const int2 *__restrict__ seg_keep,
                                                                const float *__restrict__ p, uint8_t *__restrict__ keep)
{
    const int hi = blockIdx.x, b = blockIdx.y, nsub = gridDim.x, tid = threadIdx.x;
    const int2 kc = seg_keep[hi];
    const int total = g.nc ? (g.nc - 1) * kc.x + kc.y : 0;
    const float *ph = p + ((size_t)b * g.L * g.Hkv + sub_lk[hi]) * g.Ta;
    uint8_t *kh = keep + ((size_t)b * nsub + hi) * g.Ta;
    __shared__ int hist[256];
    __shared__ uint32_t s_prefix;
    __shared__ int s_need, s_scan[NT];
    uint32_t prefix = 0, mask = 0;
    int need = total;
    if (total > 0) {
        for (int shift = 24; shift >= 0; shift -= 8) {
            hist[tid] = 0;   // NT == 256 bins
            __syncthreads();
            for (int t = tid; t < g.Ta; t += NT) {
                const uint32_t key = score_key(ph[t]);
                if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1);
            }
            __syncthreads();
            if (tid == 0) {
                int cum = 0, d = 255;
                for (; d > 0; --d) {
                    if (cum + hist[d] >= need) break;
                    cum += hist[d];
                }
                s_prefix = prefix | ((uint32_t)d << shift);
                s_need = need - cum;
            }
            __syncthreads();
            prefix = s_prefix;
            need = s_need;
            mask |= 255u << shift;
            __syncthreads();
        }
    }
    // keep: key > v, or key == v among the first `need` such positions
    int base = 0;
    for (int t0 = 0; t0 < g.Ta; t0 += NT) {
        const int t = t0 + tid;
        const float v = t < g.Ta ? ph[t] : 0.f;
        const uint32_t key = score_key(v);
        const int tie = (total > 0 && t < g.Ta && key == prefix) ? 1 : 0;
        s_scan[tid] = tie;
        __syncthreads();
        for (int o = 1; o < NT; o <<= 1) {   // inclusive prefix sum
            const int add = tid >= o ? s_scan[tid - o] : 0;
            __syncthreads();
            s_scan[tid] += add;
            __syncthreads();
        }
        if (t < g.Ta) {
            const int before = base + s_scan[tid] - tie;
            kh[t] = isnan(v) ? 2 : (total > 0 && (key > prefix || (tie && before < need)));
        }
        base += s_scan[NT - 1];
        __syncthreads();
    }
}

// p = 0 (no text tokens): a fill kernel rather than a memset, so that the launch can sit in a
// captured graph.
__global__ __launch_bounds__(NT) void prefill_zero_kernel(float *__restrict__ p, long long n)
{
    for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n; i += (long long)gridDim.x * NT) p[i] = 0.f;
}

}  // namespace

hipError_t launch_prefill_scores(const Geometry &g, const uint16_t *K, const uint16_t *q_text, float *lse,
                                 float *p, hipStream_t st)
{
    const int R = g.G * g.Tt;
    if (g.Ta == 0) return hipSuccess;
    if (R == 0) {
        const long long n = (long long)g.B * g.L * g.Hkv * g.Ta;
        hipLaunchKernelGGL(prefill_zero_kernel, dim3((unsigned)std::min<long long>((n + NT - 1) / NT, 4096)), dim3(NT), 0,
                           st, p, n);
        return hipGetLastError();
    }
    const long long nheads = (long long)g.B * g.L * g.Hkv;
    const long long n1 = (long long)((R + RS_ROWS - 1) / RS_ROWS) * nheads;
    const long long n2 = (long long)((g.Ta + CS_KEYS - 1) / CS_KEYS) * nheads;
    if (n1 > INT32_MAX || n2 > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(prefill_rowstats_kernel, dim3((unsigned)n1), dim3(NT), 0, st, g, K, q_text, lse);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(prefill_colsum_kernel, dim3((unsigned)n2), dim3(NT), 0, st, g, K, q_text, (const float *)lse, p);
    return hipGetLastError();
}

hipError_t launch_prefill_keep(const Geometry &g, int n_sub, const int32_t *sub_lk, const int2 *seg_keep, bool global,
                               const float *p, uint8_t *keep, hipStream_t st)
{
    if (n_sub == 0 || g.Ta == 0) return hipSuccess;
    if (global)
        hipLaunchKernelGGL(prefill_keep_global_kernel, dim3(n_sub, g.B), dim3(NT), 0, st, g, sub_lk, seg_keep, p, keep);
    else
        hipLaunchKernelGGL(prefill_keep_kernel, dim3(n_sub, g.B), dim3(NT), 0, st, g, sub_lk, seg_keep, p, keep);
    return hipGetLastError();
}

}  // namespace wnw
