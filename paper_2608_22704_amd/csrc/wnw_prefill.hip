// Prefill compression on the device (Method, "Prefill Compression"): the text-to-audio attention
// sums that rank a head's audio positions, and the per-segment keep selection from them.
//
// p[b][l][kv][tau] = sum over the text tokens t and the g q-heads of KV-head kv of the softmax
// weight that text token t puts on audio position tau; text token t attends to every audio row
// and to text rows 0..t.  Per KV-head this is S = Q K^T with Q the g * T_t text query rows and K
// the T_a + T_t key rows, a dense contraction, so both passes run on
// v_mfma_f32_16x16x32_bf16 (bf16 operands, fp32 accumulation):
//   pass 1 (prefill_rowstats_kernel): per query row, the softmax maximum and sum over its
//           causal key set;
//   pass 2 (prefill_colsum_kernel): per audio key, the sum over all query rows of
//           exp(s - max) / sum.  Audio keys are visible to every text row, so pass 2 needs no mask.
// Operand layout of v_mfma_f32_16x16x32_bf16 (wave64): lane l holds A row l % 16 and B column
// l % 16, each at k = 8 * (l / 16) .. + 8 (of 32); the 16x16 fp32 result holds column l % 16 of
// rows 4 * (l / 16) + i in element i.
#include "wnw_internal.h"

#include <math.h>

namespace wnw {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float LOG2E = 1.4426950408889634f;
constexpr float C2 = 0.08838834764831845f * LOG2E;   // logit scale 1 / sqrt(128), base 2
constexpr int RS_ROWS = 128;                          // query rows per pass-1 work-group (32 per wave)
constexpr int CS_KEYS = 128;                          // audio keys per pass-2 work-group (32 per wave)
constexpr int TILE = 64;                              // rows staged in LDS per iteration
constexpr int PADU = D / 8 + 1;                       // uint4 per staged row: 16 + 1 of padding

__device__ inline bf16x8_t as_bf8(uint4 u)
{
    return __builtin_bit_cast(bf16x8_t, u);
}

__device__ inline f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Stage TILE rows of D bf16 (rows >= n are zero) into padded LDS rows.
__device__ inline void stage_rows(uint4 *dst, const uint16_t *src, int r0, int n)
{
    for (int i = threadIdx.x; i < TILE * (D / 8); i += NT) {
        const int rr = i >> 4, c = i & 15, r = r0 + rr;
        dst[rr * PADU + c] = r < n ? *(const uint4 *)(src + (size_t)r * D + c * 8) : make_uint4(0, 0, 0, 0);
    }
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

// Pass 1.  Grid (ceil(g * T_t / RS_ROWS), L * H_kv, B).  Wave w owns query rows
// r0 + 32 w .. + 32 (two 16-row blocks) of KV-head (b, lk); rows r = j * T_t + t (q-head j of
// the group, text token t).  Each lane keeps an online (max, sum) for the four rows it holds in
// the result layout, over the keys of its column; the 16 columns are merged at the end.
__global__ __launch_bounds__(NT) void prefill_rowstats_kernel(Geometry g, const uint16_t *__restrict__ K,
                                                             const uint16_t *__restrict__ qt, float2 *__restrict__ stats)
{
    const int lk = blockIdx.y, b = blockIdx.z, l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, grp = lane >> 4;
    const int R = g.G * g.Tt;
    const uint16_t *Kh = K + ((size_t)b * g.L * g.Hkv + lk) * (size_t)g.T * D;
    const size_t qbase = (((size_t)b * g.L + l) * g.Hq + (size_t)kv * g.G) * g.Tt;
    const uint16_t *Qh = qt + qbase * D;
    const int rw = blockIdx.x * RS_ROWS + wave * 32;

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
    float m[2][4], s[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = rw + rb * 16 + 4 * grp + i;
            lim[rb][i] = r < R ? g.Ta + r % g.Tt : -1;
            m[rb][i] = -INFINITY;
            s[rb][i] = 0.f;
        }

    __shared__ uint4 ks[TILE * PADU];
    for (int k0 = 0; k0 < g.T; k0 += TILE) {
        __syncthreads();
        stage_rows(ks, Kh, k0, g.T);
        __syncthreads();
#pragma unroll
        for (int kb = 0; kb < TILE / 16; ++kb) {
            bf16x8_t kf[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) kf[kk] = as_bf8(ks[(kb * 16 + col) * PADU + grp + 4 * kk]);
            const int key = k0 + kb * 16 + col;
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
                f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) acc = mfma16(qf[rb][kk], kf[kk], acc);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (key > lim[rb][i]) continue;   // causal mask (and rows past the end)
                    const float x = acc[i] * C2;
                    if (x > m[rb][i]) {
                        s[rb][i] = s[rb][i] * exp2f(m[rb][i] - x) + 1.f;
                        m[rb][i] = x;
                    } else {
                        s[rb][i] += exp2f(x - m[rb][i]);
                    }
                }
            }
        }
    }
    // merge the 16 columns of each row (lanes of one group), in a fixed order
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) {
                const float m2 = __shfl_xor(m[rb][i], o), s2 = __shfl_xor(s[rb][i], o);
                merge_ms(m[rb][i], s[rb][i], m2, s2);
            }
    if (col == 0)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = rw + rb * 16 + 4 * grp + i;
                if (r < R) stats[qbase + r] = make_float2(m[rb][i], 1.f / s[rb][i]);
            }
}

// Pass 2.  Grid (ceil(T_a / CS_KEYS), L * H_kv, B).  Wave w owns audio keys k0 + 32 w .. + 32
// (two 16-key blocks, their K fragments held in registers); the work-group walks every query row
// of the KV-head in tiles of TILE rows staged in LDS with their statistics, and each lane adds
// exp2(s * C2 - max) / sum over the rows it holds for its key column.
__global__ __launch_bounds__(NT) void prefill_colsum_kernel(Geometry g, const uint16_t *__restrict__ K,
                                                           const uint16_t *__restrict__ qt,
                                                           const float2 *__restrict__ stats, float *__restrict__ p)
{
    const int lk = blockIdx.y, b = blockIdx.z, l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, grp = lane >> 4;
    const int R = g.G * g.Tt;
    const uint16_t *Kh = K + ((size_t)b * g.L * g.Hkv + lk) * (size_t)g.T * D;
    const size_t qbase = (((size_t)b * g.L + l) * g.Hq + (size_t)kv * g.G) * g.Tt;
    const uint16_t *Qh = qt + qbase * D;
    const int kw = blockIdx.x * CS_KEYS + wave * 32;

    bf16x8_t kf[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int key = kw + kb * 16 + col;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
            kf[kb][kk] = as_bf8(key < g.Ta ? *(const uint4 *)(Kh + (size_t)key * D + grp * 8 + 32 * kk)
                                           : make_uint4(0, 0, 0, 0));
    }
    float acc[2] = {0.f, 0.f};
    __shared__ uint4 qs[TILE * PADU];
    __shared__ float2 sst[TILE];
    for (int r0 = 0; r0 < R; r0 += TILE) {
        __syncthreads();
        stage_rows(qs, Qh, r0, R);
        if (threadIdx.x < TILE) {
            const int r = r0 + threadIdx.x;
            sst[threadIdx.x] = r < R ? stats[qbase + r] : make_float2(0.f, 0.f);   // a padding row adds 0
        }
        __syncthreads();
#pragma unroll
        for (int rb = 0; rb < TILE / 16; ++rb) {
            bf16x8_t qf[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) qf[kk] = as_bf8(qs[(rb * 16 + col) * PADU + grp + 4 * kk]);
            float2 st[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) st[i] = sst[rb * 16 + 4 * grp + i];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                f32x4_t sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) sc = mfma16(qf[kk], kf[kb][kk], sc);
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[kb] += exp2f(sc[i] * C2 - st[i].x) * st[i].y;
            }
        }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        acc[kb] += __shfl_xor(acc[kb], 16);
        acc[kb] += __shfl_xor(acc[kb], 32);
    }
    if (grp == 0)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int key = kw + kb * 16 + col;
            if (key < g.Ta) p[((size_t)b * g.L * g.Hkv + lk) * g.Ta + key] = acc[kb];
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
        kh[tau] = rank < k;
    }
}

}  // namespace

hipError_t launch_prefill_scores(const Geometry &g, const uint16_t *K, const uint16_t *q_text, float2 *stats,
                                 float *p, hipStream_t st)
{
    const int R = g.G * g.Tt;
    if (g.Ta == 0) return hipSuccess;
    if (R == 0) return hipMemsetAsync(p, 0, (size_t)g.B * g.L * g.Hkv * g.Ta * sizeof(float), st);
    hipLaunchKernelGGL(prefill_rowstats_kernel, dim3((R + RS_ROWS - 1) / RS_ROWS, g.L * g.Hkv, g.B), dim3(NT), 0, st, g,
                       K, q_text, stats);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(prefill_colsum_kernel, dim3((g.Ta + CS_KEYS - 1) / CS_KEYS, g.L * g.Hkv, g.B), dim3(NT), 0, st,
                       g, K, q_text, (const float2 *)stats, p);
    return hipGetLastError();
}

hipError_t launch_prefill_keep(const Geometry &g, int n_sub, const int32_t *sub_lk, const int2 *seg_keep,
                               const float *p, uint8_t *keep, hipStream_t st)
{
    if (n_sub == 0 || g.Ta == 0) return hipSuccess;
    hipLaunchKernelGGL(prefill_keep_kernel, dim3(n_sub, g.B), dim3(NT), 0, st, g, sub_lk, seg_keep, p, keep);
    return hipGetLastError();
}

}  // namespace wnw
