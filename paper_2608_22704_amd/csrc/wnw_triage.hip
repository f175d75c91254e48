// Head triage arithmetic (Method, "Head Functional Triage via Offline Calibration", with the
// calibration score details of the appendix), on given inputs: the answer tokens' queries and a
// sample's keys, their aligned audio intervals, and the loss gradients at the audio keys.  The
// model, the alignment and the autograd that produce those are outside the library.
//
//   voice_hits_kernel   per (answer token, q-head): the K audio positions with the largest
//                       logit (softmax keeps the order), ties to the lower position, counted
//                       inside the token's interval.  Logits are exact bf16 products summed in
//                       double, so the top-K decisions are those of the exact logits.
//   key_sens_kernel     per (answer token, KV-head): the mean over audio positions of the L2 norm
//                       of the key gradient.  A streaming reduction (HBM-bound).
//   wnw_triage          (host) VS and HS means, VS * HS ranking, roles, normalised importance.
#include "wnw.h"
#include "wnw_internal.h"

#include <math.h>

#include <algorithm>
#include <cstring>
#include <numeric>
#include <vector>

namespace wnw {

namespace {

constexpr int VH_ROWS = 64;   // (token, q-head) rows per work-group
constexpr int VH_SPLIT = 4;   // threads per row; key tau goes to thread tau % 4 of its tile
constexpr int VH_TILE = 64;   // keys staged in LDS per iteration
constexpr int VH_KMAX = 8;    // largest K (the paper uses 4 and 8)
constexpr int PADU = D / 8 + 1;

__device__ inline void bf16x2(uint32_t u, double &lo, double &hi)
{
    lo = (double)__uint_as_float(u << 16);
    hi = (double)__uint_as_float(u & 0xffff0000u);
}

// Grid (ceil(n_tok / tpb), L * Hkv), tpb = VH_ROWS / g tokens per work-group.  Thread (row r,
// split s): row r = token tt * g + q-head j; the thread scans the keys s, s + 4, ... of each tile
// and keeps its best eight (value descending; equal values keep the earlier, lower, position).
// The four lists of a row are merged at the end.
__global__ __launch_bounds__(NT) void voice_hits_kernel(int L, int Hq, int Hkv, int T, int Ta, int n_tok, int K,
                                                       const uint16_t *__restrict__ k, const uint16_t *__restrict__ q,
                                                       const int32_t *__restrict__ span, int32_t *__restrict__ hits)
{
    const int g = Hq / Hkv, tpb = VH_ROWS / g, lk = blockIdx.y, l = lk / Hkv, kv = lk - l * Hkv;
    const int tid = threadIdx.x, r = tid / VH_SPLIT, sp = tid % VH_SPLIT;
    const int tt = r / g, j = r - tt * g, t = blockIdx.x * tpb + tt;
    const bool active = tt < tpb && t < n_tok;
    uint32_t qv[D / 2];
    {
        const uint4 *qrow = (const uint4 *)(q + (((size_t)(active ? t : 0) * L + l) * Hq + (size_t)kv * g + j) * D);
#pragma unroll
        for (int i = 0; i < D / 8; ++i) {
            const uint4 u = active ? qrow[i] : make_uint4(0, 0, 0, 0);
            qv[4 * i] = u.x;
            qv[4 * i + 1] = u.y;
            qv[4 * i + 2] = u.z;
            qv[4 * i + 3] = u.w;
        }
    }
    double best[VH_KMAX];
    int bpos[VH_KMAX];
#pragma unroll
    for (int i = 0; i < VH_KMAX; ++i) {
        best[i] = -INFINITY;
        bpos[i] = INT32_MAX;
    }
    const uint16_t *Kh = k + (size_t)lk * T * D;
    __shared__ uint4 ks[VH_TILE * PADU];
    for (int k0 = 0; k0 < Ta; k0 += VH_TILE) {
        __syncthreads();
        for (int i = tid; i < VH_TILE * (D / 8); i += NT) {
            const int rr = i >> 4, c = i & 15, row = k0 + rr;
            ks[rr * PADU + c] = row < Ta ? *(const uint4 *)(Kh + (size_t)row * D + c * 8) : make_uint4(0, 0, 0, 0);
        }
        __syncthreads();
        for (int kr = sp; kr < VH_TILE; kr += VH_SPLIT) {
            const int tau = k0 + kr;
            if (tau >= Ta) break;
            double acc = 0.0;
#pragma unroll
            for (int c = 0; c < D / 8; ++c) {
                const uint4 u = ks[kr * PADU + c];
                const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    double k_lo, k_hi, q_lo, q_hi;
                    bf16x2(w[e], k_lo, k_hi);
                    bf16x2(qv[4 * c + e], q_lo, q_hi);
                    acc = fma(q_lo, k_lo, acc);
                    acc = fma(q_hi, k_hi, acc);
                }
            }
            if (acc > best[VH_KMAX - 1]) {
                double v = acc;
                int p = tau;
#pragma unroll
                for (int s = 0; s < VH_KMAX; ++s)
                    if (v > best[s]) {
                        const double tv = best[s];
                        const int tp = bpos[s];
                        best[s] = v;
                        bpos[s] = p;
                        v = tv;
                        p = tp;
                    }
            }
        }
    }
    __shared__ double sbest[VH_ROWS][VH_SPLIT * VH_KMAX];
    __shared__ int spos[VH_ROWS][VH_SPLIT * VH_KMAX];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < VH_KMAX; ++i) {
        sbest[r][sp * VH_KMAX + i] = best[i];
        spos[r][sp * VH_KMAX + i] = bpos[i];
    }
    __syncthreads();
    if (sp == 0 && active) {
        // top K of the row's candidates by (value descending, position ascending)
        const int a = span[2 * t], b = span[2 * t + 1];
        unsigned taken = 0;
        int c = 0;
        for (int n = 0; n < K; ++n) {
            int bi = -1;
            for (int i = 0; i < VH_SPLIT * VH_KMAX; ++i) {
                if (taken >> i & 1u) continue;
                if (bi < 0 || sbest[r][i] > sbest[r][bi] || (sbest[r][i] == sbest[r][bi] && spos[r][i] < spos[r][bi]))
                    bi = i;
            }
            taken |= 1u << bi;
            const int pos = spos[r][bi];
            c += pos >= a && pos < b;
        }
        hits[((size_t)t * L + l) * Hq + (size_t)kv * g + j] = c;
    }
}

// One work-group of KS_THREADS per (answer token, KV-head) row of T_a gradient vectors: sixteen
// threads per position (eight floats each), four positions per thread in flight; the
// per-position norms are summed in double in a fixed order.
constexpr int KS_THREADS = 1024, KS_SLOTS = KS_THREADS / 16, KS_UNROLL = 4;
typedef float f4v __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(KS_THREADS) void key_sens_kernel(int Ta, const float *__restrict__ grad,
                                                             float *__restrict__ sens)
{
    const size_t row = blockIdx.x;
    const f4v *G4 = (const f4v *)(grad + row * (size_t)Ta * D);
    const int tid = threadIdx.x, l16 = tid & 15, slot = tid >> 4;
    double acc = 0.0;
    for (int t0 = slot; t0 < Ta; t0 += KS_SLOTS * KS_UNROLL) {
        f4v a[KS_UNROLL], b[KS_UNROLL];
#pragma unroll
        for (int u = 0; u < KS_UNROLL; ++u) {
            const int tau = t0 + u * KS_SLOTS;
            if (tau < Ta) {
                a[u] = __builtin_nontemporal_load(&G4[(size_t)tau * (D / 4) + 2 * l16]);
                b[u] = __builtin_nontemporal_load(&G4[(size_t)tau * (D / 4) + 2 * l16 + 1]);
            } else {
                a[u] = b[u] = f4v{0.f, 0.f, 0.f, 0.f};
            }
        }
#pragma unroll
        for (int u = 0; u < KS_UNROLL; ++u) {
            float s2 = a[u].x * a[u].x + a[u].y * a[u].y + a[u].z * a[u].z + a[u].w * a[u].w + b[u].x * b[u].x +
                       b[u].y * b[u].y + b[u].z * b[u].z + b[u].w * b[u].w;
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) s2 += __shfl_xor(s2, o);
            if (l16 == 0 && t0 + u * KS_SLOTS < Ta) acc += sqrt((double)s2);
        }
    }
    __shared__ double red[KS_SLOTS];
    if (l16 == 0) red[slot] = acc;
    __syncthreads();
    if (tid == 0) {
        double s = 0.0;
        for (int i = 0; i < KS_SLOTS; ++i) s += red[i];
        sens[row] = (float)(s / Ta);
    }
}

thread_local char t_msg[256] = "no error";

wnw_status triage_fail(wnw_status st, const char *msg)
{
    strncpy(t_msg, msg, sizeof t_msg - 1);
    return st;
}

}  // namespace

}  // namespace wnw

using namespace wnw;

extern "C" {

const char *wnw_triage_last_error(void)
{
    return t_msg;
}

wnw_status wnw_voice_hits(int32_t layers, int32_t q_heads, int32_t kv_heads, int32_t rows, int32_t audio_len,
                          int32_t n_tok, const void *k_dev, const void *q_dev, const int32_t *span_dev, int32_t top_k,
                          int32_t *hits_dev, void *hip_stream)
{
    if (layers < 1 || kv_heads < 1 || q_heads < kv_heads || q_heads % kv_heads || audio_len < 0 || rows < audio_len ||
        n_tok < 0 || (int64_t)layers * kv_heads > 65535)
        return triage_fail(WNW_ERR_INVALID, "bad sizes");
    const int g = q_heads / kv_heads;
    if (g > VH_ROWS) return triage_fail(WNW_ERR_UNSUPPORTED, "GQA group larger than 64");
    if (top_k < 1 || top_k > VH_KMAX || top_k > audio_len)
        return triage_fail(WNW_ERR_INVALID, "top_k must be in 1..8 and at most audio_len");
    if (n_tok == 0) return WNW_OK;
    if (!k_dev || !q_dev || !span_dev || !hits_dev) return triage_fail(WNW_ERR_INVALID, "NULL pointer");
    const int tpb = VH_ROWS / g;
    hipLaunchKernelGGL(voice_hits_kernel, dim3((n_tok + tpb - 1) / tpb, layers * kv_heads), dim3(NT), 0,
                       (hipStream_t)hip_stream, layers, q_heads, kv_heads, rows, audio_len, n_tok, top_k,
                       (const uint16_t *)k_dev, (const uint16_t *)q_dev, span_dev, hits_dev);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? WNW_OK : triage_fail(WNW_ERR_HIP, hipGetErrorString(e));
}

wnw_status wnw_key_sensitivity(int32_t layers, int32_t kv_heads, int32_t audio_len, int32_t n_tok, const float *grad_dev,
                               float *sens_dev, void *hip_stream)
{
    if (layers < 1 || kv_heads < 1 || audio_len < 1 || n_tok < 0) return triage_fail(WNW_ERR_INVALID, "bad sizes");
    const int64_t n = (int64_t)n_tok * layers * kv_heads;
    if (n == 0) return WNW_OK;
    if (n > INT32_MAX) return triage_fail(WNW_ERR_UNSUPPORTED, "too many rows");
    if (!grad_dev || !sens_dev) return triage_fail(WNW_ERR_INVALID, "NULL pointer");
    hipLaunchKernelGGL(key_sens_kernel, dim3((unsigned)n), dim3(KS_THREADS), 0, (hipStream_t)hip_stream, audio_len,
                       grad_dev, sens_dev);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? WNW_OK : triage_fail(WNW_ERR_HIP, hipGetErrorString(e));
}

wnw_status wnw_triage(int32_t layers, int32_t kv_heads, int32_t group, int32_t n, const int32_t *sample,
                      const int32_t *hits, int32_t top_k, const float *sens, int32_t n_voice, int32_t n_anchor,
                      uint8_t *roles, float *importance, double *vs_out, double *hs_out)
{
    const int nh = layers * kv_heads, nq = nh * group;
    if (layers < 1 || kv_heads < 1 || group < 1 || n < 1 || top_k < 1 || n_voice < 0 || n_voice > nh || n_anchor < 0 ||
        n_anchor > n_voice)
        return triage_fail(WNW_ERR_INVALID, "bad sizes or counts");
    if (!sample || !hits || !sens || !roles || !importance) return triage_fail(WNW_ERR_INVALID, "NULL pointer");
    int ns = 0;
    for (int i = 0; i < n; ++i) {
        if (sample[i] < 0) return triage_fail(WNW_ERR_INVALID, "negative sample id");
        ns = std::max(ns, sample[i] + 1);
    }
    // per-sample means, then the mean over the samples present
    std::vector<double> hsum((size_t)ns * nq, 0.0), ssum((size_t)ns * nh, 0.0);
    std::vector<int> cnt(ns, 0);
    for (int i = 0; i < n; ++i) {
        const int s = sample[i];
        ++cnt[s];
        for (int m = 0; m < nq; ++m) hsum[(size_t)s * nq + m] += (double)hits[(size_t)i * nq + m] / top_k;
        for (int m = 0; m < nh; ++m) ssum[(size_t)s * nh + m] += (double)sens[(size_t)i * nh + m];
    }
    std::vector<double> hq(nq, 0.0), hs(nh, 0.0), vs(nh, 0.0), imp(nh);
    int used = 0;
    for (int s = 0; s < ns; ++s) {
        if (!cnt[s]) continue;
        ++used;
        for (int m = 0; m < nq; ++m) hq[m] += hsum[(size_t)s * nq + m] / cnt[s];
        for (int m = 0; m < nh; ++m) hs[m] += ssum[(size_t)s * nh + m] / cnt[s];
    }
    for (int m = 0; m < nq; ++m) hq[m] /= used;
    for (int m = 0; m < nh; ++m) hs[m] /= used;
    double mx = 0.0;
    for (int h = 0; h < nh; ++h) {
        double a = 0.0;
        for (int j = 0; j < group; ++j) a += hq[(size_t)h * group + j];
        vs[h] = a / group;
        imp[h] = vs[h] * hs[h];
        mx = std::max(mx, imp[h]);
    }
    std::vector<int> order(nh);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return imp[a] > imp[b]; });
    for (int r = 0; r < nh; ++r) roles[order[r]] = r < n_anchor ? WNW_ANCHOR : r < n_voice ? WNW_TIDAL : WNW_FIXED;
    for (int h = 0; h < nh; ++h) {
        importance[h] = mx > 0.0 ? (float)(imp[h] / mx) : 0.f;
        if (vs_out) vs_out[h] = vs[h];
        if (hs_out) hs_out[h] = hs[h];
    }
    return WNW_OK;
}

}  // extern "C"
