// Head triage arithmetic (Method, "Head Functional Triage via Offline Calibration", with the
// calibration score details of the appendix), on given inputs: the answer tokens' queries and a
// sample's keys, their aligned audio intervals, and the loss gradients at the audio keys.  The
// model, the alignment and the autograd that produce those are outside the library.
//
//   voice_hits_kernel   per (answer token, q-head): the K audio positions with the largest
//                       logit (softmax keeps the order), ties to the lower position, counted
//                       inside the token's interval.  Logits are exact bf16 products summed in
//                       double on the matrix cores; a sum of 128 products (16 significant bits
//                       each) rounds only when their magnitudes span more than ~30 binary
//                       orders, so the top-K decisions are in practice those of the exact logits.
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

constexpr int VH_ROWS = 64;   // (token, q-head) rows per work-group (16 per wavefront)
constexpr int VH_TILE = 16;   // keys staged in LDS per iteration (as doubles): one MFMA key block
static_assert(VH_TILE * (D / 8) % NT == 0, "whole 16-byte pieces per thread");
constexpr int VH_KMAX = 8;    // largest K (the paper uses 4 and 8)
static_assert(VH_TILE % 16 == 0, "whole 16-key blocks per tile");
typedef double v4d __attribute__((ext_vector_type(4)));

__device__ inline void bf16x2(uint32_t u, double &lo, double &hi)
{
    lo = (double)__uint_as_float(u << 16);
    hi = (double)__uint_as_float(u & 0xffff0000u);
}

// Work-groups: ceil(n_tok * g / VH_ROWS) row blocks per KV-head (row = answer token * g + q-head
// of the group), in XCD order so that the row blocks of one KV-head read its keys through one L2.
// Wavefront w owns 16 rows of the block.  The logits run on v_mfma_f64_16x16x4f64 (lane
// l = i + 16k supplies A[i][k] and B[k][i]; D[i][j] lands in lane j + 16 (i % 4), element i / 4):
// A is a block of 16 keys from the staged tile, B the wavefront's 16 query rows (converted to
// double once and held in registers), and lane group k feeds dimension 32k + s at step s.  Every
// key element is read from shared memory once per wavefront.  A lane ends a key block holding
// four logits of its row (keys k + 4v) and keeps the best eight of the keys it sees (value
// descending; equal values keep the earlier, lower, position); the four lists of a row (one per
// lane group) are merged at the end.  Products of bf16 values are exact in double.
__device__ inline int vh_xcd_order(int w, int n)
{
    const int q = n / 8, r = n % 8, x = w % 8;
    return x * q + min(x, r) + w / 8;
}

__global__ __launch_bounds__(NT, 4) void voice_hits_kernel(int L, int Hq, int Hkv, int T, int Ta, int n_tok, int K,
                                                       const uint16_t *__restrict__ k, const uint16_t *__restrict__ q,
                                                       const int32_t *__restrict__ span, int32_t *__restrict__ hits)
{
    const int g = Hq / Hkv, R = n_tok * g, nrb = (R + VH_ROWS - 1) / VH_ROWS;
    const int v = vh_xcd_order(blockIdx.x, gridDim.x), lk = v / nrb, rblk = v - lk * nrb;
    const int l = lk / Hkv, kv = lk - l * Hkv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kq = lane >> 4, li = lane & 15;
    const int r0 = rblk * VH_ROWS + wave * 16;
    // B operand: row r0 + li, dimensions 32 kq .. + 32
    double qd[32];
    {
        const int ra = r0 + li;
        const bool ok = ra < R;
        const int t = ok ? ra / g : 0, j = ok ? ra - t * g : 0;
        const uint4 *qrow = (const uint4 *)(q + (((size_t)t * L + l) * Hq + (size_t)kv * g + j) * D) + kq * 4;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint4 w = ok ? qrow[u] : make_uint4(0, 0, 0, 0);
            const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) bf16x2(d[e], qd[8 * u + 2 * e], qd[8 * u + 2 * e + 1]);
        }
    }
    double best[VH_KMAX];
    int bpos[VH_KMAX];
#pragma unroll
    for (int i = 0; i < VH_KMAX; ++i) {
        best[i] = -INFINITY;
        bpos[i] = INT32_MAX;
    }
    auto insert = [&](double val, int pos) {
        if (val > best[VH_KMAX - 1]) {
#pragma unroll
            for (int s = 0; s < VH_KMAX; ++s)
                if (val > best[s]) {
                    const double tv = best[s];
                    const int tp = bpos[s];
                    best[s] = val;
                    bpos[s] = pos;
                    val = tv;
                    pos = tp;
                }
        }
    };
    // key tile staged as doubles (each element converted once per work-group): key r, dimension
    // 32 kq + s at r * VH_KS + kq * 33 + s; the padding puts the 16 keys that one lane group reads
    // at a step on distinct banks.  After the loop the same memory holds the candidate lists.
    constexpr int VH_KS = 4 * 33 + 1;
    constexpr int TILE_DBL = VH_TILE * VH_KS, LIST_DBL = VH_ROWS * 4 * VH_KMAX * 3 / 2;   // lists: double + int
    __shared__ double ksd[TILE_DBL > LIST_DBL ? TILE_DBL : LIST_DBL];
    const uint16_t *Kh = k + (size_t)lk * T * D;
    // The next tile's keys are loaded into registers while the current tile is computed (each
    // thread holds VH_PF 16-byte pieces), then converted into the single shared buffer.
    constexpr int VH_PF = VH_TILE * (D / 8) / NT;
    uint4 pf[VH_PF];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int j = 0; j < VH_PF; ++j) {
            const int i = tid + j * NT, row = k0 + (i >> 4);
            pf[j] = row < Ta ? *(const uint4 *)(Kh + (size_t)row * D + (i & 15) * 8) : make_uint4(0, 0, 0, 0);
        }
    };
    fetch(0);
    for (int k0 = 0; k0 < Ta; k0 += VH_TILE) {
        __syncthreads();   // every wavefront is done with the previous tile
#pragma unroll
        for (int j = 0; j < VH_PF; ++j) {
            const int i = tid + j * NT, rr = i >> 4, c = i & 15;
            const uint32_t d[4] = {pf[j].x, pf[j].y, pf[j].z, pf[j].w};
            double *dst = ksd + rr * VH_KS + (c >> 2) * 33 + (c & 3) * 8;   // dimensions 8c .. 8c + 8
#pragma unroll
            for (int e = 0; e < 4; ++e) bf16x2(d[e], dst[2 * e], dst[2 * e + 1]);
        }
        __syncthreads();
        if (k0 + VH_TILE < Ta) fetch(k0 + VH_TILE);
        const int nk = min(VH_TILE, Ta - k0);
        for (int kb = 0; kb < nk; kb += 16) {
            // A: key k0 + kb + li, dimension 32 kq + s
            const double *ga = ksd + (kb + li) * VH_KS + kq * 33;
            v4d acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int s2 = 0; s2 < 32; ++s2) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(ga[s2], qd[s2], acc, 0, 0, 0);
            // this lane: row r0 + li, keys k0 + kb + kq + 4 e
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int p = k0 + kb + kq + 4 * e;
                if (p < Ta) insert(acc[e], p);
            }
        }
    }
    __syncthreads();   // the tile's memory takes the candidate lists
    double (*sbest)[4 * VH_KMAX] = reinterpret_cast<double (*)[4 * VH_KMAX]>(ksd);
    int (*spos)[4 * VH_KMAX] = reinterpret_cast<int (*)[4 * VH_KMAX]>(ksd + VH_ROWS * 4 * VH_KMAX);
    const int rl = wave * 16 + li;   // this lane's row within the block
#pragma unroll
    for (int i = 0; i < VH_KMAX; ++i) {
        sbest[rl][kq * VH_KMAX + i] = best[i];
        spos[rl][kq * VH_KMAX + i] = bpos[i];
    }
    __syncthreads();
    const int rg = rblk * VH_ROWS + tid;
    if (tid < VH_ROWS && rg < R) {
        // top K of the row's candidates by (value descending, position ascending)
        const int t = rg / g, j = rg - t * g;
        const int a = span[2 * t], b = span[2 * t + 1];
        unsigned taken = 0;
        int c = 0;
        for (int n = 0; n < K; ++n) {
            int bi = -1;
            for (int i = 0; i < 4 * VH_KMAX; ++i) {
                if (taken >> i & 1u) continue;
                if (bi < 0 || sbest[tid][i] > sbest[tid][bi] ||
                    (sbest[tid][i] == sbest[tid][bi] && spos[tid][i] < spos[tid][bi]))
                    bi = i;
            }
            taken |= 1u << bi;
            const int pos = spos[tid][bi];
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
    if ((int64_t)n_tok * g > INT32_MAX) return triage_fail(WNW_ERR_UNSUPPORTED, "too many answer-token rows");
    if (top_k < 1 || top_k > VH_KMAX || top_k > audio_len)
        return triage_fail(WNW_ERR_INVALID, "top_k must be in 1..8 and at most audio_len");
    if (n_tok == 0) return WNW_OK;
    if (!k_dev || !q_dev || !span_dev || !hits_dev) return triage_fail(WNW_ERR_INVALID, "NULL pointer");
    const int64_t nrb = ((int64_t)n_tok * g + VH_ROWS - 1) / VH_ROWS, nwg = nrb * layers * kv_heads;
    if (nwg > INT32_MAX) return triage_fail(WNW_ERR_UNSUPPORTED, "too many answer tokens for one launch");
    hipLaunchKernelGGL(voice_hits_kernel, dim3((unsigned)nwg), dim3(NT), 0,
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
