// HIP kernels of the WnW decode step for CDNA4 (gfx950).
//
// Work decomposition (all kernels are launched by wnw_api.hip on the caller's stream, the
// recall on a side stream):
//   anchor_attn     one work-group per (sequence, anchor KV-head, tile of TILE_A key rows): the
//                   g q-heads' logits, the tile max, exp, the per-chunk softmax mass (Eq. 2) and
//                   the unnormalised P.V partial.  Logits and masses are kept in double: the
//                   chunk ranking must agree with an fp64 reference to well under 1e-6.
//   attention       (next-step timing) anchor tiles and the static tidal/fixed tiles in one launch.
//   anchor_mass     log-sum-exp normalisers of one anchor head's tiles and its normalised
//                   chunk masses (summed over its q-heads), for the selection.
//   scores          per chunk: fixed-order sum over anchor q-heads / chunk length (mean).
//   select          one work-group per sequence: top-k by (score desc, id asc), streaks,
//                   residency, slot assignment, kept/new lists.
//   tidal_fixed     tidal and fixed heads over their kept rows + text, and tidal heads over the
//                   complements already in their slots (fp32 logits).
//                   With same-step timing its first work-groups recall: they copy newly resident
//                   complements from mapped pinned host memory into their slots and attend to them.
//   recall_copy     next-step recall (side stream): the copy only.
//   subset_combine  final merge: a tidal/fixed head's partials, or an anchor head's tiles, into
//                   output rows.
//
// Layout inside a tile: 16 lanes share one 256-byte key row (8 bf16 = 16 bytes each), so one
// wavefront load moves 4 rows (1 KiB) fully coalesced.  A wavefront owns RPL such 4-row steps
// and issues all of its K and V loads before computing, so every wavefront keeps 2 * RPL KiB in
// flight.  Dot products are reduced across the 16 lanes of a row with DPP row permutes.
#include "wnw_internal.h"

#include <hip/hip_ext.h>

#include <math.h>

#include <algorithm>
#include <atomic>

namespace wnw {

namespace {

constexpr int WAVES = NT / 64;
constexpr double SCALE_D = 0.088388347648318440550;   // 1 / sqrt(128)
constexpr float SCALE_F = 0.08838834764831845f;

__device__ inline void unpack8(const uint4 u, float f[8])
{
    f[0] = __uint_as_float(u.x << 16); f[1] = __uint_as_float(u.x & 0xffff0000u);
    f[2] = __uint_as_float(u.y << 16); f[3] = __uint_as_float(u.y & 0xffff0000u);
    f[4] = __uint_as_float(u.z << 16); f[5] = __uint_as_float(u.z & 0xffff0000u);
    f[6] = __uint_as_float(u.w << 16); f[7] = __uint_as_float(u.w & 0xffff0000u);
}

// DPP permutes inside a 16-lane row: quad_perm [1,0,3,2] (xor 1), quad_perm [2,3,0,1] (xor 2),
// row_half_mirror (lane i <-> 7-i inside each 8) and row_mirror (i <-> 15-i).  After the four
// add steps every lane of the row holds the same, bitwise identical sum.
template <int CTRL>
__device__ inline float dpp(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ inline double dpp(double v)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(u & 0xffffffffull), CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(u >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
template <typename T>
__device__ inline T sum16(T v)
{
    v += dpp<0xB1>(v);
    v += dpp<0x4E>(v);
    v += dpp<0x141>(v);
    v += dpp<0x140>(v);
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
//
// Loads: K and V rows are read fully coalesced (one wavefront instruction = 4 whole rows) with
// nontemporal loads (every byte is read once per step).  Each wavefront owns 32 rows of the tile.
//
// Logits come from v_mfma_f64_4x4x4f64 (four independent 4x4x4 blocks per wavefront).  On
// gfx950 lane l = 16k + 4*blk + x holds A_blk[x][k] and B_blk[k][x], and the result
// D_blk[i][j] lands in lane 16i + 4*blk + j.  With A = key rows and B = q^T, one instruction
// multiplies 16 keys (4 per block) by 4 q-heads over 4 dimensions; lane l feeds dimension 32k + t
// to instruction t, so it needs 64 contiguous bytes of its key row.  The coalesced K rows reach
// that layout through a per-wavefront LDS region whose 16-byte units are XOR-swizzled by the row
// (unit p of row r at r*16 + (p ^ (r & 15))), so both the stores and the operand reads are free
// of bank conflicts.  For groups of 6 or 8 q-heads, blocks 0-1 take heads 0-3 and blocks 2-3
// heads 4-7 over the same 8 keys.  Products of bf16 values are exact in double, so the logits
// match a double reference to rounding.
//
// Softmax: the four wavefronts agree on the tile maximum M (one barrier) before any exp, so the
// probabilities, their sums, the chunk masses and the P.V partials all share M and merge by
// plain sums.  exp(y) is evaluated as 2^n * 2^f with n = rint(y log2 e) and f in [-1/2, 1/2]
// taken in double and 2^f by the hardware exp2 in fp32 (relative error ~1e-7).
//
// P.V runs on v_mfma_f32_4x4x1 (16 blocks): lane l = 4*blk + j feeds B_blk[0][j] = its own V
// element (row 4i + rg, dimension 8*sub + e) and A_blk[h][0] = P[h][row 4i + rg] with h = l & 3,
// so D_blk[h][j] accumulates, per lane, the same sums a per-lane FMA loop would.
// -------------------------------------------------------------------------------------------
__device__ inline uint4 load_nt(const uint16_t *p)
{
    typedef unsigned v4u __attribute__((ext_vector_type(4)));
    const v4u a = __builtin_nontemporal_load((const v4u *)p);
    return make_uint4(a.x, a.y, a.z, a.w);
}

// Raw buffer loads for the streamed K/V tiles: the base and the byte count of a head's valid rows
// sit in scalar registers and each lane adds one 32-bit offset (the row offsets fold into the
// instruction's immediate), which saves the per-load 64-bit address arithmetic and the zeroing of
// registers that a conditional load needs; offsets at or past the byte count read zeros.  The
// K/V arrays also carry zeroed rows past every head's valid rows (reserved rows, a padding tile
// at the end), so a tile's tail reads finite data inside the allocation in any case.
// aux 2 = nontemporal (every byte is read once per step).
__device__ inline __amdgpu_buffer_rsrc_t buf_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ inline uint4 buf_load_nt(__amdgpu_buffer_rsrc_t r, unsigned off)
{
    typedef unsigned v4u __attribute__((ext_vector_type(4)));
    const v4u a = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 2));
    return make_uint4(a.x, a.y, a.z, a.w);
}

// exp(y) for y <= 0 (see above); 0 below 2^-1022
__device__ inline double exp_nonpos(double y)
{
    const double tt = y * 1.4426950408889634074;
    const double n = rint(tt);
    const float e = __builtin_amdgcn_exp2f((float)(tt - n));
    return tt < -1022.0 ? 0.0 : ldexp((double)e, (int)n);
}

// Thread index as a value the compiler may not treat as loop-invariant: tiles run inside
// grid-stride loops, and hoisting every lane-dependent index out of the loop would keep them all
// live across the tile and spill registers.
__device__ inline int lane_id_opaque()
{
    int tid = threadIdx.x;
    __asm__ volatile("" : "+v"(tid));
    return tid;
}

// Shared memory of one anchor tile.
// Values that pass between work-groups of one launch (the chunk masses, from the work-groups that
// merge them to the selection in the same launch, see last_arrival) are stored and loaded as
// agent-scope relaxed atomics: coherent across the dies' caches with no cache write-back or
// invalidation, which an agent-scope fence would cost every work-group.
__device__ inline void st_agent(double *p, double v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline double ld_agent(const double *p)
{
    return __hip_atomic_load(const_cast<double *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int G>
struct AnchorSmem {
    static constexpr int RW = TILE_A / WAVES;
    uint4 kst[WAVES][RW * 16];                // swizzled K rows; afterwards the P.V partials
    double xs[G * TILE_A];                    // probabilities (per-row chunk masses only)
    float xf[G * TILE_A];                     // probabilities in fp32, for P.V
    double wm[WAVES * G], wl[WAVES * G];
};

template <int G>
__device__ inline void anchor_tile(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *__restrict__ q,
                                   int tile, int ai, int b, AnchorSmem<G> &sm)
{
    typedef float v4f __attribute__((ext_vector_type(4)));
    constexpr int HG = G <= 4 ? 1 : 2;        // groups of 4 q-heads per logit instruction
    constexpr int KG = 16 / HG;               // keys per logit instruction
    constexpr int RW = TILE_A / WAVES;        // key rows per wavefront (32)
    constexpr int NKG = RW / KG;              // key groups per wavefront (2 or 4)
    constexpr int RPL = RW / 4;               // coalesced 4-row steps per wavefront
    constexpr int OGR = G <= 4 ? 4 : 2;       // row groups kept in the P.V partial store
    constexpr int HS = (G + 3) / 4;           // sets of 4 heads for P.V
    static_assert(NKG % 2 == 0, "key groups are processed in pairs");
    const int tid = lane_id_opaque(), lane = tid & 63, wave = tid >> 6, sub = lane & 15, rg = lane >> 4;
    const int kq = lane >> 4, blk = (lane >> 2) & 3, x4 = lane & 3;
    const int lk = t.anchor_lk[ai], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const size_t hrow = ((size_t)b * g.nA + ai) * (size_t)g.Tcap;
    const uint16_t *__restrict__ K = t.aK + hrow * D;
    const uint16_t *__restrict__ V = t.aV + hrow * D;
    const uint16_t *__restrict__ qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    const int t0 = tile * TILE_A;
    // chunk masses from wavefront sums when every wavefront's audio rows lie in one chunk and no
    // wavefront of this tile straddles the audio/text boundary
    const bool fast_mass = g.cl % RW == 0 && !(t0 < g.Ta && g.Ta < t0 + TILE_A && g.Ta % RW != 0);

    auto &kst = sm.kst;
    double *xs = sm.xs, *wm = sm.wm, *wl = sm.wl;
    float *xf = sm.xf;
    float *wo = (float *)&kst[wave][0];       // [OGR][G][D] of this wavefront

    // q (B operand: head hB, dims 32kq..32kq+31), then K and V rows
    const int hB = (HG == 1 ? 0 : (blk >> 1) * 4) + x4;
    uint4 qr[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
        qr[u] = hB < G ? *(const uint4 *)(qh + hB * D + kq * 32 + u * 8) : make_uint4(0, 0, 0, 0);
    uint4 kr[RPL], vr[RPL];
    {
        // rows at or past T read zeros
        const __amdgpu_buffer_rsrc_t rk = buf_rsrc(K, (unsigned)g.T * (D * 2)), rv = buf_rsrc(V, (unsigned)g.T * (D * 2));
        const unsigned o0 = (unsigned)(t0 + wave * RW + rg) * (D * 2) + sub * 16;
#pragma unroll
        for (int i = 0; i < RPL; ++i) kr[i] = buf_load_nt(rk, o0 + i * (4 * D * 2));
#pragma unroll
        for (int i = 0; i < RPL; ++i) vr[i] = buf_load_nt(rv, o0 + i * (4 * D * 2));
    }
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
        const int r = i * 4 + rg;
        kst[wave][r * 16 + (sub ^ (r & 15))] = kr[i];
    }
    // each wavefront reads back only its own rows: a wavefront-scope fence suffices
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // logits of (key keyD, head hD) per key group; key groups in pairs, four accumulator chains
    const int keyA = (HG == 1 ? blk * 4 : (blk & 1) * 4) + x4;
    const int keyD = (HG == 1 ? blk * 4 : (blk & 1) * 4) + kq;
    const int hD = (HG == 1 ? 0 : (blk >> 1) * 4) + x4;
    double xv[NKG];
#pragma unroll
    for (int kp = 0; kp < NKG; kp += 2) {
        double a00 = 0.0, a01 = 0.0, a10 = 0.0, a11 = 0.0;
        const int r0 = kp * KG + keyA, r1 = r0 + KG;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint4 k0 = kst[wave][r0 * 16 + ((kq * 4 + u) ^ (r0 & 15))];
            const uint4 k1 = kst[wave][r1 * 16 + ((kq * 4 + u) ^ (r1 & 15))];
            float f0[8], f1[8], qf[8];
            unpack8(k0, f0);
            unpack8(k1, f1);
            unpack8(qr[u], qf);
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const double qa = (double)qf[e], qb = (double)qf[e + 1];
                a00 = __builtin_amdgcn_mfma_f64_4x4x4f64((double)f0[e], qa, a00, 0, 0, 0);
                a10 = __builtin_amdgcn_mfma_f64_4x4x4f64((double)f1[e], qa, a10, 0, 0, 0);
                a01 = __builtin_amdgcn_mfma_f64_4x4x4f64((double)f0[e + 1], qb, a01, 0, 0, 0);
                a11 = __builtin_amdgcn_mfma_f64_4x4x4f64((double)f1[e + 1], qb, a11, 0, 0, 0);
            }
        }
        const int rr0 = t0 + wave * RW + kp * KG + keyD;
        xv[kp] = (hD < G && rr0 < g.T) ? (a00 + a01) * SCALE_D : -INFINITY;
        xv[kp + 1] = (hD < G && rr0 + KG < g.T) ? (a10 + a11) * SCALE_D : -INFINITY;
    }
    // wavefront maximum per head (lanes of one head differ in bits 2, 4, 5, and 3 when all four
    // blocks share the heads), then the tile maximum over the four wavefronts
    double m = xv[0];
#pragma unroll
    for (int kg = 1; kg < NKG; ++kg) m = fmax(m, xv[kg]);
    m = fmax(m, __shfl_xor(m, 4));
    if (HG == 1) m = fmax(m, __shfl_xor(m, 8));
    m = fmax(m, __shfl_xor(m, 16));
    m = fmax(m, __shfl_xor(m, 32));
    const bool head_lane = hD < G && kq == 0 && (HG == 1 ? blk == 0 : (blk & 1) == 0);
    if (head_lane) wm[wave * G + hD] = m;
    __syncthreads();
    if (hD < G) {
#pragma unroll
        for (int w = 0; w < WAVES; ++w) m = fmax(m, wm[w * G + hD]);
    }
    double lsum = 0.0;
#pragma unroll
    for (int kg = 0; kg < NKG; ++kg) {
        const double pv = (m == -INFINITY || xv[kg] == -INFINITY) ? 0.0 : exp_nonpos(xv[kg] - m);
        if (hD < G) {
            const int rr = wave * RW + kg * KG + keyD;
            if (!fast_mass) xs[hD * TILE_A + rr] = pv;
            xf[hD * TILE_A + rr] = (float)pv;
        }
        lsum += pv;
    }
    lsum += __shfl_xor(lsum, 4);
    if (HG == 1) lsum += __shfl_xor(lsum, 8);
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    if (head_lane) wl[wave * G + hD] = lsum;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // P.V (unnormalised, relative to M) on the matrix cores
    v4f dacc[HS][8];
#pragma unroll
    for (int hs = 0; hs < HS; ++hs)
#pragma unroll
        for (int e = 0; e < 8; ++e) dacc[hs][e] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
        const int rr = wave * RW + i * 4 + rg;
        float f[8];
        unpack8(vr[i], f);
#pragma unroll
        for (int hs = 0; hs < HS; ++hs) {
            const int h = hs * 4 + (lane & 3);
            const float pa = h < G ? xf[h * TILE_A + rr] : 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) dacc[hs][e] = __builtin_amdgcn_mfma_f32_4x4x1f32(pa, f[e], dacc[hs][e], 0, 0, 0);
        }
    }
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[h][e] = dacc[h / 4][e][h % 4];
            if (OGR == 2) acc[h][e] += __shfl_xor(acc[h][e], 32);
        }
    if (rg < OGR) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float4 *dst = (float4 *)(wo + (rg * G + h) * D + sub * 8);
            dst[0] = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
            dst[1] = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
        }
    }
    __syncthreads();

    // tile partials: maximum, sum, P.V and per-chunk masses, all relative to M
    const size_t pidx = ((size_t)b * g.nA + ai) * g.n_tiles_a + tile;
    if (tid < G) {
        double M = wm[tid], L = 0.0;
#pragma unroll
        for (int w = 1; w < WAVES; ++w) M = fmax(M, wm[w * G + tid]);
#pragma unroll
        for (int w = 0; w < WAVES; ++w) L += wl[w * G + tid];
        s.pa_m[pidx * G + tid] = M;
        s.pa_l[pidx * G + tid] = L;
    }
    for (int idx = tid; idx < G * D; idx += NT) {
        float o = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            const float *ww = (const float *)&kst[w][0];
#pragma unroll
            for (int r4 = 0; r4 < OGR; ++r4) o += ww[r4 * G * D + idx];
        }
        s.pa_o[pidx * G * D + idx] = o;
    }
    const int c_first = t0 / g.cl;
    if (fast_mass) {
        if (tid < G * g.maxc) {
            const int h = tid / g.maxc, c = c_first + (tid - h * g.maxc);
            double acc2 = 0.0;
#pragma unroll
            for (int w = 0; w < WAVES; ++w) {
                const int r0 = t0 + w * RW;
                if (r0 >= c * g.cl && r0 < (c + 1) * g.cl && r0 < g.Ta) acc2 += wl[w * G + h];
            }
            s.pa_mass[pidx * G * g.maxc + tid] = acc2;
        }
        return;
    }
    // general chunk lengths: 16 lanes per (head, chunk) entry sum a fixed stride of rows, then a
    // DPP sum (fixed order)
    for (int base = 0; base < G * g.maxc * 16; base += NT) {
        const int idx = base + tid, grp = idx >> 4, k = idx & 15;
        const bool valid = grp < G * g.maxc;
        double acc2 = 0.0;
        if (valid) {
            const int h = grp / g.maxc, c = c_first + (grp - h * g.maxc);
            const int r0 = max(c * g.cl, t0), r1 = min(min((c + 1) * g.cl, t0 + TILE_A), g.Ta);
            for (int rr = r0 + k; rr < r1; rr += 16) acc2 += xs[h * TILE_A + (rr - t0)];
        }
        acc2 = sum16(acc2);
        if (valid && k == 0) s.pa_mass[pidx * G * g.maxc + grp] = acc2;
    }
}

template <int G>
__global__ __launch_bounds__(NT, G <= 4 ? 4 : 2) void anchor_attn_kernel(Geometry g, Tiers t, StepBuffers s,
                                                                         const uint16_t *__restrict__ q)
{
    __shared__ AnchorSmem<G> sm;
    anchor_tile<G>(g, t, s, q, blockIdx.x, blockIdx.y, blockIdx.z, sm);
}

constexpr int COMBINE_THREADS = 1024;

// One output element: fp32, or bf16 rounded to nearest (ties to even; NaN stays a quiet NaN).
__device__ inline void store_out(void *out, size_t i, float v, bool bf16)
{
    if (!bf16) {
        static_cast<float *>(out)[i] = v;
        return;
    }
    const unsigned u = __float_as_uint(v);
    const unsigned r = (u & 0x7fffffffu) > 0x7f800000u ? 0x7fc0u : (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    static_cast<uint16_t *>(out)[i] = (uint16_t)r;
}

// Block-wide max / sum of G values per thread (THREADS threads, in double).
template <int G, int THREADS>
__device__ inline void block_reduce_g(double v[G], bool is_max, double (*red)[G])
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int h = 0; h < G; ++h) {
        v[h] = is_max ? wave_max(v[h]) : wave_sum(v[h]);
        if (lane == 0) red[wave][h] = v[h];
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
        double m = red[0][h];
        for (int w = 1; w < THREADS / 64; ++w) m = is_max ? fmax(m, red[w][h]) : m + red[w][h];
        v[h] = m;
    }
    __syncthreads();
}

constexpr int MASS_THREADS = 256;

// Chunk masses of one anchor KV-head (the part of the anchor merge that the selection needs):
// the log-sum-exp normalisers of its G q-heads from the tile partials, kept for the output merge
// (anchor_out_merge, in the final launch), and the normalised per-chunk softmax mass of Eq. 2
// summed over the G q-heads in order, all in double.
// Shared memory of anchor_mass_head besides fac[G][n_tiles_a].
template <int G>
struct MassSmem {
    double red[MASS_THREADS / 64][G];
    double inv_l[G];
};

// One anchor KV-head ai of sequence b, MASS_THREADS threads; fac: [G][n_tiles_a] doubles of
// shared memory.
static_assert(MASS_THREADS == NT, "the attention launch's work-groups merge the chunk masses");
template <int G>
__device__ inline void anchor_mass_head(const Geometry &g, const StepBuffers &s, int ai, int b, double *fac,
                                        MassSmem<G> &ms)
{
    const int tid = threadIdx.x;
    auto &red = ms.red;
    double *inv_l = ms.inv_l;
    const int nt = g.n_tiles_a;
    const size_t base = ((size_t)b * g.nA + ai) * nt;
    // a segment of at most MAX_CHUNK positions spans at most MAXT tiles
    constexpr int MAXT = (MAX_CHUNK + TILE_A - 2) / TILE_A + 1;
    // every load of the first round (this thread's tile maxima and sums, its segment's mass
    // partials) is issued before any is used: one memory round trip for caches of up to
    // MASS_THREADS tiles and segments
    double pm[G], pl[G], v[G][MAXT];
    const int c0 = tid, t_lo0 = c0 < g.nc ? (c0 * g.cl) / TILE_A : 0;
    const int t_hi0 = c0 < g.nc ? (min((c0 + 1) * g.cl, g.Ta) - 1) / TILE_A : -1;
#pragma unroll
    for (int h = 0; h < G; ++h) {
        pm[h] = tid < nt ? s.pa_m[(base + tid) * G + h] : -INFINITY;
        pl[h] = tid < nt ? s.pa_l[(base + tid) * G + h] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < MAXT; ++u) {
        const int i = t_lo0 + u, j = c0 - (i * TILE_A) / g.cl;
#pragma unroll
        for (int h = 0; h < G; ++h) v[h][u] = i <= t_hi0 ? s.pa_mass[((base + i) * G + h) * g.maxc + j] : 0.0;
    }
    double m[G], l[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = pm[h];
        if (tid < nt) fac[h * nt + tid] = pm[h];
    }
    for (int i = tid + MASS_THREADS; i < nt; i += MASS_THREADS)
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const double x = s.pa_m[(base + i) * G + h];
            fac[h * nt + i] = x;
            m[h] = fmax(m[h], x);
        }
    block_reduce_g<G, MASS_THREADS>(m, true, red);
#pragma unroll
    for (int h = 0; h < G; ++h) {
        l[h] = 0.0;
        if (tid < nt) {
            const double f = (m[h] > -INFINITY && pm[h] > -INFINITY) ? exp(pm[h] - m[h]) : 0.0;
            fac[h * nt + tid] = f;
            l[h] = pl[h] * f;
        }
    }
    for (int i = tid + MASS_THREADS; i < nt; i += MASS_THREADS)
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const double mi = fac[h * nt + i];
            const double f = (m[h] > -INFINITY && mi > -INFINITY) ? exp(mi - m[h]) : 0.0;
            fac[h * nt + i] = f;
            l[h] += s.pa_l[(base + i) * G + h] * f;
        }
    block_reduce_g<G, MASS_THREADS>(l, false, red);   // also publishes fac[]
    if (tid < G) {
        double M = m[0], L = l[0];
#pragma unroll
        for (int h = 1; h < G; ++h)
            if (tid == h) M = m[h], L = l[h];
        const double inv = L > 0.0 ? 1.0 / L : 0.0;
        inv_l[tid] = inv;
        s.a_stat[(((size_t)b * g.nA + ai) * G + tid) * 2] = M;
        s.a_stat[(((size_t)b * g.nA + ai) * G + tid) * 2 + 1] = inv;
    }
    __syncthreads();
    double *mass = s.mass + ((size_t)b * g.nA + ai) * (size_t)g.nc;
    for (int c = c0; c < g.nc; c += MASS_THREADS) {
        const int t_lo = (c * g.cl) / TILE_A, t_hi = (min((c + 1) * g.cl, g.Ta) - 1) / TILE_A;
        if (c != c0) {
#pragma unroll
            for (int u = 0; u < MAXT; ++u) {
                const int i = t_lo + u, j = c - (i * TILE_A) / g.cl;
#pragma unroll
                for (int h = 0; h < G; ++h) v[h][u] = i <= t_hi ? s.pa_mass[((base + i) * G + h) * g.maxc + j] : 0.0;
            }
        }
        double acc = 0.0;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            double a = 0.0;
#pragma unroll
            for (int u = 0; u < MAXT; ++u)
                if (t_lo + u <= t_hi) a += v[h][u] * fac[h * nt + t_lo + u];
            acc += a * inv_l[h];
        }
        st_agent(&mass[c], acc);
    }
}

template <int G>
__global__ __launch_bounds__(MASS_THREADS) void anchor_mass_kernel(Geometry g, StepBuffers s)
{
    extern __shared__ double fac[];      // [G][n_tiles_a]
    __shared__ MassSmem<G> ms;
    anchor_mass_head<G>(g, s, blockIdx.x, blockIdx.y, fac, ms);
}

// Output rows of one anchor KV-head's G q-heads from the tile partials and the normalisers
// anchor_mass_kernel kept (COMBINE_THREADS threads, one work-group of the final merge launch):
// per 16-byte column of the G * d outputs, the tiles are split over groups of threads summed in
// a fixed order, in double.  fac: [G][n_tiles_a] doubles of shared memory.
template <int G>
__device__ inline void anchor_out_merge(const Geometry &g, const Tiers &t, const StepBuffers &s, void *out, int ai,
                                        int b, double *fac, double *opart)
{
    constexpr int NC4 = G * D / 4, GR = COMBINE_THREADS / NC4;   // 16-byte columns, groups
    const int tid = threadIdx.x, nt = g.n_tiles_a;
    const size_t base = ((size_t)b * g.nA + ai) * nt;
    const double *st = s.a_stat + ((size_t)b * g.nA + ai) * G * 2;
    const int col = tid % NC4, grp = tid / NC4, h = col / (D / 4);
    const int i0 = grp * nt / GR, i1 = grp < GR ? (grp + 1) * nt / GR : i0;
    const float4 *po = (const float4 *)s.pa_o;
    // this thread's first PF tile partials are loaded with the maxima (one memory round trip)
    constexpr int PF = G <= 4 ? 8 : 4;
    float4 pf[PF];
#pragma unroll
    for (int u = 0; u < PF; ++u) pf[u] = i0 + u < i1 ? po[(base + i0 + u) * NC4 + col] : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int idx = tid; idx < G * nt; idx += COMBINE_THREADS) {
        const int hh = idx / nt, i = idx - hh * nt;
        const double M = st[hh * 2], mi = s.pa_m[(base + i) * G + hh];
        fac[idx] = (M > -INFINITY && mi > -INFINITY) ? exp(mi - M) : 0.0;
    }
    __syncthreads();
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
    if (grp < GR) {
#pragma unroll
        for (int u = 0; u < PF; ++u)
            if (i0 + u < i1) {
                const double f = fac[h * nt + i0 + u];
                a0 += (double)pf[u].x * f;
                a1 += (double)pf[u].y * f;
                a2 += (double)pf[u].z * f;
                a3 += (double)pf[u].w * f;
            }
#pragma unroll 4
        for (int i = i0 + PF; i < i1; ++i) {
            const float4 v = po[(base + i) * NC4 + col];
            const double f = fac[h * nt + i];
            a0 += (double)v.x * f;
            a1 += (double)v.y * f;
            a2 += (double)v.z * f;
            a3 += (double)v.w * f;
        }
        double *o = opart + ((size_t)grp * NC4 + col) * 4;
        o[0] = a0, o[1] = a1, o[2] = a2, o[3] = a3;
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll 4
        for (int r = 1; r < GR; ++r) {
            const double *o = opart + ((size_t)r * NC4 + col) * 4;
            a0 += o[0], a1 += o[1], a2 += o[2], a3 += o[3];
        }
        const double inv = st[h * 2 + 1];
        const int lk = t.anchor_lk[ai], ll = lk / g.Hkv, kv = lk - ll * g.Hkv;
        const size_t ob = (((size_t)b * g.L + ll) * g.Hq + (size_t)kv * G) * D + (size_t)col * 4;
        store_out(out, ob, (float)(a0 * inv), g.out_bf16);
        store_out(out, ob + 1, (float)(a1 * inv), g.out_bf16);
        store_out(out, ob + 2, (float)(a2 * inv), g.out_bf16);
        store_out(out, ob + 3, (float)(a3 * inv), g.out_bf16);
    }
}

// -------------------------------------------------------------------------------------------
// Chunk scores, selection, residency and slot bookkeeping: one work-group per sequence.
// -------------------------------------------------------------------------------------------
// Work-group barrier for communication through shared memory only: waits for this wavefront's
// shared-memory operations, not for its global stores (the select kernel never reads its global
// outputs back, and waiting for them at every barrier would expose their latency each time).
__device__ inline void lds_barrier()
{
    __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Counters of select_seq in shared memory (and a flag of last_arrival).
struct SelectShared {
    int ndrop, nrows, nrev, nfree, nkrows;
    int last;
};


// Per sequence b (state staged in shared memory, written back at the end).  Chunks (nchk) are
// the selection's candidates; segments (nc) are the unit of masses, residency, slots and
// recall.  With disjoint chunks a chunk is a segment; with overlapping chunks chunk c is
// segments c and c + 1.
//   scores   score_c = (sum over anchor q-heads and the chunk's segments of their mass) / |c|,
//            double, fixed order
//   select   top-k chunks by (fp32 score desc, id asc), or the caller's override
//   streaks  per chunk: 0 when selected, else +1 (capped at delta); a chunk is resident iff its
//            streak < delta, a segment iff a resident chunk covers it
//   attended this step: the resident segments of this step (same-step timing) or of the step
//            before (next-step timing)
//   slots    a segment that stops being resident frees its slot (next-step timing: one step
//            later, after this step's attention has read it); a newly resident segment whose
//            bytes still sit in a free slot (never overwritten since) takes it back with no copy;
//            the others take free slots in least-recently-freed order (never-used slots first)
//            and are listed for recall
//   lists    kept list = attended with bytes already on the device; new list = to recall
//            (attended in the same launch with same-step timing; with next-step timing the new
//            segments also follow the kept ones in the kept list, which the next step attends)
// Any number of threads (blockDim.x, a multiple of 64); sdyn: select_shared_bytes(g) bytes of
// shared memory.
__device__ inline void select_seq(const Geometry &g, const StepBuffers &s, float *__restrict__ scores,
                                  const int32_t *__restrict__ ovr, int32_t *__restrict__ selected, int b, double *sdyn,
                                  SelectShared &sh)
{
    const int tid = threadIdx.x, nthr = blockDim.x;
    const int nu = g.nc, nk = g.nchk, k = g.k, ns = g.n_slots, naq = g.nA;   // mass rows: one per anchor KV-head
    const bool nxt = g.next_step, two = g.span == 2;
    double *part = sdyn;                              // [nu] segment mass sums
    unsigned long long *ckey = (unsigned long long *)(part + nu);       // [nk] ranking keys
    unsigned long long *fkey = (unsigned long long *)(part + 2 * nu);   // [ns] free-slot keys
    float *sc = (float *)(part + 3 * nu);             // [nk] chunk scores
    int *fsel = (int *)(sc + nu);                     // [nk] selected
    int *st = fsel + nu;                              // [nk] streak
    int *sof = st + nu;                               // [nu] slot of the segment or -1
    int *slast = sof + nu;                            // [nu] slot that last received the segment
    int *fnew = slast + nu;                           // [nu] to recall
    int *fkept = fnew + nu;                           // [nu] attended from a slot already filled
    int *fdrop = fkept + nu;                          // [nu] leaves the resident set
    int *rank = fdrop + nu;                           // [nk] rank of a selected chunk
    int *busy = rank + nu;                            // [ns] 0 free, 1 owned, 2 freed after this step
    int *sdata = busy + ns;                           // [ns] segment whose bytes the slot holds
    int *since = sdata + ns;                          // [ns] step at which the slot was freed
    int *skey = since + ns;                           // [ns] ordering key of free slots
    int *freelist = skey + ns;                        // [ns] free slots in order
    int *frank = freelist + ns;                       // [ns] rank of a free slot among the free ones
    int *srows = frank + ns;                          // [nu] complement rows of the segment (all tidal heads)
    int *rank_k = srows + nu;                         // [nu] rank of a kept segment
    int *rank_n = rank_k + nu;                        // [nu] rank of a new segment
    int *bcnt = rank_n + nu;                          // [3][ceil(nu / 64)] flags set per 64-entry block
    int &ndrop = sh.ndrop, &nrows = sh.nrows, &nrev = sh.nrev, &nfree = sh.nfree, &nkrows = sh.nkrows;

    int32_t *g_streak = s.streak + (size_t)b * nk, *g_slot_of = s.slot_of + (size_t)b * nu;
    int32_t *g_slot_last = s.slot_last + (size_t)b * nu;
    int32_t *g_att = s.att + (size_t)b * nu;
    int32_t *g_data = s.slot_data + (size_t)b * ns, *g_busy = s.slot_busy + (size_t)b * ns;
    int32_t *g_since = s.slot_since + (size_t)b * ns;
    const int step = s.step[b];

    // state in: every load of up to IN_ROUNDS rounds of the work-group is issued before any store
    // to shared memory (one memory round trip while the arrays fit)
    constexpr int IN_ROUNDS = 4;
    const int n_in = max(max(nk, nu), ns);
    for (int i00 = 0; i00 < n_in; i00 += IN_ROUNDS * nthr) {
        int v_st[IN_ROUNDS], v_sof[IN_ROUNDS], v_slast[IN_ROUNDS], v_rows[IN_ROUNDS];
        int v_busy[IN_ROUNDS], v_data[IN_ROUNDS], v_since[IN_ROUNDS];
#pragma unroll
        for (int r = 0; r < IN_ROUNDS; ++r) {
            const int i = i00 + r * nthr + tid;
            v_st[r] = i < nk ? g_streak[i] : 0;
            v_sof[r] = i < nu ? g_slot_of[i] : 0;
            v_slast[r] = i < nu ? g_slot_last[i] : 0;
            v_rows[r] = i < nu ? s.seg_rows[(size_t)b * nu + i] : 0;
            v_busy[r] = i < ns ? g_busy[i] : 0;
            v_data[r] = i < ns ? g_data[i] : 0;
            v_since[r] = i < ns ? g_since[i] : 0;
        }
#pragma unroll
        for (int r = 0; r < IN_ROUNDS; ++r) {
            const int i = i00 + r * nthr + tid;
            if (i < nk) {
                st[i] = v_st[r];
                fsel[i] = 0;
            }
            if (i < nu) {
                sof[i] = v_sof[r];
                slast[i] = v_slast[r];
                srows[i] = v_rows[r];
            }
            if (i < ns) {
                busy[i] = v_busy[r] == 2 ? 0 : v_busy[r];   // frees deferred by the previous step
                sdata[i] = v_data[r];
                since[i] = v_since[r];
            }
        }
    }
    // segment masses: the anchor heads' masses of a segment summed over SCORE_PARTS fixed ranges
    // of heads, each in head order, then the ranges' sums in order.  A thread's loads are issued
    // MB at a time before any is added.
    constexpr int MB = 16;
    for (int u = tid; u < nu; u += nthr) {
        const double *m = s.mass + (size_t)b * naq * nu + u;
        double tot = 0.0, acc = 0.0;
        int p = 0, pend = naq / SCORE_PARTS;   // the range being summed and its end
        for (int a = 0; a < naq; a += MB) {
            double v[MB];
#pragma unroll
            for (int e = 0; e < MB; ++e) v[e] = a + e < naq ? ld_agent(m + (size_t)(a + e) * nu) : 0.0;
#pragma unroll
            for (int e = 0; e < MB; ++e) {
                if (a + e >= naq) break;
                while (a + e >= pend) {   // the range ends (ranges are empty when naq < SCORE_PARTS)
                    tot = p == 0 ? acc : tot + acc;
                    acc = 0.0;
                    ++p;
                    pend = (p + 1) * naq / SCORE_PARTS;
                }
                acc += v[e];
            }
        }
        for (; p < SCORE_PARTS; ++p) {
            tot = p == 0 ? acc : tot + acc;
            acc = 0.0;
        }
        part[u] = tot;
    }
    if (tid == 0) ndrop = nrows = nrev = nfree = nkrows = 0;
    lds_barrier();
    for (int c = tid; c < nk; c += nthr) {
        const bool pair = two && c + 1 < nu;
        const double acc = pair ? part[c] + part[c + 1] : part[c];
        const int len = chunk_len_of(g, c) + (pair ? chunk_len_of(g, c + 1) : 0);
        const float v = (float)(acc / (double)len);
        sc[c] = v;
        scores[(size_t)b * nk + c] = v;
        // ranking key: the fp32 score's bits made order-preserving, then the complement of the
        // id, so that a larger key is a higher score, or an equal score and a lower id
        unsigned u32 = v == 0.f ? 0u : __float_as_uint(v);   // -0 ranks as +0
        u32 = (u32 >> 31) ? ~u32 : u32 | 0x80000000u;
        ckey[c] = ((unsigned long long)u32 << 32) | (0xffffffffu - (unsigned)c);
    }
    lds_barrier();

    // selection
    if (ovr) {
        for (int i = tid; i < k; i += nthr) {
            const int c = ovr[(size_t)b * k + i];
            if (c >= 0 && c < nk) fsel[c] = 1;
        }
    } else {
        // rank of every chunk among all (the number of larger keys): P adjacent lanes per chunk
        // each compare it with a contiguous share of the chunks (independent shared-memory
        // reads, unrolled), then add their counts across the P lanes
        int P = 1;
        while (P < 32 && 2 * P * nk <= nthr) P *= 2;
        const int span = (nk + P - 1) / P;
        for (int c0 = 0; c0 < nk * P; c0 += nthr) {
            const int w = c0 + tid, c = w / P, part = w - c * P;
            int cnt = 0;
            if (c < nk) {
                const unsigned long long kc = ckey[c];
                const int ja = part * span, jb = min(nk, ja + span);
#pragma unroll 8
                for (int j = ja; j < jb; ++j) cnt += ckey[j] > kc;
            }
            for (int o = 1; o < P; o <<= 1) cnt += __shfl_xor(cnt, o);
            if (c < nk && part == 0) fsel[c] = cnt < k;
        }
    }
    lds_barrier();
    for (int c = tid; c < nk; c += nthr) st[c] = fsel[c] ? 0 : min(st[c] + 1, g.delta);
    lds_barrier();

    // segment residency, drops (counters summed per thread, then per wavefront: one shared-memory
    // atomic per wavefront)
    int c_rows = 0, c_drop = 0, c_rev = 0;
    for (int u = tid; u < nu; u += nthr) {
        const bool now = (u < nk && st[u] < g.delta) || (two && u >= 1 && u - 1 < nk && st[u - 1] < g.delta);
        const bool owned = sof[u] >= 0;     // has a slot: resident after the previous step
        fdrop[u] = owned && !now;
        fnew[u] = now && !owned;
        fkept[u] = now && owned;
        const bool att = nxt ? owned : now;
        g_att[u] = att;
        if (att) c_rows += srows[u];
        if (fdrop[u]) {
            busy[sof[u]] = nxt ? 2 : 0;
            since[sof[u]] = step;
            ++c_drop;
        }
    }
    lds_barrier();
    // revival: the segment's bytes are still in the free slot it last occupied
    for (int u = tid; u < nu; u += nthr)
        if (fnew[u]) {
            const int sl = slast[u];
            if (sl >= 0 && busy[sl] == 0 && sdata[sl] == u) {
                busy[sl] = 1;
                sof[u] = sl;
                fnew[u] = 0;
                fkept[u] = 1;
                ++c_rev;
            }
        }
    c_rows = wave_sum(c_rows);
    c_drop = wave_sum(c_drop);
    c_rev = wave_sum(c_rev);
    if ((tid & 63) == 0) {
        if (c_rows) atomicAdd(&nrows, c_rows);
        if (c_drop) atomicAdd(&ndrop, c_drop);
        if (c_rev) atomicAdd(&nrev, c_rev);
    }
    lds_barrier();

    // ranks in index order of the selected chunks (rank), the kept segments (rank_k) and the
    // new segments (rank_n), all three at once: a ballot per wavefront and flag gives each entry
    // its rank inside its 64-entry block and the block's count (kept in shared memory); after
    // one barrier each entry adds the counts of the blocks before its own
    const int nb = (nu + 63) >> 6, lane = tid & 63;
    for (int i0 = 0; i0 < nu; i0 += nthr) {
        const int i = i0 + tid;
        const unsigned long long m0 = __ballot(i < nk && fsel[i]), m1 = __ballot(i < nu && fkept[i]),
                                 m2 = __ballot(i < nu && fnew[i]);
        const unsigned long long below = (1ull << lane) - 1ull;
        if (i < nk) rank[i] = __popcll(m0 & below);
        if (i < nu) {
            rank_k[i] = __popcll(m1 & below);
            rank_n[i] = __popcll(m2 & below);
            if (lane == 0) {
                const int blk = i >> 6;
                bcnt[blk] = __popcll(m0);
                bcnt[nb + blk] = __popcll(m1);
                bcnt[2 * nb + blk] = __popcll(m2);
            }
        }
    }
    lds_barrier();
    int nsel = 0, nkept = 0, nnew = 0;
    for (int i0 = 0; i0 < nu; i0 += nthr) {
        const int i = i0 + tid, blk = i >> 6;
        int p0 = 0, p1 = 0, p2 = 0;
        for (int j = (i0 >> 6); j < blk && j < nb; ++j) {
            p0 += bcnt[j];
            p1 += bcnt[nb + j];
            p2 += bcnt[2 * nb + j];
        }
        if (i < nk) rank[i] += nsel + p0;
        if (i < nu) {
            rank_k[i] += nkept + p1;
            rank_n[i] += nnew + p2;
        }
        // totals up to the end of this round (the same for every thread)
        for (int j = i0 >> 6; j < min(nb, (i0 + nthr) >> 6); ++j) {
            nsel += bcnt[j];
            nkept += bcnt[nb + j];
            nnew += bcnt[2 * nb + j];
        }
    }
    if (selected) {
        for (int c = tid; c < nk; c += nthr)
            if (fsel[c]) selected[(size_t)b * k + rank[c]] = c;
        for (int i = nsel + tid; i < k; i += nthr) selected[(size_t)b * k + i] = -1;
    }

    // kept list: the resident segments whose bytes are on the device already (kept from the
    // previous step or revived), attended by this step (same-step timing) or by the next one.
    // With next-step timing the new list's segments follow them in the same list (below): the
    // step that reads the list finds them copied, and each tidal head streams one run of rows.
    // Bit 30 of an entry's slot: every tidal head's complement of the segment has its full
    // stride of rows (the tiles then skip the per-head row count).
    int32_t *kl = s.kept_list + (size_t)b * ns * 2;
    int c_krows = 0;
    for (int u = tid; u < nu; u += nthr)
        if (fkept[u]) {
            const int rows = srows[u];
            kl[rank_k[u] * 2] = u;
            kl[rank_k[u] * 2 + 1] = sof[u] | (rows * 2 == g.blk_rows ? 1 << 30 : 0);
            c_krows += rows;
        }
    c_krows = wave_sum(c_krows);
    if ((tid & 63) == 0 && c_krows) atomicAdd(&nkrows, c_krows);

    // free slots ordered by (holds data, freed at step, slot id): never-used first, then the
    // least recently freed.  Key: -1 for slots not free, else (holds data) * 2^30 + freed-at step.
    for (int i0 = 0; i0 < ns; i0 += nthr) {
        const int i = i0 + tid;
        const bool fr = i < ns && !busy[i];
        if (i < ns) {
            skey[i] = fr ? ((sdata[i] >= 0 ? 1 : 0) << 30) + since[i] : -1;
            // the key and the slot id in one 64-bit word (slots not free: above every free one)
            fkey[i] = fr ? ((unsigned long long)skey[i] << 32) | (unsigned)i : ~0ull;
            frank[i] = 0;
        }
        const unsigned long long bal = __ballot(fr);   // free slots: one count per wavefront
        if ((tid & 63) == 0 && bal) atomicAdd(&nfree, __popcll(bal));
    }
    lds_barrier();
    {
        // every free slot counts the free slots ordered before it; the comparisons of one slot are
        // split over `split` threads that add their counts (integer sums: any order)
        const int split = max(1, nthr / max(ns, 1)), span_j = (ns + split - 1) / split;
        for (int w = tid; w < ns * split; w += nthr) {
            const int i = w % ns, part = w / ns;
            if (skey[i] < 0) continue;
            const unsigned long long ki = fkey[i];
            int r = 0;
#pragma unroll 16
            for (int j = part * span_j, je = min(ns, (part + 1) * span_j); j < je; ++j) r += fkey[j] < ki;
            if (r) atomicAdd(&frank[i], r);
        }
    }
    lds_barrier();
    for (int i = tid; i < ns; i += nthr)
        if (skey[i] >= 0) freelist[frank[i]] = i;   // the ranks of the free slots are 0 .. nfree-1, each once
    lds_barrier();

    // segments to recall take the free slots in that order (lowest id first)
    int32_t *nl = s.new_list + (size_t)b * g.knew * 2;
    for (int u = tid; u < nu; u += nthr)
        if (fnew[u] && rank_n[u] < nfree && rank_n[u] < g.knew) {
            const int slot = freelist[rank_n[u]];
            sof[u] = slot;
            slast[u] = slot;
            busy[slot] = 1;
            sdata[slot] = u;
            nl[rank_n[u] * 2] = u;
            nl[rank_n[u] * 2 + 1] = slot;
            if (nxt) {
                kl[(nkept + rank_n[u]) * 2] = u;
                kl[(nkept + rank_n[u]) * 2 + 1] = slot | (srows[u] * 2 == g.blk_rows ? 1 << 30 : 0);
            }
            if (s.pub) {
                // the host reads this mirror once the sequence's tag is published (below)
                int32_t *hl = s.pub + g.B * 2 + (size_t)b * g.knew * 2;
                hl[rank_n[u] * 2] = u;
                hl[rank_n[u] * 2 + 1] = slot;
            }
        }
    for (int u = tid; u < nu; u += nthr)
        if (fdrop[u]) sof[u] = -1;
    lds_barrier();

    // state out
    for (int c = tid; c < nk; c += nthr) g_streak[c] = st[c];
    for (int u = tid; u < nu; u += nthr) {
        g_slot_of[u] = sof[u];
        g_slot_last[u] = slast[u];
    }
    for (int i = tid; i < ns; i += nthr) {
        g_busy[i] = busy[i];
        g_data[i] = sdata[i];
        g_since[i] = since[i];
    }
    if (tid == 0) {
        const int nn = min(nnew, min(nfree, g.knew));
        const int nlist = nxt ? nkept + nn : nkept;   // entries of the kept list
        s.counts[b * 2] = nlist;
        s.counts[b * 2 + 1] = nn;
        if (s.pub) {
            s.pub[b * 2] = nlist;
            s.pub[b * 2 + 1] = nn;
        }
        s.step[b] = step + 1;
        atomicAdd(&s.stats[0], (unsigned long long)nn);
        atomicAdd(&s.stats[1], (unsigned long long)ndrop);
        // resident segments after the step
        const int nres = nkept + nn;
        atomicAdd(&s.stats[2], (unsigned long long)nres);
        atomicAdd(&s.stats[3], (unsigned long long)nrows);
        atomicMax(&s.stats[4], (unsigned long long)nres);
        if (nnew > nn) {
            // no free slot for a newly resident segment: the slot count bounds the resident set,
            // so this never happens; if it did, tidal heads would miss a resident segment, so the
            // host is told (vector store to mapped pinned memory) and fails the context
            atomicAdd(&s.stats[5], 1ull);
            if (s.exhausted) *(volatile int32_t *)s.exhausted = 1;
        }
        atomicAdd(&s.stats[6], (unsigned long long)nrev);
        atomicAdd(&s.stats[7], (unsigned long long)nkrows);
    }
    if (s.pub) {
        // publication: the host polls this sequence's tag instead of an event after the kernel
        // (an event costs the stream a gap before the next launch).  Every wavefront waits for
        // its own stores to the mirror (and the exhaustion flag) to complete before the barrier
        // (a work-group barrier alone does not wait for global stores); the first thread's
        // system-scope fence then writes back whatever of them the cache holds, and the tag is
        // stored last, write-through
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0) {
            __threadfence_system();
            __hip_atomic_store(s.pub + g.B * 2 + (size_t)g.B * g.knew * 2 + b, s.pub_tag, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

__global__ __launch_bounds__(SEL_THREADS) void select_kernel(Geometry g, StepBuffers s, float *__restrict__ scores,
                                                             const int32_t *__restrict__ ovr, int32_t *__restrict__ selected)
{
    extern __shared__ double sdyn[];
    __shared__ SelectShared sh;
    select_seq(g, s, scores, ovr, selected, blockIdx.x, sdyn, sh);
}

// -------------------------------------------------------------------------------------------
// Tidal / fixed attention (fp32 logits).  Each wavefront runs its own softmax over its 4 * RPL
// rows (no barrier until the end); the four wavefront partials are merged in shared memory.
// -------------------------------------------------------------------------------------------
// Source rows of one key position (nullptr when the position is not in the tile) and, for the
// recall path, where to copy them.
struct RowPtr {
    const uint16_t *k, *v;
};

// One work-group = 4 wavefronts; wavefront w owns rows [w * 4 * RPL, (w + 1) * 4 * RPL) of the
// tile's row map, in sub-tiles of 32 rows (RPL = 8 or 16).  Rows are loaded fully coalesced
// (16 lanes per 256-byte row), by one of three paths chosen by the row map: consecutive rows of
// one head (`contiguous`: buffer loads, one lane offset), rows of several slot entries
// (`offsets`: buffer loads over the sequence's slot region, each lane walking its rows through
// the entries), or one pointer per row (the recall path, and slot regions of 4 GB or more).  The
// rows' validity becomes a per-wavefront mask (a ballot per load), which the logits read.
//
// Logits (fp32, exact bf16 products) on v_mfma_f32_4x4x4_16b_bf16: lane l = 4*blk + i feeds
// A_blk[i][0..3] and B_blk[0..3][i], and D_blk[i][j] lands in lane 4*blk + j, register i.
// Block blk = 8*dh + kb takes keys 4*kb .. 4*kb + 3 of the sub-tile over dimension half dh
// (sixteen instructions of four dimensions each); one cross-half add completes the dot
// products.  A comes from the wavefront's K rows staged in LDS (16-byte units swizzled by row),
// B from q staged in LDS (rows padded to 272 bytes so that the eight (head, half) reads of an
// instruction hit distinct banks).  P.V runs on v_mfma_f32_4x4x1 as in the anchor kernel.
// Shared memory of one subset tile; one instance per work-group, whichever row map it runs.
template <int G, int RPL>
struct SubsetSmem {
    static constexpr int NR = 4 * RPL, HS = (G + 3) / 4, QS = 136, MAXE = NR * WAVES;
    uint4 kst[WAVES][NR * 16];                // K rows, then the P.V partials of each wavefront
    uint16_t qs[HS * 4 * QS];                 // q, rows padded to 272 bytes
    float xf[G * WAVES * NR];                 // probabilities
    float wm[WAVES * G], wl[WAVES * G];
    // entries of a run of slot rows (slot_rows_tile; a tile's entries never exceed its rows)
    const uint16_t *kbase[MAXE];
    unsigned koff[MAXE];
    int nrows[MAXE];
};

template <int G, int RPL, class RowMap>
__device__ inline void subset_tile(const uint16_t *__restrict__ qh, const RowMap &map, float *pm, float *pl, float *po,
                                   SubsetSmem<G, RPL> &sm)
{
    typedef float v4f __attribute__((ext_vector_type(4)));
    typedef short v4s __attribute__((ext_vector_type(4)));
    constexpr int NR = 4 * RPL;               // rows per wavefront
    constexpr int NSUB = NR / 32;             // 32-row sub-tiles per wavefront
    constexpr int HS = (G + 3) / 4;           // sets of 4 heads
    constexpr int OGR = G <= 4 ? 4 : 2;       // row groups kept in the P.V partial store
    constexpr int QS = 136;                   // padded q row, in uint16
    static_assert(NR % 32 == 0, "wavefront rows come in 32-row sub-tiles");
    const int tid = lane_id_opaque(), lane = tid & 63, wave = tid >> 6, sub = lane & 15, rg = lane >> 4;
    const int j4 = lane & 3, kb = (lane >> 2) & 7, dh = lane >> 5;
    auto &kst = sm.kst;
    uint16_t *qs = sm.qs;
    float *xf = sm.xf, *wm = sm.wm, *wl = sm.wl;
    float *wo = (float *)&kst[wave][0];

    // q: loaded into a register first and written to shared memory only once the K/V loads are
    // issued, so that no wavefront waits for it before starting its stream
    static_assert(HS * 4 * (D / 8) <= NT, "one 16-byte piece of q per thread");
    const bool q_lane = tid < HS * 4 * (D / 8);
    const int qh_i = tid / (D / 8), qu = tid - qh_i * (D / 8);
    uint4 qv = make_uint4(0, 0, 0, 0);
    if (q_lane && qh_i < G) qv = *(const uint4 *)(qh + qh_i * D + qu * 8);
    uint4 kr[RPL], vr[RPL];
    bool ok[RPL];
    if constexpr (RowMap::contiguous) {
        // consecutive rows of one head: buffer loads, rows at or past R read zeros
        const __amdgpu_buffer_rsrc_t rk = buf_rsrc(map.K, (unsigned)map.R * (D * 2));
        const __amdgpu_buffer_rsrc_t rv = buf_rsrc(map.V, (unsigned)map.R * (D * 2));
        const unsigned o0 = (unsigned)(map.t0 + wave * NR + rg) * (D * 2) + sub * 16;
#pragma unroll
        for (int i = 0; i < RPL; ++i) kr[i] = buf_load_nt(rk, o0 + i * (4 * D * 2));
#pragma unroll
        for (int i = 0; i < RPL; ++i) vr[i] = buf_load_nt(rv, o0 + i * (4 * D * 2));
#pragma unroll
        for (int i = 0; i < RPL; ++i) ok[i] = map.t0 + wave * NR + i * 4 + rg < map.R;
    } else if constexpr (RowMap::offsets) {
        // rows of several slot entries: offsets in the sequence's slot region; each lane walks
        // its rows (stride 4) through the entries with one division.  Rows past the group's
        // entries or past an entry's valid rows read the first row of entry 0 (finite, masked).
        const __amdgpu_buffer_rsrc_t rs = buf_rsrc(map.base, map.bytes);
        const int cm = map.comp_max;
        const unsigned vd = (unsigned)cm * (D * 2);   // an entry's V rows follow its K rows
        const int v0 = map.first + wave * NR + rg;     // row within the entries, from entry 0's first
        // every row's entry first (one division, then steps of 4 rows), then the entries'
        // shared-memory reads back to back (one wait), then all the loads back to back
        unsigned off[RPL];
        int ent[RPL], rrs[RPL];
        {
            int e = v0 / cm, rr = v0 - e * cm;
#pragma unroll
            for (int i = 0; i < RPL; ++i) {
                if (i) {
                    rr += 4;
                    while (rr >= cm) {
                        rr -= cm;
                        ++e;
                    }
                }
                ent[i] = e < map.n_entries ? e : -1;
                rrs[i] = rr;
            }
        }
        int nrs[RPL];
        unsigned kos[RPL];
#pragma unroll
        for (int i = 0; i < RPL; ++i) {
            const int ec = ent[i] < 0 ? 0 : ent[i];
            nrs[i] = map.nrows[ec];
            kos[i] = map.koff[ec];
        }
        const unsigned off0 = map.koff[0] + sub * 16;
#pragma unroll
        for (int i = 0; i < RPL; ++i) {
            ok[i] = ent[i] >= 0 && rrs[i] < nrs[i];
            off[i] = ok[i] ? kos[i] + (unsigned)rrs[i] * (D * 2) + sub * 16 : off0;
        }
#pragma unroll
        for (int i = 0; i < RPL; ++i) kr[i] = buf_load_nt(rs, off[i]);
#pragma unroll
        for (int i = 0; i < RPL; ++i) vr[i] = buf_load_nt(rs, off[i] + vd);
    } else {
#pragma unroll
        for (int i = 0; i < RPL; ++i) {
            const RowPtr rp = map.row(wave * NR + i * 4 + rg);
            ok[i] = rp.k != nullptr;
            // device rows stream once (nontemporal); host rows keep plain loads
            if constexpr (RowMap::copies)
                kr[i] = ok[i] ? *(const uint4 *)(rp.k + sub * 8) : make_uint4(0, 0, 0, 0);
            else
                kr[i] = ok[i] ? load_nt(rp.k + sub * 8) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < RPL; ++i) {
            const RowPtr rp = map.row(wave * NR + i * 4 + rg);
            if constexpr (RowMap::copies)
                vr[i] = ok[i] ? *(const uint4 *)(rp.v + sub * 8) : make_uint4(0, 0, 0, 0);
            else
                vr[i] = ok[i] ? load_nt(rp.v + sub * 8) : make_uint4(0, 0, 0, 0);
        }
    }
    if (q_lane) *(uint4 *)(qs + qh_i * QS + qu * 8) = qv;
    // valid rows of this wavefront as a mask (bit i * 4 + rg), for the logits
    unsigned long long rowmask = 0;
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
        const unsigned long long bal = __ballot(ok[i]);   // lane rg * 16 + sub; a row's lanes agree
        rowmask |= ((bal & 1ull) | ((bal >> 15) & 2ull) | ((bal >> 30) & 4ull) | ((bal >> 45) & 8ull)) << (i * 4);
    }
    if constexpr (RowMap::copies) {
        // rows read from host memory are also written to their device slot on the way
#pragma unroll
        for (int i = 0; i < RPL; ++i)
            if (ok[i]) {
                const int r = wave * NR + i * 4 + rg;
                *(uint4 *)(map.kdst(r) + sub * 8) = kr[i];
                *(uint4 *)(map.vdst(r) + sub * 8) = vr[i];
            }
    }
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
        const int r = i * 4 + rg;
        kst[wave][r * 16 + (sub ^ (r & 15))] = kr[i];
    }
    __syncthreads();   // q staged; each wavefront's K rows are its own

    // logits: key sub*32 + 4*kb + i, head hs*4 + j4, register i of lg[sub][hs]
    v4f lg[NSUB][HS];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
        for (int hs = 0; hs < HS; ++hs) lg[sb][hs] = v4f{0.f, 0.f, 0.f, 0.f};
    const int rA = 4 * kb + j4;               // A row of this lane within a sub-tile
#pragma unroll
    for (int p8 = 0; p8 < 8; ++p8) {
        const int unit = 8 * dh + p8;
        uint4 qb[HS];
#pragma unroll
        for (int hs = 0; hs < HS; ++hs) qb[hs] = *(const uint4 *)(qs + (hs * 4 + j4) * QS + unit * 8);
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) {
            const int r = sb * 32 + rA;
            const uint4 ka = kst[wave][r * 16 + (unit ^ (r & 15))];
            const v4s a0 = __builtin_bit_cast(v4s, make_uint2(ka.x, ka.y));
            const v4s a1 = __builtin_bit_cast(v4s, make_uint2(ka.z, ka.w));
#pragma unroll
            for (int hs = 0; hs < HS; ++hs) {
                lg[sb][hs] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(a0, __builtin_bit_cast(v4s, make_uint2(qb[hs].x, qb[hs].y)),
                                                                    lg[sb][hs], 0, 0, 0);
                lg[sb][hs] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(a1, __builtin_bit_cast(v4s, make_uint2(qb[hs].z, qb[hs].w)),
                                                                    lg[sb][hs], 0, 0, 0);
            }
        }
    }
    // complete the dot products across the two dimension halves; scale and mask
    float m[HS], l[HS];
#pragma unroll
    for (int hs = 0; hs < HS; ++hs) {
        const bool hv = hs * 4 + j4 < G;
        float mm = -INFINITY;
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float x = lg[sb][hs][i];
                x += __shfl_xor(x, 32);
                const int r = sb * 32 + 4 * kb + i;   // row of this wavefront
                x = (hv && ((rowmask >> r) & 1ull)) ? x * SCALE_F : -INFINITY;
                lg[sb][hs][i] = x;
                mm = fmaxf(mm, x);
            }
        mm = fmaxf(mm, __shfl_xor(mm, 4));
        mm = fmaxf(mm, __shfl_xor(mm, 8));
        mm = fmaxf(mm, __shfl_xor(mm, 16));
        float ll = 0.f;
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float pv = (mm == -INFINITY) ? 0.f : __expf(lg[sb][hs][i] - mm);
                lg[sb][hs][i] = pv;
                ll += pv;
            }
        ll += __shfl_xor(ll, 4);
        ll += __shfl_xor(ll, 8);
        ll += __shfl_xor(ll, 16);
        m[hs] = mm;
        l[hs] = ll;
        if (hv && dh == 0) {
#pragma unroll
            for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
                for (int i = 0; i < 4; ++i) xf[(hs * 4 + j4) * (WAVES * NR) + wave * NR + sb * 32 + 4 * kb + i] = lg[sb][hs][i];
        }
        if (hv && lane < 4) {
            wm[wave * G + hs * 4 + j4] = mm;
            wl[wave * G + hs * 4 + j4] = ll;
        }
    }
    // each wavefront reads back only its own probabilities
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // P.V (unnormalised, relative to the wavefront maximum)
    v4f dacc[HS][8];
#pragma unroll
    for (int hs = 0; hs < HS; ++hs)
#pragma unroll
        for (int e = 0; e < 8; ++e) dacc[hs][e] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
        const int rr = wave * NR + i * 4 + rg;
        float f[8];
        unpack8(vr[i], f);
#pragma unroll
        for (int hs = 0; hs < HS; ++hs) {
            const int h = hs * 4 + j4;
            const float pa = h < G ? xf[h * (WAVES * NR) + rr] : 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) dacc[hs][e] = __builtin_amdgcn_mfma_f32_4x4x1f32(pa, f[e], dacc[hs][e], 0, 0, 0);
        }
    }
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[h][e] = dacc[h / 4][e][h % 4];
            if (OGR == 2) acc[h][e] += __shfl_xor(acc[h][e], 32);
        }
    // the K region of this wavefront is dead: it takes the P.V partials
    if (rg < OGR) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float4 *dst = (float4 *)(wo + (rg * G + h) * D + sub * 8);
            dst[0] = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
            dst[1] = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
        }
    }
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += NT) {
        const int h = idx / D;
        float M = wm[h];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) M = fmaxf(M, wm[w * G + h]);
        float o = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            const float mw = wm[w * G + h];
            if (mw > -INFINITY) {
                const float *ww = (const float *)&kst[w][0];
                float ow = 0.f;
#pragma unroll
                for (int r4 = 0; r4 < OGR; ++r4) ow += ww[r4 * G * D + idx];
                o += ow * __expf(mw - M);
            }
        }
        po[idx] = o;
    }
    if (tid < G) {
        float M = wm[tid];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) M = fmaxf(M, wm[w * G + tid]);
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            const float mw = wm[w * G + tid];
            if (mw > -INFINITY) L += wl[w * G + tid] * __expf(mw - M);
        }
        pm[tid] = M;
        pl[tid] = L;
    }
    __syncthreads();   // the shared buffers may be reused by the next tile of this work-group
}

// Consecutive rows of one head: rows t0 .. of the head starting at K / V, R of them valid (read
// by buffer loads, see subset_tile).
struct StaticRows {
    static constexpr bool copies = false, contiguous = true, offsets = false;
    const uint16_t *K, *V;
    int t0, R;
};

// Rows of a run of resident complements of one tidal head: the entries' rows one after the
// other (comp_max per entry, of which the first nrows are valid), starting at row `first` of the
// first entry.  The entries are staged in shared memory as (K row base, valid rows) so that the
// row map needs no global load.
struct SlotRows {
    static constexpr bool copies = false, contiguous = false, offsets = false;
    const uint16_t *const *kbase;   // [n_entries] first K row of the tidal head in the entry's slot
    const int *nrows;               // [n_entries] valid rows of the entry (complement length)
    int n_entries, comp_max, first;
    __device__ RowPtr row(int r) const
    {
        const int v = first + r, e = v / comp_max, rr = v - e * comp_max;
        if (e >= n_entries || rr >= nrows[e]) return {nullptr, nullptr};
        const uint16_t *k = kbase[e] + (size_t)rr * D;
        return {k, k + (size_t)comp_max * D};
    }
};

// The same rows as byte offsets in the sequence's slot region (buffer loads; used while the
// region stays below 4 GB).
struct SlotRowsOff {
    static constexpr bool copies = false, contiguous = false, offsets = true;
    const uint16_t *base;           // the sequence's first slot
    unsigned bytes;                 // its slot region
    const unsigned *koff;           // [n_entries] byte offset of the entry's first K row of the tidal head
    const int *nrows;               // [n_entries] valid rows of the entry (complement length)
    int n_entries, comp_max, first;
};

// Rows of one recalled complement block (a tidal head's complement of one chunk): comp_max K rows,
// then comp_max V rows, of which the first nrows are valid.  They are read from the mapped pinned
// host block and copied through to the device slot on the way.
struct RecallRows {
    static constexpr bool copies = true, contiguous = false, offsets = false;
    const uint16_t *src;     // host block
    uint16_t *dst;           // device slot block, same layout
    int nrows, comp_max;
    __device__ RowPtr row(int r) const
    {
        if (r >= nrows) return {nullptr, nullptr};
        const uint16_t *k = src + (size_t)r * D;
        return {k, k + (size_t)comp_max * D};
    }
    __device__ uint16_t *kdst(int r) const { return dst + (size_t)r * D; }
    __device__ uint16_t *vdst(int r) const { return dst + (size_t)(comp_max + r) * D; }
};

constexpr int RPL_S = TILE_S / (4 * WAVES);   // 8
constexpr int RECALL_WGS = 64;                // work-groups that recall (they fill the host link)

// Static tile j (of the sequence's n_static) of sequence b: kept rows + text of one head.
template <int G>
__device__ inline void static_tile(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, int j,
                                   int b, SubsetSmem<G, RPL_S> &sm)
{
    const int hi = t.tile_head[j];
    const HeadRows hr = t.hr[hi];
    const int tile = j - hr.tile0, rows = hr.rs + g.n_gen;
    const size_t p = (size_t)b * g.P + hr.pbase + tile;
    if (tile * TILE_S >= rows) {
        // room reserved for tokens not appended yet: an empty partial, which the merge skips
        if (threadIdx.x < G) {
            s.ps_m[p * G + threadIdx.x] = -INFINITY;
            s.ps_l[p * G + threadIdx.x] = 0.f;
        }
        for (int i = threadIdx.x; i < G * D; i += NT) s.ps_o[p * G * D + i] = 0.f;
        return;
    }
    const bool tidal = hi < g.nT;
    const int lk = tidal ? t.tidal_lk[hi] : t.fixed_lk[hi - g.nT], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const size_t hb = ((size_t)b * (tidal ? g.RsT : g.RsF) + hr.srow) * D;
    const StaticRows map{(tidal ? t.tK : t.fK) + hb, (tidal ? t.tV : t.fV) + hb, tile * TILE_S, rows};
    const uint16_t *qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    subset_tile<G, RPL_S>(qh, map, s.ps_m + p * G, s.ps_l + p * G, s.ps_o + p * G * D, sm);
}

// Rows of the listed resident complements of tidal head ti, sequence b, as a run of entries
// (see SlotRows) starting at row `first` of entry e0: n_entries entries from `list` ((segment,
// slot) pairs; bit 30 of the slot marks a segment whose complement has the full stride in every
// tidal head, so its row count needs no lookup), attended as one tile into partial p.
template <int G, int RPL>
__device__ inline void slot_rows_tile(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q,
                                      const int32_t *list, int e0, int n_entries, int first, int ti, int b, size_t p,
                                      SubsetSmem<G, RPL> &sm)
{
    const uint16_t **kbase = sm.kbase;
    unsigned *koff = sm.koff;
    int *nrows = sm.nrows;
    const HeadRows hr = t.hr[ti];
    const uint16_t *region = t.slots + (size_t)b * g.n_slots * g.chunk_elems;
    const size_t region_bytes = (size_t)g.n_slots * g.chunk_elems * sizeof(uint16_t);
    const bool by_offset = (long long)region_bytes < g.slot_off_max;   // at most 4294967295
    for (int e = threadIdx.x; e < n_entries; e += NT) {
        const int c = list[(e0 + e) * 2], sf = list[(e0 + e) * 2 + 1], slot = sf & 0xffff;
        const size_t o = (size_t)slot * g.chunk_elems + (size_t)hr.coff * D;
        kbase[e] = region + o;
        koff[e] = (unsigned)(o * sizeof(uint16_t));
        nrows[e] = (sf >> 30) & 1 ? hr.cfull : t.comp_rows[((size_t)b * g.nc + c) * g.nT + ti];
    }
    __syncthreads();
    const int lk = t.tidal_lk[ti], l = lk / g.Hkv, kv = lk - l * g.Hkv;
    const uint16_t *qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
    if (by_offset) {
        const SlotRowsOff map{region, (unsigned)region_bytes, koff, nrows, n_entries, hr.cfull, first};
        subset_tile<G, RPL>(qh, map, s.ps_m + p * G, s.ps_l + p * G, s.ps_o + p * G * D, sm);
    } else {
        const SlotRows map{kbase, nrows, n_entries, hr.cfull, first};
        subset_tile<G, RPL>(qh, map, s.ps_m + p * G, s.ps_l + p * G, s.ps_o + p * G * D, sm);
    }
}

// Item j of the kept list of tidal head ti, sequence b: the head's complements of the listed
// segments, taken as one run of rows (entries one after the other, cfull rows each), cut into
// TILE_S-row items; item j is rows [j * TILE_S, (j + 1) * TILE_S) of that run.  An item may
// start or end inside an entry, so every work-group streams a full tile whatever the complement
// length.  Returns at once when the head has fewer items this step.
template <int G>
__device__ inline void list_item(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, int j,
                                 int ti, int b, SubsetSmem<G, RPL_S> &sm)
{
    const HeadRows hr = t.hr[ti];
    const int cm = hr.cfull, cnt = s.counts[b * 2];
    const long long v0 = (long long)j * TILE_S;
    if (cm == 0 || j >= hr.ngk || v0 >= (long long)cnt * cm) return;
    const int e0 = (int)(v0 / cm), e1 = (int)min((long long)cnt - 1, (v0 + TILE_S - 1) / cm);
    const int32_t *list = s.kept_list + (size_t)b * g.n_slots * 2;
    const size_t p = (size_t)b * g.P + hr.pbase + hr.nts + j;
    const int n_entries = e1 - e0 + 1, first = (int)(v0 - (long long)e0 * cm);
    slot_rows_tile<G, RPL_S>(g, t, s, q, list, e0, n_entries, first, ti, b, p, sm);
}

// New entry e of tidal head ti, sequence b (complements copied by the host-issued recall with
// same-step timing): the whole entry in one tile.
template <int G, int RPL>
__device__ inline void new_entry(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, int e,
                                 int ti, int b, SubsetSmem<G, RPL> &sm)
{
    const HeadRows hr = t.hr[ti];
    if (hr.cfull == 0 || e >= s.counts[b * 2 + 1]) return;
    const int32_t *list = s.new_list + (size_t)b * g.knew * 2;
    const size_t p = (size_t)b * g.P + hr.pbase + hr.nts + hr.ngk + e;
    slot_rows_tile<G, RPL>(g, t, s, q, list, e, 1, 0, ti, b, p, sm);
}

// Recall work-group w of nw: walks the units (sequence, new entry, tidal head); each unit's
// complement block is read from mapped pinned memory, copied to its slot and attended to in the
// same pass.  The number of work-groups, not their width, bounds the host reads in flight.
template <int G, int RPL>
__device__ inline void recall_units(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, int w,
                                    int nw, SubsetSmem<G, RPL> &sm)
{
    int total = 0;
    for (int b = 0; b < g.B; ++b) total += s.counts[b * 2 + 1] * g.nT;
    for (int u = w; u < total; u += nw) {
        int b = 0, r = u;
        while (r >= s.counts[b * 2 + 1] * g.nT) r -= s.counts[b++ * 2 + 1] * g.nT;
        const int e = r / g.nT, ti = r - e * g.nT;
        const HeadRows hr = t.hr[ti];
        if (hr.cfull == 0) continue;   // retention 1: nothing of this head to recall
        const int c = s.new_list[((size_t)b * g.knew + e) * 2], slot = s.new_list[((size_t)b * g.knew + e) * 2 + 1];
        const size_t off = (size_t)hr.coff * D;
        const uint16_t *src = t.host_comp + ((size_t)b * g.nc + c) * g.chunk_elems + off;
        uint16_t *dst = t.slots + ((size_t)b * g.n_slots + slot) * g.chunk_elems + off;
        const int cm = hr.cfull, nr = t.comp_rows[((size_t)b * g.nc + c) * g.nT + ti];
        // rows past the segment's complement (short last segment) are zero padding: copied for a
        // byte-identical slot, not attended
        for (int j = threadIdx.x; j < (cm - nr) * 2 * (D / 8); j += NT) {
            const int half = j / ((cm - nr) * (D / 8)), rem = j - half * (cm - nr) * (D / 8);
            const size_t o = ((size_t)half * cm + nr) * D + (size_t)rem * 8;
            *(uint4 *)(dst + o) = *(const uint4 *)(src + o);
        }
        const int lk = t.tidal_lk[ti], l = lk / g.Hkv, kv = lk - l * g.Hkv;
        const uint16_t *qh = q + (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D;
        const size_t p = (size_t)b * g.P + hr.pbase + hr.nts + hr.ngk + e;
        const RecallRows map{src, dst, nr, cm};
        subset_tile<G, RPL>(qh, map, s.ps_m + p * G, s.ps_l + p * G, s.ps_o + p * G * D, sm);
    }
}

constexpr int SEL_SHARED_OFF = 512;   // bytes of counters before the mass or selection arrays

// True in every thread of the work-group that arrives last of n at the counter *cnt (an
// agent-scope atomic), which that work-group resets for the next launch.  The values passed on
// are agent-scope atomic stores (st_agent) that every wavefront waits to complete before the
// work-group counts itself in (a work-group barrier alone does not wait for global stores); the
// last work-group reads them with agent-scope atomic loads (ld_agent) after the count.
__device__ inline bool last_arrival(int32_t *cnt, int n, SelectShared &sh)
{
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        const int old = atomicAdd(cnt, 1);
        sh.last = old == n - 1;
        if (old == n - 1) atomicExch(cnt, 0);
    }
    __syncthreads();
    return sh.last;
}

// Fixed heads, tidal kept rows and tidal complements already in their slots: static tiles
// first (unless the attention launch ran them), then the items of one list (list_item).  The
// work-groups loop over those tiles with the grid's stride, so the launch holds about as many
// work-groups as the compute units keep resident and none of them is spent on an item that
// this step does not have.  With REC (same-step timing), the first RECALL_WGS work-groups copy
// the complements listed for recall from mapped pinned memory into their slots and attend to
// them: the step is bound by the host link then, and the copies start with the launch.
// With SEL (next-step timing, sel.s.arrive set), the first sel.n_mass = nA * B work-groups
// merge the anchor heads' chunk masses of this step's attention launch, one head each, and the
// last of a sequence's heads to finish runs the sequence's selection (sel.s: the lists it
// writes, which this launch does not read; the items read the lists of s).  A separate
// instantiation: the branch alone, never taken, slowed the items by about 1.5 %.
template <int G, int RPLK, bool REC, bool SEL>
__global__ __launch_bounds__(NT, REC ? (RPLK == RPL_S ? 2 : 1) : (G <= 4 ? 4 : G <= 6 ? 3 : 2)) void tidal_fixed_kernel(
    Geometry g, Tiers t, StepBuffers s, const uint16_t *__restrict__ q, int with_static, SelectArgs sel)
{
    static_assert(!(SEL && REC), "the selection joins only the launch without recall");
    union Smem {
        SubsetSmem<G, RPL_S> st;
        SubsetSmem<G, RPLK> sl;
    };
    __shared__ Smem sm;   // one block for whichever path this work-group runs
    int w = blockIdx.x, nw = gridDim.x;
    if (SEL && w < sel.n_mass) {
        const int ai = w % g.nA, b = w / g.nA;
        char *base = (char *)&sm;
        SelectShared &sh = *(SelectShared *)base;
        static_assert(sizeof(SelectShared) + sizeof(MassSmem<G>) <= SEL_SHARED_OFF, "counters before the arrays");
        anchor_mass_head<G>(g, sel.s, ai, b, (double *)(base + SEL_SHARED_OFF), *(MassSmem<G> *)(base + sizeof(SelectShared)));
        if (last_arrival(sel.s.arrive + b, g.nA, sh))
            select_seq(g, sel.s, sel.scores, sel.ovr, sel.selected, b, (double *)(base + SEL_SHARED_OFF), sh);
        return;
    }
    if constexpr (SEL) {
        w -= sel.n_mass;
        nw -= sel.n_mass;
    }
    if constexpr (REC) {
        if (w < RECALL_WGS) {
            recall_units<G, RPLK>(g, t, s, q, w, RECALL_WGS, sm.sl);
            return;
        }
        w -= RECALL_WGS;
        nw -= RECALL_WGS;
    }
    const long long n_static = with_static ? (long long)g.n_static * g.B : 0;
    // kept-list items in item-major order over (sequence, tidal head); the loop ends after the
    // last item any head has this step (a head with fewer returns at once from the ones past its
    // own)
    int kmax = 0;
    for (int b = 0; b < g.B; ++b) kmax = max(kmax, s.counts[b * 2]);
    const long long n_items = min(((long long)kmax * g.comp_max + TILE_S - 1) / TILE_S, (long long)g.ng_kept);
    const long long nh = (long long)g.nT * g.B, total = n_static + n_items * nh;
    for (long long it = w; it < total; it += nw) {
        if (it < n_static) {
            static_tile<G>(g, t, s, q, (int)(it % g.n_static), (int)(it / g.n_static), sm.st);
        } else {
            const long long i2 = it - n_static, j = i2 / nh, rest = i2 - j * nh;
            list_item<G>(g, t, s, q, (int)j, (int)(rest % g.nT), (int)(rest / g.nT), sm.st);
        }
    }
}

// Anchor tiles and the static tidal/fixed tiles (kept rows + text, which no selection changes)
// in one launch, interleaved along the grid: the anchor tiles' arithmetic (fp64 logits)
// overlaps the static tiles' streaming.  Used with next-step timing, where the static tiles need
// not wait for this step's selection.
template <int G>
__global__ __launch_bounds__(NT, G <= 4 ? 4 : 2) void attention_kernel(Geometry g, Tiers t, StepBuffers s,
                                                                       const uint16_t *__restrict__ q)
{
    union Smem {
        AnchorSmem<G> a;
        SubsetSmem<G, RPL_S> st;
    };
    __shared__ Smem sm;
    // One tile per work-group (the hardware's dynamic dispatch balances the slower anchor tiles
    // against the static ones better than a grid-stride loop: measured 98 vs 107 us).
    // The anchor tiles are spread evenly over the first half of the grid (all of it's first
    // part when they are more than half the tiles), so that the launch ends on static tiles only:
    // an anchor tile takes longer, and one dispatched last would stretch the launch's tail
    // (measured: 98.3 -> 96.2-97.1 us with the selection pinned; spread over the whole grid, or
    // over its first 70-85 %, ends later).
    const long long na = (long long)g.n_tiles_a * g.nA * g.B;
    const long long n = na + (long long)g.n_static * g.B, m = std::max(n / 2, na);
    const long long p = blockIdx.x, a0 = p < m ? p * na / m : na, a1 = p < m ? (p + 1) * na / m : na;
    if (a1 > a0) {
        // anchors before this position: a0, so this is anchor tile a0
        const int tile = (int)(a0 % g.n_tiles_a);
        const long long rest = a0 / g.n_tiles_a;
        anchor_tile<G>(g, t, s, q, tile, (int)(rest % g.nA), (int)(rest / g.nA), sm.a);
    } else {
        const long long i = p - a0;   // static tiles before this position
        static_tile<G>(g, t, s, q, (int)(i % g.n_static), (int)(i / g.n_static), sm.st);
    }
}

// Next-step timing: copy only.  Work-group w of RECALL_WGS walks the units (sequence, new entry,
// piece) and copies each piece of the entry's segment block (every tidal head's K and V
// complement rows, padding included; 32 KB per piece) from mapped pinned memory to its slot,
// eight 16-byte reads in flight per thread; the rows are attended from the next step on.  Host
// reads take ~15 us, so the link needs about a megabyte in flight: the number of work-groups,
// each holding one piece, sets the rate.
__global__ __launch_bounds__(NT) void recall_copy_kernel(Geometry g, Tiers t, StepBuffers s)
{
    constexpr int PIECE = 8 * NT;                                  // 16-byte vectors per piece
    const long long n16 = g.chunk_elems / 8;                       // 16-byte vectors per block
    const int npc = (int)((n16 + PIECE - 1) / PIECE);
    int total = 0;
    for (int b = 0; b < g.B; ++b) total += s.counts[b * 2 + 1] * npc;
    for (int u = blockIdx.x; u < total; u += gridDim.x) {
        int b = 0, r = u;
        while (r >= s.counts[b * 2 + 1] * npc) r -= s.counts[b++ * 2 + 1] * npc;
        const int e = r / npc, pc = r - e * npc;
        const int c = s.new_list[((size_t)b * g.knew + e) * 2], slot = s.new_list[((size_t)b * g.knew + e) * 2 + 1];
        const long long j0 = (long long)pc * PIECE;
        const uint4 *src = (const uint4 *)(t.host_comp + ((size_t)b * g.nc + c) * g.chunk_elems) + j0;
        uint4 *dst = (uint4 *)(t.slots + ((size_t)b * g.n_slots + slot) * g.chunk_elems) + j0;
        const int nv = (int)min((long long)PIECE, n16 - j0);
        uint4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int j = k * NT + threadIdx.x;
            if (j < nv) v[k] = src[j];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int j = k * NT + threadIdx.x;
            if (j < nv) dst[j] = v[k];
        }
    }
}

// Complements copied by hipMemcpyAsync (host-waited recall path): one entry per work-group.
template <int G, int RPL>
__global__ __launch_bounds__(NT, RPL == RPL_S ? (G <= 4 ? 4 : 3) : 2) void new_slots_kernel(Geometry g, Tiers t, StepBuffers s, const uint16_t *__restrict__ q)
{
    __shared__ SubsetSmem<G, RPL> sm;
    new_entry<G, RPL>(g, t, s, q, blockIdx.x, blockIdx.y, blockIdx.z, sm);
}

// Final merge of a step.  Work-groups 0 .. nT + nF - 1: one tidal/fixed KV-head's partials
// (static tiles, kept items, new items or entries) -> its G output rows; the next nA: one
// anchor KV-head's tile partials -> its G output rows (anchor_out_merge; the anchors' chunk
// masses were merged earlier, on the selection's path).  Per 16-byte column of the G * d outputs
// the partials are split over groups of threads and summed in a fixed order.
template <int G>
__global__ __launch_bounds__(COMBINE_THREADS) void subset_combine_kernel(Geometry g, Tiers t, StepBuffers s, void *out)
{
    const int hi = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    extern __shared__ double dsm[];      // subset heads: float [np_max][G]; anchors: double [G][n_tiles_a]
    constexpr int NC4 = G * D / 4, GR = COMBINE_THREADS / NC4, NW = COMBINE_THREADS / 64;
    __shared__ double opart[GR * NC4 * 4];
    if (hi >= g.nT + g.nF) {
        anchor_out_merge<G>(g, t, s, out, hi - g.nT - g.nF, b, dsm, opart);
        return;
    }
    float *sfac = (float *)dsm;
    const bool tidal = hi < g.nT;
    __shared__ float red[NW * G], redl[NW * G];   // per wavefront: maxima, sums
    const HeadRows hr = t.hr[hi];
    const bool recalls = tidal && hr.cfull > 0;   // no complement at retention 1
    const int nk = recalls ? (int)min(((long long)s.counts[b * 2] * hr.cfull + TILE_S - 1) / TILE_S, (long long)hr.ngk) : 0;
    // new complements with same-step timing: one partial per entry (with next-step timing they
    // are items of the kept list)
    const int nn = !recalls || g.next_step ? 0 : min(s.counts[b * 2 + 1], g.knew);
    const int nts = hr.nts, ngk = hr.ngk, nvalid = nts + nk + nn;
    auto part = [&](int j) {
        if (j < nts) return j;
        j -= nts;
        if (j < nk) return nts + j;
        return nts + ngk + (j - nk);
    };
    const size_t base = (size_t)b * g.P + hr.pbase;
    const int lane = tid & 63, wave = tid >> 6;
    const int col = tid % NC4, grp = tid / NC4, h = col / (D / 4);
    const int j0 = grp * nvalid / GR, j1 = grp < GR ? (grp + 1) * nvalid / GR : j0;
    const float4 *po = (const float4 *)s.ps_o;
    // the first loads of every phase are issued together (one memory round trip): this
    // thread's partial maximum and sum, and its first PF output partials
    constexpr int PF = G <= 2 ? 8 : (G <= 4 ? 7 : 4);   // 7 for G = 4: eight spill at 1024 threads
    float4 pf[PF];
#pragma unroll
    for (int u = 0; u < PF; ++u)
        pf[u] = j0 + u < j1 ? po[(base + part(j0 + u)) * NC4 + col] : make_float4(0.f, 0.f, 0.f, 0.f);
    float m0[G], l0[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        m0[hh] = tid < nvalid ? s.ps_m[(base + part(tid)) * G + hh] : -INFINITY;
        l0[hh] = tid < nvalid ? s.ps_l[(base + part(tid)) * G + hh] : 0.f;
    }
    float mloc[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) mloc[hh] = m0[hh];
    for (int j = tid + COMBINE_THREADS; j < nvalid; j += COMBINE_THREADS)
#pragma unroll
        for (int hh = 0; hh < G; ++hh) mloc[hh] = fmaxf(mloc[hh], s.ps_m[(base + part(j)) * G + hh]);
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        mloc[hh] = wave_max(mloc[hh]);
        if (lane == 0) red[wave * G + hh] = mloc[hh];
    }
    __syncthreads();
    float M[G], lsum[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        M[hh] = red[hh];
        for (int w = 1; w < NW; ++w) M[hh] = fmaxf(M[hh], red[w * G + hh]);
        lsum[hh] = 0.f;
    }
    if (tid < nvalid)
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            const float f = (M[hh] > -INFINITY && m0[hh] > -INFINITY) ? __expf(m0[hh] - M[hh]) : 0.f;
            sfac[tid * G + hh] = f;
            lsum[hh] += l0[hh] * f;
        }
    for (int j = tid + COMBINE_THREADS; j < nvalid; j += COMBINE_THREADS)
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            const float mj = s.ps_m[(base + part(j)) * G + hh];
            const float f = (M[hh] > -INFINITY && mj > -INFINITY) ? __expf(mj - M[hh]) : 0.f;
            sfac[j * G + hh] = f;
            lsum[hh] += s.ps_l[(base + part(j)) * G + hh] * f;
        }
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        lsum[hh] = wave_sum(lsum[hh]);
        if (lane == 0) redl[wave * G + hh] = lsum[hh];   // red still holds the maxima others read
    }
    __syncthreads();
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float4 *op = (float4 *)opart;   // [GR][NC4] float4 (the double buffer, reused)
    if (grp < GR) {
#pragma unroll
        for (int u = 0; u < PF; ++u)
            if (j0 + u < j1) {
                const float f = sfac[(j0 + u) * G + h];
                acc.x += pf[u].x * f, acc.y += pf[u].y * f, acc.z += pf[u].z * f, acc.w += pf[u].w * f;
            }
#pragma unroll 4
        for (int j = j0 + PF; j < j1; ++j) {
            const float4 v = po[(base + part(j)) * NC4 + col];
            const float f = sfac[j * G + h];
            acc.x += v.x * f, acc.y += v.y * f, acc.z += v.z * f, acc.w += v.w * f;
        }
        op[grp * NC4 + col] = acc;
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll 4
        for (int r = 1; r < GR; ++r) {
            const float4 o = op[r * NC4 + col];
            acc.x += o.x, acc.y += o.y, acc.z += o.z, acc.w += o.w;
        }
        const int lk = tidal ? t.tidal_lk[hi] : t.fixed_lk[hi - g.nT], l = lk / g.Hkv, kv = lk - l * g.Hkv;
        const size_t ob = (((size_t)b * g.L + l) * g.Hq + (size_t)kv * G) * D + (size_t)col * 4;
        float L = redl[h];
        for (int w = 1; w < NW; ++w) L += redl[w * G + h];
        const float li = L > 0.f ? 1.f / L : 0.f;
        store_out(out, ob, acc.x * li, g.out_bf16);
        store_out(out, ob + 1, acc.y * li, g.out_bf16);
        store_out(out, ob + 2, acc.z * li, g.out_bf16);
        store_out(out, ob + 3, acc.w * li, g.out_bf16);
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

// Decode-time append: grid (L * Hkv, B), one 64-thread group per head writes the token's K row
// (lanes 0-15) and V row (lanes 16-31) as sixteen 16-byte pieces each.
__global__ __launch_bounds__(64) void append_kv_kernel(Geometry g, const HeadRows *__restrict__ hr,
                                                       const int32_t *__restrict__ place, uint16_t *aK, uint16_t *aV,
                                                       uint16_t *tK, uint16_t *tV, uint16_t *fK, uint16_t *fV,
                                                       const uint16_t *__restrict__ k_new,
                                                       const uint16_t *__restrict__ v_new)
{
    const int lk = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
    if (lane >= 32) return;
    const int pl = place[lk], piece = lane & 15;
    const bool isv = lane >= 16;
    size_t row;
    uint16_t *dst;
    if (pl >= 0) {
        row = ((size_t)b * g.nA + pl) * g.Tcap + g.T;
        dst = isv ? aV : aK;
    } else {
        const int hi = -pl - 1;
        const bool tidal = hi < g.nT;
        const HeadRows h = hr[hi];
        row = (size_t)b * (tidal ? g.RsT : g.RsF) + h.srow + h.rs + g.n_gen;
        dst = tidal ? (isv ? tV : tK) : (isv ? fV : fK);
    }
    const size_t src = ((size_t)b * g.L * g.Hkv + lk) * D + piece * 8;
    *(uint4 *)(dst + row * D + piece * 8) = *(const uint4 *)((isv ? v_new : k_new) + src);
}

// Timing events of a launch that has no work: both recorded on the stream (the interval is empty).
hipError_t record_pair(hipEvent_t e0, hipEvent_t e1, hipStream_t st)
{
    hipError_t r = hipSuccess;
    if (e0) r = hipEventRecord(e0, st);
    if (e1 && r == hipSuccess) r = hipEventRecord(e1, st);
    return r;
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
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st,
                          hipEvent_t e0, hipEvent_t e1)
    {
        if (g.nA == 0 || g.n_tiles_a == 0) return record_pair(e0, e1, st);
        hipExtLaunchKernelGGL(anchor_attn_kernel<G>, dim3(g.n_tiles_a, g.nA, g.B), dim3(NT), 0, st, e0, e1, 0, g, t,
                              s, q);
        return hipGetLastError();
    }
};
template <int G>
struct AnchorMassL {
    static hipError_t run(const Geometry &g, const StepBuffers &s, hipStream_t st)
    {
        if (g.nA == 0) return hipSuccess;
        const size_t shm = (size_t)G * g.n_tiles_a * sizeof(double);
        hipLaunchKernelGGL(anchor_mass_kernel<G>, dim3(g.nA, g.B), dim3(MASS_THREADS), shm, st, g, s);
        return hipGetLastError();
    }
};
// Work-groups of a grid-stride launch: the tiles, at most as many as the compute units keep
// resident at once (the kernel's occupancy, queried once and kept in `cache`).
template <typename K>
long long resident_grid(K kernel, std::atomic<int> &cache, const Geometry &g, long long tiles)
{
    int per_cu = cache.load(std::memory_order_relaxed);
    if (per_cu == 0) {
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, NT, 0) != hipSuccess || per_cu < 1) {
            (void)hipGetLastError();
            per_cu = 1;
        }
        cache.store(per_cu, std::memory_order_relaxed);
    }
    return std::min<long long>(tiles, (long long)per_cu * std::max(g.n_cu, 1));
}

template <int G>
struct TidalFixedL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, bool recall,
                          bool with_static, long long items, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                          const SelectArgs *selp)
    {
        recall = recall && g.nT > 0 && g.k > 0 && g.comp_max > 0;
        const bool known = items >= 0 && !recall;
        SelectArgs sel{};
        if (selp) {
            sel = *selp;
            sel.n_mass = g.nA * g.B;
        }
        const long long tiles = (with_static ? (long long)g.n_static * g.B : 0) +
                                (known ? std::min<long long>(items, g.ng_kept) : g.ng_kept) * g.nT * g.B;
        if (tiles == 0 && !recall && sel.n_mass == 0) return record_pair(e0, e1, st);
        const dim3 block(NT);
        const int ws = with_static ? 1 : 0;
        static std::atomic<int> occ[4];
        if (!recall) {
            // the step's item count known on the host: one tile per work-group (the hardware
            // dispatches each work-group as another ends); else as many as stay resident, looping
            auto k = sel.n_mass ? tidal_fixed_kernel<G, RPL_S, false, true> : tidal_fixed_kernel<G, RPL_S, false, false>;
            const long long n = sel.n_mass + (known ? tiles : (tiles ? resident_grid(k, occ[sel.n_mass ? 3 : 0], g, tiles) : 0));
            hipExtLaunchKernelGGL(k, dim3((unsigned)n), block, 0, st, e0, e1, 0, g, t, s, q, ws, sel);
        } else if (g.slot_tile == TILE_S) {
            auto k = tidal_fixed_kernel<G, RPL_S, true, false>;
            const dim3 grid((unsigned)(RECALL_WGS + std::max(1LL, resident_grid(k, occ[1], g, tiles))));
            hipExtLaunchKernelGGL(k, grid, block, 0, st, e0, e1, 0, g, t, s, q, ws, SelectArgs{});
        } else {
            auto k = tidal_fixed_kernel<G, 2 * RPL_S, true, false>;
            const dim3 grid((unsigned)(RECALL_WGS + std::max(1LL, resident_grid(k, occ[2], g, tiles))));
            hipExtLaunchKernelGGL(k, grid, block, 0, st, e0, e1, 0, g, t, s, q, ws, SelectArgs{});
        }
        return hipGetLastError();
    }
};
template <int G>
struct TidalSelectFits {
    static bool run(const Geometry &g)
    {
        const size_t room = sizeof(SubsetSmem<G, RPL_S>) - SEL_SHARED_OFF;
        return g.nA > 0 && g.nc > 0 && select_shared_bytes(g) <= room && (size_t)G * g.n_tiles_a * sizeof(double) <= room;
    }
};
template <int G>
struct AttentionL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st,
                          hipEvent_t e0, hipEvent_t e1)
    {
        const long long n = (long long)g.n_tiles_a * g.nA * g.B + (long long)g.n_static * g.B;
        if (n == 0) return record_pair(e0, e1, st);
        if (n > INT32_MAX) return hipErrorInvalidValue;
        hipExtLaunchKernelGGL(attention_kernel<G>, dim3((unsigned)n), dim3(NT), 0, st, e0, e1, 0, g, t, s, q);
        return hipGetLastError();
    }
};
template <int G>
struct NewSlotsL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st)
    {
        if (g.nT == 0 || g.k == 0 || g.comp_max == 0) return hipSuccess;
        if (g.slot_tile == TILE_S)
            hipLaunchKernelGGL((new_slots_kernel<G, TILE_S / 16>), dim3(g.knew, g.nT, g.B), dim3(NT), 0, st, g, t, s, q);
        else
            hipLaunchKernelGGL((new_slots_kernel<G, TILE_S / 8>), dim3(g.knew, g.nT, g.B), dim3(NT), 0, st, g, t, s, q);
        return hipGetLastError();
    }
};
template <int G>
struct CombineL {
    static hipError_t run(const Geometry &g, const Tiers &t, const StepBuffers &s, void *out, hipStream_t st)
    {
        if (g.nT + g.nF + g.nA == 0) return hipSuccess;
        const size_t shm = std::max((size_t)(g.np_max ? g.np_max : 1) * G * sizeof(float),
                                    (size_t)G * g.n_tiles_a * sizeof(double));
        hipLaunchKernelGGL(subset_combine_kernel<G>, dim3(g.nT + g.nF + g.nA, g.B), dim3(COMBINE_THREADS), shm, st, g, t, s,
                           out);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_anchor(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st,
                         hipEvent_t e0, hipEvent_t e1)
{
    return dispatch_g<AnchorL>(g.G, g, t, s, q, st, e0, e1);
}

hipError_t launch_anchor_mass(const Geometry &g, const StepBuffers &s, hipStream_t st)
{
    return dispatch_g<AnchorMassL>(g.G, g, s, st);
}

hipError_t launch_select(const Geometry &g, const StepBuffers &s, float *scores, const int32_t *ovr,
                         int32_t *selected, hipStream_t st)
{
    if (g.nc == 0) return hipSuccess;
    hipLaunchKernelGGL(select_kernel, dim3(g.B), dim3(SEL_THREADS), select_shared_bytes(g), st, g, s, scores, ovr, selected);
    return hipGetLastError();
}

hipError_t launch_tidal_fixed(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, bool recall,
                              bool with_static, long long items, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                              const SelectArgs *sel)
{
    if (sel && (recall || !sel->s.arrive || !tidal_select_fits(g))) return hipErrorInvalidValue;
    return dispatch_g<TidalFixedL>(g.G, g, t, s, q, recall, with_static, items, st, e0, e1, sel);
}

bool tidal_select_fits(const Geometry &g)
{
    switch (g.G) {
    case 1: return TidalSelectFits<1>::run(g);
    case 2: return TidalSelectFits<2>::run(g);
    case 3: return TidalSelectFits<3>::run(g);
    case 4: return TidalSelectFits<4>::run(g);
    case 6: return TidalSelectFits<6>::run(g);
    case 8: return TidalSelectFits<8>::run(g);
    default: return false;
    }
}

hipError_t launch_attention(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st,
                            hipEvent_t e0, hipEvent_t e1)
{
    return dispatch_g<AttentionL>(g.G, g, t, s, q, st, e0, e1);
}

hipError_t launch_recall(const Geometry &g, const Tiers &t, const StepBuffers &s, hipStream_t st)
{
    if (g.nT == 0 || g.k == 0 || g.comp_max == 0) return hipSuccess;
    hipLaunchKernelGGL(recall_copy_kernel, dim3(RECALL_WGS), dim3(NT), 0, st, g, t, s);
    return hipGetLastError();
}

hipError_t launch_new_slots(const Geometry &g, const Tiers &t, const StepBuffers &s, const uint16_t *q, hipStream_t st)
{
    return dispatch_g<NewSlotsL>(g.G, g, t, s, q, st);
}

hipError_t launch_subset_combine(const Geometry &g, const Tiers &t, const StepBuffers &s, void *out, hipStream_t st)
{
    return dispatch_g<CombineL>(g.G, g, t, s, out, st);
}

hipError_t launch_append_kv(const Geometry &g, const HeadRows *hr, const int32_t *place, uint16_t *aK, uint16_t *aV,
                            uint16_t *tK, uint16_t *tV, uint16_t *fK, uint16_t *fV, const uint16_t *k_new,
                            const uint16_t *v_new, hipStream_t st)
{
    hipLaunchKernelGGL(append_kv_kernel, dim3(g.L * g.Hkv, g.B), dim3(64), 0, st, g, hr, place, aK, aV, tK, tV, fK, fV,
                       k_new, v_new);
    return hipGetLastError();
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
