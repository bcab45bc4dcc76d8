// Batched search on the matrix cores (section II-B step 5 for a tile of
// queries at once, with the filter of section III-B).
//
// Per tile of up to 32 queries:
//  1. prep_kernel: q' scaled by a power of two and rounded to float16, with
//     the per-query constants below.
//  2. mfma_scores_kernel: one pass over the code store.  Each 16-byte chunk
//     of 64 vectors (32 coordinates each) is turned into float16 centroid
//     values and multiplied with the query tile on v_mfma_f32_16x16x32_f16;
//     after a block's last chunk the approximate scores s_v <c_hat, q'> are
//     written, scaled to a float16 range, as a [query][vector] matrix, and
//     each query's largest score in the block as a [query][block] matrix.
//  3. Selection of at most KC candidates per query (KC = 256, or 512 for
//     k > 64) with a bound amin on the approximate score of every other
//     vector.  Unfiltered: block_select_kernel.  The R-th largest block
//     maximum (R = KC - 32) is a score of R distinct vectors, so at least R
//     vectors reach it, and every vector that does lies in a block whose
//     maximum reaches it: a radix selection over the block maxima lists
//     those blocks, and their vectors that reach it are the candidates
//     (about R when vectors sit at random positions; if more than KC, a
//     radix selection over the listed scores keeps the KC best).  Filtered
//     (the block maxima ignore the allowlist): select_kernel +
//     select_merge_kernel, the KC best allowed scores.
//  4. rescore_kernel: the exact score of each candidate with the
//     single-query scan's integer table (bit-identical scores), the top k of
//     them, and a certificate: with E a rigorous bound on |approximate -
//     exact| for every vector, a vector outside the candidates scores at
//     most amin + E; if that is below the k-th exact score the top k is
//     proven, otherwise the query is flagged and the caller re-runs it on
//     the single-query scan.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <type_traits>
#include <vector>

#include "kernels.h"
#include "lut.h"
#include "stream.h"
#include "topk.h"

namespace tq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

constexpr int kTile = 32;          // queries per pass over the codes: two MFMA row tiles of 16
constexpr int kCandMax = 512;      // candidates per query kept for exact rescoring (KC <= this)
constexpr int kCandMin = 64;
constexpr int kMaxBatchK = 256;    // largest k of the batched path
constexpr int BS_THREADS = 1024;   // block_select_kernel
constexpr int BS_WAVES = BS_THREADS / 64;
constexpr int kListMaxB = 8192;    // blocks a query's selection may list
constexpr int kHistCopies = 4;     // histogram copies (lane & 3), against atomic conflicts
constexpr int kHistStride = 257;   // words between copies: copies in different banks
// Selection outcome per query.
constexpr int kSelBound = 0;       // candidates + a bound amin on every other vector
constexpr int kSelOverflow = 1;    // no usable candidates: the query is not certified
constexpr int kSelAll = 2;         // every vector is a candidate
constexpr int MF_THREADS = 768;    // 12 waves: three per SIMD, 168 registers each
constexpr int MF_RING = 8;         // chunk loads in flight per wave
constexpr int kTableBytes = 256 * 32 * 4;   // byte table, 32 replicas
constexpr int SEL_THREADS = 256;
constexpr int SEL_GROUPS = 32;     // select workgroups per query
constexpr int kBoundStride = 32;  // ints between the global bounds of two queries
constexpr int kBuf = 8 * 64 + 64;  // per-wave candidate buffer: one load of 8 scores per lane + a partial 64
constexpr int kKeepVmemB = 0x1 | 0x2 | 0x4 | 0x8 | 0x80 | 0x100 | 0x200 | 0x400;

// Per-query constants written by prep_kernel.
struct QInfo {
    float f;      // stored approximate score = s_v * acc * f (acc: MFMA sum of the scaled query)
    float norm;   // approximate score = stored * norm  (s_max ||q'||_2)
    float err;    // bound on |approximate - exact| before the float16 storage
    float pad;
};

// ------------------------------------------------------------------- prep
// The query is scaled by alpha = 2^e with max|alpha q'_j| in [2^14, 2^15)
// and rounded to float16: alpha q'_j + eps_j.  With the float16 centroids
// c_l + delta_l (|delta_l| <= dmax, |c_l + delta_l| <= cmax16), the MFMA sum
// is alpha sum_j c q'_j + sum_j (alpha delta q'_j + (c + delta) eps_j), so
//   |acc / alpha - <c, q'>| <= dmax ||q'||_1 + cmax16 ||eps||_1 / alpha
// plus the float32 accumulation of d products in any order,
//   gamma_d cmax16 (||q'||_1 + ||eps||_1 / alpha),  gamma_d = d u / (1 - d u),
// u = 2^-24, and two float32 roundings when scaling (2^-23 of the same
// magnitude).  The exact score (the integer table of lut.h, d rows at
// b = 4) differs from s_v <c, q'> by the table's rounding: each entry is
// within 1/2 unit plus 2^-24 of its product, the integer sum is exact, and
// its float conversion and the product with s_v add 2^-24 each.  The table
// builder picks 2^sh > (2^31 - 1 - 2d) / (2 B'), B' = cmax tot (1 + 1e-5)
// with tot its float sum of |q'_j| (within 1e-6 of ||q'||_1), so the d/2
// units are below rho cmax ||q'||_1 in score units, rho = d (1 + 2e-5) /
// (2^31 - 1 - 2d); with the 2^-24 terms the exact score is within
// (rho + 4 * 2^-24) s_v cmax ||q'||_1 of s_v <c, q'> (cmax <= cmax16
// (1 + 2^-10): float16 rounding moves a value by at most 2^-11 of it).
// The sum of all terms times s_max is the error before storage (the factor
// 1.1 is margin only); the float16 storage of the approximate score adds at
// most 2^-11 of its magnitude plus 2^-25 norm, accounted for where the
// certificate is checked.
__global__ void prep_kernel(const float *__restrict__ Q, int nq, int d, const float *smax_p,
                            float cmax16, float dmax, _Float16 *__restrict__ q16,
                            QInfo *__restrict__ info) {
    __shared__ float red_m[SEL_THREADS / 64];
    __shared__ double red_1[SEL_THREADS / 64], red_2[SEL_THREADS / 64];
    const int q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float *row = Q + (int64_t)q * d;
    float m = 0.f;
    double s1 = 0.0, s2 = 0.0;
    for (int j = tid; j < d; j += SEL_THREADS) {
        const float v = row[j];
        m = fmaxf(m, fabsf(v));
        s1 += fabs((double)v);
        s2 += (double)v * v;
    }
    for (int o = 32; o > 0; o >>= 1) {
        m = fmaxf(m, __shfl_xor(m, o, 64));
        s1 += __shfl_xor(s1, o, 64);
        s2 += __shfl_xor(s2, o, 64);
    }
    if (lane == 0) {
        red_m[wave] = m;
        red_1[wave] = s1;
        red_2[wave] = s2;
    }
    __syncthreads();
    m = 0.f;
    s1 = 0.0;
    s2 = 0.0;
    for (int w = 0; w < SEL_THREADS / 64; ++w) {
        m = fmaxf(m, red_m[w]);
        s1 += red_1[w];
        s2 += red_2[w];
    }
    __syncthreads();   // red_1 is reused below
    const int e = m > 0.f ? 14 - ilogbf(m) : 0;
    const float alpha = ldexpf(1.0f, e);
    double se = 0.0;   // ||eps||_1
    for (int j = tid; j < d; j += SEL_THREADS) {
        const float a = row[j] * alpha;   // exact: alpha is a power of two
        const _Float16 h = (_Float16)a;
        q16[(int64_t)q * d + j] = h;
        se += fabs((double)(float)h - (double)a);
    }
    for (int o = 32; o > 0; o >>= 1) se += __shfl_xor(se, o, 64);
    if (lane == 0) red_1[wave] = se;
    __syncthreads();
    if (tid == 0) {
        se = 0.0;
        for (int w = 0; w < SEL_THREADS / 64; ++w) se += red_1[w];
        const double smax = (double)*smax_p;
        double norm = smax * sqrt(s2);
        if (!(norm > 0.0)) norm = 1.0;
        const double u = ldexp(1.0, -24);
        const double gd = d * u / (1.0 - d * u);
        const double mag = (double)cmax16 * (s1 + se / alpha);
        const double rho = d * (1.0 + 2e-5) / (2147483647.0 - 2.0 * d);
        const double tab = (rho + 4 * u) * (double)cmax16 * (1.0 + ldexp(1.0, -10)) * s1;
        const double E = (double)dmax * s1 + (double)cmax16 * se / alpha + gd * mag +
                         2 * ldexp(1.0, -23) * mag + tab;
        QInfo qi;
        qi.f = (float)(1.0 / ((double)alpha * norm));
        qi.norm = (float)norm;
        qi.err = (float)(1.1 * smax * E);
        qi.pad = 0.f;
        info[q] = qi;
    }
}

// ------------------------------------------------------------ MFMA scores
struct ScoreParams {
    const uint4 *codes;        // blocked store (b = 4)
    const float *scales;
    const _Float16 *q16;       // [nqt][d]
    const QInfo *info;         // [nqt]
    const float *cents;        // 16 levels
    _Float16 *out;             // [kTile][npad] approximate scores / norm
    _Float16 *bmax;            // [kTile][nblk] per-block maximum of out (vectors < n)
    int64_t n, nblk, npad;
    int d, chunks, nqt;
};

// Float16 centroids of the 8 4-bit fields of a stored word w (the canonical
// word rotated left by 2): element t is coordinate t of the word.  The byte
// table holds, for every byte value e, the pair (c[e & 15], c[e >> 4]) as
// two float16 -- one lookup per two coordinates.  It is replicated 32 times
// so that lane i reads only LDS bank i mod 32 (entry e of replica i is the
// 32-bit word e * 32 + i): lookups of random bytes by different lanes never
// meet in a bank.  `lb` is the lane's byte offset (lane mod 32) * 4.
__device__ inline half8 dequant8(uint32_t w, uint32_t lb) {
    typedef __attribute__((address_space(3))) const uint32_t lds_u32;
    const uint32_t cw = __builtin_amdgcn_alignbit(w, w, 2);   // canonical word
    union {
        uint32_t u[4];
        half8 h;
    } r;
    r.u[0] = *(lds_u32 *)(uintptr_t)(((cw << 7) & 0x7F80u) | lb);
    r.u[1] = *(lds_u32 *)(uintptr_t)(((cw >> 1) & 0x7F80u) | lb);
    r.u[2] = *(lds_u32 *)(uintptr_t)(((cw >> 9) & 0x7F80u) | lb);
    r.u[3] = *(lds_u32 *)(uintptr_t)(((cw >> 17) & 0x7F80u) | lb);
    return r.h;
}

// One workgroup of 12 waves per compute unit.  The byte table and the query
// tile (32 rows of d float16, rows padded by 16 bytes so the 16 rows read by
// one instruction fall in distinct banks) stay in LDS.  Waves claim the workgroup's
// 64-vector blocks one at a time from an LDS counter (one ahead, so the ring
// of MF_RING chunk loads runs on into the next block).  For a chunk, lane 16m+i
// (row m of 16 lanes) has loaded the 4 words of vector 16m+i; a 4 x 4
// transpose across the rows (two v_permlane32_swap, then two
// v_permlane16_swap) leaves word q of vectors i, 16+i, 32+i, 48+i in lane
// 16q+i: the B operands (k = 8q..8q+7, column i) of the four 16-vector
// MFMAs.
__global__ __launch_bounds__(MF_THREADS) void mfma_scores_kernel(ScoreParams p) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int ld = p.d + 8;                                   // row stride in halves
    uint32_t *T = reinterpret_cast<uint32_t *>(smem);          // byte table x 32, at 0
    _Float16 *Qs = reinterpret_cast<_Float16 *>(smem + kTableBytes);   // [kTile][ld]
    int *ctr = reinterpret_cast<int *>(smem + kTableBytes + (size_t)kTile * ld * 2);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int G = gridDim.x, g = blockIdx.x;
    const int CH = p.chunks;   // multiple of 8
    const int64_t gb0 = p.nblk * g / G, gb1 = p.nblk * (g + 1) / G;
    const int nbw = (int)(gb1 - gb0);

    // query tile, zero rows past nqt
    for (int e = tid; e < kTile * (p.d / 8); e += MF_THREADS) {
        const int r = e / (p.d / 8), c8 = e - r * (p.d / 8);
        uint4 v = make_uint4(0, 0, 0, 0);
        if (r < p.nqt) v = reinterpret_cast<const uint4 *>(p.q16 + (int64_t)r * p.d)[c8];
        *reinterpret_cast<uint4 *>(Qs + r * ld + c8 * 8) = v;
    }
    for (int e = tid; e < 256 * 32; e += MF_THREADS) {
        const int v = e >> 5;   // byte value; e & 31 is the replica
        const uint32_t lo = __builtin_bit_cast(uint16_t, (_Float16)p.cents[v & 15]);
        const uint32_t hi = __builtin_bit_cast(uint16_t, (_Float16)p.cents[v >> 4]);
        T[e] = lo | (hi << 16);
    }
    const uint32_t lb = (uint32_t)(lane & 31) * 4;
    if (tid == 0) *ctr = 0;
    // per-lane query factors: tile t, rows 4*(lane/16) + r
    float qf[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int q = 16 * t + 4 * (lane >> 4) + r;
            const float f = p.info[q < p.nqt ? q : 0].f;
            qf[t][r] = q < p.nqt ? f : 0.f;
        }
    __syncthreads();

    auto take = [&]() {
        int v = 0;
        if (lane == 0) v = atomicAdd(ctr, 1);
        return v;
    };
    int cur = __builtin_amdgcn_readfirstlane(take());
    if (cur >= nbw) return;
    int nxt = __builtin_amdgcn_readfirstlane(take());
    const uint4 *bsrc = p.codes + (gb0 + cur) * CH * 64;
    // the ring: named registers (an array would end up in scratch)
    uint4 rb0, rb1, rb2, rb3, rb4, rb5, rb6, rb7;
#define TQ_RING_LOAD(R, I)                          \
    R = load_stream(bsrc + (I) * 64 + lane);        \
    __builtin_amdgcn_sched_barrier(kKeepVmemB);
    TQ_RING_LOAD(rb0, 0)
    TQ_RING_LOAD(rb1, 1)
    TQ_RING_LOAD(rb2, 2)
    TQ_RING_LOAD(rb3, 3)
    TQ_RING_LOAD(rb4, 4)
    TQ_RING_LOAD(rb5, 5)
    TQ_RING_LOAD(rb6, 6)
    TQ_RING_LOAD(rb7, 7)
#undef TQ_RING_LOAD
    const int qrow = lane & 15, kq = lane >> 4;
    const _Float16 *qa0 = Qs + qrow * ld + kq * 8;
    const _Float16 *qa1 = Qs + (16 + qrow) * ld + kq * 8;
    while (true) {
        const int64_t blk = gb0 + cur;
        // the block after this one (or this one again past the end: cache hits)
        const uint4 *nsrc = nxt < nbw ? p.codes + (gb0 + nxt) * CH * 64 : bsrc;
        const int ticket = take();
        // unconditional loads (clamped index): a load under a branch makes the
        // wait-count pass drain the chunk ring in the loop below
        float scl[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int64_t v = blk * 64 + 16 * m + qrow;
            scl[m] = p.scales[v < p.n ? v : 0];
        }
        float4v acc[2][4];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int m = 0; m < 4; ++m) acc[t][m] = float4v{0.f, 0.f, 0.f, 0.f};
        // one chunk; the ring index is a compile-time constant at every call
        auto chunk = [&](const int c, uint4 &slot) {
            // W_q (row m) = word q of vector 16m+i.  permlane32_swap(a, b)
            // exchanges a's rows 2, 3 with b's rows 0, 1; permlane16_swap(a, b)
            // exchanges a's rows 1, 3 with b's rows 0, 2.  After both levels
            // r[m] (row q) = W_q (row m).
            const auto s02 = __builtin_amdgcn_permlane32_swap(slot.x, slot.z, false, false);
            const auto s13 = __builtin_amdgcn_permlane32_swap(slot.y, slot.w, false, false);
            const auto t01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
            const auto t23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
            const uint32_t r[4] = {t01[0], t01[1], t23[0], t23[1]};
            // refill MF_RING chunks ahead: this block, then the next one
            const int nc = c + MF_RING;
            slot = load_stream((nc < CH ? bsrc + nc * 64 : nsrc + (nc - CH) * 64) + lane);
            __builtin_amdgcn_sched_barrier(kKeepVmemB);
            const half8 a0 = *reinterpret_cast<const half8 *>(qa0 + c * 32);
            const half8 a1 = *reinterpret_cast<const half8 *>(qa1 + c * 32);
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const half8 b = dequant8(r[m], lb);
                acc[0][m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, b, acc[0][m], 0, 0, 0);
                acc[1][m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, b, acc[1][m], 0, 0, 0);
            }
        };
        static_assert(MF_RING == 8, "the chunk calls below assume a ring of 8");
        for (int c0 = 0; c0 < CH; c0 += MF_RING) {
            chunk(c0 + 0, rb0);
            chunk(c0 + 1, rb1);
            chunk(c0 + 2, rb2);
            chunk(c0 + 3, rb3);
            chunk(c0 + 4, rb4);
            chunk(c0 + 5, rb5);
            chunk(c0 + 6, rb6);
            chunk(c0 + 7, rb7);
        }
        // lane holds vectors 16m + qrow, queries 16t + 4*kq + r
        float mx[2][4];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) mx[t][r] = -INFINITY;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int64_t v = blk * 64 + 16 * m + qrow;
            const bool vin = v < p.n;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int q = 16 * t + 4 * kq + r;
                    const _Float16 h = (_Float16)(acc[t][m][r] * scl[m] * qf[t][r]);
                    if (q < p.nqt) p.out[(int64_t)q * p.npad + v] = h;
                    mx[t][r] = fmaxf(mx[t][r], vin ? (float)h : -INFINITY);
                }
        }
        // block maxima: the 16 lanes of a DPP row hold the block's 64 vectors
        // of the same queries
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float x = mx[t][r];
                x = fmaxf(x, dpp_f<kDppRowRor8>(x));
                x = fmaxf(x, dpp_f<kDppRowRor4>(x));
                x = fmaxf(x, dpp_f<kDppRowRor2>(x));
                x = fmaxf(x, dpp_f<kDppRowRor1>(x));
                const int q = 16 * t + 4 * kq + r;
                if (qrow == 0 && q < p.nqt) p.bmax[(int64_t)q * p.nblk + blk] = (_Float16)x;
            }
        if (nxt >= nbw) break;
        cur = nxt;
        nxt = __builtin_amdgcn_readfirstlane(ticket);
        bsrc = nsrc;
    }
}

// -------------------------------------------------------------- selection
struct SelectParams {
    const _Float16 *approx;    // [nqt][npad]
    const uint16_t *tenants;
    const uint64_t *allow;     // [nqt][W] or null
    float *cand_s;             // [nqt][SEL_GROUPS][KC]
    int *cand_i;
    int *gbound;               // [nqt * kBoundStride] order keys
    int64_t n, npad;
    int W;
};

// The KC = 64 S best allowed approximate scores of one query over
// 1/SEL_GROUPS of the vectors; each lane reads 8 consecutive scores per load.  A wave
// keeps its best kCand in registers; scores that pass its current bound are
// first appended to a per-wave LDS buffer, and the buffer is sorted into
// the list only when 64 have gathered -- a sort per 64 real candidates
// rather than per 64 scores read.
template <int S>
__global__ __launch_bounds__(SEL_THREADS) void select_kernel(SelectParams p) {
    constexpr int NW = SEL_THREADS / 64;
    constexpr int kCand = 64 * S, kCandS = S;
    __shared__ float st_s[NW * kCand];
    __shared__ int st_i[NW * kCand];
    __shared__ float buf_s[NW * kBuf];
    __shared__ int buf_i[NW * kBuf];
    __shared__ int wg_key;
    __shared__ uint64_t allow_s[64];
    const int g = blockIdx.x, q = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool filtered = p.allow != nullptr;
    if (tid == 0) wg_key = fkey(-INFINITY);
    if (filtered)
        for (int w = tid; w < p.W && w < 64; w += SEL_THREADS) allow_s[w] = p.allow[(int64_t)q * p.W + w];
    __syncthreads();
    int *gb = p.gbound + q * kBoundStride;
    float *bs = buf_s + wave * kBuf;
    int *bi = buf_i + wave * kBuf;
    int cnt = 0;   // wave-uniform
    const uint64_t below = (1ull << lane) - 1;
    // ranges of 512 vectors (one load per lane per wave)
    const int64_t units = p.npad / 512;
    const int64_t u0 = units * g / SEL_GROUPS, u1 = units * (g + 1) / SEL_GROUPS;
    WaveTopK<kCandS> top;
    top.reset();
    const uint4 *row = reinterpret_cast<const uint4 *>(p.approx + (int64_t)q * p.npad);
    for (int64_t u = u0 + wave; u < u1; u += NW) {
        const uint4 w = row[u * 64 + lane];
        // the global bound is read on every 4th load (each read is a trip to L2)
        const int gk = ((u - u0 - wave) & (4 * NW - 1)) == 0
                           ? __hip_atomic_load(gb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                           : top.seen_g;
        const int bk = max(max(gk, wg_key), max(top.seen_g, fkey(top.th_s)));
        const float thr = unfkey(bk);
        const _Float16 *h = reinterpret_cast<const _Float16 *>(&w);
        // append the 8 scores of each lane that pass the bound
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int64_t v = u * 512 + lane * 8 + e;
            bool ok = v < p.n;
            if (ok && filtered) {
                const int t = p.tenants[v];
                ok = (t >> 6) < p.W && ((allow_s[t >> 6] >> (t & 63)) & 1ull);
            }
            const float val = (float)h[e];
            const bool cand = ok && !(val < thr);
            const uint64_t m = __ballot(cand);
            if (cand) {
                const int pos = cnt + __popcll(m & below);
                bs[pos] = val;
                bi[pos] = (int)v;
            }
            cnt += __popcll(m);
        }
        __builtin_amdgcn_wave_barrier();
        // sort them in, 64 at a time (one copy of the sort in the code)
        while (cnt >= 64) {
            cnt -= 64;
            const float sc = bs[cnt + lane];
            const int id = bi[cnt + lane];
            __builtin_amdgcn_wave_barrier();
            top.offer_seen(sc, id, lane, kCand, &wg_key, gb, gk);
        }
    }
    if (cnt > 0) {
        const float sc = lane < cnt ? bs[lane] : -INFINITY;
        const int id = lane < cnt ? bi[lane] : INT_MAX;
        top.offer_seen(sc, id, lane, kCand, &wg_key, gb, top.seen_g);
    }
    // merge the wave lists
#pragma unroll
    for (int a = 0; a < kCandS; ++a) {
        st_s[wave * kCand + a * 64 + lane] = top.ls[a];
        st_i[wave * kCand + a * 64 + lane] = top.li[a];
    }
    __syncthreads();
    if (wave == 0) {
        for (int w = 1; w < NW; ++w) {
            float os[kCandS];
            int oi[kCandS];
#pragma unroll
            for (int a = 0; a < kCandS; ++a) {
                os[a] = st_s[w * kCand + a * 64 + lane];
                oi[a] = st_i[w * kCand + a * 64 + lane];
            }
            merge_lists<kCandS>(top.ls, top.li, os, oi, lane);
        }
        const int64_t base = ((int64_t)q * SEL_GROUPS + g) * kCand;
#pragma unroll
        for (int a = 0; a < kCandS; ++a) {
            p.cand_s[base + a * 64 + lane] = top.ls[a];
            p.cand_i[base + a * 64 + lane] = top.li[a];
        }
    }
}

// The KC = 64 S best of the SEL_GROUPS lists of each query: their ids, the
// approximate score of the KC-th, and the selection state (every allowed
// vector a candidate when fewer than KC).
template <int S>
__global__ __launch_bounds__(256) void select_merge_kernel(const float *__restrict__ cs,
                                                           const int *__restrict__ ci,
                                                           int *__restrict__ top_i,
                                                           float *__restrict__ amin,
                                                           int *__restrict__ state) {
    constexpr int kCand = 64 * S, kCandS = S;
    __shared__ float st_s[4 * kCand];
    __shared__ int st_i[4 * kCand];
    const int q = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    float ls[kCandS];
    int li[kCandS];
#pragma unroll
    for (int a = 0; a < kCandS; ++a) {
        ls[a] = -INFINITY;
        li[a] = INT_MAX;
    }
    for (int g = wave; g < SEL_GROUPS; g += 4) {
        const int64_t base = ((int64_t)q * SEL_GROUPS + g) * kCand;
        float os[kCandS];
        int oi[kCandS];
#pragma unroll
        for (int a = 0; a < kCandS; ++a) {
            os[a] = cs[base + a * 64 + lane];
            oi[a] = ci[base + a * 64 + lane];
        }
        merge_lists<kCandS>(ls, li, os, oi, lane);
    }
#pragma unroll
    for (int a = 0; a < kCandS; ++a) {
        st_s[wave * kCand + a * 64 + lane] = ls[a];
        st_i[wave * kCand + a * 64 + lane] = li[a];
    }
    __syncthreads();
    if (wave == 0) {
        for (int w = 1; w < 4; ++w) {
            float os[kCandS];
            int oi[kCandS];
#pragma unroll
            for (int a = 0; a < kCandS; ++a) {
                os[a] = st_s[w * kCand + a * 64 + lane];
                oi[a] = st_i[w * kCand + a * 64 + lane];
            }
            merge_lists<kCandS>(ls, li, os, oi, lane);
        }
#pragma unroll
        for (int a = 0; a < kCandS; ++a) top_i[(int64_t)q * kCand + a * 64 + lane] = li[a];
        const bool full = __shfl(li[kCandS - 1], 63, 64) != INT_MAX;
        if (lane == 63) {
            amin[q] = ls[kCandS - 1];
            state[q] = full ? kSelBound : kSelAll;
        }
    }
}

// ------------------------------------------- selection by block maxima
// Order-preserving map of float16 bit patterns onto 16-bit keys.
__device__ inline uint32_t hkey(uint32_t h) { return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u); }
__device__ inline float hkey_value(uint32_t key) {
    const uint32_t h = (key & 0x8000u) ? (key & 0x7FFFu) : (~key & 0xFFFFu);
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// Run by one whole wave once the histogram copies of a digit (256 bins) are
// complete: the digit d with (#keys whose digit > d) < K <= (#keys whose
// digit >= d), for 1 <= K <= #keys; out[0] = d, out[1] = #keys whose digit
// > d.  Lane l holds bins 4l .. 4l+3.
__device__ inline void find_digit(const int *hist, int K, int *out) {
    const int lane = threadIdx.x & 63;
    int c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int v = 0;
#pragma unroll
        for (int h = 0; h < kHistCopies; ++h) v += hist[h * kHistStride + 4 * lane + j];
        c[j] = v;
    }
    const int s = (c[0] + c[1]) + (c[2] + c[3]);
    int S = s;   // keys in the bins of lanes >= this one
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_down(S, o, 64);
        if (lane + o < 64) S += t;
    }
    const uint64_t ge = __ballot(S >= K);
    const int L = 63 - __builtin_clzll(ge);
    if (lane == L) {
        int above = S - s;
        int d = 4 * lane;
        for (int j = 3; j >= 0; --j) {
            if (above + c[j] >= K) {
                d = 4 * lane + j;
                break;
            }
            above += c[j];
        }
        out[0] = d;
        out[1] = above;
    }
}

struct BlockSelParams {
    const uint16_t *approx;    // [nqt][npad] float16 bit patterns
    const uint16_t *bmax;      // [nqt][nblk]
    int *top_i;                // [nqt][KC] candidate ids (INT_MAX: none)
    float *amin;               // [nqt] bound on the approximate score of non-candidates
    int *state;                // [nqt] kSel*
    int64_t n, nblk, npad;
    int KC;
};

// One workgroup per query (unfiltered), as described at the top of the
// file.  Keys are the float16 bit patterns mapped by hkey; a radix
// selection takes the high byte, then the low byte, with LDS histograms.
__global__ __launch_bounds__(BS_THREADS) void block_select_kernel(BlockSelParams p) {
    __shared__ int hist[kHistCopies * kHistStride];
    __shared__ int list[kListMaxB];
    __shared__ int sh[8];
    const int q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int KC = p.KC, R = KC - 32;
    const uint16_t *bm = p.bmax + (int64_t)q * p.nblk;
    const uint16_t *row = p.approx + (int64_t)q * p.npad;
    int *out_i = p.top_i + (int64_t)q * KC;
    int *hc = hist + (lane & 3) * kHistStride;
    auto clear_hist = [&]() {
        for (int i = tid; i < kHistCopies * kHistStride; i += BS_THREADS) hist[i] = 0;
    };
    // Visitors of the keys: block maxima (thread t: blocks t + 1024 u) and
    // the scores of the listed blocks (wave w: listed blocks w + 16 u, lane =
    // vector).  Up to BB block keys per thread and LB listed-block keys per
    // lane stay in registers across the passes (one round of loads); beyond
    // that the keys are loaded again, in rounds of RB, for every pass.
    // A round's loads are unconditional, from clamped indices, and all
    // issued before any is used (the empty asm keeps the compiler from
    // moving a load under the branch that uses it, where it would be waited
    // for on the spot and a round would run one load at a time).
    constexpr int BB = 16, LB = 40, RB = 8;
    const bool breg = p.nblk <= (int64_t)BB * BS_THREADS;
    // keys of blocks b0 + tid + 1024 u (0 past the end) into key[0..U)
    auto load_blocks = [&](int64_t b0, auto &key) {
        constexpr int U = sizeof(key) / sizeof(key[0]);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t b = b0 + tid + (int64_t)u * BS_THREADS;
            key[u] = bm[b < p.nblk ? b : p.nblk - 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) asm volatile("" : "+v"(key[u]));
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t b = b0 + tid + (int64_t)u * BS_THREADS;
            key[u] = b < p.nblk ? hkey(key[u]) : 0u;
        }
    };
    // keys of vectors vv[u] (0 past the end) into key[0..U)
    auto load_vectors = [&](const int64_t *vv, auto &key) {
        constexpr int U = sizeof(key) / sizeof(key[0]);
#pragma unroll
        for (int u = 0; u < U; ++u) key[u] = row[vv[u] < p.n ? vv[u] : p.n - 1];
#pragma unroll
        for (int u = 0; u < U; ++u) asm volatile("" : "+v"(key[u]));
#pragma unroll
        for (int u = 0; u < U; ++u) key[u] = vv[u] < p.n ? hkey(key[u]) : 0u;
    };
    uint32_t bk[BB];
    if (breg) load_blocks(0, bk);
    auto each_block = [&](auto fn) {
        if (breg) {
#pragma unroll
            for (int u = 0; u < BB; ++u) {
                const int64_t b = tid + (int64_t)u * BS_THREADS;
                if (b < p.nblk) fn(b, bk[u]);
            }
            return;
        }
        for (int64_t b0 = 0; b0 < p.nblk; b0 += (int64_t)RB * BS_THREADS) {
            uint32_t key[RB];
            load_blocks(b0, key);
#pragma unroll
            for (int u = 0; u < RB; ++u) {
                const int64_t b = b0 + tid + (int64_t)u * BS_THREADS;
                if (b < p.nblk) fn(b, key[u]);
            }
        }
    };
    uint32_t lk[LB];
    bool lreg = false;
    int nu = 0;   // listed blocks of this wave (register keys)
    auto load_listed = [&](int nl) {
        lreg = nl <= LB * BS_WAVES;
        if (!lreg) return;
        nu = nl > wave ? (nl - wave + BS_WAVES - 1) / BS_WAVES : 0;
        int64_t vv[LB];
#pragma unroll
        for (int u = 0; u < LB; ++u)
            vv[u] = u < nu ? (int64_t)list[wave + u * BS_WAVES] * 64 + lane : p.n;
        load_vectors(vv, lk);
    };
    auto each_listed = [&](int nl, auto fn) {
        if (lreg) {
#pragma unroll
            for (int u = 0; u < LB; ++u) {
                if (u >= nu) break;
                const int64_t v = (int64_t)list[wave + u * BS_WAVES] * 64 + lane;
                if (v < p.n) fn(v, lk[u]);
            }
            return;
        }
        for (int j0 = 0; j0 < nl; j0 += RB * BS_WAVES) {
            uint32_t key[RB];
            int64_t vv[RB];
#pragma unroll
            for (int u = 0; u < RB; ++u) {
                const int j = j0 + wave + u * BS_WAVES;
                vv[u] = j < nl ? (int64_t)list[j] * 64 + lane : p.n;
            }
            load_vectors(vv, key);
#pragma unroll
            for (int u = 0; u < RB; ++u) {
                const int j = j0 + wave + u * BS_WAVES;
                const int64_t v = j < nl ? (int64_t)list[j] * 64 + lane : p.n;
                if (v < p.n) fn(v, key[u]);
            }
        }
    };
    // radix selection: the K-th largest key (1 <= K <= #keys) of a visitor;
    // returns it and the number of keys above it
    auto kth = [&](auto each, int K, int &above) -> uint32_t {
        clear_hist();
        __syncthreads();
        each([&](int64_t, uint32_t key) { atomicAdd(&hc[key >> 8], 1); });
        __syncthreads();
        if (wave == 0) find_digit(hist, K, sh);
        __syncthreads();
        const int hi = sh[0], a1 = sh[1];
        clear_hist();
        __syncthreads();
        each([&](int64_t, uint32_t key) {
            if ((int)(key >> 8) == hi) atomicAdd(&hc[key & 255u], 1);
        });
        __syncthreads();
        if (wave == 0) find_digit(hist, K - a1, sh);
        __syncthreads();
        above = a1 + sh[1];
        const uint32_t t = ((uint32_t)hi << 8) | (uint32_t)sh[0];
        __syncthreads();   // sh is read before it is written again
        return t;
    };
    auto finish = [&](float am, int st) {
        if (tid == 0) {
            p.amin[q] = am;
            p.state[q] = st;
        }
    };
    // theta_a: the R-th largest block key (0, every block, when nblk <= R)
    const bool all_blocks = p.nblk <= R;
    uint32_t tha = 0;
    if (!all_blocks) {
        int above;
        tha = kth(each_block, R, above);
    }
    if (tid == 0) {
        sh[2] = 0;
        sh[3] = 0;
        sh[4] = 0;
        sh[5] = 0;
    }
    __syncthreads();
    each_block([&](int64_t b, uint32_t key) {
        if (key >= tha) {
            const int pos = atomicAdd(&sh[2], 1);
            if (pos < kListMaxB) list[pos] = (int)b;
        }
    });
    __syncthreads();
    const int nl = sh[2];
    if (nl > kListMaxB) {
        // too many blocks tie at the threshold: no candidates
        for (int i = tid; i < KC; i += BS_THREADS) out_i[i] = INT_MAX;
        finish(INFINITY, kSelOverflow);
        return;
    }
    load_listed(nl);
    if (all_blocks && p.n <= KC) {
        // every block listed and at most KC vectors: all are candidates
        each_listed(nl, [&](int64_t v, uint32_t) { out_i[atomicAdd(&sh[3], 1)] = (int)v; });
        __syncthreads();
        for (int i = sh[3] + tid; i < KC; i += BS_THREADS) out_i[i] = INT_MAX;
        finish(-INFINITY, kSelAll);
        return;
    }
    if (!all_blocks) {
        // the vectors that reach theta_a (at least R)
        each_listed(nl, [&](int64_t v, uint32_t key) {
            if (key >= tha) {
                const int pos = atomicAdd(&sh[3], 1);
                if (pos < KC) out_i[pos] = (int)v;
            }
        });
        __syncthreads();
        const int c = sh[3];
        if (c <= KC) {
            for (int i = c + tid; i < KC; i += BS_THREADS) out_i[i] = INT_MAX;
            finish(hkey_value(tha), kSelBound);
            return;
        }
    }
    // the KC best scores of the listed blocks
    int n_gt;
    const uint32_t thb = kth([&](auto fn) { each_listed(nl, fn); }, KC, n_gt);
    const int need_eq = KC - n_gt;   // keys equal to theta_b to take (>= 1)
    each_listed(nl, [&](int64_t v, uint32_t key) {
        if (key > thb) {
            out_i[atomicAdd(&sh[4], 1)] = (int)v;
        } else if (key == thb) {
            const int e = atomicAdd(&sh[5], 1);
            if (e < need_eq) out_i[n_gt + e] = (int)v;
        }
    });
    finish(hkey_value(thb), kSelBound);
}

// ------------------------------------------------------- exact rescoring
struct RescoreParams {
    const uint4 *codes;
    const float *scales;
    const float *qrot;         // [nqt][d] float32 rotated queries
    const float *cents;
    const int *top_i;          // [nqt][KC] candidates (INT_MAX: none)
    const float *amin;         // [nqt] bound on the approximate score of non-candidates
    const int *state;          // [nqt] kSel*
    const QInfo *info;
    int64_t *ids;              // [nqt][k]
    float *scores;
    int *flags;                // [nqt]: 1 = not certified
    int d, bits, chunks, lut_words, k;
};

// One workgroup per query, KC = 64 S candidate slots.
//  1. The query's integer table (as the single-query scan builds it).
//  2. Lane = candidate: wave w takes the 64 candidates of run w % S and the
//     (w / S)-th of 16 / S slices of the chunks, so all lanes read the same
//     table rows (as in the scan); partial integer sums meet in LDS (exact,
//     order-free): bit-identical to the single-query scan's scores.
//  3. Waves 0..S-1 sort their 64 exact scores; an entry's rank is its lane
//     plus, in every other sorted run, the number of entries ahead of it
//     (binary search); ranks below k are written.
//  4. Certificate: a vector outside the candidates has a stored score at
//     most amin, so its exact score is at most amin + 2^-11 |amin| +
//     2^-25 norm + err; if that is below the k-th exact score it cannot
//     enter the top k.
template <int S>
__global__ __launch_bounds__(kTableThreads) void rescore_kernel(RescoreParams p) {
    constexpr int KC = 64 * S;
    constexpr int SL = kTableWaves / S;    // chunk slices
    constexpr int CB = 12;                 // chunk loads of a lane in flight at once
    extern __shared__ __attribute__((aligned(16))) float lds[];
    float *red = lds + p.lut_words;         // 16
    int *sums = reinterpret_cast<int *>(red + 16);   // [KC]: integer sums, then ranks
    float *run_s = reinterpret_cast<float *>(sums + KC);
    int *run_i = reinterpret_cast<int *>(run_s + KC);
    int *sh = run_i + KC;                   // [0] valid count, [1] k-th exact score
    const int q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int run = wave % S, slice = wave / S;
    const int c0 = p.chunks * slice / SL, c1 = p.chunks * (slice + 1) / SL;
    const TableShape ts{p.d, p.bits, p.lut_words};
    for (int i = tid; i < KC; i += kTableThreads) sums[i] = 0;
    if (tid == 0) {
        sh[0] = 0;
        sh[1] = __float_as_int(-INFINITY);
    }
    // Loads in the order they are needed (completion is in order): the
    // query's coordinates, this lane's candidate, the certificate inputs,
    // then the candidate's chunks, in flight while the table is built.
    // Every load is unconditional, from a clamped address.
    float qv[2][4];
    load_nibble_query(ts, p.qrot + (int64_t)q * p.d, qv);
    const int v = p.top_i[(int64_t)q * KC + run * 64 + lane];
    const QInfo qi = p.info[q];
    const float amin_s = p.amin[q];
    const int st = p.state[q];
    const bool valid = v != INT_MAX;
    const int vc = valid ? v : 0;
    const uint4 *src = p.codes + ((int64_t)(vc >> 6) * p.chunks) * 64 + (vc & 63);
    const float scl = p.scales[vc];
    uint4 w[CB];
    auto load_chunks = [&](int cb) {
#pragma unroll
        for (int r = 0; r < CB; ++r) {
            const int c = cb + r < c1 ? cb + r : c0;
            w[r] = src[(int64_t)c * 64];
        }
    };
    load_chunks(c0);
    nibble_abs_sum(red, qv);
    __syncthreads();
    const int shx = build_nibble_table(lds, red, p.cents, ts, qv);
    __syncthreads();
    const char *lut = reinterpret_cast<const char *>(lds);
    int acc = 0;
    for (int cb = c0; cb < c1; cb += CB) {
        if (cb > c0) load_chunks(cb);
#pragma unroll
        for (int r = 0; r < CB; ++r)
            if (cb + r < c1) acc += nib_chunk(lut + (cb + r) * 2048, w[r]);
    }
    if (valid) atomicAdd(&sums[run * 64 + lane], acc);
    __syncthreads();
    // waves 0..S-1: sort their runs of 64 exact scores
    float s_ = -INFINITY;
    int i_ = INT_MAX;
    if (wave < S) {
        if (valid) {
            s_ = ldexpf((float)sums[run * 64 + lane] * scl, -shx);
            i_ = v;
        }
        wave_sort64(s_, i_, lane);
        run_s[wave * 64 + lane] = s_;
        run_i[wave * 64 + lane] = i_;
        const int c = __popcll(__ballot(i_ != INT_MAX));
        if (lane == 0 && c) atomicAdd(&sh[0], c);
    }
    __syncthreads();
    // rank of entry e = its place in its run + the entries ahead of it in
    // each other run (binary search); thread t searches for entry t % KC in
    // the runs (run(e) + 1 + t / KC + g * (1024 / KC)) % S
    for (int e = tid; e < KC; e += kTableThreads) sums[e] = e & 63;
    __syncthreads();
    {
        const int e = tid % KC, er = e >> 6;
        const float es = run_s[e];
        const int ei = run_i[e];
        int add = 0;
        if (ei != INT_MAX) {
            for (int o = 1 + tid / KC; o < S; o += kTableThreads / KC) {
                const int b = (er + o) % S;
                const float *rs = run_s + b * 64;
                const int *ri = run_i + b * 64;
                int pos = 0;
#pragma unroll
                for (int step = 64; step >= 1; step >>= 1)
                    if (pos + step <= 64 && better(rs[pos + step - 1], ri[pos + step - 1], es, ei))
                        pos += step;
                add += pos;
            }
        }
        if (add) atomicAdd(&sums[e], add);
    }
    __syncthreads();
    for (int e = tid; e < KC; e += kTableThreads) {
        const int ei = run_i[e];
        const int rank = sums[e];
        if (ei != INT_MAX && rank < p.k) {
            p.ids[(int64_t)q * p.k + rank] = (int64_t)ei;
            p.scores[(int64_t)q * p.k + rank] = run_s[e];
            if (rank == p.k - 1) sh[1] = __float_as_int(run_s[e]);
        }
    }
    __syncthreads();
    const int nv = sh[0];
    for (int r = nv + tid; r < p.k; r += kTableThreads) {
        p.ids[(int64_t)q * p.k + r] = -1;
        p.scores[(int64_t)q * p.k + r] = -INFINITY;
    }
    if (tid == 0) {
        const float ek = __int_as_float(sh[1]);
        const double amin = (double)amin_s * qi.norm;
        const double reach = amin + ldexp(1.0, -11) * fabs(amin) + ldexp(1.0, -25) * qi.norm +
                             (double)qi.err;
        const bool cert = st == kSelAll || (st == kSelBound && reach < (double)ek);
        p.flags[q] = cert ? 0 : 1;
    }
}

// ------------------------------------------------------ fallback helpers
// Global bounds are kept one 128-byte line apart (kBoundStride ints): every
// wave of a query's selection reads and raises its query's bound, and bounds
// of different queries sharing a line serialise each other.
__global__ void fill_order_keys(int *p, int n) {
    for (int i = threadIdx.x; i < n * kBoundStride; i += blockDim.x) p[i] = fkey(-INFINITY);
}

__global__ void gather_allow(const uint64_t *__restrict__ src, const int *__restrict__ rows, int nr,
                             int W, uint64_t *__restrict__ dst) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < (int64_t)nr * W;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(e / W);
        dst[e] = src[(int64_t)rows[r] * W + (e - (int64_t)r * W)];
    }
}

__global__ void gather_rows(const float *__restrict__ src, const int *__restrict__ rows, int nr,
                            int d, float *__restrict__ dst) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < (int64_t)nr * d;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(e / d);
        dst[e] = src[(int64_t)rows[r] * d + (e - (int64_t)r * d)];
    }
}

__global__ void scatter_results(const int64_t *__restrict__ ci, const float *__restrict__ cs,
                                const int *__restrict__ rows, int nr, int k,
                                int64_t *__restrict__ ids, float *__restrict__ scores) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < (int64_t)nr * k;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(e / k);
        const int64_t dst = (int64_t)rows[r] * k + (e - (int64_t)r * k);
        ids[dst] = ci[e];
        scores[dst] = cs[e];
    }
}

__global__ void scale_max_kernel(const float *__restrict__ s, int64_t n, int *smax_bits) {
    int m = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int b = __float_as_int(s[i]);   // scales are >= 0: bit order is value order
        m = b > m ? b : m;
    }
    for (int o = 32; o > 0; o >>= 1) {
        const int x = __shfl_xor(m, o, 64);
        m = x > m ? x : m;
    }
    if ((threadIdx.x & 63) == 0) atomicMax(smax_bits, m);
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// Candidate slots for a given k: eight per result, 64 to 512 (the
// certificate needs the KC-th approximate score, plus the error bound, to
// fall below the k-th exact one; candidates are cheap next to a re-run).
int batch_candidates(int k) {
    int kc = kCandMin;
    while (kc < 8 * k && kc < kCandMax) kc *= 2;
    return kc;
}

// Calls fn with std::integral_constant<int, KC / 64>.
template <class Fn>
void with_slots(int KC, Fn fn) {
    switch (KC) {
    case 64: fn(std::integral_constant<int, 1>()); break;
    case 128: fn(std::integral_constant<int, 2>()); break;
    case 256: fn(std::integral_constant<int, 4>()); break;
    default: fn(std::integral_constant<int, 8>()); break;
    }
}

struct BatchLayout {
    size_t q16, info, approx, bmax, cand_s, cand_i, top_i, amin, state, gbound, flags, rows, qc,
        allow_c, ids_c, scores_c, lut, total;
};

// Row length of the approximate-score matrix: whole 512-vector select units.
int64_t approx_row(const ScanShape &s) { return (s.nblk * 64 + 511) / 512 * 512; }

BatchLayout batch_layout(const ScanShape &s, int64_t nq, int k, int grid) {
    BatchLayout L{};
    size_t o = align256((size_t)nq * s.d * sizeof(float));   // rotated queries
    const int64_t npad = approx_row(s);
    L.q16 = o;
    o += align256((size_t)kTile * s.d * 2);
    L.info = o;
    o += align256(kTile * sizeof(QInfo));
    L.approx = o;
    o += align256((size_t)kTile * npad * 2);
    L.bmax = o;
    o += align256((size_t)kTile * s.nblk * 2);
    L.cand_s = o;
    o += align256((size_t)kTile * SEL_GROUPS * kCandMax * 4);
    L.cand_i = o;
    o += align256((size_t)kTile * SEL_GROUPS * kCandMax * 4);
    L.top_i = o;
    o += align256((size_t)kTile * kCandMax * 4);
    L.amin = o;
    o += align256((size_t)kTile * 4);
    L.state = o;
    o += align256((size_t)kTile * 4);
    L.gbound = o;
    o += align256(kTile * kBoundStride * 4);
    L.flags = o;
    o += align256((size_t)nq * 4);
    L.rows = o;
    o += align256((size_t)nq * 4);
    L.qc = o;
    o += align256((size_t)nq * s.d * sizeof(float));
    L.allow_c = o;
    o += align256((size_t)nq * s.W * sizeof(uint64_t));
    L.ids_c = o;
    o += align256((size_t)nq * k * 8);
    L.scores_c = o;
    o += align256((size_t)nq * k * 4);
    L.lut = o;
    o += lut_search_workspace_bytes(s, nq, k, grid);
    L.total = o + 256;
    return L;
}

}  // namespace

// LDS of the score kernel: replicated byte table, query tile, counter.
size_t score_lds_bytes(int d) {
    return kTableBytes + (size_t)kTile * (d + 8) * 2 + 16;
}

bool mfma_search_supported(const ScanShape &s, int k) {
    return s.bits == 4 && s.chunks % 8 == 0 && k <= kMaxBatchK && s.W <= 64 &&
           score_lds_bytes(s.d) <= 160 * 1024;
}

size_t mfma_search_workspace_bytes(const ScanShape &s, int64_t nq, int k, int grid) {
    return batch_layout(s, nq, k, grid).total;
}

hipError_t update_scale_max(const float *scales, int64_t n, float *smax, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    int64_t g = (n + 255) / 256;
    if (g > 2048) g = 2048;
    hipLaunchKernelGGL(scale_max_kernel, dim3((int)g), dim3(256), 0, stream, scales, n,
                       reinterpret_cast<int *>(smax));
    return hipGetLastError();
}

hipError_t mfma_search(const ScanShape &s, const uint8_t *blocked, const float *scales,
                       const float *smax, const uint16_t *tenants, const uint64_t *summaries,
                       const float *cents32, float cmax16, float dmax, const float *Qrot,
                       int64_t nq, int k,
                       const uint64_t *allow, int grid, void *ws, int64_t *ids, float *scores,
                       int *n_fallback, hipStream_t stream) {
    const BatchLayout L = batch_layout(s, nq, k, grid);
    uint8_t *w8 = static_cast<uint8_t *>(ws);
    _Float16 *q16 = reinterpret_cast<_Float16 *>(w8 + L.q16);
    QInfo *info = reinterpret_cast<QInfo *>(w8 + L.info);
    _Float16 *approx = reinterpret_cast<_Float16 *>(w8 + L.approx);
    _Float16 *bmax = reinterpret_cast<_Float16 *>(w8 + L.bmax);
    float *cand_s = reinterpret_cast<float *>(w8 + L.cand_s);
    int *cand_i = reinterpret_cast<int *>(w8 + L.cand_i);
    int *top_i = reinterpret_cast<int *>(w8 + L.top_i);
    float *amin = reinterpret_cast<float *>(w8 + L.amin);
    int *state = reinterpret_cast<int *>(w8 + L.state);
    int *gbound = reinterpret_cast<int *>(w8 + L.gbound);
    int *flags = reinterpret_cast<int *>(w8 + L.flags);
    const int64_t npad = approx_row(s);
    const size_t lds_scores = score_lds_bytes(s.d);
    const int KC = batch_candidates(k);   // candidates per query
    // table, 16 floats, integer sums and sorted (score, id) runs, two counters
    const size_t lds_rescore = (size_t)s.chunks * 2048 + 16 * 4 + (size_t)KC * 12 + 16;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)mfma_scores_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        for (int S = 1; S <= 8 && e == hipSuccess; S *= 2)
            with_slots(64 * S, [&](auto sc) {
                e = hipFuncSetAttribute((const void *)rescore_kernel<decltype(sc)::value>,
                                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            });
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    for (int64_t q0 = 0; q0 < nq; q0 += kTile) {
        const int nqt = (int)((nq - q0) < kTile ? (nq - q0) : kTile);
        hipLaunchKernelGGL(prep_kernel, dim3(nqt), dim3(SEL_THREADS), 0, stream, Qrot + q0 * s.d,
                           nqt, s.d, smax, cmax16, dmax, q16, info);
        ScoreParams sp{};
        sp.codes = reinterpret_cast<const uint4 *>(blocked);
        sp.scales = scales;
        sp.q16 = q16;
        sp.info = info;
        sp.cents = cents32;
        sp.out = approx;
        sp.bmax = bmax;
        sp.n = s.n;
        sp.nblk = s.nblk;
        sp.npad = npad;
        sp.d = s.d;
        sp.chunks = s.chunks;
        sp.nqt = nqt;
        hipLaunchKernelGGL(mfma_scores_kernel, dim3(grid), dim3(MF_THREADS), lds_scores, stream, sp);
        if (allow) {
            // the block maxima ignore the allowlist: select over every allowed score
            hipLaunchKernelGGL(fill_order_keys, dim3(1), dim3(64), 0, stream, gbound, nqt);
            SelectParams sl{};
            sl.approx = approx;
            sl.tenants = tenants;
            sl.allow = allow + q0 * s.W;
            sl.cand_s = cand_s;
            sl.cand_i = cand_i;
            sl.gbound = gbound;
            sl.n = s.n;
            sl.npad = npad;
            sl.W = s.W;
            with_slots(KC, [&](auto sc) {
                constexpr int S = decltype(sc)::value;
                hipLaunchKernelGGL(select_kernel<S>, dim3(SEL_GROUPS, nqt), dim3(SEL_THREADS), 0,
                                   stream, sl);
                hipLaunchKernelGGL(select_merge_kernel<S>, dim3(nqt), dim3(256), 0, stream, cand_s,
                                   cand_i, top_i, amin, state);
            });
        } else {
            BlockSelParams bp{};
            bp.approx = reinterpret_cast<const uint16_t *>(approx);
            bp.bmax = reinterpret_cast<const uint16_t *>(bmax);
            bp.top_i = top_i;
            bp.amin = amin;
            bp.state = state;
            bp.n = s.n;
            bp.nblk = s.nblk;
            bp.npad = npad;
            bp.KC = KC;
            hipLaunchKernelGGL(block_select_kernel, dim3(nqt), dim3(BS_THREADS), 0, stream, bp);
        }
        RescoreParams rp{};
        rp.codes = reinterpret_cast<const uint4 *>(blocked);
        rp.scales = scales;
        rp.qrot = Qrot + q0 * s.d;
        rp.cents = cents32;
        rp.top_i = top_i;
        rp.amin = amin;
        rp.state = state;
        rp.info = info;
        rp.ids = ids + q0 * k;
        rp.scores = scores + q0 * k;
        rp.flags = flags + q0;
        rp.d = s.d;
        rp.bits = s.bits;
        rp.chunks = s.chunks;
        rp.lut_words = s.chunks * 512;
        rp.k = k;
        with_slots(KC, [&](auto sc) {
            constexpr int S = decltype(sc)::value;
            hipLaunchKernelGGL(rescore_kernel<S>, dim3(nqt), dim3(kTableThreads), lds_rescore, stream,
                               rp);
        });
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // queries whose top k is not proven run on the single-query scan
    std::vector<int> hf((size_t)nq);
    hipError_t e = hipMemcpyAsync(hf.data(), flags, nq * sizeof(int), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return e;
    std::vector<int> rows;
    for (int64_t i = 0; i < nq; ++i)
        if (hf[i]) rows.push_back((int)i);
    *n_fallback = (int)rows.size();
    if (rows.empty()) return hipSuccess;
    const int nr = (int)rows.size();
    int *rows_d = reinterpret_cast<int *>(w8 + L.rows);
    float *qc = reinterpret_cast<float *>(w8 + L.qc);
    int64_t *ids_c = reinterpret_cast<int64_t *>(w8 + L.ids_c);
    float *scores_c = reinterpret_cast<float *>(w8 + L.scores_c);
    e = hipMemcpyAsync(rows_d, rows.data(), nr * sizeof(int), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(gather_rows, dim3(256), dim3(256), 0, stream, Qrot, rows_d, nr, s.d, qc);
    uint64_t *allow_c = nullptr;
    if (allow) {
        allow_c = reinterpret_cast<uint64_t *>(w8 + L.allow_c);
        hipLaunchKernelGGL(gather_allow, dim3(64), dim3(256), 0, stream, allow, rows_d, nr, s.W,
                           allow_c);
    }
    SearchFilter f;
    f.allow = allow_c;
    e = lut_search(s, blocked, scales, tenants, summaries, cents32, qc, nr, k, f, grid,
                   w8 + L.lut, lut_search_workspace_bytes(s, nq, k, grid), ids_c, scores_c, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scatter_results, dim3(256), dim3(256), 0, stream, ids_c, scores_c, rows_d, nr,
                       k, ids, scores);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(stream);   // host vectors above go out of scope
    return e;
}

}  // namespace tq
