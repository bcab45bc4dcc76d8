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
//  3. Selection of at most KC candidates per query (KC = eight per result,
//     64 to 512) with a bound amin on the approximate score of every other
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

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <type_traits>
#include <utility>
#include <vector>

#include "kernels.h"
#include "lds_dma.h"
#include "lut.h"
#include "stream.h"
#include "topk.h"

namespace tq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef float float16v __attribute__((ext_vector_type(16)));

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
constexpr int kTicketStride = 32;  // ints between two workgroups' ticket counters (own 128 B line)
// Last word of a raw buffer resource (stride 0, byte offsets): 32-bit data
// format, so untyped loads, stores and atomics are bounds-checked by bytes.
constexpr int kBufferWord3 = 0x00020000;
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
                            QInfo *__restrict__ info, int *__restrict__ zero, int nzero) {
    __shared__ float red_m[SEL_THREADS / 64];
    __shared__ double red_1[SEL_THREADS / 64], red_2[SEL_THREADS / 64];
    const int q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (q == 0)
        for (int i = tid; i < nzero; i += SEL_THREADS) zero[i] = 0;   // the score kernel's tickets
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
    _Float16 *out;             // [kTile][npad] approximate scores / norm (rows >= nqt: 0)
    _Float16 *bmax;            // [kTile][nblk] per-block maximum of out (vectors < n)
    int *tickets;              // [grid * kTicketStride] block ticket counters, zero at launch
    int64_t n, nblk, npad;
    int d, chunks, nqt;
};

// Float16 centroids of the 8 4-bit fields of a stored word w (the canonical
// word rotated left by 2): element t is coordinate t of the word.  The byte
// table holds, for every byte value e, the pair (c[e & 15], c[e >> 4]) as
// two float16 -- one lookup per two coordinates.  It is replicated NR times
// so that the lanes of a read meet distinct LDS banks whatever bytes they
// look up (entry e of replica i is the 32-bit word e * NR + i, read by lane
// i mod NR).
//  NR = 64: the word address e * 256 + 4 * lane has the byte e in byte 1 and
//    the lane's offset `lb` = 4 * lane in byte 0, so one byte permute of the
//    canonical word and lb forms it (64 KiB of table).
//  NR = 32: ((e << 7) | lb), lb = 4 * (lane mod 32), takes a shift or
//    field extract and an and-or per lookup (32 KiB of table).
template <int NR>
__device__ inline half8 dequant8_canonical(uint32_t cw, uint32_t lb) {
    typedef __attribute__((address_space(3))) const uint32_t lds_u32;
    union {
        uint32_t u[4];
        half8 h;
    } r;
    if constexpr (NR == 64) {
        // v_perm selector: byte 0 <- lb byte 0, byte 1 <- cw byte b, bytes 2, 3 <- 0
#pragma unroll
        for (int b = 0; b < 4; ++b)
            r.u[b] = *(lds_u32 *)(uintptr_t)__builtin_amdgcn_perm(cw, lb, 0x0C0C0400u + (b << 8));
    } else {
        r.u[0] = *(lds_u32 *)(uintptr_t)(((cw << 7) & 0x7F80u) | lb);
        r.u[1] = *(lds_u32 *)(uintptr_t)(((cw >> 1) & 0x7F80u) | lb);
        r.u[2] = *(lds_u32 *)(uintptr_t)(((cw >> 9) & 0x7F80u) | lb);
        r.u[3] = *(lds_u32 *)(uintptr_t)(((cw >> 17) & 0x7F80u) | lb);
    }
    return r.h;
}
template <int NR>
__device__ inline half8 dequant8(uint32_t w, uint32_t lb) {
    return dequant8_canonical<NR>(__builtin_amdgcn_alignbit(w, w, 2), lb);   // canonical word
}

// Copies of a ring slot's four words into registers of their own.  The
// exchanges below overwrite their operands in place; on the slot itself they
// make the register allocator move the slot's refill into other registers
// and copy it back at the loop's back edge, which waits for every load in
// flight (the ring drains once per eight chunks).  An opaque copy frees the
// slot for its refill at once.
__device__ inline void copy4(const uint4 &v, uint32_t &a, uint32_t &b, uint32_t &c, uint32_t &d) {
    asm volatile("v_mov_b32 %0, %4\n\tv_mov_b32 %1, %5\n\tv_mov_b32 %2, %6\n\tv_mov_b32 %3, %7"
                 : "=v"(a), "=v"(b), "=v"(c), "=v"(d)
                 : "v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w));
}

// Replicas of the score kernel's byte table: 64 where the table (64 KiB)
// and the query tile (kTile x d float16) fit the 160 KiB of LDS together.
__host__ __device__ constexpr int score_replicas(int d) {
    return 64 * 1024 + kTile * d * 2 <= 160 * 1024 ? 64 : 32;
}

// One workgroup of 12 waves per compute unit.  The byte table and the query
// tile stay in LDS; the tile is stored in the A-operand order of the MFMAs
// (chunk c, row tile t: 64 lanes x 16 bytes, lane 16 kq + i holding row
// 16 t + i, k = 32 c + 8 kq .. + 7), so each operand read is one 16-byte read
// per lane at consecutive addresses.  Waves claim the workgroup's 64-vector
// blocks one at a time from the workgroup's ticket counter in memory (one
// ahead, so the ring of MF_RING chunk loads runs on into the next block).
template <int NR>
__global__ __launch_bounds__(MF_THREADS) void mfma_scores_kernel(ScoreParams p) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    uint32_t *T = reinterpret_cast<uint32_t *>(smem);                    // byte table, at 0
    uint4 *Qf = reinterpret_cast<uint4 *>(smem + (size_t)NR * 256 * 4);   // [chunk][2][64]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int G = gridDim.x, g = blockIdx.x;
    const int CH = p.chunks;   // multiple of 8
    const int64_t gb0 = p.nblk * g / G, gb1 = p.nblk * (g + 1) / G;
    const int nbw = (int)(gb1 - gb0);

    // query tile in operand order, zero rows past nqt
    for (int e = tid; e < CH * 128; e += MF_THREADS) {
        const int c = e >> 7, t = (e >> 6) & 1, l = e & 63;
        const int r = 16 * t + (l & 15);
        uint4 v = make_uint4(0, 0, 0, 0);
        if (r < p.nqt)
            v = *reinterpret_cast<const uint4 *>(p.q16 + (int64_t)r * p.d + 32 * c + 8 * (l >> 4));
        Qf[e] = v;
    }
    for (int e = tid; e < 256 * NR; e += MF_THREADS) {
        const int v = e / NR;   // byte value; e % NR is the replica
        const uint32_t lo = __builtin_bit_cast(uint16_t, (_Float16)p.cents[v & 15]);
        const uint32_t hi = __builtin_bit_cast(uint16_t, (_Float16)p.cents[v >> 4]);
        T[e] = lo | (hi << 16);
    }
    const uint32_t lb = (uint32_t)(lane & (NR - 1)) * 4;
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

    // The ticket is a buffer atomic issued by every lane, of which only lane
    // 0's lies inside the 4-byte buffer: bounds checking drops the others'
    // adds (their value is 0).  An atomic under a branch on lane 0 instead
    // leaves the wait-count pass unsure of the loads in flight, and it then
    // drains the chunk ring inside the chunk loop.
    const __amdgpu_buffer_rsrc_t trs =
        __builtin_amdgcn_make_buffer_rsrc(p.tickets + g * kTicketStride, 0, 4, kBufferWord3);
    auto take = [&]() {
        return __builtin_amdgcn_raw_ptr_buffer_atomic_add_i32(1, trs, lane == 0 ? 0 : 4, 0, 0);
    };
    int cur = __builtin_amdgcn_readfirstlane(take());
    if (cur >= nbw) return;
    int nxt = __builtin_amdgcn_readfirstlane(take());
    const uint4 *bsrc = p.codes + (gb0 + cur) * CH * 64;   // uniform: the block's chunk 0
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
    const uint4 *qa = Qf + lane;
    const int qrow = lane & 15, kq = lane >> 4;
    // a wave scores at most the workgroup's nbw blocks: the bound ends the
    // loop even if the tickets were to stop advancing
    for (int iter = 1;; ++iter) {
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
            // r[m] (row q) = W_q (row m): word q of vectors i, 16+i, 32+i,
            // 48+i in lane 16q+i, the B operands (k = 8q..8q+7, column i) of
            // the four 16-vector MFMAs.  The exchanges work on copies, and the
            // slot is refilled right after the copy.
            uint32_t cx, cy, cz, cw;
            copy4(slot, cx, cy, cz, cw);
            // refill MF_RING chunks ahead: this block, then the next one
            {
                const int nc = c + MF_RING;
                slot = load_stream((nc < CH ? bsrc + nc * 64 : nsrc + (nc - CH) * 64) + lane);
                __builtin_amdgcn_sched_barrier(kKeepVmemB);
            }
            const auto s02 = __builtin_amdgcn_permlane32_swap(cx, cz, false, false);
            const auto s13 = __builtin_amdgcn_permlane32_swap(cy, cw, false, false);
            const auto t01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
            const auto t23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
            const uint32_t r[4] = {t01[0], t01[1], t23[0], t23[1]};
            const half8 a0 = __builtin_bit_cast(half8, qa[c * 128]);
            const half8 a1 = __builtin_bit_cast(half8, qa[c * 128 + 64]);
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const half8 b = dequant8<NR>(r[m], lb);
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
        // lane holds vectors 16m + qrow, queries 16t + 4*kq + r.  The stores
        // are unconditional (rows past nqt are zero scores in rows that the
        // workspace holds and nothing reads; the 16 lanes of a row store the
        // same block maximum): a store under a branch leaves the wait-count
        // pass unsure of the loads in flight, and it then drains the chunk
        // ring inside the chunk loop.
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
                    p.out[(int64_t)q * p.npad + v] = h;
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
                p.bmax[(int64_t)q * p.nblk + blk] = (_Float16)x;
            }
        if (nxt >= nbw || iter >= nbw) break;
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

// ============================================================ wide passes
// Passes of 65 to 256 queries (QP = 128 or 256 query slots) read the code
// store once per pass and keep no score matrix (passes of at most 64 queries
// take tiles of 32, which are faster there):
//  1. prep_kernel, then frag_kernel: the float16 queries in the A operand
//     order of v_mfma_f32_32x32x16_f16.  Piece (c, f, l) (16 bytes) holds
//     coordinates 32c + 16(f & 1) + 8(l >> 5) .. +7 of query
//     32(f >> 1) + (l & 31), so the query part of a chunk is QP * 64
//     contiguous bytes, and lane l of a wave reads fragment f (query tile
//     f / 2, k-half f & 1) at offset (f * 64 + l) * 16.
//  2. wide_scores_kernel, pilot launch: tiles of NG blocks (every pstride-th
//     tile of the store, at most one per workgroup); every approximate score
//     of their vectors is written, [query][pilot vector].
//  3. pilot_select_kernel: per query, theta = the KC-th largest allowed
//     pilot score (-inf when at most KC pilot vectors are allowed), and the
//     allowed pilot vectors that reach it as candidates.  At least KC
//     vectors of the store score theta or more.
//  4. wide_scores_kernel, main launch: every other tile; a vector whose
//     score reaches its query's theta (and whose tenant the query allows) is
//     appended to the workgroup's list for that query.
//  5. final_select_kernel: the KC best of the pilot's and the workgroups'
//     candidates, and amin = the KC-th one's score.  A vector that is not
//     taken scores below theta <= amin (never appended) or at most amin
//     (behind the KC-th), which is the bound the certificate needs.
//  6. rescore_kernel: exact scores, top k and certificate, as for tiles.
// Work items of the score kernel are steps (tile, chunk): for each, the
// workgroup stages one slab in LDS -- the chunk's query pieces and the
// chunk of each of its NG blocks -- and its eight waves multiply them: wave
// w takes block w % NG of the tile against query half w / NG (QW queries).
// Slabs go straight from global memory into a ring of NB LDS buffers
// (direct loads, NB - 2 steps ahead); one barrier per step publishes the
// next slab, whose codes are turned into MFMA operands while the current
// slab is multiplied.
constexpr int WD_THREADS = 512;
constexpr int WD_WAVES = WD_THREADS / 64;
constexpr int PS_THREADS = 1024;               // pilot_select_kernel, final_select_kernel
constexpr int kPilotMax = 65536;               // pilot vectors per query (16-bit keys in 128 KiB of LDS)
constexpr int kFinalMax = 16384;               // candidates a query's final selection gathers
constexpr int kWideMaxQ = 256;
constexpr int kWideMinQ = 64;                 // passes of more queries take the wide path (fewer: tiles of 32)
constexpr int kWideMinChunks = 8;            // chunks per vector of a wide pass: more than its slabs ahead

// Order-preserving map of float32 onto uint32; 0 marks an absent entry
// (below every finite value and -inf).
__device__ inline uint32_t ukey(float f) {
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ inline float ukey_value(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__global__ void frag_kernel(const _Float16 *__restrict__ q16, const QInfo *__restrict__ info,
                            int nqt, int QP, int d, uint4 *__restrict__ qfrag,
                            float *__restrict__ qf) {
    const int64_t per_chunk = (int64_t)QP * 4;
    const int64_t tot = (int64_t)(d / 32) * per_chunk;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < tot;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(e / per_chunk);
        const int rem = (int)(e - c * per_chunk);
        const int f = rem >> 6, l = rem & 63;   // fragment (query tile f / 2, k-half f & 1)
        const int q = 32 * (f >> 1) + (l & 31);
        uint4 v = make_uint4(0, 0, 0, 0);
        if (q < nqt)
            v = *reinterpret_cast<const uint4 *>(q16 + (int64_t)q * d + 32 * c + 16 * (f & 1) +
                                                 8 * (l >> 5));
        qfrag[e] = v;
    }
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < QP;
         q += (int64_t)gridDim.x * blockDim.x)
        qf[q] = q < nqt ? info[q].f : 0.f;
}

struct WideParams {
    const uint4 *codes;        // blocked store (b = 4)
    const float *scales;
    const uint4 *qfrag;        // [chunks][QP * 4] query pieces
    const float *qf;           // [QP] score factor (0 for unused slots)
    const float *cents;        // 16 levels
    int64_t n, nblk, ntiles;   // tiles of NG blocks
    int chunks, pstride, npil; // pilot tiles: i * pstride, i < npil
    int pilot;                 // 1: pilot launch, 0: main launch (selects the kernel)
    float *pil;                // pilot: [QP][npil * 64 NG] scores
    const float *theta;        // main: [nqt] thresholds
    const uint16_t *tenants;   // main, filtered
    const uint64_t *allow;     // main: [nqt][W] allowlists, or null
    int W, nqt;
    float *cand_s;             // main: [grid][QP][S] appended scores and ids
    int *cand_i;
    int *cand_n;               // main: [grid][QP] appended per workgroup and query
    int S;
};

constexpr int WD_NG = 4;                       // blocks per tile (wave w: block w % 4)
constexpr int WD_NH = WD_WAVES / WD_NG;        // query halves (wave w: half w / 4)

// Slab buffers in LDS per query-slot count.  A slab holds the chunk's QF
// query pieces (pieces 0..QF-1) and the chunk of each of the tile's 4 blocks
// (pieces QF..QF+3), 1 KiB each; piece i is loaded by wave i % 8 as its
// (i / 8)-th load and stored at position (i % 8) DW + i / 8, so that each
// wave's pieces are contiguous (one LDS base per wave and slab; DW = the
// most loads a wave makes per slab).  NB buffers hold the slab being
// multiplied, the next one (whose codes are turned into operands meanwhile)
// and NB - 2 in flight.
template <int QW>
struct WideShape {
    static constexpr int QP = QW * WD_NH;
    static constexpr int QF = QP / 16;                 // query pieces of a slab
    static constexpr int NI = QF + WD_NG;              // 1 KiB pieces of a slab
    static constexpr int DW = (NI + WD_WAVES - 1) / WD_WAVES;
    static constexpr int SU = WD_WAVES * DW * 64;      // uint4 of a slab
    static constexpr int NB = QW == 128 ? 5 : 7;       // slab buffers
    static constexpr int PD = NB - 1;                  // slabs requested ahead
    static constexpr size_t lds = kTableBytes + (size_t)NB * SU * 16 + 2 * 1024 +
                                  3 * (size_t)QP * 4;
    // uint4 offset of piece i within a slab
    static constexpr int pos(int i) { return ((i % WD_WAVES) * DW + i / WD_WAVES) * 64; }
};

template <int QW, bool PILOT>
__global__ __launch_bounds__(WD_THREADS) void wide_scores_kernel(WideParams p) {
    using WS = WideShape<QW>;
    constexpr int QP = WS::QP, QF = WS::QF, NI = WS::NI, SU = WS::SU, NB = WS::NB, PD = WS::PD;
    static_assert(WS::DW * 1024 <= 4096, "a wave's loads of a slab within one instruction-offset span");
    constexpr int NG = WD_NG;
    constexpr int QT = QW / 32;                // 32-query tiles of a wave
    constexpr int QU = QF * 64;                // uint4 of a slab's query part
    // 1 KiB loads of a slab per wave: load i goes to wave i % 8
    constexpr int DHI = (NI + WD_WAVES - 1) / WD_WAVES, NHI = NI - (DHI - 1) * WD_WAVES;
    static_assert(PD >= 2, "the next slab must be present a step ahead");
    extern __shared__ __attribute__((aligned(16))) char smem[];
    uint32_t *T = reinterpret_cast<uint32_t *>(smem);                 // byte table x 32
    uint4 *slab = reinterpret_cast<uint4 *>(smem + kTableBytes);      // [NB][SU]
    float *sclv = reinterpret_cast<float *>(slab + NB * SU);           // [2][256] tile scales
    float *fq = sclv + 512;                                            // [QP]
    float *th = fq + QP;                                               // [QP]
    int *cnt = reinterpret_cast<int *>(th + QP);                       // [QP]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar branches
    const int g = wave % NG, h = wave / NG;
    const int G = gridDim.x, wg = blockIdx.x;
    const int CH = p.chunks;
    const int64_t nt_all = PILOT ? p.npil : p.ntiles - p.npil;
    const int64_t my_tiles = nt_all > wg ? (nt_all - wg + G - 1) / G : 0;
    // the i-th tile of this workgroup
    auto tile_of = [&](int64_t i) -> int64_t {
        const int64_t j = wg + i * G;
        if (PILOT) return j * p.pstride;
        const int64_t r = p.pstride - 1;   // >= 1 whenever there are main tiles
        return (j / r) * p.pstride + 1 + j % r;
    };

    for (int e = tid; e < 256 * 32; e += WD_THREADS) {
        const int v = e >> 5;
        const uint32_t lo = __builtin_bit_cast(uint16_t, (_Float16)p.cents[v & 15]);
        const uint32_t hi = __builtin_bit_cast(uint16_t, (_Float16)p.cents[v >> 4]);
        T[e] = lo | (hi << 16);
    }
    for (int q = tid; q < QP; q += WD_THREADS) {
        fq[q] = p.qf[q];
        th[q] = (!PILOT && q < p.nqt) ? p.theta[q] : INFINITY;
        cnt[q] = 0;
    }
    if (my_tiles > 0) {
        const uint32_t lb = (uint32_t)(lane & 31) * 4;
        const uint32_t slab_lds = (uint32_t)(uintptr_t)slab;
        const uint32_t scl_lds = (uint32_t)(uintptr_t)sclv;
        // this wave's loads of a slab: DHI of them for waves below NHI
        const bool hi_wave = wave < NHI;
        // next slab to request: tile ordinal, tile, chunk, buffer
        int64_t ld_i = 0, ld_tile = tile_of(0);
        int ld_c = 0, ld_b = 0;
        // the j-th load of this wave for the next slab to request (piece
        // i = 8j + wave, stored at this wave's base + j KiB); request_base
        // first, once per slab
        auto request_base = [&]() {
            set_lds_base(slab_lds + (uint32_t)ld_b * (SU * 16) + (uint32_t)(wave * WS::DW) * 1024);
        };
        auto request_part = [&](auto J) {
            constexpr int j = decltype(J)::value;
            const int i = j * WD_WAVES + wave;
            if (i < NI) {   // uniform
                if (i < QF) {
                    lds_dma16_at<j, false>(p.qfrag + (int64_t)ld_c * QU + i * 64 + lane);
                } else {
                    int64_t b = ld_tile * NG + (i - QF);
                    b = b < p.nblk ? b : p.nblk - 1;
                    lds_dma16_at<j, true>(p.codes + (b * CH + ld_c) * 64 + lane);
                }
            }
        };
        auto request_done = [&]() {
            if (ld_c == 0 && wave == WD_WAVES - 1) {
                // the tile's 256 scales (4 per lane, block clamped like the codes)
                int64_t v = ld_tile * 256 + 4 * lane;
                if (v >= p.nblk * 64) v -= (ld_tile * NG + lane / 16 - (p.nblk - 1)) * 64;
                lds_dma16(p.scales + v, scl_lds + (uint32_t)(ld_i & 1) * 1024);
            }
            ld_b = ld_b + 1 == NB ? 0 : ld_b + 1;
            // past the last step the last tile's slabs are requested again (unused)
            if (++ld_c == CH) {
                ld_c = 0;
                if (ld_i + 1 < my_tiles) ld_tile = tile_of(++ld_i);
            }
        };
        auto request = [&]() {
            request_base();
            request_part(std::integral_constant<int, 0>());
            if constexpr (DHI > 1) request_part(std::integral_constant<int, 1>());
            if constexpr (DHI > 2) request_part(std::integral_constant<int, 2>());
            static_assert(DHI <= 3, "at most three loads per wave and slab");
            request_done();
        };
        // until the oldest requested slab but `ahead` has landed
        auto wait_slabs = [&](auto ahead) {
            constexpr int A = decltype(ahead)::value;
            if (hi_wave) wait_vmem<A * DHI>();
            else wait_vmem<A * (DHI - 1)>();
        };
        // B operands of a chunk: b[2m + ks] for vectors 32m .. 32m + 31 of the
        // wave's block and coordinates 16ks .. 16ks + 15 of the chunk (lane l:
        // vector 32m + (l & 31), coordinates 16ks + 8(l >> 5) .. +7).  Lane v
        // holds words 0..3 of vector v; permlane32_swap(w0, w1) leaves word 0
        // of vectors 0..31 in lanes 0..31 and word 1 of the same vectors in
        // lanes 32..63 (first result), and words 0, 1 of vectors 32..63 the
        // same way (second); likewise (w2, w3) for the second k-half.
        half8 bcur[4];
        auto operands = [&](const uint4 *sb, half8 (&b)[4]) {
            const uint4 w = sb[WS::pos(QF + g) + lane];
            const auto k0 = __builtin_amdgcn_permlane32_swap(w.x, w.y, false, false);
            const auto k1 = __builtin_amdgcn_permlane32_swap(w.z, w.w, false, false);
            b[0] = dequant8<32>(k0[0], lb);   // vectors 0..31, k-half 0
            b[1] = dequant8<32>(k1[0], lb);   // vectors 0..31, k-half 1
            b[2] = dequant8<32>(k0[1], lb);   // vectors 32..63, k-half 0
            b[3] = dequant8<32>(k1[1], lb);   // vectors 32..63, k-half 1
        };
#pragma unroll 1
        for (int x = 0; x < PD; ++x) request();
        wait_slabs(std::integral_constant<int, PD - 1>());
        lds_barrier();
        operands(slab, bcur);
        // this wave's A operands of a slab: fragment 2t + ks of its query half
        half8 acur[2 * QT];
        auto a_operands = [&](const uint4 *sb) {
#pragma unroll
            for (int f = 0; f < 2 * QT; ++f)
                acur[f] = reinterpret_cast<const half8 *>(sb)[WS::pos(h * 2 * QT + f) + lane];
        };
        a_operands(slab);

        float16v acc[QT][2];
        auto clear_acc = [&]() {
#pragma unroll
            for (int t = 0; t < QT; ++t)
#pragma unroll
                for (int m = 0; m < 2; ++m)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[t][m][e] = 0.f;
        };
        clear_acc();
        int64_t ti = 0;       // tile ordinal of the current step
        int64_t tile = tile_of(0);
        int buf = 0;          // buffer of the current step's slab
        // lane holds vectors 32m + (lane & 31) of its block and, in element e
        // of tile t, query h QW + 32t + 8(e >> 2) + 4(lane >> 5) + (e & 3)
        auto epilogue = [&]() {
            // hq is made opaque so that the per-query offsets below are
            // formed here, once per tile, rather than hoisted out of the step
            // loop into registers held across it
            int hq = h * QW + 4 * (lane >> 5);
            asm volatile("" : "+v"(hq));
            const float *ts = sclv + (ti & 1) * 256 + g * 64 + (lane & 31);
            const float scl[2] = {ts[0], ts[32]};
            const int64_t vb = (tile * NG + g) * 64 + (lane & 31);
            const bool vin[2] = {vb < p.n, vb + 32 < p.n};
            if constexpr (PILOT) {
                const int64_t prow = (int64_t)p.npil * 64 * NG;
                const int64_t pcol = (wg + ti * G) * 64 * NG + g * 64 + (lane & 31);
#pragma unroll
                for (int t = 0; t < QT; ++t)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int q = hq + 32 * t + 8 * (e >> 2) + (e & 3);
                        const float f = fq[q];
#pragma unroll
                        for (int m = 0; m < 2; ++m)
                            p.pil[q * prow + pcol + 32 * m] = vin[m] ? acc[t][m][e] * scl[m] * f : -INFINITY;
                    }
            } else {
                // which entries reach their query's threshold, without
                // branches (bit 2e + m of hit[t]) ...
                uint32_t hit[QT];
#pragma unroll
                for (int t = 0; t < QT; ++t) {
                    uint32_t hb = 0u;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        // four queries' factors and thresholds, read together
                        const float4 f4 = *reinterpret_cast<const float4 *>(fq + hq + 32 * t + 8 * i);
                        const float4 t4 = *reinterpret_cast<const float4 *>(th + hq + 32 * t + 8 * i);
                        const float fr[4] = {f4.x, f4.y, f4.z, f4.w}, tr[4] = {t4.x, t4.y, t4.z, t4.w};
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int e = 4 * i + j;
                            hb |= (vin[0] && acc[t][0][e] * scl[0] * fr[j] >= tr[j]) ? 1u << (2 * e) : 0u;
                            hb |= (vin[1] && acc[t][1][e] * scl[1] * fr[j] >= tr[j]) ? 2u << (2 * e) : 0u;
                        }
                    }
                    hit[t] = hb;
                }
                // ... then append those (rare): one entry per lane and round,
                // its value picked out of the accumulators by its bit index
                // (a fixed select chain: the accumulators stay in registers)
                uint32_t pend[QT];
#pragma unroll
                for (int t = 0; t < QT; ++t) pend[t] = hit[t];
                auto any_pending = [&]() {
                    uint32_t o = 0u;
#pragma unroll
                    for (int t = 0; t < QT; ++t) o |= pend[t];
                    return o != 0u;
                };
                while (__ballot(any_pending())) {
                    if (any_pending()) {
                        int bt = 0;   // lowest pending bit: tile bt, bit bb = 2e + m
#pragma unroll
                        for (int t = QT - 1; t >= 0; --t)
                            if (pend[t]) bt = t;
                        uint32_t word = pend[0];
#pragma unroll
                        for (int t = 1; t < QT; ++t) word = bt == t ? pend[t] : word;
                        const int bb = __builtin_ctz(word);
#pragma unroll
                        for (int t = 0; t < QT; ++t)
                            if (bt == t) pend[t] &= pend[t] - 1u;
                        float a = 0.f;
#pragma unroll
                        for (int t = 0; t < QT; ++t)
#pragma unroll
                            for (int e = 0; e < 16; ++e)
#pragma unroll
                                for (int m = 0; m < 2; ++m)
                                    a = (bt == t && bb == 2 * e + m) ? acc[t][m][e] : a;
                        const int e = bb >> 1, m = bb & 1;
                        const int q = hq + 32 * bt + 8 * (e >> 2) + (e & 3);
                        const float val = a * scl[m] * fq[q];
                        const int64_t v = vb + 32 * m;
                        bool ok = true;
                        if (p.allow) {
                            const int tn = p.tenants[v];
                            ok = (tn >> 6) < p.W &&
                                 ((p.allow[(int64_t)q * p.W + (tn >> 6)] >> (tn & 63)) & 1ull);
                        }
                        if (ok) {
                            const int slot = atomicAdd(&cnt[q], 1);
                            if (slot < p.S) {
                                const int64_t o = ((int64_t)wg * QP + q) * p.S + slot;
                                p.cand_s[o] = val;
                                p.cand_i[o] = (int)v;
                            }
                        }
                    }
                }
            }
            clear_acc();
        };
        for (;;) {
            for (int c = 0; c < CH; ++c) {
                // the next step's slab has landed (own loads), then everyone's;
                // every wave is done with the buffer the new request overwrites
                wait_slabs(std::integral_constant<int, PD - 2>());
                lds_barrier();
                // the products of slab s (operands read a step ahead) in groups
                // of two; the code word of slab s + 1 turned into the next B
                // operands, and this step's loads, are issued between the
                // groups so that they overlap the matrix cores' work
                buf = buf + 1 == NB ? 0 : buf + 1;
                const uint4 wn = slab[buf * SU + WS::pos(QF + g) + lane];
                half8 bnext[4];
                // k-half outer, so that the two products into one accumulator
                // are 2 QT products apart (a product waits for the previous
                // one into the same accumulator to finish)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                    for (int t = 0; t < QT; ++t) {
                        const half8 a = acur[2 * t + ks];
                        acc[t][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bcur[ks], acc[t][0], 0, 0, 0);
                        acc[t][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bcur[2 + ks], acc[t][1], 0, 0, 0);
                        const int grp = ks * QT + t;   // groups of two products
                        if (grp == 0) {
                            const auto k0 = __builtin_amdgcn_permlane32_swap(wn.x, wn.y, false, false);
                            const auto k1 = __builtin_amdgcn_permlane32_swap(wn.z, wn.w, false, false);
                            bnext[0] = dequant8<32>(k0[0], lb);
                            bnext[1] = dequant8<32>(k1[0], lb);
                            bnext[2] = dequant8<32>(k0[1], lb);
                            bnext[3] = dequant8<32>(k1[1], lb);
                        }
                        if (grp == 1) {
                            request_base();
                            request_part(std::integral_constant<int, 0>());
                        }
                        if constexpr (DHI > 1)
                            if (grp == 2) request_part(std::integral_constant<int, 1>());
                        if constexpr (DHI > 2)
                            if (grp == 3) request_part(std::integral_constant<int, 2>());
                        __builtin_amdgcn_sched_barrier(0);
                    }
                // loads that found no group after them
                if constexpr (DHI > 1 && 2 * QT <= 2) request_part(std::integral_constant<int, 1>());
                if constexpr (DHI > 2 && 2 * QT <= 3) request_part(std::integral_constant<int, 2>());
                request_done();
                // the next slab's A operands, read now so that they arrive
                // while this wave waits at the next barrier
                a_operands(slab + buf * SU);
#pragma unroll
                for (int m = 0; m < 4; ++m) bcur[m] = bnext[m];
            }
            epilogue();
            if (++ti == my_tiles) break;
            tile = tile_of(ti);
            // the next step's operands again (its slab stays in place until the
            // next request): not held in registers across the epilogue
            a_operands(slab + buf * SU);
            operands(slab + buf * SU, bcur);
        }
    }
    if (!PILOT) {
        __syncthreads();
        for (int q = tid; q < QP; q += WD_THREADS) p.cand_n[(int64_t)wg * QP + q] = cnt[q];
    }
}

// K-th largest of the BITS-bit keys visited by `each` (K >= 1, at most the
// number of non-zero keys; zero keys are absent): 8-bit radix passes with
// LDS histograms.  Returns the key and sets n_above to the number of
// keys above it.  Called by every thread of the workgroup.
template <int BITS, class Each>
__device__ uint32_t radix_kth(Each each, int K, int *hist, int *sh, int &n_above) {
    static_assert(BITS % 8 == 0, "8-bit digits");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int *hc = hist + (lane & 3) * kHistStride;
    uint32_t prefix = 0, pmask = 0;
    int above = 0;
    for (int pass = 0; pass < BITS / 8; ++pass) {
        const int shift = BITS - 8 - 8 * pass;
        for (int i = tid; i < kHistCopies * kHistStride; i += blockDim.x) hist[i] = 0;
        __syncthreads();
        // the lanes of a wave that share the first active lane's digit add
        // their count once (the high digits of one query's scores are mostly
        // equal, and their single-lane atomics would serialise); the others
        // add one each
        each([&](uint32_t k) {
            const bool act = k != 0u && (k & pmask) == prefix;
            const uint32_t dg = (k >> shift) & 255u;
            const uint64_t live = __ballot(act);
            if (live) {
                const int leader = __builtin_ctzll(live);
                const uint32_t dl = __builtin_amdgcn_readlane(dg, leader);
                const bool same = act && dg == dl;
                const uint64_t sm = __ballot(same);
                if (lane == leader) atomicAdd(&hc[dl], (int)__popcll(sm));
                else if (act && !same) atomicAdd(&hc[dg], 1);
            }
        });
        __syncthreads();
        if (wave == 0) find_digit(hist, K - above, sh);
        __syncthreads();
        prefix |= (uint32_t)sh[0] << shift;
        pmask |= 255u << shift;
        above += sh[1];
        __syncthreads();   // sh is read before it is written again
    }
    n_above = above;
    return prefix;
}

struct PilotParams {
    const float *pil;          // [QP][npv]
    int64_t npv;               // pilot vectors per query (npil * 64 WD_NG)
    int pstride;
    int64_t n;
    const uint16_t *tenants;
    const uint64_t *allow;     // [nqt][W] or null
    int W, KC, PCM;
    float *theta;              // [nqt]
    int *pc_n;                 // [nqt] pilot candidates (may exceed PCM: overflow)
    int *pc_i;                 // [nqt][PCM]
    float *pc_s;
};

// One workgroup per query.  The selection runs on 16-bit keys, the top half
// of the order-preserving key of each allowed pilot score, held in LDS: the
// KC-th largest such key kt gives theta = the smallest float whose key starts
// with kt, so at least KC allowed pilot vectors score theta or more, and a
// pilot vector reaches theta exactly when its 16-bit key reaches kt.
__global__ __launch_bounds__(PS_THREADS) void pilot_select_kernel(PilotParams p) {
    constexpr int TV = 64 * WD_NG;                 // vectors per pilot tile
    extern __shared__ __attribute__((aligned(16))) uint16_t k16[];   // [npv], 0: absent
    __shared__ int hist[kHistCopies * kHistStride];
    __shared__ int sh[8];
    const int q = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int npv = (int)p.npv;
    const float *row = p.pil + (int64_t)q * p.npv;
    const uint64_t *arow = p.allow ? p.allow + (int64_t)q * p.W : nullptr;
    auto vec_of = [&](int e) -> int64_t { return (int64_t)(e / TV) * p.pstride * TV + e % TV; };
    if (tid == 0) {
        sh[4] = 0;
        sh[5] = 0;
    }
    __shared__ uint64_t allow_s[64];
    if (arow)
        for (int w = tid; w < p.W; w += PS_THREADS) allow_s[w] = arow[w];
    __syncthreads();
    int cnt = 0;
    // rounds of 16 loads per thread, all issued before any is used
    constexpr int R = 16;
    for (int e0 = 0; e0 < npv; e0 += R * PS_THREADS) {
        float val[R];
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int e = e0 + tid + u * PS_THREADS;
            val[u] = row[e < npv ? e : 0];
        }
        int tn[R];
        if (arow) {
#pragma unroll
            for (int u = 0; u < R; ++u) {
                const int e = e0 + tid + u * PS_THREADS;
                tn[u] = p.tenants[vec_of(e < npv ? e : 0)];
            }
        }
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int e = e0 + tid + u * PS_THREADS;
            if (e < npv) {
                bool ok = val[u] > -INFINITY;
                if (arow)
                    ok = ok && (tn[u] >> 6) < p.W && ((allow_s[tn[u] >> 6] >> (tn[u] & 63)) & 1ull);
                k16[e] = ok ? (uint16_t)(ukey(val[u]) >> 16) : (uint16_t)0;   // a finite key's top half is >= 0x80
                cnt += ok;
            }
        }
    }
    for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
    __syncthreads();
    if (lane == 0) atomicAdd(&sh[5], cnt);
    __syncthreads();
    const int allowed = sh[5];
    uint32_t thk = 1u;   // every present key
    if (allowed > p.KC) {
        int n_above;
        thk = radix_kth<16>([&](auto fn) {
            for (int e = tid; e < npv; e += PS_THREADS) fn((uint32_t)k16[e]);
        }, p.KC, hist, sh, n_above);
    }
    if (tid == 0) p.theta[q] = allowed > p.KC ? ukey_value(thk << 16) : -INFINITY;
    for (int e = tid; e < npv; e += PS_THREADS) {
        const uint32_t k = k16[e];
        if (k != 0u && k >= thk) {
            const int pos = atomicAdd(&sh[4], 1);
            if (pos < p.PCM) {
                p.pc_i[(int64_t)q * p.PCM + pos] = (int)vec_of(e);
                p.pc_s[(int64_t)q * p.PCM + pos] = row[e];
            }
        }
    }
    __syncthreads();
    if (tid == 0) p.pc_n[q] = sh[4];
}

struct FinalParams {
    const float *theta;
    const int *pc_n;
    const int *pc_i;
    const float *pc_s;
    int PCM;
    const float *cand_s;       // [G][QP][S]
    const int *cand_i;
    const int *cand_n;         // [G][QP]
    int G, QP, S, KC;
    int *top_i;                // [nqt][KC] (INT_MAX: none)
    float *amin;
    int *state;
};

// One workgroup per query: the query's candidates gathered in LDS, then the
// KC best.
__global__ __launch_bounds__(PS_THREADS) void final_select_kernel(FinalParams p) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    uint32_t *ck = reinterpret_cast<uint32_t *>(smem);        // [kFinalMax] keys
    int *cv = reinterpret_cast<int *>(ck + kFinalMax);         // [kFinalMax] ids
    __shared__ int hist[kHistCopies * kHistStride];
    __shared__ int sh[8];
    const int q = blockIdx.x, tid = threadIdx.x;
    int *out = p.top_i + (int64_t)q * p.KC;
    __shared__ int goff[1025];                  // exclusive offsets of the workgroup lists
    __shared__ int wsum[PS_THREADS / 64];
    const int lane = tid & 63, wave = tid >> 6;
    const int n0 = p.pc_n[q];
    const int base = n0 < p.PCM ? n0 : p.PCM;
    if (tid == 0) {
        sh[3] = n0 > p.PCM;         // overflow
        sh[4] = 0;
        sh[5] = 0;
    }
    __syncthreads();
    // the G list lengths (G <= PS_THREADS), an exclusive scan over them
    int c = 0;
    if (tid < p.G) {
        c = p.cand_n[(int64_t)tid * p.QP + q];
        if (c > p.S) sh[3] = 1;
    }
    int incl = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(incl, o, 64);
        if (lane >= o) incl += t;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    goff[tid] = base + before + incl - c;
    if (tid == PS_THREADS - 1) goff[PS_THREADS] = base + before + incl;
    __syncthreads();
    const int ng = p.G < PS_THREADS ? p.G : PS_THREADS;
    const int total_all = goff[ng];
    for (int e = tid; e < base && e < kFinalMax; e += PS_THREADS) {
        ck[e] = ukey(p.pc_s[(int64_t)q * p.PCM + e]);
        cv[e] = p.pc_i[(int64_t)q * p.PCM + e];
    }
    if (!sh[3] && total_all <= kFinalMax) {
        for (int e = base + tid; e < total_all; e += PS_THREADS) {
            int lo = 0, hi = ng - 1;   // last list whose offset is <= e
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (goff[mid] <= e) lo = mid;
                else hi = mid - 1;
            }
            const int64_t src = ((int64_t)lo * p.QP + q) * p.S + (e - goff[lo]);
            ck[e] = ukey(p.cand_s[src]);
            cv[e] = p.cand_i[src];
        }
    }
    if (tid == 0) sh[2] = total_all;
    __syncthreads();
    const int tot = sh[2];
    const float theta = p.theta[q];
    if (sh[3] || tot > kFinalMax) {
        for (int i = tid; i < p.KC; i += PS_THREADS) out[i] = INT_MAX;
        if (tid == 0) {
            p.amin[q] = INFINITY;
            p.state[q] = kSelOverflow;
        }
        return;
    }
    if (tot <= p.KC) {
        // every candidate kept: all allowed vectors when theta = -inf, else
        // every vector below theta is outside
        for (int i = tid; i < p.KC; i += PS_THREADS) out[i] = i < tot ? cv[i] : INT_MAX;
        if (tid == 0) {
            p.amin[q] = theta;
            p.state[q] = theta == -INFINITY ? kSelAll : kSelBound;
        }
        return;
    }
    int n_gt;
    const uint32_t thk = radix_kth<32>([&](auto fn) {
        for (int i = tid; i < tot; i += PS_THREADS) fn(ck[i]);
    }, p.KC, hist, sh, n_gt);
    const int need_eq = p.KC - n_gt;   // keys equal to thk to take (>= 1)
    for (int i = tid; i < tot; i += PS_THREADS) {
        const uint32_t k = ck[i];
        if (k > thk) {
            out[atomicAdd(&sh[4], 1)] = cv[i];
        } else if (k == thk) {
            const int e = atomicAdd(&sh[5], 1);
            if (e < need_eq) out[n_gt + e] = cv[i];
        }
    }
    if (tid == 0) {
        p.amin[q] = ukey_value(thk);
        p.state[q] = kSelBound;
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
    size_t q16, info, approx, bmax, cand_s, cand_i, top_i, amin, state, gbound, tickets, flags, rows, qc,
        allow_c, ids_c, scores_c, lut, total;
    // wide passes
    size_t w_q16, w_info, w_qfrag, w_qf, w_pil, w_theta, w_pcn, w_pci, w_pcs, w_cs, w_ci, w_cn,
        w_top, w_amin, w_state;
};

// Geometry of a wide pass with NG blocks per tile.
struct WideGeom {
    int NG, tilev, pstride, npil, S;
    int64_t ntiles, nmain;
};

WideGeom wide_geom(const ScanShape &s, int NG, int grid, int KC) {
    WideGeom w{};
    w.NG = NG;
    w.tilev = 64 * NG;
    w.ntiles = (s.nblk + NG - 1) / NG;
    // pilot tiles: at most one per workgroup, their scores within kPilotMax per query
    const int64_t cap = std::min<int64_t>(grid, kPilotMax / w.tilev);
    w.pstride = (int)((w.ntiles + cap - 1) / cap);
    w.npil = (int)((w.ntiles + w.pstride - 1) / w.pstride);
    w.nmain = w.ntiles - w.npil;
    // theta is about the (KC ntiles / npil)-th score of the store, so a
    // workgroup appends about KC nmain / (npil grid) vectors per query
    const double per = (double)KC * (double)w.nmain / ((double)w.npil * grid);
    int S = (int)std::ceil(2.0 * per + 16.0);
    S = (S + 7) / 8 * 8;
    w.S = std::min(std::max(S, 16), 512);
    return w;
}

// Query slots of a wide pass of nqt > kWideMinQ queries.
int wide_slots(int nqt) { return nqt <= 128 ? 128 : 256; }


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
    L.tickets = o;
    o += align256((size_t)grid * kTicketStride * 4);
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
    if (nq > kWideMinQ && s.chunks >= kWideMinChunks && grid <= PS_THREADS) {
        const int KC = batch_candidates(k), PCM = 2 * KC;
        const int QP = wide_slots((int)std::min<int64_t>(nq, kWideMaxQ));
        const WideGeom w = wide_geom(s, WD_NG, grid, KC);
        auto take = [&](size_t bytes) {
            const size_t at = o;
            o += align256(bytes);
            return at;
        };
        L.w_q16 = take((size_t)QP * s.d * 2);
        L.w_info = take((size_t)QP * sizeof(QInfo));
        L.w_qfrag = take((size_t)QP * s.d * 2);
        L.w_qf = take((size_t)QP * 4);
        L.w_pil = take((size_t)QP * w.npil * w.tilev * 4);
        L.w_theta = take((size_t)QP * 4);
        L.w_pcn = take((size_t)QP * 4);
        L.w_pci = take((size_t)QP * PCM * 4);
        L.w_pcs = take((size_t)QP * PCM * 4);
        L.w_cs = take((size_t)grid * QP * w.S * 4);
        L.w_ci = take((size_t)grid * QP * w.S * 4);
        L.w_cn = take((size_t)grid * QP * 4);
        L.w_top = take((size_t)QP * KC * 4);
        L.w_amin = take((size_t)QP * 4);
        L.w_state = take((size_t)QP * 4);
    }
    L.total = o + 256;
    return L;
}

// Launches wide_scores_kernel for a pass of QP query slots (QP / 2 queries
// per wave).
hipError_t launch_wide_scores(int QP, const WideParams &wp, int grid, hipStream_t stream) {
    static bool attr[6] = {false, false, false, false, false, false};
    hipError_t err = hipSuccess;
    auto go = [&](int slot, auto kern, size_t lds) {
        if (!attr[slot]) {
            err = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                      (int)lds);
            if (err != hipSuccess) return;
            attr[slot] = true;
        }
        hipLaunchKernelGGL(kern, dim3(grid), dim3(WD_THREADS), lds, stream, wp);
        err = hipGetLastError();
    };
    const int pl = wp.pilot ? 1 : 0;
    switch (QP) {
    case 128:
        if (pl) go(1, wide_scores_kernel<64, true>, WideShape<64>::lds);
        else go(4, wide_scores_kernel<64, false>, WideShape<64>::lds);
        break;
    default:
        if (pl) go(2, wide_scores_kernel<128, true>, WideShape<128>::lds);
        else go(5, wide_scores_kernel<128, false>, WideShape<128>::lds);
        break;
    }
    return err;
}

}  // namespace

// LDS of the score kernel: replicated byte table and query tile.
size_t score_lds_bytes(int d) {
    return (size_t)score_replicas(d) * 256 * 4 + (size_t)kTile * d * 2;
}

bool mfma_search_supported(const ScanShape &s, int k) {
    return s.bits == 4 && s.chunks % 8 == 0 && k <= kMaxBatchK && s.W <= 64 && s.d <= 1792 &&
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
    int *tickets = reinterpret_cast<int *>(w8 + L.tickets);
    int *flags = reinterpret_cast<int *>(w8 + L.flags);
    const int64_t npad = approx_row(s);
    const size_t lds_scores = score_lds_bytes(s.d);
    const int KC = batch_candidates(k);   // candidates per query
    // table, 16 floats, integer sums and sorted (score, id) runs, two counters
    const size_t lds_rescore = (size_t)s.chunks * 2048 + 16 * 4 + (size_t)KC * 12 + 16;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)mfma_scores_kernel<64>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)mfma_scores_kernel<32>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        for (int S = 1; S <= 8 && e == hipSuccess; S *= 2)
            with_slots(64 * S, [&](auto sc) {
                e = hipFuncSetAttribute((const void *)rescore_kernel<decltype(sc)::value>,
                                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            });
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)final_select_kernel,
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)(kFinalMax * 8));
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)pilot_select_kernel,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, kPilotMax * 2);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    auto rescore = [&](int64_t q0, int nqt, const int *ti, const float *am, const int *st,
                       const QInfo *qi) {
        RescoreParams rp{};
        rp.codes = reinterpret_cast<const uint4 *>(blocked);
        rp.scales = scales;
        rp.qrot = Qrot + q0 * s.d;
        rp.cents = cents32;
        rp.top_i = ti;
        rp.amin = am;
        rp.state = st;
        rp.info = qi;
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
    };
    for (int64_t q0 = 0; q0 < nq;) {
        if (nq - q0 > kWideMinQ && s.chunks >= kWideMinChunks && grid <= PS_THREADS) {
            // a wide pass of up to kWideMaxQ queries
            const int nqt = (int)std::min<int64_t>(nq - q0, kWideMaxQ);
            const int QP = wide_slots(nqt);
            const int PCM = 2 * KC;
            const WideGeom w = wide_geom(s, WD_NG, grid, KC);
            _Float16 *wq16 = reinterpret_cast<_Float16 *>(w8 + L.w_q16);
            QInfo *winfo = reinterpret_cast<QInfo *>(w8 + L.w_info);
            uint4 *wqfrag = reinterpret_cast<uint4 *>(w8 + L.w_qfrag);
            float *wqf = reinterpret_cast<float *>(w8 + L.w_qf);
            float *wpil = reinterpret_cast<float *>(w8 + L.w_pil);
            float *wtheta = reinterpret_cast<float *>(w8 + L.w_theta);
            int *wpcn = reinterpret_cast<int *>(w8 + L.w_pcn);
            int *wpci = reinterpret_cast<int *>(w8 + L.w_pci);
            float *wpcs = reinterpret_cast<float *>(w8 + L.w_pcs);
            float *wcs = reinterpret_cast<float *>(w8 + L.w_cs);
            int *wci = reinterpret_cast<int *>(w8 + L.w_ci);
            int *wcn = reinterpret_cast<int *>(w8 + L.w_cn);
            int *wtop = reinterpret_cast<int *>(w8 + L.w_top);
            float *wamin = reinterpret_cast<float *>(w8 + L.w_amin);
            int *wstate = reinterpret_cast<int *>(w8 + L.w_state);
            const uint64_t *allow_p = allow ? allow + q0 * s.W : nullptr;
            hipLaunchKernelGGL(prep_kernel, dim3(nqt), dim3(SEL_THREADS), 0, stream,
                               Qrot + q0 * s.d, nqt, s.d, smax, cmax16, dmax, wq16, winfo,
                               nullptr, 0);
            const int64_t fr = (int64_t)(s.d / 32) * QP * 4;
            hipLaunchKernelGGL(frag_kernel, dim3((int)std::min<int64_t>((fr + 255) / 256, 1024)),
                               dim3(256), 0, stream, wq16, winfo, nqt, QP, s.d, wqfrag, wqf);
            WideParams wp{};
            wp.codes = reinterpret_cast<const uint4 *>(blocked);
            wp.scales = scales;
            wp.qfrag = wqfrag;
            wp.qf = wqf;
            wp.cents = cents32;
            wp.n = s.n;
            wp.nblk = s.nblk;
            wp.ntiles = w.ntiles;
            wp.chunks = s.chunks;
            wp.pstride = w.pstride;
            wp.npil = w.npil;
            wp.pil = wpil;
            wp.theta = wtheta;
            wp.tenants = tenants;
            wp.allow = allow_p;
            wp.W = s.W;
            wp.nqt = nqt;
            wp.cand_s = wcs;
            wp.cand_i = wci;
            wp.cand_n = wcn;
            wp.S = w.S;
            wp.pilot = 1;
            hipError_t e = launch_wide_scores(QP, wp, grid, stream);
            if (e != hipSuccess) return e;
            PilotParams pp{};
            pp.pil = wpil;
            pp.npv = (int64_t)w.npil * w.tilev;
            pp.pstride = w.pstride;
            pp.n = s.n;
            pp.tenants = tenants;
            pp.allow = allow_p;
            pp.W = s.W;
            pp.KC = KC;
            pp.PCM = PCM;
            pp.theta = wtheta;
            pp.pc_n = wpcn;
            pp.pc_i = wpci;
            pp.pc_s = wpcs;
            hipLaunchKernelGGL(pilot_select_kernel, dim3(nqt), dim3(PS_THREADS), (size_t)pp.npv * 2, stream,
                               pp);
            wp.pilot = 0;
            e = launch_wide_scores(QP, wp, grid, stream);
            if (e != hipSuccess) return e;
            FinalParams fp{};
            fp.theta = wtheta;
            fp.pc_n = wpcn;
            fp.pc_i = wpci;
            fp.pc_s = wpcs;
            fp.PCM = PCM;
            fp.cand_s = wcs;
            fp.cand_i = wci;
            fp.cand_n = wcn;
            fp.G = grid;
            fp.QP = QP;
            fp.S = w.S;
            fp.KC = KC;
            fp.top_i = wtop;
            fp.amin = wamin;
            fp.state = wstate;
            hipLaunchKernelGGL(final_select_kernel, dim3(nqt), dim3(PS_THREADS),
                               (size_t)kFinalMax * 8, stream, fp);
            rescore(q0, nqt, wtop, wamin, wstate, winfo);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
            q0 += nqt;
            continue;
        }
        const int nqt = (int)std::min<int64_t>(nq - q0, kTile);
        hipLaunchKernelGGL(prep_kernel, dim3(nqt), dim3(SEL_THREADS), 0, stream, Qrot + q0 * s.d,
                           nqt, s.d, smax, cmax16, dmax, q16, info, tickets, grid * kTicketStride);
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
        sp.tickets = tickets;
        if (score_replicas(s.d) == 64)
            hipLaunchKernelGGL(mfma_scores_kernel<64>, dim3(grid), dim3(MF_THREADS), lds_scores,
                               stream, sp);
        else
            hipLaunchKernelGGL(mfma_scores_kernel<32>, dim3(grid), dim3(MF_THREADS), lds_scores,
                               stream, sp);
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
        rescore(q0, nqt, top_i, amin, state, info);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        q0 += nqt;
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
