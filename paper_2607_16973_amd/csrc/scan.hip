// Single-query scan over the blocked code store (section II-B step 5,
// section III-B) on gfx950.
//
// One persistent workgroup of 16 waves per compute unit.  For every query:
//  * the workgroup builds a lookup table in LDS from the rotated query q'
//    (b in {1,2,4}: every 4-bit field of the code stream -- 4/b coordinates --
//    indexes 16 precomputed partial sums sum_t c[code_t] q'_j; b = 3: 8
//    entries c[code] q'_j per coordinate; b = 8: the 256 centroids and q'
//    itself, multiplied on the fly);
//  * each wave walks its share of 64-vector blocks: first the block's tenant
//    summary is ANDed with the allowlist and the block is skipped if nothing
//    can match -- before any code byte is read; otherwise every lane streams
//    its own vector's codes in 16-byte loads (a wave reads 1 KiB contiguous
//    per load), sums table hits in float32 and multiplies by the vector's
//    scale; vectors whose tenant is not allowed are dropped at insertion;
//  * a wave keeps its best 64*S entries in registers (bitonic sort of the 64
//    new scores, then a bitonic merge), skipping the sort when no lane beats
//    the current k-th best; the 16 wave lists are merged in LDS and the
//    workgroup's top-k goes to the workspace; a second kernel merges the
//    per-workgroup lists of each query.
#include <hip/hip_runtime.h>

#include <atomic>
#include <climits>
#include <cmath>
#include <cstdint>

#include "kernels.h"
#include "lut.h"
#include "stream.h"
#include "topk.h"

namespace tq {
namespace {

constexpr int SCAN_THREADS = kTableThreads;
constexpr int SCAN_WAVES = SCAN_THREADS / 64;
// Scheduling-barrier mask: ALU, SALU, MFMA, LDS and transcendental
// instructions may move across, memory loads and stores to HBM may not.
constexpr int kKeepVmem = 0x1 | 0x2 | 0x4 | 0x8 | 0x80 | 0x100 | 0x200 | 0x400;

enum Mode { NIBBLE = 0, TRIBIT = 1, BYTE = 2 };

struct ScanParams {
    const uint4 *codes;
    const float *scales;
    const uint16_t *tenants;
    const uint64_t *summaries;
    const uint64_t *allow;      // [nq][W] tenant allowlists, or null: every tenant
    const uint64_t *live;       // [nblk] live-slot masks (bit v: slot 64b+v not deleted), or null
    const uint64_t *slot_allow; // [nq][nblk] allowed-slot masks (instead of allow), or null
    const float *qrot;          // [nq][d] (with TQ+ calibration: kappa_j q'_j)
    const float *qconst;        // [nq] TQ+ constant term sum_j mu_j q'_j, or null
    const float *cents;         // [levels]
    float *cand_s;              // [nq][G][k]
    int *cand_i;
    int *gbound;                // [nq] order keys of a k-th-best lower bound, all workgroups
    int64_t n, nblk;
    int d, bits, chunks, W, k, nq;
    int lut_words;              // 32-bit words of LDS used by the table
};

// Slots of block b that query qi may return: the live ones (all if no slot
// was deleted), restricted to the query's allowed slots when slot-level
// allowlists are given.  Tenant allowlists are tested separately.
__device__ inline uint64_t block_mask(const ScanParams &p, int qi, int64_t b) {
    uint64_t m = p.live ? p.live[b] : ~0ull;
    if (p.slot_allow) m &= p.slot_allow[(int64_t)qi * p.nblk + b];
    return m;
}

// Constant term of query qi's scores (TQ+ calibration), 0 without.
__device__ inline float qconst_of(const ScanParams &p, int qi) {
    return p.qconst ? p.qconst[qi] : 0.f;
}

__device__ inline TableShape table_shape(const ScanParams &p) {
    return TableShape{p.d, p.bits, p.lut_words};
}

// ---------------------------------------------------------------- tables
// b in {1,2,4}: int32 fixed-point rows of 16 entries per 4-bit field (lut.h).
// b = 3: int32 fixed-point rows of 8 entries per coordinate (lut.h).
// b = 8: the 256 float32 centroids, each repeated 32 times, followed by q'
// (multiplied on the fly).  Centroid e of lane l is at byte 128 e + 4 (l % 32):
// the 32 lanes of a half-wave always read 32 different banks, whatever
// their codes.

constexpr int kByteRepWords = 256 * 32;

// Sum over the four codes of word w of c[code] q'_j; rep is the repeated
// centroids, lo = 4 (lane % 32).  Each address is a bit-field extract and a
// shift-add (the empty asm keeps the compiler from re-forming them).
__device__ inline float byte4(const char *__restrict__ rep, const float *__restrict__ q,
                              uint32_t w, uint32_t lo) {
    uint32_t e0 = __builtin_amdgcn_ubfe(w, 0, 8), e1 = __builtin_amdgcn_ubfe(w, 8, 8);
    uint32_t e2 = __builtin_amdgcn_ubfe(w, 16, 8), e3 = w >> 24;
    asm volatile("" : "+v"(e0), "+v"(e1), "+v"(e2), "+v"(e3));
    const float c0 = *reinterpret_cast<const float *>(rep + (e0 << 7) + lo);
    const float c1 = *reinterpret_cast<const float *>(rep + (e1 << 7) + lo);
    const float c2 = *reinterpret_cast<const float *>(rep + (e2 << 7) + lo);
    const float c3 = *reinterpret_cast<const float *>(rep + (e3 << 7) + lo);
    float a = c0 * q[0];
    float b = c1 * q[1];
    a = fmaf(c2, q[2], a);
    b = fmaf(c3, q[3], b);
    return a + b;
}

// The integer-table modes: the query coordinates a thread loads ahead of
// the build, and the bytes of table per 16-byte chunk of codes.
template <int MODE> struct QueryRegs { float v[2][4]; };
template <> struct QueryRegs<TRIBIT> { float v[kTriRowsPerThread]; };
template <int MODE> constexpr int kChunkTableBytes = MODE == TRIBIT ? 1280 : 2048;

template <int MODE>
__device__ inline void load_query(const TableShape &t, const float *__restrict__ q,
                                  QueryRegs<MODE> &r) {
    if constexpr (MODE == TRIBIT)
        load_tribit_query(t, q, r.v);
    else
        load_nibble_query(t, q, r.v);
}

template <int MODE>
__device__ inline void query_abs_sum(float *red, const QueryRegs<MODE> &r) {
    if constexpr (MODE == TRIBIT)
        tribit_abs_sum(red, r.v);
    else
        nibble_abs_sum(red, r.v);
}

template <int MODE>
__device__ inline int build_int_table(float *lds, const float *red, const float *cents,
                                      const TableShape &t, const QueryRegs<MODE> &r, float C) {
    if constexpr (MODE == TRIBIT)
        return build_tribit_table(lds, red, cents, t, r.v, C);
    else
        return build_nibble_table(lds, red, cents, t, r.v, C);
}

template <int MODE>
__device__ inline int int_chunk(const char *__restrict__ Lb, uint4 v) {
    if constexpr (MODE == TRIBIT)
        return tri_chunk(Lb, v);
    else
        return nib_chunk(Lb, v);
}

template <int MODE> struct AccOf { typedef int type; };
template <> struct AccOf<BYTE> { typedef float type; };

template <int MODE>
__device__ inline typename AccOf<MODE>::type chunk_sum(const float *__restrict__ lds, int c, uint4 v) {
    if constexpr (MODE == BYTE) {
        const char *rep = reinterpret_cast<const char *>(lds);
        const float *q = lds + kByteRepWords + c * 16;
        const uint32_t lo = (threadIdx.x & 31u) << 2;
        return (byte4(rep, q, v.x, lo) + byte4(rep, q + 4, v.y, lo)) +
               (byte4(rep, q + 8, v.z, lo) + byte4(rep, q + 12, v.w, lo));
    } else {
        return int_chunk<MODE>(reinterpret_cast<const char *>(lds) + c * kChunkTableBytes<MODE>, v);
    }
}

// Builds the table for one query; returns the fixed-point exponent sh of
// the integer tables, or 0.  `red` is 16 floats of LDS scratch.  C is the
// query's constant term: part of the integer tables, the starting value of
// the float sums of b = 8.
template <int MODE>
__device__ int build_table(float *lds, float *red, const ScanParams &p, const float *__restrict__ q,
                           float C) {
    const int tid = threadIdx.x;
    if constexpr (MODE == BYTE) {
        for (int e = tid; e < kByteRepWords; e += SCAN_THREADS) lds[e] = p.cents[e >> 5];
        for (int e = tid; e < p.d; e += SCAN_THREADS) lds[kByteRepWords + e] = q[e];
        return 0;
    } else {
        QueryRegs<MODE> qv;
        load_query<MODE>(table_shape(p), q, qv);
        query_abs_sum<MODE>(red, qv);
        __syncthreads();
        return build_int_table<MODE>(lds, red, p.cents, table_shape(p), qv, C);
    }
}

__global__ void fill_keys(int *p, int64_t n, int v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// LDS words from the start of dynamic LDS that the table and, after the
// scan, the merge stage (16 lists of 64*S scores and ids) may occupy; the
// regions that must survive the merge start here.
__host__ __device__ inline int aux_words(int lut_words, int S) {
    const int stage = SCAN_WAVES * 64 * S * 2;
    return lut_words > stage ? lut_words : stage;
}

// Workgroup top-k from the 16 wave lists, in three steps.
//  1. collect_survivors: entries below a proven bound -- the best k-th score
//     of any wave (LDS key) or of any workgroup (as last seen by the wave) --
//     cannot reach the top k; each wave appends its other entries to a list
//     of up to 64 in LDS, counted in *cnt (which starts at zero).
//  2. If at most 64 survive, write_survivors (one wave) sorts them and
//     writes the workgroup's k best.
//  3. Otherwise tree_merge merges the full lists pairwise through LDS.
template <int S>
__device__ inline void collect_survivors(const WaveTopK<S> &top, int wg_key, float *surv_s,
                                         int *surv_i, int *cnt, int lane) {
    const int bk = wg_key > top.seen_g ? wg_key : top.seen_g;
    const float bound = unfkey(bk);
#pragma unroll
    for (int a = 0; a < S; ++a) {
        const bool keep = top.li[a] != INT_MAX && !(top.ls[a] < bound);
        const uint64_t m = __ballot(keep);
        if (m) {
            int base = 0;
            if (lane == 0) base = atomicAdd(cnt, __popcll(m));
            base = __builtin_amdgcn_readfirstlane(base);
            const int pos = base + __popcll(m & ((1ull << lane) - 1));
            if (keep && pos < 64) {
                surv_s[pos] = top.ls[a];
                surv_i[pos] = top.li[a];
            }
        }
    }
}

template <int S>
__device__ inline void write_survivors(const float *surv_s, const int *surv_i, int total,
                                       const ScanParams &p, int64_t out, int lane) {
    float sv = lane < total ? surv_s[lane] : -INFINITY;
    int iv = lane < total ? surv_i[lane] : INT_MAX;
    wave_sort64(sv, iv, lane);
#pragma unroll
    for (int a = 0; a < S; ++a) {
        const int r = a * 64 + lane;
        if (r < p.k) {
            p.cand_s[out + r] = a == 0 ? sv : -INFINITY;
            p.cand_i[out + r] = a == 0 ? iv : INT_MAX;
        }
    }
}

// Pairwise merge of the 16 wave lists through LDS (stage_* hold 16 x 64*S
// entries); wave 0 writes the result.  Starts and ends with a barrier.
template <int S>
__device__ inline void tree_merge(WaveTopK<S> &top, float *stage_s, int *stage_i, int wave,
                                  int lane, const ScanParams &p, int64_t out) {
    __syncthreads();
#pragma unroll
    for (int a = 0; a < S; ++a) {
        stage_s[wave * 64 * S + a * 64 + lane] = top.ls[a];
        stage_i[wave * 64 * S + a * 64 + lane] = top.li[a];
    }
    __syncthreads();
    for (int step = 1; step < SCAN_WAVES; step <<= 1) {
        if ((wave & (2 * step - 1)) == 0) {
            float os[S];
            int oi[S];
            const int w = wave + step;
#pragma unroll
            for (int a = 0; a < S; ++a) {
                os[a] = stage_s[w * 64 * S + a * 64 + lane];
                oi[a] = stage_i[w * 64 * S + a * 64 + lane];
            }
            merge_lists<S>(top.ls, top.li, os, oi, lane);
#pragma unroll
            for (int a = 0; a < S; ++a) {
                stage_s[wave * 64 * S + a * 64 + lane] = top.ls[a];
                stage_i[wave * 64 * S + a * 64 + lane] = top.li[a];
            }
        }
        __syncthreads();
    }
    if (wave == 0) {
#pragma unroll
        for (int a = 0; a < S; ++a) {
            const int r = a * 64 + lane;
            if (r < p.k) {
                p.cand_s[out + r] = top.ls[a];
                p.cand_i[out + r] = top.li[a];
            }
        }
    }
    __syncthreads();
}

// The three steps with their barriers, for the block-per-wave scan: the
// table's LDS holds the survivors and the stage (misc[0]: bound key,
// misc[2]: survivor count, zero on entry and on return).
template <int S>
__device__ inline void workgroup_merge(WaveTopK<S> &top, float *stage_s, int *stage_i, int *misc,
                                       int wave, int lane, const ScanParams &p, int qi) {
    __syncthreads();   // every offer is done; the table's LDS is free
    const int64_t out = ((int64_t)qi * gridDim.x + blockIdx.x) * p.k;
    collect_survivors<S>(top, misc[0], stage_s, stage_i, misc + 2, lane);
    __syncthreads();
    const int total = misc[2];
    if (total <= 64) {
        if (wave == 0) write_survivors<S>(stage_s, stage_i, total, p, out, lane);
    } else {
        tree_merge<S>(top, stage_s, stage_i, wave, lane, p, out);
    }
    __syncthreads();   // LDS is rebuilt for the next query
    if (threadIdx.x == 0) misc[2] = 0;
}

// ALL: no top-k; every vector's score (-inf when the filter drops it) goes to
// cand_s[qi * n + vid] (vectors of skipped blocks keep what the buffer
// held: the caller fills it with -inf first).
template <int MODE, int S, int PF, bool ALL = false>
__global__ __launch_bounds__(SCAN_THREADS) void scan_kernel(ScanParams p) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    // [0, aux): the table, later the merge stage; then the fixed regions
    uint64_t *allow_s = reinterpret_cast<uint64_t *>(lds + aux_words(p.lut_words, S));
    int *misc = reinterpret_cast<int *>(allow_s + p.W);     // [0] bound key, [2] merge count
    float *red = reinterpret_cast<float *>(misc + 4);        // 16 floats
    float *stage_s = lds;                                     // reused after the scan
    int *stage_i = reinterpret_cast<int *>(lds + SCAN_WAVES * 64 * S);
    typedef typename AccOf<MODE>::type acc_t;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // wave-uniform: lets the compiler keep block and chunk indices in SGPRs
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = gridDim.x;
    const int g = blockIdx.x;
    const bool filtered = p.allow || p.live || p.slot_allow;
    const int CH = p.chunks;

    // contiguous block range of this wave
    const int64_t gb0 = p.nblk * g / G, gb1 = p.nblk * (g + 1) / G;
    const int64_t b0 = gb0 + (gb1 - gb0) * wave / SCAN_WAVES;
    const int64_t b1 = gb0 + (gb1 - gb0) * (wave + 1) / SCAN_WAVES;

    if (tid == 0) misc[2] = 0;
    for (int qi = 0; qi < p.nq; ++qi) {
        const float cq = qconst_of(p, qi);
        const int sh = build_table<MODE>(lds, red, p, p.qrot + (int64_t)qi * p.d, cq);
        if (p.allow)
            for (int w = tid; w < p.W; w += SCAN_THREADS) allow_s[w] = p.allow[(int64_t)qi * p.W + w];
        if (tid == 0) misc[0] = fkey(-INFINITY);
        __syncthreads();

        WaveTopK<S> top;
        top.reset();
        int64_t blk = b0;
        while (blk < b1) {
            // next run of consecutive blocks to scan
            int64_t r0 = blk, r1 = b1;
            if (filtered) {
                // a block is scanned when its tenant summary meets the
                // allowlist and it holds a live, allowed slot
                auto listed = [&](int64_t r) {
                    bool hit = true;
                    if (p.allow) {
                        bool h = false;
                        for (int w = lane; w < p.W; w += 64)
                            h |= (p.summaries[r * p.W + w] & allow_s[w]) != 0;
                        hit = __any(h);
                    }
                    if (hit && (p.live || p.slot_allow)) hit = block_mask(p, qi, r) != 0;
                    return hit;
                };
                // skip blocks that are not listed, then extend the run over
                // blocks that are
                for (; r0 < b1; ++r0)
                    if (listed(r0)) break;
                for (r1 = r0 + 1; r1 < b1; ++r1)
                    if (!listed(r1)) break;
                if (r0 >= b1) break;
            }
            // stream the run as one sequence of F 16-byte chunks per lane
            // wave-uniform base of the run; each lane adds its fixed 16-byte slot
            const uint4 *src = p.codes + r0 * CH * 64;
            const int64_t F = (r1 - r0) * CH;
            // Prefetch ring: the refill of buf[i] is issued as soon as chunk i
            // has been consumed.  Scheduling barriers keep every load where it
            // is written (in ring order), so each chunk waits only for its own
            // load with PF-1 younger loads still in flight.
            uint4 buf[PF];
#pragma unroll
            for (int i = 0; i < PF; ++i) {
                buf[i] = load_stream(src + (int64_t)(i < F ? i : F - 1) * 64 + lane);
                __builtin_amdgcn_sched_barrier(kKeepVmem);
            }
            int64_t f = 0;
            for (int64_t b = r0; b < r1; ++b) {
                // per-vector loads first: in-order completion means waiting
                // for them later does not drain the chunk prefetches
                const uint4 *bsrc = src + f * 64;    // this block's first chunk
                const int64_t vid = b * 64 + lane;
                const bool inside = vid < p.n;
                const float scl = p.scales[vid];
                const int ten = p.allow ? (int)p.tenants[vid] : 0;
                const uint64_t bm = filtered ? block_mask(p, qi, b) : ~0ull;
                acc_t acc = 0;
                if constexpr (MODE == BYTE) acc = cq;
                for (int c0 = 0; c0 < CH; c0 += PF) {
#pragma unroll
                    for (int i = 0; i < PF; ++i) {
                        // consume buf[i] before it is refilled, so the refill
                        // reuses its registers and only waits for this chunk
                        acc += chunk_sum<MODE>(lds, c0 + i, buf[i]);
                        // past the end of the run the refill reads the first
                        // chunk of this block again: a cache hit, no HBM traffic
                        const int64_t nf = f + c0 + i + PF;
                        const uint4 *nsrc = nf < F ? src + nf * 64 : bsrc;
                        buf[i] = load_stream(nsrc + lane);
                        __builtin_amdgcn_sched_barrier(kKeepVmem);
                    }
                }
                f += CH;
                bool ok = inside && ((bm >> lane) & 1ull);
                if (ok && p.allow) ok = (allow_s[ten >> 6] >> (ten & 63)) & 1ull;
                float sc;
                if constexpr (MODE == BYTE)
                    sc = acc * scl;
                else
                    sc = ldexpf((float)acc * scl, -sh);
                if constexpr (ALL) {
                    if (inside) p.cand_s[(int64_t)qi * p.n + vid] = ok ? sc : -INFINITY;
                } else {
                    top.offer(ok ? sc : -INFINITY, ok ? (int)vid : INT_MAX, lane, p.k, misc,
                              p.gbound + qi);
                }
            }
            blk = r1;
        }
        if constexpr (ALL)
            __syncthreads();   // every lookup done before the next table is built
        else
            workgroup_merge<S>(top, stage_s, stage_i, misc, wave, lane, p, qi);
    }
}

// Blocks per accumulation pass of the split scan: 64 blocks x 64 int32 sums
// = 16 KiB of LDS.
constexpr int kPassBlocks = 64;

// Unfiltered scan for b in {1, 2, 3, 4} with the work of a workgroup handed
// out in groups of 8 chunks (8 KiB of one block's codes) rather than whole
// blocks.
//  * Every query covers the same blocks of the workgroup, taken in passes of
//    up to 64 blocks.  The (query, pass, group) work items are numbered in
//    that order and each wave claims its next item from an LDS counter one
//    item ahead of the one it is scoring, so the ring of 8 loads always
//    holds the next group -- also across pass and query boundaries: while
//    the workgroup merges one query's lists and builds the next table, the
//    codes of the next query's first groups are already on their way.
//  * The waves, which the hardware does not run at equal speed, finish a
//    pass within one group of each other.
//  * A wave adds its integer sum for a group into the block's LDS slot with
//    an atomic add (integer: exact and order-free, so the result does not
//    depend on who scored what), then counts the group done; the wave that
//    completes a block turns its sums into scores and offers them to its
//    top-k while the other waves stream on.
//  * Per query there are three barriers: end of the scan, survivors
//    collected, next table built (the survivors' sort overlaps the build).
template <int MODE, int S>
__global__ __launch_bounds__(SCAN_THREADS) void split_scan_kernel(ScanParams p) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    // [0, aux): the table (and the tree-merge stage); then the fixed regions
    const int aux = aux_words(p.lut_words, S);
    int *accb = reinterpret_cast<int *>(lds + aux);   // [kPassBlocks][64] block sums
    int *done = accb + kPassBlocks * 64;              // [kPassBlocks] finished groups
    int *misc = done + kPassBlocks;                   // [0] bound key, [1] tickets, [2] survivors
    float *red = reinterpret_cast<float *>(misc + 4); // 16 wave sums of |q'|
    float *cents_s = red + 16;                        // 16 levels
    float *surv_s = cents_s + 16;                     // 64 survivors
    int *surv_i = reinterpret_cast<int *>(surv_s + 64);
    float *stage_s = lds;
    int *stage_i = reinterpret_cast<int *>(lds + SCAN_WAVES * 64 * S);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = gridDim.x;
    const int g = blockIdx.x;
    const int CH = p.chunks;          // multiple of 8
    const int GPB = CH >> 3;          // 8-chunk groups per block
    const int64_t gb0 = p.nblk * g / G, gb1 = p.nblk * (g + 1) / G;
    const int nbq = (int)(gb1 - gb0);                       // blocks per query
    const int NGq = nbq * GPB;                              // groups per query
    const int npass = (nbq + kPassBlocks - 1) / kPassBlocks;
    const int PG = kPassBlocks * GPB;                       // groups per full pass
    const int total = p.nq * NGq;                           // work items (host-bounded)
    const uint4 *wg_src = p.codes + gb0 * CH * 64;
    const char *lut = reinterpret_cast<const char *>(lds);
    // lane 0 takes a ticket; the wave reads it from lane 0 when it needs it
    auto take = [&](int *ctr) {
        int v = 0;
        if (lane == 0) v = atomicAdd(ctr, 1);
        return v;
    };
    // pass number, counted over all queries, of a work item
    auto stage_of = [&](int t) {
        const int q = t / NGq;
        return q * npass + (t - q * NGq) / PG;
    };

    for (int e = tid; e < kPassBlocks * 65; e += SCAN_THREADS) accb[e] = 0;   // sums and counts
    if (tid < 16) cents_s[tid] = p.cents[tid];
    if (tid == 0) {
        misc[0] = fkey(-INFINITY);
        misc[1] = 0;
        misc[2] = 0;
    }
    if (p.nq == 0) return;
    QueryRegs<MODE> qv;
    load_query<MODE>(table_shape(p), p.qrot, qv);
    const float qc0 = qconst_of(p, 0);
    query_abs_sum<MODE>(red, qv);
    __syncthreads();

    // this wave's current and next work items, and the ring holding the
    // current one's 8 chunks: claimed and requested before the first table
    // is built, so that the build overlaps the first loads
    int tk = __builtin_amdgcn_readfirstlane(take(misc + 1));
    int nxt = __builtin_amdgcn_readfirstlane(take(misc + 1));
    // wave-uniform base of a group; each lane adds its 16-byte slot
    const uint4 *csrc = wg_src + (int64_t)(tk < total ? tk % NGq : 0) * 8 * 64;
    uint4 buf[8];
    if (tk < total) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            buf[i] = load_stream(csrc + i * 64 + lane);
            __builtin_amdgcn_sched_barrier(kKeepVmem);
        }
    }
    int sh = build_int_table<MODE>(lds, red, cents_s, table_shape(p), qv, qc0);
    __syncthreads();
    for (int qi = 0; qi < p.nq; ++qi) {
        WaveTopK<S> top;
        top.reset();
        for (int ps = 0; ps < npass; ++ps) {
            if (ps > 0) __syncthreads();   // the previous pass's slots are free again
            const int sid = qi * npass + ps;
            const int64_t p0 = gb0 + (int64_t)ps * kPassBlocks;
            while (tk < total && stage_of(tk) == sid) {
                const int gp = tk - qi * NGq - ps * PG;   // group within the pass
                const int bl = gp / GPB;
                const int c0 = (gp - bl * GPB) * 8;
                const int64_t vid = (p0 + bl) * 64 + lane;
                const bool inside = vid < p.n;
                // The group that completes a block needs the vectors'
                // scales and the global bound.  Groups are claimed in order,
                // so that is almost always the block's last group: it loads
                // them ahead of its lookups; any other group that turns out
                // to complete the block loads them when it does.
                const bool last = c0 == CH - 8;
                float scl = 0.f;
                int gk = 0;
                if (last) {
                    scl = p.scales[inside ? vid : 0];
                    gk = __hip_atomic_load(p.gbound + qi, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                }
                // past the last item the refills read this group again:
                // cache hits, no HBM traffic
                const uint4 *nsrc = nxt < total ? wg_src + (int64_t)(nxt % NGq) * 8 * 64 : csrc;
                const char *Lb = lut + c0 * kChunkTableBytes<MODE>;
                int acc = 0;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    // consume buf[i], then refill it with the next group
                    acc += int_chunk<MODE>(Lb + i * kChunkTableBytes<MODE>, buf[i]);
                    buf[i] = load_stream(nsrc + i * 64 + lane);
                    __builtin_amdgcn_sched_barrier(kKeepVmem);
                }
                __builtin_amdgcn_sched_barrier(0);
                atomicAdd(&accb[bl * 64 + lane], acc);
                // LDS executes each wave's operations in order, so when the
                // count reaches GPB every group's sum is in the slot
                const int fin = __builtin_amdgcn_readfirstlane(take(done + bl));
                if (fin == GPB - 1) {
                    if (!last) {
                        scl = p.scales[inside ? vid : 0];
                        gk = __hip_atomic_load(p.gbound + qi, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                    }
                    const int sum = accb[bl * 64 + lane];
                    accb[bl * 64 + lane] = 0;
                    if (lane == 0) done[bl] = 0;
                    const float sc = ldexpf((float)sum * scl, -sh);
                    top.offer_seen(inside ? sc : -INFINITY, inside ? (int)vid : INT_MAX, lane, p.k,
                                   misc, p.gbound + qi, gk);
                }
                // the ticket after next, taken as late as possible: near the
                // end of a query a wave holds no more than two groups
                const int nxt2 = __builtin_amdgcn_readfirstlane(take(misc + 1));
                tk = nxt;
                nxt = nxt2;
                csrc = nsrc;
            }
        }
        // a wave that is done loads the next query's coordinates and |q'|
        // sum while the others finish (red was last read by this table's build)
        const bool more = qi + 1 < p.nq;
        if (more) {
            load_query<MODE>(table_shape(p), p.qrot + (int64_t)(qi + 1) * p.d, qv);
            query_abs_sum<MODE>(red, qv);
        }
        __syncthreads();   // scan done: every offer made, the bound key final
        const int64_t out = ((int64_t)qi * G + g) * p.k;
        collect_survivors<S>(top, misc[0], surv_s, surv_i, misc + 2, lane);
        __syncthreads();
        const int ns = misc[2];
        if (ns <= 64) {
            if (wave == 0) write_survivors<S>(surv_s, surv_i, ns, p, out, lane);
        } else {
            tree_merge<S>(top, stage_s, stage_i, wave, lane, p, out);   // rare: LDS of the table
        }
        if (more) sh = build_int_table<MODE>(lds, red, cents_s, table_shape(p), qv, qconst_of(p, qi + 1));
        if (tid == 0) misc[0] = fkey(-INFINITY);   // every wave has read it (previous barrier)
        __syncthreads();   // table ready; survivor count read by every wave
        if (tid == 0) misc[2] = 0;
    }
}

// Filtered scan for b in {1, 2, 3, 4}: as split_scan_kernel, over the blocks
// whose tenant summary meets the query's allowlist only.  At the start of a
// query the workgroup lists those of its blocks (by summary & allowlist, in
// windows of kListMax blocks; no code byte of a skipped block is read), then
// waves claim 8-chunk groups of the listed blocks in passes of up to 64
// blocks; the wave that completes a block drops vectors whose tenant is not
// allowed and offers the rest to its top-k.  (The listing order is not
// fixed; the result does not depend on it.)
constexpr int kListMax = 4096;

template <int MODE, int S>
__global__ __launch_bounds__(SCAN_THREADS) void split_filtered_kernel(ScanParams p) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    const int aux = aux_words(p.lut_words, S);
    int *accb = reinterpret_cast<int *>(lds + aux);   // [kPassBlocks][64] block sums
    int *done = accb + kPassBlocks * 64;              // [kPassBlocks] finished groups
    // [0] bound key, [1] and [3] group counters (alternate passes), [2] survivors
    int *misc = done + kPassBlocks;
    float *red = reinterpret_cast<float *>(misc + 4); // 16 wave sums of |q'|
    float *cents_s = red + 16;                        // 16 levels
    float *surv_s = cents_s + 16;                     // 64 survivors
    int *surv_i = reinterpret_cast<int *>(surv_s + 64);
    int *nlist = surv_i + 64;                         // listed blocks of the window
    int *list = nlist + 4;                            // [kListMax] block offsets in the window
    uint64_t *allow_s = reinterpret_cast<uint64_t *>(list + kListMax);   // [W]
    float *stage_s = lds;
    int *stage_i = reinterpret_cast<int *>(lds + SCAN_WAVES * 64 * S);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = gridDim.x;
    const int g = blockIdx.x;
    const int CH = p.chunks;          // multiple of 8
    const int GPB = CH >> 3;          // 8-chunk groups per block
    const int W = p.W;
    const int64_t gb0 = p.nblk * g / G, gb1 = p.nblk * (g + 1) / G;
    const char *lut = reinterpret_cast<const char *>(lds);
    auto take = [&](int *ctr) {
        int v = 0;
        if (lane == 0) v = atomicAdd(ctr, 1);
        return v;
    };

    for (int e = tid; e < kPassBlocks * 65; e += SCAN_THREADS) accb[e] = 0;   // sums and counts
    if (tid < 16) cents_s[tid] = p.cents[tid];
    if (tid == 0) {
        misc[0] = fkey(-INFINITY);
        misc[1] = 0;
        misc[2] = 0;
        misc[3] = 0;
    }
    if (p.nq == 0) return;
    if (p.allow)
        for (int w = tid; w < W; w += SCAN_THREADS) allow_s[w] = p.allow[w];
    QueryRegs<MODE> qv;
    load_query<MODE>(table_shape(p), p.qrot, qv);
    query_abs_sum<MODE>(red, qv);
    __syncthreads();
    int sh = build_int_table<MODE>(lds, red, cents_s, table_shape(p), qv, qconst_of(p, 0));
    __syncthreads();
    for (int qi = 0; qi < p.nq; ++qi) {
        WaveTopK<S> top;
        top.reset();
        int pass = 0;
        for (int64_t w0 = gb0; w0 < gb1; w0 += kListMax) {
            const int wn = (int)(gb1 - w0 < kListMax ? gb1 - w0 : kListMax);
            if (w0 > gb0) __syncthreads();   // the previous window's list is no longer read
            if (tid == 0) *nlist = 0;
            __syncthreads();
            for (int t = tid; t < wn; t += SCAN_THREADS) {
                const int64_t b = w0 + t;
                bool hit;
                if (p.slot_allow) {
                    hit = (block_mask(p, qi, b) != 0);
                } else {
                    hit = !p.live || p.live[b] != 0;
                    if (p.allow) {
                        const uint64_t *sm = p.summaries + b * W;
                        bool any = false;
                        for (int w = 0; w < W; ++w) any |= (sm[w] & allow_s[w]) != 0;
                        hit = hit && any;
                    }
                }
                if (hit) list[atomicAdd(nlist, 1)] = t;
            }
            __syncthreads();
            const int nl = *nlist;
            for (int l0 = 0; l0 < nl; l0 += kPassBlocks, ++pass) {
                if (l0 > 0) __syncthreads();   // the previous pass's slots are free again
                int *ctr = misc + 1 + 2 * (pass & 1);
                if (tid == 0) misc[1 + 2 * ((pass + 1) & 1)] = 0;   // the next pass's counter
                const int nb = nl - l0 < kPassBlocks ? nl - l0 : kPassBlocks;
                const int ng = nb * GPB;
                // address of group u of this pass (wave-uniform)
                auto group_src = [&](int u) {
                    const int bl = u / GPB;
                    const int64_t blk = w0 + list[l0 + bl];
                    return p.codes + (blk * CH + (int64_t)(u - bl * GPB) * 8) * 64;
                };
                int cur = __builtin_amdgcn_readfirstlane(take(ctr));
                if (cur < ng) {
                    int nxt = __builtin_amdgcn_readfirstlane(take(ctr));
                    const uint4 *csrc = group_src(cur);
                    uint4 buf[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        buf[i] = load_stream(csrc + i * 64 + lane);
                        __builtin_amdgcn_sched_barrier(kKeepVmem);
                    }
                    while (true) {
                        const int bl = cur / GPB;
                        const int c0 = (cur - bl * GPB) * 8;
                        const int64_t blk = w0 + list[l0 + bl];
                        const int64_t vid = blk * 64 + lane;
                        const bool inside = vid < p.n;
                        const bool last = c0 == CH - 8;
                        float scl = 0.f;
                        int ten = 0, gk = 0;
                        uint64_t bm = 0;
                        if (last) {
                            scl = p.scales[inside ? vid : 0];
                            ten = p.tenants[inside ? vid : 0];
                            bm = block_mask(p, qi, blk);
                            gk = __hip_atomic_load(p.gbound + qi, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT);
                        }
                        const uint4 *nsrc = nxt < ng ? group_src(nxt) : csrc;
                        const char *Lb = lut + c0 * kChunkTableBytes<MODE>;
                        int acc = 0;
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            acc += int_chunk<MODE>(Lb + i * kChunkTableBytes<MODE>, buf[i]);
                            buf[i] = load_stream(nsrc + i * 64 + lane);
                            __builtin_amdgcn_sched_barrier(kKeepVmem);
                        }
                        __builtin_amdgcn_sched_barrier(0);
                        atomicAdd(&accb[bl * 64 + lane], acc);
                        const int fin = __builtin_amdgcn_readfirstlane(take(done + bl));
                        if (fin == GPB - 1) {
                            if (!last) {
                                scl = p.scales[inside ? vid : 0];
                                ten = p.tenants[inside ? vid : 0];
                                bm = block_mask(p, qi, blk);
                                gk = __hip_atomic_load(p.gbound + qi, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                            }
                            const int sum = accb[bl * 64 + lane];
                            accb[bl * 64 + lane] = 0;
                            if (lane == 0) done[bl] = 0;
                            const bool ok = inside && ((bm >> lane) & 1ull) &&
                                            (!p.allow || ((allow_s[ten >> 6] >> (ten & 63)) & 1ull));
                            const float sc = ldexpf((float)sum * scl, -sh);
                            top.offer_seen(ok ? sc : -INFINITY, ok ? (int)vid : INT_MAX, lane, p.k,
                                           misc, p.gbound + qi, gk);
                        }
                        if (nxt >= ng) break;
                        const int nxt2 = __builtin_amdgcn_readfirstlane(take(ctr));
                        cur = nxt;
                        nxt = nxt2;
                        csrc = nsrc;
                    }
                }
            }
        }
        const bool more = qi + 1 < p.nq;
        if (more) {
            load_query<MODE>(table_shape(p), p.qrot + (int64_t)(qi + 1) * p.d, qv);
            query_abs_sum<MODE>(red, qv);
        }
        __syncthreads();   // scan done: every offer made, the bound key final
        const int64_t out = ((int64_t)qi * G + g) * p.k;
        collect_survivors<S>(top, misc[0], surv_s, surv_i, misc + 2, lane);
        __syncthreads();
        const int ns = misc[2];
        if (ns <= 64) {
            if (wave == 0) write_survivors<S>(surv_s, surv_i, ns, p, out, lane);
        } else {
            tree_merge<S>(top, stage_s, stage_i, wave, lane, p, out);   // rare: LDS of the table
        }
        if (more) {
            sh = build_int_table<MODE>(lds, red, cents_s, table_shape(p), qv, qconst_of(p, qi + 1));
            if (p.allow)
                for (int w = tid; w < W; w += SCAN_THREADS)
                    allow_s[w] = p.allow[(int64_t)(qi + 1) * W + w];
        }
        if (tid == 0) {
            misc[0] = fkey(-INFINITY);
            misc[1] = 0;
            misc[3] = 0;
        }
        __syncthreads();   // table and allowlist ready; survivor count read by every wave
        if (tid == 0) misc[2] = 0;
    }
}

template <int S>
__global__ __launch_bounds__(256) void merge_kernel(const float *__restrict__ cs,
                                                    const int *__restrict__ ci, int G, int k,
                                                    const int *__restrict__ gbound,
                                                    int64_t *__restrict__ ids,
                                                    float *__restrict__ scores) {
    __shared__ float st_s[4 * 64 * S];
    __shared__ int st_i[4 * 64 * S];
    // survivors of the bound (k <= 64)
    constexpr int MCAP = S == 1 ? 4096 : 1;
    __shared__ float sv_s[MCAP];
    __shared__ int sv_i[MCAP];
    __shared__ int nsurv;
    __shared__ int lkey;
    const int q = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    // The k best score at least the final bound gbound[q] (a proven lower
    // bound on the k-th best score) and at least the k-th entry of every
    // workgroup list, so only entries that reach both can be in the result.  For k <= 64 those entries are gathered in LDS: when at
    // most 64 survive one wave sorts them; up to MCAP, each wave folds its
    // share in sorted runs of 64 into a running top 64 and the four lists
    // are merged; beyond that (and for larger k) the lists are merged in
    // full.
    if (threadIdx.x == 0) {
        nsurv = k <= 64 ? 0 : (1 << 30);   // k > 64: the full merge
        lkey = gbound[q];
    }
    __syncthreads();
    if (k <= 64) {
        const int64_t base = (int64_t)q * G * k;
        // Each workgroup's list is sorted, and its k best are k distinct
        // vectors: the k-th entry of any list is also a lower bound on the
        // query's k-th best score, and usually a much tighter one.
        // And the lists hold disjoint vectors, so the k-th largest of any
        // lists' best entries is one too: each wave sorts the best entries
        // of 64 lists and offers its k-th.
        for (int g0 = 0; g0 < G; g0 += 256) {
            const int g = g0 + threadIdx.x;
            const int64_t e = base + (int64_t)(g < G ? g : 0) * k;
            const bool in = g < G;
            const int last_i = in ? ci[e + (k - 1)] : INT_MAX;
            const float last_s = in ? cs[e + (k - 1)] : -INFINITY;
            const int top_i = in ? ci[e] : INT_MAX;
            float top_s = in && top_i != INT_MAX ? cs[e] : -INFINITY;
            int top_g = g;
            if (last_i != INT_MAX) atomicMax(&lkey, fkey(last_s));
            if (k > 1) {   // at k = 1 a list's best entry is its k-th
                wave_sort64(top_s, top_g, lane);
                const float kth = __shfl(top_s, k - 1);
                if (lane == 0 && kth > -INFINITY) atomicMax(&lkey, fkey(kth));
            }
        }
        __syncthreads();
        const float bound = unfkey(lkey);
        // rounds of MERGE_BATCH entries per thread, loaded together (one
        // memory round trip per round instead of one per entry)
        constexpr int MERGE_BATCH = 16;
        for (int e0 = 0; e0 < G * k; e0 += 256 * MERGE_BATCH) {
            float sc[MERGE_BATCH];
            int id[MERGE_BATCH];
#pragma unroll
            for (int u = 0; u < MERGE_BATCH; ++u) {
                const int e = e0 + u * 256 + threadIdx.x;
                const bool in = e < G * k;
                sc[u] = in ? cs[base + e] : -INFINITY;
                id[u] = in ? ci[base + e] : INT_MAX;
            }
#pragma unroll
            for (int u = 0; u < MERGE_BATCH; ++u) {
                const bool keep = id[u] != INT_MAX && !(sc[u] < bound);
                const uint64_t m = __ballot(keep);
                if (m) {
                    int pos0 = 0;
                    if (lane == 0) pos0 = atomicAdd(&nsurv, __popcll(m));
                    pos0 = __shfl(pos0, 0);
                    const int pos = pos0 + __popcll(m & ((1ull << lane) - 1));
                    if (keep && pos < MCAP) {
                        sv_s[pos] = sc[u];
                        sv_i[pos] = id[u];
                    }
                }
            }
        }
    }
    __syncthreads();
    const int ns = nsurv;
    if (ns <= 64) {
        if (wave == 0) {
            float sv = lane < ns ? sv_s[lane] : -INFINITY;
            int iv = lane < ns ? sv_i[lane] : INT_MAX;
            wave_sort64(sv, iv, lane);
            for (int r = lane; r < k; r += 64) {
                const bool empty = r >= 64 || !(sv > -INFINITY);
                ids[(int64_t)q * k + r] = empty ? -1 : (int64_t)iv;
                scores[(int64_t)q * k + r] = empty ? -INFINITY : sv;
            }
        }
        return;
    }
    if (S == 1 && ns <= MCAP) {
        float ls1[1] = {-INFINITY};
        int li1[1] = {INT_MAX};
        for (int c = wave * 64; c < ns; c += 256) {
            float v = c + lane < ns ? sv_s[c + lane] : -INFINITY;
            int iv = c + lane < ns ? sv_i[c + lane] : INT_MAX;
            wave_sort64(v, iv, lane);
            merge_sorted64<1>(ls1, li1, v, iv, lane);
        }
        st_s[wave * 64 + lane] = ls1[0];
        st_i[wave * 64 + lane] = li1[0];
        __syncthreads();
        if (wave == 0) {
            for (int w = 1; w < 4; ++w) {
                const float os[1] = {st_s[w * 64 + lane]};
                const int oi[1] = {st_i[w * 64 + lane]};
                merge_lists<1>(ls1, li1, os, oi, lane);
            }
            if (lane < k) {
                const bool empty = !(ls1[0] > -INFINITY);
                ids[(int64_t)q * k + lane] = empty ? -1 : (int64_t)li1[0];
                scores[(int64_t)q * k + lane] = empty ? -INFINITY : ls1[0];
            }
        }
        return;
    }
    __syncthreads();   // the stage is reused below
    float ls[S];
    int li[S];
#pragma unroll
    for (int a = 0; a < S; ++a) {
        ls[a] = -INFINITY;
        li[a] = INT_MAX;
    }
    // wave w merges lists w, w + 4, ...; MERGE_LISTS of them are loaded
    // together (one memory round trip per batch instead of one per list)
    constexpr int MERGE_LISTS = 8;
    for (int g0 = wave; g0 < G; g0 += 4 * MERGE_LISTS) {
        float os[MERGE_LISTS][S];
        int oi[MERGE_LISTS][S];
#pragma unroll
        for (int u = 0; u < MERGE_LISTS; ++u) {
            const int g = g0 + 4 * u;
            const int64_t base = ((int64_t)q * G + (g < G ? g : 0)) * k;
#pragma unroll
            for (int a = 0; a < S; ++a) {
                const int r = a * 64 + lane;
                const bool in = g < G && r < k;
                os[u][a] = in ? cs[base + r] : -INFINITY;
                oi[u][a] = in ? ci[base + r] : INT_MAX;
            }
        }
#pragma unroll
        for (int u = 0; u < MERGE_LISTS; ++u) merge_lists<S>(ls, li, os[u], oi[u], lane);
    }
#pragma unroll
    for (int a = 0; a < S; ++a) {
        st_s[wave * 64 * S + a * 64 + lane] = ls[a];
        st_i[wave * 64 * S + a * 64 + lane] = li[a];
    }
    __syncthreads();
    if (wave == 0) {
        for (int w = 1; w < 4; ++w) {
            float os[S];
            int oi[S];
#pragma unroll
            for (int a = 0; a < S; ++a) {
                os[a] = st_s[w * 64 * S + a * 64 + lane];
                oi[a] = st_i[w * 64 * S + a * 64 + lane];
            }
            merge_lists<S>(ls, li, os, oi, lane);
        }
#pragma unroll
        for (int a = 0; a < S; ++a) {
            const int r = a * 64 + lane;
            if (r < k) {
                const bool empty = !(ls[a] > -INFINITY);
                ids[(int64_t)q * k + r] = empty ? -1 : (int64_t)li[a];
                scores[(int64_t)q * k + r] = empty ? -INFINITY : ls[a];
            }
        }
    }
}

// ---------------------------------------------------------------- large k
// Top k (kMaxK >= k > kMaxTopK) of a query's n scores by radix selection:
// scores map to order-preserving unsigned keys (larger score, larger key);
// three histogram passes over 11, 11 and 10 key bits find the key T of the
// k-th best; the vectors with a larger key and, in id order, the first ones
// with key T make up the k best (ties broken by id, as everywhere); a
// bitonic sort in LDS orders them by (score descending, id ascending).
// One workgroup of 1024 threads per query.  Entries of score -inf (vectors
// the filter dropped) become padding (-1, -inf).
constexpr int SEL_T = 1024;

__device__ inline uint32_t ukey(float f) { return (uint32_t)fkey(f) ^ 0x80000000u; }
__device__ inline float unukey(uint32_t u) { return unfkey((int)(u ^ 0x80000000u)); }

__global__ __launch_bounds__(SEL_T) void select_topk_kernel(const float *__restrict__ scores,
                                                           int64_t n, int k,
                                                           int64_t *__restrict__ ids_out,
                                                           float *__restrict__ scores_out) {
    __shared__ uint32_t hist[2048];
    __shared__ uint64_t cand[kMaxK];          // (key << 32) | (0xFFFFFFFF - id)
    __shared__ int wave_eq[SEL_T / 64];
    __shared__ uint32_t sel[4];               // [0] prefix, [1] still needed, [2] candidates
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const float *sc = scores + (int64_t)blockIdx.x * n;
    const int kk = (int64_t)k < n ? k : (int)n;       // entries to return
    uint32_t prefix = 0, pmask = 0;
    uint32_t need = (uint32_t)kk;
    if (kk > 0) {
        for (int pass = 0; pass < 3; ++pass) {
            const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
            const int bins = pass == 2 ? 1024 : 2048;
            for (int b = tid; b < 2048; b += SEL_T) hist[b] = 0;
            __syncthreads();
            for (int64_t i = tid; i < n; i += SEL_T) {
                const uint32_t u = ukey(sc[i]);
                if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & (bins - 1)], 1u);
            }
            __syncthreads();
            if (tid == 0) {
                // bin of the need-th largest key within the prefix class
                uint32_t above = 0;
                int b = bins - 1;
                for (; b > 0; --b) {
                    if (above + hist[b] >= need) break;
                    above += hist[b];
                }
                sel[0] = prefix | ((uint32_t)b << shift);
                sel[1] = need - above;
            }
            __syncthreads();
            prefix = sel[0];
            need = sel[1];
            pmask |= (uint32_t)(bins - 1) << shift;
            __syncthreads();
        }
    }
    // prefix is now the key T of the kk-th best; `need` of the keys equal to
    // T are taken, the ones with the smallest ids
    const uint32_t T = prefix;
    const int64_t len = ((n + SEL_T / 64 - 1) / (SEL_T / 64) + 63) / 64 * 64;   // per wave
    const int64_t w0 = wave * len, w1 = w0 + len < n ? w0 + len : n;
    int eq = 0;
    if (kk > 0)
        for (int64_t i = w0 + lane; i < w1; i += 64) eq += ukey(sc[i]) == T;
    for (int m = 32; m > 0; m >>= 1) eq += __shfl_xor(eq, m, 64);
    if (lane == 0) wave_eq[wave] = eq;
    if (tid == 0) sel[2] = 0;
    __syncthreads();
    if (kk > 0) {
        int before = 0;
        for (int w = 0; w < wave; ++w) before += wave_eq[w];
        for (int64_t i0 = w0; i0 < w1; i0 += 64) {
            const int64_t i = i0 + lane;
            const uint32_t u = i < w1 ? ukey(sc[i]) : 0u;
            const bool is_eq = i < w1 && u == T;
            const uint64_t m = __ballot(is_eq);
            const int rank = before + __popcll(m & ((1ull << lane) - 1));
            const bool take = (i < w1 && u > T) || (is_eq && rank < (int)need);
            if (take) {
                const uint32_t at = atomicAdd(&sel[2], 1u);
                cand[at] = ((uint64_t)u << 32) | (0xFFFFFFFFu - (uint32_t)i);
            }
            before += __popcll(m);
        }
    }
    __syncthreads();
    // pad to a power of two and sort descending
    int P = 1;
    while (P < kk) P <<= 1;
    for (int e = kk + tid; e < P; e += SEL_T) cand[e] = 0;
    __syncthreads();
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int e = tid; e < P / 2; e += SEL_T) {
                const int lo = 2 * e - (e & (stride - 1));
                const int hi = lo + stride;
                const bool desc = (lo & size) == 0;
                const uint64_t a = cand[lo], b = cand[hi];
                if ((a < b) == desc) {
                    cand[lo] = b;
                    cand[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    int64_t *io = ids_out + (int64_t)blockIdx.x * k;
    float *so = scores_out + (int64_t)blockIdx.x * k;
    for (int r = tid; r < k; r += SEL_T) {
        int64_t id = -1;
        float s = -INFINITY;
        if (r < kk) {
            const float v = unukey((uint32_t)(cand[r] >> 32));
            if (v > -INFINITY) {
                s = v;
                id = (int64_t)(0xFFFFFFFFu - (uint32_t)(cand[r] & 0xFFFFFFFFu));
            }
        }
        io[r] = id;
        so[r] = s;
    }
}

// Over-fetch post-filter (section V-C baseline): from each query's list of
// kk entries in rank order, the first k whose tenant the query's allowlist
// admits (padding -1 / -inf after them).  One wave per query.
__global__ __launch_bounds__(64) void postfilter_kernel(const int64_t *__restrict__ ids_in,
                                                       const float *__restrict__ sc_in, int kk,
                                                       const uint16_t *__restrict__ tenants,
                                                       const uint64_t *__restrict__ allow, int W,
                                                       int k, int64_t *__restrict__ ids_out,
                                                       float *__restrict__ sc_out) {
    const int q = blockIdx.x, lane = threadIdx.x;
    const int64_t *ii = ids_in + (int64_t)q * kk;
    const float *ss = sc_in + (int64_t)q * kk;
    const uint64_t *al = allow + (int64_t)q * W;
    int64_t *io = ids_out + (int64_t)q * k;
    float *so = sc_out + (int64_t)q * k;
    int kept = 0;
    for (int r0 = 0; r0 < kk && kept < k; r0 += 64) {
        const int r = r0 + lane;
        const int64_t id = r < kk ? ii[r] : -1;
        bool keep = false;
        if (id >= 0) {
            const int t = tenants[id];
            keep = (al[t >> 6] >> (t & 63)) & 1ull;
        }
        const uint64_t m = __ballot(keep);
        const int pos = kept + __popcll(m & ((1ull << lane) - 1));
        if (keep && pos < k) {
            io[pos] = id;
            so[pos] = ss[r];
        }
        kept += __popcll(m);
    }
    for (int r = (kept < k ? kept : k) + lane; r < k; r += 64) {
        io[r] = -1;
        so[r] = -INFINITY;
    }
}

int lut_words_for(const ScanShape &s) {
    if (s.bits == 8) return kByteRepWords + s.d;
    if (s.bits == 3) return s.chunks * 40 * 8;
    return s.chunks * 32 * 16;
}

// The split scans serve searches over 1-, 2-, 3- and 4-bit codes whose
// chunk count is a multiple of their 8-chunk groups, unfiltered or filtered.
bool use_split(const ScanShape &s) {
    return s.bits != 8 && s.chunks % 8 == 0;
}

size_t lds_bytes_for(const ScanShape &s, int S, bool split, bool filtered) {
    // split: block sums and counts, misc, |q'| sums, levels, 64 survivors;
    // filtered split: also the block list and the allowlist
    size_t fixed = (size_t)s.W * 8 + 16 + 64;
    if (split) {
        fixed = (size_t)kPassBlocks * 65 * 4 + 16 + 64 + 64 + 512;
        if (filtered) fixed += 16 + (size_t)kListMax * 4 + (size_t)s.W * 8;
    }
    return (size_t)aux_words(lut_words_for(s), S) * 4 + fixed;
}

// Queries per scan launch: as many as fit a 256 MiB candidate buffer, and
// few enough that the split scan's work items of one workgroup (queries x
// its 8-chunk groups) stay below 2^30.
int64_t query_chunk(const ScanShape &s, int64_t nq, int k, int grid) {
    const int64_t per = (int64_t)grid * k * (int64_t)(sizeof(float) + sizeof(int));
    int64_t qc = ((int64_t)256 << 20) / per;
    const int64_t groups = ((s.nblk + grid - 1) / grid) * (s.chunks / 8 + 1);
    const int64_t qt = ((int64_t)1 << 30) / (groups + 1);
    if (qt < qc) qc = qt;
    if (qc < 1) qc = 1;
    return nq < qc ? nq : qc;
}

template <int MODE, int S, int PF, bool ALL = false>
hipError_t launch_scan(const ScanParams &p, int grid, size_t lds, hipStream_t stream) {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)scan_kernel<MODE, S, PF, ALL>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL((scan_kernel<MODE, S, PF, ALL>), dim3(grid), dim3(SCAN_THREADS), lds, stream, p);
    return hipGetLastError();
}

// Prefetch depth: 8 chunks in flight per lane when the chunk count allows.
template <int MODE, int S>
hipError_t launch_scan_pf(const ScanParams &p, int grid, size_t lds, hipStream_t stream) {
    if (p.chunks % 8 == 0) return launch_scan<MODE, S, 8>(p, grid, lds, stream);
    if (p.chunks % 4 == 0) return launch_scan<MODE, S, 4>(p, grid, lds, stream);
    if (p.chunks % 2 == 0) return launch_scan<MODE, S, 2>(p, grid, lds, stream);
    return launch_scan<MODE, S, 1>(p, grid, lds, stream);
}

// The all-scores scan (large k), prefetching 8 chunks when the count allows.
template <int MODE>
hipError_t launch_scan_all(const ScanParams &p, int grid, size_t lds, hipStream_t stream) {
    if (p.chunks % 8 == 0) return launch_scan<MODE, 1, 8, true>(p, grid, lds, stream);
    if (p.chunks % 4 == 0) return launch_scan<MODE, 1, 4, true>(p, grid, lds, stream);
    if (p.chunks % 2 == 0) return launch_scan<MODE, 1, 2, true>(p, grid, lds, stream);
    return launch_scan<MODE, 1, 1, true>(p, grid, lds, stream);
}

template <int MODE, int S>
hipError_t launch_split(const ScanParams &p, int grid, size_t lds, hipStream_t stream) {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)split_scan_kernel<MODE, S>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)split_filtered_kernel<MODE, S>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    if (p.allow || p.live || p.slot_allow)
        hipLaunchKernelGGL((split_filtered_kernel<MODE, S>), dim3(grid), dim3(SCAN_THREADS), lds,
                           stream, p);
    else
        hipLaunchKernelGGL((split_scan_kernel<MODE, S>), dim3(grid), dim3(SCAN_THREADS), lds, stream,
                           p);
    return hipGetLastError();
}

template <int S>
hipError_t launch_scan_mode(const ScanParams &p, int grid, size_t lds, bool split,
                            hipStream_t stream) {
    if (split) {
        if (p.bits == 3) return launch_split<TRIBIT, S>(p, grid, lds, stream);
        return launch_split<NIBBLE, S>(p, grid, lds, stream);
    }
    if (p.bits == 8) return launch_scan_pf<BYTE, S>(p, grid, lds, stream);
    if (p.bits == 3) return launch_scan_pf<TRIBIT, S>(p, grid, lds, stream);
    return launch_scan_pf<NIBBLE, S>(p, grid, lds, stream);
}

}  // namespace

// The compute-unit count is asked of the runtime once per device and kept:
// every search call needs it (grid size and workspace layout), and the query
// costs about as much as a kernel launch on the host.
int device_cu_count() {
    static std::atomic<int> cached[64];
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (dev >= 0 && dev < 64) {
        const int c = cached[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (dev >= 0 && dev < 64 && cus > 0) cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

// Queries per launch of the large-k path: their scores (n floats each) fill
// at most 256 MiB.
int64_t all_scores_chunk(const ScanShape &s, int64_t nq) {
    const int64_t per = (s.n > 0 ? s.n : 1) * (int64_t)sizeof(float);
    int64_t qc = ((int64_t)256 << 20) / per;
    if (qc < 1) qc = 1;
    return nq < qc ? nq : qc;
}

size_t lut_search_workspace_bytes(const ScanShape &s, int64_t nq, int k, int grid) {
    if (k > kMaxTopK) {
        size_t b = (size_t)nq * s.d * sizeof(float);
        b = (b + 255) & ~(size_t)255;
        b += (size_t)all_scores_chunk(s, nq) * (s.n > 0 ? s.n : 1) * sizeof(float);
        b = (b + 255) & ~(size_t)255;
        return b + 256;
    }
    const int64_t qc = query_chunk(s, nq, k, grid);
    size_t b = (size_t)nq * s.d * sizeof(float);
    b = (b + 255) & ~(size_t)255;
    b += (size_t)qc * grid * k * (sizeof(float) + sizeof(int));
    b = (b + 255) & ~(size_t)255;
    b += (size_t)qc * sizeof(int);
    b = (b + 255) & ~(size_t)255;
    return b + 256;
}

// The global bounds of a top-k search in its workspace: after the rotated
// queries and the candidate lists of one query chunk.
static int *search_bounds(void *ws, const ScanShape &s, int64_t nq, int k, int grid) {
    const int64_t qc = query_chunk(s, nq, k, grid);
    uint8_t *p8 = static_cast<uint8_t *>(ws);
    p8 += ((size_t)nq * s.d * sizeof(float) + 255) & ~(size_t)255;
    uint8_t *after = p8 + (size_t)qc * grid * k * (sizeof(float) + sizeof(int));
    return reinterpret_cast<int *>((reinterpret_cast<uintptr_t>(after) + 255) & ~(uintptr_t)255);
}

int *lut_search_bounds(const ScanShape &s, int64_t nq, int k, int grid, void *ws) {
    if (nq <= 0 || k > kMaxTopK || query_chunk(s, nq, k, grid) < nq) return nullptr;
    return search_bounds(ws, s, nq, k, grid);
}

hipError_t lut_search(const ScanShape &s, const uint8_t *blocked, const float *scales,
                      const uint16_t *tenants, const uint64_t *summaries, const float *cents32,
                      const float *Qrot, int64_t nq, int k, const SearchFilter &filter, int grid,
                      void *ws, size_t ws_bytes, int64_t *ids, float *scores,
                      hipStream_t stream, const float *qconst, bool bounds_ready) {
    const uint64_t *allow = filter.allow;
    const int64_t qc = query_chunk(s, nq, k, grid);
    uint8_t *p8 = static_cast<uint8_t *>(ws);
    p8 += ((size_t)nq * s.d * sizeof(float) + 255) & ~(size_t)255;   // rotated queries live here
    float *cand_s = reinterpret_cast<float *>(p8);
    int *cand_i = reinterpret_cast<int *>(cand_s + (size_t)qc * grid * k);
    int *gbound = search_bounds(ws, s, nq, k, grid);
    (void)ws_bytes;
    if (k > kMaxTopK) {
        // every score, then a radix selection per query
        float *all = reinterpret_cast<float *>(p8);
        const int64_t qa = all_scores_chunk(s, nq);
        const size_t lds = lds_bytes_for(s, 1, false, filter.any());
        for (int64_t q0 = 0; q0 < nq; q0 += qa) {
            const int64_t m = (nq - q0) < qa ? (nq - q0) : qa;
            ScanParams p{};
            p.codes = reinterpret_cast<const uint4 *>(blocked);
            p.scales = scales;
            p.tenants = tenants;
            p.summaries = summaries;
            p.allow = allow ? allow + q0 * s.W : nullptr;
            p.live = filter.live;
            p.slot_allow = filter.slot_allow ? filter.slot_allow + q0 * s.nblk : nullptr;
            p.qrot = Qrot + q0 * s.d;
            p.qconst = qconst ? qconst + q0 : nullptr;
            p.cents = cents32;
            p.cand_s = all;
            p.n = s.n;
            p.nblk = s.nblk;
            p.d = s.d;
            p.bits = s.bits;
            p.chunks = s.chunks;
            p.W = s.W;
            p.k = k;
            p.nq = (int)m;
            p.lut_words = lut_words_for(s);
            hipLaunchKernelGGL(fill_keys, dim3(1024), dim3(256), 0, stream,
                               reinterpret_cast<int *>(all), m * s.n, (int)0xFF800000u);   // -inf
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            if (s.bits == 8)
                e = launch_scan_all<BYTE>(p, grid, lds, stream);
            else if (s.bits == 3)
                e = launch_scan_all<TRIBIT>(p, grid, lds, stream);
            else
                e = launch_scan_all<NIBBLE>(p, grid, lds, stream);
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL(select_topk_kernel, dim3((unsigned)m), dim3(SEL_T), 0, stream, all,
                               s.n, k, ids + q0 * k, scores + q0 * k);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    const int S = k <= 64 ? 1 : (k <= 128 ? 2 : 4);
    for (int64_t q0 = 0; q0 < nq; q0 += qc) {
        const int64_t m = (nq - q0) < qc ? (nq - q0) : qc;
        ScanParams p{};
        p.codes = reinterpret_cast<const uint4 *>(blocked);
        p.scales = scales;
        p.tenants = tenants;
        p.summaries = summaries;
        p.allow = allow ? allow + q0 * s.W : nullptr;
        p.live = filter.live;
        p.slot_allow = filter.slot_allow ? filter.slot_allow + q0 * s.nblk : nullptr;
        p.qrot = Qrot + q0 * s.d;
        p.qconst = qconst ? qconst + q0 : nullptr;
        p.cents = cents32;
        p.cand_s = cand_s;
        p.cand_i = cand_i;
        p.gbound = gbound;
        p.n = s.n;
        p.nblk = s.nblk;
        p.d = s.d;
        p.bits = s.bits;
        p.chunks = s.chunks;
        p.W = s.W;
        p.k = k;
        p.nq = (int)m;
        p.lut_words = lut_words_for(s);
        const bool split = use_split(s) && lds_bytes_for(s, S, true, filter.any()) <= 160 * 1024;
        const size_t lds = lds_bytes_for(s, S, split, filter.any());
        hipError_t e = hipSuccess;
        if (!(bounds_ready && q0 == 0 && m == nq)) {
            hipLaunchKernelGGL(fill_keys, dim3(1), dim3(256), 0, stream, gbound, m, kBoundInit);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        if (S == 1)
            e = launch_scan_mode<1>(p, grid, lds, split, stream);
        else if (S == 2)
            e = launch_scan_mode<2>(p, grid, lds, split, stream);
        else
            e = launch_scan_mode<4>(p, grid, lds, split, stream);
        if (e != hipSuccess) return e;
        if (S == 1)
            hipLaunchKernelGGL(merge_kernel<1>, dim3(m), dim3(256), 0, stream, cand_s, cand_i,
                               grid, k, gbound, ids + q0 * k, scores + q0 * k);
        else if (S == 2)
            hipLaunchKernelGGL(merge_kernel<2>, dim3(m), dim3(256), 0, stream, cand_s, cand_i,
                               grid, k, gbound, ids + q0 * k, scores + q0 * k);
        else
            hipLaunchKernelGGL(merge_kernel<4>, dim3(m), dim3(256), 0, stream, cand_s, cand_i,
                               grid, k, gbound, ids + q0 * k, scores + q0 * k);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t postfilter(const int64_t *ids_in, const float *sc_in, int64_t nq, int kk,
                      const uint16_t *tenants, const uint64_t *allow, int W, int k,
                      int64_t *ids_out, float *sc_out, hipStream_t stream) {
    if (nq <= 0) return hipSuccess;
    hipLaunchKernelGGL(postfilter_kernel, dim3((unsigned)nq), dim3(64), 0, stream, ids_in, sc_in, kk,
                       tenants, allow, W, k, ids_out, sc_out);
    return hipGetLastError();
}

}  // namespace tq
