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

#include <climits>
#include <cmath>
#include <cstdint>

#include "kernels.h"
#include "topk.h"

namespace tq {
namespace {

constexpr int SCAN_THREADS = 1024;
constexpr int SCAN_WAVES = SCAN_THREADS / 64;
constexpr int PF = 4;   // 16-byte chunks in flight per lane

enum Mode { NIBBLE = 0, TRIBIT = 1, BYTE = 2 };

struct ScanParams {
    const uint4 *codes;
    const float *scales;
    const uint16_t *tenants;
    const uint64_t *summaries;
    const uint64_t *allow;      // [nq][W] or null
    const float *qrot;          // [nq][d]
    const float *cents;         // [levels]
    float *cand_s;              // [nq][G][k]
    int *cand_i;
    int64_t n, nblk;
    int d, bits, chunks, W, k, nq;
    int lut_floats;             // floats of LDS used by the table
};

__device__ inline float nib8(const float *__restrict__ L, uint32_t w) {
    // 8 consecutive 4-bit fields, each indexing its own 16-entry row
    float a = L[0 * 16 + ((w >> 0) & 15)];
    float b = L[1 * 16 + ((w >> 4) & 15)];
    float c = L[2 * 16 + ((w >> 8) & 15)];
    float d = L[3 * 16 + ((w >> 12) & 15)];
    a += L[4 * 16 + ((w >> 16) & 15)];
    b += L[5 * 16 + ((w >> 20) & 15)];
    c += L[6 * 16 + ((w >> 24) & 15)];
    d += L[7 * 16 + ((w >> 28) & 15)];
    return (a + b) + (c + d);
}

__device__ inline float tri10(const float *__restrict__ L, uint32_t w) {
    float a = 0.f, b = 0.f;
#pragma unroll
    for (int t = 0; t < 10; t += 2) {
        a += L[t * 8 + ((w >> (3 * t)) & 7)];
        b += L[(t + 1) * 8 + ((w >> (3 * t + 3)) & 7)];
    }
    return a + b;
}

__device__ inline float byte4(const float *__restrict__ cents, const float *__restrict__ q,
                              uint32_t w) {
    float a = cents[w & 255] * q[0];
    float b = cents[(w >> 8) & 255] * q[1];
    a = fmaf(cents[(w >> 16) & 255], q[2], a);
    b = fmaf(cents[w >> 24], q[3], b);
    return a + b;
}

template <int MODE>
__device__ inline float chunk_sum(const float *__restrict__ lds, int c, uint4 v, int d) {
    if (MODE == NIBBLE) {
        const float *L = lds + c * 32 * 16;
        return (nib8(L, v.x) + nib8(L + 128, v.y)) + (nib8(L + 256, v.z) + nib8(L + 384, v.w));
    } else if (MODE == TRIBIT) {
        const float *L = lds + c * 40 * 8;
        return (tri10(L, v.x) + tri10(L + 80, v.y)) + (tri10(L + 160, v.z) + tri10(L + 240, v.w));
    } else {
        const float *cents = lds;          // 256 centroids
        const float *q = lds + 256 + c * 16;
        return (byte4(cents, q, v.x) + byte4(cents, q + 4, v.y)) +
               (byte4(cents, q + 8, v.z) + byte4(cents, q + 12, v.w));
    }
}

template <int MODE>
__device__ void build_table(float *lds, const ScanParams &p, const float *__restrict__ q) {
    const int tid = threadIdx.x;
    if (MODE == NIBBLE) {
        const int g = 4 / p.bits;              // coordinates per 4-bit field
        const int mask = (1 << p.bits) - 1;
        const int entries = p.lut_floats;      // positions * 16
        for (int e = tid; e < entries; e += SCAN_THREADS) {
            const int pos = e >> 4, c = e & 15;
            float v = 0.f;
            for (int t = 0; t < g; ++t) v += p.cents[(c >> (p.bits * t)) & mask] * q[pos * g + t];
            lds[e] = v;
        }
    } else if (MODE == TRIBIT) {
        const int entries = p.lut_floats;      // positions * 8
        for (int e = tid; e < entries; e += SCAN_THREADS) {
            const int j = e >> 3, c = e & 7;
            lds[e] = (j < p.d) ? p.cents[c] * q[j] : 0.f;
        }
    } else {
        for (int e = tid; e < 256; e += SCAN_THREADS) lds[e] = p.cents[e];
        for (int e = tid; e < p.d; e += SCAN_THREADS) lds[256 + e] = q[e];
    }
}

template <int MODE, int S>
__global__ __launch_bounds__(SCAN_THREADS) void scan_kernel(ScanParams p) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    uint64_t *allow_s = reinterpret_cast<uint64_t *>(lds + p.lut_floats);
    float *stage_s = lds;                                   // reused after the scan
    int *stage_i = reinterpret_cast<int *>(lds + SCAN_WAVES * 64 * S);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int G = gridDim.x;
    const int g = blockIdx.x;
    const bool filtered = p.allow != nullptr;

    for (int qi = 0; qi < p.nq; ++qi) {
        build_table<MODE>(lds, p, p.qrot + (int64_t)qi * p.d);
        if (filtered)
            for (int w = tid; w < p.W; w += SCAN_THREADS) allow_s[w] = p.allow[(int64_t)qi * p.W + w];
        __syncthreads();

        float ls[S];
        int li[S];
#pragma unroll
        for (int a = 0; a < S; ++a) {
            ls[a] = -INFINITY;
            li[a] = INT_MAX;
        }
        float th_s = -INFINITY;
        int th_i = INT_MAX;

        for (int64_t blk = g + (int64_t)G * wave; blk < p.nblk; blk += (int64_t)G * SCAN_WAVES) {
            if (filtered) {
                bool hit = false;
                for (int w = lane; w < p.W; w += 64)
                    hit |= (p.summaries[blk * p.W + w] & allow_s[w]) != 0;
                if (!__any(hit)) continue;      // nothing in this block can match
            }
            const uint4 *src = p.codes + blk * p.chunks * 64 + lane;
            uint4 buf[PF];
#pragma unroll
            for (int i = 0; i < PF; ++i)
                if (i < p.chunks) buf[i] = src[i * 64];
            float acc = 0.f;
            for (int c0 = 0; c0 < p.chunks; c0 += PF) {
#pragma unroll
                for (int i = 0; i < PF; ++i) {
                    const int c = c0 + i;
                    if (c < p.chunks) {
                        const uint4 v = buf[i];
                        if (c + PF < p.chunks) buf[i] = src[(c + PF) * 64];
                        acc += chunk_sum<MODE>(lds, c, v, p.d);
                    }
                }
            }
            const int64_t vid = blk * 64 + lane;
            bool ok = vid < p.n;
            if (ok && filtered) {
                const int t = p.tenants[vid];
                ok = (allow_s[t >> 6] >> (t & 63)) & 1ull;
            }
            float sc = ok ? acc * p.scales[vid] : -INFINITY;
            int id = ok ? (int)vid : INT_MAX;
            const bool cand = better(sc, id, th_s, th_i);
            if (__any(cand)) {
                if (!cand) {
                    sc = -INFINITY;
                    id = INT_MAX;
                }
                wave_sort64(sc, id, lane);
                merge_sorted64<S>(ls, li, sc, id, lane);
                rank_entry<S>(ls, li, p.k - 1, th_s, th_i);
            }
        }
        __syncthreads();   // table no longer needed: reuse LDS for the wave lists
#pragma unroll
        for (int a = 0; a < S; ++a) {
            stage_s[wave * 64 * S + a * 64 + lane] = ls[a];
            stage_i[wave * 64 * S + a * 64 + lane] = li[a];
        }
        __syncthreads();
        if (wave == 0) {
            for (int w = 1; w < SCAN_WAVES; ++w) {
                float os[S];
                int oi[S];
#pragma unroll
                for (int a = 0; a < S; ++a) {
                    os[a] = stage_s[w * 64 * S + a * 64 + lane];
                    oi[a] = stage_i[w * 64 * S + a * 64 + lane];
                }
                merge_lists<S>(ls, li, os, oi, lane);
            }
            const int64_t base = ((int64_t)qi * G + g) * p.k;
#pragma unroll
            for (int a = 0; a < S; ++a) {
                const int r = a * 64 + lane;
                if (r < p.k) {
                    p.cand_s[base + r] = ls[a];
                    p.cand_i[base + r] = li[a];
                }
            }
        }
        __syncthreads();   // LDS is rebuilt for the next query
    }
}

template <int S>
__global__ __launch_bounds__(256) void merge_kernel(const float *__restrict__ cs,
                                                    const int *__restrict__ ci, int G, int k,
                                                    int64_t *__restrict__ ids,
                                                    float *__restrict__ scores) {
    __shared__ float st_s[4 * 64 * S];
    __shared__ int st_i[4 * 64 * S];
    const int q = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    float ls[S];
    int li[S];
#pragma unroll
    for (int a = 0; a < S; ++a) {
        ls[a] = -INFINITY;
        li[a] = INT_MAX;
    }
    for (int g = wave; g < G; g += 4) {
        float os[S];
        int oi[S];
        const int64_t base = ((int64_t)q * G + g) * k;
#pragma unroll
        for (int a = 0; a < S; ++a) {
            const int r = a * 64 + lane;
            os[a] = (r < k) ? cs[base + r] : -INFINITY;
            oi[a] = (r < k) ? ci[base + r] : INT_MAX;
        }
        merge_lists<S>(ls, li, os, oi, lane);
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

int lut_floats_for(const ScanShape &s) {
    if (s.bits == 8) return 256 + s.d;
    if (s.bits == 3) return s.chunks * 40 * 8;
    return s.chunks * 32 * 16;
}

size_t lds_bytes_for(const ScanShape &s, int S) {
    const size_t table = (size_t)lut_floats_for(s) * 4 + (size_t)s.W * 8;
    const size_t stage = (size_t)SCAN_WAVES * 64 * S * 8;
    return table > stage ? table : stage;
}

// Queries per scan launch: as many as fit a 256 MiB candidate buffer.
int64_t query_chunk(int64_t nq, int k, int grid) {
    const int64_t per = (int64_t)grid * k * (int64_t)(sizeof(float) + sizeof(int));
    int64_t qc = ((int64_t)256 << 20) / per;
    if (qc < 1) qc = 1;
    return nq < qc ? nq : qc;
}

template <int MODE, int S>
hipError_t launch_scan(const ScanParams &p, int grid, size_t lds, hipStream_t stream) {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)scan_kernel<MODE, S>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL((scan_kernel<MODE, S>), dim3(grid), dim3(SCAN_THREADS), lds, stream, p);
    return hipGetLastError();
}

template <int S>
hipError_t launch_scan_mode(const ScanParams &p, int grid, size_t lds, hipStream_t stream) {
    if (p.bits == 8) return launch_scan<BYTE, S>(p, grid, lds, stream);
    if (p.bits == 3) return launch_scan<TRIBIT, S>(p, grid, lds, stream);
    return launch_scan<NIBBLE, S>(p, grid, lds, stream);
}

}  // namespace

int device_cu_count() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus;
}

size_t lut_search_workspace_bytes(const ScanShape &s, int64_t nq, int k, int grid) {
    const int64_t qc = query_chunk(nq, k, grid);
    size_t b = (size_t)nq * s.d * sizeof(float);
    b = (b + 255) & ~(size_t)255;
    b += (size_t)qc * grid * k * (sizeof(float) + sizeof(int));
    b = (b + 255) & ~(size_t)255;
    return b + 256;
}

hipError_t lut_search(const ScanShape &s, const uint8_t *blocked, const float *scales,
                      const uint16_t *tenants, const uint64_t *summaries, const float *cents32,
                      const float *Qrot, int64_t nq, int k, const uint64_t *allow, int grid,
                      void *ws, size_t ws_bytes, int64_t *ids, float *scores,
                      hipStream_t stream) {
    const int64_t qc = query_chunk(nq, k, grid);
    uint8_t *p8 = static_cast<uint8_t *>(ws);
    p8 += ((size_t)nq * s.d * sizeof(float) + 255) & ~(size_t)255;   // rotated queries live here
    float *cand_s = reinterpret_cast<float *>(p8);
    int *cand_i = reinterpret_cast<int *>(cand_s + (size_t)qc * grid * k);
    (void)ws_bytes;
    const int S = k <= 64 ? 1 : (k <= 128 ? 2 : 4);
    for (int64_t q0 = 0; q0 < nq; q0 += qc) {
        const int64_t m = (nq - q0) < qc ? (nq - q0) : qc;
        ScanParams p{};
        p.codes = reinterpret_cast<const uint4 *>(blocked);
        p.scales = scales;
        p.tenants = tenants;
        p.summaries = summaries;
        p.allow = allow ? allow + q0 * s.W : nullptr;
        p.qrot = Qrot + q0 * s.d;
        p.cents = cents32;
        p.cand_s = cand_s;
        p.cand_i = cand_i;
        p.n = s.n;
        p.nblk = s.nblk;
        p.d = s.d;
        p.bits = s.bits;
        p.chunks = s.chunks;
        p.W = s.W;
        p.k = k;
        p.nq = (int)m;
        p.lut_floats = lut_floats_for(s);
        const size_t lds = lds_bytes_for(s, S);
        hipError_t e;
        if (S == 1)
            e = launch_scan_mode<1>(p, grid, lds, stream);
        else if (S == 2)
            e = launch_scan_mode<2>(p, grid, lds, stream);
        else
            e = launch_scan_mode<4>(p, grid, lds, stream);
        if (e != hipSuccess) return e;
        if (S == 1)
            hipLaunchKernelGGL(merge_kernel<1>, dim3(m), dim3(256), 0, stream, cand_s, cand_i,
                               grid, k, ids + q0 * k, scores + q0 * k);
        else if (S == 2)
            hipLaunchKernelGGL(merge_kernel<2>, dim3(m), dim3(256), 0, stream, cand_s, cand_i,
                               grid, k, ids + q0 * k, scores + q0 * k);
        else
            hipLaunchKernelGGL(merge_kernel<4>, dim3(m), dim3(256), 0, stream, cand_s, cand_i,
                               grid, k, ids + q0 * k, scores + q0 * k);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace tq
