// Code-store layout conversions and tenant summaries (section III-B).
//
// Canonical layout: one little-endian bitstream per vector, coordinate j at
// bits [b*j, b*j + b), least significant bit first (d*b/8 bytes per row).
// Blocked layout (index storage): vector v belongs to 64-vector block v/64,
// lane v%64; its i-th 16-byte chunk sits at ((v/64)*chunks + i)*1024 +
// (v%64)*16, so the 64 lanes of a wave read one contiguous KiB per chunk.
// For b in {1,2,4,8} chunk i holds canonical bytes [16i, 16i+16), each
// 32-bit word rotated left by 2 bits when b in {1,2,4}; for b = 3 every
// 32-bit word holds 10 codes (bits 3t..3t+2 for code t, 2 pad bits).
// Block summaries: W = ceil(T/64) words per block, bit t set when some vector
// of the block belongs to tenant t.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace tq {
namespace {

__device__ inline uint32_t get_code3(const uint8_t *row, int j) {
    const int bit = 3 * j;
    const int byte = bit >> 3, sh = bit & 7;
    uint32_t v = row[byte];
    if (sh > 5) v |= (uint32_t)row[byte + 1] << 8;
    return (v >> sh) & 7u;
}

__global__ void canon_to_blocked_kernel(const uint8_t *__restrict__ canon,
                                        const float *__restrict__ scales, int64_t n, int d,
                                        int bits, int chunks, uint8_t *__restrict__ blocked,
                                        float *__restrict__ blocked_scales, int64_t base) {
    const int64_t rowbytes = (int64_t)d * bits / 8;
    const int64_t total = n * chunks;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / chunks;
        const int c = (int)(e % chunks);
        const int64_t v = base + i;
        uint4 *dst = reinterpret_cast<uint4 *>(blocked + ((v >> 6) * chunks + c) * 1024 + (v & 63) * 16);
        const uint8_t *row = canon + i * rowbytes;
        if (bits != 3) {
            uint4 q4 = reinterpret_cast<const uint4 *>(row)[c];
            if (blocked_rotated(bits)) {
                q4.x = rotl2(q4.x);
                q4.y = rotl2(q4.y);
                q4.z = rotl2(q4.z);
                q4.w = rotl2(q4.w);
            }
            *dst = q4;
        } else {
            uint32_t w[4];
            for (int q = 0; q < 4; ++q) {
                uint32_t word = 0;
                for (int t = 0; t < 10; ++t) {
                    const int j = (c * 4 + q) * 10 + t;
                    if (j < d) word |= get_code3(row, j) << (3 * t);
                }
                w[q] = word;
            }
            *dst = make_uint4(w[0], w[1], w[2], w[3]);
        }
        if (c == 0) blocked_scales[v] = scales[i];
    }
}

__global__ void blocked_to_canon_kernel(const uint8_t *__restrict__ blocked,
                                        const float *__restrict__ blocked_scales, int64_t n,
                                        int d, int bits, int chunks, uint8_t *__restrict__ canon,
                                        float *__restrict__ scales) {
    const int64_t rowbytes = (int64_t)d * bits / 8;
    if (bits != 3) {
        const int64_t total = n * chunks;
        for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
             e += (int64_t)gridDim.x * blockDim.x) {
            const int64_t v = e / chunks;
            const int c = (int)(e % chunks);
            const uint4 *src = reinterpret_cast<const uint4 *>(blocked + ((v >> 6) * chunks + c) * 1024 + (v & 63) * 16);
            uint4 w = *src;
            if (blocked_rotated(bits)) {
                w.x = rotr2(w.x);
                w.y = rotr2(w.y);
                w.z = rotr2(w.z);
                w.w = rotr2(w.w);
            }
            if (canon) reinterpret_cast<uint4 *>(canon + v * rowbytes)[c] = w;
            if (c == 0 && scales) scales[v] = blocked_scales[v];
        }
    } else {
        // one thread per output byte of the canonical bitstream
        const int64_t total = n * rowbytes;
        for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
             e += (int64_t)gridDim.x * blockDim.x) {
            const int64_t v = e / rowbytes;
            const int byte = (int)(e % rowbytes);
            const uint8_t *blk = blocked + (v >> 6) * chunks * 1024 + (v & 63) * 16;
            uint32_t out = 0;
            for (int t = 0; t < 8; ++t) {
                const int bit = byte * 8 + t;
                const int j = bit / 3, sh = bit % 3;
                const int word = j / 10, pos = j % 10;
                const uint32_t w = reinterpret_cast<const uint32_t *>(blk + (word >> 2) * 1024)[word & 3];
                out |= ((w >> (3 * pos + sh)) & 1u) << t;
            }
            if (canon) canon[e] = (uint8_t)out;
            if (byte == 0 && scales) scales[v] = blocked_scales[v];
        }
    }
}

__global__ void add_tenants_kernel(const uint16_t *__restrict__ tenants, int64_t n, int64_t base,
                                   int n_tenants, int W, uint16_t *__restrict__ store,
                                   unsigned long long *__restrict__ summaries, int *status) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = tenants ? tenants[i] : 0;
        if (t >= n_tenants) {
            atomicOr(status, 2);
            continue;
        }
        const int64_t v = base + i;
        store[v] = (uint16_t)t;
        atomicOr(&summaries[(v >> 6) * W + (t >> 6)], 1ull << (t & 63));
    }
}

// Marks slots [base, base + n) live.
__global__ void set_live_kernel(unsigned long long *__restrict__ live, int64_t base, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t v = base + i;
        atomicOr(&live[v >> 6], 1ull << (v & 63));
    }
}

// One 64-lane workgroup per listed block: clears the block's slots in
// `clear` from its live mask, then rebuilds its tenant summary from the
// slots still live (W words, staged in LDS).
__global__ __launch_bounds__(64) void retire_kernel(const int64_t *__restrict__ blocks,
                                                    const uint64_t *__restrict__ clear,
                                                    uint64_t *__restrict__ live,
                                                    const uint16_t *__restrict__ tenants, int W,
                                                    uint64_t *__restrict__ summaries) {
    __shared__ unsigned long long words[1024];
    const int64_t b = blocks[blockIdx.x];
    const int lane = threadIdx.x;
    const uint64_t m = live[b] & ~clear[blockIdx.x];
    for (int w = lane; w < W; w += 64) words[w] = 0;
    __syncthreads();
    if ((m >> lane) & 1ull) {
        const int t = tenants[b * 64 + lane];
        atomicOr(&words[t >> 6], 1ull << (t & 63));
    }
    __syncthreads();
    for (int w = lane; w < W; w += 64) summaries[b * W + w] = words[w];
    if (lane == 0) live[b] = m;
}

// Search results in slots -> the slots' external ids (-1 stays -1).
__global__ void map_ids_kernel(int64_t *__restrict__ ids, int64_t count,
                               const uint64_t *__restrict__ ext) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t v = ids[i];
        if (v >= 0) ids[i] = (int64_t)ext[v];
    }
}

int grid_for(int64_t items) {
    int64_t g = (items + 255) / 256;
    if (g > 8192) g = 8192;
    if (g < 1) g = 1;
    return (int)g;
}

}  // namespace

hipError_t canonical_to_blocked(const uint8_t *canon, const float *scales, int64_t n, int d,
                                int bits, uint8_t *blocked, float *blocked_scales, int64_t base,
                                hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int chunks = chunks_per_vector(d, bits);
    hipLaunchKernelGGL(canon_to_blocked_kernel, dim3(grid_for(n * chunks)), dim3(256), 0, stream,
                       canon, scales, n, d, bits, chunks, blocked, blocked_scales, base);
    return hipGetLastError();
}

hipError_t blocked_to_canonical(const uint8_t *blocked, const float *blocked_scales, int64_t n,
                                int d, int bits, uint8_t *canon, float *scales,
                                hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const int chunks = chunks_per_vector(d, bits);
    const int64_t items = bits == 3 ? n * ((int64_t)d * 3 / 8) : n * chunks;
    hipLaunchKernelGGL(blocked_to_canon_kernel, dim3(grid_for(items)), dim3(256), 0, stream,
                       blocked, blocked_scales, n, d, bits, chunks, canon, scales);
    return hipGetLastError();
}

hipError_t add_tenants(const uint16_t *tenants, int64_t n, int64_t base, int n_tenants, int W,
                       uint16_t *tenant_store, uint64_t *summaries, int *status_dev,
                       hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(add_tenants_kernel, dim3(grid_for(n)), dim3(256), 0, stream, tenants, n,
                       base, n_tenants, W, tenant_store,
                       reinterpret_cast<unsigned long long *>(summaries), status_dev);
    return hipGetLastError();
}

hipError_t set_live(uint64_t *live, int64_t base, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(set_live_kernel, dim3(grid_for(n)), dim3(256), 0, stream,
                       reinterpret_cast<unsigned long long *>(live), base, n);
    return hipGetLastError();
}

hipError_t retire_slots(const int64_t *blocks, const uint64_t *clear, int64_t nb, uint64_t *live,
                        const uint16_t *tenants, int W, uint64_t *summaries, hipStream_t stream) {
    if (nb <= 0) return hipSuccess;
    if (W > 1024) return hipErrorInvalidValue;
    hipLaunchKernelGGL(retire_kernel, dim3((unsigned)nb), dim3(64), 0, stream, blocks, clear, live,
                       tenants, W, summaries);
    return hipGetLastError();
}

hipError_t map_ids(int64_t *ids, int64_t count, const uint64_t *ext, hipStream_t stream) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(map_ids_kernel, dim3(grid_for(count)), dim3(256), 0, stream, ids, count, ext);
    return hipGetLastError();
}

}  // namespace tq
