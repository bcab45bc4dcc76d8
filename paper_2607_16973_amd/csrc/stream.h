// Loads of the code stream (device code).
//
// The scans read the whole code store once per query (or per query tile) and
// never again before it has been evicted, so its 16-byte chunks are loaded
// non-temporally: they do not displace cached data, and streaming reads of a
// store larger than the caches run measurably faster this way on gfx950.
#pragma once

#include <hip/hip_runtime.h>

namespace tq {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint4 load_stream(const uint4 *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

}  // namespace tq
