// Search without device allocation: tq_search with its workspace held in a
// file-scope device array instead of a per-call allocation.
//
// The array (TQ_NOALLOC_SCRATCH_BYTES) is part of this library's code object,
// so each GPU the library runs on holds one copy until the process ends.  Its
// device address is looked up once per device, on the first call made with
// that device current, and every later call on that device reuses it: calls
// that overlap in time on one GPU (two streams, two threads) race on it.
// Nothing in it has to start at zero -- the scan kernels write every
// candidate slot and the bounds are set by a fill kernel before each scan --
// so a call only relies on the previous call having finished on the stream.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>

#include "tq_internal.h"

namespace tq {
namespace {

constexpr size_t kScratchBytes = TQ_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // scratch's address on each device

tq_status hip_error(hipError_t e, const char *what) {
    (void)hipGetLastError();
    return fail(TQ_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// Device address of `scratch` on the current device.  The host-side name of
// the array is only a stand-in, so kernels are always given this address.
tq_status scratch_on_current_device(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_error(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(TQ_EUNSUPPORTED, "tq_search_noalloc supports devices 0.." +
                                         std::to_string(kMaxDevices - 1));
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_error(e, "hipGetSymbolAddress(scratch)");
        if (!p || (reinterpret_cast<uintptr_t>(p) & 255) != 0)
            return fail(TQ_EDEVICE, "scratch array has no 256-byte aligned device address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return TQ_OK;
}

// Results of a search over an empty index: every slot is padding.
__global__ void pad_results_kernel(int64_t *ids, float *scores, int64_t m) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        ids[i] = -1;
        scores[i] = -__builtin_huge_valf();
    }
}

}  // namespace
}  // namespace tq

using namespace tq;

extern "C" tq_status tq_search_noalloc(const tq_index *idx, const float *Q_dev, int64_t nq,
                                       int32_t k, const uint64_t *allow_dev, int64_t *ids_dev,
                                       float *scores_dev, void *stream) {
    if (!idx) return fail(TQ_EINVAL, "NULL index");
    if (nq < 0) return fail(TQ_EINVAL, "nq < 0");
    if (k < 1 || k > 4096) return fail(TQ_EINVAL, "k must be in 1..4096");
    if (nq == 0) return TQ_OK;
    if (!Q_dev || !ids_dev || !scores_dev) return fail(TQ_EINVAL, "NULL device pointer");
    int32_t d = 0, n_tenants = 0;
    int64_t n = 0;
    tq_status st = tq_index_info(idx, &d, nullptr, &n_tenants, &n, nullptr);
    if (st != TQ_OK) return st;
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count <= 0) {
        (void)hipGetLastError();
        return fail(TQ_EDEVICE, "no usable GPU");
    }
    void *ws = nullptr;
    st = scratch_on_current_device(&ws);
    if (st != TQ_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (n == 0) {
        const int64_t m = nq * k;
        const int blocks = (int)((m + 255) / 256 < 1024 ? (m + 255) / 256 : 1024);
        hipLaunchKernelGGL(pad_results_kernel, dim3(blocks), dim3(256), 0, s, ids_dev, scores_dev, m);
        e = hipGetLastError();
        return e == hipSuccess ? TQ_OK : hip_error(e, "padding");
    }
    if (!index_rotation_resident(idx))
        return fail(TQ_EINVAL, "tq_search_noalloc: the index's rotation is not on this device yet "
                               "(it is uploaded by the first tq_index_add, tq_index_calibrate or "
                               "allocating search on the index)");
    // queries per tq_search_ex call whose workspace fits in the scratch array
    size_t need = 0;
    st = tq_search_workspace_size(idx, 1, k, TQ_PATH_LUT, &need);
    if (st != TQ_OK) return st;
    if (need > kScratchBytes)
        return fail(TQ_EUNSUPPORTED, "tq_search_noalloc: one query needs " + std::to_string(need) +
                                         " bytes of scratch, more than the " +
                                         std::to_string(kScratchBytes) + " the library holds");
    int64_t qb = nq;
    for (;;) {
        st = tq_search_workspace_size(idx, qb, k, TQ_PATH_LUT, &need);
        if (st != TQ_OK) return st;
        if (need <= kScratchBytes) break;
        const int64_t next = (int64_t)((double)qb * ((double)kScratchBytes / (double)need));
        qb = next < qb ? (next > 1 ? next : 1) : qb - 1;
    }
    const int64_t words = (n_tenants + 63) / 64;
    for (int64_t q0 = 0; q0 < nq; q0 += qb) {
        const int64_t m = (nq - q0) < qb ? (nq - q0) : qb;
        st = tq_search_ex(idx, Q_dev + q0 * d, m, k, allow_dev ? allow_dev + q0 * words : nullptr,
                          TQ_PATH_LUT, ws, kScratchBytes, ids_dev + q0 * k, scores_dev + q0 * k,
                          stream);
        if (st != TQ_OK) return st;
    }
    return TQ_OK;
}
