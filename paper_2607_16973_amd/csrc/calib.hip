// TQ+ calibration (section II-B): per-coordinate moments of the rotated,
// normalised vectors of a first batch, and the per-query preparation that
// lets the scans score against the calibrated reconstruction.
//
// Fit: y = R x / ||x|| per row; mu_j = mean_r y_rj, sigma_j the population
// standard deviation, kappa_j = sigma_j sqrt(d) (the affine map
// z = (y - mu) / kappa then gives every coordinate mean 0 and variance 1/d,
// the first two moments of the law the codebook was built for).  Rows are
// processed in chunks; each coordinate's sums run in float64 over a fixed
// split of the rows into slices and are then added in slice order, so the
// result does not depend on scheduling.  The sums are taken about the first
// row's value (a shift that keeps the variance free of cancellation).
//
// Query preparation: a coded vector reconstructs as s (mu_j + kappa_j c_j),
// so its score against q' is s (C + sum_j (kappa_j q'_j) c_j), C = sum_j
// mu_j q'_j: the scans run unchanged on q''_j = kappa_j q'_j with C folded
// into every sum.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kernels.h"

namespace tq {
namespace {

constexpr int kCalibRows = 16384;   // rows rotated per chunk
constexpr int kCalibSlices = 64;    // row slices of the per-coordinate sums

// One wave per row: ||x_r|| in float64 (lane-strided sums, then a fixed
// butterfly); flags zero or non-finite norms in *status.
__global__ __launch_bounds__(256) void row_norm_kernel(const float *__restrict__ X, int64_t m, int d,
                                                       double *__restrict__ nrm, int *status) {
    const int lane = threadIdx.x & 63;
    const int64_t r = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= m) return;
    const float *x = X + r * d;
    double s = 0.0;
    for (int j = lane; j < d; j += 64) {
        const double v = (double)x[j];
        s = fma(v, v, s);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    const double v = sqrt(s);
    if (lane == 0) {
        nrm[r] = v;
        if (!(v > 0.0) || !std::isfinite(v)) atomicOr(status, 1);
    }
}

// Thread (slice, j) adds (y_rj - K_j) and its square over the slice's rows
// of this chunk to its running sums; K_j is taken from the chunk's row 0
// when `first` (the first chunk).
__global__ __launch_bounds__(256) void coord_sums_kernel(const float *__restrict__ Y, int64_t rows,
                                                         int d, const double *__restrict__ nrm,
                                                         double *__restrict__ K, bool first,
                                                         double *__restrict__ S1,
                                                         double *__restrict__ S2) {
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int j = (int)(t % d);
    const int sl = (int)(t / d);
    if (sl >= kCalibSlices) return;
    const double k = first ? (double)Y[j] / nrm[0] : K[j];
    if (first && sl == 0) K[j] = k;
    const int64_t r0 = rows * sl / kCalibSlices, r1 = rows * (sl + 1) / kCalibSlices;
    double a = first ? 0.0 : S1[(int64_t)sl * d + j];
    double b = first ? 0.0 : S2[(int64_t)sl * d + j];
    for (int64_t r = r0; r < r1; ++r) {
        const double v = (double)Y[r * d + j] / nrm[r] - k;
        a += v;
        b = fma(v, v, b);
    }
    S1[(int64_t)sl * d + j] = a;
    S2[(int64_t)sl * d + j] = b;
}

__global__ __launch_bounds__(256) void coord_finish_kernel(const double *__restrict__ S1,
                                                           const double *__restrict__ S2,
                                                           const double *__restrict__ K, int64_t m,
                                                           int d, float *__restrict__ mu,
                                                           float *__restrict__ kappa) {
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= d) return;
    double a = 0.0, b = 0.0;
    for (int sl = 0; sl < kCalibSlices; ++sl) {
        a += S1[(int64_t)sl * d + j];
        b += S2[(int64_t)sl * d + j];
    }
    const double mean = a / (double)m;            // of y - K
    double var = b / (double)m - mean * mean;
    var = var > 0.0 ? var : 0.0;
    mu[j] = (float)(K[j] + mean);
    kappa[j] = (float)(sqrt(var) * sqrt((double)d));
}

// One workgroup per query: Qout = kappa * Qin (may alias Qin; each element is
// read and written by the same thread) and qconst = sum_j mu_j q'_j (float64,
// fixed reduction order).
__global__ __launch_bounds__(256) void query_prep_kernel(const float *Qin, int d,
                                                         const float *__restrict__ mu,
                                                         const float *__restrict__ kappa,
                                                         float *Qout, float *__restrict__ qconst) {
    __shared__ double part[4];
    const int64_t q = blockIdx.x;
    const float *qi = Qin + q * d;
    float *qo = Qout + q * d;
    double c = 0.0;
    for (int j = threadIdx.x; j < d; j += 256) {
        const float v = qi[j];
        c = fma((double)mu[j], (double)v, c);
        qo[j] = v * kappa[j];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) qconst[q] = (float)((part[0] + part[1]) + (part[2] + part[3]));
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

size_t calib_workspace_bytes(int d) {
    return align256((size_t)kCalibRows * d * sizeof(float)) +
           align256((size_t)kCalibRows * sizeof(double)) + align256((size_t)d * sizeof(double)) +
           2 * align256((size_t)kCalibSlices * d * sizeof(double));
}

hipError_t calib_fit(const float *X, int64_t m, int d, const float *R, void *ws, int *status_dev,
                     float *mu, float *kappa, hipStream_t stream) {
    if (m <= 0) return hipErrorInvalidValue;
    uint8_t *p = static_cast<uint8_t *>(ws);
    float *Y = reinterpret_cast<float *>(p);
    p += align256((size_t)kCalibRows * d * sizeof(float));
    double *nrm = reinterpret_cast<double *>(p);
    p += align256((size_t)kCalibRows * sizeof(double));
    double *K = reinterpret_cast<double *>(p);
    p += align256((size_t)d * sizeof(double));
    double *S1 = reinterpret_cast<double *>(p);
    p += align256((size_t)kCalibSlices * d * sizeof(double));
    double *S2 = reinterpret_cast<double *>(p);
    const int64_t sum_threads = (int64_t)kCalibSlices * d;
    for (int64_t r0 = 0; r0 < m; r0 += kCalibRows) {
        const int64_t rows = (m - r0) < kCalibRows ? (m - r0) : kCalibRows;
        hipError_t e = rotate_rows_f32(X + r0 * d, rows, d, R, Y, stream);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(row_norm_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream,
                           X + r0 * d, rows, d, nrm, status_dev);
        hipLaunchKernelGGL(coord_sums_kernel, dim3((unsigned)((sum_threads + 255) / 256)), dim3(256),
                           0, stream, Y, rows, d, nrm, K, r0 == 0, S1, S2);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(coord_finish_kernel, dim3((unsigned)((d + 255) / 256)), dim3(256), 0, stream,
                       S1, S2, K, m, d, mu, kappa);
    return hipGetLastError();
}

hipError_t calib_queries(const float *Qin, int64_t nq, int d, const float *mu, const float *kappa,
                         float *Qout, float *qconst, hipStream_t stream) {
    if (nq <= 0) return hipSuccess;
    hipLaunchKernelGGL(query_prep_kernel, dim3((unsigned)nq), dim3(256), 0, stream, Qin, d, mu,
                       kappa, Qout, qconst);
    return hipGetLastError();
}

}  // namespace tq
