// Seeded Haar-random orthogonal rotation (section II-B, step 2).
//
// G (d x d, row-major) is filled with standard normals: SplitMix64 in its
// counter form z_i = mix(seed + (i+1) * 0x9E3779B97F4A7C15) (Steele, Lea &
// Flood 2014), 53-bit uniforms u = ((z >> 11) + 1/2) 2^-53, Box-Muller on
// consecutive pairs.  G = Q T by Householder QR; R = Q diag(sign(diag T)),
// which makes R Haar-distributed (Mezzadri 2007).  The factorisation runs in
// float64 on the host (OpenMP over columns); R is returned as float32.
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <utility>

#include "tq_internal.h"

namespace tq {
namespace {

inline uint64_t splitmix_at(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

inline double uniform53(uint64_t z) { return ((double)(z >> 11) + 0.5) * 0x1.0p-53; }

// Column-major n x n Householder QR in place; returns Q explicitly (column-
// major) and the diagonal of the triangular factor.
void householder_q(int n, std::vector<double> &A, std::vector<double> &Q,
                   std::vector<double> &diag) {
    std::vector<double> tau(n, 0.0);
    diag.assign(n, 0.0);
    // Factorisation: column k holds v_k below the diagonal (v_k[0] == 1 implied).
    for (int k = 0; k < n; ++k) {
        double *col = &A[(size_t)k * n];
        double s = 0.0;
        for (int i = k; i < n; ++i) s += col[i] * col[i];
        const double nrm = std::sqrt(s);
        const double x0 = col[k];
        const double alpha = (x0 >= 0.0) ? -nrm : nrm;
        if (nrm == 0.0) {
            tau[k] = 0.0;
            diag[k] = 0.0;
            continue;
        }
        const double v0 = x0 - alpha;
        // v = (x - alpha e_0) / v0 so that v[0] = 1; tau = -v0 / alpha
        for (int i = k + 1; i < n; ++i) col[i] /= v0;
        tau[k] = -v0 / alpha;
        diag[k] = alpha;
        col[k] = 1.0;
        const double tk = tau[k];
#pragma omp parallel for schedule(static)
        for (int j = k + 1; j < n; ++j) {
            double *cj = &A[(size_t)j * n];
            double w = 0.0;
            for (int i = k; i < n; ++i) w += col[i] * cj[i];
            w *= tk;
            for (int i = k; i < n; ++i) cj[i] -= w * col[i];
        }
        col[k] = alpha;
    }
    // Q = H_0 H_1 ... H_{n-1} I, accumulated backwards.
    Q.assign((size_t)n * n, 0.0);
    for (int i = 0; i < n; ++i) Q[(size_t)i * n + i] = 1.0;
    std::vector<double> v(n);
    for (int k = n - 1; k >= 0; --k) {
        if (tau[k] == 0.0) continue;
        const double *col = &A[(size_t)k * n];
        v[k] = 1.0;
        for (int i = k + 1; i < n; ++i) v[i] = col[i];
        const double tk = tau[k];
#pragma omp parallel for schedule(static)
        for (int j = k; j < n; ++j) {
            double *qj = &Q[(size_t)j * n];
            double w = 0.0;
            for (int i = k; i < n; ++i) w += v[i] * qj[i];
            w *= tk;
            for (int i = k; i < n; ++i) qj[i] -= w * v[i];
        }
    }
}

std::mutex g_cache_mu;
std::map<std::pair<int, uint64_t>, std::vector<float>> g_cache;

}  // namespace

bool make_rotation(int d, uint64_t seed, std::vector<float> *R32) {
    {
        std::lock_guard<std::mutex> lk(g_cache_mu);
        auto it = g_cache.find({d, seed});
        if (it != g_cache.end()) {
            *R32 = it->second;
            return true;
        }
    }
    const size_t nn = (size_t)d * d;
    // G row-major: G[r][c] = g[r*d + c].  Column-major storage of G: A[c*d + r].
    std::vector<double> A(nn);
    for (size_t p = 0; p < nn / 2; ++p) {
        const double u1 = uniform53(splitmix_at(seed, 2 * p));
        const double u2 = uniform53(splitmix_at(seed, 2 * p + 1));
        const double r = std::sqrt(-2.0 * std::log(u1));
        const double g0 = r * std::cos(2.0 * M_PI * u2);
        const double g1 = r * std::sin(2.0 * M_PI * u2);
        const size_t i0 = 2 * p, i1 = 2 * p + 1;
        A[(i0 % d) * d + i0 / d] = g0;
        A[(i1 % d) * d + i1 / d] = g1;
    }
    std::vector<double> Q, diag;
    householder_q(d, A, Q, diag);
    R32->resize(nn);
    for (int c = 0; c < d; ++c) {
        const double s = (diag[c] < 0.0) ? -1.0 : 1.0;
        const double *qc = &Q[(size_t)c * d];
        for (int r = 0; r < d; ++r) (*R32)[(size_t)r * d + c] = (float)(s * qc[r]);
    }
    std::lock_guard<std::mutex> lk(g_cache_mu);
    if (g_cache.size() > 8) g_cache.clear();
    g_cache[{d, seed}] = *R32;
    return true;
}

}  // namespace tq
