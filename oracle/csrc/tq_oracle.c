/*
 * CPU oracle: TurboQuant encode, written as the plain definition
 * (test infrastructure only -- never linked into or called by the library).
 *
 * Section II-B, steps 1-5, for one float32 row x of length d:
 *   1. normalise:  n = sqrt(sum_k x_k^2)        sequential float64 sum; every
 *                                                square of a float32 is exact
 *   2. rotate:     S_j = sum_k R[j,k] * x_k     sequential float64 sum over
 *                                                k = 0..d-1; every product of
 *                                                two float32 values is exact
 *   3. quantise:   code_j = #{ i : fl64(t_i * n) <= S_j }
 *                  i.e. the cell of S_j / n with a value on a boundary going
 *                  to the upper cell; a zero row gets code L/2 everywhere
 *   5. scale:      s = n / sqrt(sum_j c2[code_j]),  c2[c] = fl64(c_c * c_c),
 *                  sequential float64 sum over j, stored as float32
 *                  (the per-vector length-renormalisation scalar: the
 *                  reconstruction s * R^T xhat has the length of x)
 * Step 4 (bit packing) is done by the Python wrapper.  Optionally the rotated
 * values S_j are returned too (rot_out, float64 [n][d]).
 *
 * Build with -ffp-contract=off so that no multiply-add is fused: the
 * definition rounds every product and every sum on its own.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Step 3 for one row: code_j = #{ t : T[t] <= S_j } with T[t] = fl64(t_t * n),
 * the thresholds already scaled by the row's norm. */
static void quantise_row(const double *S, const double *T, int32_t d, int32_t L, uint8_t *c)
{
    for (int32_t j = 0; j < d; ++j) {
        int cnt = 0;
        for (int32_t t = 0; t < L - 1; ++t) cnt += (T[t] <= S[j]);
        c[j] = (uint8_t)cnt;
    }
}

/* Returns 0 on success, -1 on bad arguments, -2 on a non-finite input row
 * (its index is written to *bad_row). */
int tqo_encode(const float *X, int64_t n, int32_t d, const float *R,
               const double *bounds, int32_t L, uint8_t *codes,
               double *norm_out, double *rot_out, int64_t *bad_row)
{
    if (!X || !R || !bounds || !codes || n < 0 || d <= 0 || L < 2 || L > 256)
        return -1;
    /* R transposed in float64 so that the inner loop runs over j with k fixed:
     * every S_j still accumulates k = 0, 1, ..., d-1 in order. */
    double *RT = (double *)malloc(sizeof(double) * (size_t)d * (size_t)d);
    if (!RT) return -1;
    for (int32_t j = 0; j < d; ++j)
        for (int32_t k = 0; k < d; ++k)
            RT[(size_t)k * d + j] = (double)R[(size_t)j * d + k];
    int status = 0;
    int64_t first_bad = -1;

#pragma omp parallel
    {
        double *S = (double *)malloc(sizeof(double) * (size_t)d);
        double *T = (double *)malloc(sizeof(double) * (size_t)(L - 1));
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            const float *x = X + (size_t)i * d;
            uint8_t *c = codes + (size_t)i * d;
            int finite = 1;
            double n2 = 0.0;
            for (int32_t k = 0; k < d; ++k) {
                double xk = (double)x[k];
                if (!isfinite(xk)) finite = 0;
                double sq = xk * xk;
                n2 = n2 + sq;
            }
            if (!finite) {
#pragma omp critical
                {
                    if (first_bad < 0 || i < first_bad) first_bad = i;
                    status = -2;
                }
                continue;
            }
            double nrm = sqrt(n2);
            if (norm_out) norm_out[i] = nrm;
            if (nrm == 0.0) {
                memset(c, L / 2, (size_t)d);
                if (rot_out) memset(rot_out + (size_t)i * d, 0, sizeof(double) * (size_t)d);
                continue;
            }
            for (int32_t t = 0; t < L - 1; ++t) {
                double p = bounds[t] * nrm;
                T[t] = p;
            }
            for (int32_t j = 0; j < d; ++j) S[j] = 0.0;
            for (int32_t k = 0; k < d; ++k) {
                const double xk = (double)x[k];
                const double *col = RT + (size_t)k * d;
                for (int32_t j = 0; j < d; ++j) {
                    double prod = col[j] * xk;
                    S[j] = S[j] + prod;
                }
            }
            if (rot_out)
                for (int32_t j = 0; j < d; ++j) rot_out[(size_t)i * d + j] = S[j];
            quantise_row(S, T, d, L, c);
        }
        free(S);
        free(T);
    }
    free(RT);
    if (status == -2 && bad_row) *bad_row = first_bad;
    return status;
}

/* Step 3 alone, for rows already rotated: S [n][d] the sequential float64
 * sums and norms [n] the row norms of tqo_encode (rot_out, norm_out), so one
 * rotation serves several codebooks.  A zero norm gives code L/2. */
int tqo_quantise(const double *S, const double *norms, int64_t n, int32_t d,
                 const double *bounds, int32_t L, uint8_t *codes)
{
    if (!S || !norms || !bounds || !codes || n < 0 || d <= 0 || L < 2 || L > 256)
        return -1;
#pragma omp parallel
    {
        double T[255];
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            uint8_t *c = codes + (size_t)i * d;
            const double nrm = norms[i];
            if (nrm == 0.0) {
                memset(c, L / 2, (size_t)d);
                continue;
            }
            for (int32_t t = 0; t < L - 1; ++t) {
                double p = bounds[t] * nrm;
                T[t] = p;
            }
            quantise_row(S + (size_t)i * d, T, d, L, c);
        }
    }
    return 0;
}

/* Length-renormalisation scalar (step 5) for rows already coded. */
int tqo_scales(const uint8_t *codes, const double *norms, int64_t n, int32_t d,
               const double *cents, int32_t L, float *scale_out)
{
    if (!codes || !norms || !cents || !scale_out || n < 0 || d <= 0 || L < 2)
        return -1;
    double c2[256];
    for (int32_t c = 0; c < L; ++c) {
        double v = cents[c] * cents[c];
        c2[c] = v;
    }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const uint8_t *c = codes + (size_t)i * d;
        if (norms[i] == 0.0) {
            scale_out[i] = 0.0f;
            continue;
        }
        double h2 = 0.0;
        for (int32_t j = 0; j < d; ++j) h2 = h2 + c2[c[j]];
        double s = norms[i] / sqrt(h2);
        scale_out[i] = (float)s;
    }
    return 0;
}

/* TQ+ calibration (section II-B): per-coordinate shift mu_j and spread
 * kappa_j (float32, as stored by an index) move the thresholds of coordinate
 * j to a_jt = fl64(mu_j + fl64(kappa_j t_t)); coordinate j of a vector of
 * norm n gets code #{t : fl64(a_jt n) <= S_j}, S_j the sequential float64
 * dot product of tqo_encode.  mu = 0, kappa = 1 is tqo_encode. */
int tqo_encode_plus(const float *X, int64_t n, int32_t d, const float *R,
                    const double *bounds, int32_t L, const float *mu,
                    const float *kappa, uint8_t *codes, double *norm_out)
{
    if (!X || !R || !bounds || !mu || !kappa || !codes || n < 0 || d <= 0 || L < 2 || L > 256)
        return -1;
    double *A = (double *)malloc(sizeof(double) * (size_t)d * (size_t)(L - 1));
    double *RT = (double *)malloc(sizeof(double) * (size_t)d * (size_t)d);
    if (!A || !RT) {
        free(A);
        free(RT);
        return -1;
    }
    for (int32_t j = 0; j < d; ++j)
        for (int32_t t = 0; t < L - 1; ++t) {
            double p = (double)kappa[j] * bounds[t];
            double a = (double)mu[j] + p;
            A[(size_t)j * (L - 1) + t] = a;
        }
    for (int32_t j = 0; j < d; ++j)
        for (int32_t k = 0; k < d; ++k)
            RT[(size_t)k * d + j] = (double)R[(size_t)j * d + k];
    int status = 0;
#pragma omp parallel
    {
        double *S = (double *)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            const float *x = X + (size_t)i * d;
            uint8_t *c = codes + (size_t)i * d;
            int finite = 1;
            double n2 = 0.0;
            for (int32_t k = 0; k < d; ++k) {
                double xk = (double)x[k];
                if (!isfinite(xk)) finite = 0;
                double sq = xk * xk;
                n2 = n2 + sq;
            }
            if (!finite) {
#pragma omp critical
                status = -2;
                continue;
            }
            double nrm = sqrt(n2);
            if (norm_out) norm_out[i] = nrm;
            if (nrm == 0.0) {
                memset(c, L / 2, (size_t)d);
                continue;
            }
            for (int32_t j = 0; j < d; ++j) S[j] = 0.0;
            for (int32_t k = 0; k < d; ++k) {
                const double xk = (double)x[k];
                const double *col = RT + (size_t)k * d;
                for (int32_t j = 0; j < d; ++j) {
                    double prod = col[j] * xk;
                    S[j] = S[j] + prod;
                }
            }
            for (int32_t j = 0; j < d; ++j) {
                int cnt = 0;
                const double *a = A + (size_t)j * (L - 1);
                for (int32_t t = 0; t < L - 1; ++t) {
                    double thr = a[t] * nrm;
                    cnt += (thr <= S[j]);
                }
                c[j] = (uint8_t)cnt;
            }
        }
        free(S);
    }
    free(A);
    free(RT);
    return status;
}

/* TQ+ scales: the reconstruction of coordinate j is
 * yhat_j = fl64(mu_j + fl64(kappa_j c[code_j])) and s = n / sqrt(sum_j
 * fl64(yhat_j^2)) (sequential over j, float32 result); mu = 0, kappa = 1 is
 * tqo_scales. */
int tqo_scales_plus(const uint8_t *codes, const double *norms, int64_t n, int32_t d,
                    const double *cents, int32_t L, const float *mu, const float *kappa,
                    float *scale_out)
{
    if (!codes || !norms || !cents || !mu || !kappa || !scale_out || n < 0 || d <= 0 || L < 2)
        return -1;
    double *Y2 = (double *)malloc(sizeof(double) * (size_t)d * (size_t)L);
    if (!Y2) return -1;
    for (int32_t j = 0; j < d; ++j)
        for (int32_t c = 0; c < L; ++c) {
            double p = (double)kappa[j] * cents[c];
            double y = (double)mu[j] + p;
            double y2 = y * y;
            Y2[(size_t)j * L + c] = y2;
        }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const uint8_t *c = codes + (size_t)i * d;
        if (norms[i] == 0.0) {
            scale_out[i] = 0.0f;
            continue;
        }
        double h2 = 0.0;
        for (int32_t j = 0; j < d; ++j) h2 = h2 + Y2[(size_t)j * L + c[j]];
        double s = norms[i] / sqrt(h2);
        scale_out[i] = (float)s;
    }
    free(Y2);
    return 0;
}
