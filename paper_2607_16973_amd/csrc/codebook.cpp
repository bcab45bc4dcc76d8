// Analytic Lloyd-Max codebook for TurboQuant (section II-B, step 3).
//
// The coordinate law after a random rotation of a unit vector in R^d has
// density proportional to g(x) = (1 - x^2)^((d-3)/2) on [-1, 1].  A Lloyd-Max
// quantiser with L = 2^b levels satisfies (i) every boundary is the midpoint
// of its two neighbouring levels and (ii) every level is the conditional mean
// of its cell.  The law is symmetric, so the positive half (h = L/2 levels
// p_0 < ... < p_{h-1}, cell edges e_0 = 0, e_i = (p_{i-1} + p_i)/2, e_h = 1)
// is solved and mirrored.
//
// Method (independent of any table or library special function):
//  * cell mass  M0(a, b) = int_a^b g  by composite 24-point Gauss-Legendre
//    quadrature on panels no wider than sigma/4 (sigma = 1/sqrt(d)); the
//    integrand is smooth and tiny beyond 40 sigma, where integration stops;
//  * first moment M1(a, b) = int_a^b x g in closed form,
//    [(1-a^2)^((d-1)/2) - (1-b^2)^((d-1)/2)] / (d-1), evaluated through
//    expm1/log1p to avoid cancellation in narrow cells;
//  * conditions (ii) written as F_i(p) = M1_i / M0_i - p_i = 0 and solved by
//    Newton's method with the exact tridiagonal Jacobian
//      d(M1/M0)/d(e_{i+1}) =  g(e_{i+1}) (e_{i+1} - c_i) / M0_i
//      d(M1/M0)/d(e_i)     = -g(e_i)     (e_i     - c_i) / M0_i
//    and de_i/dp_{i-1} = de_i/dp_i = 1/2 (condition (i));
//  * starting point: a few Lloyd steps from Gaussian quantiles of N(0, 1/d).
// The normalising constant of the density cancels in every ratio used.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <limits>

#include "tq_internal.h"

namespace tq {
namespace {

constexpr int kGL = 24;

struct GaussLegendre {
    double x[kGL];
    double w[kGL];
    GaussLegendre() {
        // Nodes by Newton iteration on the Legendre polynomial P_n, starting
        // from the Chebyshev-like guess cos(pi (i + 3/4) / (n + 1/2)).
        const int n = kGL;
        for (int i = 0; i < n; ++i) {
            double z = std::cos(M_PI * (i + 0.75) / (n + 0.5));
            double dp = 0.0;
            for (int it = 0; it < 100; ++it) {
                double p0 = 1.0, p1 = z;
                for (int k = 2; k <= n; ++k) {
                    double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
                    p0 = p1;
                    p1 = p2;
                }
                dp = n * (z * p1 - p0) / (z * z - 1.0);
                double dz = p1 / dp;
                z -= dz;
                if (std::fabs(dz) < 1e-17) break;
            }
            // recompute derivative at the converged node
            double p0 = 1.0, p1 = z;
            for (int k = 2; k <= n; ++k) {
                double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
                p0 = p1;
                p1 = p2;
            }
            dp = n * (z * p1 - p0) / (z * z - 1.0);
            x[i] = z;
            w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
        }
    }
};

const GaussLegendre &gl() {
    static const GaussLegendre g;
    return g;
}

struct Law {
    int d;
    double e3;     // (d-3)/2
    double e1;     // (d-1)/2
    double sigma;  // 1/sqrt(d)
    double g(double x) const {  // unnormalised density
        if (x <= -1.0 || x >= 1.0) return 0.0;
        return std::exp(e3 * std::log1p(-x * x));
    }
    double pw(double x) const {  // (1-x^2)^((d-1)/2)
        if (x <= -1.0 || x >= 1.0) return 0.0;
        return std::exp(e1 * std::log1p(-x * x));
    }
    // int_a^b g, 0 <= a < b <= 1
    double mass(double a, double b) const {
        const double cap = std::min(1.0, a + 40.0 * sigma);
        if (b > cap) b = cap;
        if (b <= a) return 0.0;
        const double panel = 0.25 * sigma;
        int np = (int)std::ceil((b - a) / panel);
        if (np < 1) np = 1;
        const double h = (b - a) / np;
        const GaussLegendre &q = gl();
        double s = 0.0;
        for (int p = 0; p < np; ++p) {
            const double lo = a + p * h;
            const double mid = lo + 0.5 * h;
            double ps = 0.0;
            for (int i = 0; i < kGL; ++i) ps += q.w[i] * g(mid + 0.5 * h * q.x[i]);
            s += 0.5 * h * ps;
        }
        return s;
    }
    // int_a^b x g in closed form, 0 <= a < b <= 1:
    // [(1-a^2)^e1 - (1-b^2)^e1] / (d-1), written as
    // (1-b^2)^e1 * expm1(e1 * log1p((b-a)(b+a)/(1-b^2))) / (d-1)
    // so that narrow cells near 0 do not lose digits to cancellation.
    double moment1(double a, double b) const {
        if (b >= 1.0) return pw(a) / (d - 1.0);
        const double r = (b - a) * (b + a) / ((1.0 - b) * (1.0 + b));
        return pw(b) * std::expm1(e1 * std::log1p(r)) / (d - 1.0);
    }
    // int_a^b x^2 g by quadrature (for the distortion figure only)
    double moment2(double a, double b) const {
        const double cap = std::min(1.0, a + 40.0 * sigma);
        if (b > cap) b = cap;
        if (b <= a) return 0.0;
        const double panel = 0.25 * sigma;
        int np = (int)std::ceil((b - a) / panel);
        if (np < 1) np = 1;
        const double h = (b - a) / np;
        const GaussLegendre &q = gl();
        double s = 0.0;
        for (int p = 0; p < np; ++p) {
            const double mid = a + p * h + 0.5 * h;
            double ps = 0.0;
            for (int i = 0; i < kGL; ++i) {
                double x = mid + 0.5 * h * q.x[i];
                ps += q.w[i] * x * x * g(x);
            }
            s += 0.5 * h * ps;
        }
        return s;
    }
};

// Inverse of the standard normal CDF by Newton's method on erfc.
double norm_ppf(double p) {
    double z = 0.0;
    for (int it = 0; it < 200; ++it) {
        double cdf = 0.5 * std::erfc(-z / std::sqrt(2.0));
        double pdf = std::exp(-0.5 * z * z) / std::sqrt(2.0 * M_PI);
        double dz = (cdf - p) / pdf;
        if (dz > 2.0) dz = 2.0;
        if (dz < -2.0) dz = -2.0;
        z -= dz;
        if (std::fabs(dz) < 1e-15) break;
    }
    return z;
}

void edges_of(const std::vector<double> &p, std::vector<double> *e) {
    const int h = (int)p.size();
    e->assign(h + 1, 0.0);
    (*e)[0] = 0.0;
    for (int i = 1; i < h; ++i) (*e)[i] = 0.5 * (p[i - 1] + p[i]);
    (*e)[h] = 1.0;
}

}  // namespace

bool solve_lloyd_max(int d, int bits, CodebookTables *out) {
    if (d < 3 || bits < 1 || bits > 8) {
        set_error("solve_lloyd_max: bad (d, bits)");
        return false;
    }
    const int L = 1 << bits, h = L / 2;
    Law law{d, 0.5 * (d - 3), 0.5 * (d - 1), 1.0 / std::sqrt((double)d)};
    std::vector<double> p(h), e, c(h), m0(h), F(h);
    for (int i = 0; i < h; ++i) p[i] = law.sigma * norm_ppf((i + h + 0.5) / L);

    auto centroids = [&](const std::vector<double> &pp) {
        edges_of(pp, &e);
        for (int i = 0; i < h; ++i) {
            m0[i] = law.mass(e[i], e[i + 1]);
            c[i] = law.moment1(e[i], e[i + 1]) / m0[i];
        }
    };
    // a few Lloyd steps to settle the start inside Newton's basin
    for (int it = 0; it < 20; ++it) {
        centroids(p);
        p = c;
    }
    // Newton on F(p) = c(p) - p with the tridiagonal Jacobian
    std::vector<double> lo(h), di(h), up(h), rhs(h), best_p = p;
    double best_r = std::numeric_limits<double>::infinity();
    const double tiny = 2.0 * std::numeric_limits<double>::epsilon();
    for (int it = 0; it < 60; ++it) {
        centroids(p);
        double r = 0.0, pmax = 0.0;
        for (int i = 0; i < h; ++i) {
            F[i] = c[i] - p[i];
            r = std::max(r, std::fabs(F[i]));
            pmax = std::max(pmax, std::fabs(p[i]));
        }
        if (r < best_r) {
            best_r = r;
            best_p = p;
        }
        if (r <= tiny * pmax) break;
        if (r > 0.5 * best_r && best_r < 1e-13 * pmax) break;  // rounding floor
        for (int i = 0; i < h; ++i) {
            // derivative of c_i with respect to its lower and upper edges
            const double dlow = (i == 0) ? 0.0 : law.g(e[i]) * (c[i] - e[i]) / m0[i];
            const double dupp = (i == h - 1) ? 0.0 : law.g(e[i + 1]) * (e[i + 1] - c[i]) / m0[i];
            lo[i] = 0.5 * dlow;
            up[i] = 0.5 * dupp;
            di[i] = 0.5 * dlow + 0.5 * dupp - 1.0;
            rhs[i] = -F[i];
        }
        // Thomas algorithm
        for (int i = 1; i < h; ++i) {
            const double m = lo[i] / di[i - 1];
            di[i] -= m * up[i - 1];
            rhs[i] -= m * rhs[i - 1];
        }
        std::vector<double> dx(h);
        dx[h - 1] = rhs[h - 1] / di[h - 1];
        for (int i = h - 2; i >= 0; --i) dx[i] = (rhs[i] - up[i] * dx[i + 1]) / di[i];
        for (int i = 0; i < h; ++i) p[i] += dx[i];
        bool ok = p[0] > 0.0 && p[h - 1] < 1.0;
        for (int i = 1; i < h && ok; ++i) ok = p[i] > p[i - 1];
        if (!ok) {
            set_error("Lloyd-Max Newton iteration left the feasible region");
            return false;
        }
    }
    p = best_p;
    out->d = d;
    out->bits = bits;
    out->cents.assign(L, 0.0);
    out->bounds.assign(L - 1, 0.0);
    for (int i = 0; i < h; ++i) {
        out->cents[h + i] = p[i];
        out->cents[h - 1 - i] = -p[i];
    }
    out->bounds[h - 1] = 0.0;
    for (int i = 1; i < h; ++i) {
        const double m = 0.5 * (p[i - 1] + p[i]);
        out->bounds[h - 1 + i] = m;
        out->bounds[h - 1 - i] = -m;
    }
    // distortion: 2 * sum over positive cells of int (x - c)^2 g / int g
    edges_of(p, &e);
    double num = 0.0, den = 0.0;
    for (int i = 0; i < h; ++i) {
        const double a = e[i], b = e[i + 1];
        const double M0 = law.mass(a, b), M1 = law.moment1(a, b), M2 = law.moment2(a, b);
        num += M2 - 2.0 * p[i] * M1 + p[i] * p[i] * M0;
        den += M0;
    }
    out->mse = num / den;
    return true;
}

}  // namespace tq
