// fit_ab.cpp -- host-side fit of the smooth membership curve
// Phi(x) = 1 / (1 + a x^(2b)) to the piecewise target of Eq. 3 (1 up to
// min_dist, exp(-(x - min_dist) / spread) beyond), by damped Gauss-Newton
// with step halving on 300 points of [0, 3 spread].
#include <math.h>

#include "umap_layout.h"
#include "internal.hpp"

namespace {

struct Sample {
    double x, y;
};

double sum_sq(const Sample *s, int m, double a, double b)
{
    double c = 0.0;
    for (int t = 0; t < m; ++t) {
        double phi = s[t].x > 0.0 ? 1.0 / (1.0 + a * pow(s[t].x, 2.0 * b)) : 1.0;
        c += (phi - s[t].y) * (phi - s[t].y);
    }
    return c;
}

}  // namespace

extern "C" int umap_fit_ab(float spread, float min_dist, float *a_out, float *b_out)
{
    if (!a_out || !b_out || !(spread > 0.0f) || !(min_dist >= 0.0f) || !(min_dist < 3.0f * spread) ||
        !isfinite(spread))
        return ul::set_error(UMAP_E_INVAL, "need spread > 0 and 0 <= min_dist < 3 spread, and non-NULL outputs");
    constexpr int M = 300;
    Sample s[M];
    for (int t = 0; t < M; ++t) {
        s[t].x = 3.0 * (double)spread * t / (M - 1);
        s[t].y = s[t].x < min_dist ? 1.0 : exp(-(s[t].x - (double)min_dist) / (double)spread);
    }
    double a = 1.0, b = 1.0;
    double cost = sum_sq(s, M, a, b);
    for (int it = 0; it < 500; ++it) {
        // Jacobian of the residuals with respect to (a, b); both columns vanish at x = 0
        double h11 = 0, h12 = 0, h22 = 0, g1 = 0, g2 = 0;
        for (int t = 0; t < M; ++t) {
            const double x = s[t].x;
            if (!(x > 0.0)) continue;
            const double p = pow(x, 2.0 * b);
            const double q = 1.0 + a * p;
            const double res = 1.0 / q - s[t].y;
            const double ja = -p / (q * q);
            const double jb = -a * p * 2.0 * log(x) / (q * q);
            h11 += ja * ja;
            h12 += ja * jb;
            h22 += jb * jb;
            g1 += ja * res;
            g2 += jb * res;
        }
        const double damp = 1e-12 * (h11 + h22);
        const double det = (h11 + damp) * (h22 + damp) - h12 * h12;
        if (!(det > 0.0)) break;
        double da = -((h22 + damp) * g1 - h12 * g2) / det;
        double db = -((h11 + damp) * g2 - h12 * g1) / det;
        double step = 1.0, next = cost;
        for (int h = 0; h < 60; ++h, step *= 0.5) {
            next = sum_sq(s, M, a + step * da, b + step * db);
            if (next < cost) break;
        }
        if (!(next < cost)) break;
        a += step * da;
        b += step * db;
        const bool small = fabs(step * da) < 1e-12 * fabs(a) && fabs(step * db) < 1e-12 * fabs(b);
        cost = next;
        if (small) break;
    }
    if (!isfinite(a) || !isfinite(b) || a <= 0.0 || b <= 0.0)
        return ul::set_error(UMAP_E_INVAL, "the fit did not converge to positive (a, b)");
    *a_out = (float)a;
    *b_out = (float)b;
    return UMAP_OK;
}
