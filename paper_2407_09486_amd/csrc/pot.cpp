// Host fp64 fit of the peaks-over-threshold tail (Section IV-B cites Siffer et al. 2017).
//
// The excesses Y over the level-quantile t follow a generalised Pareto distribution
// GPD(gamma, sigma). Maximum likelihood uses Grimshaw's reduction: with x = gamma/sigma the
// score equations collapse to one equation in x,
//     w(x) = u(x) v(x) - 1 = 0,   u = mean 1/(1+xY),   v = 1 + mean log(1+xY),
// whose roots give gamma = v(x) - 1 and sigma = gamma/x. Roots are bracketed on a fixed grid of
// each admissible interval and refined by bisection; the exponential tail (gamma = 0,
// sigma = mean Y) is always a candidate, and the candidate of largest log-likelihood wins.
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "internal.h"

namespace enova {

namespace {

constexpr int kGrid = 512;
constexpr int kBisect = 200;

struct Excess {
    const double *y;
    int64_t n;

    double w(double x) const
    {
        double su = 0.0, sv = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            const double z = 1.0 + x * y[i];
            su += 1.0 / z;
            sv += std::log(z);
        }
        const double u = su / static_cast<double>(n);
        const double v = 1.0 + sv / static_cast<double>(n);
        return u * v - 1.0;
    }

    double loglik(double gamma, double sigma) const
    {
        if (!(sigma > 0.0))
            return -std::numeric_limits<double>::infinity();
        double acc = 0.0;
        if (gamma == 0.0) {
            for (int64_t i = 0; i < n; ++i)
                acc += y[i];
            return -static_cast<double>(n) * std::log(sigma) - acc / sigma;
        }
        for (int64_t i = 0; i < n; ++i) {
            const double z = 1.0 + gamma * y[i] / sigma;
            if (!(z > 0.0))
                return -std::numeric_limits<double>::infinity();
            acc += std::log(z);
        }
        return -static_cast<double>(n) * std::log(sigma) - (1.0 + 1.0 / gamma) * acc;
    }

    double mean_log(double x) const
    {
        double s = 0.0;
        for (int64_t i = 0; i < n; ++i)
            s += std::log(1.0 + x * y[i]);
        return s / static_cast<double>(n);
    }
};

// Roots of w on [a, b]: sign changes between grid points, each bisected.
void roots_on(const Excess &ex, double a, double b, std::vector<double> *out)
{
    if (!(a < b))
        return;
    std::vector<double> xs(kGrid), ws(kGrid);
    for (int i = 0; i < kGrid; ++i) {
        xs[i] = a + (b - a) * static_cast<double>(i) / static_cast<double>(kGrid - 1);
        ws[i] = ex.w(xs[i]);
    }
    for (int i = 0; i + 1 < kGrid; ++i) {
        if (ws[i] == 0.0) {
            out->push_back(xs[i]);
            continue;
        }
        if (!(ws[i] * ws[i + 1] < 0.0))
            continue;
        double lo = xs[i], hi = xs[i + 1], wlo = ws[i];
        for (int it = 0; it < kBisect; ++it) {
            const double mid = 0.5 * (lo + hi);
            if (mid <= lo || mid >= hi)
                break;
            const double wm = ex.w(mid);
            if (wm == 0.0) {
                lo = hi = mid;
                break;
            }
            if ((wm < 0.0) == (wlo < 0.0)) {
                lo = mid;
                wlo = wm;
            } else {
                hi = mid;
            }
        }
        out->push_back(0.5 * (lo + hi));
    }
    if (ws[kGrid - 1] == 0.0)
        out->push_back(xs[kGrid - 1]);
}

void fit_mle(const Excess &ex, double *gamma, double *sigma)
{
    double ysum = 0.0;
    for (int64_t i = 0; i < ex.n; ++i)
        ysum += ex.y[i];
    const double ymean = ysum / static_cast<double>(ex.n);
    const double ymin = ex.y[0], ymax = ex.y[ex.n - 1];   // excesses are sorted ascending
    const double eps = 1e-8 / ymean;
    std::vector<double> roots;
    roots_on(ex, -1.0 / ymax + eps, -eps, &roots);
    const double right = 2.0 * (ymean - ymin) / (ymin * ymin);
    if (right > 2.0 * eps)
        roots_on(ex, eps, right, &roots);
    double bg = 0.0, bs = ymean, bl = ex.loglik(0.0, ymean);
    for (double xr : roots) {
        const double g = ex.mean_log(xr);
        if (g == 0.0)
            continue;
        const double s = g / xr;
        const double ll = ex.loglik(g, s);
        if (ll > bl || (ll == bl && std::fabs(g) < std::fabs(bg))) {
            bg = g;
            bs = s;
            bl = ll;
        }
    }
    *gamma = bg;
    *sigma = bs;
}

}  // namespace

PotResult pot_from_peaks(double t, int64_t n, const double *excess, int64_t n_peaks, double q)
{
    PotResult r{};
    r.t = t;
    r.n = n;
    r.n_peaks = n_peaks;
    r.z = t;
    r.gamma = std::numeric_limits<double>::quiet_NaN();
    r.sigma = std::numeric_limits<double>::quiet_NaN();
    r.method = 0;
    double gamma, sigma;
    if (n_peaks >= 10) {
        fit_mle(Excess{excess, n_peaks}, &gamma, &sigma);
        r.method = 2;
    } else if (n_peaks >= 2) {
        double m = 0.0;
        for (int64_t i = 0; i < n_peaks; ++i)
            m += excess[i];
        m /= static_cast<double>(n_peaks);
        double s2 = 0.0;
        for (int64_t i = 0; i < n_peaks; ++i)
            s2 += (excess[i] - m) * (excess[i] - m);
        s2 /= static_cast<double>(n_peaks - 1);
        if (!(s2 > 0.0))
            return r;
        gamma = 0.5 * (1.0 - m * m / s2);
        sigma = 0.5 * m * (1.0 + m * m / s2);
        r.method = 1;
    } else {
        return r;
    }
    r.gamma = gamma;
    r.sigma = sigma;
    const double ratio = q * static_cast<double>(n) / static_cast<double>(n_peaks);
    if (std::fabs(gamma) < 1e-9)
        r.z = t - sigma * std::log(ratio);
    else
        r.z = t + sigma / gamma * (std::pow(ratio, -gamma) - 1.0);
    return r;
}

}  // namespace enova
