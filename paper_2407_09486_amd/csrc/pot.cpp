// Peaks-over-threshold tail fit (Section IV-B cites Siffer et al. 2017), in fp64.
//
// The excesses Y over the level-quantile t follow a generalised Pareto distribution
// GPD(gamma, sigma). Maximum likelihood uses Grimshaw's reduction: with x = gamma/sigma the
// score equations collapse to one equation in x,
//     u(x) v(x) = 1,   u = mean 1/(1+xY),   v = 1 + mean log(1+xY),
// whose roots give gamma = v(x) - 1 and sigma = gamma/x. It is evaluated without cancellation as
//     w(x) = b - a - a b = 0,   a = mean xY/(1+xY) = 1 - u,   b = mean log1p(xY) = v - 1.
// Roots are bracketed on geometric grids of both admissible intervals: (0, B], B =
// 2 (mean - min) / min^2, which spans many decades once there are many peaks, and
// (-1/Y_max, 0), resolved geometrically towards both ends; each bracket is refined by Newton's
// method kept inside it (all open brackets evaluated in one batch per round, w' from two more
// sums): the first point is the secant of the grid's w at the bracket's ends, a step that lands
// strictly inside is taken, else false position through the ends (Illinois), else the midpoint,
// and a bracket ends once |w| is within the rounding of the sums it is formed from, once the
// step falls below 2^-26 of the point (quadratic convergence then puts the new point within
// rounding of the root; a tighter test only meets the rounding noise of the sums), or when it
// can no longer be split.
// The exponential tail (gamma = 0, sigma = mean Y) is always a candidate, and the candidate of
// largest log-likelihood wins (ties: smaller |gamma|).
//
// The sums over the (possibly millions of) excesses come from a GpdSums evaluator; the
// library's evaluator runs them on the device where the excesses were compacted.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "internal.h"

namespace enova {

namespace {

constexpr int kGrid = 512;       // grid points per admissible interval
constexpr int kRounds = 64;      // evaluations per bracket at most

struct Bracket {
    double lo, hi;
    bool lo_neg;     // sign of w(lo)
    bool done;
    double root;
    double x;        // the point the next round evaluates
    double wlo, whi; // w at the ends (an end kept twice in a row has its w halved: Illinois)
    int side;        // the end the last evaluation replaced (-1 lo, 1 hi, 0 none yet)
};

double w_of(double sa, double sb, double n)
{
    const double a = sa / n, b = sb / n;
    return b - a - a * b;
}

double quantile_z(double t, double gamma, double sigma, double ratio)
{
    if (std::fabs(gamma) < 1e-9)
        return t - sigma * std::log(ratio);
    return t + sigma / gamma * (std::pow(ratio, -gamma) - 1.0);
}

}  // namespace

PotResult pot_small(double t, int64_t n, const double *excess, int64_t n_peaks, double q)
{
    PotResult r{};
    r.t = t;
    r.n = n;
    r.n_peaks = n_peaks;
    r.z = t;
    r.gamma = std::numeric_limits<double>::quiet_NaN();
    r.sigma = std::numeric_limits<double>::quiet_NaN();
    r.method = 0;
    if (n_peaks < 2)
        return r;
    double m = 0.0;
    for (int64_t i = 0; i < n_peaks; ++i)
        m += excess[i];
    m /= static_cast<double>(n_peaks);
    double s2 = 0.0;
    for (int64_t i = 0; i < n_peaks; ++i)
        s2 += (excess[i] - m) * (excess[i] - m);
    s2 /= static_cast<double>(n_peaks - 1);       // unbiased sample variance
    if (!(s2 > 0.0))
        return r;
    r.gamma = 0.5 * (1.0 - m * m / s2);
    r.sigma = 0.5 * m * (1.0 + m * m / s2);
    r.method = 1;
    r.z = quantile_z(t, r.gamma, r.sigma, q * static_cast<double>(n) / static_cast<double>(n_peaks));
    return r;
}

PotResult pot_mle(double t, int64_t n, int64_t n_peaks, double ysum, double ymin, double ymax,
                  double q, GpdSums &sums, bool *ok)
{
    *ok = false;
    PotResult r{};
    r.t = t;
    r.n = n;
    r.n_peaks = n_peaks;
    r.method = 2;
    const double N = static_cast<double>(n_peaks);
    const double ymean = ysum / N;
    const double eps = 1e-8 / ymean;

    // geometric grids over both admissible intervals of x
    std::vector<std::vector<double>> grids;
    const double f0 = eps * ymax;
    if (f0 < 0.5) {
        const double zlo = std::log(f0 / (1.0 - f0)), zhi = 30.0;
        std::vector<double> g(kGrid);
        for (int i = 0; i < kGrid; ++i) {
            const double z = zlo + (zhi - zlo) * static_cast<double>(i) / static_cast<double>(kGrid - 1);
            g[i] = -(1.0 / (1.0 + std::exp(-z))) / ymax;
        }
        grids.push_back(g);
    }
    const double right = 2.0 * (ymean - ymin) / (ymin * ymin);
    if (right > 2.0 * eps) {
        const double ratio = right / eps;
        std::vector<double> g(kGrid);
        for (int i = 0; i < kGrid; ++i)
            g[i] = eps * std::pow(ratio, static_cast<double>(i) / static_cast<double>(kGrid - 1));
        grids.push_back(g);
    }
    std::vector<double> xs, su, sv;
    for (auto &g : grids)
        xs.insert(xs.end(), g.begin(), g.end());
    su.resize(xs.size());
    sv.resize(xs.size());
    if (!xs.empty() && !sums.eval(xs.data(), static_cast<int>(xs.size()), su.data(), sv.data()))
        return r;
    std::vector<double> roots;
    std::vector<Bracket> br;
    for (size_t gi = 0, base = 0; gi < grids.size(); ++gi) {
        for (int i = 0; i < kGrid; ++i) {
            const double wi = w_of(su[base + i], sv[base + i], N);
            if (wi == 0.0) {
                roots.push_back(xs[base + i]);
                continue;
            }
            if (i + 1 < kGrid) {
                const double wn = w_of(su[base + i + 1], sv[base + i + 1], N);
                if (wi * wn < 0.0) {
                    const double x0 = xs[base + i], x1 = xs[base + i + 1];
                    // keep lo < hi; lo_neg is the sign of w at lo; start at the secant point
                    const double lo = x0 < x1 ? x0 : x1, hi = x0 < x1 ? x1 : x0;
                    const double xsec = x0 - wi * (x1 - x0) / (wn - wi);
                    const double x = xsec > lo && xsec < hi ? xsec : 0.5 * (lo + hi);
                    br.push_back({lo, hi, x0 < x1 ? wi < 0.0 : wn < 0.0, false, 0.0, x, x0 < x1 ? wi : wn,
                                  x0 < x1 ? wn : wi, 0});
                }
            }
        }
        base += kGrid;
    }
    // Newton's method inside every open bracket, batched
    std::vector<double> sda, sdb;
    std::vector<int> evals(br.size(), 0);
    for (int round = 0; round < kRounds; ++round) {
        xs.clear();
        std::vector<int> owner;
        for (size_t b = 0; b < br.size(); ++b)
            if (!br[b].done) {
                xs.push_back(br[b].x);
                owner.push_back(static_cast<int>(b));
            }
        if (xs.empty())
            break;
        su.assign(xs.size(), 0.0);
        sv.assign(xs.size(), 0.0);
        sda.assign(xs.size(), 0.0);
        sdb.assign(xs.size(), 0.0);
        if (!sums.eval_d(xs.data(), static_cast<int>(xs.size()), su.data(), sv.data(), sda.data(), sdb.data()))
            return r;
        for (size_t i = 0; i < xs.size(); ++i) {
            Bracket &k = br[owner[i]];
            const double x = xs[i];
            const double a = su[i] / N, b = sv[i] / N, da = sda[i] / N, db = sdb[i] / N;
            const double wv = b - a - a * b;
            const double wd = db - da - da * b - a * db;
            if (wv == 0.0) {
                k.done = true;
                k.root = x;
                continue;
            }
            const int side = (wv < 0.0) == k.lo_neg ? -1 : 1;
            if (side < 0) {
                k.lo = x;
                k.wlo = wv;
                if (k.side < 0)
                    k.whi *= 0.5;
            } else {
                k.hi = x;
                k.whi = wv;
                if (k.side > 0)
                    k.wlo *= 0.5;
            }
            k.side = side;
            const double xn = x - wv / wd;
            const bool inside = xn > k.lo && xn < k.hi;     // false for NaN
            // when the Newton step leaves the bracket: false position through the ends, else the
            // midpoint
            const double xf = k.lo - k.wlo * (k.hi - k.lo) / (k.whi - k.wlo);
            const double mid = xf > k.lo && xf < k.hi ? xf : 0.5 * (k.lo + k.hi);
            const double tol = 0x1p-26 * std::max(std::fabs(k.lo), std::fabs(k.hi));
            // |w| within the rounding of the sums it is formed from: x is a root to fp64 resolution
            if (std::fabs(wv) <= 0x1p-46 * (std::fabs(b) + std::fabs(a) + std::fabs(a * b))) {
                k.done = true;
                k.root = x;
            } else if (inside && std::fabs(xn - x) <= tol) {
                k.done = true;
                k.root = xn;
            } else if (!inside && !(mid > k.lo && mid < k.hi)) {
                k.done = true;
                k.root = mid;
            } else if (++evals[owner[i]] >= kRounds) {
                k.done = true;
                k.root = inside ? xn : mid;
            } else {
                k.x = inside ? xn : mid;
            }
        }
    }
    for (auto &k : br)
        roots.push_back(k.done ? k.root : 0.5 * (k.lo + k.hi));

    // candidates: the exponential tail and every root
    double bg = 0.0, bs = ymean;
    double bl = -N * std::log(ymean) - ysum / ymean;
    if (!roots.empty()) {
        su.assign(roots.size(), 0.0);
        sv.assign(roots.size(), 0.0);
        if (!sums.eval(roots.data(), static_cast<int>(roots.size()), su.data(), sv.data()))
            return r;
        for (size_t i = 0; i < roots.size(); ++i) {
            const double g = sv[i] / N;
            if (g == 0.0 || !std::isfinite(g))
                continue;
            const double s = g / roots[i];
            if (!(s > 0.0))
                continue;
            const double ll = -N * std::log(s) - (1.0 + 1.0 / g) * sv[i];   // sum log1p(g y / s) = sv
            if (ll > bl || (ll == bl && std::fabs(g) < std::fabs(bg))) {
                bg = g;
                bs = s;
                bl = ll;
            }
        }
    }
    r.gamma = bg;
    r.sigma = bs;
    r.z = quantile_z(t, bg, bs, q * static_cast<double>(n) / N);
    *ok = true;
    return r;
}

}  // namespace enova
