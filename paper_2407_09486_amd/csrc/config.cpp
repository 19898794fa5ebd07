// Host side of the configuration scans (Section IV-A, Eqs. (4)-(6)): parameter checks, the
// critical value of the slope's t-test, tile bookkeeping and the launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <new>

#include "config_internal.h"
#include "enova_detect.h"

using namespace enova;

namespace enova {

namespace {

// Regularised incomplete beta function I_x(a, b) by its continued fraction (the even/odd terms
// d_2m = m (b - m) x / ((a + 2m - 1)(a + 2m)), d_2m+1 = -(a + m)(a + b + m) x / ((a + 2m)(a + 2m + 1))),
// evaluated with the modified Lentz method; the symmetry I_x(a, b) = 1 - I_{1-x}(b, a) keeps x in
// the region where the fraction converges quickly.
double beta_cf(double a, double b, double x)
{
    const double tiny = 1e-300;
    double c = 1.0, d = 1.0 - (a + b) * x / (a + 1.0);
    if (std::fabs(d) < tiny)
        d = tiny;
    d = 1.0 / d;
    double f = d;
    for (int m = 1; m <= 10000; ++m) {
        const double m2 = 2.0 * m;
        double num = m * (b - m) * x / ((a + m2 - 1.0) * (a + m2));
        d = 1.0 + num * d;
        if (std::fabs(d) < tiny)
            d = tiny;
        c = 1.0 + num / c;
        if (std::fabs(c) < tiny)
            c = tiny;
        d = 1.0 / d;
        f *= d * c;
        num = -(a + m) * (a + b + m) * x / ((a + m2) * (a + m2 + 1.0));
        d = 1.0 + num * d;
        if (std::fabs(d) < tiny)
            d = tiny;
        c = 1.0 + num / c;
        if (std::fabs(c) < tiny)
            c = tiny;
        d = 1.0 / d;
        const double delta = d * c;
        f *= delta;
        if (std::fabs(delta - 1.0) < 1e-16)
            break;
    }
    return f;
}

double inc_beta(double a, double b, double x)
{
    if (x <= 0.0)
        return 0.0;
    if (x >= 1.0)
        return 1.0;
    const double lfront = std::lgamma(a + b) - std::lgamma(a) - std::lgamma(b) + a * std::log(x) + b * std::log1p(-x);
    if (x < (a + 1.0) / (a + b + 2.0))
        return std::exp(lfront) * beta_cf(a, b, x) / a;
    return 1.0 - std::exp(lfront) * beta_cf(b, a, 1.0 - x) / b;
}

}  // namespace

// The two-sided tail of |T| beyond t is I_{nu/(nu+t^2)}(nu/2, 1/2); it increases with that
// argument, so the argument at which it equals alpha is found by bisection and mapped back to t.
double student_t_critical(double alpha, int dof)
{
    const double a = 0.5 * dof, b = 0.5;
    double lo = 0.0, hi = 1.0;
    for (int it = 0; it < 400; ++it) {
        const double mid = 0.5 * (lo + hi);
        if (mid <= lo || mid >= hi)
            break;
        if (inc_beta(a, b, mid) < alpha)
            lo = mid;
        else
            hi = mid;
    }
    const double xs = 0.5 * (lo + hi);
    return std::sqrt(dof * (1.0 - xs) / xs);
}

}  // namespace enova

struct enova_config_s {
    int device = 0;
    CfgParams c{};
    int nb = 0;
    int64_t *tiles = nullptr;
    size_t tiles_cap = 0;
    int *map = nullptr;
    size_t map_cap = 0;
    bool timing = false, timed = false;
    hipEvent_t ev[2] = {nullptr, nullptr};
};

namespace {

template <typename T>
enova_status grow(T **p, size_t *cap, size_t n)
{
    if (n <= *cap)
        return ENOVA_OK;
    (void)hipFree(*p);
    *p = nullptr;
    *cap = 0;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(p), n * sizeof(T));
    if (e != hipSuccess)
        return fail(ENOVA_ENOMEM, "hipMalloc(%zu): %s", n * sizeof(T), hipGetErrorString(e));
    *cap = n;
    return ENOVA_OK;
}

}  // namespace

extern "C" {

enova_status enova_config_t_critical(double alpha, int32_t dof, double *out)
{
    if (!out)
        return fail(ENOVA_EINVAL, "NULL argument");
    if (!(alpha > 0.0 && alpha < 1.0) || dof < 1)
        return fail(ENOVA_EINVAL, "need 0 < alpha < 1 and dof >= 1");
    *out = student_t_critical(alpha, dof);
    return ENOVA_OK;
}

enova_status enova_config_init(const enova_config_params *p, enova_config *out)
{
    if (!p || !out)
        return fail(ENOVA_EINVAL, "NULL argument");
    *out = nullptr;
    if (p->metrics < 1 || p->window < 3 || p->window > 4096 || p->stride < 1)
        return fail(ENOVA_EINVAL, "need M >= 1, 3 <= W <= 4096, S >= 1");
    if (p->dtype != ENOVA_F32 && p->dtype != ENOVA_BF16)
        return fail(ENOVA_EINVAL, "bad dtype");
    const int cols[4] = {p->col_finished, p->col_running, p->col_exec_time, p->col_mem_util};
    for (int c : cols)
        if (c < 0 || c >= p->metrics)
            return fail(ENOVA_EINVAL, "metric column out of range");
    if (!(p->alpha > 0.0 && p->alpha < 1.0) || !(p->q_extreme > 0.0 && p->q_extreme < 1.0))
        return fail(ENOVA_EINVAL, "need 0 < alpha < 1 and 0 < q_extreme < 1");
    CfgParams c{p->metrics,      p->window,      p->stride,        p->dtype,       p->col_finished, p->col_running,
                p->col_exec_time, p->col_mem_util, p->alpha,        p->q_extreme,   0.0};
    c.t_crit = student_t_critical(c.alpha, c.W - 2);
    const int nb = cfg_scan_windows_per_block(c);
    if (nb < 1)
        return fail(ENOVA_EINVAL, "window x stride too large for the scan's staging");
    enova_config h = new (std::nothrow) enova_config_s;
    if (!h)
        return fail(ENOVA_ENOMEM, "host allocation");
    if (hipGetDevice(&h->device) != hipSuccess) {
        delete h;
        return fail(ENOVA_EHIP, "no current HIP device");
    }
    h->c = c;
    h->nb = nb;
    *out = h;
    return ENOVA_OK;
}

enova_status enova_config_destroy(enova_config h)
{
    if (!h)
        return ENOVA_OK;
    DeviceGuard dg(h->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(h->tiles);
    (void)hipFree(h->map);
    for (hipEvent_t e : h->ev)
        if (e)
            (void)hipEventDestroy(e);
    delete h;
    return ENOVA_OK;
}

enova_status enova_config_window_offsets(enova_config h, const int64_t *soff, int32_t n, int64_t *woff)
{
    if (!h || !soff || !woff)
        return fail(ENOVA_EINVAL, "NULL argument");
    if (n < 0)
        return fail(ENOVA_EINVAL, "n_streams < 0");
    if (soff[0] != 0)
        return fail(ENOVA_EINVAL, "stream_offsets[0] must be 0");
    const int64_t W = h->c.W, S = h->c.S;
    woff[0] = 0;
    for (int32_t s = 0; s < n; ++s) {
        const int64_t T = soff[s + 1] - soff[s];
        if (T < 0)
            return fail(ENOVA_EINVAL, "stream_offsets decrease at stream %d", s);
        woff[s + 1] = woff[s] + (T >= W ? (T - W) / S + 1 : 0);
    }
    return ENOVA_OK;
}

enova_status enova_config_scan(enova_config h, const void *x, const int64_t *soff, const int64_t *woff, int32_t n,
                               int64_t n_windows, float *out_a, float *out_b, float *out_t, uint8_t *out_sig,
                               float *out_g0, float *out_g1, hipStream_t stream)
{
    if (!h)
        return fail(ENOVA_EINVAL, "scanner is NULL");
    if (n < 0 || n_windows < 0)
        return fail(ENOVA_EINVAL, "negative sizes");
    h->timed = false;
    if (n == 0 || n_windows == 0)
        return ENOVA_OK;
    if (!x || !soff || !woff)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(h->device);
    Geometry g{};
    g.W = h->c.W;
    g.S = h->c.S;
    enova_status st = grow(&h->tiles, &h->tiles_cap, static_cast<size_t>(n) + 1);
    if (st != ENOVA_OK)
        return st;
    hipError_t e = launch_stream_scan(g, soff, woff, n, 0, h->nb, h->tiles, stream);
    if (e != hipSuccess)
        return hip_fail(e, "tile scan kernel");
    const int64_t grid = (n_windows + h->nb - 1) / h->nb + n;
    if (grid > 0x7fffffffLL)
        return fail(ENOVA_EUNSUPPORTED, "too many tiles");
    if ((st = grow(&h->map, &h->map_cap, static_cast<size_t>(grid))) != ENOVA_OK)
        return st;
    if ((e = launch_tile_map(h->tiles, n, grid, h->map, stream)) != hipSuccess)
        return hip_fail(e, "tile map kernel");
    if (h->timing && (e = hipEventRecord(h->ev[0], stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    const CfgScanOut o{out_a, out_b, out_t, out_sig, out_g0, out_g1};
    if ((e = launch_cfg_scan(h->c, h->nb, x, soff, woff, h->tiles, h->map, grid, o, stream)) != hipSuccess)
        return hip_fail(e, "scan kernel");
    if (h->timing) {
        if ((e = hipEventRecord(h->ev[1], stream)) != hipSuccess)
            return hip_fail(e, "hipEventRecord");
        h->timed = true;
    }
    return ENOVA_OK;
}

enova_status enova_config_recommend(enova_config h, const void *x, const int64_t *soff, int32_t n, uint8_t *out_sig,
                                    double *out_nl, double *out_tl, double *out_mns, double *out_gm,
                                    hipStream_t stream)
{
    if (!h)
        return fail(ENOVA_EINVAL, "scanner is NULL");
    if (n < 0)
        return fail(ENOVA_EINVAL, "n_streams < 0");
    if (n == 0)
        return ENOVA_OK;
    if (!x || !soff)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(h->device);
    const CfgStreamOut o{out_sig, out_nl, out_tl, out_mns, out_gm};
    hipError_t e = launch_cfg_stream(h->c, x, soff, n, o, stream);
    return e == hipSuccess ? ENOVA_OK : hip_fail(e, "configuration kernel");
}

enova_status enova_config_set_timing(enova_config h, int32_t enable)
{
    if (!h)
        return fail(ENOVA_EINVAL, "scanner is NULL");
    DeviceGuard dg(h->device);
    if (enable && !h->ev[0]) {
        for (hipEvent_t &ev : h->ev) {
            hipError_t e = hipEventCreate(&ev);
            if (e != hipSuccess)
                return hip_fail(e, "hipEventCreate");
        }
    }
    h->timing = enable != 0;
    h->timed = false;
    return ENOVA_OK;
}

enova_status enova_config_kernel_time(enova_config h, double *ms)
{
    if (!h || !ms)
        return fail(ENOVA_EINVAL, "NULL argument");
    *ms = 0.0;
    if (!h->timed)
        return ENOVA_OK;
    DeviceGuard dg(h->device);
    hipError_t e = hipEventSynchronize(h->ev[1]);
    float f = 0.0f;
    if (e == hipSuccess)
        e = hipEventElapsedTime(&f, h->ev[0], h->ev[1]);
    if (e != hipSuccess)
        return hip_fail(e, "event timing");
    *ms = f;
    return ENOVA_OK;
}

}  // extern "C"
