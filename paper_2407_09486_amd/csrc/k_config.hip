// Configuration scans (Section IV-A, Eqs. (4)-(6)): per-window OLS fits with the slope's t-test,
// and per-stream KDE quantiles of the last window. All statistics in fp64, every reduction in a
// fixed order.
#include <hip/hip_runtime.h>

#include <cmath>

#include "config_internal.h"

namespace enova {

namespace {

constexpr int kCfgThreads = 256;
constexpr int kCfgMaxW = 4096;   // the per-stream kernel holds one window of four columns in LDS (80 KiB at most)
constexpr size_t kCfgScanLds = 48 * 1024;

template <int DT>
__device__ __forceinline__ float load_value(const void *x, int64_t idx)
{
    if constexpr (DT == ENOVA_BF16)
        return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(x)[idx]) << 16);
    else
        return static_cast<const float *>(x)[idx];
}

// One thread per window: two passes over the window's samples in LDS (means, then centred sums).
template <int DT>
__global__ __launch_bounds__(kCfgThreads) void k_cfg_scan(CfgParams c, int nb, const void *__restrict__ x,
                                                          const int64_t *__restrict__ soff,
                                                          const int64_t *__restrict__ woff,
                                                          const int64_t *__restrict__ tile_off,
                                                          const int *__restrict__ tile_stream, CfgScanOut o)
{
    extern __shared__ float sm[];
    const int s = tile_stream[blockIdx.x];
    if (s < 0)
        return;
    const int64_t k0 = (static_cast<int64_t>(blockIdx.x) - tile_off[s]) * nb;
    const int64_t nwin = woff[s + 1] - woff[s];
    const int nw = static_cast<int>(nwin - k0 < nb ? nwin - k0 : nb);
    const int W = c.W, S = c.S, M = c.M;
    const int seg = (nw - 1) * S + W;
    const int pitch = (nb - 1) * S + W;
    float *xr = sm, *xf = sm + pitch, *xm = sm + 2 * pitch;
    const int64_t row0 = soff[s] + k0 * S;
    for (int i = threadIdx.x; i < seg; i += kCfgThreads) {
        const int64_t base = (row0 + i) * M;
        xr[i] = load_value<DT>(x, base + c.col_r);
        xf[i] = load_value<DT>(x, base + c.col_f);
        xm[i] = load_value<DT>(x, base + c.col_m);
    }
    __syncthreads();
    const int w = threadIdx.x;
    if (w >= nw)
        return;
    const float *r = xr + w * S, *f = xf + w * S, *m = xm + w * S;
    double sr = 0.0, sf = 0.0, smu = 0.0;
    for (int j = 0; j < W; ++j) {
        sr += r[j];
        sf += f[j];
        smu += m[j];
    }
    const double rm = sr / W, fm = sf / W, mm = smu / W;
    double sxx = 0.0, sxy = 0.0, syy = 0.0, sxz = 0.0;
    for (int j = 0; j < W; ++j) {
        const double dx = r[j] - rm, dy = f[j] - fm, dz = m[j] - mm;
        sxx = fma(dx, dx, sxx);
        sxy = fma(dx, dy, sxy);
        syy = fma(dy, dy, syy);
        sxz = fma(dx, dz, sxz);
    }
    double a, b, t, g0, g1;
    if (sxx == 0.0) {
        a = fm;
        b = 0.0;
        t = 0.0;
        g0 = mm;
        g1 = 0.0;
    } else {
        b = sxy / sxx;
        a = fm - b * rm;
        const double rss = fmax(syy - b * sxy, 0.0);
        t = b == 0.0 ? 0.0 : (rss == 0.0 ? copysign(HUGE_VAL, b) : b * sqrt((W - 2) * sxx / rss));
        g1 = sxz / sxx;
        g0 = mm - g1 * rm;
    }
    const int64_t out = woff[s] + k0 + w;
    if (o.a)
        o.a[out] = static_cast<float>(a);
    if (o.b)
        o.b[out] = static_cast<float>(b);
    if (o.t)
        o.t[out] = static_cast<float>(t);
    if (o.sig)
        o.sig[out] = fabs(t) > c.t_crit ? 1 : 0;
    if (o.g0)
        o.g0[out] = static_cast<float>(g0);
    if (o.g1)
        o.g1[out] = static_cast<float>(g1);
}

// Fixed-order block sum: a butterfly in each wave, then the four wave sums as (w0 + w1) +
// (w2 + w3); every thread gets the total. Two barriers (a tree over the threads took one per
// level).
static_assert(kCfgThreads == 256, "four waves");
__device__ __forceinline__ double wave_sum_cfg(double v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        v += __shfl_xor(v, m);
    return v;
}

__device__ double block_sum(double v, double *red)
{
    v = wave_sum_cfg(v);
    if ((threadIdx.x & 63) == 0)
        red[threadIdx.x >> 6] = v;
    __syncthreads();
    const double r = (red[0] + red[1]) + (red[2] + red[3]);
    __syncthreads();
    return r;
}

// Two fixed-order block sums at once.
__device__ void block_sum2(double a, double b, double *red, double &ra, double &rb)
{
    a = wave_sum_cfg(a);
    b = wave_sum_cfg(b);
    if ((threadIdx.x & 63) == 0) {
        red[threadIdx.x >> 6] = a;
        red[4 + (threadIdx.x >> 6)] = b;
    }
    __syncthreads();
    ra = (red[0] + red[1]) + (red[2] + red[3]);
    rb = (red[4] + red[5]) + (red[6] + red[7]);
    __syncthreads();
}

// Linearly interpolated sample quantile of sorted v[0..n).
__device__ double sorted_quantile(const float *v, int n, double p)
{
    const double h = (n - 1) * p;
    const int lo = static_cast<int>(floor(h));
    const int hi = lo + 1 < n ? lo + 1 : n - 1;
    return static_cast<double>(v[lo]) + (h - lo) * (static_cast<double>(v[hi]) - static_cast<double>(v[lo]));
}

// Quantile at level q of the Gaussian KDE of v[0..n) (Silverman's bandwidth): the root of its
// distribution function minus q. `sorted` is scratch of np2 floats (np2: a power of two >= n).
__device__ double kde_quantile(const float *v, int n, int np2, double q, float *sorted, double *red)
{
    for (int i = threadIdx.x; i < np2; i += kCfgThreads)
        sorted[i] = i < n ? v[i] : INFINITY;
    __syncthreads();
    // bitonic sort, ascending
    for (int k = 2; k <= np2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < np2; i += kCfgThreads) {
                const int l = i ^ j;
                if (l > i) {
                    const bool up = (i & k) == 0;
                    const float x = sorted[i], y = sorted[l];
                    if ((x > y) == up) {
                        sorted[i] = y;
                        sorted[l] = x;
                    }
                }
            }
            __syncthreads();
        }
    }
    double part = 0.0;
    for (int i = threadIdx.x; i < n; i += kCfgThreads)
        part += v[i];
    const double mean = block_sum(part, red) / n;
    part = 0.0;
    for (int i = threadIdx.x; i < n; i += kCfgThreads) {
        const double d = v[i] - mean;
        part = fma(d, d, part);
    }
    const double ss = block_sum(part, red);
    const double sd = n > 1 ? sqrt(ss / (n - 1)) : 0.0;
    const double iqr = sorted_quantile(sorted, n, 0.75) - sorted_quantile(sorted, n, 0.25);
    const double spread = iqr > 0.0 ? fmin(sd, iqr / 1.34) : sd;
    const double h = 0.9 * spread * pow(static_cast<double>(n), -0.2);
    if (h == 0.0)
        return v[0];
    // Safeguarded Newton on F(x) - q (F' is the KDE density): every evaluation also tightens the
    // bracket [lo, hi], and a step that would leave it becomes a bisection step; stops when the
    // bracket can no longer shrink, the step vanishes, or a Newton step falls below 2^-26 of the
    // bracket's magnitude (taken: quadratic convergence then puts it within rounding of the root,
    // where the sums' rounding noise would otherwise keep the iterates moving).
    double lo = sorted[0] - 10.0 * h, hi = sorted[n - 1] + 10.0 * h;
    const double scale = 1.0 / (h * 1.4142135623730951);
    const double dens = 1.0 / (h * 2.5066282746310002 * n);   // 1 / (h sqrt(2 pi) n)
    double x = 0.5 * (lo + hi);
    for (int it = 0; it < 200; ++it) {
        double pf = 0.0, pd = 0.0;
        for (int i = threadIdx.x; i < n; i += kCfgThreads) {
            const double u = (x - v[i]) * scale;
            pf += 0.5 * erfc(-u);
            pd += exp(-u * u);
        }
        double F, f1;
        block_sum2(pf, pd, red, F, f1);
        F /= n;
        f1 *= dens;
        if (F < q)
            lo = x;
        else
            hi = x;
        double nx = f1 > 0.0 ? x - (F - q) / f1 : 0.5 * (lo + hi);
        const bool newton = nx > lo && nx < hi;
        if (!newton)
            nx = 0.5 * (lo + hi);
        if (nx == x || !(0.5 * (lo + hi) > lo && 0.5 * (lo + hi) < hi))
            break;
        if (newton && fabs(nx - x) <= 0x1p-26 * fmax(fabs(lo), fabs(hi))) {
            x = nx;
            break;
        }
        x = nx;
    }
    return x;
}

// One block per stream: the last window's fits, the regime and the KDE limits.
template <int DT>
__global__ __launch_bounds__(kCfgThreads) void k_cfg_stream(CfgParams c, const void *__restrict__ x,
                                                            const int64_t *__restrict__ soff, CfgStreamOut o)
{
    extern __shared__ float cfg_dyn[];   // four columns of the window [W] each, sort scratch [np2]
    __shared__ double red[2 * kCfgThreads];
    const int s = blockIdx.x;
    const int W = c.W, S = c.S, M = c.M;
    float *vr = cfg_dyn, *vf = vr + W, *vt = vf + W, *vm = vt + W, *sorted = vm + W;
    const int64_t T = soff[s + 1] - soff[s];
    const int64_t nw = T >= W ? (T - W) / S + 1 : 0;
    if (nw == 0) {
        if (threadIdx.x == 0) {
            if (o.sig)
                o.sig[s] = 0;
            if (o.n_limit)
                o.n_limit[s] = NAN;
            if (o.t_limit)
                o.t_limit[s] = NAN;
            if (o.max_num_seqs)
                o.max_num_seqs[s] = NAN;
            if (o.gpu_memory)
                o.gpu_memory[s] = NAN;
        }
        return;
    }
    const int64_t row0 = soff[s] + (nw - 1) * S;
    for (int i = threadIdx.x; i < W; i += kCfgThreads) {
        const int64_t base = (row0 + i) * M;
        vr[i] = load_value<DT>(x, base + c.col_r);
        vf[i] = load_value<DT>(x, base + c.col_f);
        vt[i] = load_value<DT>(x, base + c.col_t);
        vm[i] = load_value<DT>(x, base + c.col_m);
    }
    __syncthreads();
    double p0 = 0.0, p1 = 0.0, p2 = 0.0;
    for (int i = threadIdx.x; i < W; i += kCfgThreads) {
        p0 += vr[i];
        p1 += vf[i];
        p2 += vm[i];
    }
    const double rm = block_sum(p0, red) / W, fm = block_sum(p1, red) / W, mm = block_sum(p2, red) / W;
    double q0 = 0.0, q1 = 0.0, q2 = 0.0, q3 = 0.0;
    for (int i = threadIdx.x; i < W; i += kCfgThreads) {
        const double dx = vr[i] - rm, dy = vf[i] - fm, dz = vm[i] - mm;
        q0 = fma(dx, dx, q0);
        q1 = fma(dx, dy, q1);
        q2 = fma(dy, dy, q2);
        q3 = fma(dx, dz, q3);
    }
    const double sxx = block_sum(q0, red), sxy = block_sum(q1, red), syy = block_sum(q2, red),
                 sxz = block_sum(q3, red);
    double t = 0.0, g0 = mm, g1 = 0.0;
    if (sxx != 0.0) {
        const double b = sxy / sxx;
        const double rss = fmax(syy - b * sxy, 0.0);
        t = b == 0.0 ? 0.0 : (rss == 0.0 ? copysign(HUGE_VAL, b) : b * sqrt((W - 2) * sxx / rss));
        g1 = sxz / sxx;
        g0 = mm - g1 * rm;
    }
    const bool sig = fabs(t) > c.t_crit;
    const double q = sig ? c.q_extreme : 0.5;
    int np2 = 1;
    while (np2 < W)
        np2 <<= 1;
    const double nl = kde_quantile(vf, W, np2, q, sorted, red);
    const double tl = kde_quantile(vt, W, np2, q, sorted, red);
    if (threadIdx.x == 0) {
        const double mns = nl * tl;
        if (o.sig)
            o.sig[s] = sig ? 1 : 0;
        if (o.n_limit)
            o.n_limit[s] = nl;
        if (o.t_limit)
            o.t_limit[s] = tl;
        if (o.max_num_seqs)
            o.max_num_seqs[s] = mns;
        if (o.gpu_memory)
            o.gpu_memory[s] = g0 + g1 * mns;
    }
}

}  // namespace

int cfg_scan_windows_per_block(const CfgParams &c)
{
    for (int nb = kCfgThreads; nb >= 1; nb >>= 1)
        if (cfg_scan_lds_bytes(c, nb) <= kCfgScanLds)
            return nb;
    return 0;
}

size_t cfg_scan_lds_bytes(const CfgParams &c, int nb)
{
    return 3 * sizeof(float) * (static_cast<size_t>(nb - 1) * c.S + c.W);
}

hipError_t launch_cfg_scan(const CfgParams &c, int nb, const void *x, const int64_t *soff, const int64_t *woff,
                           const int64_t *tile_off, const int *tile_stream, int64_t grid, const CfgScanOut &o,
                           hipStream_t st)
{
    if (grid <= 0)
        return hipSuccess;
    const size_t lds = cfg_scan_lds_bytes(c, nb);
    if (c.dtype == ENOVA_BF16)
        hipLaunchKernelGGL(k_cfg_scan<ENOVA_BF16>, dim3(static_cast<unsigned>(grid)), dim3(kCfgThreads), lds, st, c,
                           nb, x, soff, woff, tile_off, tile_stream, o);
    else
        hipLaunchKernelGGL(k_cfg_scan<ENOVA_F32>, dim3(static_cast<unsigned>(grid)), dim3(kCfgThreads), lds, st, c,
                           nb, x, soff, woff, tile_off, tile_stream, o);
    return hipGetLastError();
}

hipError_t launch_cfg_stream(const CfgParams &c, const void *x, const int64_t *soff, int n, const CfgStreamOut &o,
                             hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    if (c.W > kCfgMaxW)
        return hipErrorInvalidValue;
    int np2 = 1;
    while (np2 < c.W)
        np2 <<= 1;
    const size_t lds = sizeof(float) * (4 * static_cast<size_t>(c.W) + np2);
    const void *fn = c.dtype == ENOVA_BF16 ? reinterpret_cast<const void *>(k_cfg_stream<ENOVA_BF16>)
                                           : reinterpret_cast<const void *>(k_cfg_stream<ENOVA_F32>);
    if (lds > 64 * 1024) {   // windows beyond 3276 steps need more than the default dynamic LDS
        const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess)
            return e;
    }
    if (c.dtype == ENOVA_BF16)
        hipLaunchKernelGGL(k_cfg_stream<ENOVA_BF16>, dim3(static_cast<unsigned>(n)), dim3(kCfgThreads), lds, st, c, x,
                           soff, o);
    else
        hipLaunchKernelGGL(k_cfg_stream<ENOVA_F32>, dim3(static_cast<unsigned>(n)), dim3(kCfgThreads), lds, st, c, x,
                           soff, o);
    return hipGetLastError();
}

}  // namespace enova
