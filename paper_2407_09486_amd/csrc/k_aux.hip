// Bandwidth-bound helper kernels: reference statistics, per-stream scans, flags and the
// radix-select passes of the peaks-over-threshold calibration.
#include <hip/hip_runtime.h>

#include "gpd_math.h"
#include "internal.h"

namespace enova {

namespace {

template <int DT>
__device__ __forceinline__ float load_x(const void *x, int64_t idx)
{
    if constexpr (DT == ENOVA_F32) {
        return static_cast<const float *>(x)[idx];
    } else {
        uint32_t b = static_cast<const uint16_t *>(x)[idx];
        return __uint_as_float(b << 16);
    }
}

__device__ __forceinline__ int64_t ref_len_dev(float ref_frac, int64_t T)
{
    return static_cast<int64_t>(floor(static_cast<double>(ref_frac) * static_cast<double>(T)));
}

__device__ __forceinline__ void finish_stats(double x0, double s1, double s2, int64_t R, float *mean,
                                             float *std)
{
    if (R <= 0) {
        *mean = 0.0f;
        *std = 1.0f;
        return;
    }
    const double inv = 1.0 / static_cast<double>(R);
    const double m1 = s1 * inv;
    const double mu = x0 + m1;
    double var = s2 * inv - m1 * m1;
    var = var > 0.0 ? var : 0.0;
    double sd = sqrt(var);
    if (sd <= 1e-6 * fmax(1.0, fabs(mu)))
        sd = 1.0;   // the metric is constant over the reference prefix
    *mean = static_cast<float>(mu);
    *std = static_cast<float>(sd);
}

// Reference statistics of one stream per block. Values are shifted by the first reference
// value of their metric and accumulated in fp64 (sum and sum of squares), then reduced in a
// fixed order, so the result does not depend on the launch.
template <int DT>
__global__ __launch_bounds__(256) void k_ref_stats(const void *__restrict__ x,
                                                   const int64_t *__restrict__ soff, int M,
                                                   float ref_frac, float *__restrict__ mean,
                                                   float *__restrict__ std)
{
    __shared__ double red1[256];
    __shared__ double red2[256];
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t base = soff[s];
    const int64_t T = soff[s + 1] - base;
    const int64_t R = ref_len_dev(ref_frac, T);

    if (M <= 256 && (256 % M) == 0) {
        const int per = 256 / M;
        const int m = tid % M;
        const int r0 = tid / M;
        const double x0 = R > 0 ? static_cast<double>(load_x<DT>(x, base * M + m)) : 0.0;
        double s1 = 0.0, s2 = 0.0;
        int64_t t = r0;
        for (; t + 3 * per < R; t += 4 * per) {
            const double d0 = static_cast<double>(load_x<DT>(x, (base + t) * M + m)) - x0;
            const double d1 = static_cast<double>(load_x<DT>(x, (base + t + per) * M + m)) - x0;
            const double d2 = static_cast<double>(load_x<DT>(x, (base + t + 2 * per) * M + m)) - x0;
            const double d3 = static_cast<double>(load_x<DT>(x, (base + t + 3 * per) * M + m)) - x0;
            s1 += (d0 + d1) + (d2 + d3);
            s2 += (d0 * d0 + d1 * d1) + (d2 * d2 + d3 * d3);
        }
        for (; t < R; t += per) {
            const double d = static_cast<double>(load_x<DT>(x, (base + t) * M + m)) - x0;
            s1 += d;
            s2 += d * d;
        }
        red1[tid] = s1;
        red2[tid] = s2;
        __syncthreads();
        if (tid < M) {
            double a = 0.0, b = 0.0;
            for (int j = 0; j < per; ++j) {
                a += red1[tid + j * M];
                b += red2[tid + j * M];
            }
            finish_stats(x0, a, b, R, mean + static_cast<int64_t>(s) * M + tid,
                         std + static_cast<int64_t>(s) * M + tid);
        }
    } else {
        for (int m = tid; m < M; m += 256) {
            const double x0 = R > 0 ? static_cast<double>(load_x<DT>(x, base * M + m)) : 0.0;
            double s1 = 0.0, s2 = 0.0;
            for (int64_t t = 0; t < R; ++t) {
                const double d = static_cast<double>(load_x<DT>(x, (base + t) * M + m)) - x0;
                s1 += d;
                s2 += d * d;
            }
            finish_stats(x0, s1, s2, R, mean + static_cast<int64_t>(s) * M + m,
                         std + static_cast<int64_t>(s) * M + m);
        }
    }
}

// Stream of every tile of the matrix-core kernel (one binary search per tile, done once here
// with full occupancy instead of as a chain of dependent loads at the start of each tile).
__global__ __launch_bounds__(256) void k_tile_map(const int64_t *__restrict__ tile_off, int n,
                                                  int64_t grid, int *__restrict__ map)
{
    const int64_t total = tile_off[n];
    for (int64_t b = blockIdx.x * 256LL + threadIdx.x; b < grid; b += static_cast<int64_t>(gridDim.x) * 256) {
        int s = -1;
        if (b < total) {
            int lo = 0, hi = n - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (tile_off[mid] <= b)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            s = lo;
        }
        map[b] = s;
    }
}

// Single-block exclusive scan of a per-stream count.
__global__ __launch_bounds__(1024) void k_stream_scan(const int64_t *__restrict__ soff,
                                                      const int64_t *__restrict__ woff, int n,
                                                      int mode, int div, int W, int S,
                                                      float ref_frac, int64_t *__restrict__ out)
{
    __shared__ int64_t part[1024];
    const int tid = threadIdx.x;
    const int64_t chunk = (static_cast<int64_t>(n) + 1023) / 1024;
    const int64_t a = tid * chunk;
    const int64_t b = a + chunk < n ? a + chunk : n;
    auto count = [&](int64_t s) -> int64_t {
        int64_t c = woff[s + 1] - woff[s];
        if (mode == 1) {
            const int64_t R = ref_len_dev(ref_frac, soff[s + 1] - soff[s]);
            const int64_t cal = R >= W ? (R - W) / S + 1 : 0;
            c = cal < c ? cal : c;
        }
        return div > 1 ? (c + div - 1) / div : c;
    };
    int64_t local = 0;
    for (int64_t s = a; s < b; ++s)
        local += count(s);
    part[tid] = local;
    __syncthreads();
    if (tid == 0) {
        int64_t run = 0;
        for (int i = 0; i < 1024; ++i) {
            const int64_t v = part[i];
            part[i] = run;
            run += v;
        }
        out[n] = run;
    }
    __syncthreads();
    int64_t run = part[tid];
    for (int64_t s = a; s < b; ++s) {
        out[s] = run;
        run += count(s);
    }
}

__global__ void k_flag(const float *__restrict__ scores, int64_t n, float thr,
                       uint8_t *__restrict__ flags)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
        flags[i] = scores[i] > thr ? 1 : 0;
}

// Order-preserving map of a float to an unsigned key.
__device__ __forceinline__ uint32_t fkey(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kCalItems = 16;   // calibration scores per thread per block

// Upper-bound search: the stream s with cal_off[s] <= ci < cal_off[s+1].
__device__ __forceinline__ int find_stream(const int64_t *off, int n, int64_t ci)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (off[mid] <= ci)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

__global__ __launch_bounds__(256) void k_calib_hist(const float *__restrict__ scores,
                                                    const int64_t *__restrict__ woff,
                                                    const int64_t *__restrict__ cal_off, int n,
                                                    int64_t n_cal, int shift,
                                                    const RadixState *__restrict__ rs,
                                                    unsigned int *__restrict__ hist)
{
    __shared__ unsigned int h[256];
    const int tid = threadIdx.x;
    const uint32_t prefix = rs->prefix;
    h[tid] = 0;
    __syncthreads();
    const int64_t start = static_cast<int64_t>(blockIdx.x) * 256 * kCalItems;
    if (start < n_cal) {
        int s = find_stream(cal_off, n, start);
        for (int j = 0; j < kCalItems; ++j) {
            const int64_t ci = start + static_cast<int64_t>(j) * 256 + tid;
            if (ci >= n_cal)
                break;
            while (cal_off[s + 1] <= ci)
                ++s;
            const uint32_t key = fkey(scores[woff[s] + (ci - cal_off[s])]);
            const bool match = shift >= 24 ? true : ((key >> (shift + 8)) == prefix);
            if (match)
                atomicAdd(&h[(key >> shift) & 255u], 1u);
        }
    }
    __syncthreads();
    if (h[tid])
        atomicAdd(&hist[tid], h[tid]);
}

// The radix state's start: no prefix, the sought rank, nothing above; the bins cleared.
__global__ __launch_bounds__(256) void k_radix_init(RadixState *__restrict__ rs, int64_t rank,
                                                    unsigned int *__restrict__ hist)
{
    hist[threadIdx.x] = 0u;
    if (threadIdx.x == 0) {
        rs->prefix = 0u;
        rs->ok = 1;
        rs->rank = rank;
        rs->n_greater = 0;
    }
}

// One block of 256 threads, thread d holding bin d: an inclusive scan of the bins (in 64-bit)
// finds the digit whose range [before, before + count) holds the rank; that thread appends the
// digit to the prefix, keeps rank - before and adds the keys of the higher digits. The bins are
// cleared for the next pass.
__global__ __launch_bounds__(256) void k_radix_pick(RadixState *__restrict__ rs, unsigned int *__restrict__ hist)
{
    __shared__ int64_t wsum[4];
    const int d = threadIdx.x, lane = d & 63, wave = d >> 6;
    const int64_t c = hist[d];
    hist[d] = 0u;
    int64_t inc = c;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int64_t o = __shfl_up(inc, off);
        if (lane >= off)
            inc += o;
    }
    if (lane == 63)
        wsum[wave] = inc;
    __syncthreads();
    int64_t base = 0, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        if (w < wave)
            base += wsum[w];
        total += wsum[w];
    }
    inc += base;
    const int64_t before = inc - c;
    const int64_t rank = rs->rank;
    __syncthreads();
    if (c > 0 && rank >= before && rank < inc) {
        rs->prefix = (rs->prefix << 8) | static_cast<uint32_t>(d);
        rs->rank = rank - before;
        rs->n_greater += total - inc;
    }
    if (d == 0 && !(rank >= 0 && rank < total))
        rs->ok = 0;
}

// Peaks of the calibration set, pass 1: how many keys above key_t each block holds.
__global__ __launch_bounds__(256) void k_calib_count(const float *__restrict__ scores,
                                                     const int64_t *__restrict__ woff,
                                                     const int64_t *__restrict__ cal_off, int n,
                                                     int64_t n_cal, uint32_t key_t,
                                                     int64_t *__restrict__ block_counts)
{
    __shared__ int wsum[4];
    const int tid = threadIdx.x;
    const int64_t start = static_cast<int64_t>(blockIdx.x) * 256 * kCalItems;
    int cnt = 0;
    int s = find_stream(cal_off, n, start);
    for (int j = 0; j < kCalItems; ++j) {
        const int64_t ci = start + static_cast<int64_t>(j) * 256 + tid;
        if (ci >= n_cal)
            break;
        while (cal_off[s + 1] <= ci)
            ++s;
        cnt += fkey(scores[woff[s] + (ci - cal_off[s])]) > key_t ? 1 : 0;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        cnt += __shfl_xor(cnt, off);
    if ((tid & 63) == 0)
        wsum[tid >> 6] = cnt;
    __syncthreads();
    if (tid == 0)
        block_counts[blockIdx.x] = wsum[0] + wsum[1] + wsum[2] + wsum[3];
}

// Pass 2: write the excesses y = score - t of the peaks in calibration order (stable).
__global__ __launch_bounds__(256) void k_calib_compact(const float *__restrict__ scores,
                                                       const int64_t *__restrict__ woff,
                                                       const int64_t *__restrict__ cal_off, int n,
                                                       int64_t n_cal, uint32_t key_t, double t,
                                                       const int64_t *__restrict__ block_off,
                                                       double *__restrict__ y, int64_t cap)
{
    __shared__ int wcnt[4];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t start = static_cast<int64_t>(blockIdx.x) * 256 * kCalItems;
    int64_t run = block_off[blockIdx.x];
    int s = find_stream(cal_off, n, start);
    for (int j = 0; j < kCalItems; ++j) {
        const int64_t ci = start + static_cast<int64_t>(j) * 256 + tid;
        float v = 0.0f;
        bool hit = false;
        if (ci < n_cal) {
            while (cal_off[s + 1] <= ci)
                ++s;
            v = scores[woff[s] + (ci - cal_off[s])];
            hit = fkey(v) > key_t;
        }
        const uint64_t mask = __ballot(hit);
        const int below = __popcll(mask & ((1ull << lane) - 1ull));
        if (lane == 0)
            wcnt[wave] = __popcll(mask);
        __syncthreads();
        int before = 0;
        for (int k = 0; k < wave; ++k)
            before += wcnt[k];
        const int total = wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
        const int64_t pos = run + before + below;
        if (hit && pos < cap)
            y[pos] = static_cast<double>(v) - t;
        run += total;
        __syncthreads();
    }
}

// Exclusive scan of n int64 values by one block; out[n] receives the total.
__global__ __launch_bounds__(1024) void k_scan_i64(const int64_t *__restrict__ in, int64_t n,
                                                   int64_t *__restrict__ out)
{
    __shared__ int64_t part[1024];
    const int tid = threadIdx.x;
    const int64_t chunk = (n + 1023) / 1024;
    const int64_t a = tid * chunk;
    const int64_t b = a + chunk < n ? a + chunk : n;
    int64_t local = 0;
    for (int64_t i = a; i < b; ++i)
        local += in[i];
    part[tid] = local;
    __syncthreads();
    if (tid == 0) {
        int64_t r = 0;
        for (int i = 0; i < 1024; ++i) {
            const int64_t v = part[i];
            part[i] = r;
            r += v;
        }
        out[n] = r;
    }
    __syncthreads();
    int64_t r = part[tid];
    for (int64_t i = a; i < b; ++i) {
        out[i] = r;
        r += in[i];
    }
}

// Wave-wide sum in a fixed butterfly order (every lane ends with the same value).
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        v += __shfl_xor(v, m);
    return v;
}

// Likelihood sums of the excesses: block (g, j) covers chunk j of nsplit contiguous chunks of y
// at the kGpdX points xs[g*kGpdX ...] (each excess is loaded once for all of them) and writes
// pa = sum xy/(1+xy), pb = sum log1p(xy) per point in a fixed order (DER: also pda = sum
// y/(1+xy)^2 and pdb = sum y/(1+xy), their derivatives in x). The terms take the device form
// (hardware reciprocal refined by Newton steps, within a few ulps of the divided form).
constexpr int kGpdX = 8;
template <bool DER>
__global__ __launch_bounds__(256) void k_gpd_sums(const double *__restrict__ y, int64_t n,
                                                  const double *__restrict__ xs, int nx, int nsplit,
                                                  double *__restrict__ pa, double *__restrict__ pb,
                                                  double *__restrict__ pda, double *__restrict__ pdb)
{
    constexpr int NV = DER ? 4 : 2;   // sums per point
    __shared__ double red[4][NV * kGpdX];
    const int grp = blockIdx.x / nsplit;
    const int j = blockIdx.x - grp * nsplit;
    double x[kGpdX];
#pragma unroll
    for (int k = 0; k < kGpdX; ++k) {
        const int i = grp * kGpdX + k;
        x[k] = i < nx ? xs[i] : 0.0;
    }
    const int64_t chunk = (n + nsplit - 1) / nsplit;
    const int64_t lo = j * chunk;
    const int64_t hi = lo + chunk < n ? lo + chunk : n;
    double acc[NV][kGpdX];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int k = 0; k < kGpdX; ++k)
            acc[v][k] = 0.0;
    for (int64_t i = lo + threadIdx.x; i < hi; i += 256) {
        const double yi = y[i];
#pragma unroll
        for (int k = 0; k < kGpdX; ++k) {
            double ta, tb, r;
            gpd_terms_fast(x[k] * yi, ta, tb, r);
            acc[0][k] += ta;
            acc[1][k] += tb;
            if constexpr (DER) {
                const double yr = yi * r;
                acc[2][k] += yr * r;
                acc[3][k] += yr;
            }
        }
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int k = 0; k < kGpdX; ++k)
            acc[v][k] = wave_sum(acc[v][k]);
    if (lane == 0) {
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int k = 0; k < kGpdX; ++k)
                red[wave][v * kGpdX + k] = acc[v][k];
    }
    __syncthreads();
    if (threadIdx.x < NV * kGpdX) {
        const int v = threadIdx.x / kGpdX, k = threadIdx.x - v * kGpdX;
        const int i = grp * kGpdX + k;
        if (i < nx) {
            double *out = v == 0 ? pa : v == 1 ? pb : v == 2 ? pda : pdb;
            const int c = threadIdx.x;
            out[static_cast<int64_t>(i) * nsplit + j] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
        }
    }
}

// Sum, minimum and maximum of the excesses: block j of nblk reduces chunk j (fixed order) into
// part[3j..3j+2]; one block then combines the nblk partials in order.
__global__ __launch_bounds__(256) void k_peak_partial(const double *__restrict__ y, int64_t n,
                                                      double *__restrict__ part)
{
    __shared__ double sa[256];
    __shared__ double sb[256];
    __shared__ double sc[256];
    const int tid = threadIdx.x;
    const int64_t chunk = (n + gridDim.x - 1) / gridDim.x;
    const int64_t lo = blockIdx.x * chunk;
    const int64_t hi = lo + chunk < n ? lo + chunk : n;
    double sum = 0.0, mn = INFINITY, mx = -INFINITY;
    for (int64_t i = lo + tid; i < hi; i += 256) {
        const double v = y[i];
        sum += v;
        mn = fmin(mn, v);
        mx = fmax(mx, v);
    }
    sa[tid] = sum;
    sb[tid] = mn;
    sc[tid] = mx;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if (tid < w) {
            sa[tid] += sa[tid + w];
            sb[tid] = fmin(sb[tid], sb[tid + w]);
            sc[tid] = fmax(sc[tid], sc[tid + w]);
        }
        __syncthreads();
    }
    if (tid == 0) {
        part[3 * blockIdx.x + 0] = sa[0];
        part[3 * blockIdx.x + 1] = sb[0];
        part[3 * blockIdx.x + 2] = sc[0];
    }
}

__global__ __launch_bounds__(64) void k_peak_final(const double *__restrict__ part, int nblk,
                                                   double *__restrict__ out)
{
    if (threadIdx.x != 0)
        return;
    double sum = 0.0, mn = INFINITY, mx = -INFINITY;
    for (int j = 0; j < nblk; ++j) {
        sum += part[3 * j];
        mn = fmin(mn, part[3 * j + 1]);
        mx = fmax(mx, part[3 * j + 2]);
    }
    out[0] = sum;
    out[1] = mn;
    out[2] = mx;
}

}  // namespace

hipError_t launch_ref_stats(const Geometry &g, const void *x, const int64_t *soff, int n,
                            float *mean, float *std, hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    if (g.dtype == ENOVA_F32)
        hipLaunchKernelGGL(k_ref_stats<ENOVA_F32>, dim3(n), dim3(256), 0, st, x, soff, g.M,
                           g.ref_frac, mean, std);
    else
        hipLaunchKernelGGL(k_ref_stats<ENOVA_BF16>, dim3(n), dim3(256), 0, st, x, soff, g.M,
                           g.ref_frac, mean, std);
    return hipGetLastError();
}

hipError_t launch_stream_scan(const Geometry &g, const int64_t *soff, const int64_t *woff, int n,
                              int mode, int div, int64_t *out, hipStream_t st)
{
    hipLaunchKernelGGL(k_stream_scan, dim3(1), dim3(1024), 0, st, soff, woff, n, mode, div, g.W,
                       g.S, g.ref_frac, out);
    return hipGetLastError();
}

hipError_t launch_tile_map(const int64_t *tile_off, int n, int64_t grid, int *map, hipStream_t st)
{
    if (grid <= 0)
        return hipSuccess;
    int64_t blocks = (grid + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    hipLaunchKernelGGL(k_tile_map, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, tile_off, n,
                       grid, map);
    return hipGetLastError();
}

hipError_t launch_flag(const float *scores, int64_t n, float thr, uint8_t *flags, hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    hipLaunchKernelGGL(k_flag, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, scores, n,
                       thr, flags);
    return hipGetLastError();
}

static unsigned cal_blocks(int64_t n_cal)
{
    return static_cast<unsigned>((n_cal + 256 * kCalItems - 1) / (256 * kCalItems));
}

hipError_t launch_radix_init(RadixState *rs, int64_t rank, unsigned int *hist, hipStream_t st)
{
    hipLaunchKernelGGL(k_radix_init, dim3(1), dim3(256), 0, st, rs, rank, hist);
    return hipGetLastError();
}

hipError_t launch_calib_hist(const float *scores, const int64_t *woff, const int64_t *cal_off,
                             int n, int64_t n_cal, int shift, RadixState *rs, unsigned int *hist,
                             hipStream_t st)
{
    if (n_cal <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_calib_hist, dim3(cal_blocks(n_cal)), dim3(256), 0, st, scores, woff,
                       cal_off, n, n_cal, shift, rs, hist);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_radix_pick, dim3(1), dim3(256), 0, st, rs, hist);
    return hipGetLastError();
}

int64_t calib_blocks(int64_t n_cal) { return (n_cal + 256 * kCalItems - 1) / (256 * kCalItems); }

hipError_t launch_calib_count(const float *scores, const int64_t *woff, const int64_t *cal_off, int n,
                              int64_t n_cal, uint32_t key, int64_t *block_counts, hipStream_t st)
{
    if (n_cal <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_calib_count, dim3(cal_blocks(n_cal)), dim3(256), 0, st, scores, woff,
                       cal_off, n, n_cal, key, block_counts);
    return hipGetLastError();
}

hipError_t launch_calib_compact(const float *scores, const int64_t *woff, const int64_t *cal_off,
                                int n, int64_t n_cal, uint32_t key, double t,
                                const int64_t *block_off, double *y, int64_t cap, hipStream_t st)
{
    if (n_cal <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_calib_compact, dim3(cal_blocks(n_cal)), dim3(256), 0, st, scores, woff,
                       cal_off, n, n_cal, key, t, block_off, y, cap);
    return hipGetLastError();
}

hipError_t launch_scan_i64(const int64_t *in, int64_t n, int64_t *out, hipStream_t st)
{
    hipLaunchKernelGGL(k_scan_i64, dim3(1), dim3(1024), 0, st, in, n, out);
    return hipGetLastError();
}

// sa[i] = the chunk partials pa[i*nsplit + j] of point i added by one wave in a fixed order:
// lane l adds the chunks j = l, l + 64, ... in order, then a butterfly adds the lanes; likewise sb
// from pb. Four points per block.
__global__ __launch_bounds__(256) void k_gpd_reduce(const double *__restrict__ pa, const double *__restrict__ pb,
                                                    int nx, int nsplit, double *__restrict__ sa,
                                                    double *__restrict__ sb)
{
    const int i = blockIdx.x * 4 + static_cast<int>(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (i >= nx)
        return;
    const double *a = pa + static_cast<int64_t>(i) * nsplit, *b = pb + static_cast<int64_t>(i) * nsplit;
    double ta = 0.0, tb = 0.0;
    for (int j = lane; j < nsplit; j += 64) {
        ta += a[j];
        tb += b[j];
    }
    ta = wave_sum(ta);
    tb = wave_sum(tb);
    if (lane == 0) {
        sa[i] = ta;
        sb[i] = tb;
    }
}

hipError_t launch_gpd_reduce(const double *pa, const double *pb, int nx, int nsplit, double *sa, double *sb,
                             hipStream_t st)
{
    if (nx <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_gpd_reduce, dim3(static_cast<unsigned>((nx + 3) / 4)), dim3(256), 0, st, pa, pb, nx,
                       nsplit, sa, sb);
    return hipGetLastError();
}

int gpd_split(int64_t n, int nx)
{
    // about 2048 blocks in all (eight per compute unit: the fp64 division and log1p chains need
    // several waves per SIMD to hide their latency), and at least 1024 excesses per chunk
    const int64_t groups = (nx + kGpdX - 1) / kGpdX;
    int64_t s = (2048 + groups - 1) / (groups < 1 ? 1 : groups);
    const int64_t cap = n / 1024;
    if (s > cap)
        s = cap;
    return static_cast<int>(s < 1 ? 1 : s);
}

hipError_t launch_gpd_sums(const double *y, int64_t n, const double *xs, int nx, int nsplit,
                           double *pa, double *pb, double *pda, double *pdb, hipStream_t st)
{
    if (nx <= 0)
        return hipSuccess;
    if ((pda == nullptr) != (pdb == nullptr))
        return hipErrorInvalidValue;
    const unsigned groups = static_cast<unsigned>((nx + kGpdX - 1) / kGpdX);
    if (pda)
        hipLaunchKernelGGL(k_gpd_sums<true>, dim3(groups * nsplit), dim3(256), 0, st, y, n, xs, nx, nsplit, pa, pb,
                           pda, pdb);
    else
        hipLaunchKernelGGL(k_gpd_sums<false>, dim3(groups * nsplit), dim3(256), 0, st, y, n, xs, nx, nsplit, pa,
                           pb, pda, pdb);
    return hipGetLastError();
}

int peak_blocks(int64_t n)
{
    const int64_t b = (n + 8191) / 8192;
    return static_cast<int>(b < 1 ? 1 : (b > kPeakBlocks ? kPeakBlocks : b));
}

hipError_t launch_peak_stats(const double *y, int64_t n, double *out, double *work, hipStream_t st)
{
    const int nblk = peak_blocks(n);
    hipLaunchKernelGGL(k_peak_partial, dim3(nblk), dim3(256), 0, st, y, n, work);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_peak_final, dim3(1), dim3(64), 0, st, work, nblk, out);
    return hipGetLastError();
}

}  // namespace enova
