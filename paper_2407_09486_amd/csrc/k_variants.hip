// Detector-output variants (Section IV-B): windows materialised in chunks, normalised against the
// reference prefix or against the window itself; the encoder, heads and the decoder's full output
// run as matrix-core products (the training step's GEMM); these kernels are the pieces around
// them: staging, the latent and its KL score, and the per-window reductions of v - m'.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <type_traits>

#include "mfma_common.h"
#include "variants_internal.h"

namespace enova {

namespace {

constexpr int kExtThreads = 256;

template <int DT>
__device__ __forceinline__ float load_value(const void *x, int64_t idx)
{
    if constexpr (DT == ENOVA_BF16)
        return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(x)[idx]) << 16);
    else
        return static_cast<const float *>(x)[idx];
}

// bf16 round to nearest even, returned as the float it represents (NaN kept).
__device__ __forceinline__ float round_bf16(float v)
{
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return v;
    u += 0x7fffu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xffff0000u);
}

// One block per window of the chunk: the window's stream (from k_ext_map), its
// normalisation (reference statistics, or the window's own fp64 mean and population std with the
// reference path's guard), and its D normalised values as row i of V.
// map[i] = the stream of window w0 + i (the last s with woff[s] <= w0 + i), one thread per window:
// the binary searches run in parallel instead of heading every staging block.
__global__ __launch_bounds__(kExtThreads) void k_ext_map(const int64_t *__restrict__ woff, int n, int64_t w0, int rows,
                                                         int *__restrict__ map)
{
    const int i = blockIdx.x * kExtThreads + threadIdx.x;
    if (i >= rows)
        return;
    const int64_t gw = w0 + i;
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (woff[mid] <= gw)
            lo = mid;
        else
            hi = mid - 1;
    }
    map[i] = lo;
}

template <int DT>
__global__ __launch_bounds__(kExtThreads) void k_ext_stage(const void *__restrict__ x, const int64_t *__restrict__ soff,
                                                           const int64_t *__restrict__ woff, const int *__restrict__ map,
                                                           int64_t w0, int M, int W, int S, int norm,
                                                           const float *__restrict__ mean,
                                                           const float *__restrict__ std, float *__restrict__ V)
{
    extern __shared__ float s_norm[];   // mean [M], then 1/std [M]
    float *s_mean = s_norm, *s_rinv = s_norm + M;
    const int64_t gw = w0 + blockIdx.x;
    const int s = map[blockIdx.x];
    const int64_t row0 = soff[s] + (gw - woff[s]) * S;
    if (norm == ENOVA_NORM_WINDOW) {
        // G = 256 / MB threads per metric for a batch of MB = min(M, 256) metrics: thread
        // (g, m) = (tid / MB, tid % MB) takes every G-th step (consecutive threads read
        // consecutive metrics of a step); the G partial sums of a metric are combined in g order
        __shared__ double part[kExtThreads];
        const int MB = M < kExtThreads ? M : kExtThreads;
        const int G = kExtThreads / MB;
        for (int m0 = 0; m0 < M; m0 += MB) {
            const int m = m0 + threadIdx.x % MB, g = threadIdx.x / MB;
            const bool on = g < G && m < M;
            double a = 0.0;
            if (on)
                for (int t = g; t < W; t += G)
                    a += load_value<DT>(x, (row0 + t) * M + m);
            part[threadIdx.x] = a;
            __syncthreads();
            double mu = 0.0;
            if (on) {
                for (int i = 0; i < G; ++i)
                    mu += part[i * MB + threadIdx.x % MB];
                mu /= W;
            }
            __syncthreads();
            double q = 0.0;
            if (on)
                for (int t = g; t < W; t += G) {
                    const double d = load_value<DT>(x, (row0 + t) * M + m) - mu;
                    q = fma(d, d, q);
                }
            part[threadIdx.x] = q;
            __syncthreads();
            if (on && g == 0) {
                double ss = 0.0;
                for (int i = 0; i < G; ++i)
                    ss += part[i * MB + threadIdx.x];
                double sd = sqrt(ss / W);
                if (sd <= 1e-6 * fmax(1.0, fabs(mu)))
                    sd = 1.0;
                s_mean[m] = static_cast<float>(mu);
                s_rinv[m] = 1.0f / static_cast<float>(sd);
            }
            __syncthreads();
        }
    } else {
        for (int m = threadIdx.x; m < M; m += kExtThreads) {
            s_mean[m] = mean[static_cast<int64_t>(s) * M + m];
            s_rinv[m] = 1.0f / std[static_cast<int64_t>(s) * M + m];
        }
        __syncthreads();
    }
    const int D = W * M;
    float *out = V + static_cast<int64_t>(blockIdx.x) * D;
    for (int j = threadIdx.x; j < D; j += kExtThreads) {
        const int t = j / M, m = j - t * M;
        const float v = (load_value<DT>(x, (row0 + t) * M + m) - s_mean[m]) * s_rinv[m];
        out[j] = DT == ENOVA_BF16 ? round_bf16(v) : v;
    }
}

// The same rows as k_ext_stage, one wave per window (four per block, no LDS, no barriers), when
// M is a power of two in [4, 256] and D = 256 Q: lane l holds the 4 Q values
// j = 256 q + 4 l + u (metric (4 l + u) mod M) in registers. The lanes that hold a metric are
// those with equal l mod (M / 4), so a butterfly over the other lane bits completes each metric's
// fp64 sum (then its centred sum of squares) in every lane that needs it.
template <int DT, int Q>
__global__ __launch_bounds__(kExtThreads) void k_ext_stage_wave(const void *__restrict__ x,
                                                                const int64_t *__restrict__ soff,
                                                                const int64_t *__restrict__ woff,
                                                                const int *__restrict__ map, int64_t w0, int rows,
                                                                int M, int W, int S, int norm,
                                                                const float *__restrict__ mean,
                                                                const float *__restrict__ std, float *__restrict__ V)
{
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * (kExtThreads / 64) + static_cast<int>(threadIdx.x >> 6);
    if (i >= rows)
        return;
    const int s = map[i];
    const int64_t row0 = soff[s] + (w0 + i - woff[s]) * S;
    const int64_t base = row0 * M + 4 * lane;
    float v[Q][4];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        if constexpr (DT == ENOVA_BF16) {
            const uint2 p = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(x) + base + 256 * q);
            v[q][0] = __uint_as_float(p.x << 16);
            v[q][1] = __uint_as_float(p.x & 0xffff0000u);
            v[q][2] = __uint_as_float(p.y << 16);
            v[q][3] = __uint_as_float(p.y & 0xffff0000u);
        } else {
            const float4 p = *reinterpret_cast<const float4 *>(static_cast<const float *>(x) + base + 256 * q);
            v[q][0] = p.x;
            v[q][1] = p.y;
            v[q][2] = p.z;
            v[q][3] = p.w;
        }
    }
    float mu[4], ri[4];
    if (norm == ENOVA_NORM_WINDOW) {
        const int g = M / 4;   // lanes l and l ^ (k g) hold the same metrics
        double a[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            a[u] = 0.0;
#pragma unroll
            for (int q = 0; q < Q; ++q)
                a[u] += v[q][u];
        }
        for (int off = g; off < 64; off <<= 1)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                a[u] += __shfl_xor(a[u], off);
        double c[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            a[u] /= W;
            c[u] = 0.0;
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                const double d = v[q][u] - a[u];
                c[u] = fma(d, d, c[u]);
            }
        }
        for (int off = g; off < 64; off <<= 1)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                c[u] += __shfl_xor(c[u], off);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            double sd = sqrt(c[u] / W);
            if (sd <= 1e-6 * fmax(1.0, fabs(a[u])))
                sd = 1.0;
            mu[u] = static_cast<float>(a[u]);
            ri[u] = 1.0f / static_cast<float>(sd);
        }
    } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t e = static_cast<int64_t>(s) * M + ((4 * lane + u) & (M - 1));
            mu[u] = mean[e];
            ri[u] = 1.0f / std[e];
        }
    }
    float *out = V + static_cast<int64_t>(i) * (256 * Q) + 4 * lane;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        float o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            o[u] = (v[q][u] - mu[u]) * ri[u];
            if constexpr (DT == ENOVA_BF16)
                o[u] = round_bf16(o[u]);
        }
        *reinterpret_cast<float4 *>(out + 256 * q) = make_float4(o[0], o[1], o[2], o[3]);
    }
}

// One thread per window: mu and lv (biases [bmu | blv] added in place in ml = [mu | lv]) and
// the KL score of the posterior from N(0, I).
__global__ __launch_bounds__(64) void k_ext_latent(float *__restrict__ ml, const float *__restrict__ bml, int rows,
                                                   int L, float *__restrict__ score)
{
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= rows)
        return;
    float *mu = ml + static_cast<int64_t>(i) * 2 * L, *lv = mu + L;
    float k = 0.0f;
    for (int l = 0; l < L; ++l) {
        const float m = mu[l] + bml[l];
        const float v = lv[l] + bml[L + l];
        mu[l] = m;
        lv[l] = v;
        k += m * m + kl_g(v);
    }
    if (score)
        score[i] = 0.5f * k;
}

// One block per window: d = v - (out + bd2) over the window's D values; per metric the mean of d
// over the W steps, and the window's mean of d and of d^2. Thread (g, m) = (tid / MB, tid % MB)
// sums every G-th step of metric m (MB = min(M, 256), G = 256 / MB); a metric's partials are
// combined in g order, the metrics' totals by a tree.
__global__ __launch_bounds__(kExtThreads) void k_ext_reduce(const float *__restrict__ V, const float *__restrict__ out,
                                                            const float *__restrict__ bd2, int M, int W,
                                                            float *__restrict__ md, float *__restrict__ md_metric,
                                                            float *__restrict__ recon)
{
    __shared__ float pa[kExtThreads], pq[kExtThreads];
    const int D = W * M;
    const float *v = V + static_cast<int64_t>(blockIdx.x) * D;
    const float *o = out + static_cast<int64_t>(blockIdx.x) * D;
    const int MB = M < kExtThreads ? M : kExtThreads;
    const int G = kExtThreads / MB;
    float sd = 0.0f, sq = 0.0f;   // thread g == 0 of a metric: running totals over its metrics
    for (int m0 = 0; m0 < M; m0 += MB) {
        const int m = m0 + threadIdx.x % MB, g = threadIdx.x / MB;
        const bool on = g < G && m < M;
        float a = 0.0f, q = 0.0f;
        if (on)
            for (int t = g; t < W; t += G) {
                const int j = t * M + m;
                const float d = v[j] - (o[j] + bd2[j]);
                a += d;
                q = fmaf(d, d, q);
            }
        pa[threadIdx.x] = a;
        pq[threadIdx.x] = q;
        __syncthreads();
        if (on && g == 0) {
            float ta = 0.0f, tq = 0.0f;
            for (int i = 0; i < G; ++i) {
                ta += pa[i * MB + threadIdx.x];
                tq += pq[i * MB + threadIdx.x];
            }
            if (md_metric)
                md_metric[static_cast<int64_t>(blockIdx.x) * M + m] = ta / W;
            sd += ta;
            sq += tq;
        }
        __syncthreads();
    }
    pa[threadIdx.x] = sd;
    pq[threadIdx.x] = sq;
    __syncthreads();
    for (int w = kExtThreads / 2; w >= 1; w >>= 1) {
        if (threadIdx.x < w) {
            pa[threadIdx.x] += pa[threadIdx.x + w];
            pq[threadIdx.x] += pq[threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (md)
            md[blockIdx.x] = pa[0] / D;
        if (recon)
            recon[blockIdx.x] = pq[0] / D;
    }
}

// The reductions of k_ext_reduce from the partial sums of the decoder-output product's fused
// epilogue: P [rows][slots][M] (sums of d per metric and column slot), Q [rows][slots] (sums of
// d^2). M lanes per window (M a power of two <= 32): lane m adds its metric's slots in order, the
// window's total is a butterfly over the M lanes, and lane 0 adds the squares.
__global__ __launch_bounds__(kExtThreads) void k_ext_finish(const float *__restrict__ P, const float *__restrict__ Q,
                                                            int rows, int slots, int M, int W,
                                                            float *__restrict__ md, float *__restrict__ md_metric,
                                                            float *__restrict__ recon)
{
    const int per = kExtThreads / M;
    const int i = blockIdx.x * per + static_cast<int>(threadIdx.x) / M;
    const int m = threadIdx.x % M;
    const bool on = i < rows;
    float s = 0.0f;
    if (on) {
        const float *p = P + static_cast<int64_t>(i) * slots * M + m;
        for (int k = 0; k < slots; ++k)
            s += p[static_cast<int64_t>(k) * M];
        if (md_metric)
            md_metric[static_cast<int64_t>(i) * M + m] = s / W;
    }
    float t = s;
    for (int off = 1; off < M; off <<= 1)
        t += __shfl_xor(t, off);
    if (on && m == 0) {
        const float D = static_cast<float>(W) * static_cast<float>(M);
        if (md)
            md[i] = t / D;
        if (recon) {
            float q = 0.0f;
            const float *qq = Q + static_cast<int64_t>(i) * slots;
            for (int k = 0; k < slots; ++k)
                q += qq[k];
            recon[i] = q / D;
        }
    }
}

}  // namespace

hipError_t launch_ext_finish(const float *P, const float *Q, int rows, int slots, int M, int W, float *md,
                             float *md_metric, float *recon, hipStream_t st)
{
    if (rows <= 0)
        return hipSuccess;
    if (M < 1 || M > 32 || (M & (M - 1)) != 0)
        return hipErrorInvalidValue;
    const int per = kExtThreads / M;
    hipLaunchKernelGGL(k_ext_finish, dim3(static_cast<unsigned>((rows + per - 1) / per)), dim3(kExtThreads), 0, st, P,
                       Q, rows, slots, M, W, md, md_metric, recon);
    return hipGetLastError();
}

hipError_t launch_ext_stage(const void *x, int dtype, const int64_t *soff, const int64_t *woff, int n, int64_t w0,
                            int rows, int M, int W, int S, int norm, const float *mean, const float *std, int *map,
                            float *V, hipStream_t st)
{
    if (rows <= 0)
        return hipSuccess;
    if (M > kExtMaxM)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_ext_map, dim3(static_cast<unsigned>((rows + kExtThreads - 1) / kExtThreads)),
                       dim3(kExtThreads), 0, st, woff, n, w0, rows, map);
    const int D = W * M;
    const int q = D / 256;
    const bool aligned = reinterpret_cast<uintptr_t>(x) % (dtype == ENOVA_BF16 ? 8 : 16) == 0 &&
                         reinterpret_cast<uintptr_t>(V) % 16 == 0;
    if (aligned && M >= 4 && M <= 256 && (M & (M - 1)) == 0 && D % 256 == 0 && q >= 1 && q <= 8) {
        const dim3 grid(static_cast<unsigned>((rows + kExtThreads / 64 - 1) / (kExtThreads / 64)));
        auto go = [&](auto dt_tag, auto q_tag) {
            constexpr int DT = decltype(dt_tag)::value, QQ = decltype(q_tag)::value;
            hipLaunchKernelGGL((k_ext_stage_wave<DT, QQ>), grid, dim3(kExtThreads), 0, st, x, soff, woff, map, w0,
                               rows, M, W, S, norm, mean, std, V);
        };
        auto by_q = [&](auto dt_tag) {
            switch (q) {
            case 1: go(dt_tag, std::integral_constant<int, 1>{}); break;
            case 2: go(dt_tag, std::integral_constant<int, 2>{}); break;
            case 3: go(dt_tag, std::integral_constant<int, 3>{}); break;
            case 4: go(dt_tag, std::integral_constant<int, 4>{}); break;
            case 5: go(dt_tag, std::integral_constant<int, 5>{}); break;
            case 6: go(dt_tag, std::integral_constant<int, 6>{}); break;
            case 7: go(dt_tag, std::integral_constant<int, 7>{}); break;
            default: go(dt_tag, std::integral_constant<int, 8>{}); break;
            }
        };
        if (dtype == ENOVA_BF16)
            by_q(std::integral_constant<int, ENOVA_BF16>{});
        else
            by_q(std::integral_constant<int, ENOVA_F32>{});
        return hipGetLastError();
    }
    const size_t lds = 2 * sizeof(float) * static_cast<size_t>(M);
    if (dtype == ENOVA_BF16)
        hipLaunchKernelGGL(k_ext_stage<ENOVA_BF16>, dim3(static_cast<unsigned>(rows)), dim3(kExtThreads), lds, st, x,
                           soff, woff, map, w0, M, W, S, norm, mean, std, V);
    else
        hipLaunchKernelGGL(k_ext_stage<ENOVA_F32>, dim3(static_cast<unsigned>(rows)), dim3(kExtThreads), lds, st, x,
                           soff, woff, map, w0, M, W, S, norm, mean, std, V);
    return hipGetLastError();
}

hipError_t launch_ext_latent(float *ml, const float *bml, int rows, int L, float *score, hipStream_t st)
{
    if (rows <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_ext_latent, dim3(static_cast<unsigned>((rows + 63) / 64)), dim3(64), 0, st, ml, bml, rows, L,
                       score);
    return hipGetLastError();
}

hipError_t launch_ext_reduce(const float *V, const float *out, const float *bd2, int rows, int M, int W, float *md,
                             float *md_metric, float *recon, hipStream_t st)
{
    if (rows <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_ext_reduce, dim3(static_cast<unsigned>(rows)), dim3(kExtThreads), 0, st, V, out, bd2, M, W,
                       md, md_metric, recon);
    return hipGetLastError();
}

}  // namespace enova
