// General vector-ALU scoring kernel: any window/stride/metric count, H <= 1024, L <= 64.
//
// One block scores 16 consecutive windows (global window order). The normalised inputs are
// staged through LDS 256 columns at a time; each thread owns up to four hidden units of all
// 16 windows and streams the matching rows of the transposed W1. The remaining layers
// (Section IV-B: posterior heads, KL score, decoder mean for the Mean Difference) run on the
// hidden activations kept in LDS.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace enova {

namespace {

constexpr int VB = 16;     // windows per block
constexpr int VDC = 256;   // input columns staged per pass
constexpr int VHPT = 4;    // hidden units per thread (H <= 1024)

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

template <int DT>
__device__ __forceinline__ float load_w(const void *w, int64_t idx)
{
    return load_x<DT>(w, idx);
}

__device__ __forceinline__ float act_fn(float a, int act)
{
    if (act == ENOVA_TANH)
        return tanhf(a);
    return a < 0.0f ? 0.0f : a;   // ReLU; a NaN passes through
}

// e^u - 1 - u without cancellation near 0: Taylor series through u^8 for |u| < 0.5.
__device__ __forceinline__ float kl_g(float u)
{
    if (fabsf(u) < 0.5f) {
        float p = 1.0f / 40320.0f;
        p = p * u + 1.0f / 5040.0f;
        p = p * u + 1.0f / 720.0f;
        p = p * u + 1.0f / 120.0f;
        p = p * u + 1.0f / 24.0f;
        p = p * u + 1.0f / 6.0f;
        p = p * u + 0.5f;
        return (u * u) * p;
    }
    return expm1f(u) - u;
}

__device__ __forceinline__ int find_stream(const int64_t *off, int n, int64_t w)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (off[mid] <= w)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

template <int DT>
__global__ __launch_bounds__(256) void k_score_valu(ScoreParams p, int M, int W, int S, int H,
                                                    int L, int act, float inv_d)
{
    extern __shared__ float sm[];
    const int D = W * M;
    float *vbuf = sm;                       // [VB][VDC]
    float *hbuf = vbuf + VB * VDC;          // [VB][H]
    float *zbuf = hbuf + VB * H;            // [VB][2L]
    float *red = zbuf + VB * 2 * L;         // [VB][256]
    __shared__ int64_t xrow[VB];
    __shared__ int64_t widx[VB];
    __shared__ int sidx[VB];
    __shared__ float vsum_s[VB];
    __shared__ float score_s[VB];

    const int tid = threadIdx.x;
    const int64_t w0 = static_cast<int64_t>(blockIdx.x) * VB;
    if (tid < VB) {
        const int64_t w = w0 + tid;
        if (w < p.n_windows) {
            const int s = find_stream(p.woff, p.n_streams, w);
            const int64_t k = w - p.woff[s];
            xrow[tid] = p.soff[s] + k * S;
            widx[tid] = w;
            sidx[tid] = s;
        } else {
            xrow[tid] = 0;
            widx[tid] = -1;
            sidx[tid] = 0;
        }
    }
    __syncthreads();

    float acc[VB][VHPT];
#pragma unroll
    for (int i = 0; i < VB; ++i)
#pragma unroll
        for (int r = 0; r < VHPT; ++r)
            acc[i][r] = 0.0f;

    const int my_w = tid >> 4;      // the window this thread stages
    const int my_c = tid & 15;
    float vs = 0.0f;
    const bool my_valid = widx[my_w] >= 0;
    const int my_s = sidx[my_w];

    for (int j0 = 0; j0 < D; j0 += VDC) {
        const int nc = D - j0 < VDC ? D - j0 : VDC;
        for (int i = 0; i < VDC / 16; ++i) {
            const int c = my_c + 16 * i;
            float val = 0.0f;
            if (c < nc && my_valid) {
                const int j = j0 + c;
                const int t = j / M;
                const int m = j - t * M;
                const float xv = load_x<DT>(p.x, (xrow[my_w] + t) * M + m);
                const float mu = p.mean[static_cast<int64_t>(my_s) * M + m];
                const float rinv = 1.0f / p.std[static_cast<int64_t>(my_s) * M + m];
                val = (xv - mu) * rinv;
                if constexpr (DT == ENOVA_BF16)
                    val = static_cast<float>(static_cast<__bf16>(val));
                vs += val;
            }
            vbuf[my_w * VDC + c] = val;
        }
        __syncthreads();
        for (int c = 0; c < nc; ++c) {
#pragma unroll
            for (int r = 0; r < VHPT; ++r) {
                const int h = tid + 256 * r;
                if (h < H) {
                    const float wv = load_w<DT>(p.w1t, static_cast<int64_t>(j0 + c) * H + h);
#pragma unroll
                    for (int i = 0; i < VB; ++i)
                        acc[i][r] += wv * vbuf[i * VDC + c];
                }
            }
        }
        __syncthreads();
    }
    // window sums of v: the 16 threads of a window group reduce in a fixed order
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1)
        vs += __shfl_down(vs, off, 16);
    if (my_c == 0)
        vsum_s[my_w] = vs;

    // hidden activations
#pragma unroll
    for (int r = 0; r < VHPT; ++r) {
        const int h = tid + 256 * r;
        if (h < H) {
            const float b = p.b1[h];
#pragma unroll
            for (int i = 0; i < VB; ++i)
                hbuf[i * H + h] = act_fn(acc[i][r] + b, act);
        }
    }
    __syncthreads();
    // posterior heads: mean rows 0..L-1, log-variance rows L..2L-1
    for (int idx = tid; idx < VB * 2 * L; idx += 256) {
        const int i = idx / (2 * L);
        const int o = idx - i * 2 * L;
        const float *wr = o < L ? p.wmu + static_cast<int64_t>(o) * H
                                : p.wlv + static_cast<int64_t>(o - L) * H;
        float a = o < L ? p.bmu[o] : p.blv[o - L];
        for (int h = 0; h < H; ++h)
            a += wr[h] * hbuf[i * H + h];
        zbuf[i * 2 * L + o] = a;
    }
    __syncthreads();
    if (tid < VB) {
        float kl = 0.0f;
        for (int l = 0; l < L; ++l) {
            const float mu = zbuf[tid * 2 * L + l];
            kl += mu * mu + kl_g(zbuf[tid * 2 * L + L + l]);
        }
        score_s[tid] = 0.5f * kl;
    }
    // decoder hidden layer and its dot with the column sums of Wd2
    float part[VB];
#pragma unroll
    for (int i = 0; i < VB; ++i)
        part[i] = 0.0f;
#pragma unroll
    for (int r = 0; r < VHPT; ++r) {
        const int h = tid + 256 * r;
        if (h < H) {
            const float b = p.bd1[h];
            const float uh = p.u[h];
            for (int i = 0; i < VB; ++i) {
                float a = b;
                for (int l = 0; l < L; ++l)
                    a += p.wd1[static_cast<int64_t>(h) * L + l] * zbuf[i * 2 * L + l];
                part[i] += uh * act_fn(a, act);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < VB; ++i)
        red[i * 256 + tid] = part[i];
    __syncthreads();
    if (tid < VB) {
        float dot = 0.0f;
        for (int t = 0; t < 256; ++t)
            dot += red[tid * 256 + t];
        const int64_t w = widx[tid];
        if (w >= 0) {
            const float sc = score_s[tid];
            p.scores[w] = sc;
            if (p.md)
                p.md[w] = vsum_s[tid] * inv_d - (dot + p.sum_bd2) * inv_d;
            if (p.write_flags)
                p.flags[w] = sc > p.threshold ? 1 : 0;
        }
    }
}

}  // namespace

hipError_t launch_score_valu(const Geometry &g, const ScoreParams &p, hipStream_t st)
{
    if (p.n_windows <= 0)
        return hipSuccess;
    const int64_t blocks = (p.n_windows + VB - 1) / VB;
    const size_t lds = sizeof(float) * (VB * VDC + VB * g.H + VB * 2 * g.L + VB * 256);
    const float inv_d = 1.0f / static_cast<float>(g.D);
    if (g.dtype == ENOVA_F32)
        hipLaunchKernelGGL(k_score_valu<ENOVA_F32>, dim3(static_cast<unsigned>(blocks)), dim3(256),
                           lds, st, p, g.M, g.W, g.S, g.H, g.L, g.act, inv_d);
    else
        hipLaunchKernelGGL(k_score_valu<ENOVA_BF16>, dim3(static_cast<unsigned>(blocks)), dim3(256),
                           lds, st, p, g.M, g.W, g.S, g.H, g.L, g.act, inv_d);
    return hipGetLastError();
}

}  // namespace enova
