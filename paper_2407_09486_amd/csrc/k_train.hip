// Training kernels (Section IV-B, Eq. (9)): a general fp32 matrix-core GEMM for the forward and
// backward products of the VAE over a batch of windows, and the element-wise pieces around them
// (bias + activation, the reparameterised latent and its KL, the reconstruction term and its
// gradient, the PI-controlled KL weight, the latent gradients, activation derivatives, bias
// gradients and the Adam update). Every reduction runs in a fixed order, so a step is
// deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "internal.h"
#include "mfma_common.h"

namespace enova {

namespace {

constexpr int kGemmTile = 64;   // C tile of a block (2 x 2 waves of 32 x 32)
constexpr int kGemmK = 32;      // reduction slice staged in LDS
constexpr int kGemmPitch = kGemmTile + 4;
constexpr int kGemmTargetBlocks = 1024;   // split the reduction until a launch has about this many blocks
constexpr int kGemmMinSlice = 256;        // ... but keep every slice at least this long
constexpr int kGemmMaxSplits = 64;
constexpr int kColsumRows = 128;         // rows per block of a column sum ...
constexpr int kColsumMaxChunks = 64;     // ... in at most this many row chunks
constexpr float kLog2Pi = 1.8378770664093453f;   // log(2 pi)

// C(i, j) [+]= sum_k A(i, k) B(k, j) with A(i, k) = A[i*ai + k*ak], B(k, j) = B[k*bk + j*bj],
// C(i, j) = C[i*ldc + j]; i < m, j < n, k < kk. Two accumulator chains (even and odd k pairs)
// keep the matrix ops of a wave independent; they are added at the end.
// blockIdx.z takes the reduction slice [z kc, min(kk, (z + 1) kc)); with several slices each
// writes its own partial tile to C + z * m * ldc (summed afterwards by k_sum_splits).
template <bool ACC>
__global__ __launch_bounds__(256) void k_gemm(const float *__restrict__ A, int64_t ai, int64_t ak,
                                              const float *__restrict__ B, int64_t bk, int64_t bj,
                                              float *__restrict__ C, int64_t ldc, int m, int n, int kk, int kc)
{
    const int kbeg = blockIdx.z * kc;
    const int kend = min(kk, kbeg + kc);
    C += static_cast<int64_t>(blockIdx.z) * m * ldc;
    __shared__ float As[kGemmK][kGemmPitch];
    __shared__ float Bs[kGemmK][kGemmPitch];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wy = wave >> 1, wx = wave & 1;
    const int64_t i0 = static_cast<int64_t>(blockIdx.y) * kGemmTile;
    const int64_t j0 = static_cast<int64_t>(blockIdx.x) * kGemmTile;
    v16f acc0, acc1;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        acc0[r] = 0.0f;
        acc1[r] = 0.0f;
    }
    for (int k0 = kbeg; k0 < kend; k0 += kGemmK) {
        // stage both tiles, walking the operand's unit-stride index fastest (coalesced reads)
        for (int e = tid; e < kGemmTile * kGemmK; e += 256) {
            int ii, kx;
            if (ak == 1) {
                kx = e % kGemmK;
                ii = e / kGemmK;
            } else {
                ii = e % kGemmTile;
                kx = e / kGemmTile;
            }
            const int64_t gi = i0 + ii, gk = k0 + kx;
            As[kx][ii] = (gi < m && gk < kend) ? A[gi * ai + gk * ak] : 0.0f;
            int jj, ky;
            if (bj == 1) {
                jj = e % kGemmTile;
                ky = e / kGemmTile;
            } else {
                ky = e % kGemmK;
                jj = e / kGemmK;
            }
            const int64_t gj = j0 + jj, gk2 = k0 + ky;
            Bs[ky][jj] = (gj < n && gk2 < kend) ? B[gk2 * bk + gj * bj] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kp = 0; kp < kGemmK; kp += 4) {
            const float a0 = As[kp + (lane >> 5)][wy * 32 + (lane & 31)];
            const float b0 = Bs[kp + (lane >> 5)][wx * 32 + (lane & 31)];
            const float a1 = As[kp + 2 + (lane >> 5)][wy * 32 + (lane & 31)];
            const float b1 = Bs[kp + 2 + (lane >> 5)][wx * 32 + (lane & 31)];
            acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc1, 0, 0, 0);
        }
        __syncthreads();
    }
    const int half = lane >> 5;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int64_t gi = i0 + wy * 32 + crow(r, half);
        const int64_t gj = j0 + wx * 32 + (lane & 31);
        if (gi < m && gj < n) {
            const float v = acc0[r] + acc1[r];
            C[gi * ldc + gj] = ACC ? C[gi * ldc + gj] + v : v;
        }
    }
}

// C(i, j) [+]= sum over the slices s = 0, 1, ... (in order) of P[s][i][j].
template <bool ACC>
__global__ __launch_bounds__(256) void k_sum_splits(const float *__restrict__ P, int splits, int m, int n,
                                                    float *__restrict__ C, int64_t ldc)
{
    const int64_t total = static_cast<int64_t>(m) * n;
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
        float v = 0.0f;
        for (int sp = 0; sp < splits; ++sp)
            v += P[sp * total + e];
        const int64_t i = e / n, j = e % n;
        C[i * ldc + j] = ACC ? C[i * ldc + j] + v : v;
    }
}

template <int ACT>
__device__ __forceinline__ float dact(float a)
{
    if constexpr (ACT == ENOVA_TANH) {
        const float t = tanhf(a);
        return 1.0f - t * t;
    } else {
        return a > 0.0f ? 1.0f : 0.0f;
    }
}

// pre[i][j] += bias[j]; out[i][j] = act(pre[i][j])
template <int ACT>
__global__ __launch_bounds__(256) void k_bias_act(float *__restrict__ pre, const float *__restrict__ bias,
                                                  float *__restrict__ out, int64_t rows, int cols)
{
    const int64_t total = rows * cols;
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
        const float a = pre[e] + bias[e % cols];
        pre[e] = a;
        out[e] = act_fn<ACT>(a);
    }
}

// g[e] *= act'(pre[e])
template <int ACT>
__global__ __launch_bounds__(256) void k_dact(float *__restrict__ g, const float *__restrict__ pre, int64_t total)
{
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256)
        g[e] *= dact<ACT>(pre[e]);
}

// One thread per window: mu, lv (biases added in place), sd = e^(lv/2), z = mu + sd eps and the
// KL of q(z|m) from N(0, I).
__global__ __launch_bounds__(256) void k_latent(float *__restrict__ mu, float *__restrict__ lv,
                                                const float *__restrict__ bmu, const float *__restrict__ blv,
                                                const float *__restrict__ eps, float *__restrict__ sd,
                                                float *__restrict__ z, float *__restrict__ kl, int rows, int L)
{
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= rows)
        return;
    float k = 0.0f;
    for (int l = 0; l < L; ++l) {
        const int64_t e = static_cast<int64_t>(i) * L + l;
        const float m = mu[e] + bmu[l];
        const float v = lv[e] + blv[l];
        const float s = expf(0.5f * v);
        mu[e] = m;
        lv[e] = v;
        sd[e] = s;
        z[e] = m + s * eps[e];
        k += m * m + kl_g(v);
    }
    kl[i] = 0.5f * k;
}

// One block per window: m' = out + bd2, e = |v - m'|^2 / 2, log p = -e - D/2 log 2 pi, and in place
// of out the gradient of J, (l/B)(m' - v); an anomalous window (l < 0) whose e has reached the
// margin contributes a constant and gets a zero gradient.
__global__ __launch_bounds__(256) void k_recon(float *__restrict__ out, const float *__restrict__ bd2,
                                               const float *__restrict__ V, const float *__restrict__ labels,
                                               float *__restrict__ logp, int D, float inv_b, float margin)
{
    __shared__ float red[256];
    const int64_t row = blockIdx.x;
    const float l = labels[row];
    float sq = 0.0f;
    for (int j = threadIdx.x; j < D; j += 256) {
        const int64_t e = row * D + j;
        const float d = out[e] + bd2[j] - V[e];
        sq += d * d;
    }
    red[threadIdx.x] = sq;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if (threadIdx.x < w)
            red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const float err = 0.5f * red[0];
    const float scale = (l > 0.0f || err < margin) ? l * inv_b : 0.0f;
    for (int j = threadIdx.x; j < D; j += 256) {
        const int64_t e = row * D + j;
        out[e] = scale * (out[e] + bd2[j] - V[e]);
    }
    if (threadIdx.x == 0)
        logp[row] = -err - 0.5f * static_cast<float>(D) * kLog2Pi;
}

// One block: the KL weight of this step from the PI controller, and the step's summary
// (J, mean log p, mean KL of the normal windows, beta). State: st[0] = the integral term.
// An anomalous window enters J through -log p capped at margin + D/2 log 2 pi.
__global__ __launch_bounds__(256) void k_beta(const float *__restrict__ kl, const float *__restrict__ logp,
                                              const float *__restrict__ labels, int rows, float kl_set,
                                              float kp, float ki, float beta_min, float beta_max,
                                              float margin, float half_d_log2pi,
                                              float *__restrict__ st, float *__restrict__ beta_out,
                                              float *__restrict__ info)
{
    __shared__ double r_kl[256], r_n[256], r_lp[256], r_la[256], r_kn[256];
    double skl = 0.0, sn = 0.0, slp = 0.0, sla = 0.0, skn = 0.0;
    for (int i = threadIdx.x; i < rows; i += 256) {
        const double l = labels[i];
        const double k = kl[i];
        const double lp = logp[i];
        if (l > 0.0) {
            skl += k;
            sn += 1.0;
        }
        slp += lp;
        if (l < 0.0) {
            // anomalous: -log p capped at margin + D/2 log 2 pi
            const double err = -lp - static_cast<double>(half_d_log2pi);
            sla += (err < margin ? err : static_cast<double>(margin)) + static_cast<double>(half_d_log2pi);
        } else {
            sla += l * lp;
        }
        skn += 0.5 * (1.0 + l) * k;
    }
    r_kl[threadIdx.x] = skl;
    r_n[threadIdx.x] = sn;
    r_lp[threadIdx.x] = slp;
    r_la[threadIdx.x] = sla;
    r_kn[threadIdx.x] = skn;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if (threadIdx.x < w) {
            r_kl[threadIdx.x] += r_kl[threadIdx.x + w];
            r_n[threadIdx.x] += r_n[threadIdx.x + w];
            r_lp[threadIdx.x] += r_lp[threadIdx.x + w];
            r_la[threadIdx.x] += r_la[threadIdx.x + w];
            r_kn[threadIdx.x] += r_kn[threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double mkl = r_n[0] > 0.0 ? r_kl[0] / r_n[0] : 0.0;
        const double e = static_cast<double>(kl_set) - mkl;
        const double integ = static_cast<double>(st[0]) - static_cast<double>(ki) * e;
        const double p = e < 700.0 ? static_cast<double>(kp) / (1.0 + exp(e)) : 0.0;
        double b = p + integ + static_cast<double>(beta_min);
        b = b < beta_min ? beta_min : (b > beta_max ? beta_max : b);
        st[0] = static_cast<float>(integ);
        beta_out[0] = static_cast<float>(b);
        if (info) {
            info[0] = static_cast<float>(-(r_la[0] - b * r_kn[0]) / rows);
            info[1] = static_cast<float>(r_lp[0] / rows);
            info[2] = static_cast<float>(mkl);
            info[3] = static_cast<float>(b);
        }
    }
}

// Gradients of J at the latent: g_mu = g_z + c mu, g_lv = g_z eps sd/2 + c (e^lv - 1)/2 with
// c = (1 + l)/2 beta / B; g_z holds dJ/dz on entry and g_mu on exit.
__global__ __launch_bounds__(256) void k_latent_grad(float *__restrict__ gz, float *__restrict__ glv,
                                                     const float *__restrict__ mu, const float *__restrict__ lv,
                                                     const float *__restrict__ sd, const float *__restrict__ eps,
                                                     const float *__restrict__ labels,
                                                     const float *__restrict__ beta, int rows, int L, float inv_b)
{
    const int64_t total = static_cast<int64_t>(rows) * L;
    const float b = beta[0];
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t i = e / L;
        const float c = 0.5f * (1.0f + labels[i]) * b * inv_b;
        const float g = gz[e];
        gz[e] = g + c * mu[e];
        glv[e] = g * eps[e] * 0.5f * sd[e] + c * 0.5f * expm1f(lv[e]);
    }
}

// Column sums in two fixed-order passes: block (x, r) sums rows [r rc, (r + 1) rc) of 64 columns
// (4 row lanes of 64 threads, combined in lane order) into P[r][j]; k_sum_splits then adds the
// row chunks in order.
__global__ __launch_bounds__(256) void k_colsum_part(const float *__restrict__ X, int64_t rows, int cols,
                                                     int64_t rc, float *__restrict__ P)
{
    __shared__ float part[4][64];
    const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int j = blockIdx.x * 64 + c;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * rc;
    const int64_t r1 = r0 + rc < rows ? r0 + rc : rows;
    float s = 0.0f;
    if (j < cols)
        for (int64_t i = r0 + q; i < r1; i += 4)
            s += X[i * cols + j];
    part[q][c] = s;
    __syncthreads();
    if (q == 0 && j < cols)
        P[static_cast<int64_t>(blockIdx.y) * cols + j] = ((part[0][c] + part[1][c]) + part[2][c]) + part[3][c];
}

__global__ __launch_bounds__(256) void k_adam(float *__restrict__ p, const float *__restrict__ g,
                                              float *__restrict__ m, float *__restrict__ v, int64_t total,
                                              float lr, float b1, float b2, float eps, float c1, float c2)
{
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
        const float ge = g[e];
        const float me = b1 * m[e] + (1.0f - b1) * ge;
        const float ve = b2 * v[e] + (1.0f - b2) * ge * ge;
        m[e] = me;
        v[e] = ve;
        p[e] -= lr * (me * c1) / (sqrtf(ve * c2) + eps);
    }
}

unsigned blocks_for(int64_t total)
{
    int64_t b = (total + 255) / 256;
    return static_cast<unsigned>(b < 1 ? 1 : (b > 65536 ? 65536 : b));
}

}  // namespace

static int gemm_splits(int m, int n, int k)
{
    const int64_t tiles = static_cast<int64_t>((m + kGemmTile - 1) / kGemmTile) * ((n + kGemmTile - 1) / kGemmTile);
    if (tiles >= kGemmTargetBlocks / 2)
        return 1;
    const int by_k = (k + kGemmMinSlice - 1) / kGemmMinSlice;
    const int by_grid = static_cast<int>((kGemmTargetBlocks + tiles - 1) / tiles);
    return std::max(1, std::min({by_k, by_grid, kGemmMaxSplits}));
}

int64_t gemm_workspace_floats(int m, int n, int k)
{
    const int s = gemm_splits(m, n, k);
    return s > 1 ? static_cast<int64_t>(s) * m * n : 0;
}

hipError_t launch_gemm(const float *A, int64_t ai, int64_t ak, const float *B, int64_t bk, int64_t bj,
                       float *C, int64_t ldc, int m, int n, int k, bool accumulate, float *work, hipStream_t st)
{
    if (m <= 0 || n <= 0)
        return hipSuccess;
    const int splits = work ? gemm_splits(m, n, k) : 1;
    const int kc = splits > 1 ? ((k + splits - 1) / splits + kGemmK - 1) / kGemmK * kGemmK : std::max(k, 1);
    const int used = splits > 1 ? (k + kc - 1) / kc : 1;
    const dim3 grid(static_cast<unsigned>((n + kGemmTile - 1) / kGemmTile),
                    static_cast<unsigned>((m + kGemmTile - 1) / kGemmTile), static_cast<unsigned>(used));
    if (used > 1) {
        hipLaunchKernelGGL(k_gemm<false>, grid, dim3(256), 0, st, A, ai, ak, B, bk, bj, work,
                           static_cast<int64_t>(n), m, n, k, kc);
        const unsigned b = blocks_for(static_cast<int64_t>(m) * n);
        if (accumulate)
            hipLaunchKernelGGL(k_sum_splits<true>, dim3(b), dim3(256), 0, st, work, used, m, n, C, ldc);
        else
            hipLaunchKernelGGL(k_sum_splits<false>, dim3(b), dim3(256), 0, st, work, used, m, n, C, ldc);
    } else if (accumulate) {
        hipLaunchKernelGGL(k_gemm<true>, grid, dim3(256), 0, st, A, ai, ak, B, bk, bj, C, ldc, m, n, k, kc);
    } else {
        hipLaunchKernelGGL(k_gemm<false>, grid, dim3(256), 0, st, A, ai, ak, B, bk, bj, C, ldc, m, n, k, kc);
    }
    return hipGetLastError();
}

hipError_t launch_bias_act(float *pre, const float *bias, float *out, int64_t rows, int cols, int act,
                           hipStream_t st)
{
    const unsigned b = blocks_for(rows * cols);
    if (act == ENOVA_TANH)
        hipLaunchKernelGGL(k_bias_act<ENOVA_TANH>, dim3(b), dim3(256), 0, st, pre, bias, out, rows, cols);
    else
        hipLaunchKernelGGL(k_bias_act<ENOVA_RELU>, dim3(b), dim3(256), 0, st, pre, bias, out, rows, cols);
    return hipGetLastError();
}

hipError_t launch_dact(float *g, const float *pre, int64_t total, int act, hipStream_t st)
{
    const unsigned b = blocks_for(total);
    if (act == ENOVA_TANH)
        hipLaunchKernelGGL(k_dact<ENOVA_TANH>, dim3(b), dim3(256), 0, st, g, pre, total);
    else
        hipLaunchKernelGGL(k_dact<ENOVA_RELU>, dim3(b), dim3(256), 0, st, g, pre, total);
    return hipGetLastError();
}

hipError_t launch_latent(float *mu, float *lv, const float *bmu, const float *blv, const float *eps, float *sd,
                         float *z, float *kl, int rows, int L, hipStream_t st)
{
    hipLaunchKernelGGL(k_latent, dim3(static_cast<unsigned>((rows + 255) / 256)), dim3(256), 0, st, mu, lv, bmu,
                       blv, eps, sd, z, kl, rows, L);
    return hipGetLastError();
}

hipError_t launch_recon(float *out, const float *bd2, const float *V, const float *labels, float *logp,
                        int rows, int D, float margin, hipStream_t st)
{
    hipLaunchKernelGGL(k_recon, dim3(static_cast<unsigned>(rows)), dim3(256), 0, st, out, bd2, V, labels, logp,
                       D, 1.0f / static_cast<float>(rows), margin);
    return hipGetLastError();
}

hipError_t launch_beta(const float *kl, const float *logp, const float *labels, int rows, int D,
                       const TrainHyper &h, float *state, float *beta, float *info, hipStream_t st)
{
    hipLaunchKernelGGL(k_beta, dim3(1), dim3(256), 0, st, kl, logp, labels, rows, h.kl_set, h.kp, h.ki,
                       h.beta_min, h.beta_max, h.margin, 0.5f * static_cast<float>(D) * kLog2Pi, state, beta,
                       info);
    return hipGetLastError();
}

hipError_t launch_latent_grad(float *gz, float *glv, const float *mu, const float *lv, const float *sd,
                              const float *eps, const float *labels, const float *beta, int rows, int L,
                              hipStream_t st)
{
    hipLaunchKernelGGL(k_latent_grad, dim3(blocks_for(static_cast<int64_t>(rows) * L)), dim3(256), 0, st, gz,
                       glv, mu, lv, sd, eps, labels, beta, rows, L, 1.0f / static_cast<float>(rows));
    return hipGetLastError();
}

int64_t colsum_workspace_floats(int64_t rows, int cols)
{
    const int64_t chunks = std::min<int64_t>(kColsumMaxChunks, (rows + kColsumRows - 1) / kColsumRows);
    return std::max<int64_t>(chunks, 1) * cols;
}

hipError_t launch_colsum(const float *X, int64_t rows, int cols, float *out, float *work, hipStream_t st)
{
    if (cols <= 0)
        return hipSuccess;
    const int64_t chunks = std::max<int64_t>(1, std::min<int64_t>(kColsumMaxChunks, (rows + kColsumRows - 1) / kColsumRows));
    const int64_t rc = std::max<int64_t>(1, (rows + chunks - 1) / chunks);
    const int64_t used = rows > 0 ? (rows + rc - 1) / rc : 1;
    hipLaunchKernelGGL(k_colsum_part, dim3(static_cast<unsigned>((cols + 63) / 64), static_cast<unsigned>(used)),
                       dim3(256), 0, st, X, rows, cols, rc, work);
    hipLaunchKernelGGL(k_sum_splits<false>, dim3(blocks_for(cols)), dim3(256), 0, st, work,
                       static_cast<int>(used), 1, cols, out, static_cast<int64_t>(cols));
    return hipGetLastError();
}

hipError_t launch_adam(float *p, const float *g, float *m, float *v, int64_t total, const TrainHyper &h,
                       int64_t step, hipStream_t st)
{
    const double c1 = 1.0 / (1.0 - std::pow(static_cast<double>(h.b1), static_cast<double>(step)));
    const double c2 = 1.0 / (1.0 - std::pow(static_cast<double>(h.b2), static_cast<double>(step)));
    hipLaunchKernelGGL(k_adam, dim3(blocks_for(total)), dim3(256), 0, st, p, g, m, v, total, h.lr, h.b1, h.b2,
                       h.eps, static_cast<float>(c1), static_cast<float>(c2));
    return hipGetLastError();
}

}  // namespace enova
