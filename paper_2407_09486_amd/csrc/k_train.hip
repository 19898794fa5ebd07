// Training kernels (Section IV-B, Eq. (9)): a general fp32 matrix-core GEMM for the forward and
// backward products of the VAE over a batch of windows, and the element-wise pieces around them
// (bias + activation, the reparameterised latent and its KL, the reconstruction term and its
// gradient, the PI-controlled KL weight, the latent gradients, activation derivatives, bias
// gradients and the Adam update). Every reduction runs in a fixed order, so a step is
// deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "gemm_plan.h"
#include "train_internal.h"
#include "mfma_common.h"

namespace enova {

namespace {

// Block tiles, slice length and split limits are in gemm_plan.h.
// LDS image of one operand slice. A k-contiguous operand is staged row-major, S[row][k] with a
// pitch of kGemmK + 4 floats (16-byte rows, conflict-free 16-byte reads along k); a
// row-contiguous operand is staged k-major, S[k][row] with a pitch of ROWS + 4 floats
// (16-byte writes along rows, conflict-free 4-byte reads across lanes).
constexpr int kGemmPitch = kGemmK + 4;
// Largest leading dimension of an operand loaded with 32-bit in-tile offsets (128 rows or 32
// reduction indices of it stay below 2^31 elements); larger ones take the bounds-checked loads.
constexpr int64_t kGemmMaxLd32 = int64_t(1) << 24;
constexpr int stage_floats(int rows, bool kcont)
{
    return kcont ? rows * kGemmPitch : kGemmK * (rows + 4);
}
constexpr float kLog2Pi = 1.8378770664093453f;   // log(2 pi)

// One operand tile of a slice: ROWS rows (i of A, j of B) x 32 reduction indices. The operand is
// either "k-contiguous" (X(row, k) = X[row * ld + k]) or "row-contiguous" (X(row, k) =
// X[k * ld + row]); each thread moves ROWS / 32 4-float groups along the contiguous index.
template <bool KCONT, int ROWS>
struct Stage {
    static constexpr int kGroups = ROWS / 32;
    static constexpr int kPitchT = ROWS + 4;
    float4 v[kGroups];

    // Element (row, kx) of thread group q: KCONT walks k fastest (8 groups per row), else rows.
    static __device__ __forceinline__ void coords(int tid, int q, int &row, int &kx)
    {
        const int f = tid + 256 * q;
        if constexpr (KCONT) {
            row = f >> 3;
            kx = (f & 7) * 4;
        } else {
            kx = f / (ROWS / 4);
            row = (f % (ROWS / 4)) * 4;
        }
    }

    // The whole ROWS x 32 tile lies inside the operand and every group is 16-byte aligned: one
    // unconditional 16-byte load per group (a fixed instruction count, so the waits that follow
    // can count exactly how many loads are still in flight).
    // The tile's first element is a uniform base; each group adds a 32-bit offset that does not
    // change between slices (the caller guarantees ld <= kGemmMaxLd32), so a slice's loads need
    // no per-load 64-bit address arithmetic.
    __device__ __forceinline__ void load_full(const float *__restrict__ X, int64_t ld, int r0, int k0, int tid)
    {
        const float *base = KCONT ? X + static_cast<int64_t>(r0) * ld + k0 : X + static_cast<int64_t>(k0) * ld + r0;
        const int ld32 = static_cast<int>(ld);
#pragma unroll
        for (int q = 0; q < kGroups; ++q) {
            int row, kx;
            coords(tid, q, row, kx);
            const int off = KCONT ? row * ld32 + kx : kx * ld32 + row;
            v[q] = *reinterpret_cast<const float4 *>(base + off);
        }
    }

    // full: as load_full (a uniform branch); otherwise element by element with bounds checks.
    __device__ __forceinline__ void load(const float *__restrict__ X, int64_t ld, bool full, int r0, int rmax,
                                         int k0, int kend, int tid)
    {
        if (full) {
            load_full(X, ld, r0, k0, tid);
            return;
        }
#pragma unroll
        for (int q = 0; q < kGroups; ++q) {
            int row, kx;
            coords(tid, q, row, kx);
            float e[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int gr = r0 + row + (KCONT ? 0 : u), gk = k0 + kx + (KCONT ? u : 0);
                e[u] = (gr < rmax && gk < kend) ? X[KCONT ? static_cast<int64_t>(gr) * ld + gk
                                                          : static_cast<int64_t>(gk) * ld + gr]
                                                : 0.0f;
            }
            v[q] = make_float4(e[0], e[1], e[2], e[3]);
        }
    }

    __device__ __forceinline__ void store(float *S, int tid) const
    {
#pragma unroll
        for (int q = 0; q < kGroups; ++q) {
            int row, kx;
            coords(tid, q, row, kx);
            if constexpr (KCONT)
                *reinterpret_cast<float4 *>(&S[row * kGemmPitch + kx]) = v[q];
            else
                *reinterpret_cast<float4 *>(&S[kx * kPitchT + row]) = v[q];
        }
    }

    // The four reduction indices g*8 + 4*half + t (t = 0..3) of staged row `row`.
    static __device__ __forceinline__ float4 operand(const float *S, int row, int g, int half)
    {
        const int k = g * 8 + 4 * half;
        if constexpr (KCONT) {
            return *reinterpret_cast<const float4 *>(&S[row * kGemmPitch + k]);
        } else {
            return make_float4(S[k * kPitchT + row], S[(k + 1) * kPitchT + row], S[(k + 2) * kPitchT + row],
                               S[(k + 3) * kPitchT + row]);
        }
    }
};

// What a product does with C(i, j) once it is complete (fused element-wise steps):
//   kEpiStore:     C = v
//   kEpiBiasAct:   C = v + bias[j] (the pre-activation, kept for the backward pass), out2 = act(C)
//   kEpiDact:      C = v * act'(pre[i][j]) (pre has C's layout)
struct EpiParams {
    const float *bias;   // kEpiBiasAct, kEpiRowReduce
    float *out2;         // kEpiBiasAct: act(C), C's layout; kEpiRowReduce: group sums
    const float *pre;    // kEpiDact; kEpiRowReduce: the minuend, leading dimension ldv
    float *sq;           // kEpiRowReduce: sums of squares
    int ldv, groups;     // kEpiRowReduce
};

template <int ACT>
__device__ __forceinline__ float dact_of(float a)
{
    if constexpr (ACT == ENOVA_TANH) {
        const float t = tanhf(a);
        return 1.0f - t * t;
    } else {
        return a > 0.0f ? 1.0f : 0.0f;
    }
}

template <int EPI, int ACT>
__device__ __forceinline__ void epi_store(float *__restrict__ C, int64_t ldc, int64_t i, int64_t j, float v,
                                          const EpiParams &ep)
{
    const int64_t e = i * ldc + j;
    if constexpr (EPI == kEpiBiasAct) {
        const float a = v + ep.bias[j];
        C[e] = a;
        ep.out2[e] = act_fn<ACT>(a);
    } else if constexpr (EPI == kEpiDact) {
        C[e] = v * dact_of<ACT>(ep.pre[e]);
    } else if constexpr (EPI == kEpiStore) {
        C[e] = v;
    }
}

// A whole 32 x 32 sub-tile (rows si + crow(r, half), column gj of this lane): loads first, then
// the element-wise step and the stores.
template <int EPI, int ACT>
__device__ __forceinline__ void epi_tile(float *__restrict__ C, int64_t ldc, int si, int gj, int half, const v16f &v,
                                         const EpiParams &ep)
{
    if constexpr (EPI == kEpiBiasAct) {
        const float bj = ep.bias[gj];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t e = static_cast<int64_t>(si + crow(r, half)) * ldc + gj;
            const float a = v[r] + bj;
            C[e] = a;
            ep.out2[e] = act_fn<ACT>(a);
        }
    } else if constexpr (EPI == kEpiDact) {
        float pre[16];
#pragma unroll
        for (int r = 0; r < 16; ++r)
            pre[r] = ep.pre[static_cast<int64_t>(si + crow(r, half)) * ldc + gj];
#pragma unroll
        for (int r = 0; r < 16; ++r)
            C[static_cast<int64_t>(si + crow(r, half)) * ldc + gj] = v[r] * dact_of<ACT>(pre[r]);
    } else if constexpr (EPI == kEpiStore) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
            C[static_cast<int64_t>(si + crow(r, half)) * ldc + gj] = v[r];
    }
}

// C(i, j) [+]= sum_k A(i, k) B(k, j) for i < m, j < n over the block's reduction slice
// [z kc, min(kk, (z + 1) kc)), z = blockIdx.z; C(i, j) = C[z m ldc + i ldc + j] (with several
// slices each writes its own partial tile, summed afterwards in slice order by k_sum_splits,
// which then applies the epilogue EPI, or by the Adam step for a weight gradient; a single slice
// applies it here).
// A is k-contiguous when AK (A(i, k) = A[i lda + k]), else row-contiguous (A[k lda + i]); B is
// k-contiguous when BK (B(k, j) = B[j ldb + k]), else row-contiguous (B[k ldb + j]).
// With rowsum != NULL the blocks of the first column tile also write sum_k A(i, k) over the slice
// to rowsum[z m + i] (the bias gradient of a weight-gradient product, read from the staged tiles).
// Matrix op t of an 8-index group takes, in lane l, the reduction index 4 (l / 32) + t of the
// group for both operands (a relabelling of the sum), so one 16-byte LDS read feeds four ops.
template <bool AK, bool BK, int EPI, int ACT, int TM, int TN>
__global__ __launch_bounds__(256, 2) void k_gemm(const float *__restrict__ A, int64_t lda, bool va,
                                                 const float *__restrict__ B, int64_t ldb, bool vb,
                                                 float *__restrict__ C, int64_t ldc, float *__restrict__ rowsum,
                                                 EpiParams ep, int m, int n, int kk, int kc)
{
    // waves along the rows (WM) and columns (WN) of the tile; each covers RW x CW as MA x MB ops
    constexpr int WN = gemm_waves_n(TM, TN);
    constexpr int WM = 4 / WN;
    constexpr int RW = TM / WM, CW = TN / WN;
    constexpr int MA = RW / 32, MB = CW / 32;
    static_assert(MA >= 1 && MB >= 1 && WM * WN == 4, "tile shape");
    __shared__ __align__(16) float As[2][stage_floats(TM, AK)];
    __shared__ __align__(16) float Bs[2][stage_floats(TN, BK)];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wy = wave / WN, wx = wave % WN;
    const int half = lane >> 5, l32 = lane & 31;
    const int i0 = blockIdx.y * TM, j0 = blockIdx.x * TN;
    const int kbeg = blockIdx.z * kc;
    const int kend = min(kk, kbeg + kc);
    C += static_cast<int64_t>(blockIdx.z) * m * ldc;
    bool live_a[MA], live_b[MB];
#pragma unroll
    for (int a = 0; a < MA; ++a)
        live_a[a] = i0 + wy * RW + a * 32 < m;
#pragma unroll
    for (int b = 0; b < MB; ++b)
        live_b[b] = j0 + wx * CW + b * 32 < n;
    const bool sums = rowsum != nullptr && blockIdx.x == 0 && wx == 0;
    v16f acc[MA][MB];
#pragma unroll
    for (int a = 0; a < MA; ++a)
#pragma unroll
        for (int b = 0; b < MB; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[a][b][r] = 0.0f;
    float rs[MA];
#pragma unroll
    for (int a = 0; a < MA; ++a)
        rs[a] = 0.0f;
    // Two register stages: the global loads of slice s + 2 are issued before slice s is computed,
    // so each load has two slices of matrix work to arrive in.
    using SA = Stage<AK, TM>;
    using SB = Stage<BK, TN>;
    SA sa[2];
    SB sb[2];
    const int ns = kend > kbeg ? (kend - kbeg + kGemmK - 1) / kGemmK : 0;
    const bool rows_a = va && i0 + TM <= m, rows_b = vb && j0 + TN <= n;
    auto compute = [&](int buf) __attribute__((always_inline)) {
        // every operand read of the slice is issued before the first matrix op
        float4 av[kGemmK / 8][MA], bv[kGemmK / 8][MB];
#pragma unroll
        for (int g = 0; g < kGemmK / 8; ++g) {
#pragma unroll
            for (int a = 0; a < MA; ++a)
                av[g][a] = SA::operand(As[buf], wy * RW + a * 32 + l32, g, half);
#pragma unroll
            for (int b = 0; b < MB; ++b)
                bv[g][b] = SB::operand(Bs[buf], wx * CW + b * 32 + l32, g, half);
        }
#pragma unroll
        for (int g = 0; g < kGemmK / 8; ++g) {
            // row sums of A (used only when requested; cheaper to always form than to branch)
#pragma unroll
            for (int a = 0; a < MA; ++a)
                rs[a] += (av[g][a].x + av[g][a].y) + (av[g][a].z + av[g][a].w);
            // the four ops of one accumulator are interleaved with the other accumulators' ops
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int a = 0; a < MA; ++a)
#pragma unroll
                    for (int b = 0; b < MB; ++b) {
                        const float4 &x4 = av[g][a], &y4 = bv[g][b];
                        const float x = t == 0 ? x4.x : t == 1 ? x4.y : t == 2 ? x4.z : x4.w;
                        const float y = t == 0 ? y4.x : t == 1 ? y4.y : t == 2 ? y4.z : y4.w;
                        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, y, acc[a][b], 0, 0, 0);
                    }
        }
    };
    // The slice loop, with unconditional loads when every slice of the block is a full tile
    // (FULL) and bounds-checked loads otherwise.
    auto run = [&](auto full_tag) __attribute__((always_inline)) {
        constexpr bool FULL = decltype(full_tag)::value;
        auto fetch = [&](int sl, SA &ra, SB &rb) __attribute__((always_inline)) {
            const int k1 = kbeg + sl * kGemmK;
            if constexpr (FULL) {
                ra.load_full(A, lda, i0, k1, tid);
                rb.load_full(B, ldb, j0, k1, tid);
            } else {
                const bool kin = k1 + kGemmK <= kend;
                ra.load(A, lda, rows_a && kin, i0, m, k1, kend, tid);
                rb.load(B, ldb, rows_b && kin, j0, n, k1, kend, tid);
            }
        };
        // one slice: slice s is in LDS buffer s & 1 and slice s + 1 in registers `nx`; `fr` is free
        // With FULL every step issues the same loads and stores (past the end it re-reads the last
        // slice and fills a buffer nobody reads), so the wait before the stores counts exactly the
        // loads just issued and lets them stay in flight.
        auto step = [&](int s, SA &nxa, SB &nxb, SA &fra, SB &frb) __attribute__((always_inline)) {
            if (FULL)
                fetch(min(s + 2, ns - 1), fra, frb);
            else if (s + 2 < ns)
                fetch(s + 2, fra, frb);
            // keep the loads ahead of the matrix work (the scheduler would sink them to their use)
            __builtin_amdgcn_sched_barrier(0);
            compute(s & 1);
            __builtin_amdgcn_sched_barrier(0);
            if (FULL || s + 1 < ns) {
                nxa.store(As[(s + 1) & 1], tid);
                nxb.store(Bs[(s + 1) & 1], tid);
            }
            __syncthreads();
        };
        if (ns > 0) {
            fetch(0, sa[0], sb[0]);
            if (FULL || ns > 1)
                fetch(min(1, ns - 1), sa[1], sb[1]);
            sa[0].store(As[0], tid);
            sb[0].store(Bs[0], tid);
        }
        // FULL: let the prologue's loads land (vmcnt(0), once per block). Otherwise the wait
        // counters merged at the head of the slice loop still see them, and a register the loop
        // reuses for addresses makes every trip wait for all loads in flight.
        if constexpr (FULL)
            __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
        // pairs of steps as straight-line code (a conditional second step lets the compiler
        // merge both steps' loads at the top of the pair, which shortens the prefetch distance)
        int s = 0;
        for (; s + 1 < ns; s += 2) {
            step(s, sa[1], sb[1], sa[0], sb[0]);
            step(s + 1, sa[0], sb[0], sa[1], sb[1]);
        }
        if (s < ns)
            step(s, sa[1], sb[1], sa[0], sb[0]);
    };
    if (rows_a && rows_b && (kend - kbeg) % kGemmK == 0)
        run(std::true_type{});
    else
        run(std::false_type{});
    if (sums) {
#pragma unroll
        for (int a = 0; a < MA; ++a) {
            const float other = __shfl_xor(rs[a], 32);
            const int gi = i0 + wy * RW + a * 32 + l32;
            if (half == 0 && gi < m)
                rowsum[static_cast<int64_t>(blockIdx.z) * m + gi] = rs[a] + other;
        }
    }
    if constexpr (EPI == kEpiRowReduce) {
        // d = pre - (C + bias) summed per row: over the wave's MB sub-tiles in registers, then
        // across lanes of the same column group (xor of the lane bits at and above `groups`),
        // then the rest of the lanes for the squares. One slot per wave column group.
        const int slot = blockIdx.x * WN + wx;
        if (j0 + wx * CW >= n)
            return;
        const int slots = (n + CW - 1) / CW;
#pragma unroll
        for (int a = 0; a < MA; ++a) {
            if (!live_a[a])
                continue;
            const int si = i0 + wy * RW + a * 32;
            // the 16 rows of a lane in two halves of 8 (fewer registers next to the accumulators)
#pragma unroll
            for (int rh = 0; rh < 16; rh += 8) {
                float sd[8], sq[8];
#pragma unroll
                for (int r = 0; r < 8; ++r)
                    sd[r] = sq[r] = 0.0f;
#pragma unroll
                for (int b = 0; b < MB; ++b) {
                    const int gj = j0 + wx * CW + b * 32 + l32;
                    const bool col = gj < n;
                    const float bj = col ? ep.bias[gj] : 0.0f;
                    float v[8];
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const int gi = si + crow(rh + r, half);
                        v[r] = col && gi < m ? ep.pre[static_cast<int64_t>(gi) * ep.ldv + gj] : 0.0f;
                    }
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const int gi = si + crow(rh + r, half);
                        const float d = col && gi < m ? v[r] - (acc[a][b][rh + r] + bj) : 0.0f;
                        sd[r] += d;
                        sq[r] = fmaf(d, d, sq[r]);
                    }
                }
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    for (int off = 16; off >= ep.groups; off >>= 1)
                        sd[r] += __shfl_xor(sd[r], off);
#pragma unroll
                    for (int off = 16; off >= 1; off >>= 1)
                        sq[r] += __shfl_xor(sq[r], off);
                }
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int gi = si + crow(rh + r, half);
                    if (gi < m) {
                        const int64_t row = static_cast<int64_t>(gi) * slots + slot;
                        if (l32 < ep.groups)
                            ep.out2[row * ep.groups + l32] = sd[r];
                        if (l32 == 0)
                            ep.sq[row] = sq[r];
                    }
                }
            }
        }
        return;
    }
#pragma unroll
    for (int a = 0; a < MA; ++a)
#pragma unroll
        for (int b = 0; b < MB; ++b) {
            if (!(live_a[a] && live_b[b]))
                continue;
            const int si = i0 + wy * RW + a * 32, sj = j0 + wx * CW + b * 32, gj = sj + l32;
            if (si + 32 <= m && sj + 32 <= n) {
                // whole sub-tile inside C: the epilogue's reads are issued together
                epi_tile<EPI, ACT>(C, ldc, si, gj, half, acc[a][b], ep);
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gi = si + crow(r, half);
                    if (gi < m && gj < n)
                        epi_store<EPI, ACT>(C, ldc, gi, gj, acc[a][b][r], ep);
                }
            }
        }
}

// ---- register-streamed products -------------------------------------------------------------
// C(i, j) = sum_k A(i, k) B(k, j) on 16x16x4 fp32 matrix ops with no LDS staging and no barrier
// inside the reduction (the launch shapes and their conditions are gemm_rs_plan's). The four
// waves of a block each compute the whole block tile over every fourth 16-deep reduction step;
// their partial tiles are added in LDS in wave order at the end. An operand fragment is one
// 16-byte load per lane l (p = l % 16, g = l / 16) straight from global memory into the
// matrix-op layout:
//   k-contiguous, fragment f:     row 16 f + p, indices k0 + 4 g + c (c = 0..3, the components);
//   row-contiguous, fragment f:   index k0 + 4 g + f % 4, rows 64 (f / 4) + 4 p + c.
// Matrix op t of an iteration takes, in lane l, reduction index k0 + 4 g + t for both operands (a
// relabelling of the sum), so a 16-row output block `a` of A reads component t of fragment a
// (k-contiguous) or component a % 4 of fragment 4 (a / 4) + t (row-contiguous), and likewise for
// B's 16-column blocks. Output row slot q = 4 g + r of block a (register r) is row 16 a + q, or
// 64 (a / 4) + 4 q + a % 4 for a row-contiguous A; the same for columns with slot p.
typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float comp4(const float4 &v, int c)
{
    return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w;
}

template <bool KMODE>
__device__ __forceinline__ int rs_index(int blk, int slot)
{
    return KMODE ? 16 * blk + slot : 64 * (blk >> 2) + 4 * slot + (blk & 3);
}

// MR 16-row blocks x NC 16-column blocks per wave, PD register slots of operand prefetch. RS: the
// blocks of the first column tile also write rowsum[z m + i] = sum_k A(i, k) over the slice.
template <bool AK, bool BK, int EPI, int ACT, int MR, int NC, int PD>
__global__ __launch_bounds__(64 * kRsWaves) void k_gemm_rs(const float *__restrict__ A, int64_t lda,
                                                           const float *__restrict__ B, int64_t ldb,
                                                           float *__restrict__ C, int64_t ldc,
                                                           float *__restrict__ rowsum, EpiParams ep, int m, int kc)
{
    constexpr int WK = kRsWaves;
    constexpr int TM = 16 * MR, TN = 16 * NC;
    constexpr int NF = MR * NC;                         // output blocks of the tile
    static_assert(AK || MR % 4 == 0, "row-contiguous A comes in 64-row groups");
    static_assert(BK || NC % 4 == 0, "row-contiguous B comes in 64-column groups");
    __shared__ __align__(16) float red[WK * NF * 4 * 64];
    __shared__ float rred[WK * TM];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int p = lane & 15, g = lane >> 4;
    const int i0 = blockIdx.y * TM;
    const int j0 = blockIdx.x * TN;
    const int kw = blockIdx.z * kc + kRsStep * wave;   // first reduction index of iteration 0
    const int iters = kc / (kRsStep * WK);
    C += static_cast<int64_t>(blockIdx.z) * m * ldc;

    // per-lane bases of iteration 0 and the stride between iterations
    const float *ab = AK ? A + static_cast<int64_t>(i0 + p) * lda + kw + 4 * g
                         : A + static_cast<int64_t>(kw + 4 * g) * lda + i0 + 4 * p;
    const float *bb = BK ? B + static_cast<int64_t>(j0 + p) * ldb + kw + 4 * g
                         : B + static_cast<int64_t>(kw + 4 * g) * ldb + j0 + 4 * p;
    const int64_t astep = AK ? kRsStep * WK : static_cast<int64_t>(kRsStep) * WK * lda;
    const int64_t bstep = BK ? kRsStep * WK : static_cast<int64_t>(kRsStep) * WK * ldb;
    auto aoff = [&](int f) -> int64_t { return AK ? 16 * f * lda : (f & 3) * lda + 64 * (f >> 2); };
    auto boff = [&](int f) -> int64_t { return BK ? 16 * f * ldb : (f & 3) * ldb + 64 * (f >> 2); };

    v4f acc[MR][NC];
#pragma unroll
    for (int a = 0; a < MR; ++a)
#pragma unroll
        for (int b = 0; b < NC; ++b)
            acc[a][b] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    constexpr bool RS = !AK;
    float rs[RS ? MR : 1];
#pragma unroll
    for (int a = 0; a < (RS ? MR : 1); ++a)
        rs[a] = 0.0f;

    // One iteration's fragments, always issued in the same order (the scheduling barriers): the
    // prologue and the loop then agree on which loads are in flight at the loop head.
    float4 ar[PD][MR], br[PD][NC];
    auto fetch = [&](int it, float4 (&ra)[MR], float4 (&rb)[NC]) __attribute__((always_inline)) {
        const float *pa = ab + it * astep;
        const float *pb = bb + it * bstep;
#pragma unroll
        for (int f = 0; f < MR; ++f) {
            ra[f] = *reinterpret_cast<const float4 *>(pa + aoff(f));
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int f = 0; f < NC; ++f) {
            rb[f] = *reinterpret_cast<const float4 *>(pb + boff(f));
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // PD register slots: iteration `it` first issues the loads of iteration it + PD - 1 into the
    // slot the previous iteration freed, then runs the matrix ops of slot it % PD.
#pragma unroll
    for (int u = 0; u < PD - 1; ++u) {
        fetch(u < iters ? u : iters - 1, ar[u], br[u]);
        __builtin_amdgcn_sched_barrier(0);
    }
    // let the prologue's loads land (vmcnt(0), once per block): the loop head then merges only
    // the loop's own in-flight loads, whose wait counts stay exact
    __builtin_amdgcn_s_waitcnt(0x0F70);
    for (int i = 0; i < iters; i += PD) {
#pragma unroll
        for (int u = 0; u < PD; ++u) {
            // past the last iteration the last one is fetched again (never read): loads stay in
            // range. The barriers keep the loads here (the scheduler would sink them to their use).
            const int nx = i + u + PD - 1;
            fetch(nx < iters ? nx : iters - 1, ar[(u + PD - 1) % PD], br[(u + PD - 1) % PD]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int a = 0; a < MR; ++a) {
                    const float av = AK ? comp4(ar[u][a], t) : comp4(ar[u][4 * (a >> 2) + t], a & 3);
                    if constexpr (RS)
                        rs[a] += av;
#pragma unroll
                    for (int b = 0; b < NC; ++b) {
                        const float bv = BK ? comp4(br[u][b], t) : comp4(br[u][4 * (b >> 2) + t], b & 3);
                        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[a][b], 0, 0, 0);
                    }
                }
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // partial tiles and row sums (the latter over the four lane groups first) into LDS
#pragma unroll
    for (int a = 0; a < MR; ++a)
#pragma unroll
        for (int b = 0; b < NC; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                red[((wave * NF + a * NC + b) * 4 + r) * 64 + lane] = acc[a][b][r];
    if constexpr (RS) {
#pragma unroll
        for (int a = 0; a < MR; ++a) {
            rs[a] += __shfl_xor(rs[a], 16);
            rs[a] += __shfl_xor(rs[a], 32);
            if (g == 0)
                rred[wave * TM + a * 16 + p] = rs[a];
        }
    }
    __syncthreads();
    // wave w finishes the output blocks f = w, w + 4, ... (partials added in wave order)
    for (int f = wave; f < NF; f += WK) {
        const int a = f / NC, b = f - (f / NC) * NC;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float s = 0.0f;
#pragma unroll
            for (int w2 = 0; w2 < WK; ++w2)
                s += red[((w2 * NF + f) * 4 + r) * 64 + lane];
            v[r] = s;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
            epi_store<EPI, ACT>(C, ldc, i0 + rs_index<AK>(a, 4 * g + r), j0 + rs_index<BK>(b, p), v[r], ep);
    }
    if constexpr (RS) {
        if (rowsum != nullptr && blockIdx.x == 0 && wave == 0 && g == 0) {
#pragma unroll
            for (int a = 0; a < MR; ++a) {
                float s = 0.0f;
#pragma unroll
                for (int w2 = 0; w2 < WK; ++w2)
                    s += rred[w2 * TM + a * 16 + p];
                rowsum[static_cast<int64_t>(blockIdx.z) * m + i0 + rs_index<AK>(a, p)] = s;
            }
        }
    }
}

// C(i, j) = epilogue(sum over the slices s = 0, 1, ... (in order) of P[s][i][j]) for i < m, j < n,
// and, with rowsum != NULL, rowsum[i] = sum over the slices of R[s][i].
template <int EPI, int ACT>
__global__ __launch_bounds__(256) void k_sum_splits(const float *__restrict__ P, const float *__restrict__ R,
                                                    int splits, int m, int n, float *__restrict__ C, int64_t ldc,
                                                    float *__restrict__ rowsum, EpiParams ep)
{
    const int64_t total = static_cast<int64_t>(m) * n;
    const int64_t all = total + (rowsum ? m : 0);
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < all; e += static_cast<int64_t>(gridDim.x) * 256) {
        const bool main = e < total;
        const float *src = main ? P + e : R + (e - total);
        const int64_t stride = main ? total : m;
        float v = 0.0f;
        int sp = 0;
        for (; sp + 8 <= splits; sp += 8) {
            float t[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                t[u] = src[(sp + u) * stride];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                v += t[u];
        }
        for (; sp < splits; ++sp)
            v += src[sp * stride];
        if (main)
            epi_store<EPI, ACT>(C, ldc, e / n, e % n, v, ep);
        else
            rowsum[e - total] = v;
    }
}

// One thread per window. ml holds [mu | lv] per window (2L floats, biases [bmu | blv] added in
// place); sd = e^(lv/2), z = mu + sd eps and the KL of q(z|m) from N(0, I).
__global__ __launch_bounds__(64) void k_latent(float *__restrict__ ml, const float *__restrict__ bml,
                                               const float *__restrict__ eps, float *__restrict__ sd,
                                               float *__restrict__ z, float *__restrict__ kl, int rows, int L)
{
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= rows)
        return;
    float *mu = ml + static_cast<int64_t>(i) * 2 * L, *lv = mu + L;
    float k = 0.0f;
    for (int l = 0; l < L; ++l) {
        const int64_t e = static_cast<int64_t>(i) * L + l;
        const float m = mu[l] + bml[l];
        const float v = lv[l] + bml[L + l];
        const float s = expf(0.5f * v);
        mu[l] = m;
        lv[l] = v;
        sd[e] = s;
        z[e] = m + s * eps[e];
        k += m * m + kl_g(v);
    }
    kl[i] = 0.5f * k;
}

// The same with one thread per (window, latent index) when L is a power of two <= 64: coalesced
// accesses, and the window's KL summed over its L lanes by a butterfly.
__global__ __launch_bounds__(256) void k_latent_lanes(float *__restrict__ ml, const float *__restrict__ bml,
                                                      const float *__restrict__ eps, float *__restrict__ sd,
                                                      float *__restrict__ z, float *__restrict__ kl, int rows, int L)
{
    const int64_t t = blockIdx.x * 256LL + threadIdx.x;
    const int64_t i = t / L;
    const int l = static_cast<int>(t - i * L);
    const bool on = i < rows;
    float k = 0.0f;
    if (on) {
        float *mu = ml + i * 2 * L;
        const float m = mu[l] + bml[l];
        const float v = mu[L + l] + bml[L + l];
        const float s = expf(0.5f * v);
        mu[l] = m;
        mu[L + l] = v;
        sd[t] = s;
        z[t] = m + s * eps[t];
        k = m * m + kl_g(v);
    }
    for (int off = 1; off < L; off <<= 1)
        k += __shfl_xor(k, off);
    if (on && l == 0)
        kl[i] = 0.5f * k;
}

// One wave per window (four per block) when D is a multiple of 4 and at most 2048: lane l holds
// the differences j = 256 q + 4 l + u in registers, the window's error is a butterfly over the
// wave, and no LDS or barrier is involved. Same outputs as k_recon.
template <int Q>
__global__ __launch_bounds__(256) void k_recon_wave(float *__restrict__ out, const float *__restrict__ bd2,
                                                    const float *__restrict__ V, const float *__restrict__ labels,
                                                    float *__restrict__ logp, int rows, int D, float inv_b,
                                                    float margin)
{
    const int lane = threadIdx.x & 63;
    const int64_t row = blockIdx.x * 4LL + (threadIdx.x >> 6);
    if (row >= rows)
        return;
    float *o = out + row * D;
    const float *v = V + row * D;
    float4 d[Q];
    float sq = 0.0f;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = 256 * q + 4 * lane;
        if (j < D) {
            const float4 a = *reinterpret_cast<const float4 *>(o + j);
            const float4 b = *reinterpret_cast<const float4 *>(bd2 + j);
            const float4 c = *reinterpret_cast<const float4 *>(v + j);
            d[q] = make_float4(a.x + b.x - c.x, a.y + b.y - c.y, a.z + b.z - c.z, a.w + b.w - c.w);
        } else {
            d[q] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
        sq += (d[q].x * d[q].x + d[q].y * d[q].y) + (d[q].z * d[q].z + d[q].w * d[q].w);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        sq += __shfl_xor(sq, off);
    const float l = labels[row];
    const float err = 0.5f * sq;
    const float scale = (l > 0.0f || err < margin) ? l * inv_b : 0.0f;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = 256 * q + 4 * lane;
        if (j < D)
            *reinterpret_cast<float4 *>(o + j) =
                make_float4(scale * d[q].x, scale * d[q].y, scale * d[q].z, scale * d[q].w);
    }
    if (lane == 0)
        logp[row] = -err - 0.5f * static_cast<float>(D) * kLog2Pi;
}

// One block per window: m' = out + bd2, e = |v - m'|^2 / 2, log p = -e - D/2 log 2 pi, and in place
// of out the gradient of J, (l/B)(m' - v); an anomalous window (l < 0) whose e has reached the
// margin contributes a constant and gets a zero gradient. PER > 0: the window's D <= 256 PER
// differences stay in registers between the reduction and the write; PER = 0 recomputes them.
template <int PER>
__global__ __launch_bounds__(256) void k_recon(float *__restrict__ out, const float *__restrict__ bd2,
                                               const float *__restrict__ V, const float *__restrict__ labels,
                                               float *__restrict__ logp, int D, float inv_b, float margin)
{
    __shared__ float red[256];
    const int64_t row = blockIdx.x;
    const float l = labels[row];
    float *o = out + row * D;
    const float *v = V + row * D;
    float d[PER > 0 ? PER : 1];
    float sq = 0.0f;
    if constexpr (PER > 0) {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int j = threadIdx.x + 256 * u;
            d[u] = j < D ? o[j] + bd2[j] - v[j] : 0.0f;
            sq += d[u] * d[u];
        }
    } else {
        for (int j = threadIdx.x; j < D; j += 256) {
            const float t = o[j] + bd2[j] - v[j];
            sq += t * t;
        }
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
    if constexpr (PER > 0) {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int j = threadIdx.x + 256 * u;
            if (j < D)
                o[j] = scale * d[u];
        }
    } else {
        for (int j = threadIdx.x; j < D; j += 256)
            o[j] = scale * (o[j] + bd2[j] - v[j]);
    }
    if (threadIdx.x == 0)
        logp[row] = -err - 0.5f * static_cast<float>(D) * kLog2Pi;
}

// One block: the KL weight of this step from the PI controller, and the step's summary
// (J, mean log p, mean KL of the normal windows, beta). State: st[0] = the integral term.
// An anomalous window enters J through -log p capped at margin + D/2 log 2 pi.
// It also advances the Adam step count k (held on the device, so a step's launches carry no
// per-step host value) and writes the bias corrections 1/(1 - b1^k), 1/(1 - b2^k) to corr.
__global__ __launch_bounds__(1024) void k_beta(const float *__restrict__ kl, const float *__restrict__ logp,
                                              const float *__restrict__ labels, int rows, float kl_set,
                                              float kp, float ki, float beta_min, float beta_max,
                                              float margin, float half_d_log2pi,
                                              float *__restrict__ st, float *__restrict__ beta_out,
                                              float *__restrict__ info, float b1, float b2,
                                              long long *__restrict__ step, float *__restrict__ corr)
{
    // per thread (fixed stride), per wave (butterfly), then the 16 wave sums in wave order
    __shared__ double r[5][16];
    double a[5] = {0.0, 0.0, 0.0, 0.0, 0.0};   // KL of normal windows, their count, log p, J terms, KL terms
    // 8 elements per thread per round, all loaded before any is added
    for (int i0 = 0; i0 < rows; i0 += 8 * 1024) {
        float fl[8], fk[8], fp[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * 1024 + static_cast<int>(threadIdx.x);
            const bool in = i < rows;
            fl[u] = in ? labels[i] : 0.0f;   // a zero label adds nothing below
            fk[u] = in ? kl[i] : 0.0f;
            fp[u] = in ? logp[i] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const double l = fl[u], k = fk[u], lp = fp[u];
            if (l > 0.0) {
                a[0] += k;
                a[1] += 1.0;
            }
            a[2] += lp;
            if (l < 0.0) {
                // anomalous: -log p capped at margin + D/2 log 2 pi
                const double err = -lp - static_cast<double>(half_d_log2pi);
                a[3] += (err < margin ? err : static_cast<double>(margin)) + static_cast<double>(half_d_log2pi);
            } else {
                a[3] += l * lp;
            }
            a[4] += 0.5 * (1.0 + l) * k;
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
        for (int q = 0; q < 5; ++q)
            a[q] += __shfl_xor(a[q], off);
    if ((threadIdx.x & 63) == 0)
#pragma unroll
        for (int q = 0; q < 5; ++q)
            r[q][threadIdx.x >> 6] = a[q];
    __syncthreads();
    if (threadIdx.x == 0) {
        double s_kl = 0.0, s_n = 0.0, s_lp = 0.0, s_la = 0.0, s_kn = 0.0;
        for (int w = 0; w < 16; ++w) {
            s_kl += r[0][w];
            s_n += r[1][w];
            s_lp += r[2][w];
            s_la += r[3][w];
            s_kn += r[4][w];
        }
        const double mkl = s_n > 0.0 ? s_kl / s_n : 0.0;
        const double e = static_cast<double>(kl_set) - mkl;
        const double integ = static_cast<double>(st[0]) - static_cast<double>(ki) * e;
        const double p = e < 700.0 ? static_cast<double>(kp) / (1.0 + exp(e)) : 0.0;
        double b = p + integ + static_cast<double>(beta_min);
        b = b < beta_min ? beta_min : (b > beta_max ? beta_max : b);
        st[0] = static_cast<float>(integ);
        beta_out[0] = static_cast<float>(b);
        if (info) {
            info[0] = static_cast<float>(-(s_la - b * s_kn) / rows);
            info[1] = static_cast<float>(s_lp / rows);
            info[2] = static_cast<float>(mkl);
            info[3] = static_cast<float>(b);
        }
    } else if (threadIdx.x == 64 || threadIdx.x == 65) {
        // the Adam step count and its two bias corrections, in a second wave beside the
        // controller (both lanes take one pow together; the count is read before lane 64 stores it)
        const int c = static_cast<int>(threadIdx.x) - 64;
        const long long k_adam = step[0] + 1;
        const double bc = static_cast<double>(c == 0 ? b1 : b2);
        corr[c] = static_cast<float>(1.0 / (1.0 - pow(bc, static_cast<double>(k_adam))));
        if (c == 0)
            step[0] = k_adam;
    }
}

// Gradients of J at the latent: g_mu = g_z + c mu, g_lv = g_z eps sd/2 + c (e^lv - 1)/2 with
// c = (1 + l)/2 beta / B, written as [g_mu | g_lv] per window (the layout of ml).
__global__ __launch_bounds__(256) void k_latent_grad(const float *__restrict__ gz, float *__restrict__ gml,
                                                     const float *__restrict__ ml, const float *__restrict__ sd,
                                                     const float *__restrict__ eps, const float *__restrict__ labels,
                                                     const float *__restrict__ beta, int rows, int L, float inv_b)
{
    const int64_t total = static_cast<int64_t>(rows) * L;
    const float b = beta[0];
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t i = e / L;
        const int l = static_cast<int>(e - i * L);
        const float c = 0.5f * (1.0f + labels[i]) * b * inv_b;
        const float g = gz[e];
        const float *row = ml + i * 2 * L;
        float *out = gml + i * 2 * L;
        out[l] = g + c * row[l];
        out[L + l] = g * eps[e] * 0.5f * sd[e] + c * 0.5f * expm1f(row[L + l]);
    }
}

// Adam on every flat parameter. An entry inside one of the `sums` ranges first adds its
// gradient's slices in slice order and stores the result in g; every other entry reads g. The
// slices are loaded 16 at a time while 16 remain, then 8 at a time, so a thin product's 64
// slices take four round trips to memory.
__global__ __launch_bounds__(256) void k_adam(float *__restrict__ p, float *__restrict__ g,
                                              float *__restrict__ m, float *__restrict__ v, int64_t total,
                                              float lr, float b1, float b2, float eps,
                                              const float *__restrict__ corr, GradSums sums)
{
    const float c1 = corr[0], c2 = corr[1];
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += static_cast<int64_t>(gridDim.x) * 256) {
        bool summed = false;
        float ge = 0.0f;
#pragma unroll
        for (int q = 0; q < kMaxGradSums; ++q) {
            if (q >= sums.n)
                break;
            const int64_t i = e - sums.s[q].begin;
            if (i < 0 || i >= sums.s[q].count)
                continue;
            const float *src = sums.s[q].src + i;
            const int64_t stride = sums.s[q].stride;
            const int splits = sums.s[q].splits;
            int sp = 0;
            for (; sp + 16 <= splits; sp += 16) {
                float t[16];
#pragma unroll
                for (int u = 0; u < 16; ++u)
                    t[u] = src[(sp + u) * stride];
#pragma unroll
                for (int u = 0; u < 16; ++u)
                    ge += t[u];
            }
            for (; sp + 8 <= splits; sp += 8) {
                float t[8];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    t[u] = src[(sp + u) * stride];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    ge += t[u];
            }
            for (; sp < splits; ++sp)
                ge += src[sp * stride];
            summed = true;
        }
        if (summed)
            g[e] = ge;
        else
            ge = g[e];
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

namespace {

template <bool AK, bool BK, int EPI, int ACT>
void gemm_run(dim3 grid, hipStream_t st, const float *A, int64_t lda, bool va, const float *B, int64_t ldb, bool vb,
              float *C, int64_t ldc, float *rowsum, const EpiParams &ep, int m, int n, int k, int kc)
{
    int tm, tn;
    gemm_tile(m, n, tm, tn);
    if (tn == kGemmThin)
        hipLaunchKernelGGL((k_gemm<AK, BK, EPI, ACT, kGemmTile, kGemmThin>), grid, dim3(256), 0, st, A, lda, va, B,
                           ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
    else if (tm == kGemmThin)
        hipLaunchKernelGGL((k_gemm<AK, BK, EPI, ACT, kGemmThin, kGemmTile>), grid, dim3(256), 0, st, A, lda, va, B,
                           ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
    else
        hipLaunchKernelGGL((k_gemm<AK, BK, EPI, ACT, kGemmTile, kGemmTile>), grid, dim3(256), 0, st, A, lda, va, B,
                           ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
}

template <int EPI, int ACT>
void gemm_layouts(bool a_k, bool b_k, dim3 grid, hipStream_t st, const float *A, int64_t lda, bool va,
                  const float *B, int64_t ldb, bool vb, float *C, int64_t ldc, float *rowsum, const EpiParams &ep,
                  int m, int n, int k, int kc)
{
    if (a_k && b_k)
        gemm_run<true, true, EPI, ACT>(grid, st, A, lda, va, B, ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
    else if (a_k)
        gemm_run<true, false, EPI, ACT>(grid, st, A, lda, va, B, ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
    else if (b_k)
        gemm_run<false, true, EPI, ACT>(grid, st, A, lda, va, B, ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
    else
        gemm_run<false, false, EPI, ACT>(grid, st, A, lda, va, B, ldb, vb, C, ldc, rowsum, ep, m, n, k, kc);
}

template <int EPI, int ACT>
void sum_run(unsigned blocks, hipStream_t st, const float *P, const float *R, int splits, int m, int n, float *C,
             int64_t ldc, float *rowsum, const EpiParams &ep)
{
    hipLaunchKernelGGL((k_sum_splits<EPI, ACT>), dim3(blocks), dim3(256), 0, st, P, R, splits, m, n, C, ldc, rowsum,
                       ep);
}

// The register-streamed kernel of plan kind `kind` for the operand layouts.
template <int EPI, int ACT>
void rs_layouts(int kind, bool a_k, bool b_k, dim3 grid, hipStream_t st, const float *A, int64_t lda,
                const float *B, int64_t ldb, float *C, int64_t ldc, float *rowsum, const EpiParams &ep, int m, int kc)
{
    // each kernel's tile is rs_shape(kind): tm = 16 MR, tn = 16 NC, pd register slots
    const dim3 block(64 * kRsWaves);
    if (kind == kRsK4 && b_k)
        hipLaunchKernelGGL((k_gemm_rs<true, true, EPI, ACT, 2, 8, 2>), grid, block, 0, st, A, lda, B, ldb, C, ldc,
                           rowsum, ep, m, kc);
    else if (kind == kRsK4)
        hipLaunchKernelGGL((k_gemm_rs<true, false, EPI, ACT, 2, 8, 2>), grid, block, 0, st, A, lda, B, ldb, C, ldc,
                           rowsum, ep, m, kc);
    else
        hipLaunchKernelGGL((k_gemm_rs<false, false, EPI, ACT, 4, 4, 2>), grid, block, 0, st, A, lda, B, ldb, C, ldc,
                           rowsum, ep, m, kc);
    (void)a_k;
}

// The epilogue kind and activation as template arguments.
template <template <int, int> class F, typename... Args>
void with_epilogue(int kind, int act, Args &&...args)
{
    if (kind == kEpiBiasAct) {
        if (act == ENOVA_TANH)
            F<kEpiBiasAct, ENOVA_TANH>::run(args...);
        else
            F<kEpiBiasAct, ENOVA_RELU>::run(args...);
    } else if (kind == kEpiDact) {
        if (act == ENOVA_TANH)
            F<kEpiDact, ENOVA_TANH>::run(args...);
        else
            F<kEpiDact, ENOVA_RELU>::run(args...);
    } else if (kind == kEpiRowReduce) {
        F<kEpiRowReduce, ENOVA_RELU>::run(args...);
    } else {
        F<kEpiStore, ENOVA_RELU>::run(args...);
    }
}

// rs_layouts with the epilogue kind and activation as template arguments (store, bias +
// activation, activation derivative: the kinds gemm_rs_plan accepts).
template <typename... Args>
void rs_epilogue(int kind, int act, Args &&...args)
{
    if (kind == kEpiBiasAct) {
        if (act == ENOVA_TANH)
            rs_layouts<kEpiBiasAct, ENOVA_TANH>(args...);
        else
            rs_layouts<kEpiBiasAct, ENOVA_RELU>(args...);
    } else if (kind == kEpiDact) {
        if (act == ENOVA_TANH)
            rs_layouts<kEpiDact, ENOVA_TANH>(args...);
        else
            rs_layouts<kEpiDact, ENOVA_RELU>(args...);
    } else {
        rs_layouts<kEpiStore, ENOVA_RELU>(args...);
    }
}

template <int EPI, int ACT>
struct GemmF {
    template <typename... Args>
    static void run(Args &&...args)
    {
        gemm_layouts<EPI, ACT>(args...);
    }
};

template <int EPI, int ACT>
struct SumF {
    template <typename... Args>
    static void run(Args &&...args)
    {
        sum_run<EPI, ACT>(args...);
    }
};

}  // namespace

hipError_t launch_gemm(const GemmEpilogue &epi, const float *A, int64_t ai, int64_t ak, const float *B, int64_t bk,
                       int64_t bj, float *C, int64_t ldc, int m, int n, int k, float *rowsum, float *work,
                       int64_t work_floats, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1, GemmSplit *defer)
{
    if (defer) {
        *defer = GemmSplit{};
        if (epi.kind != kEpiStore || ldc != n)
            return hipErrorInvalidValue;
    }
    if (m <= 0 || n <= 0)
        return hipSuccess;
    // each operand needs a unit stride along the reduction index or along its row index
    if ((ak != 1 && ai != 1) || (bk != 1 && bj != 1))
        return hipErrorInvalidValue;
    const bool a_k = ak == 1, b_k = bk == 1;
    const int64_t lda = a_k ? ai : ak, ldb = b_k ? bj : bk;
    const bool va = lda % 4 == 0 && lda <= kGemmMaxLd32 && reinterpret_cast<uintptr_t>(A) % 16 == 0;
    const bool vb = ldb % 4 == 0 && ldb <= kGemmMaxLd32 && reinterpret_cast<uintptr_t>(B) % 16 == 0;
    if (epi.kind == kEpiRowReduce &&
        (epi.groups < 1 || epi.groups > 32 || (epi.groups & (epi.groups - 1)) != 0 || !epi.sq || !epi.out2))
        return hipErrorInvalidValue;
    const EpiParams epp{epi.bias, epi.out2, epi.pre, epi.sq, epi.ldv, epi.groups};
    {
        // whole tiles with aligned operands: the register-streamed kernel
        const bool epi_rs = epi.kind == kEpiStore || epi.kind == kEpiBiasAct || epi.kind == kEpiDact;
        const RsPlan rp = gemm_rs_plan(m, n, k, a_k, b_k, epi_rs, va && vb, work != nullptr, work_floats);
        if (rp.kind != kRsNone) {
            const RsShape sh = rs_shape(rp.kind);
            const dim3 rgrid(static_cast<unsigned>(n / sh.tn), static_cast<unsigned>(m / sh.tm),
                             static_cast<unsigned>(rp.used));
            hipError_t e = hipSuccess;
            if (ev0 && (e = hipEventRecord(ev0, st)) != hipSuccess)
                return e;
            if (rp.used == 1) {
                rs_epilogue(epi.kind, epi.act, rp.kind, a_k, b_k, rgrid, st, A, lda, B, ldb, C, ldc, rowsum, epp, m,
                            rp.kc);
                if ((e = hipGetLastError()) != hipSuccess)
                    return e;
                return ev1 ? hipEventRecord(ev1, st) : hipSuccess;
            }
            float *part_rows = rowsum ? work + static_cast<int64_t>(rp.used) * m * n : nullptr;
            rs_layouts<kEpiStore, ENOVA_RELU>(rp.kind, a_k, b_k, rgrid, st, A, lda, B, ldb, work,
                                              static_cast<int64_t>(n), part_rows, EpiParams{}, m, rp.kc);
            if ((e = hipGetLastError()) != hipSuccess)
                return e;
            if (ev1 && (e = hipEventRecord(ev1, st)) != hipSuccess)
                return e;
            if (defer) {
                *defer = GemmSplit{work, part_rows, rp.used};
                return hipSuccess;
            }
            const unsigned blocks = blocks_for(static_cast<int64_t>(m) * n + (rowsum ? m : 0));
            with_epilogue<SumF>(epi.kind, epi.act, blocks, st, static_cast<const float *>(work),
                                static_cast<const float *>(part_rows), rp.used, m, n, C, ldc, rowsum, epp);
            return hipGetLastError();
        }
    }
    // never more slices than the caller's workspace holds (a row reduction is never split)
    const GemmPlan plan = gemm_plan(m, n, k, work && epi.kind != kEpiRowReduce, work_floats);
    const int kc = plan.kc, used = plan.used;
    const dim3 grid(static_cast<unsigned>((n + plan.tn - 1) / plan.tn), static_cast<unsigned>((m + plan.tm - 1) / plan.tm),
                    static_cast<unsigned>(used));
    hipError_t e = hipSuccess;
    if (ev0 && (e = hipEventRecord(ev0, st)) != hipSuccess)
        return e;
    if (used == 1) {
        with_epilogue<GemmF>(epi.kind, epi.act, a_k, b_k, grid, st, A, lda, va, B, ldb, vb, C, ldc, rowsum, epp, m, n,
                             k, kc);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        return ev1 ? hipEventRecord(ev1, st) : hipSuccess;
    }
    // partial tiles, then one pass that sums them in slice order and applies the epilogue
    float *part_rows = rowsum ? work + static_cast<int64_t>(used) * m * n : nullptr;
    gemm_layouts<kEpiStore, ENOVA_RELU>(a_k, b_k, grid, st, A, lda, va, B, ldb, vb, work, static_cast<int64_t>(n),
                                        part_rows, EpiParams{}, m, n, k, kc);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (ev1 && (e = hipEventRecord(ev1, st)) != hipSuccess)
        return e;
    if (defer) {
        *defer = GemmSplit{work, part_rows, used};
        return hipSuccess;
    }
    const unsigned blocks = blocks_for(static_cast<int64_t>(m) * n + (rowsum ? m : 0));
    with_epilogue<SumF>(epi.kind, epi.act, blocks, st, static_cast<const float *>(work),
                        static_cast<const float *>(part_rows), used, m, n, C, ldc, rowsum, epp);
    return hipGetLastError();
}

hipError_t launch_latent(float *ml, const float *bml, const float *eps, float *sd, float *z, float *kl, int rows,
                         int L, hipStream_t st)
{
    if (L <= 64 && (L & (L - 1)) == 0) {
        const int64_t threads = static_cast<int64_t>(rows) * L;
        hipLaunchKernelGGL(k_latent_lanes, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st, ml, bml,
                           eps, sd, z, kl, rows, L);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_latent, dim3(static_cast<unsigned>((rows + 63) / 64)), dim3(64), 0, st, ml, bml, eps, sd, z,
                       kl, rows, L);
    return hipGetLastError();
}

hipError_t launch_recon(float *out, const float *bd2, const float *V, const float *labels, float *logp,
                        int rows, int D, float margin, hipStream_t st)
{
    const float inv_b = 1.0f / static_cast<float>(rows);
    const bool vec = D % 4 == 0 && D <= 2048 && reinterpret_cast<uintptr_t>(out) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(V) % 16 == 0 && reinterpret_cast<uintptr_t>(bd2) % 16 == 0;
    if (vec) {
        const dim3 wgrid(static_cast<unsigned>((rows + 3) / 4));
        const int q = (D + 255) / 256;
        switch (q) {
        case 1: hipLaunchKernelGGL(k_recon_wave<1>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        case 2: hipLaunchKernelGGL(k_recon_wave<2>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        case 3: hipLaunchKernelGGL(k_recon_wave<3>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        case 4: hipLaunchKernelGGL(k_recon_wave<4>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        case 5: hipLaunchKernelGGL(k_recon_wave<5>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        case 6: hipLaunchKernelGGL(k_recon_wave<6>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        case 7: hipLaunchKernelGGL(k_recon_wave<7>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        default: hipLaunchKernelGGL(k_recon_wave<8>, wgrid, dim3(256), 0, st, out, bd2, V, labels, logp, rows, D, inv_b, margin); break;
        }
        return hipGetLastError();
    }
    const dim3 grid(static_cast<unsigned>(rows));
    if (D <= 256)
        hipLaunchKernelGGL(k_recon<1>, grid, dim3(256), 0, st, out, bd2, V, labels, logp, D, inv_b, margin);
    else if (D <= 512)
        hipLaunchKernelGGL(k_recon<2>, grid, dim3(256), 0, st, out, bd2, V, labels, logp, D, inv_b, margin);
    else if (D <= 1024)
        hipLaunchKernelGGL(k_recon<4>, grid, dim3(256), 0, st, out, bd2, V, labels, logp, D, inv_b, margin);
    else if (D <= 2048)
        hipLaunchKernelGGL(k_recon<8>, grid, dim3(256), 0, st, out, bd2, V, labels, logp, D, inv_b, margin);
    else
        hipLaunchKernelGGL(k_recon<0>, grid, dim3(256), 0, st, out, bd2, V, labels, logp, D, inv_b, margin);
    return hipGetLastError();
}

hipError_t launch_beta(const float *kl, const float *logp, const float *labels, int rows, int D,
                       const TrainHyper &h, float *state, float *beta, float *info, long long *step, float *corr,
                       hipStream_t st)
{
    hipLaunchKernelGGL(k_beta, dim3(1), dim3(1024), 0, st, kl, logp, labels, rows, h.kl_set, h.kp, h.ki,
                       h.beta_min, h.beta_max, h.margin, 0.5f * static_cast<float>(D) * kLog2Pi, state, beta,
                       info, h.b1, h.b2, step, corr);
    return hipGetLastError();
}

hipError_t launch_latent_grad(const float *gz, float *gml, const float *ml, const float *sd, const float *eps,
                              const float *labels, const float *beta, int rows, int L, hipStream_t st)
{
    hipLaunchKernelGGL(k_latent_grad, dim3(blocks_for(static_cast<int64_t>(rows) * L)), dim3(256), 0, st, gz, gml,
                       ml, sd, eps, labels, beta, rows, L, 1.0f / static_cast<float>(rows));
    return hipGetLastError();
}

hipError_t launch_adam(float *p, float *g, float *m, float *v, int64_t total, const TrainHyper &h,
                       const float *corr, const GradSums &sums, hipStream_t st)
{
    if (sums.n < 0 || sums.n > kMaxGradSums)
        return hipErrorInvalidValue;
    for (int q = 0; q < sums.n; ++q) {
        const GradSum &r = sums.s[q];
        if (r.begin < 0 || r.count < 0 || r.begin + r.count > total || r.splits < 1 || !r.src || r.stride < r.count)
            return hipErrorInvalidValue;
    }
    hipLaunchKernelGGL(k_adam, dim3(blocks_for(total)), dim3(256), 0, st, p, g, m, v, total, h.lr, h.b1, h.b2,
                       h.eps, corr, sums);
    return hipGetLastError();
}

}  // namespace enova
