// Streaming detection kernels: the ring of each stream's last W steps, the matrix-core scoring of
// every stream's newest window, and per-stream streaming peaks-over-threshold (SPOT, Siffer et
// al. -- the POT method Section IV-B cites; Section V runs the detector in a stream-computing
// job).
//
// Scoring: a block scores the newest windows of 16 streams (Section IV-B: normalise, encoder,
// heads, KL score, decoder hidden layer for the md). Unlike the sliding-window batch kernel, no
// two windows share data, so nothing is staged: each wave streams its share of the reduction
// from the rings straight into registers and the four waves' partial sums meet in LDS once
// (the scoring section below).
//
// SPOT refits run on the device, one block per stream with a new peak, with the batch fit's
// method: Grimshaw's reduction bracketed on geometric 512-point grids of both admissible
// intervals, each bracket refined to fp64 resolution (here by Newton's method kept inside the
// bracket), the exponential tail always a candidate.
#include <hip/hip_runtime.h>

#include <cmath>

#include "gpd_math.h"
#include "stream_internal.h"
#include "mfma_common.h"

namespace enova {

namespace {

constexpr int kStreamThreads = 64 * kStreamWaves;

struct StreamShape {
    int M, S, W, Mp, Q, CPR;
    int iters;        // reduction iterations of each wave (a multiple of the window prefetch depth)
    float inv_d;
};

// ---- ring append ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_stream_append(const T *__restrict__ x, int n, int M, int W,
                                                       int slot, T *__restrict__ ring)
{
    const int64_t total = static_cast<int64_t>(n) * M;
    for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < total; i += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t s = i / M;
        const int m = static_cast<int>(i - s * M);
        const T v = x[i];
        ring[(s * 2 * W + slot) * M + m] = v;
        ring[(s * 2 * W + slot + W) * M + m] = v;
    }
}

// ---- scoring of the newest windows ----------------------------------------------------------
// A block scores kStreamNb = 16 windows (one per stream). No two of them share data, so nothing
// is staged: each wave streams its own share of the reduction straight from HBM into
// registers. Reduction step j covers chunks 4j .. 4j+3 of every window (chunk kappa = q*CPR + c:
// chunk c of super-row q, the packed W1's order); wave w takes the steps j = w mod 4, lane l
// loads chunk 4j + l/16 of window l%16 (the B operand of the 16x16 matrix ops) and the W1
// fragments of the same step arrive from L2 (the A operand). The four waves' partial hidden
// sums meet in LDS and are added in a fixed order; the epilogue then chains heads and decoder on
// 16x16x4 fp32 matrix ops from the accumulator layout (lane l, register r: row 4*(l/16) + r,
// column l%16), which is the B-operand layout of the next op with its reduction index permuted
// to match (the packed head and decoder weights carry that permutation).
typedef float v4f __attribute__((ext_vector_type(4)));

template <int DT>
__device__ __forceinline__ v4f mfma_step(uint4 a, uint4 b, v4f c)
{
    if constexpr (DT == ENOVA_F32) {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        return __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    } else {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b),
                                                       c, 0, 0, 0);
    }
}

// The normalised chunk: (x - mean) / std of its elements (rounded to bf16 for the bf16
// detector), zeros where ok is false; sum gains the values as they enter the matrix ops.
template <int DT, int EPC>
__device__ __forceinline__ uint4 normalise_chunk(uint4 raw, const float (&mu)[EPC], const float (&is)[EPC],
                                                 bool ok, float &sum)
{
    float xv[EPC];
    if constexpr (DT == ENOVA_F32) {
        xv[0] = __uint_as_float(raw.x);
        xv[1] = __uint_as_float(raw.y);
        xv[2] = __uint_as_float(raw.z);
        xv[3] = __uint_as_float(raw.w);
    } else {
        xv[0] = bf16_lo(raw.x);
        xv[1] = bf16_hi(raw.x);
        xv[2] = bf16_lo(raw.y);
        xv[3] = bf16_hi(raw.y);
        xv[4] = bf16_lo(raw.z);
        xv[5] = bf16_hi(raw.z);
        xv[6] = bf16_lo(raw.w);
        xv[7] = bf16_hi(raw.w);
    }
    float v[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e)
        v[e] = ok ? (xv[e] - mu[e]) * is[e] : 0.0f;
    uint4 out;
    if constexpr (DT == ENOVA_F32) {
        out.x = __float_as_uint(v[0]);
        out.y = __float_as_uint(v[1]);
        out.z = __float_as_uint(v[2]);
        out.w = __float_as_uint(v[3]);
        sum += (v[0] + v[1]) + (v[2] + v[3]);
    } else {
        out.x = pack_bf16x2(v[0], v[1]);
        out.y = pack_bf16x2(v[2], v[3]);
        out.z = pack_bf16x2(v[4], v[5]);
        out.w = pack_bf16x2(v[6], v[7]);
        sum += ((bf16_lo(out.x) + bf16_hi(out.x)) + (bf16_lo(out.y) + bf16_hi(out.y))) +
               ((bf16_lo(out.z) + bf16_hi(out.z)) + (bf16_lo(out.w) + bf16_hi(out.w)));
    }
    return out;
}

// Chunk kappa of window s gathered element by element (any metric count and padding).
template <int DT>
__device__ __forceinline__ uint4 gather_chunk(const StreamScoreParams &p, const StreamShape &g, int s, bool live,
                                              int kappa, float &sum)
{
    constexpr int EPC = DT == ENOVA_F32 ? 4 : 8;
    const int q = kappa / g.CPR;
    const int c = kappa - q * g.CPR;
    float v[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
        const int jj = c * EPC + e;
        const int tt = jj / g.Mp;
        const int m = jj - tt * g.Mp;
        const int step = q * g.S + tt;
        float val = 0.0f;
        if (live && q < g.Q && m < g.M && step < g.W) {
            const int64_t at = (static_cast<int64_t>(s) * 2 * g.W + p.first_slot + step) * g.M + m;
            const int64_t sm = static_cast<int64_t>(s) * g.M + m;
            val = (load_x<DT>(p.ring, at) - p.mean[sm]) * (1.0f / p.std[sm]);
        }
        v[e] = val;
    }
    uint4 out;
    if constexpr (DT == ENOVA_F32) {
        out.x = __float_as_uint(v[0]);
        out.y = __float_as_uint(v[1]);
        out.z = __float_as_uint(v[2]);
        out.w = __float_as_uint(v[3]);
        sum += (v[0] + v[1]) + (v[2] + v[3]);
    } else {
        out.x = pack_bf16x2(v[0], v[1]);
        out.y = pack_bf16x2(v[2], v[3]);
        out.z = pack_bf16x2(v[4], v[5]);
        out.w = pack_bf16x2(v[6], v[7]);
        sum += ((bf16_lo(out.x) + bf16_hi(out.x)) + (bf16_lo(out.y) + bf16_hi(out.y))) +
               ((bf16_lo(out.z) + bf16_hi(out.z)) + (bf16_lo(out.w) + bf16_hi(out.w)));
    }
    return out;
}

// NHB 16-row hidden blocks (Hp = 16 NHB). VEC: the window is a contiguous run of the ring whose
// chunks hold whole groups of metrics, and each lane normalises the same EPC metrics at every
// step (M divides 4 EPC), so the chunks are loaded raw PB steps ahead and normalised with
// per-lane constants; otherwise every chunk is gathered element by element.
template <int DT, int NHB, int ACT, bool VEC>
__global__ __launch_bounds__(kStreamThreads) void k_stream_score(StreamScoreParams p, StreamShape g)
{
    constexpr int EPC = DT == ENOVA_F32 ? 4 : 8;
    constexpr int PA = stream_pa(NHB), PB = stream_pb(DT), U = PA > PB ? PA : PB;
    constexpr int OWN = (NHB + kStreamWaves - 1) / kStreamWaves;   // hidden blocks of a wave's epilogue
    extern __shared__ float lds[];
    float *xp = lds;                                   // [wave][hb][r][lane] encoder partial sums
    float *xz = xp + kStreamWaves * NHB * 4 * 64;      // [wave][head][r][lane] head partial sums
    float *xs = xz + kStreamWaves * 2 * 4 * 64;        // [wave][window] partial window sums
    float *xd = xs + kStreamWaves * kStreamNb;         // [wave][window] partial u . hd

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int n = lane & 15;
    const int grp = lane >> 4;
    const int s = blockIdx.x * kStreamNb + n;
    const bool live = s < p.n_streams;
    const int sc = live ? s : 0;                       // addresses of dead lanes stay in stream 0
    const int WM = g.W * g.M;

    v4f acc[NHB];
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
        acc[hb] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    float wsum = 0.0f;

    // iteration i of this wave is reduction step 4i + wave: lane chunk 16 i + 4 wave + grp
    const int kap0 = 4 * wave + grp;
    const uint4 *ap = p.w1p + static_cast<size_t>(wave) * NHB * 64 + lane;
    constexpr size_t kIterA = static_cast<size_t>(4) * NHB * 64;   // fragments per iteration
    uint4 a[PA][NHB];
#pragma unroll
    for (int k = 0; k < PA; ++k)
#pragma unroll
        for (int hb = 0; hb < NHB; ++hb)
            a[k][hb] = ap[k * kIterA + hb * 64];

    if constexpr (VEC) {
        float mu[EPC], is[EPC];
        {
            const float *mp = p.mean + static_cast<int64_t>(sc) * g.M + (grp * EPC) % g.M;
            const float *sp = p.std + static_cast<int64_t>(sc) * g.M + (grp * EPC) % g.M;
#pragma unroll
            for (int h = 0; h < EPC / 4; ++h) {
                const float4 m4 = reinterpret_cast<const float4 *>(mp)[h];
                const float4 s4 = reinterpret_cast<const float4 *>(sp)[h];
                mu[4 * h + 0] = m4.x;
                mu[4 * h + 1] = m4.y;
                mu[4 * h + 2] = m4.z;
                mu[4 * h + 3] = m4.w;
                is[4 * h + 0] = 1.0f / s4.x;
                is[4 * h + 1] = 1.0f / s4.y;
                is[4 * h + 2] = 1.0f / s4.z;
                is[4 * h + 3] = 1.0f / s4.w;
            }
        }
        const int64_t wbase = (static_cast<int64_t>(sc) * 2 * g.W + p.first_slot) * g.M;
        auto load_raw = [&](int it) __attribute__((always_inline)) -> uint4 {
            const int e0 = (16 * it + kap0) * EPC;
            const int64_t at = live && e0 < WM ? wbase + e0 : 0;
            if constexpr (DT == ENOVA_F32)
                return *reinterpret_cast<const uint4 *>(static_cast<const float *>(p.ring) + at);
            else
                return *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p.ring) + at);
        };
        uint4 b[PB];
#pragma unroll
        for (int k = 0; k < PB; ++k)
            b[k] = load_raw(k);
        for (int i = 0; i < g.iters; i += U) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int it = i + u;
                const bool ok = live && (16 * it + kap0) * EPC < WM;
                const uint4 bv = normalise_chunk<DT, EPC>(b[u % PB], mu, is, ok, wsum);
                b[u % PB] = load_raw(it + PB);
#pragma unroll
                for (int hb = 0; hb < NHB; ++hb)
                    acc[hb] = mfma_step<DT>(a[u % PA][hb], bv, acc[hb]);
                // iterations up to iters + PA - 1 are read: the packed W1 carries them as zeros
#pragma unroll
                for (int hb = 0; hb < NHB; ++hb)
                    a[u % PA][hb] = ap[(it + PA) * kIterA + hb * 64];
            }
        }
    } else {
        for (int i = 0; i < g.iters; i += PA) {
#pragma unroll
            for (int u = 0; u < PA; ++u) {
                const int it = i + u;
                const uint4 bv = gather_chunk<DT>(p, g, sc, live, 16 * it + kap0, wsum);
#pragma unroll
                for (int hb = 0; hb < NHB; ++hb)
                    acc[hb] = mfma_step<DT>(a[u][hb], bv, acc[hb]);
#pragma unroll
                for (int hb = 0; hb < NHB; ++hb)
                    a[u][hb] = ap[(it + PA) * kIterA + hb * 64];
            }
        }
    }

    // ---- the four waves' partial sums, added in a fixed order ----
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
            xp[((wave * NHB + hb) * 4 + r) * 64 + lane] = acc[hb][r];
    wsum += __shfl_xor(wsum, 16);
    wsum += __shfl_xor(wsum, 32);
    if (grp == 0)
        xs[wave * kStreamNb + n] = wsum;
    __syncthreads();

    // hidden activations of the blocks hb = wave + 4 t feed this wave's share of the heads
    v4f zm = v4f{0.0f, 0.0f, 0.0f, 0.0f}, zl = zm;
#pragma unroll
    for (int t = 0; t < OWN; ++t) {
        const int hb = wave + kStreamWaves * t;
        if (hb < NHB) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float h = 0.0f;
#pragma unroll
                for (int w2 = 0; w2 < kStreamWaves; ++w2)
                    h += xp[((w2 * NHB + hb) * 4 + r) * 64 + lane];
                const float hv = act_fn<ACT>(h + p.b1[16 * hb + 4 * grp + r]);
                zm = __builtin_amdgcn_mfma_f32_16x16x4f32(p.whp[((hb * 4 + r) * 2 + 0) * 64 + lane], hv, zm, 0, 0, 0);
                zl = __builtin_amdgcn_mfma_f32_16x16x4f32(p.whp[((hb * 4 + r) * 2 + 1) * 64 + lane], hv, zl, 0, 0, 0);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        xz[((wave * 2 + 0) * 4 + r) * 64 + lane] = zm[r];
        xz[((wave * 2 + 1) * 4 + r) * 64 + lane] = zl[r];
    }
    __syncthreads();
    // mean and log-variance of latent 4 grp + r, window n (every wave the same sums)
    float mu[4], kl = 0.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float m = 0.0f, lv = 0.0f;
#pragma unroll
        for (int w2 = 0; w2 < kStreamWaves; ++w2) {
            m += xz[((w2 * 2 + 0) * 4 + r) * 64 + lane];
            lv += xz[((w2 * 2 + 1) * 4 + r) * 64 + lane];
        }
        mu[r] = m + p.bh[4 * grp + r];
        lv += p.bh[16 + 4 * grp + r];
        kl += mu[r] * mu[r] + kl_g(lv);
    }
    kl += __shfl_xor(kl, 16);
    kl += __shfl_xor(kl, 32);

    // decoder hidden layer at z = mu for the same hidden blocks, dotted with u
    float dot = 0.0f;
#pragma unroll
    for (int t = 0; t < OWN; ++t) {
        const int hb = wave + kStreamWaves * t;
        if (hb < NHB) {
            v4f d = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int r = 0; r < 4; ++r)
                d = __builtin_amdgcn_mfma_f32_16x16x4f32(p.wd1p[(hb * 4 + r) * 64 + lane], mu[r], d, 0, 0, 0);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int h = 16 * hb + 4 * grp + r;
                dot += p.u[h] * act_fn<ACT>(d[r] + p.bd1[h]);
            }
        }
    }
    dot += __shfl_xor(dot, 16);
    dot += __shfl_xor(dot, 32);
    if (grp == 0)
        xd[wave * kStreamNb + n] = dot;
    __syncthreads();
    if (wave == 0 && grp == 0 && live) {
        float ws = 0.0f, dt = 0.0f;
#pragma unroll
        for (int w2 = 0; w2 < kStreamWaves; ++w2) {
            ws += xs[w2 * kStreamNb + n];
            dt += xd[w2 * kStreamNb + n];
        }
        p.scores[s] = 0.5f * kl;
        if (p.md)
            p.md[s] = ws * g.inv_d - (dt + p.sum_bd2) * g.inv_d;
    }
}

using StreamKernel = void (*)(StreamScoreParams, StreamShape);

template <int DT, int ACT, bool VEC>
StreamKernel pick_stream(int nhb)
{
    switch (nhb) {
    case 2: return k_stream_score<DT, 2, ACT, VEC>;
    case 4: return k_stream_score<DT, 4, ACT, VEC>;
    case 8: return k_stream_score<DT, 8, ACT, VEC>;
    case 16: return k_stream_score<DT, 16, ACT, VEC>;
    default: return nullptr;
    }
}

template <int DT, int ACT>
StreamKernel pick_stream(int nhb, bool vec)
{
    return vec ? pick_stream<DT, ACT, true>(nhb) : pick_stream<DT, ACT, false>(nhb);
}

StreamKernel pick_stream(const Geometry &g)
{
    const bool relu = g.act == ENOVA_RELU;
    const int nhb = g.Hp / 16;
    const bool vec = stream_vec(g);
    if (g.dtype == ENOVA_F32)
        return relu ? pick_stream<ENOVA_F32, ENOVA_RELU>(nhb, vec) : pick_stream<ENOVA_F32, ENOVA_TANH>(nhb, vec);
    return relu ? pick_stream<ENOVA_BF16, ENOVA_RELU>(nhb, vec) : pick_stream<ENOVA_BF16, ENOVA_TANH>(nhb, vec);
}

size_t stream_lds(const Geometry &g)
{
    const size_t nhb = static_cast<size_t>(g.Hp / 16);
    return (kStreamWaves * nhb * 4 * 64 + kStreamWaves * 2 * 4 * 64 + 2 * kStreamWaves * kStreamNb) * sizeof(float);
}

// ---- SPOT -------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t fkey(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float fkey_inv(uint32_t k)
{
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Start of one stream per block: t = the calibration scores' order statistic at
// ceil(level n) - 1 (radix select on order-preserving keys), the peaks c - t for c > t in
// calibration order (stable compaction), n = the number of calibration scores.
__global__ __launch_bounds__(256) void k_spot_init(const float *__restrict__ cal,
                                                   const int64_t *__restrict__ cal_off, double level,
                                                   SpotState st)
{
    __shared__ unsigned int hist[256];
    __shared__ uint32_t sh_prefix;
    __shared__ int64_t sh_rank;
    __shared__ int scan[256];
    __shared__ int64_t sh_np;
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t lo = cal_off[s];
    const int64_t ns = cal_off[s + 1] - lo;
    const float *c = cal + lo;
    if (ns == 0) {
        if (tid == 0) {
            st.t[s] = INFINITY;
            st.z[s] = INFINITY;
            st.cnt[s] = 0;
            st.npk[s] = 0;
            st.mark[s] = 0;
        }
        return;
    }
    for (int64_t i = tid; i < ns; i += 256)
        if (!isfinite(c[i]))
            st.err[0] = 2;
    int64_t rank = static_cast<int64_t>(ceil(level * static_cast<double>(ns))) - 1;
    if (rank < 0)
        rank = 0;
    if (tid == 0) {
        sh_prefix = 0;
        sh_rank = rank;
    }
    for (int shift = 24; shift >= 0; shift -= 8) {
        hist[tid] = 0;
        __syncthreads();
        const uint32_t prefix = sh_prefix;
        for (int64_t i = tid; i < ns; i += 256) {
            const uint32_t k = fkey(c[i]);
            if (shift == 24 || (k >> (shift + 8)) == (prefix >> (shift + 8)))
                atomicAdd(&hist[(k >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            int64_t r = sh_rank, cum = 0;
            int b = 0;
            for (; b < 255; ++b) {
                if (cum + hist[b] > static_cast<uint64_t>(r))
                    break;
                cum += hist[b];
            }
            sh_rank = r - cum;
            sh_prefix = prefix | (static_cast<uint32_t>(b) << shift);
        }
        __syncthreads();
    }
    const float tf = fkey_inv(sh_prefix);
    const double t = static_cast<double>(tf);
    // stable compaction of the peaks
    if (tid == 0)
        sh_np = 0;
    __syncthreads();
    double *pk = st.peaks + static_cast<int64_t>(s) * st.cap;
    for (int64_t base = 0; base < ns; base += 256) {
        const int64_t i = base + tid;
        const float ci = i < ns ? c[i] : 0.0f;
        const int f = (i < ns && ci > tf) ? 1 : 0;
        scan[tid] = f;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {
            const int v = tid >= off ? scan[tid - off] : 0;
            __syncthreads();
            scan[tid] += v;
            __syncthreads();
        }
        const int64_t pos = sh_np + scan[tid] - f;
        if (f && pos < st.cap)
            pk[pos] = static_cast<double>(ci) - t;
        __syncthreads();
        if (tid == 255)
            sh_np += scan[255];
        __syncthreads();
    }
    if (tid == 0) {
        if (sh_np > st.cap)
            st.err[0] = 1;
        st.t[s] = t;
        st.z[s] = t;
        st.cnt[s] = ns;
        st.npk[s] = static_cast<int>(sh_np < st.cap ? sh_np : st.cap);
        st.mark[s] = 1;
    }
}

// One score per stream: an alarm leaves the model alone; otherwise the observation counts and
// an exceedance of t joins the peaks (the stream's z is refitted by k_spot_fit). Streams
// without calibration, or with a full peak store, only compare.
__global__ __launch_bounds__(256) void k_spot_update(const float *__restrict__ scores, int n, SpotState st,
                                                     uint8_t *__restrict__ flags)
{
    const int s = blockIdx.x * 256 + threadIdx.x;
    if (s >= n)
        return;
    const float x = scores[s];
    uint8_t f = 0;
    if (!isnan(x)) {
        const double xd = static_cast<double>(x);
        const double t = st.t[s];
        const int np = st.npk[s];
        if (xd > st.z[s]) {
            f = 1;
        } else if (!isinf(t) && np < st.cap) {
            st.cnt[s] += 1;
            if (xd > t) {
                st.peaks[static_cast<int64_t>(s) * st.cap + np] = xd - t;
                st.npk[s] = np + 1;
                st.mark[s] = 1;
                st.list[atomicAdd(st.count + st.cur, 1)] = s;
            }
        }
    }
    if (flags)
        flags[s] = f;
}

constexpr int kFitGrid = 512;       // grid points per admissible interval
constexpr int kFitRounds = 64;      // evaluations per bracket at most
constexpr int kFitMaxBrackets = 64; // sign changes kept per fit
constexpr int kFitThreads = 1024;   // threads of a refit block (16 waves: four per SIMD)
constexpr int kFitWaves = kFitThreads / 64;
constexpr int kFitMaxPoints = 2 * kFitGrid;
constexpr int kFitLdsPeaks = 4096;  // a stream with at most this many peaks refits from an LDS copy
static_assert(kFitMaxPoints <= kFitThreads, "one point per thread");

struct FitShared {
    double yl[kFitLdsPeaks];     // the stream's peaks
    double xs[kFitMaxPoints];
    double sa[kFitMaxPoints];
    double sb[kFitMaxPoints];
    double red[3][kFitWaves + 1];
    double blo[kFitMaxBrackets], bhi[kFitMaxBrackets], broot[kFitMaxBrackets], bx[kFitMaxBrackets];
    double bwlo[kFitMaxBrackets], bwhi[kFitMaxBrackets];   // w at the bracket's ends (Illinois-scaled)
    int bneg[kFitMaxBrackets], bdone[kFitMaxBrackets], bround[kFitMaxBrackets], bside[kFitMaxBrackets];
    double roots[2 * kFitMaxBrackets];
    int batch[kFitWaves];        // the brackets the waves refine in this evaluation
    int wcount[2][kFitWaves];    // per-wave counts of roots and of sign changes
    int nbr, nroots, npts, ngrid, nbatch;
};

__device__ __forceinline__ double fit_w(double sa, double sb, double n)
{
    const double a = sa / n, b = sb / n;
    return b - a - a * b;
}

__device__ __forceinline__ double fit_quantile(double t, double gamma, double sigma, double ratio)
{
    if (fabs(gamma) < 1e-9)
        return t - sigma * log(ratio);
    return t + sigma / gamma * (pow(ratio, -gamma) - 1.0);
}

// sa/sb at the first npts (<= kFitMaxPoints) points of sh.xs over all N excesses (with
// nw > 0: sa = w(sa, sb, nw) = b - a - a b instead). The points go
// in groups of four; the T threads of a group (T a power of two, at most 64, consecutive lanes
// of one wave) each sum every T-th excess for the group's four points side by side (independent
// dependency chains), and the T partial sums are added by a fixed butterfly. A fixed order.
__device__ void fit_eval(FitShared &sh, const double *y, int N, double nw = 0.0)
{
    const int np = sh.npts;
    const int groups = (np + 3) / 4;
    int T = 1;
    while (T < 64 && 2 * T * groups <= kFitThreads)
        T *= 2;
    const int gi = static_cast<int>(threadIdx.x) / T;
    const int part = static_cast<int>(threadIdx.x) % T;
    double x[4], a[4], b[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int p = 4 * gi + k;
        x[k] = gi < groups && p < np ? sh.xs[p] : 0.0;
        a[k] = 0.0;
        b[k] = 0.0;
    }
    if (gi < groups) {
        for (int i = part; i < N; i += T) {
            const double yi = y[i];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                double ta, tb;
                gpd_terms_fast(x[k] * yi, ta, tb);
                a[k] += ta;
                b[k] += tb;
            }
        }
    }
    // every lane of the wave takes part in the butterfly (T divides 64)
    for (int off = T / 2; off >= 1; off >>= 1) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a[k] += __shfl_xor(a[k], off);
            b[k] += __shfl_xor(b[k], off);
        }
    }
    if (gi < groups && part == 0) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int p = 4 * gi + k;
            if (p < np) {
                sh.sa[p] = nw > 0.0 ? fit_w(a[k], b[k], nw) : a[k];
                sh.sb[p] = b[k];
            }
        }
    }
    __syncthreads();
}

// Fixed-order block reductions of one value per thread: a butterfly in each wave, then the wave
// results in wave order. block_reduce3 forms the sum of v0, the minimum of v1 and the maximum of
// v2 together; block_sum the sum of v.
__device__ void block_reduce3(FitShared &sh, double &v0, double &v1, double &v2)
{
    for (int off = 32; off >= 1; off >>= 1) {
        v0 += __shfl_xor(v0, off);
        v1 = fmin(v1, __shfl_xor(v1, off));
        v2 = fmax(v2, __shfl_xor(v2, off));
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        sh.red[0][wave] = v0;
        sh.red[1][wave] = v1;
        sh.red[2][wave] = v2;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double r0 = sh.red[0][0], r1 = sh.red[1][0], r2 = sh.red[2][0];
        for (int w = 1; w < kFitWaves; ++w) {
            r0 += sh.red[0][w];
            r1 = fmin(r1, sh.red[1][w]);
            r2 = fmax(r2, sh.red[2][w]);
        }
        sh.red[0][kFitWaves] = r0;
        sh.red[1][kFitWaves] = r1;
        sh.red[2][kFitWaves] = r2;
    }
    __syncthreads();
    v0 = sh.red[0][kFitWaves];
    v1 = sh.red[1][kFitWaves];
    v2 = sh.red[2][kFitWaves];
    __syncthreads();
}

__device__ double block_sum(FitShared &sh, double v)
{
    double lo = INFINITY, hi = -INFINITY;
    block_reduce3(sh, v, lo, hi);
    return v;
}

// Refit of z for one marked stream by one block: N_t <= 1 gives t; 2 <= N_t < 10 the method of
// moments with the unbiased sample variance; N_t >= 10 maximum likelihood.
__device__ void spot_fit_stream(FitShared &sh, int s, double q, const SpotState &st)
{
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int N = st.npk[s];
    const double t = st.t[s];
    const double n = static_cast<double>(st.cnt[s]);
    const double *yg = st.peaks + static_cast<int64_t>(s) * st.cap;
    double z = t;
    if (N >= 2) {
        // the peaks are read once per pass below: from an LDS copy when they fit
        const double *y = N <= kFitLdsPeaks ? sh.yl : yg;
        double ps = 0.0, pmin = INFINITY, pmax = -INFINITY;
        for (int i = tid; i < N; i += kFitThreads) {
            const double v = yg[i];
            if (N <= kFitLdsPeaks)
                sh.yl[i] = v;
            ps += v;
            pmin = fmin(pmin, v);
            pmax = fmax(pmax, v);
        }
        block_reduce3(sh, ps, pmin, pmax);     // its barriers also publish the LDS copy
        const double ysum = ps, ymin = pmin, ymax = pmax;
        const double Nd = static_cast<double>(N);
        const double ymean = ysum / Nd;
        if (N < 10) {
            double pv = 0.0;
            for (int i = tid; i < N; i += kFitThreads)
                pv += (y[i] - ymean) * (y[i] - ymean);
            const double s2 = block_sum(sh, pv) / (Nd - 1.0);
            if (s2 > 0.0 && wave == 0) {
                const double gamma = 0.5 * (1.0 - ymean * ymean / s2);
                const double sigma = 0.5 * ymean * (1.0 + ymean * ymean / s2);
                z = fit_quantile(t, gamma, sigma, q * n / Nd);
            }
        } else {
            // geometric grids over both admissible intervals of x = gamma / sigma
            const double eps = 1e-8 / ymean;
            const double f0 = eps * ymax;
            const double right = 2.0 * (ymean - ymin) / (ymin * ymin);
            const bool has_left = f0 < 0.5, has_right = right > 2.0 * eps;
            const int right_at = has_left ? kFitGrid : 0;
            // threads 0 .. kFitGrid-1 the left grid, the others the right one
            static_assert(2 * kFitGrid <= kFitThreads, "a grid point per thread");
            {
                const int i = tid % kFitGrid;
                if (tid < kFitGrid && has_left) {
                    const double zlo = log(f0 / (1.0 - f0)), zhi = 30.0;
                    const double zz = zlo + (zhi - zlo) * static_cast<double>(i) / static_cast<double>(kFitGrid - 1);
                    sh.xs[i] = -(1.0 / (1.0 + exp(-zz))) / ymax;
                }
                if (tid >= kFitGrid && tid < 2 * kFitGrid && has_right)
                    sh.xs[right_at + i] = eps * pow(right / eps, static_cast<double>(i) / static_cast<double>(kFitGrid - 1));
            }
            if (tid == 0) {
                sh.ngrid = (has_left ? 1 : 0) + (has_right ? 1 : 0);
                sh.npts = sh.ngrid * kFitGrid;
            }
            __syncthreads();
            fit_eval(sh, y, N, Nd);
            // every grid point: an exact root, and/or a sign change to the next point of its grid;
            // both kept in grid order (wave ballots, then the waves in order)
            {
                const int i = tid;
                int root = 0, br = 0;
                if (i < sh.npts) {
                    const int gi = i % kFitGrid;
                    const double wi = sh.sa[i];
                    if (wi == 0.0)
                        root = 1;
                    else if (gi + 1 < kFitGrid && wi * sh.sa[i + 1] < 0.0)
                        br = 1;
                }
                const uint64_t mr = __ballot(root), mb = __ballot(br);
                const uint64_t below = lane ? (~uint64_t{0} >> (64 - lane)) : 0;
                if (lane == 0) {
                    sh.wcount[0][wave] = __popcll(mr);
                    sh.wcount[1][wave] = __popcll(mb);
                }
                __syncthreads();
                int r_at = __popcll(mr & below), b_at = __popcll(mb & below);
                int nr = 0, nb = 0;
                for (int w = 0; w < kFitWaves; ++w) {
                    if (w < wave) {
                        r_at += sh.wcount[0][w];
                        b_at += sh.wcount[1][w];
                    }
                    nr += sh.wcount[0][w];
                    nb += sh.wcount[1][w];
                }
                if (root && r_at < 2 * kFitMaxBrackets)
                    sh.roots[r_at] = sh.xs[i];
                if (br && b_at < kFitMaxBrackets) {
                    const double x0 = sh.xs[i], x1 = sh.xs[i + 1];
                    const double wi = sh.sa[i], wn = sh.sa[i + 1];
                    const double lo = x0 < x1 ? x0 : x1, hi = x0 < x1 ? x1 : x0;
                    sh.blo[b_at] = lo;
                    sh.bhi[b_at] = hi;
                    sh.bwlo[b_at] = x0 < x1 ? wi : wn;
                    sh.bwhi[b_at] = x0 < x1 ? wn : wi;
                    sh.bneg[b_at] = x0 < x1 ? (wi < 0.0) : (wn < 0.0);
                    sh.bdone[b_at] = 0;
                    sh.bround[b_at] = 0;
                    sh.bside[b_at] = 0;
                    sh.broot[b_at] = 0.0;
                    // the first point: the secant of w through the bracket's ends (the grid has w
                    // there), else the midpoint
                    const double xsec = x0 - wi * (x1 - x0) / (wn - wi);
                    sh.bx[b_at] = xsec > lo && xsec < hi ? xsec : 0.5 * (lo + hi);
                }
                if (tid == 0) {
                    sh.nroots = nr < 2 * kFitMaxBrackets ? nr : 2 * kFitMaxBrackets;
                    sh.nbr = nb < kFitMaxBrackets ? nb : kFitMaxBrackets;
                }
                __syncthreads();
            }
            // Newton's method on w inside each bracket: one wave per open bracket evaluates w and
            // w' at the bracket's current point (first the secant point of the grid values) over
            // all peaks (lane l sums the peaks l, l + 64, ..., a butterfly adds the lanes), and
            // its lane 0 keeps the bracket on the sign of w, taking the Newton step when it lands
            // strictly inside and otherwise false position through the ends (Illinois), else the
            // midpoint. A bracket ends at a zero of w to the rounding of its sums, with the step
            // taken once it falls below 2^-26 of the point, when the bracket can no longer be
            // split, or after kFitRounds evaluations.
            for (;;) {
                if (tid == 0) {
                    sh.nbatch = 0;
                    for (int b = 0; b < sh.nbr && sh.nbatch < kFitWaves; ++b)
                        if (!sh.bdone[b])
                            sh.batch[sh.nbatch++] = b;
                }
                __syncthreads();
                if (sh.nbatch == 0)
                    break;
                if (wave < sh.nbatch) {
                    const int b = sh.batch[wave];
                    const double x = sh.bx[b];
                    double sa = 0.0, sb = 0.0, sda = 0.0, sdb = 0.0;
                    for (int i = lane; i < N; i += 64) {
                        const double yi = y[i];
                        double ta, tb, r;
                        gpd_terms_fast(x * yi, ta, tb, r);
                        sa += ta;
                        sb += tb;
                        sdb += yi * r;
                        sda += (yi * r) * r;
                    }
                    for (int off = 32; off >= 1; off >>= 1) {
                        sa += __shfl_xor(sa, off);
                        sb += __shfl_xor(sb, off);
                        sda += __shfl_xor(sda, off);
                        sdb += __shfl_xor(sdb, off);
                    }
                    if (lane == 0) {
                        const double a = sa / Nd, bm = sb / Nd, da = sda / Nd, db = sdb / Nd;
                        const double wv = bm - a - a * bm;
                        const double wd = db - da - da * bm - a * db;
                        const int it = sh.bround[b] + 1;
                        sh.bround[b] = it;
                        if (wv == 0.0) {
                            sh.bdone[b] = 1;
                            sh.broot[b] = x;
                        } else {
                            double lo = sh.blo[b], hi = sh.bhi[b];
                            double wlo = sh.bwlo[b], whi = sh.bwhi[b];
                            // the end that x replaces takes w(x); an end kept twice in a row has
                            // its w halved (Illinois), so the false-position fallback keeps
                            // shrinking the bracket from both sides
                            const int side = (wv < 0.0) == (sh.bneg[b] != 0) ? -1 : 1;
                            if (side < 0) {
                                lo = x;
                                wlo = wv;
                                if (sh.bside[b] < 0)
                                    whi *= 0.5;
                            } else {
                                hi = x;
                                whi = wv;
                                if (sh.bside[b] > 0)
                                    wlo *= 0.5;
                            }
                            sh.bside[b] = side;
                            sh.bwlo[b] = wlo;
                            sh.bwhi[b] = whi;
                            const double xn = x - wv / wd;
                            const bool inside = xn > lo && xn < hi;     // false for NaN
                            // when the Newton step leaves the bracket: false position through the
                            // ends, else the midpoint
                            const double xf = lo - wlo * (hi - lo) / (whi - wlo);
                            const double mid = xf > lo && xf < hi ? xf : 0.5 * (lo + hi);
                            // |w| within the rounding of the sums it is formed from: x is a root
                            // to fp64 resolution (where w is flat, no step test would tell more)
                            const bool flat = fabs(wv) <= 0x1p-46 * (fabs(bm) + fabs(a) + fabs(a * bm));
                            // converged once the step is below 2^-26 of the point: from there the
                            // step's quadratic convergence lands within rounding of the root (a
                            // tighter test only meets the rounding noise of the sums, and the
                            // iterates then wander inside the bracket)
                            const double tol = 0x1p-26 * fmax(fabs(lo), fabs(hi));
                            sh.blo[b] = lo;
                            sh.bhi[b] = hi;
                            if (flat) {
                                sh.bdone[b] = 1;
                                sh.broot[b] = x;
                            } else if (inside && fabs(xn - x) <= tol) {
                                sh.bdone[b] = 1;
                                sh.broot[b] = xn;
                            } else if (!inside && !(mid > lo && mid < hi)) {
                                sh.bdone[b] = 1;
                                sh.broot[b] = mid;
                            } else if (it >= kFitRounds) {
                                sh.bdone[b] = 1;
                                sh.broot[b] = inside ? xn : mid;
                            } else {
                                sh.bx[b] = inside ? xn : mid;
                            }
                        }
                    }
                }
                __syncthreads();
            }
            // candidates: the exponential tail and every root
            if (tid == 0) {
                for (int b = 0; b < sh.nbr && sh.nroots < 2 * kFitMaxBrackets; ++b)
                    sh.roots[sh.nroots++] = sh.bdone[b] ? sh.broot[b] : 0.5 * (sh.blo[b] + sh.bhi[b]);
                for (int r = 0; r < sh.nroots; ++r)
                    sh.xs[r] = sh.roots[r];
                sh.npts = sh.nroots;
            }
            __syncthreads();
            fit_eval(sh, y, N);
            // the choice and the quantile in one wave (only thread 0 stores z; the other waves'
            // copies of these fp64 chains would share its SIMDs' issue slots)
            if (wave == 0) {
                double bg = 0.0, bs = ymean;
                double bl = -Nd * log(ymean) - ysum / ymean;
                for (int r = 0; r < sh.nroots; ++r) {
                    const double gm = sh.sb[r] / Nd;
                    if (gm == 0.0 || !isfinite(gm))
                        continue;
                    const double sg = gm / sh.roots[r];
                    if (!(sg > 0.0))
                        continue;
                    const double ll = -Nd * log(sg) - (1.0 + 1.0 / gm) * sh.sb[r];
                    if (ll > bl || (ll == bl && fabs(gm) < fabs(bg))) {
                        bg = gm;
                        bs = sg;
                        bl = ll;
                    }
                }
                z = fit_quantile(t, bg, bs, q * n / Nd);
            }
        }
    }
    if (tid == 0) {
        st.z[s] = z;
        st.mark[s] = 0;
    }
    __syncthreads();
}

// One block per stream, the unmarked ones leaving at once (the start of a streaming set).
__global__ __launch_bounds__(kFitThreads) void k_spot_fit_all(double q, SpotState st)
{
    __shared__ FitShared sh;
    if (st.mark[blockIdx.x])
        spot_fit_stream(sh, blockIdx.x, q, st);
}

// The streams the last update listed, one block each (a grid of one block per stream, the blocks
// past the list's length leaving at once). The next push's update counts in the other counter,
// which block 0 clears (no block of this launch reads it).
__global__ __launch_bounds__(kFitThreads) void k_spot_fit_list(double q, SpotState st)
{
    __shared__ FitShared sh;
    if (blockIdx.x == 0 && threadIdx.x == 0)
        st.count[st.cur ^ 1] = 0;
    if (static_cast<int>(blockIdx.x) < st.count[st.cur])
        spot_fit_stream(sh, st.list[blockIdx.x], q, st);
}

}  // namespace

hipError_t launch_stream_append(const Geometry &g, const void *x_step, int n, int64_t step, void *ring,
                                hipStream_t st)
{
    const int64_t total = static_cast<int64_t>(n) * g.M;
    if (total <= 0)
        return hipSuccess;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    const int slot = static_cast<int>(step % g.W);
    if (g.dtype == ENOVA_F32)
        hipLaunchKernelGGL(k_stream_append<float>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                           static_cast<const float *>(x_step), n, g.M, g.W, slot, static_cast<float *>(ring));
    else
        hipLaunchKernelGGL(k_stream_append<uint16_t>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                           static_cast<const uint16_t *>(x_step), n, g.M, g.W, slot,
                           static_cast<uint16_t *>(ring));
    return hipGetLastError();
}

bool stream_score_supported(const Geometry &g)
{
    return g.mfma_ok && pick_stream(g) != nullptr && stream_lds(g) <= kLdsLimit;
}

hipError_t prepare_stream_score(const Geometry &g)
{
    StreamKernel k = pick_stream(g);
    if (!k)
        return hipErrorInvalidValue;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(stream_lds(g)));
}

hipError_t launch_stream_score(const Geometry &g, const StreamScoreParams &p, hipStream_t st)
{
    if (p.n_streams <= 0)
        return hipSuccess;
    StreamKernel k = pick_stream(g);
    if (!k)
        return hipErrorInvalidValue;
    StreamShape sh;
    sh.M = g.M;
    sh.S = g.S;
    sh.W = g.W;
    sh.Mp = g.Mp;
    sh.Q = g.Q;
    sh.CPR = g.CPR;
    sh.iters = stream_iters(g);
    sh.inv_d = 1.0f / static_cast<float>(g.D);
    const unsigned grid = static_cast<unsigned>((p.n_streams + kStreamNb - 1) / kStreamNb);
    hipLaunchKernelGGL(k, dim3(grid), dim3(kStreamThreads), stream_lds(g), st, p, sh);
    return hipGetLastError();
}

hipError_t launch_spot_init(const float *cal, const int64_t *cal_off, int n, double level,
                            const SpotState &s, hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_spot_init, dim3(static_cast<unsigned>(n)), dim3(256), 0, st, cal, cal_off, level, s);
    return hipGetLastError();
}

hipError_t launch_spot_update(const float *scores, int n, const SpotState &s, uint8_t *flags,
                              hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_spot_update, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, st,
                       scores, n, s, flags);
    return hipGetLastError();
}

hipError_t launch_spot_fit(int n, double q, const SpotState &s, bool all, hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    if (all) {
        hipLaunchKernelGGL(k_spot_fit_all, dim3(static_cast<unsigned>(n)), dim3(kFitThreads), 0, st, q, s);
    } else {
        hipLaunchKernelGGL(k_spot_fit_list, dim3(static_cast<unsigned>(n)), dim3(kFitThreads), 0, st, q, s);
    }
    return hipGetLastError();
}

}  // namespace enova
