// Streaming detection kernels: the ring of each stream's last W steps, the matrix-core scoring of
// every stream's newest window, and per-stream streaming peaks-over-threshold (SPOT, Siffer et
// al. -- the POT method Section IV-B cites; Section V runs the detector in a stream-computing
// job).
//
// Scoring: the newest windows of NBS streams form one tile. Unlike the sliding-window batch
// kernel, no two windows of a tile share data, so each window's D inputs are staged in LDS in
// the padded chunk order of the packed W1 (chunk kappa = q*CPR + c: chunk c of super-row q),
// KS chunks at a time, and the encoder contraction C[h][n] = sum_k W1[h][k] V[n][k] runs on the
// matrix cores slice by slice; the epilogue is the batch kernel's.
//
// SPOT refits run on the device, one block per stream with a new peak, with the batch fit's
// method: Grimshaw's reduction bracketed on geometric 512-point grids of both admissible
// intervals and refined by k-section, the exponential tail always a candidate.
#include <hip/hip_runtime.h>

#include <cmath>

#include "gpd_math.h"
#include "stream_internal.h"
#include "mfma_common.h"

namespace enova {

namespace {

constexpr int kStreamWaves = 4;
constexpr int kStreamThreads = 64 * kStreamWaves;
constexpr size_t kStreamSliceBytes = 48 * 1024;   // LDS for one staged slice of a tile

struct StreamShape {
    int M, S, W, Mp, Q, CPR, KC, KS, KCP, HBT;
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
// HBW hidden blocks per wave, WH waves along the hidden rows, 4/WH window groups of 32 windows.
template <int DT, int HBW, int WH, int ACT>
__global__ __launch_bounds__(kStreamThreads) void k_stream_score(StreamScoreParams p, StreamShape g)
{
    constexpr int NW = kStreamWaves, NT = kStreamThreads;
    constexpr int WN = NW / WH;
    constexpr int NBS = 32 * WN;                   // windows (streams) per tile
    constexpr int EPC = DT == ENOVA_F32 ? 4 : 8;
    extern __shared__ uint4 lds[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const int wh = wave % WH;
    const int wn = wave / WH;
    const int s0 = blockIdx.x * NBS;
    const int M = g.M, Mp = g.Mp, S = g.S, W = g.W, Q = g.Q, CPR = g.CPR, KS = g.KS, KCP = g.KCP;
    const int HBT = g.HBT, HP = 32 * HBT;

    // LDS: the staged slice (later the epilogue's exchange area), window sums, small vectors
    const size_t buf_chunks = static_cast<size_t>(NBS) * KCP;
    constexpr int XCHG = WH > 1 ? epi_xchg_floats(NW, 1) : 0;
    const size_t span = buf_chunks > XCHG / 4 ? buf_chunks : XCHG / 4;
    uint4 *buf = lds;
    float *wsum = reinterpret_cast<float *>(lds + span);
    float *s_b1 = wsum + NBS;
    float *s_bd1 = s_b1 + HP;
    float *s_u = s_bd1 + HP;
    float *s_bh = s_u + HP;
    for (int i = tid; i < HP; i += NT) {
        s_b1[i] = p.b1[i];
        s_bd1[i] = p.bd1[i];
        s_u[i] = p.u[i];
    }
    if (tid < 32)
        s_bh[tid] = p.bh[tid];

    const int nl = wn * 32 + (lane & 31);          // this lane's window in the tile
    const int brow = nl * KCP;
    v16f acc[HBW][1];
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc[hb][0][r] = 0.0f;
    v16f acc2[HBW];                                // fp32: the odd reduction slots
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc2[hb][r] = 0.0f;
    float my_sum = 0.0f;                           // thread nl < NBS: window nl's sum of v

    // padding-free windows (M a multiple of the chunk's elements) stage with vector loads
    const bool linear = Mp == M && M % EPC == 0;
    const uint4 *ap = p.w1p + (wh * HBW) * 64 + lane;
    for (int k0 = 0; k0 < g.KC; k0 += KS) {
        const int ks = g.KC - k0 < KS ? g.KC - k0 : KS;   // a multiple of 16
        __syncthreads();                                   // the previous slice is consumed
        if (linear) {
            // chunk kappa is elements [kappa*EPC, +EPC) of the window, contiguous in the ring,
            // with consecutive metrics: one 16-byte load of x and EPC/4 of mean and std each;
            // SU chunks per thread in flight
            constexpr int SU = 4;
            for (int base = tid; base < NBS * ks; base += NT * SU) {
                uint4 raw[SU];
                float4 mu[SU][EPC / 4], sd[SU][EPC / 4];
                bool ok[SU];
#pragma unroll
                for (int u = 0; u < SU; ++u) {
                    const int idx = base + u * NT;
                    const int w = idx / ks;
                    const int kc = idx - w * ks;
                    const int s = s0 + w;
                    const int e0 = (k0 + kc) * EPC;
                    ok[u] = idx < NBS * ks && s < p.n_streams && e0 < W * M;
                    if (ok[u]) {
                        const int64_t at = (static_cast<int64_t>(s) * 2 * W + p.first_slot) * M + e0;
                        if constexpr (DT == ENOVA_F32)
                            raw[u] = *reinterpret_cast<const uint4 *>(static_cast<const float *>(p.ring) + at);
                        else
                            raw[u] = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p.ring) + at);
                        const int64_t sm = static_cast<int64_t>(s) * M + e0 % M;
#pragma unroll
                        for (int h = 0; h < EPC / 4; ++h) {
                            mu[u][h] = reinterpret_cast<const float4 *>(p.mean + sm)[h];
                            sd[u][h] = reinterpret_cast<const float4 *>(p.std + sm)[h];
                        }
                    }
                }
#pragma unroll
                for (int u = 0; u < SU; ++u) {
                    const int idx = base + u * NT;
                    if (idx >= NBS * ks)
                        continue;
                    const int w = idx / ks;
                    const int kc = idx - w * ks;
                    float v[EPC];
                    if (ok[u]) {
                        float xv[EPC], mv[EPC], sv[EPC];
                        if constexpr (DT == ENOVA_F32) {
                            xv[0] = __uint_as_float(raw[u].x);
                            xv[1] = __uint_as_float(raw[u].y);
                            xv[2] = __uint_as_float(raw[u].z);
                            xv[3] = __uint_as_float(raw[u].w);
                        } else {
                            xv[0] = bf16_lo(raw[u].x);
                            xv[1] = bf16_hi(raw[u].x);
                            xv[2] = bf16_lo(raw[u].y);
                            xv[3] = bf16_hi(raw[u].y);
                            xv[4] = bf16_lo(raw[u].z);
                            xv[5] = bf16_hi(raw[u].z);
                            xv[6] = bf16_lo(raw[u].w);
                            xv[7] = bf16_hi(raw[u].w);
                        }
#pragma unroll
                        for (int h = 0; h < EPC / 4; ++h) {
                            mv[4 * h + 0] = mu[u][h].x;
                            mv[4 * h + 1] = mu[u][h].y;
                            mv[4 * h + 2] = mu[u][h].z;
                            mv[4 * h + 3] = mu[u][h].w;
                            sv[4 * h + 0] = sd[u][h].x;
                            sv[4 * h + 1] = sd[u][h].y;
                            sv[4 * h + 2] = sd[u][h].z;
                            sv[4 * h + 3] = sd[u][h].w;
                        }
#pragma unroll
                        for (int e = 0; e < EPC; ++e)
                            v[e] = (xv[e] - mv[e]) * (1.0f / sv[e]);
                    } else {
#pragma unroll
                        for (int e = 0; e < EPC; ++e)
                            v[e] = 0.0f;
                    }
                    uint4 out;
                    if constexpr (DT == ENOVA_F32) {
                        out.x = __float_as_uint(v[0]);
                        out.y = __float_as_uint(v[1]);
                        out.z = __float_as_uint(v[2]);
                        out.w = __float_as_uint(v[3]);
                    } else {
                        out.x = pack_bf16x2(v[0], v[1]);
                        out.y = pack_bf16x2(v[2], v[3]);
                        out.z = pack_bf16x2(v[4], v[5]);
                        out.w = pack_bf16x2(v[6], v[7]);
                    }
                    buf[w * KCP + kc] = out;
                }
            }
        } else {
            for (int idx = tid; idx < NBS * ks; idx += NT) {
                const int w = idx / ks;
                const int kc = idx - w * ks;
                const int kappa = k0 + kc;
                const int q = kappa / CPR;
                const int c = kappa - q * CPR;
                const int s = s0 + w;
                float v[EPC];
    #pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const int jj = c * EPC + e;
                    const int tt = jj / Mp;
                    const int m = jj - tt * Mp;
                    const int step = q * S + tt;
                    float val = 0.0f;
                    if (s < p.n_streams && q < Q && m < M && step < W) {
                        const int64_t at = (static_cast<int64_t>(s) * 2 * W + p.first_slot + step) * M + m;
                        const float x = load_x<DT>(p.ring, at);
                        const int64_t sm = static_cast<int64_t>(s) * M + m;
                        val = (x - p.mean[sm]) * (1.0f / p.std[sm]);
                    }
                    v[e] = val;
                }
                uint4 out;
                if constexpr (DT == ENOVA_F32) {
                    out.x = __float_as_uint(v[0]);
                    out.y = __float_as_uint(v[1]);
                    out.z = __float_as_uint(v[2]);
                    out.w = __float_as_uint(v[3]);
                } else {
                    out.x = pack_bf16x2(v[0], v[1]);
                    out.y = pack_bf16x2(v[2], v[3]);
                    out.z = pack_bf16x2(v[4], v[5]);
                    out.w = pack_bf16x2(v[6], v[7]);
                }
                buf[w * KCP + kc] = out;
            }
        }
        __syncthreads();
        if (tid < NBS) {
            // the window's sum of the staged (rounded) values, in a fixed order
            for (int kc = 0; kc < ks; ++kc) {
                const uint4 q4 = buf[tid * KCP + kc];
                if constexpr (DT == ENOVA_F32) {
                    my_sum += __uint_as_float(q4.x) + __uint_as_float(q4.y) + __uint_as_float(q4.z) +
                              __uint_as_float(q4.w);
                } else {
                    my_sum += bf16_lo(q4.x) + bf16_hi(q4.x) + bf16_lo(q4.y) + bf16_hi(q4.y) +
                              bf16_lo(q4.z) + bf16_hi(q4.z) + bf16_lo(q4.w) + bf16_hi(q4.w);
                }
            }
        }
        // contraction over the slice: step i covers chunks 2i (lanes 0..31) and 2i+1 (32..63).
        // W1 fragments run PD steps ahead in a register ring (a step is only a few matrix ops);
        // fp32 alternates two accumulators so consecutive ops do not wait on each other.
        constexpr int PD = 8;
        static_assert(PD <= kPrefetchSteps, "the packed W1 carries kPrefetchSteps zero steps");
        const int nsteps = ks / 2;                 // a multiple of PD
        const int64_t st0 = k0 / 2;
        uint4 a[PD][HBW];
#pragma unroll
        for (int j = 0; j < PD; ++j)
#pragma unroll
            for (int hb = 0; hb < HBW; ++hb)
                a[j][hb] = ap[((st0 + j) * HBT + hb) * 64];
        for (int i = 0; i < nsteps; i += PD) {
#pragma unroll
            for (int j = 0; j < PD; ++j) {
                const uint4 bq = buf[brow + 2 * (i + j) + half];
                if constexpr (DT == ENOVA_F32) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float bv = __uint_as_float(e == 0 ? bq.x : e == 1 ? bq.y : e == 2 ? bq.z : bq.w);
#pragma unroll
                        for (int hb = 0; hb < HBW; ++hb) {
                            const float av = __uint_as_float(e == 0 ? a[j][hb].x : e == 1 ? a[j][hb].y
                                                            : e == 2 ? a[j][hb].z : a[j][hb].w);
                            if (e & 1)
                                acc2[hb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc2[hb], 0, 0, 0);
                            else
                                acc[hb][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[hb][0], 0, 0, 0);
                        }
                    }
                } else {
#pragma unroll
                    for (int hb = 0; hb < HBW; ++hb)
                        acc[hb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(v8bf, a[j][hb]), __builtin_bit_cast(v8bf, bq), acc[hb][0], 0, 0, 0);
                }
                // steps up to KC/2 + PD - 1 are read: the packed W1 carries zero steps past the end
#pragma unroll
                for (int hb = 0; hb < HBW; ++hb)
                    a[j][hb] = ap[((st0 + i + j + PD) * HBT + hb) * 64];
            }
        }
    }
    if constexpr (DT == ENOVA_F32) {
#pragma unroll
        for (int hb = 0; hb < HBW; ++hb)
            acc[hb][0] += acc2[hb];
    }
    __syncthreads();                               // the staging buffer becomes the exchange area
    if (tid < NBS)
        wsum[tid] = my_sum;
    __syncthreads();

    const EpiArgs ea{p.whp, p.wd1p, s_b1, s_bd1, s_u, s_bh, reinterpret_cast<float *>(buf),
                     lane, half, wave, wh, wn};
    score_epilogue<DT, HBW, 1, WH, NW, ACT>(acc, ea, [&](int, float sc, float dot) __attribute__((always_inline)) {
        const int s = s0 + nl;
        if (wh == 0 && half == 0 && s < p.n_streams) {
            p.scores[s] = sc;
            if (p.md)
                p.md[s] = wsum[nl] * g.inv_d - (dot + p.sum_bd2) * g.inv_d;
        }
    });
}

using StreamKernel = void (*)(StreamScoreParams, StreamShape);

template <int DT, int ACT>
StreamKernel pick_stream(int hb)
{
    switch (hb) {
    case 1: return k_stream_score<DT, 1, 1, ACT>;
    case 2: return k_stream_score<DT, 1, 2, ACT>;
    case 4: return k_stream_score<DT, 1, 4, ACT>;
    case 8: return k_stream_score<DT, 2, 4, ACT>;
    default: return nullptr;
    }
}

StreamKernel pick_stream(const Geometry &g)
{
    const bool relu = g.act == ENOVA_RELU;
    if (g.dtype == ENOVA_F32)
        return relu ? pick_stream<ENOVA_F32, ENOVA_RELU>(g.HB) : pick_stream<ENOVA_F32, ENOVA_TANH>(g.HB);
    return relu ? pick_stream<ENOVA_BF16, ENOVA_RELU>(g.HB) : pick_stream<ENOVA_BF16, ENOVA_TANH>(g.HB);
}

// Tile shape of the streaming kernel for g: windows per tile, chunks per slice and LDS bytes.
struct StreamPlan {
    int nbs, ks, kcp;
    size_t lds;
};

StreamPlan stream_plan(const Geometry &g)
{
    StreamPlan sp{};
    const int wh = g.HB < 4 ? g.HB : 4;
    sp.nbs = 32 * (kStreamWaves / wh);
    int ks = static_cast<int>(kStreamSliceBytes / (static_cast<size_t>(sp.nbs) * 16)) - 1;
    ks = ks / 16 * 16;
    if (ks < 16)
        ks = 16;
    if (ks > g.KC)
        ks = g.KC;
    sp.ks = ks;
    sp.kcp = ks + 1;                               // odd pitch: the 32 windows of a fragment read spread over the banks
    const size_t buf = static_cast<size_t>(sp.nbs) * sp.kcp * 16;
    const size_t xchg = wh > 1 ? static_cast<size_t>(epi_xchg_floats(kStreamWaves, 1)) * sizeof(float) : 0;
    sp.lds = (buf > xchg ? buf : xchg) + (static_cast<size_t>(sp.nbs) + 3 * static_cast<size_t>(g.Hp) + 32) * sizeof(float);
    return sp;
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
                st.list[atomicAdd(st.count, 1)] = s;
            }
        }
    }
    if (flags)
        flags[s] = f;
}

constexpr int kFitGrid = 512;       // grid points per admissible interval
constexpr int kFitInterior = 63;    // k-section points per bracket and round
constexpr int kFitRounds = 40;
constexpr int kFitMaxBrackets = 64; // sign changes kept per fit
constexpr int kFitBatch = 16;       // brackets refined per evaluation batch

struct FitShared {
    double xs[2 * kFitGrid];
    double sa[2 * kFitGrid];
    double sb[2 * kFitGrid];
    double red[256], red2[256];
    double blo[kFitMaxBrackets], bhi[kFitMaxBrackets], broot[kFitMaxBrackets];
    int bneg[kFitMaxBrackets], bdone[kFitMaxBrackets], bround[kFitMaxBrackets];
    double roots[2 * kFitMaxBrackets];
    int batch[kFitBatch];
    int coll[kFitBatch];         // 1: the batch bracket's points are not strictly inside it
    int scan[256];
    int nbr, nroots, npts, ngrid, nbatch;
    double ysum, ymin, ymax;
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

// sa/sb at the first npts (<= 1024) points of sh.xs over all N excesses. Many points: each
// thread takes up to four; few points: T threads share a point (power of two, T * npts <= 256),
// each summing every T-th excess, and the T partial sums are added in order. A fixed order
// either way.
__device__ void fit_eval(FitShared &sh, const double *y, int N)
{
    const int np = sh.npts;
    if (np > 128) {
        // up to four points per thread, evaluated side by side (independent dependency chains)
        double x[4], a[4], b[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int p = threadIdx.x + 256 * k;
            x[k] = p < np ? sh.xs[p] : 0.0;
            a[k] = 0.0;
            b[k] = 0.0;
        }
        for (int i = 0; i < N; ++i) {
            const double yi = y[i];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                double ta, tb;
                gpd_terms(x[k] * yi, ta, tb);
                a[k] += ta;
                b[k] += tb;
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int p = threadIdx.x + 256 * k;
            if (p < np) {
                sh.sa[p] = a[k];
                sh.sb[p] = b[k];
            }
        }
        __syncthreads();
        return;
    }
    int T = 1;
    while (T < 64 && 2 * T * np <= 256)
        T *= 2;
    const int per = 256 / T;
    const int part = threadIdx.x % T;
    for (int p0 = 0; p0 < np; p0 += per) {
        const int p = p0 + static_cast<int>(threadIdx.x) / T;
        double a = 0.0, b = 0.0;
        if (p < np) {
            const double x = sh.xs[p];
            for (int i = part; i < N; i += T) {
                double ta, tb;
                gpd_terms(x * y[i], ta, tb);
                a += ta;
                b += tb;
            }
        }
        if (T == 1) {
            if (p < np) {
                sh.sa[p] = a;
                sh.sb[p] = b;
            }
        } else {
            sh.red[threadIdx.x] = a;
            sh.red2[threadIdx.x] = b;
            __syncthreads();
            if (part == 0 && p < np) {
                double sa = 0.0, sb = 0.0;
                for (int k = 0; k < T; ++k) {
                    sa += sh.red[threadIdx.x + k];
                    sb += sh.red2[threadIdx.x + k];
                }
                sh.sa[p] = sa;
                sh.sb[p] = sb;
            }
            __syncthreads();
        }
    }
    __syncthreads();
}

// w = b - a - a b at the first npts points, into sh.sa (every thread a share).
__device__ void fit_w_all(FitShared &sh, double n)
{
    for (int p = threadIdx.x; p < sh.npts; p += 256)
        sh.sa[p] = fit_w(sh.sa[p], sh.sb[p], n);
    __syncthreads();
}

// Fixed-order block reduction (sum, min or max) of one value per thread.
template <int OP>
__device__ double block_reduce(FitShared &sh, double v)
{
    sh.red[threadIdx.x] = v;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if (threadIdx.x < w) {
            const double o = sh.red[threadIdx.x + w];
            double &m = sh.red[threadIdx.x];
            m = OP == 0 ? m + o : (OP == 1 ? fmin(m, o) : fmax(m, o));
        }
        __syncthreads();
    }
    const double r = sh.red[0];
    __syncthreads();
    return r;
}

// Refit of z for one marked stream by one block: N_t <= 1 gives t; 2 <= N_t < 10 the method of
// moments with the unbiased sample variance; N_t >= 10 maximum likelihood.
__device__ void spot_fit_stream(FitShared &sh, int s, double q, const SpotState &st)
{
    const int tid = threadIdx.x;
    const int N = st.npk[s];
    const double t = st.t[s];
    const double n = static_cast<double>(st.cnt[s]);
    const double *y = st.peaks + static_cast<int64_t>(s) * st.cap;
    double z = t;
    if (N >= 2) {
        double ps = 0.0, pmin = INFINITY, pmax = -INFINITY;
        for (int i = tid; i < N; i += 256) {
            ps += y[i];
            pmin = fmin(pmin, y[i]);
            pmax = fmax(pmax, y[i]);
        }
        const double ysum = block_reduce<0>(sh, ps);
        const double ymin = block_reduce<1>(sh, pmin);
        const double ymax = block_reduce<2>(sh, pmax);
        const double Nd = static_cast<double>(N);
        const double ymean = ysum / Nd;
        if (N < 10) {
            double pv = 0.0;
            for (int i = tid; i < N; i += 256)
                pv += (y[i] - ymean) * (y[i] - ymean);
            const double s2 = block_reduce<0>(sh, pv) / (Nd - 1.0);
            if (s2 > 0.0) {
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
            const int left_at = 0, right_at = has_left ? kFitGrid : 0;
            for (int i = tid; i < kFitGrid; i += 256) {
                if (has_left) {
                    const double zlo = log(f0 / (1.0 - f0)), zhi = 30.0;
                    const double zz = zlo + (zhi - zlo) * static_cast<double>(i) / static_cast<double>(kFitGrid - 1);
                    sh.xs[left_at + i] = -(1.0 / (1.0 + exp(-zz))) / ymax;
                }
                if (has_right)
                    sh.xs[right_at + i] = eps * pow(right / eps, static_cast<double>(i) / static_cast<double>(kFitGrid - 1));
            }
            if (tid == 0) {
                sh.ngrid = (has_left ? 1 : 0) + (has_right ? 1 : 0);
                sh.npts = sh.ngrid * kFitGrid;
                sh.nbr = 0;
                sh.nroots = 0;
            }
            __syncthreads();
            fit_eval(sh, y, N);
            fit_w_all(sh, Nd);
            // every grid point: an exact root, and/or a sign change to the next point of its grid;
            // both kept in grid order (ordered compaction over the block)
            for (int p0 = 0; p0 < sh.npts; p0 += 256) {
                const int i = p0 + tid;
                int root = 0, br = 0;
                if (i < sh.npts) {
                    const int gi = i % kFitGrid;
                    const double wi = sh.sa[i];
                    if (wi == 0.0)
                        root = 1;
                    else if (gi + 1 < kFitGrid && wi * sh.sa[i + 1] < 0.0)
                        br = 1;
                }
                sh.scan[tid] = root | (br << 16);
                __syncthreads();
                for (int off = 1; off < 256; off <<= 1) {
                    const int v = tid >= off ? sh.scan[tid - off] : 0;
                    __syncthreads();
                    sh.scan[tid] += v;
                    __syncthreads();
                }
                const int incl = sh.scan[tid];
                const int r_at = sh.nroots + (incl & 0xffff) - root;
                const int b_at = sh.nbr + (incl >> 16) - br;
                if (root && r_at < 2 * kFitMaxBrackets)
                    sh.roots[r_at] = sh.xs[i];
                if (br && b_at < kFitMaxBrackets) {
                    const double x0 = sh.xs[i], x1 = sh.xs[i + 1];
                    const double wi = sh.sa[i], wn = sh.sa[i + 1];
                    sh.blo[b_at] = x0 < x1 ? x0 : x1;
                    sh.bhi[b_at] = x0 < x1 ? x1 : x0;
                    sh.bneg[b_at] = x0 < x1 ? (wi < 0.0) : (wn < 0.0);
                    sh.bdone[b_at] = 0;
                    sh.bround[b_at] = 0;
                    sh.broot[b_at] = 0.0;
                }
                __syncthreads();
                if (tid == 255) {
                    const int nr = sh.nroots + (incl & 0xffff), nb = sh.nbr + (incl >> 16);
                    sh.nroots = nr < 2 * kFitMaxBrackets ? nr : 2 * kFitMaxBrackets;
                    sh.nbr = nb < kFitMaxBrackets ? nb : kFitMaxBrackets;
                }
                __syncthreads();
            }
            // k-section, up to kFitBatch open brackets per evaluation: the points and w are
            // computed by all threads, one thread keeps the brackets
            for (;;) {
                if (tid == 0) {
                    sh.nbatch = 0;
                    for (int b = 0; b < sh.nbr && sh.nbatch < kFitBatch; ++b) {
                        if (sh.bdone[b])
                            continue;
                        if (sh.bround[b] >= kFitRounds) {
                            sh.bdone[b] = 1;
                            sh.broot[b] = 0.5 * (sh.blo[b] + sh.bhi[b]);
                            continue;
                        }
                        sh.coll[sh.nbatch] = 0;
                        sh.batch[sh.nbatch++] = b;
                    }
                    sh.npts = sh.nbatch * kFitInterior;
                }
                __syncthreads();
                if (sh.nbatch == 0)
                    break;
                for (int i = tid; i < sh.npts; i += 256) {
                    const int k = i / kFitInterior, j = i - k * kFitInterior + 1;
                    const int b = sh.batch[k];
                    const double lo = sh.blo[b], hi = sh.bhi[b];
                    sh.xs[i] = lo + (hi - lo) * static_cast<double>(j) / (kFitInterior + 1);
                }
                __syncthreads();
                for (int i = tid; i < sh.npts; i += 256) {
                    // a bracket that can no longer shrink: its points are not strictly inside
                    const int k = i / kFitInterior, j = i - k * kFitInterior + 1;
                    const int b = sh.batch[k];
                    const double prev = j == 1 ? sh.blo[b] : sh.xs[i - 1];
                    if (!(sh.xs[i] > prev) || !(sh.xs[i] < sh.bhi[b]))
                        sh.coll[k] = 1;
                }
                fit_eval(sh, y, N);
                fit_w_all(sh, Nd);
                if (tid == 0) {
                    for (int k = 0; k < sh.nbatch; ++k) {
                        const int b = sh.batch[k];
                        if (sh.coll[k]) {
                            sh.bdone[b] = 1;
                            sh.broot[b] = 0.5 * (sh.blo[b] + sh.bhi[b]);
                            continue;
                        }
                        double new_lo = sh.blo[b], new_hi = sh.bhi[b];
                        for (int j = 0; j < kFitInterior; ++j) {
                            const int pi = k * kFitInterior + j;
                            const double wj = sh.sa[pi];
                            if (wj == 0.0) {
                                sh.bdone[b] = 1;
                                sh.broot[b] = sh.xs[pi];
                                break;
                            }
                            if ((wj < 0.0) != (sh.bneg[b] != 0)) {
                                new_hi = sh.xs[pi];
                                break;
                            }
                            new_lo = sh.xs[pi];
                        }
                        if (!sh.bdone[b]) {
                            sh.blo[b] = new_lo;
                            sh.bhi[b] = new_hi;
                        }
                        sh.bround[b] += 1;
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
    if (tid == 0) {
        st.z[s] = z;
        st.mark[s] = 0;
    }
    __syncthreads();
}

// One block per stream, the unmarked ones leaving at once (the start of a streaming set).
__global__ __launch_bounds__(256) void k_spot_fit_all(double q, SpotState st)
{
    __shared__ FitShared sh;
    if (st.mark[blockIdx.x])
        spot_fit_stream(sh, blockIdx.x, q, st);
}

// The streams the last update listed, spread over a fixed grid of blocks (a push refits a few
// percent of the streams; launching a block per stream would mostly launch empty blocks).
__global__ __launch_bounds__(256) void k_spot_fit_list(double q, SpotState st)
{
    __shared__ FitShared sh;
    const int cnt = *st.count;
    for (int i = blockIdx.x; i < cnt; i += gridDim.x)
        spot_fit_stream(sh, st.list[i], q, st);
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
    return g.mfma_ok && pick_stream(g) != nullptr && stream_plan(g).lds <= kLdsLimit;
}

hipError_t prepare_stream_score(const Geometry &g)
{
    StreamKernel k = pick_stream(g);
    if (!k)
        return hipErrorInvalidValue;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(kLdsLimit));
}

hipError_t launch_stream_score(const Geometry &g, const StreamScoreParams &p, hipStream_t st)
{
    if (p.n_streams <= 0)
        return hipSuccess;
    StreamKernel k = pick_stream(g);
    if (!k)
        return hipErrorInvalidValue;
    const StreamPlan sp = stream_plan(g);
    StreamShape sh;
    sh.M = g.M;
    sh.S = g.S;
    sh.W = g.W;
    sh.Mp = g.Mp;
    sh.Q = g.Q;
    sh.CPR = g.CPR;
    sh.KC = g.KC;
    sh.KS = sp.ks;
    sh.KCP = sp.kcp;
    sh.HBT = g.HB;
    sh.inv_d = 1.0f / static_cast<float>(g.D);
    const unsigned grid = static_cast<unsigned>((p.n_streams + sp.nbs - 1) / sp.nbs);
    hipLaunchKernelGGL(k, dim3(grid), dim3(kStreamThreads), sp.lds, st, p, sh);
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
    hipError_t e = hipMemsetAsync(s.count, 0, sizeof(int), st);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_spot_update, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, st,
                       scores, n, s, flags);
    return hipGetLastError();
}

hipError_t launch_spot_fit(int n, double q, const SpotState &s, bool all, hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    if (all) {
        hipLaunchKernelGGL(k_spot_fit_all, dim3(static_cast<unsigned>(n)), dim3(256), 0, st, q, s);
    } else {
        int dev = 0, cus = 256;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            cus = 256;
        const int blocks = n < 2 * cus ? n : 2 * cus;
        hipLaunchKernelGGL(k_spot_fit_list, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, q, s);
    }
    return hipGetLastError();
}

}  // namespace enova
