// Fused detector-output variants (Section IV-B) for fp32 detectors: the KL score, md, the
// per-metric md vector and the reconstruction error of every window in one launch, without
// materialising the normalised windows.
//
// A tile is 256 consecutive windows of one stream. Its raw super-rows are staged in LDS once
// (coalesced 16-byte loads, no arithmetic), exactly as the scoring kernel stages its normalised
// ones, so one staged element again feeds up to Q windows (implicit im2col). Normalisation
// v = (x - mean) / std is per window and per metric (the window's own fp64 statistics, or the
// stream's reference statistics), so it cannot be applied at staging; instead every lane
// normalises the window fragments it feeds to the matrix cores, in registers:
//
//   * the lane that carries window n and lane half h meets only the metrics of one or two fixed
//     16-byte metric chunks (the reduction walks chunk 2i + h at step i, and a super-row holds a
//     whole number of metric chunks), so it computes those metrics' statistics of its own window
//     from the staged rows (one fp64 shifted pass) and keeps 1/std and -mean/std in registers;
//   * each window fragment read from LDS is turned into v with one fused multiply-add per
//     element before the encoder's 32x32x2 matrix ops (four per fragment and hidden block).
//
// The epilogue chains the posterior heads and the decoder's hidden layer on the matrix cores as
// the scoring kernel does (the 32x32 accumulator layout is the next op's B operand), keeps the
// decoder hidden activations hd in registers and runs the decoder output m' = Wd2 hd + bd2 as a
// further chain: output block ob (32 consecutive elements j = 32 ob + row of the window) has, in
// lane l and register r, element 32 ob + 8 (r/4) + 4 (l/32) + r%4 -- four consecutive elements,
// i.e. one 16-byte chunk, per group of four registers, and always a chunk of the lane's own
// metrics. So v is rebuilt from the staged row with the lane's constants, d = v - m' is reduced
// per metric and squared in registers, and only the per-window results are written.
#include <hip/hip_runtime.h>

#include "mfma_common.h"
#include "variants_internal.h"

namespace enova {

namespace {

constexpr int kFusedWaves = 4;
constexpr int kFusedNbw = 2;   // 32-window blocks per wave

__device__ __forceinline__ float4 fma4(float4 x, float4 a, float4 b)
{
    return make_float4(fmaf(x.x, a.x, b.x), fmaf(x.y, a.y, b.y), fmaf(x.z, a.z, b.z), fmaf(x.w, a.w, b.w));
}

__device__ __forceinline__ float comp(float4 v, int e)
{
    return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
}

// HB: 32-row hidden blocks (hidden units padded to 32 HB); MC: 16-byte metric chunks per step
// (M = 4 MC). Every wave owns all hidden rows and two 32-window blocks.
template <int HB, int MC, int ACT>
__global__ __launch_bounds__(kFusedWaves * 64, 2) void k_ext_fused(ExtFusedParams p, ExtFusedShape g)
{
    constexpr int NT = kFusedWaves * 64;
    constexpr int NBW = kFusedNbw;
    constexpr int NB = kExtFusedNb;
    static_assert(NB == kFusedWaves * NBW * 32, "tile");
    constexpr int CH = MC == 4 ? 2 : 1;   // metric chunks a lane meets
    constexpr int HP = 32 * HB;
    constexpr int N_WHP = HB * 16 * 64, N_WD1P = HB * 8 * 64;
    constexpr int N_CONST = N_WHP + N_WD1P + 3 * HP + 32;
    static_assert(N_CONST % 4 == 0, "16-byte constant block");
    extern __shared__ uint4 lds[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;

    // ---- tile -> (stream, first window)
    const int64_t b = blockIdx.x;
    const int s = p.tile_stream[b];
    if (s < 0)
        return;
    const int64_t k0 = (b - p.tile_off[s]) * NB;
    const int64_t ns = p.woff[s + 1] - p.woff[s];
    const int nv = static_cast<int>(ns - k0 < NB ? ns - k0 : NB);
    const int64_t srow = p.soff[s];
    const int64_t T = p.soff[s + 1] - srow;
    const int Q = g.Q, CPR = g.CPR, CPRP = g.CPRP, S = g.S, W = g.W;
    constexpr int M = 4 * MC;
    const int nrows = nv + Q - 1 + g.spare;

    // LDS: heads fragments, decoder hidden-layer fragments, b1, bd1, u, head biases (the host's
    // contiguous block), bd2, then the raw super-rows at a pitch of CPRP chunks
    float *s_whp = reinterpret_cast<float *>(lds);
    float *s_wd1p = s_whp + N_WHP;
    float *s_b1 = s_wd1p + N_WD1P;
    float *s_bd1 = s_b1 + HP;
    float *s_bh = s_bd1 + 2 * HP;
    float *s_bd2 = s_whp + N_CONST;   // [D]
    uint4 *seg = lds + N_CONST / 4 + g.D / 4;
    {
        const float4 *src = reinterpret_cast<const float4 *>(p.cst);
        float4 *dst = reinterpret_cast<float4 *>(s_whp);
        for (int i = tid; i < N_CONST / 4; i += NT)
            dst[i] = src[i];
        const float4 *src2 = reinterpret_cast<const float4 *>(p.bd2);
        float4 *dst2 = reinterpret_cast<float4 *>(s_bd2);
        for (int i = tid; i < g.D / 4; i += NT)
            dst2[i] = src2[i];
    }

    // ---- stage the tile's super-rows: one contiguous span of the stream (zero past its end)
    {
        constexpr int SU = 8;
        const int n_chunks = nrows * CPR;
        const int64_t avail = (T - k0 * S) * (M / 4);   // whole chunks left in the stream
        const uint4 *src = reinterpret_cast<const uint4 *>(p.x + (srow + k0 * S) * M);
        for (int base = tid; base < n_chunks; base += NT * SU) {
            uint4 v[SU];
#pragma unroll
            for (int u = 0; u < SU; ++u) {
                const int idx = base + u * NT;
                v[u] = make_uint4(0u, 0u, 0u, 0u);
                if (idx < n_chunks && idx < avail)
                    v[u] = src[idx];
            }
#pragma unroll
            for (int u = 0; u < SU; ++u) {
                const int idx = base + u * NT;
                if (idx < n_chunks) {
                    const int r = idx / CPR;
                    seg[r * CPRP + (idx - r * CPR)] = v[u];
                }
            }
        }
    }
    __syncthreads();

    const int wn0 = wave * NBW * 32;
    const bool wave_active = wn0 < nv;
    if (!wave_active)
        return;   // no barrier follows
    int rb[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int n = wn0 + nb * 32 + (lane & 31);
        rb[nb] = (n < nv ? n : nv - 1) * CPRP;   // idle columns evaluate a valid window
    }
    // the metric chunk of this lane's j-th constant set
    auto mchunk = [&](int j) { return MC == 4 ? 2 * j + half : (MC == 2 ? half : 0); };

    // ---- per-window normalisation constants: v = x * ca + cb (ca = 1/std, cb = -mean/std)
    float4 ca[NBW][CH], cb[NBW][CH];
    if (p.norm == ENOVA_NORM_WINDOW) {
        const double inv_w = 1.0 / W;
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                // element (t, metric) of the window: super-row t / S, chunk (t % S) MC + metric chunk
                const int c0 = rb[nb] + mchunk(j);
                const float4 k4 = reinterpret_cast<const float4 &>(seg[c0]);
                double s1[4] = {0.0, 0.0, 0.0, 0.0}, s2[4] = {0.0, 0.0, 0.0, 0.0};
                int q = 0, ts = 0;
                for (int t = 0; t < W; ++t) {
                    const float4 x4 = reinterpret_cast<const float4 &>(seg[c0 + q * CPRP + ts * MC]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const double d = static_cast<double>(comp(x4, e)) - static_cast<double>(comp(k4, e));
                        s1[e] += d;
                        s2[e] = fma(d, d, s2[e]);
                    }
                    if (++ts == S) {
                        ts = 0;
                        ++q;
                    }
                }
                float av[4], bv[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // shifted sums (shift = the window's first value): mean and population std
                    const double mean = static_cast<double>(comp(k4, e)) + s1[e] * inv_w;
                    double var = (s2[e] - s1[e] * s1[e] * inv_w) * inv_w;
                    var = var > 0.0 ? var : 0.0;
                    double sd = sqrt(var);
                    if (sd <= 1e-6 * fmax(1.0, fabs(mean)))
                        sd = 1.0;   // constant metric inside the window
                    av[e] = static_cast<float>(1.0 / sd);
                    bv[e] = static_cast<float>(-mean / sd);
                }
                ca[nb][j] = make_float4(av[0], av[1], av[2], av[3]);
                cb[nb][j] = make_float4(bv[0], bv[1], bv[2], bv[3]);
            }
    } else {
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            const int64_t e0 = static_cast<int64_t>(s) * M + 4 * mchunk(j);
            float av[4], bv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const double sd = static_cast<double>(p.std[e0 + e]);
                av[e] = static_cast<float>(1.0 / sd);
                bv[e] = static_cast<float>(-static_cast<double>(p.mean[e0 + e]) / sd);
            }
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                ca[nb][j] = make_float4(av[0], av[1], av[2], av[3]);
                cb[nb][j] = make_float4(bv[0], bv[1], bv[2], bv[3]);
            }
        }
    }

    // ---- encoder: C[h][n] = sum_k W1[h][k] v[n][k], window fragments normalised in registers
    v16f acc[HB][NBW];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[hb][nb][r] = 0.0f;
    {
        const int nsteps = g.KC / 2;   // a multiple of PD
        const uint4 *ap = p.w1p + lane;
        const int dpitch = CPRP - CPR;
        int cc = half % CPR;
        int koff = (half / CPR) * CPRP + cc;
        auto advance = [&]() {
            const bool wrap = cc + 2 >= CPR;
            cc = cc + 2 - (wrap ? CPR : 0);
            koff += 2 + (wrap ? dpitch : 0);
        };
        constexpr int PD = 2, PB = 1, RB = 2 * PB;
        uint4 a[PD][HB], bq[RB][NBW];
#pragma unroll
        for (int j = 0; j < PD; ++j) {
#pragma unroll
            for (int hb = 0; hb < HB; ++hb)
                a[j][hb] = ap[(j * HB + hb) * 64];
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
            bq[0][nb] = seg[rb[nb] + koff];
        advance();
        // prefetches past the last step read the packed W1's zero steps and the spare rows
        const uint4 *api = ap + PD * HB * 64;
        for (int i = 0; i < nsteps; i += PD) {
#pragma unroll
            for (int j = 0; j < PD; ++j) {
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    bq[(j + PB) % RB][nb] = seg[rb[nb] + koff];
                advance();
                // step i + j meets metric chunk (2 (i + j) + half) mod MC: constant set j mod 2
                const int cj = CH == 2 ? (j & 1) : 0;
                float4 vb[NBW];
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    vb[nb] = fma4(reinterpret_cast<const float4 &>(bq[j % RB][nb]), ca[nb][cj], cb[nb][cj]);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int hb = 0; hb < HB; ++hb) {
                        const float av = __uint_as_float(e == 0 ? a[j][hb].x : e == 1 ? a[j][hb].y
                                                        : e == 2 ? a[j][hb].z : a[j][hb].w);
#pragma unroll
                        for (int nb = 0; nb < NBW; ++nb)
                            acc[hb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, comp(vb[nb], e), acc[hb][nb],
                                                                               0, 0, 0);
                    }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int hb = 0; hb < HB; ++hb)
                    a[j][hb] = api[(j * HB + hb) * 64];
            }
            api += PD * HB * 64;
        }
    }

    // ---- posterior heads and KL score (rows 0..15 mean, 16..31 log-variance)
    v16f z[NBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            z[i][r] = 0.0f;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float wv = s_whp[(hb * 16 + r) * 64 + lane];
            const float bias = s_b1[hb * 32 + crow(r, half)];
#pragma unroll
            for (int i = 0; i < NBW; ++i)
                z[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(wv, act_fn<ACT>(acc[hb][i][r] + bias), z[i], 0, 0, 0);
        }
    float kl[NBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
        kl[i] = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            z[i][r] += s_bh[crow(r, half)];
            if (r < 8)
                kl[i] += z[i][r] * z[i][r];
            else
                kl[i] += kl_g(z[i][r]);
        }
        kl[i] += __shfl_xor(kl[i], 32);
    }

    // ---- decoder, one window block at a time: the hidden layer hd = act(Wd1 mu + bd1) (the
    // decoder output's B operands), then the output blocks, each reduced against v in registers
    const bool decode = p.decode != 0;
    float4 sm[NBW][CH];
    float sq[NBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
        sq[i] = 0.0f;
#pragma unroll
        for (int j = 0; j < CH; ++j)
            sm[i][j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    if (decode) {
        // Wd2 fragments of one output block (HB * 4 16-byte loads) run one block ahead in a
        // register ring: fragment (ob, hb, r4) is replaced right after its four matrix ops by the
        // same fragment of block ob + 1 (of block 0 after the last block, for the next window block)
        const int nob = g.D / 32;
        constexpr int PF = HB * 4;
        const float4 *wa = p.wd2p + lane;
        float4 ar[PF];
#pragma unroll
        for (int f = 0; f < PF; ++f)
            ar[f] = wa[f * 64];
#pragma unroll
        for (int i = 0; i < NBW; ++i) {
            v16f hd[HB];
#pragma unroll
            for (int hb = 0; hb < HB; ++hb) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    hd[hb][r] = 0.0f;
#pragma unroll
                for (int r = 0; r < 8; ++r)
                    hd[hb] = __builtin_amdgcn_mfma_f32_32x32x2f32(s_wd1p[(hb * 8 + r) * 64 + lane], z[i][r], hd[hb], 0,
                                                                  0, 0);
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    hd[hb][r] = act_fn<ACT>(hd[hb][r] + s_bd1[hb * 32 + crow(r, half)]);
            }
            for (int ob = 0; ob < nob; ++ob) {
                const float4 *wnext = wa + (ob + 1 == nob ? 0 : (ob + 1) * PF * 64);
                v16f o;
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    o[r] = 0.0f;
#pragma unroll
                for (int f = 0; f < PF; ++f) {
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        o = __builtin_amdgcn_mfma_f32_32x32x2f32(comp(ar[f], e), hd[f / 4][4 * (f % 4) + e], o, 0, 0,
                                                                 0);
                    __builtin_amdgcn_sched_barrier(0);
                    ar[f] = wnext[f * 64];
                }
                // registers 4 gq .. 4 gq + 3 hold the chunk (8 ob + 2 gq + half) of the window,
                // i.e. step t = chunk / MC, metric chunk = chunk mod MC (constant set gq mod 2
                // when MC = 4)
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    const int t = (8 * ob + 2 * gq + half) / MC;
                    const int cj = CH == 2 ? (gq & 1) : 0;
                    const int off = S == 1 ? t * CPRP + mchunk(cj) : (t / S) * CPRP + (t % S) * MC + mchunk(cj);
                    const float4 bd = reinterpret_cast<const float4 *>(s_bd2)[ob * 8 + 2 * gq + half];
                    const float4 x4 = reinterpret_cast<const float4 &>(seg[rb[i] + off]);
                    const float4 v4 = fma4(x4, ca[i][cj], cb[i][cj]);
                    const float d0 = (v4.x - bd.x) - o[4 * gq + 0];
                    const float d1 = (v4.y - bd.y) - o[4 * gq + 1];
                    const float d2 = (v4.z - bd.z) - o[4 * gq + 2];
                    const float d3 = (v4.w - bd.w) - o[4 * gq + 3];
                    sm[i][cj].x += d0;
                    sm[i][cj].y += d1;
                    sm[i][cj].z += d2;
                    sm[i][cj].w += d3;
                    sq[i] = fmaf(d0, d0, sq[i]);
                    sq[i] = fmaf(d1, d1, sq[i]);
                    sq[i] = fmaf(d2, d2, sq[i]);
                    sq[i] = fmaf(d3, d3, sq[i]);
                }
            }
        }
    }

    // ---- results: the two lane halves of a window hold different metric chunks (M >= 8) or
    // different steps of the same chunk (M = 4)
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
        const int n = wn0 + i * 32 + (lane & 31);
        float tot = 0.0f;
        if constexpr (MC == 1) {
            sm[i][0].x += __shfl_xor(sm[i][0].x, 32);
            sm[i][0].y += __shfl_xor(sm[i][0].y, 32);
            sm[i][0].z += __shfl_xor(sm[i][0].z, 32);
            sm[i][0].w += __shfl_xor(sm[i][0].w, 32);
            tot = (sm[i][0].x + sm[i][0].y) + (sm[i][0].z + sm[i][0].w);
        } else {
#pragma unroll
            for (int j = 0; j < CH; ++j)
                tot += (sm[i][j].x + sm[i][j].y) + (sm[i][j].z + sm[i][j].w);
            tot += __shfl_xor(tot, 32);
        }
        const float sqt = sq[i] + __shfl_xor(sq[i], 32);
        if (n >= nv)
            continue;
        const int64_t w = p.woff[s] + k0 + n;
        if (half == 0) {
            if (p.scores)
                p.scores[w] = 0.5f * kl[i];
            if (decode && p.md)
                p.md[w] = tot * g.inv_d;
            if (decode && p.rec)
                p.rec[w] = sqt * g.inv_d;
        }
        if (decode && p.mdm && (MC > 1 || half == 0)) {
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                float *dst = p.mdm + w * M + 4 * mchunk(j);
                dst[0] = sm[i][j].x * g.inv_w;
                dst[1] = sm[i][j].y * g.inv_w;
                dst[2] = sm[i][j].z * g.inv_w;
                dst[3] = sm[i][j].w * g.inv_w;
            }
        }
    }
}

using FusedKernel = void (*)(ExtFusedParams, ExtFusedShape);

template <int ACT>
FusedKernel pick_mc(int hb, int mc)
{
    switch (hb * 8 + mc) {
    case 1 * 8 + 1: return k_ext_fused<1, 1, ACT>;
    case 1 * 8 + 2: return k_ext_fused<1, 2, ACT>;
    case 1 * 8 + 4: return k_ext_fused<1, 4, ACT>;
    case 2 * 8 + 1: return k_ext_fused<2, 1, ACT>;
    case 2 * 8 + 2: return k_ext_fused<2, 2, ACT>;
    case 2 * 8 + 4: return k_ext_fused<2, 4, ACT>;
    default: break;
    }
    switch (hb * 8 + mc) {
    case 4 * 8 + 1: return k_ext_fused<4, 1, ACT>;
    case 4 * 8 + 2: return k_ext_fused<4, 2, ACT>;
    default: break;
    }
    if constexpr (ACT == ENOVA_RELU) {   // with tanh, 128 hidden units and 16 metrics exceed the registers
        if (hb == 4 && mc == 4)
            return k_ext_fused<4, 4, ACT>;
    }
    return nullptr;
}

FusedKernel pick_fused(const Geometry &g)
{
    if (!ext_fused_supported(g))
        return nullptr;
    return g.act == ENOVA_RELU ? pick_mc<ENOVA_RELU>(g.HB, g.M / 4) : pick_mc<ENOVA_TANH>(g.HB, g.M / 4);
}

}  // namespace

size_t ext_fused_lds_bytes(const Geometry &g)
{
    const size_t n_const = static_cast<size_t>(g.HB) * (16 * 64 + 8 * 64) + 3 * static_cast<size_t>(g.Hp) + 32;
    const size_t rows = static_cast<size_t>(kExtFusedNb + g.Q - 1 + g.spare);
    return (n_const + static_cast<size_t>(g.D)) * sizeof(float) + rows * g.CPRP * 16;
}

bool ext_fused_supported(const Geometry &g)
{
    return g.mfma_ok && !g.ring && g.dtype == ENOVA_F32 && (g.M == 4 || g.M == 8 || g.M == 16) && g.Mp == g.M &&
           (g.HB <= 2 || (g.HB == 4 && (g.act == ENOVA_RELU || g.M <= 8))) && g.L <= 16 && g.D % 32 == 0 &&
           g.KC % 4 == 0 && ext_fused_lds_bytes(g) <= kLdsLimit / 2;
}

hipError_t prepare_ext_fused(const Geometry &g)
{
    FusedKernel k = pick_fused(g);
    if (!k)
        return hipErrorInvalidValue;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(kLdsLimit));
}

hipError_t launch_ext_fused(const Geometry &g, const ExtFusedParams &p, int64_t grid, hipStream_t st)
{
    if (grid <= 0)
        return hipSuccess;
    FusedKernel k = pick_fused(g);
    if (!k)
        return hipErrorInvalidValue;
    ExtFusedShape sh;
    sh.S = g.S;
    sh.W = g.W;
    sh.Q = g.Q;
    sh.CPR = g.CPR;
    sh.CPRP = g.CPRP;
    sh.KC = g.KC;
    sh.spare = g.spare;
    sh.D = g.D;
    sh.inv_w = 1.0f / static_cast<float>(g.W);
    sh.inv_d = 1.0f / static_cast<float>(g.D);
    hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(grid)), dim3(kFusedWaves * 64), ext_fused_lds_bytes(g), st, p,
                       sh);
    return hipGetLastError();
}

}  // namespace enova
