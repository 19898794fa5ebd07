// Device pieces shared by the matrix-core scoring kernels (the sliding-window batch kernel and
// the streaming kernel over each stream's newest window): element helpers, the bf16 hi/lo split
// and the epilogue that chains the posterior heads, the KL score and the decoder's hidden layer
// on the matrix cores straight from the encoder's accumulators (Section IV-B).
//
// The accumulator layout of a 32x32 MFMA block (lane l, register r holds row
// 8*(r/4) + 4*(l/32) + r%4 and column l%32) is exactly the B-operand layout a following
// 32x32x2 fp32 MFMA needs when its reduction index is permuted the same way (and, eight
// registers at a time, the B operand of a 32x32x16 bf16 MFMA), so the rest of the detector
// chains on the matrix cores without leaving registers:
//   hidden  h  = act(C + b1)
//   heads   [mu; logvar] = Wh h + bh          (32 x Hp, Wh pre-permuted on the host)
//   score   1/2 sum_l (mu_l^2 + e^lv_l - 1 - lv_l)       (lane-pair reduction)
//   decoder hd = act(Wd1 mu + bd1),  u . hd with u the column sums of Wd2 (for the md)
#pragma once

#include <hip/hip_runtime.h>

#include "internal.h"

namespace enova {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

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

template <int ACT>
__device__ __forceinline__ float act_fn(float a)
{
    if constexpr (ACT == ENOVA_TANH)
        return tanhf(a);
    else
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

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b)
{
    const __bf16 ha = static_cast<__bf16>(a);
    const __bf16 hb = static_cast<__bf16>(b);
    return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, ha)) |
           (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, hb)) << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// x = hi + lo as two bf16 vectors, lo the rounded remainder. With a bf16 weight split the same
// way, hi*hi + hi*lo + lo*hi (fp32 accumulation) carries about 16 significant bits: the bf16
// workload's posterior heads and decoder layer run on three bf16 matrix ops instead of the
// eight times slower fp32 ones.
__device__ __forceinline__ void split_bf16x8(const float (&x)[8], v8bf &hi, v8bf &lo)
{
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const __bf16 h = static_cast<__bf16>(x[t]);
        hi[t] = h;
        lo[t] = static_cast<__bf16>(x[t] - static_cast<float>(h));
    }
}

__device__ __forceinline__ v16f mfma3_bf16(uint4 a_hi, uint4 a_lo, v8bf b_hi, v8bf b_lo, v16f c)
{
    const v8bf ah = __builtin_bit_cast(v8bf, a_hi), al = __builtin_bit_cast(v8bf, a_lo);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b_hi, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b_lo, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b_hi, c, 0, 0, 0);
}

// Row of the accumulator register r for lane half g inside a 32x32 block.
__device__ __forceinline__ int crow(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Arguments of the epilogue.
struct EpiArgs {
    const float *whp;    // heads fragments: fp32 [HBT][16][64], or bf16 hi/lo [HBT][2][2][64] x 16 B
    const float *wd1p;   // decoder hidden-layer fragments: fp32 [HBT][8][64], or bf16 hi/lo [HBT][2][64] x 16 B
    const float *b1, *bd1, *u;   // [HBT * 32] each
    const float *bh;             // [32]: mu biases (padded to 16), log-variance biases (padded to 16)
    float *xchg;                 // LDS of epi_xchg_floats(NW, NBW) floats, used when WH > 1
    int lane, half, wave, wh, wn;
};

// Window blocks per epilogue pass (two at most, to bound registers) and the LDS floats the
// partial-sum exchange of a layout with WH > 1 needs.
template <int NBW>
struct EpiPass {
    static constexpr int NG = NBW > 2 ? 2 : NBW;
};
constexpr int epi_xchg_floats(int nw, int nbw) { return nw * (nbw > 2 ? 2 : nbw) * (16 + 1) * 64; }

// Epilogue of a wave that holds the encoder accumulators acc[hb][nb] of its HB hidden blocks
// (global blocks wh*HB + hb) and NBW 32-window blocks. The NW waves form WH groups along the
// hidden rows; with WH > 1 every wave of a window group adds the WH partial sums in the same
// fixed order through LDS, so every wave calls this (it synchronises the block). The NG blocks
// of a pass run as independent MFMA chains. store(nb, score, dot) is called by every lane of
// every wave for each window block; dot = u . hd is complete in every lane of the wave (both
// lane halves), score = 1/2 sum_l (mu_l^2 + e^lv_l - 1 - lv_l).
template <int DT, int HB, int NBW, int WH, int NW, int ACT, typename StoreFn>
__device__ __forceinline__ void score_epilogue(v16f (&acc)[HB][NBW], const EpiArgs &e, StoreFn store)
{
    constexpr int NG = EpiPass<NBW>::NG;
    const int lane = e.lane, half = e.half, wave = e.wave, wh = e.wh, wn = e.wn;
    float *xz = e.xchg;                                    // [NW][NG][16][64] head partials
    float *xd = xz + NW * NG * 16 * 64;                    // [NW][NG][64] decoder partials
#pragma unroll
    for (int g0 = 0; g0 < NBW; g0 += NG) {
        // a pass re-reads the small LDS vectors: kept live across passes they cost registers
        asm volatile("" ::: "memory");
        // hidden activations (bias + act, one 32-row block at a time) feed the posterior heads:
        // rows 0..15 mean, 16..31 log-variance (this wave's share of the hidden rows)
        v16f z[NG];
#pragma unroll
        for (int i = 0; i < NG; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                z[i][r] = 0.0f;
#pragma unroll
        for (int hb = 0; hb < HB; ++hb) {
            const int hbg = wh * HB + hb;
            if constexpr (DT == ENOVA_F32) {
                // reduction index of matrix op r: hidden rows crow(r, 0), crow(r, 1)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float wv = e.whp[(hbg * 16 + r) * 64 + lane];
                    const float bias = e.b1[hbg * 32 + crow(r, half)];
#pragma unroll
                    for (int i = 0; i < NG; ++i)
                        z[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            wv, act_fn<ACT>(acc[hb][g0 + i][r] + bias), z[i], 0, 0, 0);
                }
            } else {
                // reduction slot (g, t) of op m: hidden row crow(8m + t, g); weights packed as
                // [hidden block][m][hi, lo][lane] 16-byte fragments
                const uint4 *wsrc = reinterpret_cast<const uint4 *>(e.whp);
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    const uint4 wa_hi = wsrc[((hbg * 2 + m) * 2 + 0) * 64 + lane];
                    const uint4 wa_lo = wsrc[((hbg * 2 + m) * 2 + 1) * 64 + lane];
#pragma unroll
                    for (int i = 0; i < NG; ++i) {
                        float hv[8];
#pragma unroll
                        for (int t = 0; t < 8; ++t) {
                            const int r = 8 * m + t;
                            const float bias = e.b1[hbg * 32 + crow(r, half)];
                            hv[t] = act_fn<ACT>(acc[hb][g0 + i][r] + bias);
                        }
                        v8bf h_hi, h_lo;
                        split_bf16x8(hv, h_hi, h_lo);
                        z[i] = mfma3_bf16(wa_hi, wa_lo, h_hi, h_lo, z[i]);
                    }
                }
            }
        }
        if constexpr (WH > 1) {
            // every wave of the window group adds the WH partials in the same fixed order
            __syncthreads();          // the segment, or the previous pass's exchange, is no longer read
#pragma unroll
            for (int i = 0; i < NG; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    xz[((wave * NG + i) * 16 + r) * 64 + lane] = z[i][r];
            __syncthreads();
#pragma unroll
            for (int i = 0; i < NG; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float t = 0.0f;
#pragma unroll
                    for (int w2 = 0; w2 < WH; ++w2)
                        t += xz[(((wn * WH + w2) * NG + i) * 16 + r) * 64 + lane];
                    z[i][r] = t;
                }
        }
        float kl[NG];
#pragma unroll
        for (int i = 0; i < NG; ++i) {
            kl[i] = 0.0f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                z[i][r] += e.bh[crow(r, half)];
                if (r < 8)
                    kl[i] += z[i][r] * z[i][r];
                else
                    kl[i] += kl_g(z[i][r]);
            }
            kl[i] += __shfl_xor(kl[i], 32);
        }
        // decoder hidden layer at z = mu, dotted with the column sums of Wd2 (mu is held in
        // registers 0..7: latent crow(r, half))
        float dot[NG];
#pragma unroll
        for (int i = 0; i < NG; ++i)
            dot[i] = 0.0f;
        v8bf mu_hi[NG], mu_lo[NG];
        if constexpr (DT == ENOVA_BF16) {
#pragma unroll
            for (int i = 0; i < NG; ++i) {
                float mv[8];
#pragma unroll
                for (int t = 0; t < 8; ++t)
                    mv[t] = z[i][t];
                split_bf16x8(mv, mu_hi[i], mu_lo[i]);
            }
        }
#pragma unroll
        for (int hb = 0; hb < HB; ++hb) {
            const int hbg = wh * HB + hb;
            v16f d[NG];
#pragma unroll
            for (int i = 0; i < NG; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    d[i][r] = 0.0f;
            if constexpr (DT == ENOVA_F32) {
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const float wv = e.wd1p[(hbg * 8 + r) * 64 + lane];
#pragma unroll
                    for (int i = 0; i < NG; ++i)
                        d[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(wv, z[i][r], d[i], 0, 0, 0);
                }
            } else {
                // weights packed as [hidden block][hi, lo][lane] 16-byte fragments
                const uint4 *wsrc = reinterpret_cast<const uint4 *>(e.wd1p);
                const uint4 wd_hi = wsrc[(hbg * 2 + 0) * 64 + lane];
                const uint4 wd_lo = wsrc[(hbg * 2 + 1) * 64 + lane];
#pragma unroll
                for (int i = 0; i < NG; ++i)
                    d[i] = mfma3_bf16(wd_hi, wd_lo, mu_hi[i], mu_lo[i], d[i]);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int h = hbg * 32 + crow(r, half);
                const float uh = e.u[h];
                const float bh = e.bd1[h];
#pragma unroll
                for (int i = 0; i < NG; ++i)
                    dot[i] += uh * act_fn<ACT>(d[i][r] + bh);
            }
        }
        if constexpr (WH > 1) {
#pragma unroll
            for (int i = 0; i < NG; ++i)
                xd[(wave * NG + i) * 64 + lane] = dot[i];
            __syncthreads();
#pragma unroll
            for (int i = 0; i < NG; ++i) {
                float t = 0.0f;
#pragma unroll
                for (int w2 = 0; w2 < WH; ++w2)
                    t += xd[((wn * WH + w2) * NG + i) * 64 + lane];
                dot[i] = t;
            }
        }
#pragma unroll
        for (int i = 0; i < NG; ++i) {
            dot[i] += __shfl_xor(dot[i], 32);
            store(g0 + i, 0.5f * kl[i], dot[i]);
        }
    }
}

}  // namespace

}  // namespace enova
