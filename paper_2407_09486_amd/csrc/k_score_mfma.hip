// Matrix-core (MFMA) scoring kernel for gfx950.
//
// A tile is Nb consecutive windows of one stream. Its Nb+Q-1 super-rows are read from HBM
// once (coalesced 16-byte loads), normalised with the stream's reference statistics and
// written to LDS (rounded to bf16 for the bf16 workload); then the encoder's first layer --
// the dense contraction of Section IV-B's VAE, 2*H*D flops per window -- runs as
//
//     C[h][n] = sum_k W1[h][k] * V[n][k]      (A = W1 from L2, B = windows from LDS)
//
// on v_mfma_f32_32x32x2_f32 (fp32) or v_mfma_f32_32x32x16_bf16 (bf16 operands, fp32
// accumulation). Window n's row of V is never materialised: its chunk kappa = q*CPR + c is
// chunk c of LDS super-row (n + q), so one staged element feeds up to Q windows.
//
// The accumulator layout of a 32x32 MFMA block (lane l, register r holds row
// 8*(r/4) + 4*(l/32) + r%4 and column l%32) is exactly the B-operand layout a following
// 32x32x2 fp32 MFMA needs when its reduction index is permuted the same way (and, eight
// registers at a time, the B operand of a 32x32x16 bf16 MFMA), so the rest of the detector
// chains on the matrix cores without leaving registers:
//   hidden  h  = act(C + b1)
//   heads   [mu; logvar] = Wh h + bh          (32 x Hp, Wh pre-permuted on the host)
//   score   1/2 sum_l (mu_l^2 + e^lv_l - 1 - lv_l)       (lane-pair reduction)
//   decoder hd = act(Wd1 mu + bd1),  mean(m') = (u . hd + sum bd2) / D
//   md      mean(v) - mean(m'),  mean(v) from per-super-row sums kept in LDS.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace enova {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

struct MfmaShape {
    int M, S, W, Mp, Q, CPR, CPRP, KC;
    int spare;       // staged super-rows after a tile's last window's Q - 1
    int tail_rows;   // steps of the window's last super-row that belong to the window
    float inv_d;
};

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

// Wave layout: the NW waves form WH groups along the hidden rows and NW/WH groups along the
// windows. A wave owns HB 32-row hidden blocks and NBW 32-window blocks; with WH > 1 the waves
// of a window group share its B fragments and their posterior-head partial sums are reduced
// through LDS.
// CL: the epilogue weights are copied into LDS with each tile (else read from L2, leaving the
// LDS to a larger segment).
template <int DT, int HB, int NBW, int WH, int NW, int ACT, bool CL>
__global__ __launch_bounds__(NW * 64, (NW == 4 && ACT == ENOVA_RELU && WH == 1) ? 2 : 1)
void k_score_mfma(ScoreParams p, MfmaShape g)
{
    constexpr int NT = NW * 64;                   // threads of the block
    constexpr int WN = NW / WH;                   // window groups
    constexpr int HBT = HB * WH;                  // hidden blocks of the tile
    constexpr int NB = WN * NBW * 32;             // windows per tile
    constexpr int EPC = DT == ENOVA_F32 ? 4 : 8;  // elements per 16-byte chunk
    extern __shared__ uint4 lds[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const int wh = wave % WH;                     // hidden-row group of this wave
    const int wn = wave / WH;                     // window group of this wave

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

    const int Q = g.Q, CPR = g.CPR, CPRP = g.CPRP, M = g.M, Mp = g.Mp, S = g.S;
    // staged super-rows: the tile's nv + Q - 1 plus spare rows read only by zero-weight chunks
    const int nrows = nv + Q - 1 + g.spare;
    // LDS: the epilogue's weights (heads, decoder hidden layer, b1, bd1, u, head biases) when
    // CL, then the segment, the per-column statistics and offsets of a super-row, and the row
    // sums (with WH > 1 the segment's space is reused after the main loop to exchange partial
    // sums)
    constexpr int HP = 32 * HBT;
    constexpr int N_WHP = HBT * 16 * 64, N_WD1P = HBT * 8 * 64;
    constexpr int N_CONST = CL ? N_WHP + N_WD1P + 3 * HP + 32 : 0;
    constexpr int N_XCHG = WH > 1 ? NW * (NBW > 2 ? 2 : NBW) * (16 + 1) * 64 : 0;   // floats
    float *s_whp = reinterpret_cast<float *>(lds);
    float *s_wd1p = s_whp + N_WHP;
    uint4 *seg = lds + N_CONST / 4;
    const int rows_alloc = NB + Q - 1 + g.spare;
    const size_t seg_chunks = static_cast<size_t>(rows_alloc) * CPRP;
    const size_t seg_span = seg_chunks > N_XCHG / 4 ? seg_chunks : N_XCHG / 4;
    // per element j of a super-row (j = c*EPC + e < S*Mp): its metric's mean and 1/std (0 for
    // padding) and its offset from the row's first element in the stream (-1 for padding)
    const int SMp = CPR * EPC;
    float *cmean = reinterpret_cast<float *>(seg + seg_span);
    float *crinv = cmean + SMp;
    int *coff = reinterpret_cast<int *>(crinv + SMp);
    float *rs = reinterpret_cast<float *>(coff + SMp);
    float *ps = rs + rows_alloc;
    // b1, bd1, u and the head biases: inside the copied block when CL, else after the row sums
    float *s_b1 = CL ? s_wd1p + N_WD1P : ps + rows_alloc;
    float *s_bd1 = s_b1 + HP;
    float *s_u = s_bd1 + HP;
    float *s_bh = s_u + HP;

    if constexpr (CL) {
        // the host lays the epilogue weights out contiguously in this LDS order; copy them with
        // several 16-byte loads in flight per thread
        constexpr int N4 = N_CONST / 4;
        constexpr int CU = 4;
        const float4 *src = reinterpret_cast<const float4 *>(p.whp);
        float4 *dst = reinterpret_cast<float4 *>(s_whp);
        constexpr int FULL = N4 / (NT * CU) * (NT * CU);
        for (int base = tid; base < FULL; base += NT * CU) {
            float4 t[CU];
#pragma unroll
            for (int u = 0; u < CU; ++u)
                t[u] = src[base + u * NT];
#pragma unroll
            for (int u = 0; u < CU; ++u)
                dst[base + u * NT] = t[u];
        }
        for (int i = FULL + tid; i < N4; i += NT)
            dst[i] = src[i];
    } else {
        for (int i = tid; i < HP; i += NT) {
            s_b1[i] = p.b1[i];
            s_bd1[i] = p.bd1[i];
            s_u[i] = p.u[i];
        }
        if (tid < 32)
            s_bh[tid] = p.bh[tid];
    }
    for (int j = tid; j < SMp; j += NT) {
        const int tt = j / Mp;
        const int m = j - tt * Mp;
        if (m < M) {
            cmean[j] = p.mean[static_cast<int64_t>(s) * M + m];
            crinv[j] = 1.0f / p.std[static_cast<int64_t>(s) * M + m];
            coff[j] = tt * M + m;
        } else {
            cmean[j] = 0.0f;
            crinv[j] = 0.0f;
            coff[j] = -1;
        }
    }
    __syncthreads();

    // ---- stage: super-row r of the tile covers stream steps (k0 + r)*S .. +S-1
    const int64_t step0 = k0 * S;
    const int64_t eavail = (T - step0) * M;        // stream elements from super-row 0 on
    const bool linear = (Mp == M) && (((srow + step0) * M) % EPC == 0);
    const int64_t ebase = (srow + step0) * M;      // element index of super-row 0
    // Each thread keeps SU chunk loads in flight, and the next SU are issued before the current
    // ones are normalised (one load per loop trip would serialise a full HBM round trip per
    // chunk). Its chunks are tid + i*NT; their (row, column) advance by (NT / CPR, NT % CPR)
    // with a carry instead of a division each.
    constexpr int SU = 8;
    const int n_chunks = nrows * CPR;
    const int dr = NT / CPR, dc = NT - (NT / CPR) * CPR;
    int cr = tid / CPR, ccol = tid - (tid / CPR) * CPR;
    auto load_batch = [&](int base, uint4 (&raw)[SU], bool (&vec)[SU]) {
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            const int idx = base + u * NT;
            vec[u] = idx < n_chunks && linear && static_cast<int64_t>(idx + 1) * EPC <= eavail;
            if (vec[u]) {
                const int64_t e0 = ebase + static_cast<int64_t>(idx) * EPC;
                if constexpr (DT == ENOVA_F32)
                    raw[u] = *reinterpret_cast<const uint4 *>(static_cast<const float *>(p.x) + e0);
                else
                    raw[u] = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p.x) + e0);
            }
        }
    };
    auto store_batch = [&](int base, const uint4 (&raw)[SU], const bool (&vec)[SU]) {
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            const int idx = base + u * NT;
            const int r = cr, c = ccol;
            ccol += dc;
            cr += dr;
            if (ccol >= CPR) {
                ccol -= CPR;
                ++cr;
            }
            if (idx >= n_chunks)
                continue;
            const float *mu = cmean + c * EPC;
            const float *ri = crinv + c * EPC;
            float v[EPC];
            if (vec[u]) {
                if constexpr (DT == ENOVA_F32) {
                    v[0] = __uint_as_float(raw[u].x);
                    v[1] = __uint_as_float(raw[u].y);
                    v[2] = __uint_as_float(raw[u].z);
                    v[3] = __uint_as_float(raw[u].w);
                } else {
                    v[0] = bf16_lo(raw[u].x);
                    v[1] = bf16_hi(raw[u].x);
                    v[2] = bf16_lo(raw[u].y);
                    v[3] = bf16_hi(raw[u].y);
                    v[4] = bf16_lo(raw[u].z);
                    v[5] = bf16_hi(raw[u].z);
                    v[6] = bf16_lo(raw[u].w);
                    v[7] = bf16_hi(raw[u].w);
                }
#pragma unroll
                for (int e = 0; e < EPC; ++e)
                    v[e] = (v[e] - mu[e]) * ri[e];
            } else {
                // padding, the stream's end, or a row start that is not 16-byte aligned
                const int64_t rel = static_cast<int64_t>(r) * S * M;
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const int off = coff[c * EPC + e];
                    float val = 0.0f;
                    if (off >= 0 && rel + off < eavail)
                        val = (load_x<DT>(p.x, ebase + rel + off) - mu[e]) * ri[e];
                    v[e] = val;
                }
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
            seg[r * CPRP + c] = out;
        }
    };
    {
        uint4 raw0[SU], raw1[SU];
        bool vec0[SU], vec1[SU];
        load_batch(tid, raw0, vec0);
        for (int base = tid; base < n_chunks; base += 2 * NT * SU) {
            load_batch(base + NT * SU, raw1, vec1);
            store_batch(base, raw0, vec0);
            load_batch(base + 2 * NT * SU, raw0, vec0);
            store_batch(base + NT * SU, raw1, vec1);
        }
    }
    __syncthreads();

    // ---- per-super-row sums of the staged values (full row, and the window's tail part)
    const int tail_elems = g.tail_rows * Mp;
    for (int r = tid; r < nrows; r += NT) {
        float full = 0.0f, part = 0.0f;
        for (int c = 0; c < CPR; ++c) {
            const uint4 q4 = seg[r * CPRP + c];
            float e[EPC];
            if constexpr (DT == ENOVA_F32) {
                e[0] = __uint_as_float(q4.x);
                e[1] = __uint_as_float(q4.y);
                e[2] = __uint_as_float(q4.z);
                e[3] = __uint_as_float(q4.w);
            } else {
                e[0] = bf16_lo(q4.x);
                e[1] = bf16_hi(q4.x);
                e[2] = bf16_lo(q4.y);
                e[3] = bf16_hi(q4.y);
                e[4] = bf16_lo(q4.z);
                e[5] = bf16_hi(q4.z);
                e[6] = bf16_lo(q4.w);
                e[7] = bf16_hi(q4.w);
            }
#pragma unroll
            for (int k = 0; k < EPC; ++k) {
                full += e[k];
                if (c * EPC + k < tail_elems)
                    part += e[k];
            }
        }
        rs[r] = full;
        ps[r] = part;
    }

    // ---- main contraction
    int rb[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int n = wn * NBW * 32 + nb * 32 + (lane & 31);
        rb[nb] = (n < nv ? n : nv - 1) * CPRP;   // idle columns re-read a valid window
    }
    v16f acc[HB][NBW];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[hb][nb][r] = 0.0f;

    const bool wave_active = wn * NBW * 32 < nv;
    const int nsteps = g.KC / 2;                 // even: KC is a multiple of 4
    // A fragments of step i: w1p[(i * HBT + hb) * 64 + lane]; this wave's blocks start at wh * HB
    const uint4 *ap = p.w1p + wh * HB * 64 + lane;
    // LDS chunk offset of this lane's chunk kappa = 2*i + half inside a window:
    // (kappa / CPR) * CPRP + kappa % CPR, advanced without branches
    const int dpitch = CPRP - CPR;
    int cc = half % CPR;
    int koff = (half / CPR) * CPRP + cc;
    auto advance = [&]() {
        const bool wrap = cc + 2 >= CPR;
        cc = cc + 2 - (wrap ? CPR : 0);
        koff += 2 + (wrap ? dpitch : 0);
    };
    auto mma = [&](const uint4 (&a)[HB], const uint4 (&bq)[NBW]) {
        if constexpr (DT == ENOVA_F32) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
#pragma unroll
                for (int hb = 0; hb < HB; ++hb) {
                    const float av = __uint_as_float(e == 0 ? a[hb].x : e == 1 ? a[hb].y
                                                    : e == 2 ? a[hb].z : a[hb].w);
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb) {
                        const float bv = __uint_as_float(e == 0 ? bq[nb].x : e == 1 ? bq[nb].y
                                                        : e == 2 ? bq[nb].z : bq[nb].w);
                        acc[hb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[hb][nb], 0, 0, 0);
                    }
                }
            }
        } else {
#pragma unroll
            for (int hb = 0; hb < HB; ++hb) {
                const v8bf av = __builtin_bit_cast(v8bf, a[hb]);
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    acc[hb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        av, __builtin_bit_cast(v8bf, bq[nb]), acc[hb][nb], 0, 0, 0);
            }
        }
    };
    __syncthreads();
    if (wave_active) {
        // W1 fragments run PD steps ahead in a register ring, window fragments PB steps ahead
        // (ring of 2*PB) from LDS: an fp32 step is 4*HB*NBW matrix ops, a bf16 step only
        // HB*NBW, so bf16 needs the deeper rings to cover an L2 round trip. The loop is unrolled
        // by PD so every ring slot is a compile-time register set.
        // (bf16 with one wave per hidden group runs two waves per SIMD, and four hidden blocks
        // per wave hold 16 registers per step: a shallower W1 ring for both; the eight-wave
        // layout has 256 registers per wave and a short LDS latency to cover: one window step)
        constexpr int PD = DT == ENOVA_F32 ? 2 : ((WH == 1 || HB >= 4) ? 4 : 8);
        constexpr int PB = (DT == ENOVA_F32 || NW == 8) ? 1 : 2;
        constexpr int RB = 2 * PB;
        static_assert(PD % RB == 0 && PD <= kPrefetchSteps && PB <= kPrefetchRows, "prefetch rings");
        uint4 a[PD][HB], b[RB][NBW];
#pragma unroll
        for (int j = 0; j < PD; ++j) {
#pragma unroll
            for (int hb = 0; hb < HB; ++hb)
                a[j][hb] = ap[(j * HBT + hb) * 64];
            // issue the ring in step order: the wait counts inserted at the loop head must hold
            // for the first trip too, and a reordered prologue makes them wait for the newest loads
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int j = 0; j < PB; ++j) {
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                b[j][nb] = seg[rb[nb] + koff];
            advance();
        }
        // koff now points PB steps ahead. Prefetches past the last step read the zero steps the
        // host appends to the packed W1 and the spare LDS rows, so no index needs clamping.
        const uint4 *api = ap + PD * HBT * 64;
        for (int i = 0; i < nsteps; i += PD) {
#pragma unroll
            for (int j = 0; j < PD; ++j) {
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb)
                    b[(j + PB) % RB][nb] = seg[rb[nb] + koff];
                advance();
                if constexpr (DT == ENOVA_F32) {
                    // keep the prefetches ahead of this step's matrix ops (the scheduler would
                    // sink them)
                    __builtin_amdgcn_sched_barrier(0);
                    mma(a[j], b[j % RB]);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int hb = 0; hb < HB; ++hb)
                        a[j][hb] = api[(j * HBT + hb) * 64];
                } else {
                    mma(a[j], b[j % RB]);
#pragma unroll
                    for (int hb = 0; hb < HB; ++hb)
                        a[j][hb] = api[(j * HBT + hb) * 64];
                    // A bf16 matrix op is short, and a wave issues in order: slot the step's
                    // other instructions between the matrix ops instead of in one run (the
                    // window-fragment reads first, each W1 reload right after the last op that
                    // reads its register)
#pragma unroll
                    for (int t = 0; t < HB * NBW; ++t) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // matrix op
                        if (t < NBW)
                            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
                        if ((t + 1) % NBW == 0)
                            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // global read
                        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);   // vector ALU
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            api += PD * HBT * 64;
        }
    }
    if constexpr (WH == 1) {
        if (!wave_active)
            return;
    }

    // ---- epilogue, NG window blocks per pass (weights from LDS, or L2 when the segment needs
    // the LDS); the NG blocks of a pass run as independent MFMA chains
    constexpr int NG = NBW > 2 ? 2 : NBW;
    float *xz = reinterpret_cast<float *>(seg);            // [NW][NG][16][64] head partials
    float *xd = xz + NW * NG * 16 * 64;                    // [NW][NG][64] decoder partials
    const bool storer = WH == 1 || (wh == 0 && wave_active);
#pragma unroll
    for (int g0 = 0; g0 < NBW; g0 += NG) {
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
                    const float wv = CL ? s_whp[(hbg * 16 + r) * 64 + lane] : p.whp[(hbg * 16 + r) * 64 + lane];
                    const float bias = s_b1[hbg * 32 + crow(r, half)];
#pragma unroll
                    for (int i = 0; i < NG; ++i)
                        z[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            wv, act_fn<ACT>(acc[hb][g0 + i][r] + bias), z[i], 0, 0, 0);
                }
            } else {
                // reduction slot (g, t) of op m: hidden row crow(8m + t, g); weights packed as
                // [hidden block][m][hi, lo][lane] 16-byte fragments
                const uint4 *wsrc = reinterpret_cast<const uint4 *>(CL ? s_whp : p.whp);
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
                            const float bias = s_b1[hbg * 32 + crow(r, half)];
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
                z[i][r] += s_bh[crow(r, half)];
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
                    const float wv = CL ? s_wd1p[(hbg * 8 + r) * 64 + lane] : p.wd1p[(hbg * 8 + r) * 64 + lane];
#pragma unroll
                    for (int i = 0; i < NG; ++i)
                        d[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(wv, z[i][r], d[i], 0, 0, 0);
                }
            } else {
                // weights packed as [hidden block][hi, lo][lane] 16-byte fragments
                const uint4 *wsrc = reinterpret_cast<const uint4 *>(CL ? s_wd1p : p.wd1p);
                const uint4 wd_hi = wsrc[(hbg * 2 + 0) * 64 + lane];
                const uint4 wd_lo = wsrc[(hbg * 2 + 1) * 64 + lane];
#pragma unroll
                for (int i = 0; i < NG; ++i)
                    d[i] = mfma3_bf16(wd_hi, wd_lo, mu_hi[i], mu_lo[i], d[i]);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int h = hbg * 32 + crow(r, half);
                const float uh = s_u[h];
                const float bh = s_bd1[h];
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
            const int nb = g0 + i;
            dot[i] += __shfl_xor(dot[i], 32);

            // window mean of the staged inputs: super-rows rb .. rb+Q-1, the last one partially
            const int n = wn * NBW * 32 + nb * 32 + (lane & 31);
            float vsum = 0.0f;
            const int row0 = rb[nb] / CPRP;
            for (int qq = half; qq < Q - 1; qq += 2)
                vsum += rs[row0 + qq];
            if (((Q - 1) & 1) == half)
                vsum += ps[row0 + Q - 1];
            vsum += __shfl_xor(vsum, 32);

            if (storer && half == 0 && n < nv) {
                const int64_t w = p.woff[s] + k0 + n;
                const float sc = 0.5f * kl[i];
                p.scores[w] = sc;
                if (p.md)
                    p.md[w] = vsum * g.inv_d - (dot[i] + p.sum_bd2) * g.inv_d;
                if (p.write_flags)
                    p.flags[w] = sc > p.threshold ? 1 : 0;
            }
        }
    }
}

using ScoreKernel = void (*)(ScoreParams, MfmaShape);

template <int DT, int ACT>
ScoreKernel pick_layout(int hbw, int nbw, int wh, int nw, bool cl)
{
    if (wh == 1 && nw == 4 && cl) {
        switch (hbw) {
        case 1: return nbw == 4 ? k_score_mfma<DT, 1, 4, 1, 4, ACT, true> : nullptr;
        case 2: return nbw == 4 ? k_score_mfma<DT, 2, 4, 1, 4, ACT, true> : nullptr;
        case 4: return nbw == 2 ? k_score_mfma<DT, 4, 2, 1, 4, ACT, true> : nullptr;
        case 8:   // bf16 with eight hidden blocks uses a split layout below
            if constexpr (DT == ENOVA_F32)
                return nbw == 1 ? k_score_mfma<DT, 8, 1, 1, 4, ACT, true> : nullptr;
            else
                return nullptr;
        default: return nullptr;
        }
    }
    if constexpr (DT == ENOVA_BF16) {
        if (wh == 4 && nw == 8 && hbw == 2 && nbw == 4 && !cl)
            return k_score_mfma<DT, 2, 4, 4, 8, ACT, false>;
    }
    return nullptr;
}

// The instantiation for a geometry: storage type, wave layout and activation.
ScoreKernel pick(const Geometry &g)
{
    const bool relu = g.act == ENOVA_RELU;
    if (g.dtype == ENOVA_F32)
        return relu ? pick_layout<ENOVA_F32, ENOVA_RELU>(g.HBW, g.NBW, g.WH, g.NW, g.cl)
                    : pick_layout<ENOVA_F32, ENOVA_TANH>(g.HBW, g.NBW, g.WH, g.NW, g.cl);
    return relu ? pick_layout<ENOVA_BF16, ENOVA_RELU>(g.HBW, g.NBW, g.WH, g.NW, g.cl)
                : pick_layout<ENOVA_BF16, ENOVA_TANH>(g.HBW, g.NBW, g.WH, g.NW, g.cl);
}

}  // namespace

// Allow the chosen instantiation the full 160 KiB of LDS.
hipError_t prepare_score_mfma(const Geometry &g)
{
    ScoreKernel k = pick(g);
    if (!k)
        return hipErrorInvalidValue;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(kLdsLimit));
}

hipError_t launch_score_mfma(const Geometry &g, const ScoreParams &p, int64_t grid, hipStream_t st)
{
    if (grid <= 0)
        return hipSuccess;
    ScoreKernel k = pick(g);
    if (!k)
        return hipErrorInvalidValue;
    MfmaShape sh;
    sh.M = g.M;
    sh.S = g.S;
    sh.W = g.W;
    sh.Mp = g.Mp;
    sh.Q = g.Q;
    sh.CPR = g.CPR;
    sh.CPRP = g.CPRP;
    sh.KC = g.KC;
    sh.spare = g.spare;
    sh.tail_rows = g.W - (g.Q - 1) * g.S;
    sh.inv_d = 1.0f / static_cast<float>(g.D);
    hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(grid)), dim3(64 * g.NW), g.lds_bytes, st, p, sh);
    return hipGetLastError();
}

// Wave layout for a hidden-block count HB: hidden blocks and 32-window blocks per wave, waves
// along the hidden rows, waves per block.
void mfma_layout(int dtype, int hb, int *hbw, int *nbw, int *wh, int *nw)
{
    if (dtype == ENOVA_BF16 && hb == 8) {
        // bf16 matrix ops are 4x faster than fp32 ones, and every tile streams all of W1 from
        // L2: the tile must hold as many windows as LDS allows (256; the epilogue weights then
        // stay in L2). Eight waves, two per SIMD, keep the matrix cores busy while the other
        // wave of the SIMD waits: 4 x 2 waves of 64 hidden rows x 128 windows.
        *hbw = 2;
        *nbw = 4;
        *wh = 4;
        *nw = 8;
        return;
    }
    *wh = 1;
    *nw = 4;
    *hbw = hb;
    *nbw = hb <= 2 ? 4 : (hb == 4 ? 2 : 1);
}

}  // namespace enova
