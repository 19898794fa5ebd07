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
// The posterior heads, the KL score and the decoder's hidden layer then chain on the matrix
// cores straight from the accumulators (score_epilogue); the md adds the window mean of the
// staged inputs from per-super-row sums kept in LDS.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "mfma_common.h"

namespace enova {

namespace {

struct MfmaShape {
    int M, S, W, Mp, Q, CPR, CPRP, KC;
    int spare;       // staged super-rows after a tile's last window's Q - 1
    int tail_rows;   // steps of the window's last super-row that belong to the window
    float inv_d;
};

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
    constexpr int N_XCHG = WH > 1 ? epi_xchg_floats(NW, NBW) : 0;   // floats
    float *s_whp = reinterpret_cast<float *>(lds);
    float *s_wd1p = s_whp + N_WHP;
    const float *e_whp = CL ? s_whp : p.whp;      // epilogue fragments: the copied block, or L2
    const float *e_wd1p = CL ? s_wd1p : p.wd1p;
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

    // ---- epilogue (weights from LDS when CL, else from L2)
    const bool storer = WH == 1 || (wh == 0 && wave_active);
    const EpiArgs ea{e_whp, e_wd1p, s_b1, s_bd1, s_u, s_bh, reinterpret_cast<float *>(seg),
                     lane, half, wave, wh, wn};
    score_epilogue<DT, HB, NBW, WH, NW, ACT>(acc, ea, [&](int nb, float sc, float dot) __attribute__((always_inline)) {
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
            p.scores[w] = sc;
            if (p.md)
                p.md[w] = vsum * g.inv_d - (dot + p.sum_bd2) * g.inv_d;
            if (p.write_flags)
                p.flags[w] = sc > p.threshold ? 1 : 0;
        }
    });
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
