// Matrix-core scoring kernel of the bf16 detectors with 193..256 hidden units (gfx950).
//
// The same computation as k_score_mfma (Section IV-B: normalise, encoder, posterior heads, KL
// score, decoder hidden layer for the md) with a layout built around the bf16 matrix op
// v_mfma_f32_16x16x32_bf16 and around keeping two tiles in flight on every compute unit:
//
//  * A tile is 128 consecutive windows of one stream; a block of four waves scores it, wave w
//    owning hidden rows 64w .. 64w+63 (four 16-row blocks) for all 128 windows (eight 16-window
//    blocks): 32 matrix ops per 32-deep reduction step, A = W1 fragments streamed from L2,
//    B = window fragments from LDS.
//  * The window is cut into Q super-rows of S steps (as in k_score_mfma); window n at reduction
//    super-row q reads tile super-row n + q. The LDS holds a ring of R >= 136 super-rows (R a
//    multiple of 8) instead of all 127 + Q of them: before the loop the first 130 are staged;
//    during super-row step q one wave loads, normalises and writes super-row q + 130 (first read
//    two steps later) into the slot of a super-row no window reads any more, and a barrier after
//    every second step publishes it.
//    That keeps a block's LDS under half a compute unit's, so two blocks run per compute unit
//    and one block's staging and epilogue overlap the other's matrix work.
//  * Chunk c (16 bytes, 8 bf16) of tile super-row r, held in ring slot r mod R, lives at
//    (r mod R) * P + (c ^ key(r)), key(r) = (r & 7) << 1: the 16 windows of a fragment read 16
//    consecutive super-rows at one chunk column, and this XOR makes that 128-bit LDS read free of
//    bank conflicts on gfx950 (measured with rocprofv3's SQ_LDS_BANK_CONFLICT on the kernel's
//    exact read sequence: 0 with this key, 33% of LDS cycles with r & 15, 50% with an odd row
//    pitch). Keyed by the super-row, not the slot, the key is the same for every window block.
//    P = the super-row's chunks rounded up to a multiple of 16: whole XOR groups and whole groups
//    of four reduction steps; padding chunks hold zeros and meet zero weights.
//
// Epilogue: the 16x16 accumulator layout (lane l, register r: row 4*(l/16) + r, column l%16)
// supplies the B operands of the following ops directly: two hidden blocks' accumulators are the
// eight reduction slots of a 16x16x32 heads op, and the mean head's accumulator is the four
// reduction slots of a 16x16x16 decoder op; weights are pre-permuted to match on the host and,
// with the activations, split into bf16 hi + lo parts (three ops, about 16 significant bits).
// The four waves' partial head sums are added through LDS in a fixed order, so a window's
// score does not depend on which block or batch computed it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "internal.h"
#include "mfma_common.h"

namespace enova {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));

constexpr int kNT = 64 * kRingWaves;     // threads of a block
constexpr int kBlk = kRingNb / 16;       // 16-window blocks of a tile
constexpr int kHbw = 4;                  // 16-row hidden blocks of a wave
constexpr int kHbt = kHbw * kRingWaves;  // 16-row hidden blocks of the tile (256 rows)
constexpr int kPd = 2;                   // W1 fragment prefetch depth (reduction steps)
static_assert(kHbt * 16 == kRingHidden, "four waves of 64 hidden rows");
static_assert(kPd <= kPrefetchSteps, "W1 prefetch runs into the appended zero steps");

struct RingShape {
    int M, S, Mp, Q, CPR;
    int P;            // LDS chunks per ring slot (multiple of 16)
    int KS;           // reduction steps per super-row: P / 4 (a multiple of kPd)
    int R;            // ring slots (multiple of 8, >= kRingNb + 8)
    int SMp;          // elements of a super-row: S * Mp = 8 * CPR
    int tail_elems;   // elements of a window's last super-row that belong to the window
    int rs_rows;      // entries of the row-sum arrays: kRingNb + Q + 1
    int ring_floats;  // floats of the ring region (also the epilogue's exchange buffer)
    int cus;          // compute units of the device
    int start_sleeps; // s_sleep(127) rounds of the first wave's second blocks before their tile
    float inv_d;
};

__device__ __forceinline__ v4f mfma16x32(uint4 a, uint4 b, v4f c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c,
                                                   0, 0, 0);
}

__device__ __forceinline__ v4f mfma16x16(uint2 a, v4s b, v4f c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(v4s, a), b, c, 0, 0, 0);
}

// x = hi + lo for four values (see split_bf16x8)
__device__ __forceinline__ void split_bf16x4(const float (&x)[4], v4s &hi, v4s &lo)
{
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const __bf16 h = static_cast<__bf16>(x[t]);
        hi[t] = __builtin_bit_cast(short, h);
        lo[t] = __builtin_bit_cast(short, static_cast<__bf16>(x[t] - static_cast<float>(h)));
    }
}

// Block barrier that publishes LDS only: this wave's LDS operations complete, then s_barrier. Unlike
// __syncthreads() it leaves global loads in flight (its workgroup fence would wait for every
// outstanding load, draining the W1 prefetch at each super-row step); the memory clobber keeps
// the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// XOR key of the chunks of tile super-row r in its ring slot (see the layout note above)
__device__ __forceinline__ int ring_key(int r) { return (r & 7) << 1; }

__device__ __forceinline__ void unpack8(const uint4 q, float (&e)[8])
{
    e[0] = bf16_lo(q.x);
    e[1] = bf16_hi(q.x);
    e[2] = bf16_lo(q.y);
    e[3] = bf16_hi(q.y);
    e[4] = bf16_lo(q.z);
    e[5] = bf16_hi(q.z);
    e[6] = bf16_lo(q.w);
    e[7] = bf16_hi(q.w);
}

template <int ACT>
__global__ __launch_bounds__(kNT, 2) void k_score_ring(ScoreParams p, RingShape g)
{
    extern __shared__ uint4 lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = lane >> 4;     // lane group: reduction slots 8*grp.. of an op, result rows 4*grp..
    const int col = lane & 15;     // window (or weight row) of this lane inside a 16-block

    // ---- tile -> (stream, first window)
    const int64_t b = blockIdx.x;
    const int s = p.tile_stream[b];
    if (s < 0)
        return;
    const int64_t k0 = (b - p.tile_off[s]) * kRingNb;
    const int64_t ns = p.woff[s + 1] - p.woff[s];
    const int nv = static_cast<int>(ns - k0 < kRingNb ? ns - k0 : kRingNb);
    const int64_t srow = p.soff[s];
    const int64_t T = p.soff[s + 1] - srow;
    const int M = g.M, Mp = g.Mp, S = g.S, Q = g.Q, P = g.P, KS = g.KS, R = g.R, CPR = g.CPR;

    // ---- LDS: ring [R][P] chunks (reused by the epilogue's exchange), the per-element
    // statistics and offsets of a super-row, row sums, and the epilogue's small vectors
    uint4 *ring = lds;
    // element e of chunk c of a super-row: its metric's mean and 1/std (0 for padding) and its
    // offset from the super-row's first element in the stream (-1 for padding), element-major
    // ([e][c], P entries per e) so that lanes reading consecutive chunks read consecutive words
    float *cmean = reinterpret_cast<float *>(lds) + g.ring_floats;
    float *crinv = cmean + 8 * P;
    int *coff = reinterpret_cast<int *>(crinv + 8 * P);
    float *rs = reinterpret_cast<float *>(coff + 8 * P);
    float *ps = rs + g.rs_rows;
    float *s_b1 = ps + g.rs_rows;
    float *s_bd1 = s_b1 + kRingHidden;
    float *s_u = s_bd1 + kRingHidden;
    float *s_bh = s_u + kRingHidden;

    for (int i = tid; i < kRingHidden; i += kNT) {
        s_b1[i] = p.b1[i];
        s_bd1[i] = p.bd1[i];
        s_u[i] = p.u[i];
    }
    if (tid < 32)
        s_bh[tid] = p.bh[tid];
    // Two blocks run per compute unit. The dispatcher starts blocks b and b + cus together on one
    // compute unit, and tiles take equally long, so the pair -- and every pair dispatched into the
    // slots they free -- would stay in step and wait on HBM in the same staging phases. The first
    // wave's second blocks start about half a tile late instead, once; the pairs after them
    // inherit the offset, so one block's staging and epilogue run under the other's matrix work.
    if (blockIdx.x >= g.cus && blockIdx.x < 2 * g.cus) {
        for (int i = 0; i < g.start_sleeps; ++i)
            __builtin_amdgcn_s_sleep(127);
    }
    for (int j = tid; j < 8 * P; j += kNT) {
        const int e = j / P, c = j - (j / P) * P;
        const int jj = c * 8 + e;                 // element of the super-row
        const int tt = jj / Mp;
        const int m = jj - tt * Mp;
        const int t = e * P + c;
        if (jj < g.SMp && m < M) {
            cmean[t] = p.mean[static_cast<int64_t>(s) * M + m];
            crinv[t] = 1.0f / p.std[static_cast<int64_t>(s) * M + m];
            coff[t] = tt * M + m;
        } else {
            cmean[t] = 0.0f;
            crinv[t] = 0.0f;
            coff[t] = -1;
        }
    }
    __syncthreads();

    // ---- staging helpers: tile super-row r covers stream steps (k0 + r) * S .. + S - 1
    const int64_t step0 = k0 * S;
    const int64_t eavail = (T - step0) * M;        // stream elements from tile super-row 0 on
    const bool linear = (Mp == M) && (((srow + step0) * M) % 8 == 0);
    const int64_t ebase = (srow + step0) * M;
    const uint16_t *xb = static_cast<const uint16_t *>(p.x);
    // issue the 16-byte load of chunk c of super-row r when it is whole, aligned and in the stream
    auto fetch = [&](int r, int c, uint4 &raw) -> bool {
        const int64_t e0 = (static_cast<int64_t>(r) * CPR + c) * 8;
        const bool vec = c < CPR && linear && e0 + 8 <= eavail;
        if (vec)
            raw = *reinterpret_cast<const uint4 *>(xb + ebase + e0);
        return vec;
    };
    // the normalised chunk (zero for padding and beyond the stream), rounded to bf16
    auto finish = [&](int r, int c, const uint4 &raw, bool vec, float (&v)[8]) {
        if (c >= CPR) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                v[e] = 0.0f;
            return;
        }
        if (vec) {
            unpack8(raw, v);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                v[e] = (v[e] - cmean[e * P + c]) * crinv[e * P + c];
        } else {
            const int64_t rel = static_cast<int64_t>(r) * S * M;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int off = coff[e * P + c];
                float val = 0.0f;
                if (off >= 0 && rel + off < eavail)
                    val = (load_x<ENOVA_BF16>(p.x, ebase + rel + off) - cmean[e * P + c]) * crinv[e * P + c];
                v[e] = val;
            }
        }
    };
    auto pack = [](const float (&v)[8]) {
        uint4 out;
        out.x = pack_bf16x2(v[0], v[1]);
        out.y = pack_bf16x2(v[2], v[3]);
        out.z = pack_bf16x2(v[4], v[5]);
        out.w = pack_bf16x2(v[6], v[7]);
        return out;
    };
    // row sums of the staged (bf16) values of super-row r: lane c < P holds chunk c; every lane of
    // the wave takes part in the fixed-order butterfly
    const int tail_elems = g.tail_elems;
    auto row_sums = [&](int r, int c, const uint4 &q, bool have) {
        float full = 0.0f, part = 0.0f;
        if (have) {
            float e[8];
            unpack8(q, e);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                full += e[k];
                if (c * 8 + k < tail_elems)
                    part += e[k];
            }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            full += __shfl_xor(full, o);
            part += __shfl_xor(part, o);
        }
        if (c == 0) {
            rs[r] = full;
            ps[r] = part;
        }
    };

    const int rows_need = nv + Q - 1;            // tile super-rows any valid window reads
    // ---- stage super-rows 0 .. kRingNb + 1 into slots 0 .. kRingNb + 1, every load of a thread in flight
    // at once (one HBM round trip for the usual shapes); the super-rows the loop streams in later
    // are touched once per 128-byte line meanwhile, so their loads hit L2
    {
        constexpr int SU = 20;
        const int n_chunks = (kRingNb + 2) * P;
        const int lines_per_row = P / 8;
        const int n_pre = rows_need > kRingNb + 2 ? (rows_need - kRingNb - 2) * lines_per_row : 0;
        float sink = 0.0f;
        for (int i = tid; i < n_pre; i += kNT) {
            const int r = kRingNb + 2 + i / lines_per_row;
            const int64_t e0 = (static_cast<int64_t>(r) * CPR + (i % lines_per_row) * 8) * 8;
            if (e0 < eavail)
                sink += load_x<ENOVA_BF16>(p.x, ebase + e0);
        }
        for (int base = tid; base < n_chunks; base += kNT * SU) {
            uint4 raw[SU];
            bool vec[SU];
#pragma unroll
            for (int u = 0; u < SU; ++u) {
                const int idx = base + u * kNT;
                const int r = idx / P, c = idx - (idx / P) * P;
                vec[u] = idx < n_chunks && fetch(r, c, raw[u]);
            }
#pragma unroll
            for (int u = 0; u < SU; ++u) {
                const int idx = base + u * kNT;
                if (idx < n_chunks) {
                    const int r = idx / P, c = idx - (idx / P) * P;
                    float v[8];
                    finish(r, c, raw[u], vec[u], v);
                    ring[r * P + (c ^ ring_key(r))] = pack(v);
                }
            }
        }
        asm volatile("" ::"v"(sink));          // keeps the line touches (their values are not used)
    }
    __syncthreads();
    for (int r = wave; r <= kRingNb + 1; r += kRingWaves) {
        uint4 q = make_uint4(0, 0, 0, 0);
        if (lane < P)
            q = ring[r * P + (lane ^ ring_key(r))];
        row_sums(r, lane, q, lane < P);
    }

    // ---- main contraction: acc[hb][nb] = W1 rows of hidden block 4*wave + hb x windows of block nb
    v4f acc[kHbw][kBlk];
#pragma unroll
    for (int hb = 0; hb < kHbw; ++hb)
#pragma unroll
        for (int nb = 0; nb < kBlk; ++nb)
            acc[hb][nb] = v4f{0.0f, 0.0f, 0.0f, 0.0f};

    const int nblk = (nv + 15) >> 4;             // 16-window blocks holding a valid window
    // A fragments of step i, hidden block hb: w1r[(i * kHbt + hb) * 64 + lane]
    const uint4 *ap = p.w1r + (wave * kHbw) * 64 + lane;

    // the contraction for the tile's NBA active 16-window blocks (a compile-time count, so the
    // unrolled step has no branches)
    // The contraction for the tile's NBA active 16-window blocks, with KSC reduction steps per
    // super-row (0: KS at run time; the usual count is unrolled so the compiler's wait counts stay
    // exact across the whole super-row step). Compile-time counts keep the unrolled step free of
    // branches.
    auto run = [&](auto nba_tag, auto ks_tag) {
        constexpr int NBA = decltype(nba_tag)::value;
        constexpr int KSC = decltype(ks_tag)::value;
        uint4 a[kPd][kHbw];
#pragma unroll
        for (int j = 0; j < kPd; ++j)
#pragma unroll
            for (int hb = 0; hb < kHbw; ++hb)
                a[j][hb] = ap[(j * kHbt + hb) * 64];
        const uint4 *api = ap + kPd * kHbt * 64;
        // one reduction step: block nb's four ops, then the next step's fragment of block nb into
        // the register the ops just read (NEXT: the super-row's last step, whose next fragments are
        // those of the next super-row step, one slot further), then the W1 fragments of the step
        // kPd ahead into the registers of this step's. The order is pinned: left to itself the scheduler sinks every load to
        // just before its use.
        uint4 bq[NBA];
        int bofs[NBA];                             // LDS chunk offset of each active block's ring slot
        const int RP = R * P;
        auto step = [&](auto next_tag, uint4 (&av)[kHbw], int cnext, const uint4 *anext) {
            constexpr bool NEXT = decltype(next_tag)::value;
#pragma unroll
            for (int nb = 0; nb < NBA; ++nb) {
#pragma unroll
                for (int hb = 0; hb < kHbw; ++hb)
                    acc[hb][nb] = mfma16x32(av[hb], bq[nb], acc[hb][nb]);
                int o = bofs[nb];
                if constexpr (NEXT) {                // the block's slot in the next super-row step
                    o += P;
                    o = o == RP ? 0 : o;
                }
                bq[nb] = ring[o + cnext];
            }
#pragma unroll
            for (int hb = 0; hb < kHbw; ++hb)
                av[hb] = anext[hb * 64];
#pragma unroll
            for (int nb = 0; nb < NBA; ++nb) {
                __builtin_amdgcn_sched_group_barrier(0x008, kHbw, 0);   // the block's matrix ops
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // its next fragment (LDS)
            }
            __builtin_amdgcn_sched_group_barrier(0x020, kHbw, 0);       // W1 reloads (global)
            __builtin_amdgcn_sched_barrier(0);
        };
        // LDS chunk offset of each active block's ring slot: block nb reads slot s0 + 16 nb (mod R)
        auto offsets = [&](int s0, int (&bo)[NBA]) {
#pragma unroll
            for (int nb = 0; nb < NBA; ++nb) {
                const int sl = s0 + 16 * nb;
                bo[nb] = (sl >= R ? sl - R : sl) * P;
            }
        };
        int sl0 = col;                            // ring slot of tile super-row col + q
        int sn = kRingNb + 2;                     // ring slot of this step's new super-row q + kRingNb + 2
        int xo = ring_key(col);                   // XOR key of every block's super-row 16 nb + col + q
        offsets(sl0, bofs);
#pragma unroll
        for (int nb = 0; nb < NBA; ++nb)
            bq[nb] = ring[bofs[nb] + (grp ^ xo)];
        for (int q = 0; q < Q; ++q) {
            // this step's new super-row: wave q % 4 loads it now and writes it after the matrix work
            const int rn = q + kRingNb + 2;
            const bool stager = (q & (kRingWaves - 1)) == wave && rn < rows_need;
            // the stager's per-lane values are recomputed from an opaque copy of the lane index,
            // so they are not kept live (or spilled) across the matrix work
            int ln = lane;
            asm volatile("" : "+v"(ln));
            // every lane of every wave issues the load, with no branch (only the stager uses it; a
            // lane without a whole in-stream chunk reads the packed W1 instead and ignores it): a
            // load under a branch would leave the compiler unsure which loads are pending at the
            // next wait, and it would then wait for all of them, the W1 prefetch included
            const int64_t se0 = (static_cast<int64_t>(rn) * CPR + ln) * 8;
            const bool svec = ln < CPR && rn < rows_need && linear && se0 + 8 <= eavail;
            const uint4 sraw = *(svec ? reinterpret_cast<const uint4 *>(xb + ebase + se0) : p.w1r);
            // the next super-row step's slots and key: its first fragments are read during this
            // step's last reduction step (super-rows q + 1 .. q + kRingNb, all published by now)
            const int sl1 = sl0 + 1 == R ? 0 : sl0 + 1;
            const int xo1 = ring_key(col + q + 1);
            // all steps but the last kPd, then those (the very last one reads ahead into the next
            // super-row step), so no step needs a branch
            auto group = [&](int sp) {
#pragma unroll
                for (int j = 0; j < kPd; ++j)
                    step(std::false_type{}, a[j], (4 * (sp + j + 1) + grp) ^ xo, api + j * kHbt * 64);
                api += kPd * kHbt * 64;
            };
            if constexpr (KSC > 0) {
#pragma unroll
                for (int sp = 0; sp < KSC - kPd; sp += kPd)
                    group(sp);
            } else {
                for (int sp = 0; sp < KS - kPd; sp += kPd)
                    group(sp);
            }
            {
                const int sp = (KSC > 0 ? KSC : KS) - kPd;
#pragma unroll
                for (int j = 0; j + 1 < kPd; ++j)
                    step(std::false_type{}, a[j], (4 * (sp + j + 1) + grp) ^ xo, api + j * kHbt * 64);
                step(std::true_type{}, a[kPd - 1], grp ^ xo1, api + (kPd - 1) * kHbt * 64);
                api += kPd * kHbt * 64;
            }
            if (stager) {
                const int sl = sn;                // held super-row rn - R (or nothing): no longer read
                asm volatile("" : "+v"(ln));
                float v[8];
                finish(rn, ln, sraw, svec, v);
                const uint4 out = pack(v);
                if (ln < P)
                    ring[sl * P + (ln ^ ring_key(rn))] = out;
                row_sums(rn, ln, out, ln < P);
            }
            sl0 = sl1;
            xo = xo1;
            offsets(sl0, bofs);
            sn = sn + 1 == R ? 0 : sn + 1;
            // a barrier after every odd step (and the last): the super-row staged at step q is first
            // read in step q + 2 (by the next-fragment read of its last reduction step), and one of
            // q, q + 1 is odd; the slot it overwrites was last read in step q - 6, and no wave runs
            // more than three steps ahead of another
            if ((q & 1) || q == Q - 1)
                lds_barrier();
        }
    };
    auto go = [&](auto nba_tag) {
        if (KS == 8)
            run(nba_tag, std::integral_constant<int, 8>{});
        else
            run(nba_tag, std::integral_constant<int, 0>{});
    };
    switch (nblk) {
    case 8: go(std::integral_constant<int, 8>{}); break;
    case 7: go(std::integral_constant<int, 7>{}); break;
    case 6: go(std::integral_constant<int, 6>{}); break;
    case 5: go(std::integral_constant<int, 5>{}); break;
    case 4: go(std::integral_constant<int, 4>{}); break;
    case 3: go(std::integral_constant<int, 3>{}); break;
    case 2: go(std::integral_constant<int, 2>{}); break;
    default: go(std::integral_constant<int, 1>{}); break;
    }
    static_assert(kBlk == 8, "one contraction variant per active block count");

    // ---- epilogue. Heads: wave partials over its 64 hidden rows, hidden activations as the B
    // operand (slots 0..3: rows 4*grp + t of block 2m, slots 4..7: of block 2m + 1)
    const uint4 *whr = p.whr;     // [wave][m][zb][hi, lo][lane]
    v4f zp[2][kBlk];
#pragma unroll
    for (int zb = 0; zb < 2; ++zb)
#pragma unroll
        for (int nb = 0; nb < kBlk; ++nb)
            zp[zb][nb] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        uint4 wa[2][2];
#pragma unroll
        for (int zb = 0; zb < 2; ++zb)
#pragma unroll
            for (int hl = 0; hl < 2; ++hl)
                wa[zb][hl] = whr[((((wave * 2 + m) * 2 + zb) * 2) + hl) * 64 + lane];
        const int h0 = 16 * (kHbw * wave + 2 * m) + 4 * grp;
#pragma unroll
        for (int nb = 0; nb < kBlk; ++nb) {
            float hv[8];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                hv[t] = act_fn<ACT>(acc[2 * m][nb][t] + s_b1[h0 + t]);
                hv[4 + t] = act_fn<ACT>(acc[2 * m + 1][nb][t] + s_b1[h0 + 16 + t]);
            }
            v8bf hh, hlo;
            split_bf16x8(hv, hh, hlo);
            const uint4 bh = __builtin_bit_cast(uint4, hh), bl = __builtin_bit_cast(uint4, hlo);
#pragma unroll
            for (int zb = 0; zb < 2; ++zb) {
                zp[zb][nb] = mfma16x32(wa[zb][0], bh, zp[zb][nb]);
                zp[zb][nb] = mfma16x32(wa[zb][0], bl, zp[zb][nb]);
                zp[zb][nb] = mfma16x32(wa[zb][1], bh, zp[zb][nb]);
            }
        }
    }
    // exchange: wave w then adds the four partials of window blocks 2w, 2w + 1 in wave order
    float *xz = reinterpret_cast<float *>(lds);     // [wave][zb][nb][r][lane]
#pragma unroll
    for (int zb = 0; zb < 2; ++zb)
#pragma unroll
        for (int nb = 0; nb < kBlk; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                xz[(((wave * 2 + zb) * kBlk + nb) * 4 + r) * 64 + lane] = zp[zb][nb][r];
    __syncthreads();
    constexpr int kOwn = kBlk / kRingWaves;          // window blocks a wave finishes
    v4f z[2][kOwn];
#pragma unroll
    for (int zb = 0; zb < 2; ++zb)
#pragma unroll
        for (int i = 0; i < kOwn; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float t = 0.0f;
#pragma unroll
                for (int w2 = 0; w2 < kRingWaves; ++w2)
                    t += xz[(((w2 * 2 + zb) * kBlk + kOwn * wave + i) * 4 + r) * 64 + lane];
                z[zb][i][r] = t;
            }
    // biases, KL score (latent 4*grp + r of this lane; the four lane groups add up)
    float kl[kOwn];
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
        kl[i] = 0.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float mu = z[0][i][r] + s_bh[4 * grp + r];
            const float lv = z[1][i][r] + s_bh[16 + 4 * grp + r];
            z[0][i][r] = mu;
            kl[i] += mu * mu + kl_g(lv);
        }
        kl[i] += __shfl_xor(kl[i], 16);
        kl[i] += __shfl_xor(kl[i], 32);
    }
    // decoder hidden layer at z = mu (B operand: the mean head's accumulator), dotted with u
    v4s mh[kOwn], ml[kOwn];
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
        float mv[4] = {z[0][i][0], z[0][i][1], z[0][i][2], z[0][i][3]};
        split_bf16x4(mv, mh[i], ml[i]);
    }
    float dot[kOwn];
#pragma unroll
    for (int i = 0; i < kOwn; ++i)
        dot[i] = 0.0f;
    const uint2 *wdr = p.wdr;     // [hidden block][hi, lo][lane]
#pragma unroll 4
    for (int hb = 0; hb < kHbt; ++hb) {
        const uint2 wh = wdr[(hb * 2 + 0) * 64 + lane];
        const uint2 wl = wdr[(hb * 2 + 1) * 64 + lane];
#pragma unroll
        for (int i = 0; i < kOwn; ++i) {
            v4f d = v4f{0.0f, 0.0f, 0.0f, 0.0f};
            d = mfma16x16(wh, mh[i], d);
            d = mfma16x16(wh, ml[i], d);
            d = mfma16x16(wl, mh[i], d);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int h = 16 * hb + 4 * grp + r;
                dot[i] += s_u[h] * act_fn<ACT>(d[r] + s_bd1[h]);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
        dot[i] += __shfl_xor(dot[i], 16);
        dot[i] += __shfl_xor(dot[i], 32);
        // window mean of the staged inputs: super-rows n .. n+Q-1, the last one partially
        const int n = 16 * (kOwn * wave + i) + col;
        float vs = 0.0f;
        for (int qq = grp; qq < Q - 1; qq += 4)
            vs += rs[n + qq];
        if (((Q - 1) & 3) == grp)
            vs += ps[n + Q - 1];
        vs += __shfl_xor(vs, 16);
        vs += __shfl_xor(vs, 32);
        if (grp == 0 && n < nv) {
            const int64_t w = p.woff[s] + k0 + n;
            const float sc = 0.5f * kl[i];
            p.scores[w] = sc;
            if (p.md)
                p.md[w] = vs * g.inv_d - (dot[i] + p.sum_bd2) * g.inv_d;
            if (p.write_flags)
                p.flags[w] = sc > p.threshold ? 1 : 0;
        }
    }
}

RingShape ring_shape(const Geometry &g)
{
    RingShape sh;
    sh.M = g.M;
    sh.S = g.S;
    sh.Mp = g.Mp;
    sh.Q = g.Q;
    sh.CPR = g.CPR;
    sh.P = g.RP;
    sh.KS = g.RP / 4;
    sh.R = g.RR;
    sh.SMp = g.S * g.Mp;
    sh.tail_elems = (g.W - (g.Q - 1) * g.S) * g.Mp;
    sh.rs_rows = kRingNb + g.Q + 1;
    sh.ring_floats = g.ring_floats;
    sh.inv_d = 1.0f / static_cast<float>(g.D);
    sh.cus = 0;
    sh.start_sleeps = 0;
    return sh;
}

using RingKernel = void (*)(ScoreParams, RingShape);

RingKernel pick_ring(const Geometry &g)
{
    return g.act == ENOVA_RELU ? k_score_ring<ENOVA_RELU> : k_score_ring<ENOVA_TANH>;
}

}  // namespace

size_t ring_lds_bytes(int P, int Q, int ring_floats)
{
    return sizeof(float) * (static_cast<size_t>(ring_floats) + 3 * 8 * static_cast<size_t>(P) +
                            2 * static_cast<size_t>(kRingNb + Q + 1) + 3 * static_cast<size_t>(kRingHidden) + 32);
}

hipError_t prepare_score_ring(const Geometry &g)
{
    return hipFuncSetAttribute(reinterpret_cast<const void *>(pick_ring(g)),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(g.ring_lds));
}

hipError_t launch_score_ring(const Geometry &g, const ScoreParams &p, int64_t grid, hipStream_t st)
{
    if (grid <= 0)
        return hipSuccess;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess)
        return e;
    RingShape sh = ring_shape(g);
    sh.cus = cus;
    // half a tile of delay when the grid is several waves deep: a tile is 2 * kRingNb * 256 * D
    // flops at about 4 TFLOP/s per block; one s_sleep(127) round is about 4 us
    if (grid >= 8 * static_cast<int64_t>(cus)) {
        const double half_tile_us = 0.5 * 2.0 * kRingNb * kRingHidden * static_cast<double>(g.D) / 4e12 * 1e6;
        sh.start_sleeps = static_cast<int>(std::min(64.0, half_tile_us / 4.0));
    }
    hipLaunchKernelGGL(pick_ring(g), dim3(static_cast<unsigned>(grid)), dim3(kNT), g.ring_lds, st, p, sh);
    return hipGetLastError();
}

}  // namespace enova
