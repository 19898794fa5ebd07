// Launch planning of the fp32 matrix-core product (block tile, reduction slices, workspace) and
// of the chunking of the detector-output variant pass. Plain C++ with no device code, so the
// planner builds and is checked on the host as well as inside the library.
#pragma once

#include <algorithm>
#include <cstdint>

namespace enova {

// C tile of a block (4 waves, each a grid of 32 x 32 matrix ops): 128 x 128 as 2 x 2 waves of
// 64 x 64; for a product with at most 32 columns 128 x 32 as 4 x 1 waves of 32 x 32, and with at
// most 32 rows (and more columns) 32 x 128 as 1 x 4 waves, so a thin product does no padded work.
constexpr int kGemmTile = 128;
constexpr int kGemmThin = 32;
constexpr int kGemmK = 32;               // reduction slice staged in LDS (double-buffered)
constexpr int kGemmTargetBlocks = 256;   // split the reduction until a launch has about this many blocks
constexpr int kGemmMinSlice = 128;       // ... but keep every slice at least this long
constexpr int kGemmMaxSplits = 128;

// Waves of a TM x TN block tile along its columns.
constexpr int gemm_waves_n(int tm, int tn)
{
    return 4 / (tn == kGemmTile ? (tm == kGemmTile ? 2 : 1) : 4);
}

// The block tile of an m x n product (rows, columns): thin products get a 32-wide side, and so
// does one whose 128 x 128 tiles would leave most of the chip idle (its longer side is cut into
// 4x as many tiles, so it needs fewer reduction slices, or none).
inline void gemm_tile(int m, int n, int &tm, int &tn)
{
    tm = kGemmTile;
    tn = kGemmTile;
    if (n <= kGemmThin) {
        tn = kGemmThin;
    } else if (m <= kGemmThin) {
        tm = kGemmThin;
    } else {
        const int64_t tiles = static_cast<int64_t>((m + kGemmTile - 1) / kGemmTile) * ((n + kGemmTile - 1) / kGemmTile);
        if (tiles < kGemmTargetBlocks / 2) {
            if (m >= n)
                tm = kGemmThin;
            else
                tn = kGemmThin;
        }
    }
}

// Reduction slices wanted for an m x n x k product (1: none).
inline int gemm_splits(int m, int n, int k)
{
    int tm, tn;
    gemm_tile(m, n, tm, tn);
    const int64_t tiles = static_cast<int64_t>((m + tm - 1) / tm) * ((n + tn - 1) / tn);
    if (tiles >= kGemmTargetBlocks / 2)
        return 1;
    const int by_k = (k + kGemmMinSlice - 1) / kGemmMinSlice;
    const int by_grid = static_cast<int>((kGemmTargetBlocks + tiles - 1) / tiles);
    return std::max(1, std::min({by_k, by_grid, kGemmMaxSplits}));
}

// Floats of one slice's partial results: the m x n tile and the m row sums.
inline int64_t gemm_slice_floats(int m, int n)
{
    return static_cast<int64_t>(m) * n + m;
}

// Workspace an m x n x k product needs to split as far as it wants (0: it does not split).
inline int64_t gemm_workspace_floats(int m, int n, int k)
{
    const int s = gemm_splits(m, n, k);
    return s > 1 ? static_cast<int64_t>(s) * gemm_slice_floats(m, n) : 0;
}

// Column slots of an m x n product whose epilogue reduces per row (at most (n + 31) / 32).
inline int gemm_reduce_slots(int m, int n)
{
    int tm, tn;
    gemm_tile(m, n, tm, tn);
    const int cw = tn / gemm_waves_n(tm, tn);
    return (n + cw - 1) / cw;
}

struct GemmPlan {
    int tm, tn;     // block tile
    int kc;         // reduction indices per slice (a multiple of kGemmK when split)
    int used;       // slices launched: ceil(k / kc); their partials need used * slice floats
};

// The launch of an m x n x k product. It splits only when `may_split` (a workspace is given and
// the epilogue allows it) and never into more slices than `work_floats` floats of workspace hold:
// used * gemm_slice_floats(m, n) <= work_floats whenever used > 1.
inline GemmPlan gemm_plan(int m, int n, int k, bool may_split, int64_t work_floats)
{
    GemmPlan p{};
    gemm_tile(m, n, p.tm, p.tn);
    int splits = may_split ? gemm_splits(m, n, k) : 1;
    const int64_t per_slice = gemm_slice_floats(m, n);
    while (splits > 1 && static_cast<int64_t>(splits) * per_slice > work_floats)
        --splits;
    p.kc = splits > 1 ? ((k + splits - 1) / splits + kGemmK - 1) / kGemmK * kGemmK : std::max(k, 1);
    p.used = splits > 1 ? (k + p.kc - 1) / p.kc : 1;
    return p;
}

// ---------------------------------------------------------------------------------------------
// Register-streamed products (k_gemm_rs): no LDS staging and no barrier inside the reduction.
// The four waves of a block each cover every fourth 16-deep step of the block's reduction range
// for the whole tile; the partial tiles are added in LDS in wave order. Every operand fragment is
// one 16-byte load per lane straight from global memory: along the reduction index for a
// k-contiguous operand, along its rows for a row-contiguous one. Only whole tiles and whole
// prefetch groups are planned; anything else takes k_gemm.
//   kRsK4: k-contiguous A, either B, a reduction of at least 512, fewer than 128 tiles of
//          128 x 128; 32 x 128 tiles
//   kRsR4: both row-contiguous (weight gradients); 64 x 64 tiles, the reduction also split over
//          blocks when the tiles are few (partials summed in slice order)
// ---------------------------------------------------------------------------------------------
enum { kRsNone = 0, kRsK4 = 1, kRsR4 = 3 };
constexpr int kRsStep = 16;          // reduction indices per wave iteration
constexpr int kRsWaves = 4;          // waves of a block, along the reduction
struct RsShape {
    int tm, tn;      // block tile
    int pd;          // register slots of operand prefetch (loads run pd - 1 iterations ahead; the
                     // unroll of the reduction loop)
};
constexpr RsShape rs_shape(int kind) { return kind == kRsK4 ? RsShape{32, 128, 2} : RsShape{64, 64, 2}; }
// Reduction indices one block covers per unrolled loop trip.
constexpr int rs_k_unit(int kind) { return kRsStep * kRsWaves * rs_shape(kind).pd; }

struct RsPlan {
    int kind;        // kRsNone: use k_gemm
    int kc;          // reduction indices per slice (k when not split)
    int used;        // slices
};

// Slices a kRsR4 product wants: about kGemmTargetBlocks blocks, each slice a whole number of
// loop trips.
inline int rs_r4_splits(int m, int n, int k, int64_t work_floats)
{
    const int64_t tiles = static_cast<int64_t>(m / rs_shape(kRsR4).tm) * (n / rs_shape(kRsR4).tn);
    const int unit = rs_k_unit(kRsR4);
    const int64_t want = (kGemmTargetBlocks + tiles - 1) / tiles;
    int s = 1;
    for (int c = 2; c <= kGemmMaxSplits && c <= want; ++c)
        if (k % (c * unit) == 0 && static_cast<int64_t>(c) * gemm_slice_floats(m, n) <= work_floats)
            s = c;
    return s;
}

// The register-streamed launch of an m x n x k product, or kind kRsNone. `epi_ok`: the epilogue
// is one the kernel applies (store, bias + activation, activation derivative); `vec`: both
// operands are 16-byte aligned with leading dimensions that are multiples of 4. Splits (kRsR4
// only) obey the same workspace bound as gemm_plan: used * gemm_slice_floats(m, n) <= work_floats.
inline RsPlan gemm_rs_plan(int m, int n, int k, bool a_k, bool b_k, bool epi_ok, bool vec, bool may_split,
                           int64_t work_floats)
{
    RsPlan p{kRsNone, 0, 0};
    if (!epi_ok || !vec || m <= 0 || n <= 0 || k <= 0)
        return p;
    // kRsK4 only where k_gemm's 128 x 128 tiles would leave most of the chip idle (it then cuts
    // 32-wide tiles, the shape this kernel beats); with many tiles k_gemm's LDS reuse wins
    const int64_t tiles128 = static_cast<int64_t>((m + kGemmTile - 1) / kGemmTile) * ((n + kGemmTile - 1) / kGemmTile);
    if (a_k && k >= 512 && m % 32 == 0 && n % 128 == 0 && k % rs_k_unit(kRsK4) == 0 &&
        tiles128 < kGemmTargetBlocks / 2) {
        p = RsPlan{kRsK4, k, 1};
    } else if (!a_k && !b_k && m % 64 == 0 && n % 64 == 0 && k % rs_k_unit(kRsR4) == 0) {
        const int s = may_split ? rs_r4_splits(m, n, k, work_floats) : 1;
        p = RsPlan{kRsR4, k / s, s};
    }
    return p;
}

// Workspace a register-streamed product wants (0: none, or it does not take that kernel).
inline int64_t gemm_rs_workspace_floats(int m, int n, int k, bool a_k, bool b_k)
{
    const RsPlan p = gemm_rs_plan(m, n, k, a_k, b_k, true, true, true, int64_t{1} << 60);
    return p.used > 1 ? static_cast<int64_t>(p.used) * gemm_slice_floats(m, n) : 0;
}

// Split workspace (floats) of one training step over a batch of B windows: every product of the
// step as (m, n, k) -- forward encoder, heads, decoder hidden and output; backward the decoder
// output's weight and input gradients, the decoder hidden layer's, the heads', the encoder's
// weight gradient.
inline int64_t train_gemm_workspace(int B, int D, int H, int L)
{
    // (m, n, k, A k-contiguous, B k-contiguous)
    const int shapes[][5] = {{B, H, D, 1, 1},     {B, 2 * L, H, 1, 1}, {B, H, L, 1, 1}, {B, D, H, 1, 1},
                             {D, H, B, 0, 0},     {B, H, D, 1, 0},     {H, L, B, 0, 0}, {B, L, H, 1, 0},
                             {2 * L, H, B, 0, 0}, {B, H, 2 * L, 1, 0}, {H, D, B, 0, 0}};
    int64_t ws = 0;
    for (const auto &sh : shapes) {
        ws = std::max(ws, gemm_workspace_floats(sh[0], sh[1], sh[2]));
        ws = std::max(ws, gemm_rs_workspace_floats(sh[0], sh[1], sh[2], sh[3] != 0, sh[4] != 0));
    }
    return ws;
}

// The step's four weight-gradient products (both operands row-contiguous, k = B) leave their
// slice partials for the Adam step to sum, so each has a workspace region of its own:
// which = 0 dWd2 (D x H), 1 dWd1 (H x L), 2 the heads' [dWmu; dWlv] (2L x H), 3 dW1 (H x D).
constexpr int kTrainGradProducts = 4;
inline void train_grad_shape(int B, int D, int H, int L, int which, int &m, int &n, int &k)
{
    const int shapes[kTrainGradProducts][2] = {{D, H}, {H, L}, {2 * L, H}, {H, D}};
    m = shapes[which][0];
    n = shapes[which][1];
    k = B;
}
inline int64_t train_grad_workspace(int B, int D, int H, int L, int which)
{
    int m, n, k;
    train_grad_shape(B, D, H, L, which, m, n, k);
    return std::max(gemm_workspace_floats(m, n, k), gemm_rs_workspace_floats(m, n, k, false, false));
}

// ---------------------------------------------------------------------------------------------
// Variant pass: windows are evaluated densely in chunks of `variants_chunk` rows, the last chunk
// shorter. Its four products per chunk (rows x H x D encoder, rows x 2L x H heads, rows x H x L
// decoder hidden, rows x D x H decoder output) share one split workspace sized for the full and
// the last chunk.
// ---------------------------------------------------------------------------------------------

// Windows per chunk: about 1 GiB of V (every chunk pays each kernel's fixed launch cost once), at
// least 256 and at most 262144 rows, never more than the windows there are.
inline int variants_chunk(int D, int64_t n_windows)
{
    int64_t c = (int64_t{1} << 28) / D;
    c = std::max<int64_t>(256, std::min<int64_t>(c, 262144));
    return static_cast<int>(std::min<int64_t>(c, std::max<int64_t>(n_windows, 1)));
}

// Rows of the last chunk of n_windows >= 1 windows in chunks of B.
inline int variants_last_rows(int64_t n_windows, int B)
{
    return static_cast<int>(n_windows - (n_windows - 1) / B * B);
}

// Split workspace (floats) of the variant pass's products over chunks of B rows and a last chunk.
inline int64_t variants_gemm_workspace(int B, int last, int D, int H, int L)
{
    int64_t ws = 0;
    for (const int rows : {B, last}) {
        const int shapes[][3] = {{rows, H, D}, {rows, 2 * L, H}, {rows, H, L}, {rows, D, H}};
        for (const auto &sh : shapes)
            ws = std::max(ws, gemm_workspace_floats(sh[0], sh[1], sh[2]));
    }
    return ws;
}

}  // namespace enova
