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

// Split workspace (floats) of one training step over a batch of B windows: every product of the
// step as (m, n, k) -- forward encoder, heads, decoder hidden and output; backward the decoder
// output's weight and input gradients, the decoder hidden layer's, the heads', the encoder's
// weight gradient.
inline int64_t train_gemm_workspace(int B, int D, int H, int L)
{
    const int shapes[][3] = {{B, H, D}, {B, 2 * L, H}, {B, H, L},     {B, D, H},     {D, H, B}, {B, H, D},
                             {H, L, B}, {B, L, H},     {2 * L, H, B}, {B, H, 2 * L}, {H, D, B}};
    int64_t ws = 0;
    for (const auto &sh : shapes)
        ws = std::max(ws, gemm_workspace_floats(sh[0], sh[1], sh[2]));
    return ws;
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
