// Internal declarations of libenova_detect: kernel parameter blocks and launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

#include "enova_detect.h"

namespace enova {

// ---------------------------------------------------------------------------------------------
// Geometry of the matrix-core path.
//
// The window of W steps x M metrics is cut into Q = ceil(W/S) "super-rows" of S consecutive
// steps (S*Mp elements, Mp = M padded so a super-row is a whole number of 16-byte chunks).
// Window k of a stream consists of super-rows k .. k+Q-1 of that stream, so a tile of Nb
// consecutive windows needs only Nb+Q-1 super-rows staged in LDS: every staged element is
// normalised once and then read by up to Q windows (implicit im2col of a strided 1-D
// convolution). The reduction index is walked chunk by chunk: chunk kappa = q*CPR + c is
// 16-byte chunk c of the window's super-row q.
// ---------------------------------------------------------------------------------------------
struct Geometry {
    int M, W, S, H, L, D;   // true sizes
    int dtype, act;
    float ref_frac;
    int epc;                // elements per 16-byte chunk: 4 (f32) or 8 (bf16)
    int Mp;                 // metrics padded so that S*Mp % epc == 0
    int Q;                  // super-rows per window
    int CPR;                // chunks per super-row
    int CPRP;               // LDS row pitch in chunks (odd, so 16 consecutive rows hit distinct banks)
    int KC;                 // chunks per window, rounded up to a multiple of 2*kPrefetchSteps
    int spare;              // staged super-rows after a tile's last window's Q - 1
    int Hp;                 // hidden width padded to 32*HB
    int HB;                 // 32-row hidden blocks of the tile (Hp = 32*HB)
    int HBW;                // hidden blocks per wave
    int NBW;                // 32-window blocks per wave
    int WH;                 // waves along the hidden rows (NW/WH along the windows)
    int NW;                 // waves per block of the matrix-core kernel (4 or 8)
    bool cl;                // epilogue weights staged in LDS (else read from L2)
    int Nb;                 // windows per tile
    size_t lds_bytes;       // dynamic LDS of the matrix-core kernel
    bool mfma_ok;
    // bf16 detectors with 193..256 hidden units take the ring kernel (k_score_ring.hip) instead:
    // 128-window tiles, a ring of RR super-rows of RP chunks in LDS, two blocks per compute unit
    bool ring;
    int RP, RR;
    int ring_floats;        // floats of the ring region (at least the epilogue's 64 KiB exchange)
    size_t ring_lds;        // dynamic LDS of the ring kernel
};

constexpr int kRingNb = 128;        // windows per tile of the ring kernel
constexpr int kRingWaves = 4;       // waves per block: 64 hidden rows each
constexpr int kRingHidden = 256;    // hidden units the ring kernel is laid out for (padded)
// dynamic LDS of the ring kernel for ring slots of P chunks, Q super-rows per window
size_t ring_lds_bytes(int P, int Q, int ring_floats);

constexpr int kWaves = 4;                 // waves per block of the other kernels
constexpr int kThreads = 64 * kWaves;
constexpr size_t kLdsLimit = 160 * 1024;
// The reduction index is padded to a multiple of 2*kPrefetchSteps chunks (the matrix-core
// kernel's deepest W1 prefetch ring, in two-chunk steps); the packed W1 carries kPrefetchSteps
// zero steps after the last one, and Geometry::spare staged super-rows follow a tile's windows
// (enough for the padded chunks and kPrefetchRows steps of window-fragment prefetch), so every
// prefetch past the last step reads valid memory.
constexpr int kPrefetchSteps = 8;
constexpr int kPrefetchRows = 2;

// Fixed device scratch of the allocation-free scoring entry point: kScratchBytes per device.
// scratch_setup returns this device's copy (device must be current); the lookup happens once per
// device and is then cached.
constexpr size_t kScratchBytes = size_t{16} << 20;
hipError_t scratch_setup(int device, void **out);

// Error reporting of the C entry points: records the message returned by enova_last_error().
enova_status fail(enova_status st, const char *fmt, ...);
enova_status hip_fail(hipError_t e, const char *what);

// Keeps the caller's current device and switches to another for a call's duration.
struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess)
            return;
        ok = prev == dev || hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard()
    {
        if (ok && prev >= 0)
            (void)hipSetDevice(prev);
    }
};

bool plan_geometry(const enova_detect_config &cfg, Geometry *g);
// Wave layout of the matrix-core kernel for dtype and hb 32-row hidden blocks: hidden blocks and
// 32-window blocks per wave, waves along the hidden rows, waves per block.
void mfma_layout(int dtype, int hb, int *hbw, int *nbw, int *wh, int *nw);
// Lets the instantiation chosen for g use the full LDS of a compute unit.
hipError_t prepare_score_mfma(const Geometry &g);

// Parameter block of the scoring kernels (passed by value).
struct ScoreParams {
    const void *x;
    const int64_t *soff;
    const int64_t *woff;
    const int64_t *tile_off;     // matrix-core kernel only: first tile of each stream
    const int *tile_stream;      // matrix-core kernel only: stream of each block (-1: none)
    int n_streams;
    int64_t n_windows;
    const float *mean;
    const float *std;
    // matrix-core packed weights
    const uint4 *w1p;            // [KC/2][HB][64 lanes] 16-byte A fragments
    const float *whp;            // [HB][16][64] heads (mu rows 0..15, log-var rows 16..31)
    const float *wd1p;           // [HB][8][64]  decoder hidden layer
    // vector-kernel weights
    const void *w1t;             // [D][H] transposed W1 (float or bf16 bits)
    const float *wmu, *wlv, *wd1;
    // shared small vectors (padded to Hp / 32)
    const float *b1;             // [Hp]
    const float *bh;             // [32]: bmu (padded to 16), blv (padded to 16)
    const float *bmu, *blv;      // [L]
    const float *bd1;            // [Hp]
    const float *u;              // [Hp] column sums of Wd2
    // ring kernel: W1 as 16x16x32 A fragments [steps + kPrefetchSteps][16][64 lanes], the heads as
    // bf16 hi/lo fragments [wave][2][2][hi, lo][64], the decoder hidden layer [16][hi, lo][64]
    const uint4 *w1r;
    const uint4 *whr;
    const uint2 *wdr;
    float sum_bd2;
    float threshold;
    int write_flags;
    float *scores;
    float *md;
    uint8_t *flags;
};

// Launchers (return the launch error).
hipError_t launch_ref_stats(const Geometry &g, const void *x, const int64_t *soff, int n,
                            float *mean, float *std, hipStream_t st);
// out[s] = sum_{r<s} ceil(count(s)/div) for count(s) = (mode 0) windows of stream s,
// (mode 1) calibration windows of stream s. out has n+1 entries.
hipError_t launch_stream_scan(const Geometry &g, const int64_t *soff, const int64_t *woff, int n,
                              int mode, int div, int64_t *out, hipStream_t st);
// map[b] = the stream whose tiles include tile b (tile_off has n+1 entries), -1 for
// tile_off[n] <= b < grid.
hipError_t launch_tile_map(const int64_t *tile_off, int n, int64_t grid, int *map, hipStream_t st);
hipError_t launch_score_valu(const Geometry &g, const ScoreParams &p, hipStream_t st);
hipError_t launch_score_mfma(const Geometry &g, const ScoreParams &p, int64_t grid, hipStream_t st);
hipError_t prepare_score_ring(const Geometry &g);
hipError_t launch_score_ring(const Geometry &g, const ScoreParams &p, int64_t grid, hipStream_t st);
hipError_t launch_flag(const float *scores, int64_t n, float thr, uint8_t *flags, hipStream_t st);
// Radix select over the calibration scores' float keys, every pass's digit picked on the device.
// The state lives in device memory: the key prefix chosen so far, the rank still sought among
// the keys that share it, the count of keys above it, and ok = 0 if a pass lost the rank.
struct RadixState {
    uint32_t prefix;
    int32_t ok;
    int64_t rank;
    int64_t n_greater;
};
// rs = {0, 1, rank, 0}; hist (256 bins) cleared.
hipError_t launch_radix_init(RadixState *rs, int64_t rank, unsigned int *hist, hipStream_t st);
// One pass: the histogram of the 8-bit digit at `shift` among keys whose bits above shift+8 equal
// rs->prefix, then (one block) the digit holding rs->rank: rs updated, hist cleared again.
hipError_t launch_calib_hist(const float *scores, const int64_t *woff, const int64_t *cal_off,
                             int n, int64_t n_cal, int shift, RadixState *rs,
                             unsigned int *hist, hipStream_t st);
// Stable compaction of the calibration scores whose key exceeds `key`:
// calib_blocks() blocks; pass 1 counts per block, an exclusive scan gives each block's output
// offset, pass 2 writes the excesses score - t in calibration order.
int64_t calib_blocks(int64_t n_cal);
hipError_t launch_calib_count(const float *scores, const int64_t *woff, const int64_t *cal_off, int n,
                              int64_t n_cal, uint32_t key, int64_t *block_counts, hipStream_t st);
hipError_t launch_calib_compact(const float *scores, const int64_t *woff, const int64_t *cal_off,
                                int n, int64_t n_cal, uint32_t key, double t,
                                const int64_t *block_off, double *y, int64_t cap, hipStream_t st);
hipError_t launch_scan_i64(const int64_t *in, int64_t n, int64_t *out, hipStream_t st);
// Partial likelihood sums at the points xs: pa[i*nsplit + j] = sum xs[i] y/(1 + xs[i] y) and
// pb[i*nsplit + j] = sum log1p(xs[i] y) over the j-th of nsplit contiguous chunks of y (fixed-order
// fp64 sums, device terms within a few ulps of gpd_terms); with pda and pdb (else NULL) also
// their derivatives in x, sum y/(1 + xs[i] y)^2 and sum y/(1 + xs[i] y). gpd_split gives nsplit
// for n excesses and nx points.
int gpd_split(int64_t n, int nx);
hipError_t launch_gpd_sums(const double *y, int64_t n, const double *xs, int nx, int nsplit,
                           double *pa, double *pb, double *pda, double *pdb, hipStream_t st);
// sa[i], sb[i] = the chunk partials of point i added in a fixed order (one wave per point).
hipError_t launch_gpd_reduce(const double *pa, const double *pb, int nx, int nsplit, double *sa, double *sb,
                             hipStream_t st);
// out = {sum y, min y, max y}; work holds 3 * kPeakBlocks doubles of block partials
constexpr int kPeakBlocks = 256;
hipError_t launch_peak_stats(const double *y, int64_t n, double *out, double *work, hipStream_t st);

// Peaks-over-threshold fit (fp64). The likelihood sums over the excesses are supplied by an
// evaluator, so they can run where the excesses live.
struct PotResult {
    double z, t, gamma, sigma;
    int64_t n, n_peaks;
    int method;   // 0: the threshold is t, 1: method of moments, 2: maximum likelihood
};
struct GpdSums {
    virtual ~GpdSums() = default;
    // sa[i] = sum xs[i] y / (1 + xs[i] y), sb[i] = sum log1p(xs[i] y); false on failure
    virtual bool eval(const double *xs, int nx, double *su, double *sv) = 0;
    // the same sums and their derivatives in x: sda[i] = sum y / (1 + xs[i] y)^2,
    // sdb[i] = sum y / (1 + xs[i] y)
    virtual bool eval_d(const double *xs, int nx, double *su, double *sv, double *sda, double *sdb) = 0;
};
// Maximum likelihood (n_peaks >= 10) given the excesses' sum, minimum and maximum.
PotResult pot_mle(double t, int64_t n, int64_t n_peaks, double ysum, double ymin, double ymax,
                  double q, GpdSums &sums, bool *ok);
// Method of moments / degenerate cases (n_peaks < 10) from the excesses on the host.
PotResult pot_small(double t, int64_t n, const double *excess, int64_t n_peaks, double q);

}  // namespace enova
