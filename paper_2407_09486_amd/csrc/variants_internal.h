// Internal declarations of the detector-output variants (chunked dense evaluation of windows).
#pragma once

#include "train_internal.h"

namespace enova {

constexpr int kExtMaxM = 4096;   // metrics whose normalisation (2M floats) a staging block keeps in LDS

// Rows i < rows of V [rows][W*M] = window w0 + i (global window index) normalised per `norm`
// (ENOVA_NORM_REFERENCE: mean/std [n][M]; ENOVA_NORM_WINDOW: the window's own statistics);
// map holds `rows` ints of scratch (each window's stream).
hipError_t launch_ext_stage(const void *x, int dtype, const int64_t *soff, const int64_t *woff, int n, int64_t w0,
                            int rows, int M, int W, int S, int norm, const float *mean, const float *std, int *map,
                            float *V, hipStream_t st);
// ml [rows][2L] = [mu | lv] without biases; adds bml = [bmu | blv] in place and writes the KL
// score of each row (score may be NULL).
hipError_t launch_ext_latent(float *ml, const float *bml, int rows, int L, float *score, hipStream_t st);
// Per row: md = mean(v - m'), md_metric [rows][M] = mean over the steps per metric, recon =
// mean((v - m')^2), with m' = out + bd2 (any output may be NULL).
// The same outputs from the partial sums of a kEpiRowReduce decoder-output product with M
// column groups (M a power of two <= 32): P [rows][slots][M], Q [rows][slots].
hipError_t launch_ext_finish(const float *P, const float *Q, int rows, int slots, int M, int W, float *md,
                             float *md_metric, float *recon, hipStream_t st);
hipError_t launch_ext_reduce(const float *V, const float *out, const float *bd2, int rows, int M, int W, float *md,
                             float *md_metric, float *recon, hipStream_t st);

// ---------------------------------------------------------------------------------------------
// Fused variant pass (k_ext_fused.hip): fp32 detectors with 4, 8 or 16 metrics, at most 128
// hidden units (64 with tanh and 16 metrics), at most 16 latent units and W*M a multiple of 32.
// One block per tile of kExtFusedNb consecutive windows of a stream (tile_off / tile_stream as
// the scoring kernel's), every output written directly.
// ---------------------------------------------------------------------------------------------
constexpr int kExtFusedNb = 256;
struct ExtFusedParams {
    const float *x;
    const int64_t *soff, *woff, *tile_off;
    const int *tile_stream;
    const float *mean, *std;     // reference statistics [n][M] (reference normalisation only)
    const uint4 *w1p;            // the scoring kernel's encoder A fragments
    const float *cst;            // the scoring kernel's block: heads, decoder hidden layer, b1, bd1, u, bh
    const float4 *wd2p;          // [D/32][HB][4][64 lanes]: Wd2[32 ob + l%32][32 hb + crow(4 r4 + e, l/32)], e = 0..3
    const float *bd2;            // [D]
    float *scores, *md, *mdm, *rec;   // any may be NULL
    int norm;                    // ENOVA_NORM_REFERENCE or ENOVA_NORM_WINDOW
    int decode;                  // 0: scores only (the decoder is skipped)
};
struct ExtFusedShape {
    int S, W, Q, CPR, CPRP, KC, spare, D;
    float inv_w, inv_d;
};
bool ext_fused_supported(const Geometry &g);
size_t ext_fused_lds_bytes(const Geometry &g);
hipError_t prepare_ext_fused(const Geometry &g);
hipError_t launch_ext_fused(const Geometry &g, const ExtFusedParams &p, int64_t grid, hipStream_t st);

}  // namespace enova
