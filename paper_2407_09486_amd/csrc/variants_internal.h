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

}  // namespace enova
