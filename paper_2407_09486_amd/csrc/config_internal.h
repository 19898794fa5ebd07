// Internal declarations of the configuration scans (windowed OLS and t-test, KDE limits).
#pragma once

#include "internal.h"

namespace enova {

struct CfgParams {
    int M, W, S, dtype;
    int col_f, col_r, col_t, col_m;
    double alpha, q_extreme;
    double t_crit;   // t_{1-alpha/2, W-2}
};

// Windows per block of the scan and the LDS it stages: NB consecutive windows of one stream need
// (NB - 1) S + W steps of the three columns n^r, n^f, m^u.
int cfg_scan_windows_per_block(const CfgParams &c);
size_t cfg_scan_lds_bytes(const CfgParams &c, int nb);

struct CfgScanOut {
    float *a, *b, *t;
    uint8_t *sig;
    float *g0, *g1;
};

// Blocks follow tile_off / tile_stream (tiles of nb windows per stream, -1: no tile).
hipError_t launch_cfg_scan(const CfgParams &c, int nb, const void *x, const int64_t *soff, const int64_t *woff,
                           const int64_t *tile_off, const int *tile_stream, int64_t grid, const CfgScanOut &o,
                           hipStream_t st);

struct CfgStreamOut {
    uint8_t *sig;
    double *n_limit, *t_limit, *max_num_seqs, *gpu_memory;
};
hipError_t launch_cfg_stream(const CfgParams &c, const void *x, const int64_t *soff, int n, const CfgStreamOut &o,
                             hipStream_t st);

// Student's t: two-sided critical value by bisection on the distribution function (regularised
// incomplete beta function by its continued fraction).
double student_t_critical(double alpha, int dof);

}  // namespace enova
