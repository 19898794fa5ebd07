// Internal declarations of the streaming path (per-stream rings, newest-window scoring, SPOT).
#pragma once

#include "internal.h"

namespace enova {

// ---------------------------------------------------------------------------------------------
// Streaming detection: n streams advance one step per push; each keeps its last W steps in a
// ring of 2W slots (every step is written twice, at slot c % W and c % W + W, so the newest W
// steps are always contiguous), and its own SPOT threshold.
// ---------------------------------------------------------------------------------------------
struct StreamScoreParams {
    const void *ring;            // [n][2W][M], the detector's dtype
    int n_streams;
    int first_slot;              // slot of the newest window's first step (the same in every stream)
    const float *mean, *std;     // [n][M]
    const uint4 *w1p;            // W1 as 16x16 fragments [stream_w1_steps][Hp/16][64 lanes]
    const float *whp, *wd1p;     // heads [Hp/16][4][2][64] and decoder [Hp/16][4][64] fragments
    const float *b1, *bd1, *u, *bh;
    float sum_bd2;
    float *scores;               // [n]
    float *md;                   // [n] or null
};
// Scoring kernel of the newest windows: kStreamNb windows per block of kStreamWaves waves; wave w
// takes the reduction steps j = w mod 4 (four 16-byte chunks of every window each), one
// iteration per step, with W1 fragments fetched stream_pa iterations ahead and, when the window
// is a contiguous run of whole metric groups (stream_vec), window chunks stream_pb ahead.
constexpr int kStreamNb = 16;
constexpr int kStreamWaves = 4;
constexpr int stream_pa(int nhb) { return nhb >= 16 ? 2 : nhb >= 8 ? 4 : 8; }
constexpr int stream_pb(int dtype) { return dtype == ENOVA_F32 ? 8 : 16; }
inline bool stream_vec(const Geometry &g)
{
    return g.Mp == g.M && g.M % g.epc == 0 && (4 * g.epc) % g.M == 0;
}
// Iterations of every wave: KC / 16 rounded up to a multiple of the window prefetch depth.
inline int stream_iters(const Geometry &g)
{
    const int u = stream_pb(g.dtype);
    return (g.KC / 16 + u - 1) / u * u;
}
// Reduction steps of the packed W1: every iteration's step plus the prefetch's overrun (zeros
// past the window's KC chunks).
inline int stream_w1_steps(const Geometry &g) { return 4 * (stream_iters(g) + stream_pa(g.Hp / 16)); }

// x_step [n][M] becomes step number `step` (0-based) of every stream.
hipError_t launch_stream_append(const Geometry &g, const void *x_step, int n, int64_t step, void *ring,
                                hipStream_t st);
// Lets the streaming scoring kernel of g use the LDS it needs; false if g does not fit.
bool stream_score_supported(const Geometry &g);
hipError_t prepare_stream_score(const Geometry &g);
hipError_t launch_stream_score(const Geometry &g, const StreamScoreParams &p, hipStream_t st);

// Per-stream SPOT state (device arrays of n entries; peaks [n][cap]).
struct SpotState {
    double *t, *z;               // level quantile and threshold (+inf: no calibration)
    int64_t *cnt;                // observations counted (calibration + later non-alarms)
    int *npk;                    // stored peaks
    double *peaks;               // excesses over t, arrival order
    int cap;
    uint8_t *mark;               // 1: z must be refitted
    int *err;                    // set to 1 if a stream's calibration peaks exceed cap
    int *list;                   // [n]: streams that took a new peak in this push (any order)
    int *count;                  // [2]: entries of list, alternating between pushes: a push's update
                                 // counts in count[cur], its refit reads that and clears the other
    int cur;                     // this push's counter (0 or 1)
};
hipError_t launch_spot_init(const float *cal, const int64_t *cal_off, int n, double level,
                            const SpotState &s, hipStream_t st);
hipError_t launch_spot_update(const float *scores, int n, const SpotState &s, uint8_t *flags,
                              hipStream_t st);
// Refits z: every marked stream (all = true), or the streams listed by the last update.
hipError_t launch_spot_fit(int n, double q, const SpotState &s, bool all, hipStream_t st);

}  // namespace enova
