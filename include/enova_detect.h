/*
 * enova_detect.h -- C ABI of the MI355X (gfx950) batched sliding-window anomaly scorer.
 *
 * What it computes is the performance-detection module of ENOVA (arXiv 2407.09486,
 * Section IV-B, Fig. 3): monitoring metrics of many LLM-service instances (Table II:
 * arrivals, running/pending requests, execution time, GPU memory and GPU utilisation,
 * each observed over a window of consecutive steps) are normalised, encoded by a VAE
 * whose posterior q(z|m) is a diagonal Gaussian, scored by the KL-divergence of that
 * posterior from the standard-normal prior, thresholded by peaks-over-threshold, and
 * given a scale-up/scale-down direction by the Mean Difference between the input
 * window and its reconstruction.
 *
 * Conventions for every entry point:
 *   - every function returns an enova_status; none aborts, throws or exits;
 *   - arguments are validated on the host before any launch; a failing call writes no output;
 *   - "device" pointers are HIP device (or managed) memory of the device the detector was
 *     created on; "host" pointers are ordinary host memory;
 *   - the caller owns every buffer it passes; the library owns the detector handle, the
 *     device copies of the weights and its internal workspace;
 *   - calls on one detector must not overlap (the workspace is reused); distinct detectors
 *     are independent;
 *   - enova_last_error() returns a description of the last failure on the calling thread.
 *
 * Data layout:
 *   x: row-major [total_steps][M]: step-major, the M metrics of a step contiguous; the
 *      streams are concatenated, stream s occupying rows [stream_offsets[s], stream_offsets[s+1]).
 *   Window k of stream s covers rows [k*S, k*S + W) of that stream (k = 0, 1, ... while
 *   k*S + W <= T_s; a partial tail is dropped); its flattened input index is j = t*M + m.
 *   Window outputs are CSR too: window k of stream s is element window_offsets[s] + k.
 */
#ifndef ENOVA_DETECT_H
#define ENOVA_DETECT_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct enova_detector_s *enova_detector;   /* opaque; owned by the library */

typedef enum {
    ENOVA_OK = 0,
    ENOVA_EINVAL = 1,        /* a null required pointer, a size out of range, a bad enum */
    ENOVA_ESHAPE = 2,        /* shapes are valid but the request has no data to act on */
    ENOVA_ENOMEM = 3,        /* device or host allocation failed */
    ENOVA_EHIP = 4,          /* a HIP runtime call or a kernel launch failed */
    ENOVA_EUNSUPPORTED = 5,  /* a valid request this library does not implement */
    ENOVA_ENUMERIC = 6       /* non-finite values where finite ones are required */
} enova_status;

typedef enum { ENOVA_F32 = 0, ENOVA_BF16 = 1 } enova_dtype;     /* storage / MFMA type of x and W1 */
typedef enum { ENOVA_RELU = 0, ENOVA_TANH = 1 } enova_act;       /* hidden activation of encoder and decoder */
typedef enum {
    ENOVA_KERNEL_AUTO = 0,   /* the matrix-core kernel when the shape allows it, else the vector kernel */
    ENOVA_KERNEL_VALU = 1,   /* always the general vector-ALU kernel */
    ENOVA_KERNEL_MFMA = 2    /* always the matrix-core kernel; EUNSUPPORTED if the shape does not fit */
} enova_kernel;

/*
 * Detector shape (Section IV-B: one hidden layer of width H, a diagonal-Gaussian latent
 * of width L with mean and log-variance heads, prior N(0, I); the decoder's mean head
 * reconstructs the window).
 *   metrics M >= 1, window W >= 1, stride S >= 1, hidden H >= 1, latent 1 <= L <= 64,
 *   W*M <= 65536, ref_frac in (0, 1]: the reference prefix of a stream of T steps is its
 *   first floor((double)ref_frac * T) steps.
 */
typedef struct {
    int32_t metrics, window, stride, hidden, latent;
    int32_t dtype;           /* enova_dtype */
    int32_t act;             /* enova_act */
    int32_t kernel;          /* enova_kernel */
    float ref_frac;          /* default 0.5 */
} enova_detect_config;

/*
 * Detector weights: HOST pointers, row-major [out][in] (as torch.nn.Linear stores them).
 * They are copied (and repacked for the kernels) by enova_detect_init; the caller may free
 * them afterwards. D = W*M; the flattened input index is j = t*M + m.
 */
typedef struct {
    const void *w1;   const float *b1;    /* [H][D] (float, or bf16 bit patterns for ENOVA_BF16), [H] */
    const float *wmu; const float *bmu;   /* [L][H], [L]   posterior mean head        */
    const float *wlv; const float *blv;   /* [L][H], [L]   posterior log-variance head */
    const float *wd1; const float *bd1;   /* [H][L], [H]   decoder hidden layer        */
    const float *wd2; const float *bd2;   /* [D][H], [D]   decoder mean head (only its column sums are kept) */
} enova_detect_weights;

/* Create a detector on the current HIP device. Errors: EINVAL (config or weights), ENOMEM, EHIP. */
enova_status enova_detect_init(const enova_detect_config *config, const enova_detect_weights *weights,
                               enova_detector *out);

/* Free a detector and all its device memory (synchronises the device). NULL is a no-op. */
enova_status enova_detect_destroy(enova_detector det);

/*
 * Host helper (window enumeration of Table II's observation windows).
 *   stream_offsets_host [n_streams+1]: [0] = 0, non-decreasing (EINVAL otherwise).
 *   window_offsets_host [n_streams+1] receives the exclusive scan of the per-stream window
 *   counts n_s = T_s >= W ? (T_s - W) / S + 1 : 0; its last entry is the total window count N.
 */
enova_status enova_detect_window_offsets(enova_detector det, const int64_t *stream_offsets_host,
                                         int32_t n_streams, int64_t *window_offsets_host);

/*
 * Reference statistics (Section IV-B: metrics are normalised before entering the VAE).
 * Per stream and metric, mean and population standard deviation over the reference
 * prefix (accumulated in fp64, stored as fp32). A prefix of zero steps gives mean 0 and
 * std 1; a std <= 1e-6 * max(1, |mean|) (a metric constant over the reference) becomes 1.
 *   x              device, [stream_offsets[n]][M], the detector's dtype
 *   stream_offsets device [n+1]
 *   out_mean, out_std device [n][M] float
 * Asynchronous on `stream`.
 */
enova_status enova_detect_ref_stats(enova_detector det, const void *x, const int64_t *stream_offsets,
                                    int32_t n_streams, float *out_mean, float *out_std,
                                    hipStream_t stream);

/*
 * Score every window (Section IV-B: KL-divergence of q(z|m) from p(z); Mean Difference
 * between m and its reconstruction m' for the direction; anomaly iff the KL exceeds the
 * threshold).
 *   x              device [stream_offsets[n]][M], the detector's dtype (float or bf16 bits)
 *   stream_offsets device [n+1]: [0] = 0, non-decreasing (precondition, not checked on device)
 *   window_offsets device [n+1]: as produced by enova_detect_window_offsets (precondition)
 *   n_streams      >= 0;   n_windows = window_offsets[n_streams] (precondition)
 *   ref_mean, ref_std  device [n][M] float, or both NULL: then computed as by
 *                  enova_detect_ref_stats into the detector's workspace
 *   threshold      flags are written as score > threshold; NaN: out_flags is not written
 *   out_scores     device [n_windows] float: 1/2 sum_l (mu_l^2 + e^lv_l - 1 - lv_l)
 *   out_md         device [n_windows] float or NULL: mean(v) - mean(m'), in normalised units;
 *                  positive means the window sits above its reconstruction (scale up)
 *   out_flags      device [n_windows] uint8 or NULL
 * Inputs are expected finite; a NaN input propagates to that window's score and md, and its
 * flag is 0. Nothing outside [0, n_windows) is written. Asynchronous on `stream`.
 * Errors: EINVAL, EUNSUPPORTED (ENOVA_KERNEL_MFMA with an unsupported shape), ENOMEM, EHIP.
 */
enova_status enova_detect_score(enova_detector det, const void *x, const int64_t *stream_offsets,
                                const int64_t *window_offsets, int32_t n_streams, int64_t n_windows,
                                const float *ref_mean, const float *ref_std, float threshold,
                                float *out_scores, float *out_md, uint8_t *out_flags,
                                hipStream_t stream);

/*
 * enova_detect_score without any allocation, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, hosts that forbid hipMalloc). Arguments,
 * results and errors are those of enova_detect_score, with the same kernels; it calls no
 * hipMalloc, hipFree or allocating routine, and records no timing events (kernel timing reports
 * nothing for it). Its workspace -- the reference statistics when ref_mean/ref_std are NULL
 * (2 * n_streams * M floats), and for the matrix-core kernel the tile offsets
 * ((n_streams + 1) int64) and block-to-stream map ((n_windows + Nb - 1) / Nb + n_streams ints,
 * Nb = windows per tile: 128-512 by shape), each rounded up to 256 bytes -- lives in a fixed
 * 16 MiB device array that the library holds on every GPU it runs on until the process ends,
 * shared by all detectors on that GPU. A call that needs more returns ENOVA_ESHAPE before any
 * launch. Every part of that workspace is fully rewritten by each call before it is read, so no
 * clearing is needed between calls; calls that overlap on one GPU (on different streams, or from
 * several threads) race on the array and must be serialised by the caller.
 */
enova_status enova_detect_score_noalloc(enova_detector det, const void *x, const int64_t *stream_offsets,
                                        const int64_t *window_offsets, int32_t n_streams, int64_t n_windows,
                                        const float *ref_mean, const float *ref_std, float threshold,
                                        float *out_scores, float *out_md, uint8_t *out_flags,
                                        hipStream_t stream);

/*
 * Peaks-over-threshold threshold (Section IV-B, citing Siffer et al. 2017), static and global:
 * the calibration set is the scores of the windows lying wholly inside each stream's reference
 * prefix (k*S + W <= floor(ref_frac*T_s)); t is its order statistic at ceil(level*n) - 1
 * (ascending, 0-based); the excesses Y = {c - t : c > t} are fitted by a generalised Pareto
 * distribution (N_t >= 10: maximum likelihood by Grimshaw's reduction in fp64 -- the roots of
 * its one-variable equation are bracketed on a 512-point grid of each admissible interval and
 * refined by Newton steps kept inside each bracket, with the likelihood sums over the excesses
 * reduced on the device in a fixed order; 2 <= N_t < 10: method of moments with the unbiased
 * sample variance;
 * N_t <= 1: the threshold is t) and
 *   z_q = t + sigma/gamma * ((q n / N_t)^(-gamma) - 1)   (z_q = t - sigma ln(q n / N_t) if gamma = 0).
 *   scores         device [n_windows] float (as written by enova_detect_score)
 *   level in (0,1), q in (0,1)  (defaults 0.98 and 1e-3)
 *   out_threshold  HOST float
 *   out_info       HOST double[6] or NULL: t, n, N_t, gamma, sigma, method (0 t, 1 moments, 2 MLE)
 *   out_flags      device [n_windows] uint8 or NULL: score > z_q for every window
 * Synchronises `stream` (it returns a host value). ESHAPE if no window is a calibration window.
 */
enova_status enova_detect_threshold(enova_detector det, const float *scores,
                                    const int64_t *stream_offsets, const int64_t *window_offsets,
                                    int32_t n_streams, int64_t n_windows, double level, double q,
                                    float *out_threshold, double *out_info, uint8_t *out_flags,
                                    hipStream_t stream);

/*
 * Streaming detection. Section V runs the detector inside a stream-computing job, and the
 * peaks-over-threshold method Section IV-B cites (Siffer et al. 2017) is a streaming one (SPOT).
 * A streaming set holds n streams that advance together: every enova_stream_push appends one
 * step of M metrics to each stream; once every stream has seen c = W + k*S steps (k >= 0), the
 * push scores each stream's newest window (its last W steps, normalised with the reference
 * statistics given at creation) exactly as enova_detect_score scores that window, and updates
 * each stream's own threshold by SPOT:
 *   start   t_s = the order statistic at ceil(level*n_s) - 1 of the stream's n_s calibration
 *           scores, its peaks {c - t_s : c > t_s} in calibration order, and z_s fitted as by
 *           enova_detect_threshold over that stream alone (no calibration score: t_s = z_s =
 *           +inf and the stream never changes, so it never flags);
 *   s > z_s          flag 1; the stream's model is left as it is (an alarm is not learnt);
 *   t_s < s <= z_s   flag 0; s - t_s joins the peaks, n_s += 1, z_s is refitted on all peaks;
 *   s <= t_s         flag 0; n_s += 1 (z_s moves at the next peak);   NaN: flag 0, no change.
 * Once a stream stores peak_cap peaks its model is frozen (its scores are still compared).
 * The refits run on the device (one block per stream with a new peak) with the batch fit's
 * method; a push is asynchronous on `stream`. Calls on one streaming set must not overlap, and
 * the detector must outlive its streaming sets; the set uses the detector's matrix-core
 * weights (EUNSUPPORTED for a shape the matrix-core kernel does not take).
 */
typedef struct enova_stream_s *enova_stream;   /* opaque; owned by the library */

/*
 *   n_streams        >= 1
 *   ref_mean, ref_std  device [n][M] float (e.g. from enova_detect_ref_stats); copied
 *   calib_scores     device float: stream s's calibration scores at
 *                    [calib_offsets[s], calib_offsets[s+1]), e.g. its windows inside its
 *                    reference prefix as scored by enova_detect_score
 *   calib_offsets    HOST [n+1] int64, [0] = 0, non-decreasing
 *   level, q         in (0, 1), as for enova_detect_threshold
 *   peak_cap         >= 1: peaks stored per stream (device memory n * peak_cap * 8 bytes)
 * Synchronises `stream`. Errors: EINVAL (arguments; a stream whose calibration peaks exceed
 * peak_cap), ENUMERIC (a non-finite calibration score), EUNSUPPORTED, ENOMEM, EHIP.
 */
enova_status enova_stream_create(enova_detector det, int32_t n_streams, const float *ref_mean,
                                 const float *ref_std, const float *calib_scores,
                                 const int64_t *calib_offsets, double level, double q,
                                 int32_t peak_cap, enova_stream *out, hipStream_t stream);

/*
 *   x_step       device [n][M], the detector's dtype: the next step of every stream
 *   out_scores   device [n] float or NULL: the newest window's score when a window was due
 *   out_md       device [n] float or NULL: its md
 *   out_flags    device [n] uint8 or NULL: 1 where the score exceeds the stream's threshold
 *                (as it stood before this score)
 *   out_due      HOST int32 or NULL: 1 if this push scored windows, else 0 (then nothing is
 *                written to the device outputs)
 * Asynchronous on `stream`. The threshold update and the refit of the streams that took a new
 * peak run on a stream of the set's own (default priority), ordered by events: the update after
 * this push's scores, later work on `stream` after the update (its flags are then written), the
 * next push's update and any enova_stream_state after the refit. The refit thus overlaps the
 * next push's append and scoring, and every push and state read sees the thresholds in push
 * order.
 * Errors: EINVAL, EHIP.
 */
enova_status enova_stream_push(enova_stream s, const void *x_step, float *out_scores, float *out_md,
                               uint8_t *out_flags, int32_t *out_due, hipStream_t stream);

/* Per-stream SPOT state into HOST arrays [n] (each may be NULL): t, z, n, stored peaks, after
 * the last push's refit. Synchronises `stream`. */
enova_status enova_stream_state(enova_stream s, double *t, double *z, int64_t *n, int32_t *n_peaks,
                                hipStream_t stream);

/* With the detector's kernel timing enabled (enova_detect_set_timing), a push that scored
 * windows brackets its scoring kernel and its SPOT kernels (update and refit) with HIP events;
 * this waits for the last such push and reports milliseconds (0 if none ran). */
enova_status enova_stream_kernel_times(enova_stream s, double *score_kernel_ms, double *spot_kernels_ms);

/* Free a streaming set (synchronises the device). NULL is a no-op. */
enova_status enova_stream_destroy(enova_stream s);

/*
 * Training (Section IV-B, Eq. (9)): one step of semi-supervised ELBO training of the detector's
 * VAE on a batch of B labelled, normalised windows,
 *   L = 1/B sum_i [ l_i log p(m_i | z_i) - (1 + l_i)/2 beta(k) KL(q(z | m_i) || p(z)) ],
 * l_i = +1 (normal) or -1 (anomalous), with z_i = mu_i + exp(lv_i / 2) eps_i one reparameterised
 * sample (eps given by the caller), a unit-variance Gaussian decoder
 * (log p = -|v - m'|^2 / 2 - D/2 log 2 pi), beta(k) set before the backward pass by a PI
 * controller on the mean KL of the batch's normal windows (e = kl_set - KL, P = kp / (1 + e^e),
 * I <- I - ki e, beta = clamp(P + I + beta_min, beta_min, beta_max), I starts at 0), and an Adam
 * step (lr, b1, b2, eps; step count k from 1) on J = -L. As printed, L has no upper bound in the
 * anomalous windows' term -log p (training on anomalies diverges); a finite anomaly_margin m
 * caps that term at min(e_i, m) + D/2 log 2 pi, e_i = |v_i - m'_i|^2 / 2, so an anomalous window
 * is pushed away only until its reconstruction error reaches m. Everything runs on the device in fp32
 * (matrix-core GEMMs with fixed-order reductions, so a step is deterministic); the parameters,
 * the Adam moments and the controller state live in the trainer.
 */
typedef struct enova_trainer_s *enova_trainer;   /* opaque; owned by the library */

typedef struct {
    int32_t inputs;          /* D >= 1 (W * M of the detector) */
    int32_t hidden, latent;  /* H >= 1, L >= 1 */
    int32_t act;             /* enova_act */
    float lr, adam_b1, adam_b2, adam_eps;            /* e.g. 1e-3, 0.9, 0.999, 1e-8 */
    float kl_set, kp, ki, beta_min, beta_max;        /* e.g. 3, 0.01, 1e-4, 0, 1 */
    float anomaly_margin;    /* > 0; +INFINITY: Eq. (9) as printed (see below) */
} enova_train_config;

/* Parameters or gradients in the layout of enova_detect_weights (w1 always fp32 here). */
typedef struct {
    float *w1, *b1, *wmu, *bmu, *wlv, *blv, *wd1, *bd1, *wd2, *bd2;
} enova_train_params;

/* Create a trainer on the current device from initial HOST weights (w1 fp32). Errors: EINVAL,
 * ENOMEM, EHIP. */
enova_status enova_train_init(const enova_train_config *config, const enova_detect_weights *init,
                              enova_trainer *out);

/*
 *   V         device [B][D] float: the normalised windows (flattened j = t*M + m)
 *   labels    device [B] float: +1 or -1
 *   eps       device [B][L] float: the reparameterisation noise
 *   out_info  device [4] float or NULL: J, mean log p, mean KL of the normal windows, beta(k)
 * Asynchronous on `stream`. The step's launches are captured once into a HIP graph (on a stream
 * of the trainer's own) and the graph is replayed while V, labels, eps, out_info and the batch
 * size stay the same (the contents may change between steps); any other arguments capture it
 * again, which first waits for the device. Steps taken with timing on, or with graph replay
 * off, launch their kernels one by one on `stream`; a caller that captures the step into a
 * graph of its own turns replay off. Errors: EINVAL, ENOMEM, EHIP.
 */
enova_status enova_train_step(enova_trainer t, const float *V, const float *labels, const float *eps,
                              int32_t batch, float *out_info, hipStream_t stream);

/* Graph replay of the step (see enova_train_step): on (non-zero, the default) or off. Turning it
 * off frees the captured graph (waiting for the device). Errors: EINVAL. */
enova_status enova_train_set_graph(enova_trainer t, int32_t enable);

/* Copy the current parameters, or the last step's gradients of J, into HOST arrays (each may be
 * NULL). Synchronises `stream`. */
enova_status enova_train_params_get(enova_trainer t, const enova_train_params *out, hipStream_t stream);
enova_status enova_train_grads_get(enova_trainer t, const enova_train_params *out, hipStream_t stream);

/*
 * Timing: when enabled, every following step brackets the kernel of each of its matrix products
 * (not the pass that adds the partial results of a split product) and the whole step with HIP
 * events on its stream; enova_train_kernel_times waits for the last step's events and reports
 * the summed milliseconds of those kernels and of the whole step (0 when the last step was not
 * timed).
 */
enova_status enova_train_set_timing(enova_trainer t, int32_t enable);
enova_status enova_train_kernel_times(enova_trainer t, double *gemm_ms, double *step_ms);

/* Free a trainer (synchronises the device). NULL is a no-op. */
enova_status enova_train_destroy(enova_trainer t);

/*
 * Detector-output variants (Section IV-B). Every window is normalised against its stream's
 * reference statistics (ENOVA_NORM_REFERENCE, as enova_detect_score) or against itself
 * (ENOVA_NORM_WINDOW: per metric the window's own mean and
 * population std, a std <= 1e-6 max(1, |mean|) counting as 1 -- the literal reading of
 * per-window normalisation); then the encoder, the KL score, and the decoder's full output
 * m' = Wd2 act(Wd1 mu + bd1) + bd2 at z = mu. Per window: out_scores (the KL score),
 * out_md = mean_j (v_j - m'_j), out_md_metric [N][M] = mean over the W steps of (v - m') per
 * metric, out_recon_err = mean_j (v_j - m'_j)^2 (device outputs; any may be NULL; with the last
 * three NULL the decoder is not evaluated). ref_mean /
 * ref_std as in enova_detect_score (NULL: computed; ignored for ENOVA_NORM_WINDOW). M <= 4096.
 * enova_detect_ext_mode tells whether a detector's windows take one fused launch or are
 * evaluated in chunks.
 * The products run in fp32 on the matrix cores (x and W1 of a bf16 detector are bf16 values;
 * v is rounded to bf16 as in enova_detect_score). Asynchronous. Errors: EINVAL, EUNSUPPORTED,
 * ENOMEM, EHIP.
 */
typedef enum { ENOVA_NORM_REFERENCE = 0, ENOVA_NORM_WINDOW = 1 } enova_norm;

enova_status enova_detect_score_ext(enova_detector det, const void *x, const int64_t *stream_offsets,
                                    const int64_t *window_offsets, int32_t n_streams, int64_t n_windows,
                                    const float *ref_mean, const float *ref_std, int32_t norm, float *out_scores,
                                    float *out_md, float *out_md_metric, float *out_recon_err, hipStream_t stream);

/* With timing enabled (enova_detect_set_timing), the last enova_detect_score_ext call's duration
 * from its first to its last kernel, milliseconds. */
enova_status enova_detect_ext_time(enova_detector det, double *ms);

/* How enova_detect_score_ext evaluates this detector's windows (fixed at init): *fused = 1 for
 * one launch per call that stages each tile's raw steps once and keeps every window's v, hidden
 * layers and decoder output on chip (fp32 detectors of 4, 8 or 16 metrics, at most 128 hidden
 * units -- 64 with tanh and 16 metrics --, at most 16 latent units, W*M a multiple of 32, and a
 * tile that fits half a compute unit's LDS); 0 for the chunked evaluation of normalised windows
 * in device memory. Errors: EINVAL. */
enova_status enova_detect_ext_mode(enova_detector det, int32_t *fused);

/*
 * Configuration scans (Section IV-A, Eqs. (4)-(6), Table II) over the same monitoring series.
 * Whether the finished-request rate n^f still depends on the number of running requests n^r is
 * decided per window by an ordinary-least-squares fit n^f = a + b n^r (the relation n^f = f(n^r) of Eq. (5)) and a two-sided t-test of
 * the slope at level alpha (t = b / sqrt(RSS / ((W - 2) Sxx)), significant iff
 * |t| > t_{1-alpha/2, W-2}; a window with constant n^r has b = 0, a = mean n^f, t = 0); the
 * GPU memory relation m^u = g0 + g1 n^r is fitted by OLS on the same window. Per stream, the last
 * window then gives n_limit and t^r_limit as quantiles of a Gaussian kernel density estimate
 * (Silverman's bandwidth 0.9 min(sd, IQR/1.34) W^(-1/5), sd if IQR = 0, a point mass if the window
 * is constant) of n^f and of t^r: at level q_extreme when the relation is significant (n^f has not
 * reached its limit, so the limit lies in the upper tail), at 0.5 otherwise (n^f sits at its
 * limit); max_num_seqs = n_limit t^r_limit (Eq. (4)) and gpu_memory = g0 + g1 max_num_seqs
 * (Eq. (6)). Windows are the detector's: W steps, stride S, from step 0 of each stream. All
 * statistics are computed in fp64.
 */
typedef struct enova_config_s *enova_config;   /* opaque; owned by the library */

typedef struct {
    int32_t metrics, window, stride;   /* M >= 1; 3 <= W <= 4096; S >= 1 */
    int32_t dtype;                     /* enova_dtype of x */
    int32_t col_finished, col_running, col_exec_time, col_mem_util;   /* metric columns of n^f, n^r, t^r, m^u */
    double alpha;                      /* in (0, 1), e.g. 0.05 */
    double q_extreme;                  /* in (0, 1), e.g. 0.99 */
} enova_config_params;

/* Two-sided critical value t_{1-alpha/2, dof} of Student's t (host helper). Errors: EINVAL. */
enova_status enova_config_t_critical(double alpha, int32_t dof, double *out);

/* Create a configuration scanner on the current device. Errors: EINVAL, ENOMEM, EHIP. */
enova_status enova_config_init(const enova_config_params *params, enova_config *out);
enova_status enova_config_destroy(enova_config c);

/* Host helper: the window CSR of the scanner's W and S (as enova_detect_window_offsets). */
enova_status enova_config_window_offsets(enova_config c, const int64_t *stream_offsets_host,
                                         int32_t n_streams, int64_t *window_offsets_host);

/*
 * Every window of every stream (device pointers; outputs [n_windows] float or uint8, any may be
 * NULL): OLS of n^f on n^r (intercept, slope, t statistic, significant), OLS of m^u on n^r
 * (intercept, slope). x: [stream_offsets[n]][M] in the scanner's dtype. Asynchronous.
 * Errors: EINVAL, ENOMEM, EHIP.
 */
enova_status enova_config_scan(enova_config c, const void *x, const int64_t *stream_offsets,
                               const int64_t *window_offsets, int32_t n_streams, int64_t n_windows,
                               float *out_intercept, float *out_slope, float *out_t,
                               uint8_t *out_significant, float *out_mem_intercept, float *out_mem_slope,
                               hipStream_t stream);

/*
 * The configuration read off each stream's last window (device outputs [n_streams], any may be
 * NULL): significant (0/1), n_limit, t^r_limit, max_num_seqs, gpu_memory (NaN and 0 for a stream
 * shorter than W). Asynchronous. Errors: EINVAL, EHIP.
 */
enova_status enova_config_recommend(enova_config c, const void *x, const int64_t *stream_offsets,
                                    int32_t n_streams, uint8_t *out_significant, double *out_n_limit,
                                    double *out_t_limit, double *out_max_num_seqs, double *out_gpu_memory,
                                    hipStream_t stream);

/* Kernel timing of the last enova_config_scan (its scan kernel) when enabled, milliseconds. */
enova_status enova_config_set_timing(enova_config c, int32_t enable);
enova_status enova_config_kernel_time(enova_config c, double *scan_kernel_ms);

/* flags[i] = scores[i] > threshold for i < n_windows (device pointers). Asynchronous. */
enova_status enova_detect_flag(enova_detector det, const float *scores, int64_t n_windows,
                               float threshold, uint8_t *out_flags, hipStream_t stream);

/*
 * Kernel timing: when enabled, enova_detect_score brackets its scoring kernel (and, when it
 * computes them, the reference-statistics kernel) with HIP events on `stream`;
 * enova_detect_kernel_times waits for the last call's events and reports milliseconds
 * (a kernel that did not run reports 0).
 */
enova_status enova_detect_set_timing(enova_detector det, int32_t enable);
enova_status enova_detect_kernel_times(enova_detector det, double *score_kernel_ms,
                                       double *stats_kernel_ms);

/* Which scoring kernel the detector uses: 1 vector-ALU, 2 matrix-core (MFMA). */
enova_status enova_detect_kernel_kind(enova_detector det, int32_t *kind);

const char *enova_status_str(enova_status status);
const char *enova_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ENOVA_DETECT_H */
