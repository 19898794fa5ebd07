/*
 * Oracle for the ENOVA performance-detection scoring path -- TEST INFRASTRUCTURE.
 *
 * Plain, slow, fp64 loops that follow the detector of Section IV-B step by step.
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
 * load this; the product path never does. It shares no code, header or constant
 * with the HIP library.
 *
 * Steps (Section IV-B, "Performance Detection Module"):
 *   1. windows: window k of a stream covers steps [k*S, k*S+W) (Table II's
 *      observation windows), windows start at step 0, a partial tail is dropped;
 *   2. reference statistics: per stream and metric, mean and population std over
 *      the reference prefix (the first R = floor(ref_frac*T) steps) -- the inputs
 *      are normalised before entering the VAE;
 *   3. v_j = (x[k*S+t][m] - mean_m) / std_m, flattened j = t*M + m;
 *   4. VAE encoder q(z|m): h = act(W1 v + b1), mu = Wmu h + bmu, lv = Wlv h + blv;
 *   5. score = KL(N(mu, diag e^lv) || N(0, I)) = 1/2 sum_l (mu_l^2 + e^lv_l - 1 - lv_l);
 *   6. Mean Difference between m and its reconstruction m' = Wd2 act(Wd1 mu + bd1) + bd2:
 *      md = (1/D) sum_j (v_j - m'_j)  (the decoder is materialised in full here).
 * Thresholding (peaks-over-threshold) is in the Python half of the oracle.
 *
 * For the bf16 workload the normalised value is stored as bfloat16: step 3 is
 * evaluated in fp64, v = (x - mean) / std, and v is then rounded once to the
 * nearest bfloat16 (ties to even). Everything after that stays fp64 here.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ACT_RELU 0
#define ACT_TANH 1

static double act_fn(double a, int kind)
{
    if (kind == ACT_TANH)
        return tanh(a);
    return a < 0.0 ? 0.0 : a;      /* ReLU; a NaN passes through */
}

/*
 * Nearest bfloat16 value of a double, ties to the even significand (one rounding
 * straight from fp64, never through fp32). bfloat16 keeps 8 significant bits and
 * fp32's exponent range: the spacing of representable values at |d| in
 * [2^(e-1), 2^e) is 2^(e-8), and below the smallest normal (2^-126) the spacing is
 * the subnormal step 2^-133. A result beyond the largest finite bfloat16
 * (0x7f7f = (2 - 2^-7) * 2^127) is an infinity of the same sign, as in IEEE
 * round-to-nearest.
 */
double oracle_bf16_round(double d)
{
    if (!isfinite(d) || d == 0.0)
        return d;
    int e;
    frexp(d, &e);                                   /* |d| = f * 2^e, f in [0.5, 1) */
    int qe = e - 8;
    if (qe < -133)
        qe = -133;
    double q = ldexp(1.0, qe);
    double r = nearbyint(d / q) * q;                /* d / q is exact; default mode ties to even */
    const double maxbf = ldexp(255.0, 120);         /* (2 - 2^-7) * 2^127 */
    if (fabs(r) > maxbf)
        return d > 0 ? INFINITY : -INFINITY;
    return r;
}

void oracle_bf16_round_array(const double *in, double *out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_bf16_round(in[i]);
}

/* Reference statistics over x[0..R) of one stream (row-major [T][M]). */
void oracle_ref_stats(const double *x, int64_t R, int M, double *mean, double *std)
{
    for (int m = 0; m < M; ++m) {
        if (R <= 0) {
            mean[m] = 0.0;
            std[m] = 1.0;
            continue;
        }
        double s = 0.0;
        for (int64_t t = 0; t < R; ++t)
            s += x[t * M + m];
        double mu = s / (double)R;
        double ss = 0.0;
        for (int64_t t = 0; t < R; ++t) {
            double d = x[t * M + m] - mu;
            ss += d * d;
        }
        double sd = sqrt(ss / (double)R);
        if (sd <= 1e-6 * fmax(1.0, fabs(mu)))
            sd = 1.0;                                /* metric constant over the reference */
        mean[m] = mu;
        std[m] = sd;
    }
}

typedef struct {
    const double *w1, *b1, *wmu, *bmu, *wlv, *blv, *wd1, *bd1, *wd2, *bd2;
} oracle_weights;

/*
 * One window. Scratch `buf` holds at least 2*D + 2*H + 2*L doubles. If `dbg` is
 * non-NULL it receives v[D], h[H], mu[L], lv[L], hd[H], mrec[D] in that order.
 */
static void score_window(const double *xs, int M, int W, int S, int64_t k, int H, int L, int act,
                         const oracle_weights *wt, const double *mean, const double *std, int bf16,
                         double *buf, double *score, double *md, double *md_scale, double *dbg)
{
    const int D = W * M;
    double *v = buf, *h = v + D, *mu = h + H, *lv = mu + L, *hd = lv + L, *mrec = hd + H;

    /* step 3: normalise */
    for (int t = 0; t < W; ++t) {
        for (int m = 0; m < M; ++m) {
            double val = (xs[(k * S + t) * M + m] - mean[m]) / std[m];
            v[t * M + m] = bf16 ? oracle_bf16_round(val) : val;
        }
    }
    /* step 4: encoder */
    for (int i = 0; i < H; ++i) {
        double a = wt->b1[i];
        for (int j = 0; j < D; ++j)
            a += wt->w1[(int64_t)i * D + j] * v[j];
        h[i] = act_fn(a, act);
    }
    for (int l = 0; l < L; ++l) {
        double a = wt->bmu[l], b = wt->blv[l];
        for (int i = 0; i < H; ++i) {
            a += wt->wmu[l * H + i] * h[i];
            b += wt->wlv[l * H + i] * h[i];
        }
        mu[l] = a;
        lv[l] = b;
    }
    /* step 5: KL of the posterior from the standard-normal prior */
    double kl = 0.0;
    for (int l = 0; l < L; ++l)
        kl += mu[l] * mu[l] + expm1(lv[l]) - lv[l];
    *score = 0.5 * kl;
    /* step 6: decoder mean at z = mu, and the mean difference */
    for (int i = 0; i < H; ++i) {
        double a = wt->bd1[i];
        for (int l = 0; l < L; ++l)
            a += wt->wd1[i * L + l] * mu[l];
        hd[i] = act_fn(a, act);
    }
    double diff = 0.0, mag = 0.0;
    for (int j = 0; j < D; ++j) {
        double r = wt->bd2[j];
        for (int i = 0; i < H; ++i)
            r += wt->wd2[(int64_t)j * H + i] * hd[i];
        mrec[j] = r;
        diff += v[j] - r;
        mag += fabs(v[j]) + fabs(r);
    }
    *md = diff / (double)D;
    if (md_scale)
        *md_scale = mag / (double)D;     /* mean|v| + mean|m'|: the scale md is compared at */
    if (dbg) {
        memcpy(dbg, v, sizeof(double) * D);
        memcpy(dbg + D, h, sizeof(double) * H);
        memcpy(dbg + D + H, mu, sizeof(double) * L);
        memcpy(dbg + D + H + L, lv, sizeof(double) * L);
        memcpy(dbg + D + H + 2 * L, hd, sizeof(double) * H);
        memcpy(dbg + D + 2 * H + 2 * L, mrec, sizeof(double) * D);
    }
}

/* Single window with every intermediate exposed (for the oracle's own pins). */
void oracle_window_debug(const double *xs, int M, int W, int S, int64_t k, int H, int L, int act,
                         const double *w1, const double *b1, const double *wmu, const double *bmu,
                         const double *wlv, const double *blv, const double *wd1, const double *bd1,
                         const double *wd2, const double *bd2, const double *mean, const double *std,
                         int bf16, double *score, double *md, double *dbg)
{
    oracle_weights wt = {w1, b1, wmu, bmu, wlv, blv, wd1, bd1, wd2, bd2};
    const int D = W * M;
    double *buf = (double *)malloc(sizeof(double) * (2 * (size_t)D + 2 * (size_t)H + 2 * (size_t)L));
    score_window(xs, M, W, S, k, H, L, act, &wt, mean, std, bf16, buf, score, md, NULL, dbg);
    free(buf);
}

/*
 * Batch driver over CSR streams.
 *   x            [stream_off[n]][M]
 *   win_off      [n+1] output position of each stream's first window
 *   win_count    [n]   windows to score per stream (<= the stream's window count)
 *   ref_len      [n]   R_s, the reference-prefix length of each stream
 *   ext_mean/std [n][M] or NULL (then computed from the reference prefix)
 *   out_mean/std [n][M] receive the statistics used (may be NULL)
 * Returns the number of threads used.
 */
int oracle_score_batch(const double *x, const int64_t *stream_off, int n, int M, int W, int S,
                       int H, int L, int act, const int64_t *ref_len,
                       const double *w1, const double *b1, const double *wmu, const double *bmu,
                       const double *wlv, const double *blv, const double *wd1, const double *bd1,
                       const double *wd2, const double *bd2, int bf16,
                       const double *ext_mean, const double *ext_std,
                       const int64_t *win_off, const int64_t *win_count,
                       double *score, double *md, double *md_scale, double *out_mean, double *out_std,
                       int nthreads)
{
    oracle_weights wt = {w1, b1, wmu, bmu, wlv, blv, wd1, bd1, wd2, bd2};
    const int D = W * M;
    int used = 1;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#endif
    double *mean = (double *)malloc(sizeof(double) * ((size_t)n * M + 1));
    double *std = (double *)malloc(sizeof(double) * ((size_t)n * M + 1));

#pragma omp parallel for schedule(dynamic, 1)
    for (int s = 0; s < n; ++s) {
        if (ext_mean) {
            for (int m = 0; m < M; ++m) {
                mean[(size_t)s * M + m] = ext_mean[(size_t)s * M + m];
                std[(size_t)s * M + m] = ext_std[(size_t)s * M + m];
            }
        } else {
            oracle_ref_stats(x + stream_off[s] * M, ref_len[s], M, mean + (size_t)s * M,
                             std + (size_t)s * M);
        }
    }

    /* flatten the (stream, window) work list */
    int64_t total = 0;
    for (int s = 0; s < n; ++s)
        total += win_count[s];
    int64_t *first = (int64_t *)malloc(sizeof(int64_t) * (n + 1));
    first[0] = 0;
    for (int s = 0; s < n; ++s)
        first[s + 1] = first[s] + win_count[s];

#pragma omp parallel
    {
#ifdef _OPENMP
#pragma omp single
        used = omp_get_num_threads();
#endif
        double *buf = (double *)malloc(sizeof(double) * (2 * (size_t)D + 2 * (size_t)H + 2 * (size_t)L));
#pragma omp for schedule(dynamic, 64)
        for (int64_t g = 0; g < total; ++g) {
            int lo = 0, hi = n - 1;          /* stream s with first[s] <= g < first[s+1] */
            while (lo < hi) {
                int mid = (lo + hi + 1) / 2;
                if (first[mid] <= g)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            int s = lo;
            int64_t k = g - first[s];
            double sc, dm, ms;
            score_window(x + stream_off[s] * M, M, W, S, k, H, L, act, &wt, mean + (size_t)s * M,
                         std + (size_t)s * M, bf16, buf, &sc, &dm, &ms, NULL);
            score[win_off[s] + k] = sc;
            md[win_off[s] + k] = dm;
            if (md_scale)
                md_scale[win_off[s] + k] = ms;
        }
        free(buf);
    }
    if (out_mean)
        memcpy(out_mean, mean, sizeof(double) * (size_t)n * M);
    if (out_std)
        memcpy(out_std, std, sizeof(double) * (size_t)n * M);
    free(first);
    free(mean);
    free(std);
    return used;
}

/*
 * Sampled windows: pair i is window pk[i] of stream ps[i]. Reference statistics are computed
 * for every stream that appears (or taken from ext_mean/ext_std [n][M]).
 */
int oracle_score_pairs(const double *x, const int64_t *stream_off, int n, int M, int W, int S,
                       int H, int L, int act, const int64_t *ref_len,
                       const double *w1, const double *b1, const double *wmu, const double *bmu,
                       const double *wlv, const double *blv, const double *wd1, const double *bd1,
                       const double *wd2, const double *bd2, int bf16,
                       const double *ext_mean, const double *ext_std,
                       const int32_t *ps, const int64_t *pk, int64_t npairs,
                       double *score, double *md, double *md_scale, int nthreads)
{
    oracle_weights wt = {w1, b1, wmu, bmu, wlv, blv, wd1, bd1, wd2, bd2};
    const int D = W * M;
    int used = 1;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#endif
    double *mean = (double *)malloc(sizeof(double) * ((size_t)n * M + 1));
    double *std = (double *)malloc(sizeof(double) * ((size_t)n * M + 1));
    char *need = (char *)calloc((size_t)n + 1, 1);
    for (int64_t i = 0; i < npairs; ++i)
        need[ps[i]] = 1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int s = 0; s < n; ++s) {
        if (!need[s])
            continue;
        if (ext_mean) {
            for (int m = 0; m < M; ++m) {
                mean[(size_t)s * M + m] = ext_mean[(size_t)s * M + m];
                std[(size_t)s * M + m] = ext_std[(size_t)s * M + m];
            }
        } else {
            oracle_ref_stats(x + stream_off[s] * M, ref_len[s], M, mean + (size_t)s * M,
                             std + (size_t)s * M);
        }
    }
#pragma omp parallel
    {
#ifdef _OPENMP
#pragma omp single
        used = omp_get_num_threads();
#endif
        double *buf = (double *)malloc(sizeof(double) * (2 * (size_t)D + 2 * (size_t)H + 2 * (size_t)L));
#pragma omp for schedule(dynamic, 16)
        for (int64_t i = 0; i < npairs; ++i) {
            const int s = ps[i];
            double ms;
            score_window(x + stream_off[s] * M, M, W, S, pk[i], H, L, act, &wt, mean + (size_t)s * M,
                         std + (size_t)s * M, bf16, buf, &score[i], &md[i], &ms, NULL);
            if (md_scale)
                md_scale[i] = ms;
        }
        free(buf);
    }
    free(need);
    free(mean);
    free(std);
    return used;
}
