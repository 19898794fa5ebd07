// Host side of libenova_detect: argument validation, weight repacking, workspace management
// and kernel launches behind the C ABI of include/enova_detect.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "enova_detect.h"
#include "internal.h"
#include "stream_internal.h"
#include "variants_internal.h"

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace enova {

enova_status fail(enova_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

enova_status hip_fail(hipError_t e, const char *what)
{
    return fail(ENOVA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace enova

using namespace enova;

namespace {

float bf16_bits_to_float(uint16_t b)
{
    uint32_t u = static_cast<uint32_t>(b) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// Round to nearest even; a NaN stays a (quiet) NaN.
uint16_t float_to_bf16_bits(float f)
{
    uint32_t u;
    std::memcpy(&u, &f, sizeof(u));
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return static_cast<uint16_t>((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

}  // namespace

struct enova_detector_s {
    Geometry g{};
    int device = 0;
    int kind = 1;                 // 1 vector-ALU, 2 matrix-core
    // weights
    void *w1p = nullptr;          // matrix-core A fragments
    void *ring_w = nullptr;       // ring kernel: W1, heads and decoder fragments (one allocation)
    const uint4 *w1r = nullptr, *whr = nullptr;
    const uint2 *wdr = nullptr;
    void *stream_w = nullptr;     // streaming kernel: W1, heads and decoder fragments (one allocation)
    const uint4 *w1s = nullptr;
    const float *whs = nullptr, *wds = nullptr;
    void *ext_w = nullptr;        // fused variant pass: decoder-output fragments of Wd2
    const float4 *wd2p = nullptr;
    void *w1t = nullptr;          // [D][H] transposed W1
    float *small = nullptr;       // every small weight array, one allocation
    float *b1 = nullptr, *bh = nullptr, *bmu = nullptr, *blv = nullptr, *wmu = nullptr,
          *wlv = nullptr, *wd1 = nullptr, *bd1 = nullptr, *u = nullptr, *whp = nullptr,
          *wd1p = nullptr;
    float sum_bd2 = 0.0f;
    // workspace
    float *stats = nullptr;
    size_t stats_cap = 0;         // floats
    int64_t *tiles = nullptr;
    size_t tiles_cap = 0;         // entries
    int *tile_map = nullptr;      // stream of each matrix-core block
    size_t tile_map_cap = 0;      // entries
    int64_t *cal = nullptr;
    size_t cal_cap = 0;
    unsigned int *hist = nullptr; // 256 radix bins, then the radix state (RadixState at bin 256)
    double *peaks = nullptr;      // excesses over the level quantile, calibration order
    size_t peaks_cap = 0;
    int64_t *blk = nullptr;       // per-block peak counts, then their exclusive scan
    size_t blk_cap = 0;
    double *gx = nullptr;         // evaluation points of the GPD likelihood sums, then the sums
    size_t gx_cap = 0;
    double *gpin = nullptr;       // pinned host staging of those points and sums
    size_t gpin_cap = 0;
    // this device's fixed scratch (kScratchBytes, shared by every detector on the device), the
    // only workspace of enova_detect_score_noalloc
    void *scratch = nullptr;
    // dense fp32 weights of the output variants: W1 [H][D], [Wmu; Wlv] [2L][H], [bmu | blv] [2L],
    // Wd1 [H][L], Wd2 [D][H], bd2 [D] (one allocation)
    float *dense = nullptr;
    float *d_w1 = nullptr, *d_wml = nullptr, *d_bml = nullptr, *d_wd1 = nullptr, *d_wd2 = nullptr,
          *d_bd2 = nullptr;
    // workspace of the output variants (one chunk of windows; the fused pass's tile scan and map)
    float *ext_ws = nullptr;
    size_t ext_ws_cap = 0;        // floats
    // timing
    bool timing = false;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    hipEvent_t ext_ev[2] = {nullptr, nullptr};
    bool ran_stats = false, ran_score = false, ran_ext = false;
};

namespace enova {

bool plan_geometry(const enova_detect_config &cfg, Geometry *g)
{
    g->M = cfg.metrics;
    g->W = cfg.window;
    g->S = cfg.stride;
    g->H = cfg.hidden;
    g->L = cfg.latent;
    g->D = cfg.window * cfg.metrics;
    g->dtype = cfg.dtype;
    g->act = cfg.act;
    g->ref_frac = cfg.ref_frac;
    g->epc = cfg.dtype == ENOVA_F32 ? 4 : 8;
    int mp = g->M;
    while ((static_cast<int64_t>(g->S) * mp) % g->epc)
        ++mp;
    g->Mp = mp;
    g->Q = (g->W + g->S - 1) / g->S;
    const int64_t cpr = static_cast<int64_t>(g->S) * g->Mp / g->epc;
    g->CPR = static_cast<int>(cpr);
    g->CPRP = (g->CPR % 2 == 0) ? g->CPR + 1 : g->CPR;
    int64_t kc = static_cast<int64_t>(g->Q) * g->CPR;
    kc = (kc + 2 * kPrefetchSteps - 1) / (2 * kPrefetchSteps) * (2 * kPrefetchSteps);
    g->KC = static_cast<int>(kc);
    // the furthest chunk a window fragment prefetch reads: kPrefetchRows steps past the last
    const int64_t kmax = kc + 2 * kPrefetchRows - 1;
    g->spare = static_cast<int>(kmax / g->CPR - g->Q + 2);
    int hb = 1;
    while (hb < 8 && 32 * hb < g->H)
        hb *= 2;
    g->HB = hb;
    g->Hp = 32 * hb;
    mfma_layout(g->dtype, hb, &g->HBW, &g->NBW, &g->WH, &g->NW);
    g->Nb = (g->NW / g->WH) * g->NBW * 32;
    // epilogue weights (heads, decoder hidden layer, b1, bd1, u, head biases), the segment, its
    // row sums and the stream statistics
    const size_t n_const = static_cast<size_t>(hb) * (16 * 64 + 8 * 64) + 3 * static_cast<size_t>(g->Hp) + 32;
    // with several waves along the hidden rows, the segment's space later holds the exchange of
    // head and decoder partial sums
    const size_t rows = static_cast<size_t>(g->Nb + g->Q - 1 + g->spare);
    const size_t seg_bytes = rows * g->CPRP * 16;
    const size_t xchg_bytes = g->WH > 1 ? static_cast<size_t>(g->NW) * std::min(g->NBW, 2) * 17 * 64 * sizeof(float) : 0;
    // the split bf16 layout keeps its epilogue weights in L2 to leave LDS to a 256-window tile
    g->cl = g->WH == 1;
    // (without the copied block, b1, bd1, u and the head biases still get LDS of their own)
    const size_t n_small = 3 * static_cast<size_t>(g->Hp) + 32;
    g->lds_bytes = (g->cl ? n_const : n_small) * sizeof(float) + std::max(seg_bytes, xchg_bytes) +
                   rows * 2 * sizeof(float) + 3 * sizeof(float) * static_cast<size_t>(g->S) * g->Mp;
    g->mfma_ok = g->H <= 256 && g->L <= 16 && cpr < (1 << 20) && kc < (1 << 24) &&
                 g->lds_bytes <= kLdsLimit;
    // bf16 with 193..256 hidden units: the ring kernel when a block fits half a compute unit's LDS
    // (a ring slot is one super-row of at most 64 chunks, i.e. one chunk per lane of a wave)
    g->ring = false;
    g->RP = g->RR = g->ring_floats = 0;
    g->ring_lds = 0;
    if (g->mfma_ok && g->dtype == ENOVA_BF16 && g->H > 192 && g->H <= kRingHidden && g->L <= 16) {
        const int P = (g->CPR + 15) / 16 * 16;   // whole groups of four 4-chunk reduction steps
        const int R = (kRingNb + 2 + 7) / 8 * 8;
        const int64_t ring_f = std::max<int64_t>(static_cast<int64_t>(R) * P * 4,
                                                 static_cast<int64_t>(kRingWaves) * 2 * (kRingNb / 16) * 4 * 64);
        if (P <= 64) {
            const size_t lds = ring_lds_bytes(P, g->Q, static_cast<int>(ring_f));
            if (lds <= kLdsLimit / 2) {
                g->ring = true;
                g->RP = P;
                g->RR = R;
                g->ring_floats = static_cast<int>(ring_f);
                g->ring_lds = lds;
                g->Nb = kRingNb;
            }
        }
    }
    if (!g->mfma_ok) {
        g->Hp = ((g->H + 31) / 32) * 32;
    }
    return g->mfma_ok;
}

}  // namespace enova

namespace {

template <typename T>
enova_status dev_upload(T **dst, const void *src, size_t bytes)
{
    if (bytes == 0)
        bytes = 16;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(dst), bytes);
    if (e != hipSuccess)
        return fail(ENOVA_ENOMEM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
    if (src) {
        e = hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess)
            return hip_fail(e, "hipMemcpy weights");
    }
    return ENOVA_OK;
}

template <typename T>
enova_status ensure(T **buf, size_t *cap, size_t need)
{
    if (need <= *cap && *buf)
        return ENOVA_OK;
    if (*buf) {
        (void)hipFree(*buf);
        *buf = nullptr;
        *cap = 0;
    }
    size_t n = std::max<size_t>(need, 64);
    hipError_t e = hipMalloc(reinterpret_cast<void **>(buf), n * sizeof(T));
    if (e != hipSuccess)
        return fail(ENOVA_ENOMEM, "workspace hipMalloc(%zu): %s", n * sizeof(T), hipGetErrorString(e));
    *cap = n;
    return ENOVA_OK;
}

// Fragments of the ring kernel (bf16 detectors with 193..256 hidden units), one allocation:
//  W1      step i = q * KS + sp (KS = P / 4), hidden block hb (16 rows), lane l: the 8 bf16 of
//          W1[16 hb + l % 16] at the elements of chunk 4 sp + l / 16 of super-row q (zero past the
//          window, the hidden width or the super-row's chunks); kPrefetchSteps zero steps follow.
//  heads   [wave w][m][zb][hi, lo][lane l] 8 bf16: row l % 16 of Wmu (zb = 0) or Wlv (zb = 1), zero
//          past L, at hidden rows 16 (4w + 2m) + 4 (l / 16) + t (t < 4) and
//          16 (4w + 2m + 1) + 4 (l / 16) + t - 4 (t >= 4) -- the accumulator rows the lane holds.
//  decoder [hidden block hb][hi, lo][lane l] 4 bf16: Wd1[16 hb + l % 16][4 (l / 16) + t].
// Weights of the heads and the decoder are split into bf16 hi + lo (the remainder rounded).
enova_status pack_ring(enova_detector d, const enova_detect_weights *w)
{
    const Geometry &g = d->g;
    const int H = g.H, L = g.L, D = g.D;
    const int KS = g.RP / 4, NS = g.Q * KS;
    constexpr int HBT = kRingHidden / 16;
    const size_t n_w1 = static_cast<size_t>(NS + kPrefetchSteps) * HBT * 64;   // 16-byte fragments
    const size_t n_wh = static_cast<size_t>(kRingWaves) * 2 * 2 * 2 * 64;       // 16-byte fragments
    const size_t n_wd = static_cast<size_t>(HBT) * 2 * 64;                      // 8-byte fragments
    std::vector<uint16_t> buf((n_w1 + n_wh) * 8 + n_wd * 4, 0);
    uint16_t *w1r = buf.data(), *whr = w1r + n_w1 * 8, *wdr = whr + n_wh * 8;
    const uint16_t *w1 = static_cast<const uint16_t *>(w->w1);
    for (int i = 0; i < NS; ++i) {
        const int q = i / KS, sp = i - q * KS;
        for (int hb = 0; hb < HBT; ++hb)
            for (int lane = 0; lane < 64; ++lane) {
                const int h = 16 * hb + (lane & 15);
                const int c = 4 * sp + (lane >> 4);
                if (h >= H || c >= g.CPR)
                    continue;
                uint16_t *dst = w1r + ((static_cast<size_t>(i) * HBT + hb) * 64 + lane) * 8;
                for (int e = 0; e < 8; ++e) {
                    const int jj = c * 8 + e;
                    const int tt = jj / g.Mp, m = jj - (jj / g.Mp) * g.Mp;
                    const int t = q * g.S + tt;
                    if (t < g.W && m < g.M)
                        dst[e] = w1[static_cast<int64_t>(h) * D + static_cast<int64_t>(t) * g.M + m];
                }
            }
    }
    auto split = [](float v, uint16_t &hi, uint16_t &lo) {
        hi = float_to_bf16_bits(v);
        lo = float_to_bf16_bits(v - bf16_bits_to_float(hi));
    };
    for (int wv = 0; wv < kRingWaves; ++wv)
        for (int m = 0; m < 2; ++m)
            for (int zb = 0; zb < 2; ++zb) {
                const size_t base = (((static_cast<size_t>(wv) * 2 + m) * 2 + zb) * 2) * 64;
                for (int lane = 0; lane < 64; ++lane) {
                    const int row = lane & 15, grp = lane >> 4;
                    for (int t = 0; t < 8; ++t) {
                        const int h = t < 4 ? 16 * (4 * wv + 2 * m) + 4 * grp + t
                                            : 16 * (4 * wv + 2 * m + 1) + 4 * grp + (t - 4);
                        float v = 0.0f;
                        if (h < H && row < L)
                            v = zb == 0 ? w->wmu[row * H + h] : w->wlv[row * H + h];
                        uint16_t hi, lo;
                        split(v, hi, lo);
                        whr[(base + lane) * 8 + t] = hi;
                        whr[(base + 64 + lane) * 8 + t] = lo;
                    }
                }
            }
    for (int hb = 0; hb < HBT; ++hb)
        for (int lane = 0; lane < 64; ++lane)
            for (int t = 0; t < 4; ++t) {
                const int h = 16 * hb + (lane & 15);
                const int l = 4 * (lane >> 4) + t;
                float v = 0.0f;
                if (h < H && l < L)
                    v = w->wd1[h * L + l];
                uint16_t hi, lo;
                split(v, hi, lo);
                wdr[((static_cast<size_t>(hb) * 2 + 0) * 64 + lane) * 4 + t] = hi;
                wdr[((static_cast<size_t>(hb) * 2 + 1) * 64 + lane) * 4 + t] = lo;
            }
    enova_status st = dev_upload(&d->ring_w, buf.data(), buf.size() * sizeof(uint16_t));
    if (st != ENOVA_OK)
        return st;
    const uint4 *base = static_cast<const uint4 *>(d->ring_w);
    d->w1r = base;
    d->whr = base + n_w1;
    d->wdr = reinterpret_cast<const uint2 *>(base + n_w1 + n_wh);
    const hipError_t e = prepare_score_ring(g);
    return e == hipSuccess ? ENOVA_OK : hip_fail(e, "configure the ring scoring kernel");
}

// Fragments of the streaming kernel's 16x16 matrix ops: W1 as A fragments
// [stream_w1_steps][Hp/16][64 lanes] x 16 bytes (lane l: hidden row 16 hb + l%16, chunk
// 4 step + l/16 in the detector's chunk order, zeros past the window), the heads as
// [Hp/16][4][2][64] floats (op (hb, r) of head 0 = mean, 1 = log-variance: lane l holds the head
// row l%16 at hidden unit 16 hb + 4 (l/16) + r) and the decoder's hidden layer as [Hp/16][4][64]
// floats (op (hb, r): lane l holds Wd1[16 hb + l%16][4 (l/16) + r]).
enova_status pack_stream(enova_detector d, const enova_detect_weights *w)
{
    const Geometry &g = d->g;
    const int H = g.H, L = g.L, D = g.D, NHB = g.Hp / 16;
    const bool bf = g.dtype == ENOVA_BF16;
    const int steps = stream_w1_steps(g);
    const size_t n_w1 = static_cast<size_t>(steps) * NHB * 64;   // 16-byte fragments
    const size_t n_wh = static_cast<size_t>(NHB) * 4 * 2 * 64;   // floats
    const size_t n_wd = static_cast<size_t>(NHB) * 4 * 64;       // floats
    std::vector<uint32_t> buf(n_w1 * 4 + n_wh + n_wd, 0u);
    for (int j = 0; j < steps; ++j)
        for (int hb = 0; hb < NHB; ++hb)
            for (int lane = 0; lane < 64; ++lane) {
                const int h = 16 * hb + (lane & 15);
                const int kappa = 4 * j + (lane >> 4);
                if (h >= H || kappa >= g.KC)
                    continue;
                const int q = kappa / g.CPR;
                const int c = kappa - q * g.CPR;
                uint16_t bits[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                float vals[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                for (int e = 0; e < g.epc; ++e) {
                    const int jj = c * g.epc + e;
                    const int tt = jj / g.Mp;
                    const int m = jj - tt * g.Mp;
                    const int t = q * g.S + tt;
                    if (q < g.Q && t < g.W && m < g.M) {
                        const int64_t at = static_cast<int64_t>(h) * D + static_cast<int64_t>(t) * g.M + m;
                        if (bf)
                            bits[e] = static_cast<const uint16_t *>(w->w1)[at];
                        else
                            vals[e] = static_cast<const float *>(w->w1)[at];
                    }
                }
                uint32_t *dst = &buf[((static_cast<size_t>(j) * NHB + hb) * 64 + lane) * 4];
                if (bf) {
                    for (int e = 0; e < 4; ++e)
                        dst[e] = static_cast<uint32_t>(bits[2 * e]) | (static_cast<uint32_t>(bits[2 * e + 1]) << 16);
                } else {
                    std::memcpy(dst, vals, 16);
                }
            }
    float *wh = reinterpret_cast<float *>(buf.data() + n_w1 * 4);
    float *wd = wh + n_wh;
    for (int hb = 0; hb < NHB; ++hb)
        for (int r = 0; r < 4; ++r)
            for (int lane = 0; lane < 64; ++lane) {
                const int row = lane & 15;
                const int hh = 16 * hb + 4 * (lane >> 4) + r;
                if (hh < H && row < L) {
                    wh[((hb * 4 + r) * 2 + 0) * 64 + lane] = w->wmu[row * H + hh];
                    wh[((hb * 4 + r) * 2 + 1) * 64 + lane] = w->wlv[row * H + hh];
                }
                const int hd = 16 * hb + row;
                const int l = 4 * (lane >> 4) + r;
                if (hd < H && l < L)
                    wd[(hb * 4 + r) * 64 + lane] = w->wd1[hd * L + l];
            }
    enova_status st = dev_upload(&d->stream_w, buf.data(), buf.size() * sizeof(uint32_t));
    if (st != ENOVA_OK)
        return st;
    d->w1s = static_cast<const uint4 *>(d->stream_w);
    d->whs = reinterpret_cast<const float *>(d->w1s + n_w1);
    d->wds = d->whs + n_wh;
    const hipError_t e = prepare_stream_score(g);
    return e == hipSuccess ? ENOVA_OK : hip_fail(e, "configure the streaming scoring kernel");
}

// Row of register r for lane half g inside a 32x32 matrix-op accumulator block.
int crow(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Decoder-output fragments of the fused variant pass (32x32x2 fp32 ops whose B operand is the
// decoder hidden layer's accumulator): Wd2 as [D/32][HB][4][64 lanes] x 4 floats, where lane l,
// component e of (ob, hb, r4) holds Wd2[32 ob + l%32][32 hb + crow(4 r4 + e, l/32)] (zero past
// H).
enova_status pack_ext_fused(enova_detector d, const enova_detect_weights *w)
{
    const Geometry &g = d->g;
    const int H = g.H, D = g.D, HB = g.HB, nob = D / 32;
    const size_t n_w = static_cast<size_t>(nob) * HB * 4 * 64 * 4;
    std::vector<float> buf(n_w, 0.0f);
    for (int ob = 0; ob < nob; ++ob)
        for (int hb = 0; hb < HB; ++hb)
            for (int r4 = 0; r4 < 4; ++r4)
                for (int lane = 0; lane < 64; ++lane)
                    for (int e = 0; e < 4; ++e) {
                        const int j = 32 * ob + (lane & 31);
                        const int h = 32 * hb + crow(4 * r4 + e, lane >> 5);
                        if (h < H)
                            buf[((((static_cast<size_t>(ob) * HB + hb) * 4 + r4) * 64 + lane) * 4) + e] =
                                w->wd2[static_cast<int64_t>(j) * H + h];
                    }
    enova_status st = dev_upload(&d->ext_w, buf.data(), buf.size() * sizeof(float));
    if (st != ENOVA_OK)
        return st;
    d->wd2p = static_cast<const float4 *>(d->ext_w);
    const hipError_t e = prepare_ext_fused(g);
    return e == hipSuccess ? ENOVA_OK : hip_fail(e, "configure the fused variant kernel");
}

void free_detector(enova_detector d)
{
    if (!d)
        return;
    void *ptrs[] = {d->w1p, d->w1t, d->small, d->stats, d->tiles, d->tile_map, d->cal, d->hist,
                    d->peaks, d->blk, d->gx, d->dense, d->ext_ws, d->ring_w, d->stream_w, d->ext_w};
    for (void *p : ptrs)
        if (p)
            (void)hipFree(p);
    if (d->gpin)
        (void)hipHostFree(d->gpin);
    for (hipEvent_t e : d->ev)
        if (e)
            (void)hipEventDestroy(e);
    for (hipEvent_t e : d->ext_ev)
        if (e)
            (void)hipEventDestroy(e);
    delete d;
}

enova_status check_config(const enova_detect_config *c)
{
    if (!c)
        return fail(ENOVA_EINVAL, "config is NULL");
    if (c->metrics < 1 || c->window < 1 || c->stride < 1 || c->hidden < 1 || c->latent < 1)
        return fail(ENOVA_EINVAL, "metrics, window, stride, hidden and latent must be >= 1");
    if (c->latent > 64)
        return fail(ENOVA_EINVAL, "latent %d > 64", c->latent);
    if (static_cast<int64_t>(c->window) * c->metrics > 65536)
        return fail(ENOVA_EINVAL, "window*metrics = %lld > 65536",
                    static_cast<long long>(c->window) * c->metrics);
    if (c->dtype != ENOVA_F32 && c->dtype != ENOVA_BF16)
        return fail(ENOVA_EINVAL, "unknown dtype %d", c->dtype);
    if (c->act != ENOVA_RELU && c->act != ENOVA_TANH)
        return fail(ENOVA_EINVAL, "unknown activation %d", c->act);
    if (c->kernel < ENOVA_KERNEL_AUTO || c->kernel > ENOVA_KERNEL_MFMA)
        return fail(ENOVA_EINVAL, "unknown kernel choice %d", c->kernel);
    if (!(c->ref_frac > 0.0f && c->ref_frac <= 1.0f))
        return fail(ENOVA_EINVAL, "ref_frac must be in (0, 1]");
    return ENOVA_OK;
}

// Likelihood sums of the GPD fit, evaluated on the device over the compacted excesses.
struct DeviceGpdSums : GpdSums {
    enova_detector d;
    const double *y;
    int64_t n;
    hipStream_t st;
    enova_status status = ENOVA_OK;
    DeviceGpdSums(enova_detector d_, const double *y_, int64_t n_, hipStream_t s_)
        : d(d_), y(y_), n(n_), st(s_) {}
    bool eval(const double *xs, int nx, double *sa, double *sb) override
    {
        return run(xs, nx, sa, sb, nullptr, nullptr);
    }
    bool eval_d(const double *xs, int nx, double *sa, double *sb, double *sda, double *sdb) override
    {
        return run(xs, nx, sa, sb, sda, sdb);
    }
    // the sums at nx points (with sda and sdb, else NULL, also their derivatives)
    bool run(const double *xs, int nx, double *sa, double *sb, double *sda, double *sdb)
    {
        if (nx <= 0)
            return true;
        const int nv = sda ? 4 : 2;      // sums per point
        const int ns = gpd_split(n, nx);
        const size_t np = static_cast<size_t>(nx) * ns;
        status = ensure(&d->gx, &d->gx_cap, 5 * static_cast<size_t>(nx) + 4 * np);
        if (status != ENOVA_OK)
            return false;
        // pinned host staging: the points, then the sums per point (5 nx doubles at most)
        if (d->gpin_cap < 5 * static_cast<size_t>(nx)) {
            if (d->gpin)
                (void)hipHostFree(d->gpin);
            d->gpin = nullptr;
            d->gpin_cap = 0;
            const size_t cap = std::max<size_t>(5 * static_cast<size_t>(nx), 5 * 1024);
            if (hipHostMalloc(reinterpret_cast<void **>(&d->gpin), cap * sizeof(double)) != hipSuccess) {
                d->gpin = nullptr;
                status = fail(ENOVA_ENOMEM, "pinned host buffer of %zu doubles", cap);
                return false;
            }
            d->gpin_cap = cap;
        }
        // device: x, the sums [nv][nx], then the chunk partials [nv][nx][ns]
        double *dx = d->gx, *ds = dx + nx, *dp = ds + 4 * static_cast<size_t>(nx);
        double *dpart[4] = {dp, dp + np, dp + 2 * np, dp + 3 * np};
        double *hx = d->gpin, *hs = hx + nx;
        std::copy(xs, xs + nx, hx);
        hipError_t e;
        if ((e = hipMemcpyAsync(dx, hx, sizeof(double) * nx, hipMemcpyHostToDevice, st)) != hipSuccess ||
            (e = launch_gpd_sums(y, n, dx, nx, ns, dpart[0], dpart[1], sda ? dpart[2] : nullptr,
                                 sda ? dpart[3] : nullptr, st)) != hipSuccess ||
            (e = launch_gpd_reduce(dpart[0], dpart[1], nx, ns, ds, ds + nx, st)) != hipSuccess ||
            (sda && (e = launch_gpd_reduce(dpart[2], dpart[3], nx, ns, ds + 2 * nx, ds + 3 * nx, st)) != hipSuccess) ||
            (e = hipMemcpyAsync(hs, ds, sizeof(double) * nv * nx, hipMemcpyDeviceToHost, st)) != hipSuccess ||
            (e = hipStreamSynchronize(st)) != hipSuccess) {
            status = hip_fail(e, "GPD likelihood sums");
            return false;
        }
        std::copy(hs, hs + nx, sa);
        std::copy(hs + nx, hs + 2 * nx, sb);
        if (sda) {
            std::copy(hs + 2 * nx, hs + 3 * nx, sda);
            std::copy(hs + 3 * nx, hs + 4 * nx, sdb);
        }
        return true;
    }
};

}  // namespace

extern "C" {

const char *enova_status_str(enova_status s)
{
    switch (s) {
    case ENOVA_OK: return "ok";
    case ENOVA_EINVAL: return "invalid argument";
    case ENOVA_ESHAPE: return "nothing to act on for this shape";
    case ENOVA_ENOMEM: return "out of memory";
    case ENOVA_EHIP: return "HIP runtime error";
    case ENOVA_EUNSUPPORTED: return "unsupported request";
    case ENOVA_ENUMERIC: return "non-finite values";
    }
    return "unknown status";
}

const char *enova_last_error(void) { return g_last_error.c_str(); }

enova_status enova_detect_init(const enova_detect_config *config, const enova_detect_weights *w,
                               enova_detector *out)
{
    if (!out)
        return fail(ENOVA_EINVAL, "out is NULL");
    *out = nullptr;
    enova_status st = check_config(config);
    if (st != ENOVA_OK)
        return st;
    if (!w || !w->w1 || !w->b1 || !w->wmu || !w->bmu || !w->wlv || !w->blv || !w->wd1 || !w->bd1 ||
        !w->wd2 || !w->bd2)
        return fail(ENOVA_EINVAL, "a weight pointer is NULL");

    enova_detector d = new (std::nothrow) enova_detector_s();
    if (!d)
        return fail(ENOVA_ENOMEM, "host allocation");
    Geometry &g = d->g;
    plan_geometry(*config, &g);
    if (config->kernel == ENOVA_KERNEL_MFMA && !g.mfma_ok) {
        // the message reads the geometry, which the detector owns: format it before the free
        st = fail(ENOVA_EUNSUPPORTED,
                  "matrix-core kernel needs hidden <= 256, latent <= 16 and a tile that fits LDS "
                  "(H=%d L=%d LDS=%zu)", g.H, g.L, g.lds_bytes);
        free_detector(d);
        return st;
    }
    if (config->kernel == ENOVA_KERNEL_VALU || !g.mfma_ok) {
        if (g.H > 1024) {
            st = fail(ENOVA_EUNSUPPORTED, "hidden width %d > 1024 is not supported", g.H);
            free_detector(d);
            return st;
        }
        d->kind = 1;
    } else {
        d->kind = 2;
    }
    if (hipGetDevice(&d->device) != hipSuccess) {
        free_detector(d);
        return fail(ENOVA_EHIP, "no current HIP device");
    }
    {
        // the device address of this device's fixed scratch, looked up with the device current
        const hipError_t e = scratch_setup(d->device, &d->scratch);
        if (e != hipSuccess) {
            free_detector(d);
            return hip_fail(e, "device scratch lookup");
        }
    }

    const int H = g.H, L = g.L, D = g.D, Hp = g.Hp;
    const bool bf = g.dtype == ENOVA_BF16;
    auto w1v = [&](int h, int j) -> float {
        if (bf)
            return bf16_bits_to_float(static_cast<const uint16_t *>(w->w1)[static_cast<int64_t>(h) * D + j]);
        return static_cast<const float *>(w->w1)[static_cast<int64_t>(h) * D + j];
    };

    // small arrays: b1[Hp] bd1[Hp] u[Hp] bh[32] bmu[L] blv[L] wmu[L*H] wlv[L*H] wd1[H*L]
    //               whp[HB*16*64] wd1p[HB*8*64]
    const size_t n_whp = d->kind == 2 ? static_cast<size_t>(g.HB) * 16 * 64 : 0;
    const size_t n_wd1p = d->kind == 2 ? static_cast<size_t>(g.HB) * 8 * 64 : 0;
    // every sub-array starts on a 16-byte boundary (the kernels copy them with 16-byte loads)
    size_t o = 0;
    auto take = [&o](size_t n) {
        const size_t at = o;
        o += (n + 3) / 4 * 4;
        return at;
    };
    // the matrix-core kernel copies whp, wd1p, b1, bd1, u, bh as one contiguous block into LDS
    const size_t o_whp = take(n_whp);
    const size_t o_wd1p = take(n_wd1p);
    const size_t o_b1 = take(Hp);
    const size_t o_bd1 = take(Hp);
    const size_t o_u = take(Hp);
    const size_t o_bh = take(32);
    const size_t o_bmu = take(L);
    const size_t o_blv = take(L);
    const size_t o_wmu = take(static_cast<size_t>(L) * H);
    const size_t o_wlv = take(static_cast<size_t>(L) * H);
    const size_t o_wd1 = take(static_cast<size_t>(H) * L);
    std::vector<float> small(o, 0.0f);

    for (int h = 0; h < H; ++h) {
        small[o_b1 + h] = w->b1[h];
        small[o_bd1 + h] = w->bd1[h];
        double cs = 0.0;
        for (int j = 0; j < D; ++j)
            cs += static_cast<double>(w->wd2[static_cast<int64_t>(j) * H + h]);
        small[o_u + h] = static_cast<float>(cs);
    }
    double sb = 0.0;
    for (int j = 0; j < D; ++j)
        sb += static_cast<double>(w->bd2[j]);
    d->sum_bd2 = static_cast<float>(sb);
    for (int l = 0; l < L; ++l) {
        small[o_bmu + l] = w->bmu[l];
        small[o_blv + l] = w->blv[l];
        if (l < 16) {
            small[o_bh + l] = w->bmu[l];
            small[o_bh + 16 + l] = w->blv[l];
        }
    }
    std::memcpy(&small[o_wmu], w->wmu, sizeof(float) * L * H);
    std::memcpy(&small[o_wlv], w->wlv, sizeof(float) * L * H);
    std::memcpy(&small[o_wd1], w->wd1, sizeof(float) * H * L);
    if (d->kind == 2 && bf) {
        // bf16 workload: the heads and decoder weights as bf16 hi + lo fragments of the
        // 32x32x16 matrix op; reduction slot (g, t) of heads op m is hidden row crow(8m + t, g),
        // of the decoder op latent crow(t, g)
        uint16_t *whb = reinterpret_cast<uint16_t *>(&small[o_whp]);
        uint16_t *wdb = reinterpret_cast<uint16_t *>(&small[o_wd1p]);
        for (int hb = 0; hb < g.HB; ++hb)
            for (int m = 0; m < 2; ++m)
                for (int lane = 0; lane < 64; ++lane)
                    for (int t = 0; t < 8; ++t) {
                        const int row = lane & 31;          // 0..15 mean head, 16..31 log-variance
                        const int h = hb * 32 + crow(8 * m + t, lane >> 5);
                        float v = 0.0f;
                        if (h < H) {
                            if (row < 16 && row < L)
                                v = w->wmu[row * H + h];
                            else if (row >= 16 && row - 16 < L)
                                v = w->wlv[(row - 16) * H + h];
                        }
                        const uint16_t hi = float_to_bf16_bits(v);
                        const uint16_t lo = float_to_bf16_bits(v - bf16_bits_to_float(hi));
                        whb[((((static_cast<size_t>(hb) * 2 + m) * 2 + 0) * 64 + lane) * 8) + t] = hi;
                        whb[((((static_cast<size_t>(hb) * 2 + m) * 2 + 1) * 64 + lane) * 8) + t] = lo;
                    }
        for (int hb = 0; hb < g.HB; ++hb)
            for (int lane = 0; lane < 64; ++lane)
                for (int t = 0; t < 8; ++t) {
                    const int h = hb * 32 + (lane & 31);
                    const int l = crow(t, lane >> 5);
                    float v = 0.0f;
                    if (h < H && l < L)
                        v = w->wd1[h * L + l];
                    const uint16_t hi = float_to_bf16_bits(v);
                    const uint16_t lo = float_to_bf16_bits(v - bf16_bits_to_float(hi));
                    wdb[(((static_cast<size_t>(hb) * 2 + 0) * 64 + lane) * 8) + t] = hi;
                    wdb[(((static_cast<size_t>(hb) * 2 + 1) * 64 + lane) * 8) + t] = lo;
                }
    } else if (d->kind == 2) {
        for (int hb = 0; hb < g.HB; ++hb)
            for (int r = 0; r < 16; ++r)
                for (int lane = 0; lane < 64; ++lane) {
                    const int row = lane & 31;              // 0..15 mean head, 16..31 log-variance head
                    const int h = hb * 32 + crow(r, lane >> 5);
                    float v = 0.0f;
                    if (h < H) {
                        if (row < 16 && row < L)
                            v = w->wmu[row * H + h];
                        else if (row >= 16 && row - 16 < L)
                            v = w->wlv[(row - 16) * H + h];
                    }
                    small[o_whp + (static_cast<size_t>(hb) * 16 + r) * 64 + lane] = v;
                }
        for (int hb = 0; hb < g.HB; ++hb)
            for (int r = 0; r < 8; ++r)
                for (int lane = 0; lane < 64; ++lane) {
                    const int h = hb * 32 + (lane & 31);
                    const int l = crow(r, lane >> 5);
                    float v = 0.0f;
                    if (h < H && l < L)
                        v = w->wd1[h * L + l];
                    small[o_wd1p + (static_cast<size_t>(hb) * 8 + r) * 64 + lane] = v;
                }
    }
    st = dev_upload(&d->small, small.data(), small.size() * sizeof(float));
    if (st != ENOVA_OK) {
        free_detector(d);
        return st;
    }
    d->b1 = d->small + o_b1;
    d->bd1 = d->small + o_bd1;
    d->u = d->small + o_u;
    d->bh = d->small + o_bh;
    d->bmu = d->small + o_bmu;
    d->blv = d->small + o_blv;
    d->wmu = d->small + o_wmu;
    d->wlv = d->small + o_wlv;
    d->wd1 = d->small + o_wd1;
    d->whp = d->small + o_whp;
    d->wd1p = d->small + o_wd1p;

    {
        // dense fp32 copies for the output variants (16-byte aligned sub-arrays)
        size_t od = 0;
        auto takd = [&od](size_t n) {
            const size_t at = od;
            od += (n + 3) / 4 * 4;
            return at;
        };
        const size_t p_w1 = takd(static_cast<size_t>(H) * D), p_wml = takd(2 * static_cast<size_t>(L) * H),
                     p_bml = takd(2 * static_cast<size_t>(L)), p_wd1 = takd(static_cast<size_t>(H) * L),
                     p_wd2 = takd(static_cast<size_t>(D) * H), p_bd2 = takd(D);
        std::vector<float> dn(od, 0.0f);
        for (int h = 0; h < H; ++h)
            for (int j = 0; j < D; ++j)
                dn[p_w1 + static_cast<size_t>(h) * D + j] = w1v(h, j);
        std::memcpy(&dn[p_wml], w->wmu, sizeof(float) * L * H);
        std::memcpy(&dn[p_wml + static_cast<size_t>(L) * H], w->wlv, sizeof(float) * L * H);
        std::memcpy(&dn[p_bml], w->bmu, sizeof(float) * L);
        std::memcpy(&dn[p_bml + L], w->blv, sizeof(float) * L);
        std::memcpy(&dn[p_wd1], w->wd1, sizeof(float) * H * L);
        std::memcpy(&dn[p_wd2], w->wd2, sizeof(float) * static_cast<size_t>(D) * H);
        std::memcpy(&dn[p_bd2], w->bd2, sizeof(float) * D);
        st = dev_upload(&d->dense, dn.data(), dn.size() * sizeof(float));
        if (st != ENOVA_OK) {
            free_detector(d);
            return st;
        }
        d->d_w1 = d->dense + p_w1;
        d->d_wml = d->dense + p_wml;
        d->d_bml = d->dense + p_bml;
        d->d_wd1 = d->dense + p_wd1;
        d->d_wd2 = d->dense + p_wd2;
        d->d_bd2 = d->dense + p_bd2;
    }

    if (d->kind == 1) {
        // transposed W1 [D][H] in the storage type
        const size_t esz = bf ? 2 : 4;
        std::vector<unsigned char> wt(static_cast<size_t>(D) * H * esz);
        for (int h = 0; h < H; ++h)
            for (int j = 0; j < D; ++j) {
                const size_t dst = (static_cast<size_t>(j) * H + h) * esz;
                const size_t src = (static_cast<size_t>(h) * D + j) * esz;
                std::memcpy(&wt[dst], static_cast<const unsigned char *>(w->w1) + src, esz);
            }
        st = dev_upload(&d->w1t, wt.data(), wt.size());
    } else {
        // A fragments: step i, hidden block hb, lane -> 16 bytes of W1[h][chunk 2i + lane/32]
        // kPrefetchSteps zero steps follow the last one: the kernel's W1 prefetch runs past it
        const int steps = g.KC / 2;
        const size_t frag = static_cast<size_t>(steps + kPrefetchSteps) * g.HB * 64;
        std::vector<uint32_t> pk(frag * 4, 0u);
        for (int i = 0; i < steps; ++i)
            for (int hb = 0; hb < g.HB; ++hb)
                for (int lane = 0; lane < 64; ++lane) {
                    const int h = hb * 32 + (lane & 31);
                    const int kappa = 2 * i + (lane >> 5);
                    const int q = kappa / g.CPR;
                    const int c = kappa - q * g.CPR;
                    float vals[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    uint16_t bits[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    for (int e = 0; e < g.epc; ++e) {
                        const int jj = c * g.epc + e;
                        const int tt = jj / g.Mp;
                        const int m = jj - tt * g.Mp;
                        const int t = q * g.S + tt;
                        if (h < H && t < g.W && m < g.M && q < g.Q) {
                            const int64_t j = static_cast<int64_t>(t) * g.M + m;
                            if (bf)
                                bits[e] = static_cast<const uint16_t *>(w->w1)[static_cast<int64_t>(h) * D + j];
                            else
                                vals[e] = w1v(h, static_cast<int>(j));
                        }
                    }
                    uint32_t *dst = &pk[((static_cast<size_t>(i) * g.HB + hb) * 64 + lane) * 4];
                    if (bf) {
                        for (int e = 0; e < 4; ++e)
                            dst[e] = static_cast<uint32_t>(bits[2 * e]) |
                                     (static_cast<uint32_t>(bits[2 * e + 1]) << 16);
                    } else {
                        std::memcpy(dst, vals, 16);
                    }
                }
        st = dev_upload(&d->w1p, pk.data(), pk.size() * sizeof(uint32_t));
        if (st == ENOVA_OK) {
            hipError_t e = prepare_score_mfma(g);
            if (e != hipSuccess)
                st = hip_fail(e, "configure matrix-core kernel");
        }
        if (st == ENOVA_OK && g.ring)
            st = pack_ring(d, w);
        if (st == ENOVA_OK && stream_score_supported(g))
            st = pack_stream(d, w);
        if (st == ENOVA_OK && ext_fused_supported(g))
            st = pack_ext_fused(d, w);
    }
    if (st == ENOVA_OK) {
        static_assert(sizeof(RadixState) <= 8 * sizeof(unsigned int), "radix state after the bins");
        hipError_t e = hipMalloc(reinterpret_cast<void **>(&d->hist), (256 + 8) * sizeof(unsigned int));
        if (e != hipSuccess)
            st = fail(ENOVA_ENOMEM, "hipMalloc(hist)");
    }
    if (st != ENOVA_OK) {
        free_detector(d);
        return st;
    }
    *out = d;
    return ENOVA_OK;
}

enova_status enova_detect_destroy(enova_detector det)
{
    if (!det)
        return ENOVA_OK;
    DeviceGuard dg(det->device);
    (void)hipDeviceSynchronize();
    free_detector(det);
    return ENOVA_OK;
}

enova_status enova_detect_window_offsets(enova_detector det, const int64_t *soff, int32_t n,
                                         int64_t *woff)
{
    if (!det || !soff || !woff)
        return fail(ENOVA_EINVAL, "NULL argument");
    if (n < 0)
        return fail(ENOVA_EINVAL, "n_streams < 0");
    if (soff[0] != 0)
        return fail(ENOVA_EINVAL, "stream_offsets[0] must be 0");
    const int64_t W = det->g.W, S = det->g.S;
    woff[0] = 0;
    for (int32_t s = 0; s < n; ++s) {
        const int64_t T = soff[s + 1] - soff[s];
        if (T < 0)
            return fail(ENOVA_EINVAL, "stream_offsets decrease at stream %d", s);
        woff[s + 1] = woff[s] + (T >= W ? (T - W) / S + 1 : 0);
    }
    return ENOVA_OK;
}

enova_status enova_detect_ref_stats(enova_detector det, const void *x, const int64_t *soff,
                                    int32_t n, float *out_mean, float *out_std, hipStream_t stream)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    if (n < 0)
        return fail(ENOVA_EINVAL, "n_streams < 0");
    if (n == 0)
        return ENOVA_OK;
    if (!x || !soff || !out_mean || !out_std)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(det->device);
    hipError_t e = launch_ref_stats(det->g, x, soff, n, out_mean, out_std, stream);
    if (e != hipSuccess)
        return hip_fail(e, "reference statistics kernel");
    return ENOVA_OK;
}

namespace {

// The scoring path's workspace: reference statistics [2][n][M] floats (when the caller gives
// none), the matrix-core kernel's first tile of each stream [n+1] and stream of each block [grid].
struct ScoreWork {
    float *stats = nullptr;
    int64_t *tiles = nullptr;
    int *tile_map = nullptr;
};

// Bytes of the fixed-scratch layout of that workspace, each part on a 256-byte boundary.
size_t noalloc_bytes(const Geometry &g, int kind, int32_t n, int64_t grid, bool stats, size_t *o_tiles,
                     size_t *o_map)
{
    auto up = [](size_t v) { return (v + 255) / 256 * 256; };
    size_t o = stats ? up(2 * static_cast<size_t>(n) * g.M * sizeof(float)) : 0;
    *o_tiles = o;
    if (kind == 2)
        o += up((static_cast<size_t>(n) + 1) * sizeof(int64_t));
    *o_map = o;
    if (kind == 2)
        o += up(static_cast<size_t>(grid > 0 ? grid : 1) * sizeof(int));
    return o;
}

// Both scoring entry points. noalloc: the workspace is carved from the device's fixed scratch
// (no allocation, no timing events); otherwise it is the detector's grow-only workspace.
enova_status score_common(enova_detector det, const void *x, const int64_t *soff, const int64_t *woff, int32_t n,
                          int64_t n_windows, const float *ref_mean, const float *ref_std, float threshold,
                          float *out_scores, float *out_md, uint8_t *out_flags, hipStream_t stream, bool noalloc)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    if (n < 0 || n_windows < 0)
        return fail(ENOVA_EINVAL, "n_streams and n_windows must be >= 0");
    if ((ref_mean == nullptr) != (ref_std == nullptr))
        return fail(ENOVA_EINVAL, "ref_mean and ref_std must both be given or both be NULL");
    det->ran_stats = det->ran_score = false;
    if (n == 0 || n_windows == 0)
        return ENOVA_OK;
    if (!x || !soff || !woff || !out_scores)
        return fail(ENOVA_EINVAL, "NULL argument");
    const bool want_flags = out_flags != nullptr && !std::isnan(threshold);
    const Geometry &g = det->g;
    const int64_t grid = det->kind == 2 ? (n_windows + g.Nb - 1) / g.Nb + n : 0;
    if (grid > 0x7fffffffLL)
        return fail(ENOVA_EUNSUPPORTED, "too many tiles (%lld)", static_cast<long long>(grid));
    if (det->kind != 2 && (n_windows + 15) / 16 > 0x7fffffffLL)
        return fail(ENOVA_EUNSUPPORTED, "too many windows");
    ScoreWork wk;
    if (noalloc) {
        size_t o_tiles = 0, o_map = 0;
        const size_t need = noalloc_bytes(g, det->kind, n, grid, !ref_mean, &o_tiles, &o_map);
        if (need > kScratchBytes)
            return fail(ENOVA_ESHAPE,
                        "the allocation-free call needs %zu bytes of device scratch for %d streams and %lld "
                        "windows; it has %zu",
                        need, n, static_cast<long long>(n_windows), kScratchBytes);
        if (!det->scratch)
            return fail(ENOVA_EHIP, "device scratch unavailable");
        unsigned char *base = static_cast<unsigned char *>(det->scratch);
        wk.stats = reinterpret_cast<float *>(base);
        wk.tiles = reinterpret_cast<int64_t *>(base + o_tiles);
        wk.tile_map = reinterpret_cast<int *>(base + o_map);
    }
    DeviceGuard dg(det->device);
    if (!dg.ok)
        return fail(ENOVA_EHIP, "cannot select the detector's device");
    hipError_t e;
    const bool timing = det->timing && !noalloc;
    if (timing && !det->ev[0]) {
        for (auto &ev : det->ev)
            if ((e = hipEventCreate(&ev)) != hipSuccess)
                return hip_fail(e, "hipEventCreate");
    }
    if (!noalloc) {
        enova_status st = ENOVA_OK;
        if (!ref_mean)
            st = ensure(&det->stats, &det->stats_cap, 2 * static_cast<size_t>(n) * g.M);
        if (st == ENOVA_OK && det->kind == 2) {
            st = ensure(&det->tiles, &det->tiles_cap, static_cast<size_t>(n) + 1);
            if (st == ENOVA_OK)
                st = ensure(&det->tile_map, &det->tile_map_cap, static_cast<size_t>(grid > 0 ? grid : 1));
        }
        if (st != ENOVA_OK)
            return st;
        wk.stats = det->stats;
        wk.tiles = det->tiles;
        wk.tile_map = det->tile_map;
    }
    if (!ref_mean) {
        ref_mean = wk.stats;
        ref_std = wk.stats + static_cast<size_t>(n) * g.M;
        if (timing)
            (void)hipEventRecord(det->ev[0], stream);
        e = launch_ref_stats(g, x, soff, n, wk.stats, wk.stats + static_cast<size_t>(n) * g.M, stream);
        if (e != hipSuccess)
            return hip_fail(e, "reference statistics kernel");
        if (timing)
            (void)hipEventRecord(det->ev[1], stream);
        det->ran_stats = timing;
    }
    ScoreParams p{};
    p.x = x;
    p.soff = soff;
    p.woff = woff;
    p.n_streams = n;
    p.n_windows = n_windows;
    p.mean = ref_mean;
    p.std = ref_std;
    p.w1p = static_cast<const uint4 *>(det->w1p);
    p.whp = det->whp;
    p.wd1p = det->wd1p;
    p.w1t = det->w1t;
    p.wmu = det->wmu;
    p.wlv = det->wlv;
    p.wd1 = det->wd1;
    p.b1 = det->b1;
    p.bh = det->bh;
    p.bmu = det->bmu;
    p.blv = det->blv;
    p.bd1 = det->bd1;
    p.u = det->u;
    p.w1r = det->w1r;
    p.whr = det->whr;
    p.wdr = det->wdr;
    p.sum_bd2 = det->sum_bd2;
    p.threshold = threshold;
    p.write_flags = want_flags ? 1 : 0;
    p.scores = out_scores;
    p.md = out_md;
    p.flags = out_flags;
    if (det->kind == 2) {
        e = launch_stream_scan(g, soff, woff, n, 0, g.Nb, wk.tiles, stream);
        if (e != hipSuccess)
            return hip_fail(e, "tile scan kernel");
        p.tile_off = wk.tiles;
        e = launch_tile_map(wk.tiles, n, grid, wk.tile_map, stream);
        if (e != hipSuccess)
            return hip_fail(e, "tile map kernel");
        p.tile_stream = wk.tile_map;
        if (timing)
            (void)hipEventRecord(det->ev[2], stream);
        e = g.ring ? launch_score_ring(g, p, grid, stream) : launch_score_mfma(g, p, grid, stream);
    } else {
        if (timing)
            (void)hipEventRecord(det->ev[2], stream);
        e = launch_score_valu(g, p, stream);
    }
    if (e != hipSuccess)
        return hip_fail(e, "scoring kernel");
    if (timing)
        (void)hipEventRecord(det->ev[3], stream);
    det->ran_score = timing;
    return ENOVA_OK;
}

}  // namespace

enova_status enova_detect_score(enova_detector det, const void *x, const int64_t *soff,
                                const int64_t *woff, int32_t n, int64_t n_windows,
                                const float *ref_mean, const float *ref_std, float threshold,
                                float *out_scores, float *out_md, uint8_t *out_flags,
                                hipStream_t stream)
{
    return score_common(det, x, soff, woff, n, n_windows, ref_mean, ref_std, threshold, out_scores, out_md,
                        out_flags, stream, false);
}

enova_status enova_detect_score_noalloc(enova_detector det, const void *x, const int64_t *soff,
                                        const int64_t *woff, int32_t n, int64_t n_windows,
                                        const float *ref_mean, const float *ref_std, float threshold,
                                        float *out_scores, float *out_md, uint8_t *out_flags,
                                        hipStream_t stream)
{
    return score_common(det, x, soff, woff, n, n_windows, ref_mean, ref_std, threshold, out_scores, out_md,
                        out_flags, stream, true);
}

enova_status enova_detect_score_ext(enova_detector det, const void *x, const int64_t *soff, const int64_t *woff,
                                    int32_t n, int64_t n_windows, const float *ref_mean, const float *ref_std,
                                    int32_t norm, float *out_scores, float *out_md, float *out_md_metric,
                                    float *out_recon, hipStream_t stream)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    if (n < 0 || n_windows < 0)
        return fail(ENOVA_EINVAL, "n_streams and n_windows must be >= 0");
    if (norm != ENOVA_NORM_REFERENCE && norm != ENOVA_NORM_WINDOW)
        return fail(ENOVA_EINVAL, "bad normalisation mode");
    if ((ref_mean == nullptr) != (ref_std == nullptr))
        return fail(ENOVA_EINVAL, "ref_mean and ref_std must both be given or both be NULL");
    det->ran_ext = false;
    if (n == 0 || n_windows == 0)
        return ENOVA_OK;
    if (!x || !soff || !woff)
        return fail(ENOVA_EINVAL, "NULL argument");
    const Geometry &g = det->g;
    if (g.M > kExtMaxM)
        return fail(ENOVA_EUNSUPPORTED, "output variants support at most %d metrics", kExtMaxM);
    DeviceGuard dg(det->device);
    if (!dg.ok)
        return fail(ENOVA_EHIP, "cannot select the detector's device");
    hipError_t e;
    if (det->timing && !det->ext_ev[0]) {
        for (auto &ev : det->ext_ev)
            if ((e = hipEventCreate(&ev)) != hipSuccess)
                return hip_fail(e, "hipEventCreate");
    }
    const int D = g.D, H = g.H, L = g.L, M = g.M;
    if (det->wd2p) {
        // fused pass: one block per 256-window tile, every output written directly
        const int64_t grid = (n_windows + kExtFusedNb - 1) / kExtFusedNb + n;
        if (grid > 0x7fffffffLL)
            return fail(ENOVA_EUNSUPPORTED, "too many tiles (%lld)", static_cast<long long>(grid));
        const bool stats = norm == ENOVA_NORM_REFERENCE && !ref_mean;
        // workspace: reference statistics [2][n][M] floats, first tile of each stream [n+1]
        // int64, stream of each block [grid] ints
        const size_t n_st = stats ? (2 * static_cast<size_t>(n) * M + 3) / 4 * 4 : 0;
        const size_t n_tiles = 2 * (static_cast<size_t>(n) + 1);
        enova_status st = ensure(&det->ext_ws, &det->ext_ws_cap, n_st + n_tiles + static_cast<size_t>(grid) + 4);
        if (st != ENOVA_OK)
            return st;
        int64_t *tiles = reinterpret_cast<int64_t *>(det->ext_ws + n_st);
        int *tmap = reinterpret_cast<int *>(tiles + n + 1);
        if (det->timing)
            (void)hipEventRecord(det->ext_ev[0], stream);
        if (stats) {
            ref_mean = det->ext_ws;
            ref_std = det->ext_ws + static_cast<size_t>(n) * M;
            if ((e = launch_ref_stats(g, x, soff, n, det->ext_ws, det->ext_ws + static_cast<size_t>(n) * M,
                                      stream)) != hipSuccess)
                return hip_fail(e, "reference statistics kernel");
        }
        if ((e = launch_stream_scan(g, soff, woff, n, 0, kExtFusedNb, tiles, stream)) != hipSuccess)
            return hip_fail(e, "tile scan kernel");
        if ((e = launch_tile_map(tiles, n, grid, tmap, stream)) != hipSuccess)
            return hip_fail(e, "tile map kernel");
        ExtFusedParams fp{};
        fp.x = static_cast<const float *>(x);
        fp.soff = soff;
        fp.woff = woff;
        fp.tile_off = tiles;
        fp.tile_stream = tmap;
        fp.mean = ref_mean;
        fp.std = ref_std;
        fp.w1p = static_cast<const uint4 *>(det->w1p);
        fp.cst = det->whp;
        fp.wd2p = det->wd2p;
        fp.bd2 = det->d_bd2;
        fp.scores = out_scores;
        fp.md = out_md;
        fp.mdm = out_md_metric;
        fp.rec = out_recon;
        fp.norm = norm;
        fp.decode = (out_md || out_md_metric || out_recon) ? 1 : 0;
        if ((e = launch_ext_fused(g, fp, grid, stream)) != hipSuccess)
            return hip_fail(e, "fused variant kernel");
        if (det->timing)
            (void)hipEventRecord(det->ext_ev[1], stream);
        det->ran_ext = true;
        return ENOVA_OK;
    }
    const int B = variants_chunk(D, n_windows);
    // workspace: V, out [B][D]; a1, h, a2, hd [B][H]; ml [B][2L]; the products' split partials,
    // for a full chunk and for the last, shorter one
    const int last = variants_last_rows(n_windows, B);
    const int64_t wsg = variants_gemm_workspace(B, last, D, H, L);
    // With M a power of two <= 32 the decoder-output product reduces v - m' in its epilogue
    // (per window, metric and column slot) instead of writing m'; `out` then holds those sums.
    const bool fused = M <= 32 && (M & (M - 1)) == 0;
    const bool decode = out_md || out_md_metric || out_recon;
    const int slots = fused ? std::max(gemm_reduce_slots(B, D), gemm_reduce_slots(last, D)) : 0;
    auto up4 = [](size_t v) { return (v + 3) / 4 * 4; };   // every sub-buffer 16-byte aligned
    const size_t nBD = up4(static_cast<size_t>(B) * D), nBH = up4(static_cast<size_t>(B) * H),
                 nML = up4(static_cast<size_t>(B) * 2 * L);
    const size_t nP = up4(static_cast<size_t>(B) * slots * M), nQ = up4(static_cast<size_t>(B) * slots);
    const size_t nOut = fused ? nP + nQ : nBD;
    const size_t nMap = up4(static_cast<size_t>(B));   // the chunk's window -> stream map (ints)
    const size_t need = nBD + nOut + 4 * nBH + nML + nMap + static_cast<size_t>(wsg) + 16;
    enova_status st = ensure(&det->ext_ws, &det->ext_ws_cap, need);
    if (st != ENOVA_OK)
        return st;
    float *V = det->ext_ws, *out = V + nBD, *a1 = out + nOut, *h = a1 + nBH, *a2 = h + nBH, *hd = a2 + nBH,
          *ml = hd + nBH, *mapf = ml + nML, *gw = mapf + nMap;
    int *wmap = reinterpret_cast<int *>(mapf);
    if (det->timing)
        (void)hipEventRecord(det->ext_ev[0], stream);
    if (norm == ENOVA_NORM_REFERENCE && !ref_mean) {
        st = ensure(&det->stats, &det->stats_cap, 2 * static_cast<size_t>(n) * M);
        if (st != ENOVA_OK)
            return st;
        ref_mean = det->stats;
        ref_std = det->stats + static_cast<size_t>(n) * M;
        if ((e = launch_ref_stats(g, x, soff, n, det->stats, det->stats + static_cast<size_t>(n) * M, stream)) !=
            hipSuccess)
            return hip_fail(e, "reference statistics kernel");
    }
    GemmEpilogue plain{};
    GemmEpilogue enc;
    enc.kind = kEpiBiasAct;
    enc.act = g.act;
    enc.bias = det->b1;
    enc.out2 = h;
    GemmEpilogue dec = enc;
    dec.bias = det->bd1;
    dec.out2 = hd;
    GemmEpilogue red;   // fused reductions of d = v - (product + bd2)
    red.kind = kEpiRowReduce;
    red.bias = det->d_bd2;
    red.pre = V;
    red.ldv = D;
    red.groups = M;
    red.out2 = out;
    red.sq = out + nP;
    for (int64_t w0 = 0; w0 < n_windows; w0 += B) {
        const int rows = static_cast<int>(std::min<int64_t>(B, n_windows - w0));
        e = launch_ext_stage(x, g.dtype, soff, woff, n, w0, rows, M, g.W, g.S, norm, ref_mean, ref_std, wmap, V,
                             stream);
        if (e == hipSuccess)   // a1 = V W1^T + b1, h = act(a1)
            e = launch_gemm(enc, V, D, 1, det->d_w1, 1, D, a1, H, rows, H, D, nullptr, gw, wsg, stream);
        if (e == hipSuccess)   // [mu | lv] = h [Wmu; Wlv]^T
            e = launch_gemm(plain, h, H, 1, det->d_wml, 1, H, ml, 2 * L, rows, 2 * L, H, nullptr, gw, wsg, stream);
        if (e == hipSuccess)
            e = launch_ext_latent(ml, det->d_bml, rows, L, out_scores ? out_scores + w0 : nullptr, stream);
        if (e != hipSuccess)
            return hip_fail(e, "output-variant kernels");
        if (!decode)   // only scores requested: the decoder is not needed
            continue;
        if (e == hipSuccess)   // a2 = mu Wd1^T + bd1, hd = act(a2)
            e = launch_gemm(dec, ml, 2 * L, 1, det->d_wd1, 1, L, a2, H, rows, H, L, nullptr, gw, wsg, stream);
        float *o_md = out_md ? out_md + w0 : nullptr, *o_mdm = out_md_metric ? out_md_metric + w0 * M : nullptr,
              *o_rec = out_recon ? out_recon + w0 : nullptr;
        if (fused) {
            if (e == hipSuccess)   // decoder output, reduced against V in the epilogue
                e = launch_gemm(red, hd, H, 1, det->d_wd2, 1, H, out, D, rows, D, H, nullptr, gw, wsg, stream);
            if (e == hipSuccess)
                e = launch_ext_finish(out, out + nP, rows, gemm_reduce_slots(rows, D), M, g.W, o_md, o_mdm, o_rec,
                                      stream);
        } else {
            if (e == hipSuccess)   // decoder output without bd2
                e = launch_gemm(plain, hd, H, 1, det->d_wd2, 1, H, out, D, rows, D, H, nullptr, gw, wsg, stream);
            if (e == hipSuccess)
                e = launch_ext_reduce(V, out, det->d_bd2, rows, M, g.W, o_md, o_mdm, o_rec, stream);
        }
        if (e != hipSuccess)
            return hip_fail(e, "output-variant kernels");
    }
    if (det->timing)
        (void)hipEventRecord(det->ext_ev[1], stream);
    det->ran_ext = true;
    return ENOVA_OK;
}

enova_status enova_detect_ext_time(enova_detector det, double *ms)
{
    if (!det || !ms)
        return fail(ENOVA_EINVAL, "NULL argument");
    *ms = 0.0;
    if (!det->timing || !det->ran_ext || !det->ext_ev[1])
        return ENOVA_OK;
    DeviceGuard dg(det->device);
    hipError_t e = hipEventSynchronize(det->ext_ev[1]);
    float f = 0.0f;
    if (e == hipSuccess)
        e = hipEventElapsedTime(&f, det->ext_ev[0], det->ext_ev[1]);
    if (e != hipSuccess)
        return hip_fail(e, "event timing");
    *ms = f;
    return ENOVA_OK;
}

enova_status enova_detect_flag(enova_detector det, const float *scores, int64_t n_windows,
                               float threshold, uint8_t *out_flags, hipStream_t stream)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    if (n_windows < 0)
        return fail(ENOVA_EINVAL, "n_windows < 0");
    if (n_windows == 0)
        return ENOVA_OK;
    if (!scores || !out_flags)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(det->device);
    hipError_t e = launch_flag(scores, n_windows, threshold, out_flags, stream);
    if (e != hipSuccess)
        return hip_fail(e, "flag kernel");
    return ENOVA_OK;
}

enova_status enova_detect_threshold(enova_detector det, const float *scores, const int64_t *soff,
                                    const int64_t *woff, int32_t n, int64_t n_windows, double level,
                                    double q, float *out_threshold, double *out_info,
                                    uint8_t *out_flags, hipStream_t stream)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    if (!out_threshold)
        return fail(ENOVA_EINVAL, "out_threshold is NULL");
    if (!(level > 0.0 && level < 1.0) || !(q > 0.0 && q < 1.0))
        return fail(ENOVA_EINVAL, "level and q must lie in (0, 1)");
    if (n < 0 || n_windows < 0)
        return fail(ENOVA_EINVAL, "n_streams and n_windows must be >= 0");
    if (n == 0 || n_windows == 0)
        return fail(ENOVA_ESHAPE, "no windows to calibrate on");
    if (!scores || !soff || !woff)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(det->device);
    const Geometry &g = det->g;
    enova_status st = ensure(&det->cal, &det->cal_cap, static_cast<size_t>(n) + 1);
    if (st != ENOVA_OK)
        return st;
    hipError_t e = launch_stream_scan(g, soff, woff, n, 1, 1, det->cal, stream);
    if (e != hipSuccess)
        return hip_fail(e, "calibration scan kernel");
    int64_t n_cal = 0;
    if ((e = hipMemcpyAsync(&n_cal, det->cal + n, sizeof(int64_t), hipMemcpyDeviceToHost, stream)) !=
            hipSuccess ||
        (e = hipStreamSynchronize(stream)) != hipSuccess)
        return hip_fail(e, "calibration count");
    if (n_cal <= 0)
        return fail(ENOVA_ESHAPE, "no window lies inside a reference prefix");

    // exact order statistic at ceil(level*n) - 1 by a 4-pass radix select over float keys, each
    // pass's digit picked on the device (no host round trip until the key is known)
    int64_t rank = static_cast<int64_t>(std::ceil(level * static_cast<double>(n_cal))) - 1;
    if (rank < 0)
        rank = 0;
    if (rank > n_cal - 1)
        rank = n_cal - 1;
    RadixState *rs = reinterpret_cast<RadixState *>(det->hist + 256);
    if ((e = launch_radix_init(rs, rank, det->hist, stream)) != hipSuccess)
        return hip_fail(e, "radix select start");
    for (int shift = 24; shift >= 0; shift -= 8)
        if ((e = launch_calib_hist(scores, woff, det->cal, n, n_cal, shift, rs, det->hist, stream)) != hipSuccess)
            return hip_fail(e, "calibration histogram kernel");
    RadixState rh{};
    if ((e = hipMemcpyAsync(&rh, rs, sizeof(rh), hipMemcpyDeviceToHost, stream)) != hipSuccess ||
        (e = hipStreamSynchronize(stream)) != hipSuccess)
        return hip_fail(e, "radix select state");
    if (!rh.ok)
        return fail(ENOVA_EHIP, "radix select lost the order statistic");
    const int64_t n_greater = rh.n_greater;
    const uint32_t key_t = rh.prefix;
    const uint32_t bits = (key_t & 0x80000000u) ? (key_t & 0x7fffffffu) : ~key_t;
    float t_f;
    std::memcpy(&t_f, &bits, 4);
    if (!std::isfinite(t_f))
        return fail(ENOVA_ENUMERIC, "non-finite calibration score at the level quantile");
    // stable compaction of the excesses y = score - t of every calibration score above t; with
    // ten or more, their sum, minimum and maximum right behind it (one round trip for both)
    PotResult r{};
    const double t_d = static_cast<double>(t_f);
    double ps[3] = {0.0, 0.0, 0.0};
    if (n_greater > 0) {
        const int64_t nblk = calib_blocks(n_cal);
        if ((st = ensure(&det->peaks, &det->peaks_cap, static_cast<size_t>(n_greater))) != ENOVA_OK ||
            (st = ensure(&det->blk, &det->blk_cap, 2 * static_cast<size_t>(nblk) + 2)) != ENOVA_OK ||
            (st = ensure(&det->gx, &det->gx_cap, 4 + 3 * kPeakBlocks)) != ENOVA_OK)
            return st;
        int64_t *cnt = det->blk, *off = det->blk + nblk + 1;
        if ((e = launch_calib_count(scores, woff, det->cal, n, n_cal, key_t, cnt, stream)) != hipSuccess ||
            (e = launch_scan_i64(cnt, nblk, off, stream)) != hipSuccess ||
            (e = launch_calib_compact(scores, woff, det->cal, n, n_cal, key_t, t_d, off, det->peaks,
                                      n_greater, stream)) != hipSuccess)
            return hip_fail(e, "peak compaction");
        if (n_greater >= 10 && (e = launch_peak_stats(det->peaks, n_greater, det->gx, det->gx + 4, stream)) !=
                                   hipSuccess)
            return hip_fail(e, "peak statistics");
        int64_t total = 0;
        if ((e = hipMemcpyAsync(&total, off + nblk, sizeof(int64_t), hipMemcpyDeviceToHost, stream)) !=
                hipSuccess ||
            (n_greater >= 10 &&
             (e = hipMemcpyAsync(ps, det->gx, sizeof(ps), hipMemcpyDeviceToHost, stream)) != hipSuccess) ||
            (e = hipStreamSynchronize(stream)) != hipSuccess)
            return hip_fail(e, "peak count");
        if (total != n_greater)
            return fail(ENOVA_EHIP, "peak count mismatch (%lld vs %lld)", static_cast<long long>(total),
                        static_cast<long long>(n_greater));
    }
    if (n_greater >= 10) {
        if (!std::isfinite(ps[0]) || !std::isfinite(ps[2]))
            return fail(ENOVA_ENUMERIC, "non-finite calibration score");
        DeviceGpdSums ev(det, det->peaks, n_greater, stream);
        bool ok = false;
        r = pot_mle(t_d, n_cal, n_greater, ps[0], ps[1], ps[2], q, ev, &ok);
        if (!ok)
            return ev.status != ENOVA_OK ? ev.status : fail(ENOVA_ENUMERIC, "GPD fit failed");
    } else {
        double ex[16];
        if (n_greater > 0) {
            if ((e = hipMemcpyAsync(ex, det->peaks, sizeof(double) * n_greater, hipMemcpyDeviceToHost,
                                    stream)) != hipSuccess ||
                (e = hipStreamSynchronize(stream)) != hipSuccess)
                return hip_fail(e, "peak copy");
            for (int64_t i = 0; i < n_greater; ++i)
                if (!std::isfinite(ex[i]))
                    return fail(ENOVA_ENUMERIC, "non-finite calibration score");
            std::sort(ex, ex + n_greater);
        }
        r = pot_small(t_d, n_cal, ex, n_greater, q);
    }
    const float thr = static_cast<float>(r.z);
    *out_threshold = thr;
    if (out_info) {
        out_info[0] = r.t;
        out_info[1] = static_cast<double>(r.n);
        out_info[2] = static_cast<double>(r.n_peaks);
        out_info[3] = r.gamma;
        out_info[4] = r.sigma;
        out_info[5] = r.method;
    }
    if (out_flags) {
        e = launch_flag(scores, n_windows, thr, out_flags, stream);
        if (e != hipSuccess)
            return hip_fail(e, "flag kernel");
        if ((e = hipStreamSynchronize(stream)) != hipSuccess)
            return hip_fail(e, "flag kernel");
    }
    return ENOVA_OK;
}

enova_status enova_detect_set_timing(enova_detector det, int32_t enable)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    det->timing = enable != 0;
    return ENOVA_OK;
}

enova_status enova_detect_kernel_times(enova_detector det, double *score_ms, double *stats_ms)
{
    if (!det)
        return fail(ENOVA_EINVAL, "detector is NULL");
    DeviceGuard dg(det->device);
    float a = 0.0f, b = 0.0f;
    hipError_t e;
    if (det->timing && det->ran_score && det->ev[2]) {
        if ((e = hipEventSynchronize(det->ev[3])) != hipSuccess ||
            (e = hipEventElapsedTime(&a, det->ev[2], det->ev[3])) != hipSuccess)
            return hip_fail(e, "score kernel timing");
    }
    if (det->timing && det->ran_stats && det->ev[0]) {
        if ((e = hipEventSynchronize(det->ev[1])) != hipSuccess ||
            (e = hipEventElapsedTime(&b, det->ev[0], det->ev[1])) != hipSuccess)
            return hip_fail(e, "stats kernel timing");
    }
    if (score_ms)
        *score_ms = a;
    if (stats_ms)
        *stats_ms = b;
    return ENOVA_OK;
}

enova_status enova_detect_ext_mode(enova_detector det, int32_t *fused)
{
    if (!det || !fused)
        return fail(ENOVA_EINVAL, "NULL argument");
    *fused = det->wd2p ? 1 : 0;
    return ENOVA_OK;
}

enova_status enova_detect_kernel_kind(enova_detector det, int32_t *kind)
{
    if (!det || !kind)
        return fail(ENOVA_EINVAL, "NULL argument");
    *kind = det->kind;
    return ENOVA_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------------------------
// Streaming detection
// ---------------------------------------------------------------------------------------------
struct enova_stream_s {
    enova_detector det = nullptr;
    int n = 0;
    int64_t steps = 0;            // steps pushed so far (the same for every stream)
    double q = 1e-3;
    void *ring = nullptr;         // [n][2W][M]
    float *mean = nullptr, *std = nullptr;   // [n][M]
    float *scores = nullptr;      // [n] when the caller does not ask for scores
    SpotState spot{};
    hipEvent_t ev[3] = {nullptr, nullptr, nullptr};   // score start, score end / spot start, spot end
    bool timed = false;           // the last scoring push recorded ev
    // the threshold update and the refit run on the set's own stream (default priority), so a
    // push's refit overlaps the next push's append and scoring: the update waits for the push's
    // scores (score_ev), `stream` waits for the update (upd_ev: flags written, scores read), and
    // a state read waits for the refit (fit_ev)
    hipStream_t fit_stream = nullptr;
    hipEvent_t score_ev = nullptr, upd_ev = nullptr, fit_ev = nullptr;
    bool fit_pending = false;
};

namespace {

void free_stream(enova_stream s)
{
    if (!s)
        return;
    void *ptrs[] = {s->ring, s->mean, s->std, s->scores, s->spot.t, s->spot.z, s->spot.cnt,
                    s->spot.npk, s->spot.peaks, s->spot.mark, s->spot.err, s->spot.list,
                    s->spot.count};
    for (void *p : ptrs)
        if (p)
            (void)hipFree(p);
    for (hipEvent_t e : s->ev)
        if (e)
            (void)hipEventDestroy(e);
    if (s->score_ev)
        (void)hipEventDestroy(s->score_ev);
    if (s->upd_ev)
        (void)hipEventDestroy(s->upd_ev);
    if (s->fit_ev)
        (void)hipEventDestroy(s->fit_ev);
    if (s->fit_stream)
        (void)hipStreamDestroy(s->fit_stream);
    delete s;
}

template <typename T>
enova_status dev_alloc(T **dst, size_t count)
{
    hipError_t e = hipMalloc(reinterpret_cast<void **>(dst), std::max<size_t>(count, 1) * sizeof(T));
    if (e != hipSuccess) {
        *dst = nullptr;
        return fail(ENOVA_ENOMEM, "hipMalloc(%zu): %s", count * sizeof(T), hipGetErrorString(e));
    }
    return ENOVA_OK;
}

}  // namespace

extern "C" {

enova_status enova_stream_create(enova_detector det, int32_t n, const float *ref_mean, const float *ref_std,
                                 const float *calib_scores, const int64_t *calib_offsets, double level,
                                 double q, int32_t peak_cap, enova_stream *out, hipStream_t stream)
{
    if (!det || !ref_mean || !ref_std || !calib_offsets || !out)
        return fail(ENOVA_EINVAL, "NULL argument");
    *out = nullptr;
    if (n < 1)
        return fail(ENOVA_EINVAL, "n_streams must be >= 1");
    if (!(level > 0.0 && level < 1.0) || !(q > 0.0 && q < 1.0))
        return fail(ENOVA_EINVAL, "level and q must lie in (0, 1)");
    if (peak_cap < 1)
        return fail(ENOVA_EINVAL, "peak_cap must be >= 1");
    if (calib_offsets[0] != 0)
        return fail(ENOVA_EINVAL, "calib_offsets[0] must be 0");
    for (int32_t i = 0; i < n; ++i)
        if (calib_offsets[i + 1] < calib_offsets[i])
            return fail(ENOVA_EINVAL, "calib_offsets must be non-decreasing");
    const int64_t n_cal = calib_offsets[n];
    if (n_cal > 0 && !calib_scores)
        return fail(ENOVA_EINVAL, "calib_scores is NULL");
    const Geometry &g = det->g;
    if (det->kind != 2 || !det->w1s)
        return fail(ENOVA_EUNSUPPORTED, "streaming needs the matrix-core kernel's shapes");
    DeviceGuard dg(det->device);
    hipError_t e = hipSuccess;

    enova_stream s = new (std::nothrow) enova_stream_s;
    if (!s)
        return fail(ENOVA_ENOMEM, "host allocation");
    s->det = det;
    s->n = n;
    s->q = q;
    const size_t esz = g.dtype == ENOVA_F32 ? 4 : 2;
    const size_t nm = static_cast<size_t>(n) * g.M;
    enova_status st = ENOVA_OK;
    int64_t *d_off = nullptr;
    if ((st = dev_alloc(reinterpret_cast<unsigned char **>(&s->ring), nm * 2 * g.W * esz)) != ENOVA_OK ||
        (st = dev_alloc(&s->mean, nm)) != ENOVA_OK || (st = dev_alloc(&s->std, nm)) != ENOVA_OK ||
        (st = dev_alloc(&s->scores, n)) != ENOVA_OK || (st = dev_alloc(&s->spot.t, n)) != ENOVA_OK ||
        (st = dev_alloc(&s->spot.z, n)) != ENOVA_OK || (st = dev_alloc(&s->spot.cnt, n)) != ENOVA_OK ||
        (st = dev_alloc(&s->spot.npk, n)) != ENOVA_OK ||
        (st = dev_alloc(&s->spot.peaks, static_cast<size_t>(n) * peak_cap)) != ENOVA_OK ||
        (st = dev_alloc(&s->spot.mark, n)) != ENOVA_OK || (st = dev_alloc(&s->spot.err, 1)) != ENOVA_OK ||
        (st = dev_alloc(&s->spot.list, n)) != ENOVA_OK || (st = dev_alloc(&s->spot.count, 2)) != ENOVA_OK ||
        (st = dev_alloc(&d_off, static_cast<size_t>(n) + 1)) != ENOVA_OK) {
        (void)hipFree(d_off);
        free_stream(s);
        return st;
    }
    s->spot.cap = peak_cap;
    int err = 0;
    if ((e = hipMemsetAsync(s->ring, 0, nm * 2 * g.W * esz, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(s->mean, ref_mean, nm * sizeof(float), hipMemcpyDeviceToDevice, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(s->std, ref_std, nm * sizeof(float), hipMemcpyDeviceToDevice, stream)) != hipSuccess ||
        (e = hipMemsetAsync(s->spot.err, 0, sizeof(int), stream)) != hipSuccess ||
        (e = hipMemsetAsync(s->spot.count, 0, 2 * sizeof(int), stream)) != hipSuccess ||
        (e = hipMemcpyAsync(d_off, calib_offsets, (static_cast<size_t>(n) + 1) * sizeof(int64_t),
                            hipMemcpyHostToDevice, stream)) != hipSuccess ||
        (e = launch_spot_init(n_cal > 0 ? calib_scores : s->scores, d_off, n, level, s->spot, stream)) != hipSuccess ||
        (e = hipMemcpyAsync(&err, s->spot.err, sizeof(int), hipMemcpyDeviceToHost, stream)) != hipSuccess ||
        (e = hipStreamSynchronize(stream)) != hipSuccess) {
        (void)hipFree(d_off);
        free_stream(s);
        return hip_fail(e, "streaming set start");
    }
    (void)hipFree(d_off);
    if (err == 2) {
        free_stream(s);
        return fail(ENOVA_ENUMERIC, "non-finite calibration score");
    }
    if (err == 1) {
        free_stream(s);
        return fail(ENOVA_EINVAL, "a stream's calibration peaks exceed peak_cap");
    }
    if ((e = launch_spot_fit(n, q, s->spot, true, stream)) != hipSuccess || (e = hipStreamSynchronize(stream)) != hipSuccess) {
        free_stream(s);
        return hip_fail(e, "streaming threshold fit");
    }
    *out = s;
    return ENOVA_OK;
}

enova_status enova_stream_push(enova_stream s, const void *x_step, float *out_scores, float *out_md,
                               uint8_t *out_flags, int32_t *out_due, hipStream_t stream)
{
    if (!s || !x_step)
        return fail(ENOVA_EINVAL, "NULL argument");
    enova_detector det = s->det;
    const Geometry &g = det->g;
    DeviceGuard dg(det->device);
    hipError_t e = launch_stream_append(g, x_step, s->n, s->steps, s->ring, stream);
    if (e != hipSuccess)
        return hip_fail(e, "streaming append kernel");
    s->steps += 1;
    const bool due = s->steps >= g.W && (s->steps - g.W) % g.S == 0;
    if (out_due)
        *out_due = due ? 1 : 0;
    if (!due)
        return ENOVA_OK;
    StreamScoreParams p{};
    p.ring = s->ring;
    p.n_streams = s->n;
    p.first_slot = static_cast<int>(s->steps % g.W);
    p.mean = s->mean;
    p.std = s->std;
    p.w1p = det->w1s;
    p.whp = det->whs;
    p.wd1p = det->wds;
    p.b1 = det->b1;
    p.bd1 = det->bd1;
    p.u = det->u;
    p.bh = det->bh;
    p.sum_bd2 = det->sum_bd2;
    p.scores = out_scores ? out_scores : s->scores;
    p.md = out_md;
    const bool timed = det->timing;
    if (timed && !s->ev[0]) {
        for (hipEvent_t &ev : s->ev)
            if ((e = hipEventCreate(&ev)) != hipSuccess)
                return hip_fail(e, "timing events");
    }
    if (timed)
        (void)hipEventRecord(s->ev[0], stream);
    if ((e = launch_stream_score(g, p, stream)) != hipSuccess)
        return hip_fail(e, "streaming scoring kernel");
    if (timed)
        (void)hipEventRecord(s->ev[1], stream);
    if (!s->fit_stream) {
        if ((e = hipStreamCreateWithFlags(&s->fit_stream, hipStreamNonBlocking)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&s->score_ev, hipEventDisableTiming)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&s->upd_ev, hipEventDisableTiming)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&s->fit_ev, hipEventDisableTiming)) != hipSuccess)
            return hip_fail(e, "streaming refit stream");
    }
    // on the set's stream, behind the previous push's refit (whose thresholds it compares with,
    // and whose peaks, counts and list it rewrites): this push's update, then its refit, which
    // overlaps the next push's append and scoring on `stream`
    if ((e = hipEventRecord(s->score_ev, stream)) != hipSuccess ||
        (e = hipStreamWaitEvent(s->fit_stream, s->score_ev, 0)) != hipSuccess)
        return hip_fail(e, "streaming threshold order");
    s->spot.cur ^= 1;   // this push's list counter (cleared by the previous push's refit)
    if ((e = launch_spot_update(p.scores, s->n, s->spot, out_flags, s->fit_stream)) != hipSuccess)
        return hip_fail(e, "streaming threshold update");
    if ((e = hipEventRecord(s->upd_ev, s->fit_stream)) != hipSuccess ||
        (e = launch_spot_fit(s->n, s->q, s->spot, false, s->fit_stream)) != hipSuccess ||
        (e = hipEventRecord(s->fit_ev, s->fit_stream)) != hipSuccess)
        return hip_fail(e, "streaming refit");
    if (timed)
        (void)hipEventRecord(s->ev[2], s->fit_stream);
    // later work on `stream` sees this push's flags, and may overwrite the scores the update read
    if ((e = hipStreamWaitEvent(stream, s->upd_ev, 0)) != hipSuccess)
        return hip_fail(e, "streaming threshold order");
    s->fit_pending = true;
    s->timed = timed;
    return ENOVA_OK;
}

enova_status enova_stream_state(enova_stream s, double *t, double *z, int64_t *n, int32_t *n_peaks,
                                hipStream_t stream)
{
    if (!s)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(s->det->device);
    const size_t k = static_cast<size_t>(s->n);
    hipError_t e = hipSuccess;
    if (s->fit_pending && (e = hipStreamWaitEvent(stream, s->fit_ev, 0)) != hipSuccess)
        return hip_fail(e, "streaming refit wait");
    if ((t && (e = hipMemcpyAsync(t, s->spot.t, k * sizeof(double), hipMemcpyDeviceToHost, stream)) != hipSuccess) ||
        (z && (e = hipMemcpyAsync(z, s->spot.z, k * sizeof(double), hipMemcpyDeviceToHost, stream)) != hipSuccess) ||
        (n && (e = hipMemcpyAsync(n, s->spot.cnt, k * sizeof(int64_t), hipMemcpyDeviceToHost, stream)) != hipSuccess) ||
        (n_peaks && (e = hipMemcpyAsync(n_peaks, s->spot.npk, k * sizeof(int32_t), hipMemcpyDeviceToHost, stream)) != hipSuccess) ||
        (e = hipStreamSynchronize(stream)) != hipSuccess)
        return hip_fail(e, "streaming state copy");
    return ENOVA_OK;
}

enova_status enova_stream_kernel_times(enova_stream s, double *score_ms, double *spot_ms)
{
    if (!s)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(s->det->device);
    float a = 0.0f, b = 0.0f;
    hipError_t e;
    if (s->timed) {
        if ((e = hipEventSynchronize(s->ev[2])) != hipSuccess ||
            (e = hipEventElapsedTime(&a, s->ev[0], s->ev[1])) != hipSuccess ||
            (e = hipEventElapsedTime(&b, s->ev[1], s->ev[2])) != hipSuccess)
            return hip_fail(e, "streaming kernel timing");
    }
    if (score_ms)
        *score_ms = a;
    if (spot_ms)
        *spot_ms = b;
    return ENOVA_OK;
}

enova_status enova_stream_destroy(enova_stream s)
{
    if (!s)
        return ENOVA_OK;
    DeviceGuard dg(s->det->device);
    (void)hipDeviceSynchronize();
    free_stream(s);
    return ENOVA_OK;
}

}  // extern "C"
