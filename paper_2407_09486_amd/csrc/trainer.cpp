// Host side of the training entry points (Section IV-B, Eq. (9)): parameter, gradient and Adam
// buffers, the batch workspace, and the launch sequence of one ELBO step, replayed as a HIP graph.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <new>

#include "enova_detect.h"
#include "train_internal.h"

using namespace enova;

namespace {

// The parameters in the order of enova_detect_weights. In the flat buffers they are stored as
// w1, b1, wmu, wlv, bmu, blv, wd1, bd1, wd2, bd2, so that [wmu; wlv] ([2L][H]) and [bmu | blv]
// form the weights and biases of one fused head product.
enum { P_W1, P_B1, P_WMU, P_BMU, P_WLV, P_BLV, P_WD1, P_BD1, P_WD2, P_BD2, P_COUNT };
constexpr int kStoreOrder[P_COUNT] = {P_W1, P_B1, P_WMU, P_WLV, P_BMU, P_BLV, P_WD1, P_BD1, P_WD2, P_BD2};

}  // namespace

struct enova_trainer_s {
    int device = 0;
    int D = 0, H = 0, L = 0, act = 0;
    TrainHyper hyper{};
    int64_t off[P_COUNT] = {}, size[P_COUNT] = {}, total = 0;   // flat-buffer layout (floats)
    float *p = nullptr, *g = nullptr, *m = nullptr, *v = nullptr;
    float *state = nullptr;          // [0] PI integral, [1] beta of the step, [2..3] Adam bias corrections
    long long *step = nullptr;       // Adam step count, advanced on the device
    // batch workspace
    int cap = 0;
    float *a1 = nullptr, *h = nullptr, *a2 = nullptr, *hd = nullptr, *gh = nullptr;   // [B][H]
    float *ml = nullptr, *gml = nullptr;                                           // [B][2L]: [mu | lv]
    float *sd = nullptr, *z = nullptr, *gz = nullptr;                              // [B][L]
    float *out = nullptr;                                                          // [B][D]
    float *kl = nullptr, *logp = nullptr;                                          // [B]
    float *work = nullptr;                                                         // split-reduction partials
    int64_t work_cap = 0;
    // timing: an event pair around every product of the last step and around the whole step
    static constexpr int kMaxEvents = 2 * 16 + 2;
    bool timed = false;
    int n_events = 0;
    hipEvent_t ev[kMaxEvents] = {};
    // graph replay: the launches of one step, captured on the private stream `gstream` for one set of
    // step arguments and buffer generation, replayed while both stay the same
    bool use_graph = true;
    hipStream_t gstream = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    const void *key[4] = {};         // V, labels, eps, out_info of the captured step
    int key_batch = 0;
    uint64_t gen = 1, key_gen = 0;   // gen advances with every reallocation of a step buffer
};

namespace {

void free_trainer(enova_trainer t)
{
    if (!t)
        return;
    if (t->exec)
        (void)hipGraphExecDestroy(t->exec);
    if (t->graph)
        (void)hipGraphDestroy(t->graph);
    if (t->gstream)
        (void)hipStreamDestroy(t->gstream);
    void *ptrs[] = {t->p,  t->g,  t->m,  t->v,  t->state, t->step, t->a1,  t->h,  t->a2,   t->hd,
                    t->gh, t->ml, t->gml, t->sd, t->z,  t->gz,    t->out,  t->kl, t->logp, t->work};
    for (void *q : ptrs)
        if (q)
            (void)hipFree(q);
    for (hipEvent_t e : t->ev)
        if (e)
            (void)hipEventDestroy(e);
    delete t;
}

enova_status alloc_floats(float **dst, size_t n)
{
    hipError_t e = hipMalloc(reinterpret_cast<void **>(dst), std::max<size_t>(n, 1) * sizeof(float));
    if (e != hipSuccess) {
        *dst = nullptr;
        return fail(ENOVA_ENOMEM, "hipMalloc(%zu): %s", n * sizeof(float), hipGetErrorString(e));
    }
    return ENOVA_OK;
}

// Workspace of a step over B windows: the products whose slices are summed right away share the
// first train_gemm_workspace floats; each weight-gradient product, whose slices the Adam step sums,
// has a region of its own after them (off[1 + which], cap[1 + which]).
struct StepWork {
    int64_t off[1 + kTrainGradProducts], cap[1 + kTrainGradProducts], total;
};
StepWork step_work(const enova_trainer t, int B)
{
    StepWork w{};
    w.cap[0] = train_gemm_workspace(B, t->D, t->H, t->L);
    for (int q = 0; q < kTrainGradProducts; ++q)
        w.cap[1 + q] = train_grad_workspace(B, t->D, t->H, t->L, q);
    for (int q = 0; q <= kTrainGradProducts; ++q) {
        w.off[q] = w.total;
        w.total += w.cap[q];
    }
    return w;
}

int64_t workspace_floats(const enova_trainer t, int B)
{
    return step_work(t, B).total;
}

// Grows the batch buffers to B rows (freeing the old ones synchronises the device).
enova_status ensure_batch(enova_trainer t, int B)
{
    enova_status st;
    const int64_t ws = workspace_floats(t, B);
    if (ws > t->work_cap) {
        ++t->gen;
        (void)hipFree(t->work);
        t->work = nullptr;
        t->work_cap = 0;
        if ((st = alloc_floats(&t->work, static_cast<size_t>(ws))) != ENOVA_OK)
            return st;
        t->work_cap = ws;
    }
    if (B <= t->cap)
        return ENOVA_OK;
    ++t->gen;
    float **bh[] = {&t->a1, &t->h, &t->a2, &t->hd, &t->gh};
    float **bl[] = {&t->sd, &t->z, &t->gz};
    float **b2[] = {&t->ml, &t->gml};
    float **b1[] = {&t->kl, &t->logp};
    for (float **q : bh)
        (void)hipFree(*q), *q = nullptr;
    for (float **q : bl)
        (void)hipFree(*q), *q = nullptr;
    for (float **q : b2)
        (void)hipFree(*q), *q = nullptr;
    for (float **q : b1)
        (void)hipFree(*q), *q = nullptr;
    (void)hipFree(t->out);
    t->out = nullptr;
    t->cap = 0;
    for (float **q : bh)
        if ((st = alloc_floats(q, static_cast<size_t>(B) * t->H)) != ENOVA_OK)
            return st;
    for (float **q : bl)
        if ((st = alloc_floats(q, static_cast<size_t>(B) * t->L)) != ENOVA_OK)
            return st;
    for (float **q : b2)
        if ((st = alloc_floats(q, static_cast<size_t>(B) * 2 * t->L)) != ENOVA_OK)
            return st;
    for (float **q : b1)
        if ((st = alloc_floats(q, static_cast<size_t>(B))) != ENOVA_OK)
            return st;
    if ((st = alloc_floats(&t->out, static_cast<size_t>(B) * t->D)) != ENOVA_OK)
        return st;
    t->cap = B;
    return ENOVA_OK;
}

enova_status copy_out(enova_trainer t, const float *src, const enova_train_params *out, hipStream_t stream)
{
    float *dst[P_COUNT] = {out->w1, out->b1, out->wmu, out->bmu, out->wlv, out->blv, out->wd1, out->bd1,
                           out->wd2, out->bd2};
    hipError_t e = hipSuccess;
    for (int k = 0; k < P_COUNT && e == hipSuccess; ++k)
        if (dst[k])
            e = hipMemcpyAsync(dst[k], src + t->off[k], t->size[k] * sizeof(float), hipMemcpyDeviceToHost,
                               stream);
    if (e == hipSuccess)
        e = hipStreamSynchronize(stream);
    return e == hipSuccess ? ENOVA_OK : hip_fail(e, "trainer copy");
}

}  // namespace

extern "C" {

enova_status enova_train_init(const enova_train_config *c, const enova_detect_weights *w, enova_trainer *out)
{
    if (!c || !w || !out)
        return fail(ENOVA_EINVAL, "NULL argument");
    *out = nullptr;
    if (c->inputs < 1 || c->hidden < 1 || c->latent < 1 || (c->act != ENOVA_RELU && c->act != ENOVA_TANH))
        return fail(ENOVA_EINVAL, "bad trainer shape");
    if (!(c->lr > 0.0f) || !(c->adam_b1 >= 0.0f && c->adam_b1 < 1.0f) || !(c->adam_b2 >= 0.0f && c->adam_b2 < 1.0f) ||
        !(c->adam_eps > 0.0f) || !(c->beta_min <= c->beta_max) || !(c->anomaly_margin > 0.0f))
        return fail(ENOVA_EINVAL, "bad trainer hyper-parameters");
    const void *src[P_COUNT] = {w->w1, w->b1, w->wmu, w->bmu, w->wlv, w->blv, w->wd1, w->bd1, w->wd2, w->bd2};
    for (const void *q : src)
        if (!q)
            return fail(ENOVA_EINVAL, "NULL weight array");
    enova_trainer t = new (std::nothrow) enova_trainer_s;
    if (!t)
        return fail(ENOVA_ENOMEM, "host allocation");
    if (hipGetDevice(&t->device) != hipSuccess) {
        delete t;
        return fail(ENOVA_EHIP, "no current HIP device");
    }
    t->D = c->inputs;
    t->H = c->hidden;
    t->L = c->latent;
    t->act = c->act;
    t->hyper = TrainHyper{c->lr,     c->adam_b1,  c->adam_b2,  c->adam_eps,       c->kl_set,
                          c->kp,     c->ki,       c->beta_min, c->beta_max, c->anomaly_margin};
    const int64_t D = t->D, H = t->H, L = t->L;
    const int64_t sizes[P_COUNT] = {H * D, H, L * H, L, L * H, L, H * L, H, D * H, D};
    for (int q : kStoreOrder) {
        t->off[q] = t->total;
        t->size[q] = sizes[q];
        t->total += sizes[q];
    }
    const size_t total = static_cast<size_t>(t->total);
    enova_status st;
    if ((st = alloc_floats(&t->p, total)) != ENOVA_OK || (st = alloc_floats(&t->g, total)) != ENOVA_OK ||
        (st = alloc_floats(&t->m, total)) != ENOVA_OK || (st = alloc_floats(&t->v, total)) != ENOVA_OK ||
        (st = alloc_floats(&t->state, 4)) != ENOVA_OK) {
        free_trainer(t);
        return st;
    }
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&t->step), sizeof(long long));
    if (e != hipSuccess) {
        t->step = nullptr;
        free_trainer(t);
        return fail(ENOVA_ENOMEM, "hipMalloc(step count): %s", hipGetErrorString(e));
    }
    for (int k = 0; k < P_COUNT && e == hipSuccess; ++k)
        e = hipMemcpy(t->p + t->off[k], src[k], sizes[k] * sizeof(float), hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemset(t->m, 0, total * sizeof(float));
    if (e == hipSuccess)
        e = hipMemset(t->v, 0, total * sizeof(float));
    if (e == hipSuccess)
        e = hipMemset(t->g, 0, total * sizeof(float));
    if (e == hipSuccess)
        e = hipMemset(t->state, 0, 4 * sizeof(float));
    if (e == hipSuccess)
        e = hipMemset(t->step, 0, sizeof(long long));
    if (e == hipSuccess)
        e = hipStreamCreateWithFlags(&t->gstream, hipStreamNonBlocking);
    if (e != hipSuccess) {
        free_trainer(t);
        return hip_fail(e, "trainer upload");
    }
    *out = t;
    return ENOVA_OK;
}

}  // extern "C"

namespace {

// The launches of one step on stream s (events around the products when timing is on).
hipError_t enqueue_step(enova_trainer t, const float *V, const float *labels, const float *eps, int B,
                        float *info, hipStream_t s)
{
    const int D = t->D, H = t->H, L = t->L, act = t->act;
    float *P = t->p, *G = t->g;
    const int64_t *o = t->off;
    hipError_t e = hipSuccess;
    auto run = [&](hipError_t r) {
        if (e == hipSuccess)
            e = r;
    };
    int ne = 0;
    auto mark = [&]() {
        if (t->timed && ne < enova_trainer_s::kMaxEvents)
            run(hipEventRecord(t->ev[ne++], s));
    };
    // every product of the step; with timing on, its product kernel is bracketed by two events.
    // A weight-gradient product (grad = which, train_grad_shape) splits into its own workspace
    // region and leaves the slices to the Adam step.
    const StepWork wk = step_work(t, B);
    GradSums sums;
    auto gemm = [&](const GemmEpilogue &ep, const float *A, int64_t ai, int64_t ak, const float *Bm, int64_t bk,
                    int64_t bj, float *C, int64_t ldc, int m, int n, int k, float *rowsum, int grad = -1) {
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (t->timed && ne + 2 < enova_trainer_s::kMaxEvents) {
            e0 = t->ev[ne++];
            e1 = t->ev[ne++];
        }
        const int r = grad < 0 ? 0 : 1 + grad;
        GemmSplit sp;
        run(launch_gemm(ep, A, ai, ak, Bm, bk, bj, C, ldc, m, n, k, rowsum, t->work + wk.off[r], wk.cap[r], s, e0,
                        e1, grad < 0 ? nullptr : &sp));
        if (sp.splits > 0) {
            if (sums.n + 2 > kMaxGradSums) {
                run(hipErrorInvalidValue);
                return;
            }
            const int64_t mn = static_cast<int64_t>(m) * n;
            sums.s[sums.n++] = GradSum{C - G, mn, sp.part, mn, sp.splits};
            if (rowsum)
                sums.s[sums.n++] = GradSum{rowsum - G, m, sp.rows, m, sp.splits};
        }
    };
    const GemmEpilogue plain{};
    auto bias_act = [&](const float *bias, float *out) {
        GemmEpilogue ep;
        ep.kind = kEpiBiasAct;
        ep.act = act;
        ep.bias = bias;
        ep.out2 = out;
        return ep;
    };
    auto dact = [&](const float *pre) {
        GemmEpilogue ep;
        ep.kind = kEpiDact;
        ep.act = act;
        ep.pre = pre;
        return ep;
    };
    mark();
    // forward: a1 = V W1^T + b1, h = act(a1)
    gemm(bias_act(P + o[P_B1], t->h), V, D, 1, P + o[P_W1], 1, D, t->a1, H, B, H, D, nullptr);
    // fused heads [mu | lv] = h [Wmu; Wlv]^T, reparameterised latent and KL
    gemm(plain, t->h, H, 1, P + o[P_WMU], 1, H, t->ml, 2 * L, B, 2 * L, H, nullptr);
    run(launch_latent(t->ml, P + o[P_BMU], eps, t->sd, t->z, t->kl, B, L, s));
    // decoder: a2 = z Wd1^T + bd1, hd = act(a2), m' = hd Wd2^T (+ bd2) -> log p and dJ/dm'
    gemm(bias_act(P + o[P_BD1], t->hd), t->z, L, 1, P + o[P_WD1], 1, L, t->a2, H, B, H, L, nullptr);
    gemm(plain, t->hd, H, 1, P + o[P_WD2], 1, H, t->out, D, B, D, H, nullptr);
    run(launch_recon(t->out, P + o[P_BD2], V, labels, t->logp, B, D, t->hyper.margin, s));
    // beta(k) from this batch's KL, before the backward pass; the Adam step count and corrections
    run(launch_beta(t->kl, t->logp, labels, B, D, t->hyper, t->state, t->state + 1, info, t->step, t->state + 2,
                    s));
    // backward through the decoder (G = dJ/dm' in out); bias gradients are the row sums of G^T
    gemm(plain, t->out, 1, D, t->hd, H, 1, G + o[P_WD2], H, D, H, B, G + o[P_BD2], 0);    // dWd2 = G^T hd
    gemm(dact(t->a2), t->out, D, 1, P + o[P_WD2], H, 1, t->gh, H, B, H, D, nullptr);      // dJ/da2
    gemm(plain, t->gh, 1, H, t->z, L, 1, G + o[P_WD1], L, H, L, B, G + o[P_BD1], 1);      // dWd1 = G^T z
    gemm(plain, t->gh, H, 1, P + o[P_WD1], L, 1, t->gz, L, B, L, H, nullptr);             // dJ/dz = G Wd1
    // latent: [dJ/dmu | dJ/dlv], then the fused heads' gradients and dJ/da1 = (G_ml [Wmu; Wlv]) act'(a1)
    run(launch_latent_grad(t->gz, t->gml, t->ml, t->sd, eps, labels, t->state + 1, B, L, s));
    gemm(plain, t->gml, 1, 2 * L, t->h, H, 1, G + o[P_WMU], H, 2 * L, H, B, G + o[P_BMU], 2);
    gemm(dact(t->a1), t->gml, 2 * L, 1, P + o[P_WMU], H, 1, t->gh, H, B, H, 2 * L, nullptr);
    gemm(plain, t->gh, 1, H, V, D, 1, G + o[P_W1], D, H, D, B, G + o[P_B1], 3);            // dW1 = G^T V
    // Adam, forming the split weight gradients from their slices first
    run(launch_adam(P, G, t->m, t->v, t->total, t->hyper, t->state + 2, sums, s));
    mark();
    t->n_events = ne;
    return e;
}

// Free the captured graph; a replay of it may still be in flight, so the device is drained first.
void drop_graph(enova_trainer t)
{
    if (t->exec) {
        (void)hipDeviceSynchronize();
        (void)hipGraphExecDestroy(t->exec);
    }
    if (t->graph)
        (void)hipGraphDestroy(t->graph);
    t->exec = nullptr;
    t->graph = nullptr;
    t->key_gen = 0;
}

// Capture the step's launches on the private stream (nothing runs while capturing) and
// instantiate them; on any failure no graph is kept.
hipError_t capture_step(enova_trainer t, const float *V, const float *labels, const float *eps, int B, float *info)
{
    drop_graph(t);
    hipError_t e = hipStreamBeginCapture(t->gstream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess)
        return e;
    const hipError_t le = enqueue_step(t, V, labels, eps, B, info, t->gstream);
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(t->gstream, &g);
    if (le != hipSuccess || e != hipSuccess) {
        if (g)
            (void)hipGraphDestroy(g);
        return le != hipSuccess ? le : e;
    }
    hipGraphExec_t x = nullptr;
    if ((e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0)) != hipSuccess) {
        (void)hipGraphDestroy(g);
        return e;
    }
    t->graph = g;
    t->exec = x;
    t->key[0] = V;
    t->key[1] = labels;
    t->key[2] = eps;
    t->key[3] = info;
    t->key_batch = B;
    t->key_gen = t->gen;
    return hipSuccess;
}

}  // namespace

extern "C" {

enova_status enova_train_step(enova_trainer t, const float *V, const float *labels, const float *eps,
                              int32_t B, float *info, hipStream_t s)
{
    if (!t || !V || !labels || !eps)
        return fail(ENOVA_EINVAL, "NULL argument");
    if (B < 1)
        return fail(ENOVA_EINVAL, "batch must be >= 1");
    DeviceGuard dg(t->device);
    enova_status st = ensure_batch(t, B);
    if (st != ENOVA_OK)
        return st;
    if (t->timed || !t->use_graph) {
        const hipError_t e = enqueue_step(t, V, labels, eps, B, info, s);
        return e == hipSuccess ? ENOVA_OK : hip_fail(e, "training kernels");
    }
    t->n_events = 0;
    const bool same = t->exec && t->key_gen == t->gen && t->key_batch == B && t->key[0] == V &&
                      t->key[1] == labels && t->key[2] == eps && t->key[3] == info;
    if (!same) {
        const hipError_t e = capture_step(t, V, labels, eps, B, info);
        if (e != hipSuccess)
            return hip_fail(e, "capturing the training step");
    }
    const hipError_t e = hipGraphLaunch(t->exec, s);
    return e == hipSuccess ? ENOVA_OK : hip_fail(e, "hipGraphLaunch");
}

enova_status enova_train_params_get(enova_trainer t, const enova_train_params *out, hipStream_t stream)
{
    if (!t || !out)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(t->device);
    return copy_out(t, t->p, out, stream);
}

enova_status enova_train_grads_get(enova_trainer t, const enova_train_params *out, hipStream_t stream)
{
    if (!t || !out)
        return fail(ENOVA_EINVAL, "NULL argument");
    DeviceGuard dg(t->device);
    return copy_out(t, t->g, out, stream);
}

enova_status enova_train_set_graph(enova_trainer t, int32_t enable)
{
    if (!t)
        return fail(ENOVA_EINVAL, "NULL trainer");
    DeviceGuard dg(t->device);
    t->use_graph = enable != 0;
    if (!t->use_graph)
        drop_graph(t);
    return ENOVA_OK;
}

enova_status enova_train_set_timing(enova_trainer t, int32_t enable)
{
    if (!t)
        return fail(ENOVA_EINVAL, "NULL trainer");
    DeviceGuard dg(t->device);
    if (enable && !t->ev[0]) {
        for (hipEvent_t &e : t->ev) {
            hipError_t r = hipEventCreate(&e);
            if (r != hipSuccess)
                return hip_fail(r, "hipEventCreate");
        }
    }
    t->timed = enable != 0;
    t->n_events = 0;
    return ENOVA_OK;
}

enova_status enova_train_kernel_times(enova_trainer t, double *gemm_ms, double *step_ms)
{
    if (!t || !gemm_ms || !step_ms)
        return fail(ENOVA_EINVAL, "NULL argument");
    *gemm_ms = *step_ms = 0.0;
    const int ne = t->n_events;
    if (ne < 2)
        return ENOVA_OK;
    DeviceGuard dg(t->device);
    hipError_t r = hipEventSynchronize(t->ev[ne - 1]);
    if (r != hipSuccess)
        return hip_fail(r, "hipEventSynchronize");
    // events: [step start] (gemm start, gemm end)* [step end]
    double g = 0.0;
    for (int i = 1; i + 1 <= ne - 2; i += 2) {
        float ms = 0.0f;
        if ((r = hipEventElapsedTime(&ms, t->ev[i], t->ev[i + 1])) != hipSuccess)
            return hip_fail(r, "hipEventElapsedTime");
        g += ms;
    }
    float all = 0.0f;
    if ((r = hipEventElapsedTime(&all, t->ev[0], t->ev[ne - 1])) != hipSuccess)
        return hip_fail(r, "hipEventElapsedTime");
    *gemm_ms = g;
    *step_ms = all;
    return ENOVA_OK;
}

enova_status enova_train_destroy(enova_trainer t)
{
    if (!t)
        return ENOVA_OK;
    DeviceGuard dg(t->device);
    (void)hipDeviceSynchronize();
    free_trainer(t);
    return ENOVA_OK;
}

}  // extern "C"
