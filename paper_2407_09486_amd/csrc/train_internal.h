// Internal declarations of the training step (matrix-core products and element-wise kernels).
#pragma once

#include "gemm_plan.h"
#include "internal.h"

namespace enova {

// ---------------------------------------------------------------------------------------------
// Training (fp32): C(i, j) [+]= sum_k A(i, k) B(k, j), A(i, k) = A[i*ai + k*ak],
// B(k, j) = B[k*bk + j*bj], C(i, j) = C[i*ldc + j]; and the element-wise steps around it.
// ---------------------------------------------------------------------------------------------
struct TrainHyper {
    float lr, b1, b2, eps;
    float kl_set, kp, ki, beta_min, beta_max;
    float margin;   // cap of an anomalous window's reconstruction error (+inf: none)
};
// A long reduction over few output tiles is split into slices whose partial tiles go to `work`
// (gemm_workspace_floats(m, n, k) floats, gemm_plan.h; NULL: no split) and are then summed in slice order.
// rowsum (or NULL) receives sum_k A(i, k) for every i < m. The epilogue fuses the element-wise
// step that follows a product: store; C = product + bias[j] with out2 = act(C); or
// C = product * act'(pre) (pre in C's layout).
// kEpiRowReduce writes no C: with d(i, j) = pre[i*ldv + j] - (product + bias[j]) and column j
// belonging to group j mod groups (groups a power of two <= 32), it writes for every row i and
// column slot s (gemm_reduce_slots(m, n) slots of consecutive columns)
//   out2[(i*slots + s)*groups + c] = sum of d over the slot's columns of group c,
//   sq[i*slots + s]                = sum of d^2 over the slot's columns;
// such a product is never split.
enum { kEpiStore = 0, kEpiBiasAct = 1, kEpiDact = 2, kEpiRowReduce = 3 };
struct GemmEpilogue {
    int kind = kEpiStore;
    int act = ENOVA_RELU;
    const float *bias = nullptr;
    float *out2 = nullptr;
    const float *pre = nullptr;
    float *sq = nullptr;    // kEpiRowReduce
    int ldv = 0;            // kEpiRowReduce: leading dimension of pre
    int groups = 0;         // kEpiRowReduce
};
// A split product's slice partials left for a later pass: part [splits][m][n] and rows
// [splits][m] (NULL without row sums), in `work`; splits == 0 when the product did not split and
// C (and rowsum) already hold the result.
struct GemmSplit {
    const float *part = nullptr, *rows = nullptr;
    int splits = 0;
};
// ev0 / ev1 (or NULL) are recorded around the product kernel itself (not the slice sum).
// `work` holds work_floats floats; a product splits only as far as they allow (none when work is
// NULL). With `defer` (a plain store into C with ldc == n only) a split product's slices are not
// summed: *defer describes them, and C and rowsum are left untouched.
hipError_t launch_gemm(const GemmEpilogue &epi, const float *A, int64_t ai, int64_t ak, const float *B, int64_t bk,
                       int64_t bj, float *C, int64_t ldc, int m, int n, int k, float *rowsum, float *work,
                       int64_t work_floats, hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr,
                       GemmSplit *defer = nullptr);
// ml: [rows][2L] = [mu | lv] per window (biases bml = [bmu | blv] added in place).
hipError_t launch_latent(float *ml, const float *bml, const float *eps, float *sd, float *z, float *kl, int rows,
                         int L, hipStream_t st);
hipError_t launch_recon(float *out, const float *bd2, const float *V, const float *labels, float *logp,
                        int rows, int D, float margin, hipStream_t st);
// state[0] = the controller's integral term, beta = this step's KL weight; step = the Adam step
// count (advanced here), corr [2] = its bias corrections for launch_adam.
hipError_t launch_beta(const float *kl, const float *logp, const float *labels, int rows, int D,
                       const TrainHyper &h, float *state, float *beta, float *info, long long *step, float *corr,
                       hipStream_t st);
// gz: [rows][L] = dJ/dz; gml: [rows][2L] = [dJ/dmu | dJ/dlv].
hipError_t launch_latent_grad(const float *gz, float *gml, const float *ml, const float *sd, const float *eps,
                              const float *labels, const float *beta, int rows, int L, hipStream_t st);
// The gradient of the flat range [begin, begin + count) as the sum of a deferred product's slices:
// g[begin + i] = sum over s = 0, 1, ..., splits - 1 (in order) of src[s * stride + i].
struct GradSum {
    int64_t begin, count;
    const float *src;
    int64_t stride;
    int splits;
};
constexpr int kMaxGradSums = 2 * kTrainGradProducts;   // a weight and a bias range per product
struct GradSums {
    int n = 0;
    GradSum s[kMaxGradSums] = {};
};
// One Adam step over the flat parameters; the ranges in `sums` first form their gradient from the
// slices (and store it in g), every other entry of g is read as it is.
hipError_t launch_adam(float *p, float *g, float *m, float *v, int64_t total, const TrainHyper &h,
                       const float *corr, const GradSums &sums, hipStream_t st);

}  // namespace enova
