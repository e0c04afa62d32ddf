// Launchers of the head kernels (see head.hip): gate logits, logit + isotonic
// calibration, log loss, the output-layer backward, gate-gradient finalisation
// and weighted column sums. bf16 storage; widths are multiples of 8.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rdcn {

struct CalArgs {
    int K;              // buckets
    float lo, step;
    const float* w;     // [K]
    const float* b;     // [1]
    const float* e;     // [B, K] per-sample embedding values
};

// s[b] = x[b, :] . g + c   (x [B, ldx] bf16, or f16 with x_f16; g [n] bf16, c [1] bf16)
hipError_t launch_gate_logit(int64_t B, int n, const void* x, bool x_f16, int64_t ldx, const void* g, const void* c,
                             float* s, hipStream_t st);
// y[b] = aL[b, :] . w_out + b_out (aL f16); y_cal[b] = calibrated y; y2 (optional) = second copy of y.
hipError_t launch_head_out(int64_t B, int n, const void* aL, const void* w_out, const void* b_out, const CalArgs& c,
                           float* y, float* y2, float* y_cal, hipStream_t st);
// loss[b] = softplus(z) - label z, grad[b] = (sigmoid(z) - label) * scale (either output may be NULL).
hipError_t launch_logloss(int64_t B, const float* z, const float* label, float scale, float* loss, float* grad,
                          hipStream_t st);
// From dLoss/dy_cal (aL f16): grad_e [B, K], gy [B] = dLoss/dy, the top layer's pre-activation
// gradient G [B, n] (bf16) and, when sL != NULL, its gate-logit gradient gs [B].
hipError_t launch_head_out_bwd(int64_t B, int n, const void* aL, const float* sL, const void* w_out, const float* y,
                               const CalArgs& c, const float* g_cal, float* grad_e, float* gy, void* G, float* gs,
                               hipStream_t st);
// gs[m] = (1 - sigmoid(s[m])) * sum over t < ntiles of part[t * B + m] (in t order).
hipError_t launch_gate_finalize(int64_t B, int ntiles, const float* part, const float* s, float* gs,
                                hipStream_t st);
// out[j] = sum over rows b (in row order within chunks, then chunk order) of X[b, j] * (wgt ? wgt[b] : 1),
// X float, bf16 or f16 (f16: n and ldx multiples of 8) with row stride ldx; `part` holds
// colsum_chunks(B) * n floats.
enum ColType { COL_F32 = 0, COL_BF16 = 1, COL_F16 = 2 };
int64_t colsum_chunks(int64_t B);
hipError_t launch_colsum_w(int64_t B, int64_t n, const void* X, int64_t ldx, ColType xt, const float* wgt,
                           float* part, float* out, hipStream_t st);

// out_i = sum over b < B of x_i[b] (float vectors), for up to VEC_SUMS_MAX vectors in one
// launch; each sum is taken in a fixed order (deterministic).
constexpr int VEC_SUMS_MAX = 16;
struct VecSums {
    int n;
    const float* x[VEC_SUMS_MAX];
    float* out[VEC_SUMS_MAX];
};
hipError_t launch_vec_sums(int64_t B, const VecSums& v, hipStream_t st);

}  // namespace rdcn
