// Head kernels for gfx950: the layers after the cross stack (section "Dense
// Gating and Large MLP") up to the calibrated logit (section "Isotonic
// Calibration Layer", equation (calibration)) and its log loss.
//
// The MLP layers themselves are GEMMs with fused epilogues (gemm.hip,
// EPI_MLP_FWD / EPI_MLP_BWD); this file holds the row-wise and column-wise work
// around them. Every row-wise kernel gives one sample to one 64-lane wave and
// reads its row with 16-byte loads; reductions across lanes are xor-butterflies
// in a fixed order, so every result is deterministic.
//
// Calibration: t = y - lo; the bucket k is the number of bounds step*j
// (j = 1 .. K-1, each rounded to float) that t exceeds, i.e. the largest j with
// t - step*j > 0 (or 0); v_i = step below k, t - step*k at k; and
// y_cal = b + sum_{i <= k} ReLU(e_i + w_i) v_i. Below lo and above lo + K*step
// the first and last buckets extend linearly.
#include "device_common.h"
#include "head.h"
#include "mlp_common.h"

namespace rdcn {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ void ld8(const bf16_t* p, float* v) { st<bf16_t>::unpack(*(const u32x4_t*)p, v); }
__device__ __forceinline__ void ld8(const _Float16* p, float* v) { unpack_f16x8(*(const u32x4_t*)p, v); }
__device__ __forceinline__ void ld8(const float* p, float* v) {
    st<float>::unpack(*(const u32x4_t*)p, v);
    st<float>::unpack(*(const u32x4_t*)(p + 4), v + 4);
}

// Bucket index of t: the count of bounds step*j (j = 1 .. K-1) below t, over the wave.
__device__ __forceinline__ int bucket_of(float t, float step, int K, int lane) {
    int cnt = 0;
    for (int j = 1 + lane; j < K; j += 64) cnt += t > step * (float)j ? 1 : 0;
    return wave_sum_i(cnt);
}

constexpr int ROWS_PER_BLOCK = 4;  // one wave per row, 256 threads

inline unsigned row_blocks(int64_t B) {
    int64_t b = (B + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK;
    if (b > 16384) b = 16384;
    return (unsigned)(b > 0 ? b : 1);
}

template <typename TX>
__global__ __launch_bounds__(256) void k_gate_logit(int64_t B, int n, const TX* __restrict__ x, int64_t ldx,
                                                    const bf16_t* __restrict__ g, const bf16_t* __restrict__ c,
                                                    float* __restrict__ s) {
    const int lane = threadIdx.x & 63;
    const float cb = bf16_to_f32(*c);
    for (int64_t row = (int64_t)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6); row < B;
         row += (int64_t)gridDim.x * ROWS_PER_BLOCK) {
        const TX* xr = x + row * ldx;
        float acc = 0.f;
        for (int col = lane * 8; col < n; col += 512) {
            float xv[8], gv[8];
            ld8(xr + col, xv);
            ld8(g + col, gv);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc = fmaf(xv[e], gv[e], acc);
        }
        acc = wave_sum(acc);
        if (lane == 0) s[row] = acc + cb;
    }
}

template <typename TA>
__global__ __launch_bounds__(256) void k_head_out(int64_t B, int n, const TA* __restrict__ aL,
                                                  const bf16_t* __restrict__ w_out, const bf16_t* __restrict__ b_out,
                                                  CalArgs c, float* __restrict__ y, float* __restrict__ y2,
                                                  float* __restrict__ y_cal) {
    const int lane = threadIdx.x & 63;
    const float bo = bf16_to_f32(*b_out), cb = *c.b;
    for (int64_t row = (int64_t)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6); row < B;
         row += (int64_t)gridDim.x * ROWS_PER_BLOCK) {
        const TA* ar = aL + row * n;
        float acc = 0.f;
        for (int col = lane * 8; col < n; col += 512) {
            float av[8], wv[8];
            ld8(ar + col, av);
            ld8(w_out + col, wv);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc = fmaf(av[e], wv[e], acc);
        }
        const float yv = wave_sum(acc) + bo;
        const float t = yv - c.lo;
        const int k = bucket_of(t, c.step, c.K, lane);
        const float vk = t - c.step * (float)k;
        const float* er = c.e + row * c.K;
        float cal = 0.f;
        for (int i = lane; i <= k; i += 64) cal = fmaf(relu_f(er[i] + c.w[i]), i < k ? c.step : vk, cal);
        cal = wave_sum(cal);
        if (lane == 0) {
            y[row] = yv;
            if (y2) y2[row] = yv;
            y_cal[row] = cb + cal;
        }
    }
}

__global__ __launch_bounds__(256) void k_logloss(int64_t B, const float* __restrict__ z,
                                                 const float* __restrict__ label, float scale,
                                                 float* __restrict__ loss, float* __restrict__ grad) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < B; i += (int64_t)gridDim.x * 256) {
        const float zv = z[i], lv = label[i];
        if (loss) loss[i] = fmaxf(zv, 0.f) + log1pf(expf(-fabsf(zv))) - lv * zv;
        if (grad) grad[i] = (sigmoid_f(zv) - lv) * scale;
    }
}

template <typename TA>
__global__ __launch_bounds__(256) void k_head_out_bwd(int64_t B, int n, const TA* __restrict__ aL,
                                                      const float* __restrict__ sL,
                                                      const bf16_t* __restrict__ w_out, const float* __restrict__ y,
                                                      CalArgs c, const float* __restrict__ g_cal,
                                                      float* __restrict__ grad_e, float* __restrict__ gy_out,
                                                      bf16_t* __restrict__ G, float* __restrict__ gs) {
    const int lane = threadIdx.x & 63;
    for (int64_t row = (int64_t)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6); row < B;
         row += (int64_t)gridDim.x * ROWS_PER_BLOCK) {
        const float t = y[row] - c.lo;
        const int k = bucket_of(t, c.step, c.K, lane);
        const float vk = t - c.step * (float)k;
        const float gc = g_cal[row];
        const float* er = c.e + row * c.K;
        float* ge = grad_e + row * c.K;
        for (int i = lane; i < c.K; i += 64) {
            const float v = i < k ? c.step : (i == k ? vk : 0.f);
            ge[i] = er[i] + c.w[i] > 0.f ? gc * v : 0.f;
        }
        const float gy = gc * relu_f(er[k] + c.w[k]);
        const float rho = sL ? sigmoid_f(sL[row]) : 1.f;
        const TA* ar = aL + row * n;
        bf16_t* gr = G + row * n;
        float dot = 0.f;
        for (int col = lane * 8; col < n; col += 512) {
            float av[8], wv[8], o[8];
            ld8(ar + col, av);
            ld8(w_out + col, wv);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float ga = gy * wv[e];
                dot = fmaf(ga, av[e], dot);
                o[e] = av[e] > 0.f ? rho * ga : 0.f;
            }
            *(u32x4_t*)(gr + col) = st<bf16_t>::pack(o);
        }
        dot = wave_sum(dot);
        if (lane == 0) {
            gy_out[row] = gy;
            if (sL) gs[row] = (1.f - rho) * dot;
        }
    }
}

__global__ __launch_bounds__(256) void k_gate_finalize(int64_t B, int ntiles, const float* __restrict__ part,
                                                       const float* __restrict__ s, float* __restrict__ gs) {
    for (int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x; m < B; m += (int64_t)gridDim.x * 256) {
        float acc = 0.f;
#pragma unroll 8
        for (int t = 0; t < ntiles; ++t) acc += part[(int64_t)t * B + m];
        gs[m] = (1.f - sigmoid_f(s[m])) * acc;
    }
}

constexpr int COLSUM_ROWS = 64;  // rows per chunk (16 per wave)

// part[chunk, j] = sum over the chunk's rows of X[b, j] * wgt[b]. A block of four
// waves covers 64 * VEC columns (VEC = 8: 16-byte loads); wave w takes rows
// w, w + 4, ... of the chunk, and the four wave sums are added in wave order.
template <typename T, int VEC>
__global__ __launch_bounds__(256) void k_colsum_w(int64_t B, int64_t n, const T* __restrict__ X, int64_t ldx,
                                                  const float* __restrict__ wgt, float* __restrict__ part) {
    __shared__ float red[4][64 * VEC];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t j = ((int64_t)blockIdx.x * 64 + lane) * VEC;
    const int64_t b0 = (int64_t)blockIdx.y * COLSUM_ROWS;
    const int64_t b1 = b0 + COLSUM_ROWS < B ? b0 + COLSUM_ROWS : B;
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    if (j < n) {
        // unrolled so that four rows' loads are in flight together (the sums stay in row order)
#pragma unroll 4
        for (int64_t b = b0 + wave; b < b1; b += 4) {
            const float wv = wgt ? wgt[b] : 1.f;
            float v[VEC];
            if constexpr (VEC == 8) {
                ld8(X + b * ldx + j, v);
            } else {
                v[0] = st<T>::load(X + b * ldx + j);
            }
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] = fmaf(v[e], wv, acc[e]);
        }
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) red[wave][lane * VEC + e] = acc[e];
    __syncthreads();
    if (wave == 0 && j < n) {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            part[(int64_t)blockIdx.y * n + j + e] =
                ((red[0][lane * VEC + e] + red[1][lane * VEC + e]) + red[2][lane * VEC + e]) + red[3][lane * VEC + e];
    }
}

// out[j] = sum over chunks of part[chunk, j]: four slices of the chunks summed in
// order, then the slices in order.
__global__ __launch_bounds__(256) void k_chunk_reduce(int64_t nchunks, int64_t n, const float* __restrict__ part,
                                                      float* __restrict__ out) {
    __shared__ float red[4][64];
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 64 + tx;
    float acc = 0.f;
    if (j < n)
#pragma unroll 4
        for (int64_t c = ty; c < nchunks; c += 4) acc += part[c * n + j];
    red[ty][tx] = acc;
    __syncthreads();
    if (ty == 0 && j < n) out[j] = ((red[0][tx] + red[1][tx]) + red[2][tx]) + red[3][tx];
}

// One block per vector: 256 threads take rows t, t + 256, ...; the thread sums are
// added in a fixed tree order.
__global__ __launch_bounds__(256) void k_vec_sums(int64_t B, VecSums v) {
    __shared__ float red[256];
    const int i = blockIdx.x, t = threadIdx.x;
    const float* x = v.x[i];
    float acc = 0.f;
#pragma unroll 4
    for (int64_t b = t; b < B; b += 256) acc += x[b];
    red[t] = acc;
    __syncthreads();
    for (int o = 128; o >= 1; o >>= 1) {
        if (t < o) red[t] += red[t + o];
        __syncthreads();
    }
    if (t == 0) *v.out[i] = red[0];
}

}  // namespace

hipError_t launch_vec_sums(int64_t B, const VecSums& v, hipStream_t st) {
    if (v.n <= 0) return hipSuccess;
    if (v.n > VEC_SUMS_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_vec_sums, dim3((unsigned)v.n), dim3(256), 0, st, B, v);
    return hipGetLastError();
}

hipError_t launch_gate_logit(int64_t B, int n, const void* x, bool x_f16, int64_t ldx, const void* g, const void* c,
                             float* s, hipStream_t st) {
    if (B == 0) return hipSuccess;
    if (x_f16)
        hipLaunchKernelGGL(k_gate_logit<_Float16>, dim3(row_blocks(B)), dim3(256), 0, st, B, n, (const _Float16*)x, ldx,
                           (const bf16_t*)g, (const bf16_t*)c, s);
    else
        hipLaunchKernelGGL(k_gate_logit<bf16_t>, dim3(row_blocks(B)), dim3(256), 0, st, B, n, (const bf16_t*)x, ldx,
                           (const bf16_t*)g, (const bf16_t*)c, s);
    return hipGetLastError();
}

hipError_t launch_head_out(int64_t B, int n, const void* aL, const void* w_out, const void* b_out, const CalArgs& c,
                           float* y, float* y2, float* y_cal, hipStream_t st) {
    if (B == 0) return hipSuccess;
    hipLaunchKernelGGL(k_head_out<_Float16>, dim3(row_blocks(B)), dim3(256), 0, st, B, n, (const _Float16*)aL,
                       (const bf16_t*)w_out, (const bf16_t*)b_out, c, y, y2, y_cal);
    return hipGetLastError();
}

hipError_t launch_logloss(int64_t B, const float* z, const float* label, float scale, float* loss, float* grad,
                          hipStream_t st) {
    if (B == 0) return hipSuccess;
    int64_t blocks = (B + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_logloss, dim3((unsigned)blocks), dim3(256), 0, st, B, z, label, scale, loss, grad);
    return hipGetLastError();
}

hipError_t launch_head_out_bwd(int64_t B, int n, const void* aL, const float* sL, const void* w_out, const float* y,
                               const CalArgs& c, const float* g_cal, float* grad_e, float* gy, void* G, float* gs,
                               hipStream_t st) {
    if (B == 0) return hipSuccess;
    hipLaunchKernelGGL(k_head_out_bwd<_Float16>, dim3(row_blocks(B)), dim3(256), 0, st, B, n, (const _Float16*)aL, sL,
                       (const bf16_t*)w_out, y, c, g_cal, grad_e, gy, (bf16_t*)G, gs);
    return hipGetLastError();
}

hipError_t launch_gate_finalize(int64_t B, int ntiles, const float* part, const float* s, float* gs,
                                hipStream_t st) {
    if (B == 0) return hipSuccess;
    int64_t blocks = (B + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_gate_finalize, dim3((unsigned)blocks), dim3(256), 0, st, B, ntiles, part, s, gs);
    return hipGetLastError();
}

int64_t colsum_chunks(int64_t B) { return B > 0 ? (B + COLSUM_ROWS - 1) / COLSUM_ROWS : 1; }

hipError_t launch_colsum_w(int64_t B, int64_t n, const void* X, int64_t ldx, ColType xt, const float* wgt,
                           float* part, float* out, hipStream_t st) {
    if (n == 0) return hipSuccess;
    const int64_t nch = colsum_chunks(B);
    if (B == 0) {  // one chunk of zeros
        hipLaunchKernelGGL(k_chunk_reduce, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, st, (int64_t)0, n,
                           part, out);
        return hipGetLastError();
    }
    const bool vec = n % 8 == 0 && ldx % 8 == 0;
    const int64_t cols_per_block = 64 * (vec ? 8 : 1);
    const dim3 grid((unsigned)((n + cols_per_block - 1) / cols_per_block), (unsigned)nch);
    if (xt == COL_F16) {
        if (!vec) return hipErrorInvalidValue;
        hipLaunchKernelGGL((k_colsum_w<_Float16, 8>), grid, dim3(256), 0, st, B, n, (const _Float16*)X, ldx, wgt, part);
    } else if (xt == COL_BF16) {
        if (vec) hipLaunchKernelGGL((k_colsum_w<bf16_t, 8>), grid, dim3(256), 0, st, B, n, (const bf16_t*)X, ldx, wgt, part);
        else hipLaunchKernelGGL((k_colsum_w<bf16_t, 1>), grid, dim3(256), 0, st, B, n, (const bf16_t*)X, ldx, wgt, part);
    } else {
        if (vec) hipLaunchKernelGGL((k_colsum_w<float, 8>), grid, dim3(256), 0, st, B, n, (const float*)X, ldx, wgt, part);
        else hipLaunchKernelGGL((k_colsum_w<float, 1>), grid, dim3(256), 0, st, B, n, (const float*)X, ldx, wgt, part);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_chunk_reduce, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, st, nch, n, part, out);
    return hipGetLastError();
}

}  // namespace rdcn
