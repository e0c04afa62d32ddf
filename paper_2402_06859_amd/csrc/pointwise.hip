// Backward elementwise work of the cross layer x_{l+1} = x0 * t + x_l with
// t = U h + b, given g = dLoss/dx_{l+1}:
//   gt = g * x0          (operand of the U-side gradient products, storage type)
//   gx0 (+)= g * t       (x0 is the multiplier of every layer)
//   gb = sum over the batch of g * x0, as per-row-block partial column sums
// followed by a deterministic reduction of the partials (fixed order).
#include "device_common.h"
#include "kernels.h"

namespace rdcn {

namespace {

template <typename T>
__device__ __forceinline__ void ld4(const T* p, float* v);
template <>
__device__ __forceinline__ void ld4<float>(const float* p, float* v) {
    const f32x4_t x = *(const f32x4_t*)p;
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}
template <>
__device__ __forceinline__ void ld4<bf16_t>(const bf16_t* p, float* v) {
    const uint2 w = *(const uint2*)p;
    v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xffff0000u);
    v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xffff0000u);
}
template <typename T>
__device__ __forceinline__ void st4(T* p, const float* v);
template <>
__device__ __forceinline__ void st4<float>(float* p, const float* v) {
    *(f32x4_t*)p = f32x4_t{v[0], v[1], v[2], v[3]};
}
template <>
__device__ __forceinline__ void st4<bf16_t>(bf16_t* p, const float* v) {
    *(uint2*)p = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}

// 8 consecutive values at p (float: as two halves, the second at p + off4, where off4
// is 4, or 0 when only the first half lies inside the row; bf16 rows have a multiple
// of 8 columns, so their 16 bytes are always inside).
template <typename T>
__device__ __forceinline__ void ld8(const T* p, int off4, float* v);
template <>
__device__ __forceinline__ void ld8<float>(const float* p, int off4, float* v) {
    ld4<float>(p, v);
    ld4<float>(p + off4, v + 4);
}
template <>
__device__ __forceinline__ void ld8<bf16_t>(const bf16_t* p, int, float* v) {
    const u32x4_t w = *(const u32x4_t*)p;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        v[2 * h] = __uint_as_float(w[h] << 16);
        v[2 * h + 1] = __uint_as_float(w[h] & 0xffff0000u);
    }
}

// Store 8 values (float: the second half only when has4; bf16: all 16 bytes).
template <typename T>
__device__ __forceinline__ void st8(T* p, bool has4, const float* v);
template <>
__device__ __forceinline__ void st8<float>(float* p, bool has4, const float* v) {
    st4<float>(p, v);
    if (has4) st4<float>(p + 4, v + 4);
}
template <>
__device__ __forceinline__ void st8<bf16_t>(bf16_t* p, bool, const float* v) {
    *(u32x4_t*)p = u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                           pack_bf16x2(v[6], v[7])};
}

// Block = 16 column groups of 8 columns x 16 row slices (128 columns: each row
// segment a block touches is 256 bytes of every bf16 array and 512 of every float
// one; blocks of 64 columns and 128 rows were 5% slower). Thread (ty, tx) handles
// columns c .. c+7 (two 4-column halves; d is a multiple of 4) of rows
// b0 + ty + 16 k, k < PW_RPT: every load of its rows is issued before any of them
// is used. Its column sums are then added over ty in fixed order, giving one
// partial row per block.
constexpr int PW_COLS = 128;              // columns per block
constexpr int PW_TX = PW_COLS / 8;        // column groups
constexpr int PW_TY = 256 / PW_TX;        // row slices
constexpr int PW_RPT = 4;                 // rows per thread
constexpr int PW_ROWS = PW_TY * PW_RPT;   // rows per block

template <typename T>
__global__ __launch_bounds__(256) void k_bwd_pointwise(int64_t B, int64_t d, const void* gin, int gin_f32,
                                                       const T* __restrict__ x0, const T* __restrict__ t,
                                                       float* __restrict__ gx0, int first, T* __restrict__ gt,
                                                       float* __restrict__ part) {
    __shared__ float red[PW_TY][PW_COLS + 4];
    const int tx = threadIdx.x % PW_TX, ty = threadIdx.x / PW_TX;
    const int64_t c = (int64_t)blockIdx.x * PW_COLS + tx * 8;
    const int64_t b0 = (int64_t)blockIdx.y * PW_ROWS;
    float cs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (c < d) {
        // (float) the second half past d re-reads the first; nothing of it is stored
        const int off4 = c + 4 < d ? 4 : 0;
        float g[PW_RPT][8], xv[PW_RPT][8], tv[PW_RPT][8], acc[PW_RPT][8];
        int64_t row[PW_RPT];
#pragma unroll
        for (int k = 0; k < PW_RPT; ++k) {
            const int64_t b = b0 + ty + PW_TY * k;
            row[k] = (b < B ? b : b0) * d;  // rows past B re-read row b0 and are not stored
        }
        if (gin_f32) {
#pragma unroll
            for (int k = 0; k < PW_RPT; ++k) ld8<float>((const float*)gin + row[k] + c, off4, g[k]);
        } else {
#pragma unroll
            for (int k = 0; k < PW_RPT; ++k) ld8<T>((const T*)gin + row[k] + c, off4, g[k]);
        }
#pragma unroll
        for (int k = 0; k < PW_RPT; ++k) {
            ld8<T>(x0 + row[k] + c, off4, xv[k]);
            ld8<T>(t + row[k] + c, off4, tv[k]);
            if (!first) ld8<float>(gx0 + row[k] + c, off4, acc[k]);
        }
#pragma unroll
        for (int k = 0; k < PW_RPT; ++k) {
            if (b0 + ty + PW_TY * k >= B) continue;
            float gtv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float a = first ? 0.f : acc[k][e];
                gtv[e] = g[k][e] * xv[k][e];
                acc[k][e] = fmaf(g[k][e], tv[k][e], a);
                cs[e] += gtv[e];
            }
            st8<T>(gt + row[k] + c, off4 != 0, gtv);
            st8<float>(gx0 + row[k] + c, off4 != 0, acc[k]);
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) red[ty][tx * 8 + e] = cs[e];
    __syncthreads();
    // PW_COLS threads finish the block's columns, each adding the row slices in order
    if (threadIdx.x < PW_COLS) {
        const int col = threadIdx.x;
        const int64_t cc = (int64_t)blockIdx.x * PW_COLS + col;
        float s = red[0][col];
        for (int y = 1; y < PW_TY; ++y) s += red[y][col];
        if (cc < d) part[(int64_t)blockIdx.y * d + cc] = s;
    }
}

// out[c] = sum over the nrb partial rows, in row order within each of 16
// slices and then slice order.
__global__ __launch_bounds__(256) void k_colsum(const float* __restrict__ part, int nrb, int64_t d,
                                                float* __restrict__ out) {
    __shared__ float red[16][64 + 4];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int64_t c = (int64_t)blockIdx.x * 64 + tx * 4;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    if (c < d) {
        // unrolled so that eight rows' loads are in flight together (the sums stay in row order)
#pragma unroll 8
        for (int y = ty; y < nrb; y += 16) {
            float p[4];
            ld4<float>(part + (int64_t)y * d + c, p);
#pragma unroll
            for (int e = 0; e < 4; ++e) s[e] += p[e];
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) red[ty][tx * 4 + e] = s[e];
    __syncthreads();
    if (ty == 0 && c < d) {
        for (int y = 1; y < 16; ++y)
#pragma unroll
            for (int e = 0; e < 4; ++e) s[e] += red[y][tx * 4 + e];
        st4<float>(out + c, s);
    }
}

__global__ __launch_bounds__(256) void k_fill_zero(float* __restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0.f;
}

}  // namespace

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

int pointwise_rows_per_block(int64_t, int64_t) { return PW_ROWS; }

hipError_t launch_bwd_pointwise(int64_t B, int64_t d, const void* gin, bool gin_f32, const void* x0, const void* t,
                                float* gx0, bool first, void* gt, float* part, bool bf16, hipStream_t s) {
    if (B == 0) return hipSuccess;
    dim3 grid((unsigned)((d + PW_COLS - 1) / PW_COLS), (unsigned)((B + PW_ROWS - 1) / PW_ROWS));
    if (bf16)
        hipLaunchKernelGGL(k_bwd_pointwise<bf16_t>, grid, dim3(256), 0, s, B, d, gin, (int)gin_f32,
                           (const bf16_t*)x0, (const bf16_t*)t, gx0, (int)first, (bf16_t*)gt, part);
    else
        hipLaunchKernelGGL(k_bwd_pointwise<float>, grid, dim3(256), 0, s, B, d, gin, (int)gin_f32,
                           (const float*)x0, (const float*)t, gx0, (int)first, (float*)gt, part);
    return hipGetLastError();
}

hipError_t launch_colsum(const float* part, int nrb, int64_t d, float* out, hipStream_t s) {
    if (nrb == 0) return launch_fill_zero(out, d, s);
    hipLaunchKernelGGL(k_colsum, dim3((unsigned)((d + 63) / 64)), dim3(256), 0, s, part, nrb, d, out);
    return hipGetLastError();
}

}  // namespace rdcn
