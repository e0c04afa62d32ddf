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

// Block = 16 column groups of 4 columns x 16 row slices. Thread (ty, tx) handles
// columns c .. c+3 and rows b0 + ty, b0 + ty + 16, ...; its column sums are then
// added over ty in fixed order, giving one partial row per block.
constexpr int PW_ROWS = 128;  // rows per block

template <typename T>
__global__ __launch_bounds__(256) void k_bwd_pointwise(int64_t B, int64_t d, const void* gin, int gin_f32,
                                                       const T* __restrict__ x0, const T* __restrict__ t,
                                                       float* __restrict__ gx0, int first, T* __restrict__ gt,
                                                       float* __restrict__ part) {
    __shared__ float red[16][64 + 4];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int64_t c = (int64_t)blockIdx.x * 64 + tx * 4;
    const int64_t b0 = (int64_t)blockIdx.y * PW_ROWS;
    int64_t b1 = b0 + PW_ROWS;
    if (b1 > B) b1 = B;
    float cs[4] = {0.f, 0.f, 0.f, 0.f};
    if (c < d) {
        for (int64_t b = b0 + ty; b < b1; b += 16) {
            const int64_t i = b * d + c;
            float g[4], xv[4], tv[4], acc[4], gtv[4];
            if (gin_f32) ld4<float>((const float*)gin + i, g);
            else ld4<T>((const T*)gin + i, g);
            ld4<T>(x0 + i, xv);
            ld4<T>(t + i, tv);
            if (first) {
                acc[0] = acc[1] = acc[2] = acc[3] = 0.f;
            } else {
                ld4<float>(gx0 + i, acc);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                gtv[e] = g[e] * xv[e];
                acc[e] = fmaf(g[e], tv[e], acc[e]);
                cs[e] += gtv[e];
            }
            st4<T>(gt + i, gtv);
            st4<float>(gx0 + i, acc);
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) red[ty][tx * 4 + e] = cs[e];
    __syncthreads();
    if (ty == 0 && c < d) {
        float s[4] = {red[0][tx * 4], red[0][tx * 4 + 1], red[0][tx * 4 + 2], red[0][tx * 4 + 3]};
        for (int y = 1; y < 16; ++y)
#pragma unroll
            for (int e = 0; e < 4; ++e) s[e] += red[y][tx * 4 + e];
        st4<float>(part + (int64_t)blockIdx.y * d + c, s);
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
    dim3 grid((unsigned)((d + 63) / 64), (unsigned)((B + PW_ROWS - 1) / PW_ROWS));
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
