// Device helpers shared by the MLP epilogues (gemm.hip) and the head kernels
// (head.hip): both sides must evaluate the gate identically.
#pragma once
#include <hip/hip_runtime.h>

namespace rdcn {

// Logistic function in float; the branch keeps exp from overflowing.
__device__ __forceinline__ float sigmoid_f(float x) {
    if (x >= 0.f) return 1.f / (1.f + expf(-x));
    const float e = expf(x);
    return e / (1.f + e);
}

// ReLU that keeps a NaN input NaN.
__device__ __forceinline__ float relu_f(float x) { return x < 0.f ? 0.f : x; }

}  // namespace rdcn
