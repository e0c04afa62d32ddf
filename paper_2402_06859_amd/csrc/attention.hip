// Per-sample attention over the low-rank coordinates (section "Residual DCN",
// second paragraph: value/query/key copies of the low-rank map, an attention
// score matrix inserted between the low-rank maps, a temperature, and a skip
// connection).
//
// For one sample, the r low-rank coordinates are r scalar tokens:
//   S_ij = q_i k_j / tau,  A = softmax over j,  o = A v,  h = beta v + alpha o.
// A is never stored. Because S_ij = q_i k_j / tau is linear in k_j, the row
// maximum is q_i max_j k_j / tau when q_i >= 0 and q_i min_j k_j / tau
// otherwise (rounded multiplication is monotone, so the same holds in float),
// which removes the usual online-softmax rescaling: every exponent is
// exp2(c_i k_j - c_i k*_i) <= 1 with c_i = q_i log2(e) / tau.
//
// One workgroup per sample; k and v (and, in the backward column pass, the
// per-row coefficients) are staged in LDS as floats and read as broadcasts.
#include "device_common.h"
#include "kernels.h"

namespace rdcn {

namespace {

constexpr float LOG2E = 1.4426950408889634f;

__device__ __forceinline__ void block_minmax(float lo, float hi, float* red, float& out_lo, float& out_hi) {
    // wave reduction then across waves (blockDim <= 1024)
    for (int off = 32; off > 0; off >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, off));
        hi = fmaxf(hi, __shfl_xor(hi, off));
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = (blockDim.x + 63) >> 6;
    if (lane == 0) {
        red[wave] = lo;
        red[16 + wave] = hi;
    }
    __syncthreads();
    lo = red[0];
    hi = red[16];
    for (int w = 1; w < nw; ++w) {
        lo = fminf(lo, red[w]);
        hi = fmaxf(hi, red[16 + w]);
    }
    out_lo = lo;
    out_hi = hi;
}

// Forward. P = [v | q | k] per sample in float (row stride ldp), h out (row stride ldh).
template <typename T>
__global__ __launch_bounds__(256) void k_attn_fwd(int64_t B, int r, float alpha, float beta, float inv_tau,
                                                 const float* __restrict__ P, int64_t ldp, T* __restrict__ H,
                                                 T* __restrict__ H2, int64_t ldh) {
    extern __shared__ float smem[];
    float* sk = smem;          // [r]
    float* sv = smem + r;      // [r]
    float* red = smem + 2 * r; // [32]
    const int64_t b = blockIdx.x;
    const float* pv = P + b * ldp;
    const float* pq = pv + r;
    const float* pk = pv + 2 * r;
    float lo = INFINITY, hi = -INFINITY;
    for (int j = threadIdx.x; j < r; j += blockDim.x) {
        const float kj = pk[j];
        sk[j] = kj;
        sv[j] = pv[j];
        lo = fminf(lo, kj);
        hi = fmaxf(hi, kj);
    }
    float kmin, kmax;
    block_minmax(lo, hi, red, kmin, kmax);  // includes a barrier after sk/sv are written
    for (int i = threadIdx.x; i < r; i += blockDim.x) {
        const float c = pq[i] * (LOG2E * inv_tau);
        const float mneg = -(c * (c >= 0.f ? kmax : kmin));
        float z0 = 0.f, z1 = 0.f, s0 = 0.f, s1 = 0.f;
        int j = 0;
        for (; j + 1 < r; j += 2) {
            const float e0 = __builtin_amdgcn_exp2f(fmaf(c, sk[j], mneg));
            const float e1 = __builtin_amdgcn_exp2f(fmaf(c, sk[j + 1], mneg));
            z0 += e0;
            z1 += e1;
            s0 = fmaf(e0, sv[j], s0);
            s1 = fmaf(e1, sv[j + 1], s1);
        }
        if (j < r) {
            const float e0 = __builtin_amdgcn_exp2f(fmaf(c, sk[j], mneg));
            z0 += e0;
            s0 = fmaf(e0, sv[j], s0);
        }
        const float o = (s0 + s1) / (z0 + z1);
        const float hv = beta * sv[i] + alpha * o;
        st<T>::store(H + b * ldh + i, hv);
        if (H2) st<T>::store(H2 + b * ldh + i, hv - st<T>::load(H + b * ldh + i));  // lo part of a hi + lo pair
    }
}

// Backward. gh = dLoss/dh (float, row stride ldg). Writes gP = [gv | gq | gk].
//   row pass (thread per query i):   Z_i = sum_j e_ij, o_i = sum_j e_ij v_j / Z_i,
//       gq_i = go_i/(Z_i tau) * (sum_j e_ij v_j k_j - o_i sum_j e_ij k_j),  go = alpha gh
//   column pass (thread per key j):  with a_i = go_i q_i/(Z_i tau), b_i = a_i o_i, c_i = go_i / Z_i
//       gk_j = v_j sum_i e_ij a_i - sum_i e_ij b_i,   gv_j = beta gh_j + sum_i e_ij c_i
// e_ij = exp2(c'_i k_j - c'_i k*_i) is recomputed identically in both passes.
template <typename T>
__global__ __launch_bounds__(256) void k_attn_bwd(int64_t B, int r, float alpha, float beta, float inv_tau,
                                                 const float* __restrict__ P, int64_t ldp, const float* __restrict__ GH,
                                                 int64_t ldg, T* __restrict__ GP, int64_t ldgp) {
    extern __shared__ float smem[];
    float* sk = smem;
    float* sv = smem + r;
    float* sc = smem + 2 * r;   // c'_i
    float* sm = smem + 3 * r;   // -c'_i k*_i
    float* sa = smem + 4 * r;   // a_i
    float* sb = smem + 5 * r;   // b_i
    float* sg = smem + 6 * r;   // c_i = go_i / Z_i
    float* red = smem + 7 * r;  // [32]
    const int64_t b = blockIdx.x;
    const float* pv = P + b * ldp;
    const float* pq = pv + r;
    const float* pk = pv + 2 * r;
    const float* gh = GH + b * ldg;
    T* gv_out = GP + b * ldgp;
    T* gq_out = gv_out + r;
    T* gk_out = gv_out + 2 * r;
    float lo = INFINITY, hi = -INFINITY;
    for (int j = threadIdx.x; j < r; j += blockDim.x) {
        const float kj = pk[j];
        sk[j] = kj;
        sv[j] = pv[j];
        lo = fminf(lo, kj);
        hi = fmaxf(hi, kj);
    }
    float kmin, kmax;
    block_minmax(lo, hi, red, kmin, kmax);
    for (int i = threadIdx.x; i < r; i += blockDim.x) {
        const float q = pq[i];
        const float c = q * (LOG2E * inv_tau);
        const float mneg = -(c * (c >= 0.f ? kmax : kmin));
        float z = 0.f, s = 0.f, w1 = 0.f, w2 = 0.f;
        for (int j = 0; j < r; ++j) {
            const float e = __builtin_amdgcn_exp2f(fmaf(c, sk[j], mneg));
            const float kj = sk[j];
            const float ev = e * sv[j];
            z += e;
            s += ev;
            w1 = fmaf(ev, kj, w1);
            w2 = fmaf(e, kj, w2);
        }
        const float rz = 1.0f / z;
        const float o = s * rz;
        const float go = alpha * gh[i];
        const float a = go * q * rz * inv_tau;
        st<T>::store(gq_out + i, go * rz * inv_tau * (w1 - o * w2));
        sc[i] = c;
        sm[i] = mneg;
        sa[i] = a;
        sb[i] = a * o;
        sg[i] = go * rz;
    }
    __syncthreads();
    for (int j = threadIdx.x; j < r; j += blockDim.x) {
        const float kj = sk[j];
        float c1 = 0.f, c2 = 0.f, c3 = 0.f;
        for (int i = 0; i < r; ++i) {
            const float e = __builtin_amdgcn_exp2f(fmaf(sc[i], kj, sm[i]));
            c1 = fmaf(e, sa[i], c1);
            c2 = fmaf(e, sb[i], c2);
            c3 = fmaf(e, sg[i], c3);
        }
        st<T>::store(gk_out + j, sv[j] * c1 - c2);
        st<T>::store(gv_out + j, beta * gh[j] + c3);
    }
}

int attn_threads(int r) {
    int t = ((r + 63) / 64) * 64;
    return t > 256 ? 256 : t;
}

}  // namespace

hipError_t launch_attn_fwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp, void* H,
                           void* H2, int64_t ldh, bool bf16, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const size_t lds = sizeof(float) * (2 * (size_t)r + 32);
    const int th = attn_threads(r);
    if (bf16)
        hipLaunchKernelGGL(k_attn_fwd<bf16_t>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                           (const float*)P, ldp, (bf16_t*)H, (bf16_t*)H2, ldh);
    else
        hipLaunchKernelGGL(k_attn_fwd<float>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                           (const float*)P, ldp, (float*)H, (float*)H2, ldh);
    return hipGetLastError();
}

hipError_t launch_attn_bwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp,
                           const float* GH, int64_t ldg, void* GP, int64_t ldgp, bool bf16, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const size_t lds = sizeof(float) * (7 * (size_t)r + 32);
    const int th = attn_threads(r);
    if (bf16)
        hipLaunchKernelGGL(k_attn_bwd<bf16_t>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                           (const float*)P, ldp, GH, ldg, (bf16_t*)GP, ldgp);
    else
        hipLaunchKernelGGL(k_attn_bwd<float>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                           (const float*)P, ldp, GH, ldg, (float*)GP, ldgp);
    return hipGetLastError();
}

}  // namespace rdcn
