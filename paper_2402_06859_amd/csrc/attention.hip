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

// ---------------------------------------------------------------------------
// bf16 models: the exponentials are computed on the vector ALU, but every
// weighted sum over them runs on the matrix cores. For a 16-row x 32-key block
// of one sample, each lane computes the 8 values e_ij of its row i = lane % 16
// for keys 8 (lane / 16) .. +7, which is exactly the B-operand layout of
// v_mfma_f32_16x16x32_f16; the A operand is a small per-sample matrix X^T whose
// rows are the quantities to be summed against e (v, 1, v k, k, or the column
// coefficients of the backward), each stored as an f16 hi + lo pair scaled by a
// power of two so the pair keeps about 21 significant bits. e itself is rounded
// to f16 (relative 2^-11); all sums of one row use the same rounded e, so the
// normalisation by Z is consistent. Output lane l holds quantities
// 4 (l / 16) .. +3 of row l % 16.
// ---------------------------------------------------------------------------
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pk_f16(float a, float b) {
    const f16x2_t v = {(_Float16)a, (_Float16)b};
    return __builtin_bit_cast(uint32_t, v);
}

// power of two >= |m| (1 for m == 0), so x / scale lies in [-1, 1]
__device__ __forceinline__ float pow2_ceil(float m) {
    if (!(m > 0.f)) return 1.f;
    int e;
    const float f = frexpf(m, &e);  // m = f * 2^e, f in [0.5, 1)
    (void)f;
    return ldexpf(1.f, e);
}

__device__ __forceinline__ float block_max_abs(float x, float* red) {
    for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0) red[wave] = x;
    __syncthreads();
    return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// X^T row n, keys j0 .. j0+7 as an f16 A fragment (rows >= nx read as zero).
__device__ __forceinline__ f16x8_t xfrag(const _Float16* sx, int rpad, int n, int nx, int j0) {
    if (n >= nx) return f16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    return __builtin_bit_cast(f16x8_t, *(const u32x4_t*)(sx + n * rpad + j0));
}

// e for one row (c, m) and 8 keys kv[0..7], packed as the B fragment.
__device__ __forceinline__ f16x8_t efrag(float c, float m, const float* kv) {
    float e[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) e[t] = __builtin_amdgcn_exp2f(fmaf(c, kv[t], m));
    const u32x4_t w = {pk_f16(e[0], e[1]), pk_f16(e[2], e[3]), pk_f16(e[4], e[5]), pk_f16(e[6], e[7])};
    return __builtin_bit_cast(f16x8_t, w);
}

constexpr int ATT_RT = 4;  // 16-row tiles a wave keeps in flight (register blocking)

// Row pass over all keys for the row tiles rt = first + 4 q (q < ATT_RT, rt < ntile):
// acc[q] += X^T (rows nx) . E^T over keys.
__device__ __forceinline__ void row_pass(const float* sk, const float* sc, const float* sm, const _Float16* sx, int nx,
                                         int rpad, int first, int ntile, int lane, f32x4_t (&acc)[ATT_RT]) {
    const int g = lane >> 4, n = lane & 15;
    float c[ATT_RT], m[ATT_RT];
#pragma unroll
    for (int q = 0; q < ATT_RT; ++q) {
        acc[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int rt = first + 4 * q;
        const int i = (rt < ntile ? rt : 0) * 16 + n;
        c[q] = sc[i];
        m[q] = sm[i];
    }
    for (int j0 = 0; j0 < rpad; j0 += 32) {
        const int jj = j0 + 8 * g;
        float kv[8];
        *(u32x4_t*)kv = *(const u32x4_t*)(sk + jj);
        *(u32x4_t*)(kv + 4) = *(const u32x4_t*)(sk + jj + 4);
        const f16x8_t a = xfrag(sx, rpad, n, nx, jj);
#pragma unroll
        for (int q = 0; q < ATT_RT; ++q) {
            if (first + 4 * q < ntile)
                acc[q] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, efrag(c[q], m[q], kv), acc[q], 0, 0, 0);
        }
    }
}

// Shared per-sample setup: k, v, row constants; returns kmin/kmax via LDS.
// Padded keys / rows (index >= r) get k = 0, c = 0, m = 0 and zero X^T entries.
__device__ __forceinline__ void setup_rows(const float* pv, const float* pq, const float* pk, int r, int rpad,
                                           float inv_tau, float* sk, float* sv, float* sc, float* sm, float* red) {
    float lo = INFINITY, hi = -INFINITY;
    for (int j = threadIdx.x; j < rpad; j += blockDim.x) {
        const float kj = j < r ? pk[j] : 0.f;
        sk[j] = kj;
        sv[j] = j < r ? pv[j] : 0.f;
        if (j < r) {
            lo = fminf(lo, kj);
            hi = fmaxf(hi, kj);
        }
    }
    float kmin, kmax;
    block_minmax(lo, hi, red, kmin, kmax);
    for (int i = threadIdx.x; i < rpad; i += blockDim.x) {
        const float c = i < r ? pq[i] * (LOG2E * inv_tau) : 0.f;
        sc[i] = c;
        sm[i] = i < r ? -(c * (c >= 0.f ? kmax : kmin)) : 0.f;
    }
}

// Write quantity x_j / s as an f16 hi + lo pair into rows (hi_row, hi_row + 1) of X^T.
__device__ __forceinline__ void put_pair(_Float16* sx, int rpad, int hi_row, int j, float xs) {
    const _Float16 h = (_Float16)xs;
    sx[hi_row * rpad + j] = h;
    sx[(hi_row + 1) * rpad + j] = (_Float16)(xs - (float)h);
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_fwd_mfma(int r, int rpad, float alpha, float beta, float inv_tau,
                                                      const float* __restrict__ P, int64_t ldp, T* __restrict__ H,
                                                      T* __restrict__ H2, int64_t ldh) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    float* sk = smem;              // [rpad]
    float* sv = sk + rpad;         // [rpad]
    float* sc = sv + rpad;         // [rpad]
    float* sm = sc + rpad;         // [rpad]
    float* red = sm + rpad;        // [32]
    _Float16* sx = (_Float16*)(red + 32);  // X^T: 3 rows x rpad (v hi, v lo, 1)
    const int64_t b = blockIdx.x;
    const float* pv = P + b * ldp;
    setup_rows(pv, pv + r, pv + 2 * r, r, rpad, inv_tau, sk, sv, sc, sm, red);
    float vmax = 0.f;
    for (int j = threadIdx.x; j < r; j += blockDim.x) vmax = fmaxf(vmax, fabsf(sv[j]));
    const float vs = pow2_ceil(block_max_abs(vmax, red));
    for (int j = threadIdx.x; j < rpad; j += blockDim.x) {
        put_pair(sx, rpad, 0, j, sv[j] / vs);
        sx[2 * rpad + j] = (_Float16)(j < r ? 1.f : 0.f);
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ntile = rpad / 16;
    for (int first = wave; first < ntile; first += 4 * ATT_RT) {
        f32x4_t acc[ATT_RT];
        row_pass(sk, sc, sm, sx, 3, rpad, first, ntile, lane, acc);
        if (lane < 16) {
#pragma unroll
            for (int q = 0; q < ATT_RT; ++q) {
                const int i = (first + 4 * q) * 16 + lane;
                if (first + 4 * q < ntile && i < r) {
                    const float o = (acc[q].x + acc[q].y) * vs / acc[q].z;
                    const float hv = beta * sv[i] + alpha * o;
                    st<T>::store(H + b * ldh + i, hv);
                    if (H2) st<T>::store(H2 + b * ldh + i, hv - st<T>::load(H + b * ldh + i));
                }
            }
        }
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_bwd_mfma(int r, int rpad, float alpha, float beta, float inv_tau,
                                                      const float* __restrict__ P, int64_t ldp,
                                                      const float* __restrict__ GH, int64_t ldg, T* __restrict__ GP,
                                                      int64_t ldgp) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    float* sk = smem;
    float* sv = sk + rpad;
    float* sc = sv + rpad;
    float* sm = sc + rpad;
    float* sa = sm + rpad;   // a_i = go_i q_i / (Z_i tau)
    float* sb = sa + rpad;   // b_i = a_i o_i
    float* sg = sb + rpad;   // c_i = go_i / Z_i
    float* red = sg + rpad;  // [32]
    _Float16* sx = (_Float16*)(red + 32);  // X^T rows: v hi/lo, 1, 0, v k hi/lo, k hi/lo   (8 x rpad)
    _Float16* sy = sx + 8 * rpad;          // Y^T rows: a hi/lo, b hi/lo, c hi/lo             (6 x rpad)
    const int64_t b = blockIdx.x;
    const float* pv = P + b * ldp;
    const float* pq = pv + r;
    const float* gh = GH + b * ldg;
    setup_rows(pv, pq, pv + 2 * r, r, rpad, inv_tau, sk, sv, sc, sm, red);
    float mv = 0.f, mvk = 0.f, mk = 0.f;
    for (int j = threadIdx.x; j < r; j += blockDim.x) {
        mv = fmaxf(mv, fabsf(sv[j]));
        mvk = fmaxf(mvk, fabsf(sv[j] * sk[j]));
        mk = fmaxf(mk, fabsf(sk[j]));
    }
    const float vs = pow2_ceil(block_max_abs(mv, red));
    const float vks = pow2_ceil(block_max_abs(mvk, red));
    const float ks = pow2_ceil(block_max_abs(mk, red));
    for (int j = threadIdx.x; j < rpad; j += blockDim.x) {
        put_pair(sx, rpad, 0, j, sv[j] / vs);
        sx[2 * rpad + j] = (_Float16)(j < r ? 1.f : 0.f);
        sx[3 * rpad + j] = (_Float16)0.f;
        put_pair(sx, rpad, 4, j, sv[j] * sk[j] / vks);
        put_pair(sx, rpad, 6, j, sk[j] / ks);
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ntile = rpad / 16;
    // row pass: Z, S = sum e v, W1 = sum e v k, W2 = sum e k per query row
    for (int first = wave; first < ntile; first += 4 * ATT_RT) {
        f32x4_t acc[ATT_RT];
        row_pass(sk, sc, sm, sx, 8, rpad, first, ntile, lane, acc);
#pragma unroll
        for (int q = 0; q < ATT_RT; ++q) {
            // lanes 16..31 hold (W1 hi, W1 lo, W2 hi, W2 lo) of row lane - 16
            const float w1 = __shfl((acc[q].x + acc[q].y) * vks, lane + 16);
            const float w2 = __shfl((acc[q].z + acc[q].w) * ks, lane + 16);
            const int i = (first + 4 * q) * 16 + lane;
            if (lane < 16 && first + 4 * q < ntile) {
                if (i < r) {
                    const float z = acc[q].z;
                    const float o = (acc[q].x + acc[q].y) * vs / z;
                    const float go = alpha * gh[i];
                    const float rz = 1.0f / z;
                    const float a = go * pq[i] * rz * inv_tau;
                    st<T>::store(GP + b * ldgp + r + i, go * rz * inv_tau * (w1 - o * w2));
                    sa[i] = a;
                    sb[i] = a * o;
                    sg[i] = go * rz;
                } else {
                    sa[i] = sb[i] = sg[i] = 0.f;
                }
            }
        }
    }
    __syncthreads();
    float ma = 0.f, mb = 0.f, mc = 0.f;
    for (int i = threadIdx.x; i < r; i += blockDim.x) {
        ma = fmaxf(ma, fabsf(sa[i]));
        mb = fmaxf(mb, fabsf(sb[i]));
        mc = fmaxf(mc, fabsf(sg[i]));
    }
    const float as = pow2_ceil(block_max_abs(ma, red));
    const float bs = pow2_ceil(block_max_abs(mb, red));
    const float cs = pow2_ceil(block_max_abs(mc, red));
    for (int i = threadIdx.x; i < rpad; i += blockDim.x) {
        put_pair(sy, rpad, 0, i, sa[i] / as);
        put_pair(sy, rpad, 2, i, sb[i] / bs);
        put_pair(sy, rpad, 4, i, sg[i] / cs);
    }
    __syncthreads();
    // column pass: for keys j, sum over rows i of e_ij (a_i, b_i, c_i);
    // lane (j = lane % 16, g) computes e for rows 8 g .. +7 of a 32-row chunk.
    const int g = lane >> 4, n = lane & 15;
    for (int first = wave; first < ntile; first += 4 * ATT_RT) {
        f32x4_t acc[ATT_RT];
        float kj[ATT_RT];
#pragma unroll
        for (int q = 0; q < ATT_RT; ++q) {
            acc[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            const int ct = first + 4 * q;
            kj[q] = sk[(ct < ntile ? ct : 0) * 16 + n];
        }
        for (int i0 = 0; i0 < rpad; i0 += 32) {
            const int ii = i0 + 8 * g;
            float cv[8], mv8[8];
            *(u32x4_t*)cv = *(const u32x4_t*)(sc + ii);
            *(u32x4_t*)(cv + 4) = *(const u32x4_t*)(sc + ii + 4);
            *(u32x4_t*)mv8 = *(const u32x4_t*)(sm + ii);
            *(u32x4_t*)(mv8 + 4) = *(const u32x4_t*)(sm + ii + 4);
            const f16x8_t a = xfrag(sy, rpad, n, 6, ii);
#pragma unroll
            for (int q = 0; q < ATT_RT; ++q) {
                if (first + 4 * q < ntile) {
                    float e[8];
#pragma unroll
                    for (int t = 0; t < 8; ++t) e[t] = __builtin_amdgcn_exp2f(fmaf(cv[t], kj[q], mv8[t]));
                    const u32x4_t w = {pk_f16(e[0], e[1]), pk_f16(e[2], e[3]), pk_f16(e[4], e[5]), pk_f16(e[6], e[7])};
                    acc[q] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, __builtin_bit_cast(f16x8_t, w), acc[q], 0, 0, 0);
                }
            }
        }
#pragma unroll
        for (int q = 0; q < ATT_RT; ++q) {
            const float c3 = __shfl((acc[q].x + acc[q].y) * cs, lane + 16);
            const int j = (first + 4 * q) * 16 + lane;
            if (lane < 16 && first + 4 * q < ntile && j < r) {
                const float c1 = (acc[q].x + acc[q].y) * as;
                const float c2 = (acc[q].z + acc[q].w) * bs;
                st<T>::store(GP + b * ldgp + 2 * r + j, sv[j] * c1 - c2);
                st<T>::store(GP + b * ldgp + j, beta * gh[j] + c3);
            }
        }
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
    if (bf16) {
        const int rpad = (r + 31) / 32 * 32;
        const size_t lds = sizeof(float) * (4 * (size_t)rpad + 32) + sizeof(_Float16) * 3 * (size_t)rpad;
        hipLaunchKernelGGL(k_attn_fwd_mfma<bf16_t>, dim3((unsigned)B), dim3(256), lds, s, r, rpad, alpha, beta,
                           1.0f / tau, (const float*)P, ldp, (bf16_t*)H, (bf16_t*)H2, ldh);
        return hipGetLastError();
    }
    const size_t lds = sizeof(float) * (2 * (size_t)r + 32);
    const int th = attn_threads(r);
        hipLaunchKernelGGL(k_attn_fwd<float>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                           (const float*)P, ldp, (float*)H, (float*)H2, ldh);
    return hipGetLastError();
}

hipError_t launch_attn_bwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp,
                           const float* GH, int64_t ldg, void* GP, int64_t ldgp, bool bf16, hipStream_t s) {
    if (B == 0) return hipSuccess;
    if (bf16) {
        const int rpad = (r + 31) / 32 * 32;
        const size_t lds = sizeof(float) * (7 * (size_t)rpad + 32) + sizeof(_Float16) * 14 * (size_t)rpad;
        hipLaunchKernelGGL(k_attn_bwd_mfma<bf16_t>, dim3((unsigned)B), dim3(256), lds, s, r, rpad, alpha, beta,
                           1.0f / tau, (const float*)P, ldp, GH, ldg, (bf16_t*)GP, ldgp);
        return hipGetLastError();
    }
    const size_t lds = sizeof(float) * (7 * (size_t)r + 32);
    const int th = attn_threads(r);
        hipLaunchKernelGGL(k_attn_bwd<float>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                           (const float*)P, ldp, GH, ldg, (float*)GP, ldgp);
    return hipGetLastError();
}

}  // namespace rdcn
