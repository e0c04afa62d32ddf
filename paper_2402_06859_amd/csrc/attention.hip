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
#include <type_traits>

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
// bf16 models: the exponentials are computed on the vector ALU, every weighted
// sum over them runs on the matrix cores. For a 16-row x 32-key block of one
// sample, each lane computes the 8 values e_ij of its row i = lane % 16 for keys
// 8 (lane / 16) .. +7, which is exactly the B-operand layout of
// v_mfma_f32_16x16x32_f16 with K running over keys; the A operand is a small
// per-sample matrix X^T whose rows are the quantities summed against e (v, 1,
// v k, k), each stored as an f16 hi + lo pair scaled by a power of two so the
// pair keeps about 21 significant bits. e itself is rounded to f16 (relative
// 2^-11); all sums of one row use the same rounded e, so the normalisation by Z
// is consistent. Output lane l holds quantities 4 (l / 16) .. +3 of row l % 16.
//
// One wave owns up to ATT_NT 16-row tiles of one sample and loops over all keys,
// so row sums never leave its registers and the setup needs no workgroup
// barrier; a sample with more rows is split over W = ceil(tiles / ATT_NT) waves
// of one workgroup.
//
// The forward saves each row's o_i and Z_i. The backward then needs every e_ij
// only once: the row sums (over keys) take e in the layout above, and the column
// sums (over rows, weighted by per-row coefficients that depend on o_i and Z_i)
// take the same values transposed: the wave writes its 32-row x 32-key block of
// e to LDS and reads it back with ds_read_b64_tr_b16, which delivers the B
// operand with K running over rows.
// ---------------------------------------------------------------------------
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int ATT_NT = 16;  // 16-row tiles per wave

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

// A wave-uniform float (the same value in every lane) moved to a scalar register.
__device__ __forceinline__ float uniform_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x)));
}

__device__ __forceinline__ float wave_max(float x) {
    for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
    return x;
}
__device__ __forceinline__ float wave_min(float x) {
    for (int off = 32; off > 0; off >>= 1) x = fminf(x, __shfl_xor(x, off));
    return x;
}

// The X^T / Y^T operand matrices (a few rows of f16, row stride ld, ld a multiple
// of 32) keep entry j of row n in 8-element chunk (j / 8) XOR (n & 3): the rows one
// fragment read touches then fall in different LDS banks.
__device__ __forceinline__ int xoff(int n, int j, int ld) { return n * ld + ((((j >> 3) ^ n) & 3) | ((j >> 3) & ~3)) * 8 + (j & 7); }

// Row n (< nx, else zero) of an operand matrix, entries j0 .. j0+7 (j0 % 8 == 0).
__device__ __forceinline__ f16x8_t xfrag(const _Float16* sx, int ld, int n, int nx, int j0) {
    if (n >= nx) return f16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    return __builtin_bit_cast(f16x8_t, *(const u32x4_t*)(sx + xoff(n, j0, ld)));
}

// Key order inside one 32-key chunk. Lane (g, n)'s 8 K slots of a fragment hold
// keys j0 + 4 g + t (t < 4) and j0 + 16 + 4 g + (t - 4) (t >= 4): the layout in
// which two 16x16x16 MFMA outputs (keys j0 .. +15 and j0 + 16 .. +31) leave the
// exponent arguments. Everything indexed by key within a chunk (X^T fragments,
// the LDS e block) follows it; sums over K do not depend on the order.
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t pack_e(const float (&e)[8]) {
    return u32x4_t{pk_f16(e[0], e[1]), pk_f16(e[2], e[3]), pk_f16(e[4], e[5]), pk_f16(e[6], e[7])};
}

// e for one row (c, m) and the lane's 8 keys kv[0..7] (in the order above),
// exponent arguments by FMA.
__device__ __forceinline__ u32x4_t efrag(float c, float m, const float* kv) {
    float e[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) e[t] = __builtin_amdgcn_exp2f(fmaf(c, kv[t], m));
    return pack_e(e);
}

// Exponent arguments on the matrix cores: x = c k + m as a 16 (keys) x 16 (rows)
// product with K = 5 of 16 slots used, from f16 hi + lo parts of c, k and m:
//   keys (A, lane (g, n), key n):   g = 0: (k_hi, k_hi, 1, 1)   g = 1: (k_lo, 0, 0, 0)
//   rows (B, lane (g, n), row n):   (c_hi, c_lo, m_hi, m_lo) for every g
// giving c_hi k_hi + c_lo k_hi + m_hi + m_lo + c_hi k_lo: every product is exact in
// the float accumulator and only c_lo k_lo (relative 2^-22 of c k) is left out.
__device__ __forceinline__ f16x4_t key_frag(float k, int g) {
    const _Float16 hi = (_Float16)k, lo = (_Float16)(k - (float)hi);
    if (g == 0) return f16x4_t{hi, hi, (_Float16)1.f, (_Float16)1.f};
    if (g == 1) return f16x4_t{lo, (_Float16)0.f, (_Float16)0.f, (_Float16)0.f};
    return f16x4_t{(_Float16)0.f, (_Float16)0.f, (_Float16)0.f, (_Float16)0.f};
}

__device__ __forceinline__ f16x4_t row_rec(float c, float m) {
    const _Float16 ch = (_Float16)c, mh = (_Float16)m;
    return f16x4_t{ch, (_Float16)(c - (float)ch), mh, (_Float16)(m - (float)mh)};
}

__device__ __forceinline__ u32x4_t efrag_mfma(const f16x4_t& k0, const f16x4_t& k1, const f16x4_t& rec) {
    const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
    const f32x4_t x0 = __builtin_amdgcn_mfma_f32_16x16x16f16(k0, rec, z, 0, 0, 0);
    const f32x4_t x1 = __builtin_amdgcn_mfma_f32_16x16x16f16(k1, rec, z, 0, 0, 0);
    float e[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        e[t] = __builtin_amdgcn_exp2f(x0[t]);
        e[4 + t] = __builtin_amdgcn_exp2f(x1[t]);
    }
    return pack_e(e);
}

// X^T fragment of row n (< nx, else zero) for the chunk at j0, keys in the order above.
__device__ __forceinline__ f16x8_t xfrag_perm(const _Float16* sx, int ld, int n, int nx, int j0, int g) {
    if (n >= nx) return f16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    const f16x4_t lo = *(const f16x4_t*)(sx + xoff(n, j0 + 4 * g, ld));
    const f16x4_t hi = *(const f16x4_t*)(sx + xoff(n, j0 + 16 + 4 * g, ld));
    return f16x8_t{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
}

// The lane's 8 keys (order above) from the float key array.
__device__ __forceinline__ void keys_perm(const float* sk, int j0, int g, float (&kv)[8]) {
    *(u32x4_t*)kv = *(const u32x4_t*)(sk + j0 + 4 * g);
    *(u32x4_t*)(kv + 4) = *(const u32x4_t*)(sk + j0 + 16 + 4 * g);
}

// Exponent arguments go through the matrix cores when every c, m and k of the
// wave fits f16 with margin; otherwise (extreme logits) through FMAs. The forward
// and the backward take the same decision from the same values.
constexpr float ATT_F16_SAFE = 16384.f;

// Write quantity x / s as an f16 hi + lo pair into rows (row, row + 1) of X^T.
__device__ __forceinline__ void put_pair(_Float16* sx, int ld, int row, int j, float xs) {
    const _Float16 h = (_Float16)xs;
    sx[xoff(row, j, ld)] = h;
    sx[xoff(row + 1, j, ld)] = (_Float16)(xs - (float)h);
}

// Which sample and which block of row tiles a wave owns.
struct WaveRows {
    int64_t b;   // sample
    int w;       // part of the sample (0 .. W-1)
    int t0, nt;  // first tile, tiles owned
};
__device__ __forceinline__ WaveRows wave_rows(int W, int ntile) {
    WaveRows o;
    const int64_t gw = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    o.b = gw / W;
    o.w = (int)(gw - o.b * W);
    const int per = (((ntile + W - 1) / W) + 1) & ~1;  // even, <= ATT_NT for the W chosen at launch
    o.t0 = o.w * per;
    o.nt = ntile - o.t0 < per ? ntile - o.t0 : per;
    if (o.nt < 0) o.nt = 0;
    // wave-uniform: keep them in scalar registers
    o.b = ((int64_t)__builtin_amdgcn_readfirstlane((int)(o.b >> 32)) << 32) |
          (uint32_t)__builtin_amdgcn_readfirstlane((int)(o.b & 0xffffffff));
    o.w = __builtin_amdgcn_readfirstlane(o.w);
    o.t0 = __builtin_amdgcn_readfirstlane(o.t0);
    o.nt = __builtin_amdgcn_readfirstlane(o.nt);
    return o;
}

// Setup reads every per-sample operand a lane needs with one batch of loads
// (indices clamped to the valid range, so each load is issued; values past r are
// replaced by zeros), then works from registers.
//   keys / values: lane holds j = 64 u + lane, u < KPL (KPL * 64 >= rpad)
//   the wave's rows: lane holds il = 64 u + lane, u < RPL (RPL * 64 >= 16 NT)
template <int KPL>
__device__ __forceinline__ void load_keys(const float* pv, const float* pk, int r, int lane, float (&k)[KPL],
                                          float (&v)[KPL]) {
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        const int j = 64 * u + lane;
        const int jc = j < r ? j : r - 1;
        k[u] = pk[jc];
        v[u] = pv[jc];
    }
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        if (64 * u + lane >= r) k[u] = v[u] = 0.f;
    }
}

template <int NT>
struct RowsPerLane {
    static constexpr int value = (16 * NT + 63) / 64;
};

// rows t0 * 16 + il of quantity x (zero past r or past the rows in range)
template <int RPL>
__device__ __forceinline__ void load_rows(const float* x, int r, int t0, int nrows, int lane, float (&out)[RPL]) {
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        const int il = 64 * u + lane, i = t0 * 16 + il;
        out[u] = x[i < r ? i : r - 1];
    }
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        const int il = 64 * u + lane, i = t0 * 16 + il;
        if (!(il < nrows && i < r)) out[u] = 0.f;
    }
}

// key range over the keys held (valid keys only)
template <int KPL>
__device__ __forceinline__ void key_range(const float (&k)[KPL], int r, int lane, float& kmin, float& kmax) {
    float lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        if (64 * u + lane < r) {
            lo = fminf(lo, k[u]);
            hi = fmaxf(hi, k[u]);
        }
    }
    kmin = wave_min(lo);
    kmax = wave_max(hi);
}

// (c_i, m_i) = (q_i log2(e) / tau, -c_i k*_i) of rows il = 64 u + lane < 16 NT into
// scm[il] (rows past r: c = m = 0; q holds zeros there): as floats, or, when every
// c, m of rows il < nrows and every key fits f16 (returned, wave-uniform), as the
// f16 record row_rec of the matrix-core path.
template <int NT, int RPL>
__device__ __forceinline__ bool put_row_consts(const float (&q)[RPL], int lane, int nrows, float inv_tau,
                                               float kmin, float kmax, float2* scm) {
    float c[RPL], m[RPL], big = fmaxf(fabsf(kmin), fabsf(kmax));
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        c[u] = q[u] * (LOG2E * inv_tau);
        m[u] = -(c[u] * (c[u] >= 0.f ? kmax : kmin));
        if (64 * u + lane < nrows) big = fmaxf(big, fmaxf(fabsf(c[u]), fabsf(m[u])));
    }
    const bool fast = wave_max(big) < ATT_F16_SAFE;  // false for NaN too
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        const int il = 64 * u + lane;
        if (il < 16 * NT) {
            if (fast) *(f16x4_t*)(scm + il) = row_rec(c[u], m[u]);
            else scm[il] = make_float2(c[u], m[u]);
        }
    }
    return fast;
}

// LDS words per wave of the forward: keys, row constants, X^T (3 rows).
__host__ __device__ constexpr int attn_fwd_wave_floats(int rpad) { return rpad + 2 * 16 * ATT_NT + 3 * rpad / 2; }

// NT: tiles computed per wave (a power of two >= the tiles it owns; the extra ones
// are computed on harmless row constants and discarded).
// KB: 256-key batches a lane's registers cover (4 KB >= rpad / 64).
template <typename T, int NT, int KB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_attn_fwd_mfma(int64_t B, int r, int rpad, int W, float alpha, float beta,
                                                      float inv_tau, const float* __restrict__ P, int64_t ldp,
                                                      T* __restrict__ H, T* __restrict__ H2, int64_t ldh,
                                                      float* __restrict__ stats) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ntile = rpad / 16;
    const WaveRows wr = wave_rows(W, ntile);
    if (wr.b >= B) return;
    float* sk = smem + wave * attn_fwd_wave_floats(rpad);  // [rpad] keys
    float2* scm = (float2*)(sk + rpad);                       // [16 ATT_NT] row constants
    _Float16* sx = (_Float16*)(scm + 16 * ATT_NT);            // X^T: 3 rows x rpad (v hi, v lo, 1)
    const float* pv = P + wr.b * ldp;
    constexpr int KPL = 4 * KB;
    constexpr int RPL = RowsPerLane<NT>::value;
    float kr[KPL], vr[KPL], qr[RPL];
    load_keys<KPL>(pv, pv + 2 * r, r, lane, kr, vr);
    load_rows<RPL>(pv + r, r, wr.t0, 16 * NT, lane, qr);
    float kmin, kmax;
    key_range<KPL>(kr, r, lane, kmin, kmax);
    float vmax = 0.f;
#pragma unroll
    for (int u = 0; u < KPL; ++u) vmax = fmaxf(vmax, fabsf(vr[u]));
    const float vs = uniform_f(pow2_ceil(wave_max(vmax))), ivs = 1.0f / vs;  // exact: vs is a power of two
    const int ldx = rpad;
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        const int j = 64 * u + lane;
        if (j < rpad) {
            sk[j] = kr[u];
            put_pair(sx, ldx, 0, j, vr[u] * ivs);
            sx[xoff(2, j, ldx)] = (_Float16)(j < r ? 1.f : 0.f);
        }
    }
    const bool fast = put_row_consts<NT, RPL>(qr, lane, 16 * wr.nt, inv_tau, kmin, kmax, scm);
    __builtin_amdgcn_wave_barrier();
    const int g = lane >> 4, n = lane & 15;
    f32x4_t acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto chunks = [&](auto fast_c) {
        constexpr bool FAST = decltype(fast_c)::value;
        for (int j0 = 0; j0 < rpad; j0 += 32) {
            float kv[8];
            f16x4_t k0, k1;
            if (FAST) {
                k0 = key_frag(sk[j0 + n], g);
                k1 = key_frag(sk[j0 + 16 + n], g);
            } else {
                keys_perm(sk, j0, g, kv);
            }
            const f16x8_t a = xfrag_perm(sx, ldx, n, 3, j0, g);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                u32x4_t e;
                if (FAST) {
                    e = efrag_mfma(k0, k1, *(const f16x4_t*)(scm + 16 * t + n));
                } else {
                    const float2 cm = scm[16 * t + n];
                    e = efrag(cm.x, cm.y, kv);
                }
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, __builtin_bit_cast(f16x8_t, e), acc[t], 0, 0, 0);
            }
        }
    };
    if (fast) chunks(std::true_type{});
    else chunks(std::false_type{});
    if (lane < 16) {
        float* so = stats + wr.b * 2 * (int64_t)r;
        float vi[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {  // all loads first
            const int i = (wr.t0 + t) * 16 + lane;
            vi[t] = pv[i < r ? i : r - 1];
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int i = (wr.t0 + t) * 16 + lane;
            if (t < wr.nt && i < r) {
                const float z = acc[t].z;
                const float o = (acc[t].x + acc[t].y) * vs * __builtin_amdgcn_rcpf(z);
                const float hv = beta * vi[t] + alpha * o;
                st<T>::store(H + wr.b * ldh + i, hv);
                if (H2) st<T>::store(H2 + wr.b * ldh + i, hv - st<T>::round(hv));
                so[i] = o;
                so[r + i] = z;
            }
        }
    }
}

// LDS of the backward. Per sample (shared by its W waves): keys and X^T (4 rows).
// Per wave: row constants, Y^T (6 rows of the wave's rows), one 32 x 32 f16 block
// of e, and (W > 1) two column-partial slots.
__host__ __device__ constexpr int attn_bwd_sample_floats(int rpad) { return 3 * rpad; }
__host__ __device__ constexpr int attn_bwd_slot_offset() { return 2 * 16 * ATT_NT + 3 * (16 * ATT_NT) + 512; }
__host__ __device__ constexpr int attn_bwd_wave_floats(int W) { return attn_bwd_slot_offset() + (W > 1 ? 2 * 96 : 0); }
__host__ __device__ constexpr int attn_bwd_block_floats(int rpad, int W) {
    return (4 / W) * attn_bwd_sample_floats(rpad) + 4 * attn_bwd_wave_floats(W);
}

// ds_read_b64_tr_b16 of the e block: lane (g, i) receives e[8 g + t][16 h + i]
// for t = 0..7 (rows t < 4 from the first read, t >= 4 from the second). Block
// rows hold 32 keys as four 16-byte chunks, chunk index XOR ((row >> 2) & 3).
__device__ __forceinline__ f16x8_t e_transposed(const _Float16* se, int h, int lane) {
    const int g = lane >> 4, i = lane & 15;
    const int chunk = 2 * h + ((i & 3) >> 1);
    const int r0 = 8 * g + (i >> 2), r1 = r0 + 4;
    const int o0 = r0 * 32 + ((chunk ^ ((r0 >> 2) & 3)) * 8) + 4 * (i & 1);
    const int o1 = r1 * 32 + ((chunk ^ ((r1 >> 2) & 3)) * 8) + 4 * (i & 1);
    const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4_t*)(se + o0));
    const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4_t*)(se + o1));
    const s16x8_t v = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    return __builtin_bit_cast(f16x8_t, v);
}

// Backward. Row sums W1_i = sum_j e v_j k_j, W2_i = sum_j e k_j give
// dq_i = go_i / (Z_i tau) (W1_i - o_i W2_i); column sums C1_j = sum_i e a_i,
// C2_j = sum_i e a_i o_i, C3_j = sum_i e go_i / Z_i with a_i = go_i q_i / (Z_i tau)
// give dk_j = v_j C1_j - C2_j and dv_j = beta gh_j + C3_j (go = alpha gh).
template <typename T, int W, int NT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_attn_bwd_mfma(int64_t B, int r, int rpad, float alpha, float beta,
                                                      float inv_tau, const float* __restrict__ P, int64_t ldp,
                                                      const float* __restrict__ stats,
                                                      const float* __restrict__ GH, int64_t ldg,
                                                      T* __restrict__ GP, int64_t ldgp) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ntile = rpad / 16;
    const WaveRows wr = wave_rows(W, ntile);
    const bool live = wr.b < B;
    if (W == 1 && !live) return;  // with W > 1 every wave takes part in the barriers
    constexpr int RW = 16 * ATT_NT;
    float* sk = smem + (wave / W) * attn_bwd_sample_floats(rpad);  // [rpad] keys (shared by the sample's waves)
    _Float16* sx = (_Float16*)(sk + rpad);                           // 4 rows: v k hi/lo, k hi/lo
    float* pw = smem + (4 / W) * attn_bwd_sample_floats(rpad) + wave * attn_bwd_wave_floats(W);
    float2* scm = (float2*)pw;                   // [RW] row constants
    _Float16* sy = (_Float16*)(scm + RW);        // 6 rows: a hi/lo, a o hi/lo, go/Z hi/lo
    _Float16* se = sy + 6 * RW;                  // 32 x 32 e block
    const int ldx = rpad, ldy = RW;
    float* slot = pw + attn_bwd_slot_offset();   // 2 x 96 column partials (W > 1)
    const int g = lane >> 4, n = lane & 15;
    const int64_t b = live ? wr.b : 0;
    const float* pv = P + b * ldp;
    const float* pq = pv + r;
    const float* pk = pv + 2 * r;
    const float* gh = GH + b * ldg;
    const float* so = stats + b * 2 * (int64_t)r;
    constexpr int KPL = W == 1 ? 4 : 16;
    constexpr int RPL = RowsPerLane<NT>::value;
    float kr[KPL], vr[KPL], qr[RPL], ghr[RPL], orr[RPL], zr[RPL];
    load_keys<KPL>(pv, pk, r, lane, kr, vr);
    load_rows<RPL>(pq, r, wr.t0, 16 * wr.nt, lane, qr);
    load_rows<RPL>(gh, r, wr.t0, 16 * wr.nt, lane, ghr);
    load_rows<RPL>(so, r, wr.t0, 16 * wr.nt, lane, orr);
    load_rows<RPL>(so + r, r, wr.t0, 16 * wr.nt, lane, zr);
    // every wave reduces over all keys; each writes its share of the sample's key arrays
    float kmin, kmax;
    key_range<KPL>(kr, r, lane, kmin, kmax);
    float mvk = 0.f, mk = 0.f;
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        mvk = fmaxf(mvk, fabsf(vr[u] * kr[u]));
        mk = fmaxf(mk, fabsf(kr[u]));
    }
    const float vks = uniform_f(pow2_ceil(wave_max(mvk))), ks = uniform_f(pow2_ceil(wave_max(mk)));
    const float ivks = 1.0f / vks, iks = 1.0f / ks;  // exact: powers of two
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        const int j = 64 * u + lane;
        if (j < rpad && u % W == wr.w) {
            sk[j] = kr[u];
            put_pair(sx, ldx, 0, j, vr[u] * kr[u] * ivks);
            put_pair(sx, ldx, 2, j, kr[u] * iks);
        }
    }
    // per-row coefficients of the wave's rows (zero past its rows)
    float ca[RPL], cb[RPL], cg[RPL];
    float ma = 0.f, mb = 0.f, mc = 0.f;
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        const float go = alpha * ghr[u], rz = zr[u] != 0.f ? __builtin_amdgcn_rcpf(zr[u]) : 0.f;
        ca[u] = go * qr[u] * rz * inv_tau;
        cb[u] = ca[u] * orr[u];
        cg[u] = go * rz;
        ma = fmaxf(ma, fabsf(ca[u]));
        mb = fmaxf(mb, fabsf(cb[u]));
        mc = fmaxf(mc, fabsf(cg[u]));
    }
    const float as = uniform_f(pow2_ceil(wave_max(ma))), bs = uniform_f(pow2_ceil(wave_max(mb)));
    const float cs = uniform_f(pow2_ceil(wave_max(mc)));
    const float ias = 1.0f / as, ibs = 1.0f / bs, ics = 1.0f / cs;  // exact: powers of two
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        const int il = 64 * u + lane;
        if (il < 16 * NT) {
            put_pair(sy, ldy, 0, il, ca[u] * ias);
            put_pair(sy, ldy, 2, il, cb[u] * ibs);
            put_pair(sy, ldy, 4, il, cg[u] * ics);
        }
    }
    // row constants from q (load_rows zeroed q past the wave's rows; rows of
    // other waves only feed discarded tiles)
    const bool fast = put_row_consts<NT, RPL>(qr, lane, 16 * wr.nt, inv_tau, kmin, kmax, scm);
    if (W > 1) __syncthreads();
    else __builtin_amdgcn_wave_barrier();

    f32x4_t acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto chunks = [&](auto fast_c) {
        constexpr bool FAST = decltype(fast_c)::value;
        for (int chunk = 0, j0 = 0; j0 < rpad; j0 += 32, ++chunk) {
            float kv[8];
            f16x4_t k0, k1;
            if (FAST) {
                k0 = key_frag(sk[j0 + n], g);
                k1 = key_frag(sk[j0 + 16 + n], g);
            } else {
                keys_perm(sk, j0, g, kv);
            }
            const f16x8_t ax = xfrag_perm(sx, ldx, n, 4, j0, g);
            // operands of this chunk's column epilogue, loaded now so the loads overlap the chunk
            float ev[2], eg[2];
    #pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int j = W == 1 ? j0 + 16 * h + n : j0 + (lane & 31);
                const int jc = j < r ? j : r - 1;
                ev[h] = pv[jc];
                eg[h] = gh[jc];
            }
            f32x4_t col[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
    #pragma unroll
            for (int p = 0; p < NT / 2; ++p) {
                // the wave's LDS operations run in order, so this pair's writes follow
                // the previous pair's transposed reads of the same block
                __builtin_amdgcn_wave_barrier();
    #pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int t = 2 * p + q;
                    u32x4_t e;
                    if (FAST) {
                        e = efrag_mfma(k0, k1, *(const f16x4_t*)(scm + 16 * t + n));
                    } else {
                        const float2 cm = scm[16 * t + n];
                        e = efrag(cm.x, cm.y, kv);
                    }
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ax, __builtin_bit_cast(f16x8_t, e), acc[t], 0, 0, 0);
                    // keys 4 g .. +3 and 16 + 4 g .. +3 of row 16 q + n, into their block chunks
                    const int row = 16 * q + n, sw = (row >> 2) & 3;
                    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
                    *(u32x2_t*)(se + row * 32 + (((g >> 1) ^ sw) * 8) + 4 * (g & 1)) = u32x2_t{e.x, e.y};
                    *(u32x2_t*)(se + row * 32 + (((2 + (g >> 1)) ^ sw) * 8) + 4 * (g & 1)) = u32x2_t{e.z, e.w};
                }
                const f16x8_t ay = xfrag(sy, ldy, n, 6, 32 * p + 8 * g);
    #pragma unroll
                for (int h = 0; h < 2; ++h)
                    col[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ay, e_transposed(se, h, lane), col[h], 0, 0, 0);
            }
            // lanes 0..15: (a hi, a lo, a o hi, a o lo) of key n (+16 h); lanes 16..31: (go/Z hi, lo)
            if (W == 1) {
                if (lane < 32) {
    #pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int j = j0 + 16 * h + n;
                        if (j < r) {
                            if (lane < 16) {
                                const float c1 = (col[h].x + col[h].y) * as, c2 = (col[h].z + col[h].w) * bs;
                                st<T>::store(GP + b * ldgp + 2 * r + j, ev[h] * c1 - c2);
                            } else {
                                st<T>::store(GP + b * ldgp + j, beta * eg[h] + (col[h].x + col[h].y) * cs);
                            }
                        }
                    }
                }
            } else {
                float* sl = slot + (chunk & 1) * 96;
                if (lane < 32) {
    #pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        if (lane < 16) {
                            sl[16 * h + n] = (col[h].x + col[h].y) * as;
                            sl[32 + 16 * h + n] = (col[h].z + col[h].w) * bs;
                        } else {
                            sl[64 + 16 * h + n] = (col[h].x + col[h].y) * cs;
                        }
                    }
                }
                __syncthreads();
                // the sample's first wave adds the W partials in wave order
                if (live && wr.w == 0 && lane < 32) {
                    const int j = j0 + lane;
                    float c1 = 0.f, c2 = 0.f, c3 = 0.f;
    #pragma unroll
                    for (int w = 0; w < W; ++w) {
                        const float* so2 = smem + (4 / W) * attn_bwd_sample_floats(rpad) +
                                           (wave + w) * attn_bwd_wave_floats(W) + attn_bwd_slot_offset() + (chunk & 1) * 96;
                        c1 += so2[lane];
                        c2 += so2[32 + lane];
                        c3 += so2[64 + lane];
                    }
                    if (j < r) {
                        st<T>::store(GP + b * ldgp + 2 * r + j, ev[0] * c1 - c2);
                        st<T>::store(GP + b * ldgp + j, beta * eg[0] + c3);
                    }
                }
            }
        }
    };
    if (fast) chunks(std::true_type{});
    else chunks(std::false_type{});
    if (live && lane < 16) {
        float gi[NT], oi[NT], zi[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {  // all loads first
            const int i = (wr.t0 + t) * 16 + lane, ic = i < r ? i : r - 1;
            gi[t] = gh[ic];
            oi[t] = so[ic];
            zi[t] = so[r + ic];
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int i = (wr.t0 + t) * 16 + lane;
            if (t < wr.nt && i < r) {
                const float w1 = (acc[t].x + acc[t].y) * vks, w2 = (acc[t].z + acc[t].w) * ks;
                const float go = alpha * gi[t], rz = __builtin_amdgcn_rcpf(zi[t]);
                st<T>::store(GP + b * ldgp + r + i, go * rz * inv_tau * (w1 - oi[t] * w2));
            }
        }
    }
}

int attn_threads(int r) {
    int t = ((r + 63) / 64) * 64;
    return t > 256 ? 256 : t;
}

}  // namespace

// waves per sample: 1, 2 or 4 (a workgroup of 4 waves holds whole samples)
static int attn_waves(int rpad) {
    const int ntile = rpad / 16;
    return ntile <= ATT_NT ? 1 : ntile <= 2 * ATT_NT ? 2 : 4;
}
// tiles computed per wave: the power of two (>= 2) covering the tiles one wave owns
static int attn_tiles(int rpad, int W) {
    const int ntile = rpad / 16;
    const int per = (((ntile + W - 1) / W) + 1) & ~1;
    int nt = 2;
    while (nt < per) nt *= 2;
    return nt;
}

hipError_t launch_attn_fwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp, void* H,
                           void* H2, int64_t ldh, float* stats, bool bf16, hipStream_t s) {
    if (B == 0) return hipSuccess;
    if (bf16) {
        if (r > 4 * 16 * ATT_NT || !stats) return hipErrorInvalidValue;
        const int rpad = (r + 31) / 32 * 32;
        const int W = attn_waves(rpad);
        const int NT = attn_tiles(rpad, W);
        const int64_t blocks = (B * W + 3) / 4;
        const size_t lds = 4 * sizeof(float) * (size_t)attn_fwd_wave_floats(rpad);
#define RDCN_AFWD(NTV, KBV)                                                                                          \
    hipLaunchKernelGGL((k_attn_fwd_mfma<bf16_t, NTV, KBV>), dim3((unsigned)blocks), dim3(256), lds, s, B, r, rpad, W, \
                       alpha, beta, 1.0f / tau, (const float*)P, ldp, (bf16_t*)H, (bf16_t*)H2, ldh, stats)
        if (NT == 2) RDCN_AFWD(2, 1);
        else if (NT == 4) RDCN_AFWD(4, 1);
        else if (NT == 8) RDCN_AFWD(8, 1);
        else if (W == 1) RDCN_AFWD(16, 1);
        else RDCN_AFWD(16, 4);
#undef RDCN_AFWD
        return hipGetLastError();
    }
    const size_t lds = sizeof(float) * (2 * (size_t)r + 32);
    const int th = attn_threads(r);
    hipLaunchKernelGGL(k_attn_fwd<float>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                       (const float*)P, ldp, (float*)H, (float*)H2, ldh);
    return hipGetLastError();
}

hipError_t launch_attn_bwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp,
                           const float* stats, const float* GH, int64_t ldg, void* GP, int64_t ldgp, bool bf16,
                           hipStream_t s) {
    if (B == 0) return hipSuccess;
    if (bf16) {
        if (r > 4 * 16 * ATT_NT || !stats) return hipErrorInvalidValue;
        const int rpad = (r + 31) / 32 * 32;
        const int W = attn_waves(rpad);
        const int NT = attn_tiles(rpad, W);
        const int64_t blocks = (B * W + 3) / 4;
        const size_t lds = sizeof(float) * (size_t)attn_bwd_block_floats(rpad, W);
#define RDCN_ABWD(WV, NTV)                                                                                          \
    hipLaunchKernelGGL((k_attn_bwd_mfma<bf16_t, WV, NTV>), dim3((unsigned)blocks), dim3(256), lds, s, B, r, rpad,     \
                       alpha, beta, 1.0f / tau, (const float*)P, ldp, stats, GH, ldg, (bf16_t*)GP, ldgp)
        if (W == 1) {
            if (NT == 2) RDCN_ABWD(1, 2);
            else if (NT == 4) RDCN_ABWD(1, 4);
            else if (NT == 8) RDCN_ABWD(1, 8);
            else RDCN_ABWD(1, 16);
        } else if (W == 2) {
            if (NT == 8) RDCN_ABWD(2, 8);
            else RDCN_ABWD(2, 16);
        } else {
            if (NT == 8) RDCN_ABWD(4, 8);
            else RDCN_ABWD(4, 16);
        }
#undef RDCN_ABWD
        return hipGetLastError();
    }
    const size_t lds = sizeof(float) * (7 * (size_t)r + 32);
    const int th = attn_threads(r);
    hipLaunchKernelGGL(k_attn_bwd<float>, dim3((unsigned)B), dim3(th), lds, s, B, r, alpha, beta, 1.0f / tau,
                       (const float*)P, ldp, GH, ldg, (float*)GP, ldgp);
    return hipGetLastError();
}

}  // namespace rdcn
