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
// sum over them runs on the matrix cores. For a 32-row x 32-key block of one
// sample, one v_mfma_f32_32x32x8_f16 leaves each lane 16 values e_ij of its row
// i = lane % 32, 8 of which form the B operand of a v_mfma_f32_16x16x32_f16 with
// K running over 16 keys (rows n and n + 16 share its columns and go to output
// slots 0-7 and 8-15; the A operand is zero in the other half); the A operand is a small
// per-sample matrix X^T whose rows are the quantities summed against e (v, 1,
// v k, k), each stored as an f16 hi + lo pair scaled by a power of two so the
// pair keeps about 21 significant bits. e itself is rounded to f16 (relative
// 2^-11); all sums of one row use the same rounded e, so the normalisation by Z
// is consistent. Output lane l holds quantities 4 (l / 16 % 2) .. +3 of row
// l % 16 (+16 for l >= 32).
//
// In the forward one wave owns up to ATT_NT 16-row tiles of one sample and loops
// over all keys, so row sums never leave its registers; a sample with more rows
// is split over W = ceil(tiles / ATT_NT) waves of one workgroup, which share the
// sample's keys and X^T in LDS.
//
// The forward saves each row's o_i and Z_i and, from the same MFMAs (four more
// rows of X^T), the two row sums the query gradient needs. The backward is then
// left with column sums only (over rows, weighted by per-row coefficients that
// depend on o_i and Z_i): it computes the exponent arguments with the forward's
// product transposed (row records as the A operand, key fragments as B), which
// hands every lane the e values of one key for 16 rows: B operands with K
// running over rows. No e_ij is stored or exchanged between lanes.
// ---------------------------------------------------------------------------
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int ATT_NT = 16;  // 16-row tiles per wave
// 16-key tiles the backward carries through one pass over a sample's rows (four:
// the row records and Y^T fragment read per 32-row block serve 64 keys; eight spill)
constexpr int ATT_BWD_KT = 4;

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

// Key order inside one 32-key chunk of the FMA (slow) path. Lane (g, n)'s 8 K slots
// of a fragment hold keys j0 + 4 g + t (t < 4) and j0 + 16 + 4 g + (t - 4) (t >= 4).
// Everything indexed by key within a chunk (X^T fragments, the lane's keys) follows
// it; sums over K do not depend on the order.
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

// Exponent arguments on the matrix cores: x = c k + m as a 32 (keys) x 32 (rows)
// product with K = 5 of 8 slots used, from f16 hi + lo parts of c, k and m:
//   keys (lane half g, key l % 32):   g = 0: (k_hi, k_hi, 1, 1)   g = 1: (k_lo, 0, 0, 0)
//   rows (lane half g, row l % 32):   (c_hi, c_lo, m_hi, m_lo) for both halves
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

// X^T fragment of row n (< nx, else zero) for the chunk at j0, keys in the order above.
__device__ __forceinline__ f16x8_t xfrag_perm(const _Float16* sx, int ld, int n, int nx, int j0, int g) {
    if (n >= nx) return f16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    const f16x4_t lo = *(const f16x4_t*)(sx + xoff(n, j0 + 4 * g, ld));
    const f16x4_t hi = *(const f16x4_t*)(sx + xoff(n, j0 + 16 + 4 * g, ld));
    return f16x8_t{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
}

typedef float f32x16_t __attribute__((ext_vector_type(16)));

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

// (c_i, m_i) = (q_i log2(e) / tau, -c_i k*_i) of rows 64 u + lane (rows past r hold
// q = 0, so c = m = 0), and the largest |c|, |m| over rows below nrows together with
// the key range (wave-uniform). The exponent arguments go through the matrix cores
// when that maximum stays below ATT_F16_SAFE.
template <int RPL>
__device__ __forceinline__ float row_consts(const float (&q)[RPL], int lane, int nrows, float inv_tau, float kmin,
                                            float kmax, float (&c)[RPL], float (&m)[RPL]) {
    float big = fmaxf(fabsf(kmin), fabsf(kmax));
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        c[u] = q[u] * (LOG2E * inv_tau);
        m[u] = -(c[u] * (c[u] >= 0.f ? kmax : kmin));
        if (64 * u + lane < nrows) big = fmaxf(big, fmaxf(fabsf(c[u]), fabsf(m[u])));
    }
    return wave_max(big);
}

// Largest of the W per-wave values in the sample's slots (each wave wrote slot[k] of
// its own area at stride `stride` floats; slot0 is the first wave's area).
template <int W>
__device__ __forceinline__ float sample_max(const float* slot0, int stride, int k) {
    float x = slot0[k];
#pragma unroll
    for (int w = 1; w < W; ++w) x = fmaxf(x, slot0[w * stride + k]);
    return x;
}

// X^T of the forward: f16 hi + lo pairs of quantities summed against e, row stride
// rpad. Quantity rows (the MFMA's M index): 0, 1: v / vs; 2: 1 for the real keys;
// 3: zero (not stored); 4, 5: v k / vks; 6, 7: k / ks. Output lanes 0-15 get
// (sum e v, sum e) for o and Z, lanes 16-31 the backward's row sums
// W1 = sum_j e v_j k_j and W2 = sum_j e k_j, from the same MFMAs.
constexpr int ATT_XROWS = 7;
__device__ __forceinline__ int xrow(int n) { return n < 3 ? n : n - 1; }
__device__ __forceinline__ f16x8_t xfrag_fwd(const _Float16* sx, int ld, int n, int j0, int g) {
    if (n == 3 || n > 7) return f16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    return xfrag_perm(sx, ld, xrow(n), ATT_XROWS, j0, g);
}

// Exponent arguments of 32 keys x 32 rows from one v_mfma_f32_32x32x8_f16 (the key
// and row records of key_frag / row_rec use only 8 K slots): lane l gets row l % 32 and
// keys 8 a + 4 (l / 32) + t in element 4 a + t. Elements 8 p .. 8 p + 7 are the B
// operand of a 16x16x32 weighted sum over keys 16 p .. 16 p + 15 whose columns are
// rows n (lanes 0-15, 32-47) and n + 16 (lanes 16-31, 48-63): frag32 gives the
// quantities of row n to output slots 0-7 and those of row n + 16 to slots 8-15.
// X^T fragment for such a sum at keys jb .. jb + 15: lane (g4, q) with q % 8 a
// quantity row (row 3 and rows of the other half read as zero).
__device__ __forceinline__ f16x8_t frag32(const _Float16* sx, int ld, int lane, int jb) {
    const int qs = lane & 15, g4 = lane >> 4, q = qs & 7, h = g4 >> 1;
    if ((qs >> 3) != (g4 & 1) || q == 3) return f16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    const int row = xrow(q);
    const f16x4_t lo = *(const f16x4_t*)(sx + xoff(row, jb + 4 * h, ld));
    const f16x4_t hi = *(const f16x4_t*)(sx + xoff(row, jb + 8 + 4 * h, ld));
    return f16x8_t{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
}

// LDS of the forward. Per sample (shared by its W waves): keys, X^T. Per wave: row
// constants and one slot for the range check.
__host__ __device__ constexpr int attn_fwd_sample_floats(int rpad) { return rpad + ATT_XROWS * rpad / 2; }
__host__ __device__ constexpr int attn_fwd_wave_floats() { return 2 * 16 * ATT_NT + 4; }
__host__ __device__ constexpr int attn_fwd_block_floats(int rpad, int W) {
    return (4 / W) * attn_fwd_sample_floats(rpad) + 4 * attn_fwd_wave_floats();
}

// NT: tiles computed per wave (a power of two >= the tiles it owns; the extra ones
// are computed on harmless row constants and discarded).
// KB: 256-key batches a lane's registers cover (4 KB >= rpad / 64).
// stats: [o | Z | W1 | W2] per sample, row stride 4 r.
template <typename T, int W, int NT, int KB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_attn_fwd_mfma(int64_t B, int r, int rpad, float alpha, float beta,
                                                      float inv_tau, const float* __restrict__ P, int64_t ldp,
                                                      T* __restrict__ H, void* __restrict__ H2, int64_t ldh,
                                                      bool h2_f16, float* __restrict__ stats, int* err) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ntile = rpad / 16;
    const WaveRows wr = wave_rows(W, ntile);
    const bool live = wr.b < B;
    if (W == 1 && !live) return;  // with W > 1 every wave takes part in the barriers
    float* sk = smem + (wave / W) * attn_fwd_sample_floats(rpad);  // [rpad] keys (shared by the sample's waves)
    _Float16* sx = (_Float16*)(sk + rpad);                           // X^T (ATT_XROWS stored rows)
    float* pw = smem + (4 / W) * attn_fwd_sample_floats(rpad);
    float2* scm = (float2*)(pw + wave * attn_fwd_wave_floats());   // [16 ATT_NT] row constants
    float* slot = pw + wave * attn_fwd_wave_floats() + 2 * 16 * ATT_NT;
    const int64_t b = live ? wr.b : 0;
    const float* pv = P + b * ldp;
    constexpr int KPL = 4 * KB;
    constexpr int RPL = RowsPerLane<NT>::value;
    float kr[KPL], vr[KPL], qr[RPL];
    load_keys<KPL>(pv, pv + 2 * r, r, lane, kr, vr);
    load_rows<RPL>(pv + r, r, wr.t0, 16 * NT, lane, qr);
    float kmin, kmax;
    key_range<KPL>(kr, r, lane, kmin, kmax);
    float vmax = 0.f, mvk = 0.f, mk = 0.f;
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        vmax = fmaxf(vmax, fabsf(vr[u]));
        mvk = fmaxf(mvk, fabsf(vr[u] * kr[u]));
        mk = fmaxf(mk, fabsf(kr[u]));
    }
    // exact scalings: powers of two, identical in every wave of the sample (all see all keys)
    const float vs = uniform_f(pow2_ceil(wave_max(vmax))), ivs = 1.0f / vs;
    const float vks = uniform_f(pow2_ceil(wave_max(mvk))), ivks = 1.0f / vks;
    const float ks = uniform_f(pow2_ceil(wave_max(mk))), iks = 1.0f / ks;
    const int ldx = rpad;
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        const int j = 64 * u + lane;
        if (j < rpad && u % W == wr.w) {
            sk[j] = kr[u];
            put_pair(sx, ldx, 0, j, vr[u] * ivs);
            sx[xoff(2, j, ldx)] = (_Float16)(j < r ? 1.f : 0.f);
            put_pair(sx, ldx, xrow(4), j, vr[u] * kr[u] * ivks);
            put_pair(sx, ldx, xrow(6), j, kr[u] * iks);
        }
    }
    float c[RPL], m[RPL];
    float big = row_consts<RPL>(qr, lane, 16 * wr.nt, inv_tau, kmin, kmax, c, m);
    if (W > 1) {  // one decision per sample, as in the backward
        if (lane == 0) slot[0] = big;
        __syncthreads();
        big = uniform_f(sample_max<W>(pw + (wave - wr.w) * attn_fwd_wave_floats() + 2 * 16 * ATT_NT,
                                      attn_fwd_wave_floats(), 0));
    }
    const bool fast = big < ATT_F16_SAFE;  // false for NaN too
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
        const int il = 64 * u + lane;
        if (il < 16 * NT) {
            if (fast) *(f16x4_t*)(scm + il) = row_rec(c[u], m[u]);
            else scm[il] = make_float2(c[u], m[u]);
        }
    }
    if (W > 1) __syncthreads();
    else __builtin_amdgcn_wave_barrier();
    const int g = lane >> 4, n = lane & 15;
    f32x4_t acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto chunks = [&](auto fast_c) {
        constexpr bool FAST = decltype(fast_c)::value;
        for (int j0 = 0; j0 < rpad; j0 += 32) {
            if (FAST) {
                // 32-row tiles: acc[tt] holds rows 32 tt + n (lanes 0-31) and 32 tt + 16 + n
                const f16x4_t kf = key_frag(sk[j0 + (lane & 31)], lane >> 5);
                const f16x8_t a0 = frag32(sx, ldx, lane, j0), a1 = frag32(sx, ldx, lane, j0 + 16);
                const f32x16_t z16 = {};
                // the next tile's arguments are issued before this tile's exponentials, so
                // the matrix core computes them while the wave's exponentials run
                f32x16_t xn = __builtin_amdgcn_mfma_f32_32x32x8f16(kf, *(const f16x4_t*)(scm + (lane & 31)), z16, 0, 0, 0);
#pragma unroll
                for (int tt = 0; tt < NT / 2; ++tt) {
                    const f32x16_t x = xn;
                    if (tt + 1 < NT / 2) {
                        const f16x4_t rec = *(const f16x4_t*)(scm + 32 * (tt + 1) + (lane & 31));
                        xn = __builtin_amdgcn_mfma_f32_32x32x8f16(kf, rec, z16, 0, 0, 0);
                    }
                    float e0[8], e1[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        e0[u] = __builtin_amdgcn_exp2f(x[u]);
                        e1[u] = __builtin_amdgcn_exp2f(x[8 + u]);
                    }
                    acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, __builtin_bit_cast(f16x8_t, pack_e(e0)), acc[tt], 0, 0, 0);
                    acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, __builtin_bit_cast(f16x8_t, pack_e(e1)), acc[tt], 0, 0, 0);
                }
            } else {
                float kv[8];
                keys_perm(sk, j0, g, kv);
                const f16x8_t a = xfrag_fwd(sx, ldx, n, j0, g);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const float2 cm = scm[16 * t + n];
                    const u32x4_t e = efrag(cm.x, cm.y, kv);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, __builtin_bit_cast(f16x8_t, e), acc[t], 0, 0, 0);
                }
            }
        }
    };
    if (fast) chunks(std::true_type{});
    else chunks(std::false_type{});
    // Which row and quantities each lane's accumulators hold. Fast path: 32-row tiles,
    // lane (g4, n) has quantities 4 (g4 & 1) .. +3 of row 16 (2 t + g4 / 2) + n. Slow
    // path: 16-row tiles, lanes 0-31 only, quantities 4 (lane / 16) .. +3 of row 16 t + n.
    const int na = fast ? NT / 2 : NT;
    const bool act = fast || lane < 32;
    const bool lo = fast ? ((lane >> 4) & 1) == 0 : lane < 16;
    if (live && act) {
        // lo lanes: (sum e v, sum e) of their row -> h, o, Z; the others: (W1, W2)
        float* so = stats + b * 4 * (int64_t)r;
        float vi[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {  // all loads first
            const int t16 = fast ? 2 * t + (lane >> 5) : t;
            const int i = (wr.t0 + t16) * 16 + n;
            vi[t] = pv[i < r ? i : r - 1];
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int t16 = fast ? 2 * t + (lane >> 5) : t;
            const int i = (wr.t0 + t16) * 16 + n;
            if (t < na && t16 < wr.nt && i < r) {
                const float s01 = acc[t].x + acc[t].y, z = acc[t].z;
                const float o = s01 * vs * __builtin_amdgcn_rcpf(z);
                if (lo) {
                    const float hv = beta * vi[t] + alpha * o;
                    st<T>::store(H + b * ldh + i, hv);
                    if (H2 && h2_f16) {  // h as f16, the up projection's operand
                        ((_Float16*)H2)[b * ldh + i] = (_Float16)hv;
                        if (fabsf(hv) >= F16_OVERFLOW) atomicOr(err, 2);  // f16 range bit of the error word
                    } else if (H2) {     // lo part of a hi + lo pair
                        st<T>::store((T*)H2 + b * ldh + i, hv - st<T>::round(hv));
                    }
                }
                so[(lo ? 0 : 2 * r) + i] = lo ? o : s01 * vks;
                so[(lo ? r : 3 * r) + i] = lo ? z : (z + acc[t].w) * ks;
            }
        }
    }
}

// LDS of the backward, per sample (shared by its W waves): keys, row constants (8
// bytes per row), Y^T (6 rows of f16 and two rows of zeros, row stride rpad); per
// wave four slots for the range check and the three scales.
__host__ __device__ constexpr int attn_bwd_sample_floats(int rpad) { return rpad + 2 * rpad + 4 * rpad; }

// The backward's Y^T fragment, laid out as frag32's with K over rows and the 6
// quantity rows stored as they are. Every lane loads: the lanes whose slots hold no
// quantity (the other half's, and quantities 6 and 7) read row 7, which holds zeros,
// so the fragment needs no per-lane branches.
__device__ __forceinline__ f16x8_t yfrag32(const _Float16* sy, int ld, int lane, int jb) {
    const int qs = lane & 15, g4 = lane >> 4, q = qs & 7, h = g4 >> 1;
    const int row = ((qs >> 3) != (g4 & 1) || q >= 6) ? 7 : q;
    const f16x4_t lo = *(const f16x4_t*)(sy + xoff(row, jb + 4 * h, ld));
    const f16x4_t hi = *(const f16x4_t*)(sy + xoff(row, jb + 8 + 4 * h, ld));
    return f16x8_t{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
}
__host__ __device__ constexpr int attn_bwd_wave_floats() { return 4; }
__host__ __device__ constexpr int attn_bwd_block_floats(int rpad, int W) {
    return (4 / W) * attn_bwd_sample_floats(rpad) + 4 * attn_bwd_wave_floats();
}

// Backward. With the forward's row sums W1 and W2, dq_i = go_i / (Z_i tau) (W1_i - o_i W2_i)
// needs no exponentials. The column sums C1_j = sum_i e_ij a_i, C2_j = sum_i e_ij a_i o_i,
// C3_j = sum_i e_ij go_i / Z_i (a_i = go_i q_i / (Z_i tau)) give dk_j = v_j C1_j - C2_j and
// dv_j = beta gh_j + C3_j (go = alpha gh). They run on the matrix cores with K over rows:
// the exponent arguments come out of v_mfma_f32_32x32x8_f16 with the row records as A
// and the key fragments as B (the forward's product with its operands swapped, so each
// e_ij is computed exactly as in the forward), which leaves lane l holding e of key
// l % 32 for 16 rows of a 32-row block: the B operands of two v_mfma_f32_16x16x32_f16
// against Y^T (rows: a hi, a lo, a o hi, a o lo, go/Z hi, lo), keys n and n + 16 in
// output slots 0-7 and 8-15 (frag32).
// A sample's waves split its keys (16 ATT_BWD_KT at a time); every wave runs over all rows.
template <typename T, int W, int KB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_attn_bwd_mfma(int64_t B, int r, int rpad, float alpha, float beta,
                                                      float inv_tau, const float* __restrict__ P, int64_t ldp,
                                                      const float* __restrict__ stats,
                                                      const float* __restrict__ GH, int64_t ldg,
                                                      T* __restrict__ GP, int64_t ldgp) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t gw = (int64_t)blockIdx.x * 4 + wave;
    const int64_t bsm = gw / W;
    const int w = __builtin_amdgcn_readfirstlane((int)(gw - bsm * W));
    const bool live = bsm < B;
    if (W == 1 && !live) return;  // with W > 1 every wave takes part in the barriers
    const int64_t b = live ? bsm : 0;
    float* sk = smem + (wave / W) * attn_bwd_sample_floats(rpad);  // [rpad] keys
    float2* scm = (float2*)(sk + rpad);                              // [rpad] row constants
    _Float16* sy = (_Float16*)(scm + rpad);                          // Y^T, 6 rows
    float* slots = smem + (4 / W) * attn_bwd_sample_floats(rpad);
    float* slot = slots + wave * attn_bwd_wave_floats();
    const int ldy = rpad;
    const float* pv = P + b * ldp;
    const float* pq = pv + r;
    const float* pk = pv + 2 * r;
    const float* gh = GH + b * ldg;
    const float* so = stats + b * 4 * (int64_t)r;
    constexpr int KPL = 4 * KB;      // keys (and rows) per lane: 64 KPL >= rpad
    constexpr int RPW = KPL / W;     // rows per lane of this wave's share: 64 (s W + w) + lane
    float kr[KPL];
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        const int j = 64 * u + lane;
        kr[u] = pk[j < r ? j : r - 1];
    }
#pragma unroll
    for (int u = 0; u < KPL; ++u)
        if (64 * u + lane >= r) kr[u] = 0.f;
    float kmin, kmax;
    key_range<KPL>(kr, r, lane, kmin, kmax);
    // this wave's rows: the forward's statistics, dq, and the column-sum coefficients
    float qr[RPW], ghr[RPW], orr[RPW], zr[RPW], w1[RPW], w2[RPW];
#pragma unroll
    for (int s = 0; s < RPW; ++s) {
        const int i = 64 * (s * W + w) + lane, ic = i < r ? i : r - 1;
        qr[s] = pq[ic];
        ghr[s] = gh[ic];
        orr[s] = so[ic];
        zr[s] = so[r + ic];
        w1[s] = so[2 * r + ic];
        w2[s] = so[3 * r + ic];
    }
    float ca[RPW], cb[RPW], cg[RPW], c[RPW], m[RPW];
    float big = fmaxf(fabsf(kmin), fabsf(kmax)), ma = 0.f, mb = 0.f, mc = 0.f;
#pragma unroll
    for (int s = 0; s < RPW; ++s) {
        const int i = 64 * (s * W + w) + lane;
        const bool ok = i < r;
        const float q = ok ? qr[s] : 0.f, go = ok ? alpha * ghr[s] : 0.f;
        const float rz = ok && zr[s] != 0.f ? __builtin_amdgcn_rcpf(zr[s]) : 0.f;
        if (live && ok) st<T>::store(GP + b * ldgp + r + i, go * rz * inv_tau * (w1[s] - orr[s] * w2[s]));
        ca[s] = go * q * rz * inv_tau;
        cb[s] = ca[s] * orr[s];
        cg[s] = go * rz;
        c[s] = q * (LOG2E * inv_tau);
        m[s] = -(c[s] * (c[s] >= 0.f ? kmax : kmin));
        if (ok) big = fmaxf(big, fmaxf(fabsf(c[s]), fabsf(m[s])));
        ma = fmaxf(ma, fabsf(ca[s]));
        mb = fmaxf(mb, fabsf(cb[s]));
        mc = fmaxf(mc, fabsf(cg[s]));
    }
    big = wave_max(big);
    ma = wave_max(ma);
    mb = wave_max(mb);
    mc = wave_max(mc);
    if (W > 1) {  // maxima over the sample's rows
        if (lane == 0) {
            slot[0] = big;
            slot[1] = ma;
            slot[2] = mb;
            slot[3] = mc;
        }
        __syncthreads();
        const float* s0 = slots + (wave - w) * attn_bwd_wave_floats();
        big = sample_max<W>(s0, attn_bwd_wave_floats(), 0);
        ma = sample_max<W>(s0, attn_bwd_wave_floats(), 1);
        mb = sample_max<W>(s0, attn_bwd_wave_floats(), 2);
        mc = sample_max<W>(s0, attn_bwd_wave_floats(), 3);
    }
    const bool fast = uniform_f(big) < ATT_F16_SAFE;  // the forward's decision (false for NaN too)
    const float as = uniform_f(pow2_ceil(ma)), bs = uniform_f(pow2_ceil(mb)), cs = uniform_f(pow2_ceil(mc));
    const float ias = 1.0f / as, ibs = 1.0f / bs, ics = 1.0f / cs;  // exact: powers of two
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
        const int j = 64 * u + lane;
        if (j < rpad && u % W == w) sk[j] = kr[u];
    }
#pragma unroll
    for (int s = 0; s < RPW; ++s) {
        const int i = 64 * (s * W + w) + lane;
        if (i < rpad) {
            if (fast) *(f16x4_t*)(scm + i) = row_rec(c[s], m[s]);
            else scm[i] = make_float2(c[s], m[s]);
            put_pair(sy, ldy, 0, i, ca[s] * ias);
            put_pair(sy, ldy, 2, i, cb[s] * ibs);
            put_pair(sy, ldy, 4, i, cg[s] * ics);
            sy[xoff(6, i, ldy)] = (_Float16)0.f;
            sy[xoff(7, i, ldy)] = (_Float16)0.f;
        }
    }
    if (W > 1) __syncthreads();
    else __builtin_amdgcn_wave_barrier();
    if (!live) return;

    const int g = lane >> 4, n = lane & 15;
    constexpr int KT = ATT_BWD_KT;
    // Fast path: 32-key blocks. Arguments of 32 rows x 32 keys from one 32x32x8 MFMA
    // (row records as A, key records as B: lane l gets key l % 32), then two column
    // sums per block whose output lane (g4, n) holds quantities 4 (g4 & 1) .. +3 of
    // key n + 16 (g4 / 2).
    auto keys32 = [&]() {
        constexpr int KB2 = KT / 2;
        for (int j0 = 16 * KT * w; j0 < rpad; j0 += 16 * KT * W) {
            f16x4_t kf[KB2];
            float ev[KB2], eg[KB2];
#pragma unroll
            for (int q = 0; q < KB2; ++q) {
                const int jl = j0 + 32 * q + (lane & 31), jp = jl < rpad ? jl : rpad - 1;
                kf[q] = key_frag(sk[jp], lane >> 5);
                const int j = j0 + 32 * q + n + 16 * (lane >> 5), jc = j < r ? j : r - 1;
                ev[q] = pv[jc];
                eg[q] = gh[jc];
            }
            f32x4_t col[KB2];
#pragma unroll
            for (int q = 0; q < KB2; ++q) col[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            const f32x16_t z16 = {};
            for (int i0 = 0; i0 < rpad; i0 += 32) {
                const f16x4_t rec = *(const f16x4_t*)(scm + i0 + (lane & 31));
                const f16x8_t y0 = yfrag32(sy, ldy, lane, i0), y1 = yfrag32(sy, ldy, lane, i0 + 16);
                f32x16_t x[KB2];
#pragma unroll
                for (int q = 0; q < KB2; ++q) x[q] = __builtin_amdgcn_mfma_f32_32x32x8f16(rec, kf[q], z16, 0, 0, 0);
#pragma unroll
                for (int q = 0; q < KB2; ++q) {
                    float e0[8], e1[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        e0[u] = __builtin_amdgcn_exp2f(x[q][u]);
                        e1[u] = __builtin_amdgcn_exp2f(x[q][8 + u]);
                    }
                    col[q] = __builtin_amdgcn_mfma_f32_16x16x32_f16(y0, __builtin_bit_cast(f16x8_t, pack_e(e0)), col[q], 0, 0, 0);
                    col[q] = __builtin_amdgcn_mfma_f32_16x16x32_f16(y1, __builtin_bit_cast(f16x8_t, pack_e(e1)), col[q], 0, 0, 0);
                }
            }
#pragma unroll
            for (int q = 0; q < KB2; ++q) {
                const int j = j0 + 32 * q + n + 16 * (lane >> 5);
                if (j < r) {
                    if (((lane >> 4) & 1) == 0) {
                        const float c1 = (col[q].x + col[q].y) * as, c2 = (col[q].z + col[q].w) * bs;
                        st<T>::store(GP + b * ldgp + 2 * r + j, ev[q] * c1 - c2);
                    } else {
                        st<T>::store(GP + b * ldgp + j, beta * eg[q] + (col[q].x + col[q].y) * cs);
                    }
                }
            }
        }
    };
    // Slow path (arguments by FMA): 16-key tiles, lane (g, n) holds e of key n for
    // rows 4 g .. +3 and 16 + 4 g .. +3 of each 32-row block.
    auto keys_fma = [&]() {
        for (int j0 = 16 * KT * w; j0 < rpad; j0 += 16 * KT * W) {
            // keys j0 + 16 q + n of this lane (q < KT; past rpad the last key stands in and
            // nothing is stored); their epilogue operands, loaded now
            float kv[KT], ev[KT], eg[KT];
#pragma unroll
            for (int q = 0; q < KT; ++q) {
                const int j = j0 + 16 * q + n, jp = j < rpad ? j : rpad - 1, jc = j < r ? j : r - 1;
                kv[q] = sk[jp];
                ev[q] = pv[jc];
                eg[q] = gh[jc];
            }
            f32x4_t col[KT];
#pragma unroll
            for (int q = 0; q < KT; ++q) col[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            for (int i0 = 0; i0 < rpad; i0 += 32) {
                const f16x8_t ay = xfrag_perm(sy, ldy, n, 6, i0, g);
                u32x4_t e[KT];
                {
                    // rows i0 + 4 g + t and i0 + 16 + 4 g + t (t < 4) of this lane's keys
                    float2 cm[8];
                    *(f32x4_t*)&cm[0] = *(const f32x4_t*)(scm + i0 + 4 * g);
                    *(f32x4_t*)&cm[2] = *(const f32x4_t*)(scm + i0 + 4 * g + 2);
                    *(f32x4_t*)&cm[4] = *(const f32x4_t*)(scm + i0 + 16 + 4 * g);
                    *(f32x4_t*)&cm[6] = *(const f32x4_t*)(scm + i0 + 16 + 4 * g + 2);
#pragma unroll
                    for (int q = 0; q < KT; ++q) {
                        float ex[8];
#pragma unroll
                        for (int t = 0; t < 8; ++t) ex[t] = __builtin_amdgcn_exp2f(fmaf(cm[t].x, kv[q], cm[t].y));
                        e[q] = pack_e(ex);
                    }
                }
#pragma unroll
                for (int q = 0; q < KT; ++q)
                    col[q] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ay, __builtin_bit_cast(f16x8_t, e[q]), col[q], 0, 0, 0);
            }
            // lanes 0..15: (a hi, a lo, a o hi, a o lo) of key n (+16 q); lanes 16..31: (go/Z hi, lo)
            if (lane < 32) {
#pragma unroll
                for (int q = 0; q < KT; ++q) {
                    const int j = j0 + 16 * q + n;
                    if (j < r) {
                        if (lane < 16) {
                            const float c1 = (col[q].x + col[q].y) * as, c2 = (col[q].z + col[q].w) * bs;
                            st<T>::store(GP + b * ldgp + 2 * r + j, ev[q] * c1 - c2);
                        } else {
                            st<T>::store(GP + b * ldgp + j, beta * eg[q] + (col[q].x + col[q].y) * cs);
                        }
                    }
                }
            }
        }
    };
    if (fast) keys32();
    else keys_fma();
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
                           void* H2, bool h2_f16, int64_t ldh, float* stats, int* err, bool bf16, hipStream_t s) {
    if (B == 0) return hipSuccess;
    if (bf16) {
        if (r > 4 * 16 * ATT_NT || !stats) return hipErrorInvalidValue;
        const int rpad = (r + 31) / 32 * 32;
        const int W = attn_waves(rpad);
        const int NT = attn_tiles(rpad, W);
        const int64_t blocks = (B * W + 3) / 4;
        const size_t lds = sizeof(float) * (size_t)attn_fwd_block_floats(rpad, W);
#define RDCN_AFWD(WV, NTV, KBV)                                                                                     \
    hipLaunchKernelGGL((k_attn_fwd_mfma<bf16_t, WV, NTV, KBV>), dim3((unsigned)blocks), dim3(256), lds, s, B, r, rpad, \
                       alpha, beta, 1.0f / tau, (const float*)P, ldp, (bf16_t*)H, H2, ldh, h2_f16, stats, err)
        if (W == 1) {
            if (NT == 2) RDCN_AFWD(1, 2, 1);
            else if (NT == 4) RDCN_AFWD(1, 4, 1);
            else if (NT == 8) RDCN_AFWD(1, 8, 1);
            else RDCN_AFWD(1, 16, 1);
        } else if (W == 2) {
            RDCN_AFWD(2, 16, 4);
        } else {
            RDCN_AFWD(4, 16, 4);
        }
#undef RDCN_AFWD
        return hipGetLastError();
    }
    if (h2_f16) return hipErrorInvalidValue;  // float models have no f16 activations
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
        const int64_t blocks = (B * W + 3) / 4;
        const size_t lds = sizeof(float) * (size_t)attn_bwd_block_floats(rpad, W);
#define RDCN_ABWD(WV, KBV)                                                                                          \
    hipLaunchKernelGGL((k_attn_bwd_mfma<bf16_t, WV, KBV>), dim3((unsigned)blocks), dim3(256), lds, s, B, r, rpad,     \
                       alpha, beta, 1.0f / tau, (const float*)P, ldp, stats, GH, ldg, (bf16_t*)GP, ldgp)
        if (W == 1) RDCN_ABWD(1, 1);
        else if (W == 2) RDCN_ABWD(2, 4);
        else RDCN_ABWD(4, 4);
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
