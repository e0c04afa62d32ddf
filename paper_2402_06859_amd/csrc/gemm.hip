// bf16 MFMA GEMMs with fused epilogues for gfx950, plus a float VALU GEMM for
// float-storage models.
//
// C[m, n] = scale * sum_k A(m, k) B(n, k), float accumulate. Each operand is
// either K-contiguous (row-major [rows, K]) or K-strided ([K, rows], rows
// contiguous). All six products of the low-rank cross layer map onto this:
//   forward  down  P = x_l W^T      both K-contiguous
//            up    t = h U^T        both K-contiguous (+ cross epilogue)
//   backward gh    = gt U           B K-strided
//            g    += gP W           B K-strided (+ residual epilogue)
//            gU    = gt^T h         both K-strided (split-K over the batch)
//            gW    = gP^T x_l       both K-strided (split-K over the batch)
//
// Tiling: 256 threads = 4 waves in a 2 x 2 grid; a wave owns a (BM/2) x (BN/2)
// block of 16 x 16 MFMA tiles (v_mfma_f32_16x16x32_bf16). Tiles of A and B are
// staged in LDS as [row][k] with a 16-byte row pad, double-buffered, with one
// barrier per K step of 64; the next K step's global loads are in flight
// while the current one is multiplied. A K-strided operand is read as 8 x 8
// blocks (8 k-rows of 16 bytes), transposed in registers and written to LDS
// in the same [row][k] layout, so the MFMA feed is identical for every case.
// The MFMA is issued with B as its first operand, so each lane ends up with
// four consecutive output columns of one row: epilogue loads and stores are
// 8- or 16-byte vectors along the rows of x0, x_l, t and g.
#include "device_common.h"
#include "gemm.h"

namespace rdcn {

namespace {

constexpr int BK = 64;
constexpr int LDS_LD = BK + 8;  // bf16 elements per LDS row (16-byte pad)

template <typename T>
__device__ __forceinline__ void load4(const T* p, float* v);
template <>
__device__ __forceinline__ void load4<float>(const float* p, float* v) {
    const f32x4_t x = *(const f32x4_t*)p;
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}
template <>
__device__ __forceinline__ void load4<bf16_t>(const bf16_t* p, float* v) {
    const uint2 w = *(const uint2*)p;
    v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xffff0000u);
    v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xffff0000u);
}
template <typename T>
__device__ __forceinline__ void store4(T* p, const float* v);
template <>
__device__ __forceinline__ void store4<float>(float* p, const float* v) {
    *(f32x4_t*)p = f32x4_t{v[0], v[1], v[2], v[3]};
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, const float* v) {
    *(uint2*)p = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}

// Epilogue on four consecutive columns n .. n+3 of row m (n + 3 < N guaranteed).
template <typename T>
__device__ __forceinline__ void epilogue4(const GemmArgs& g, int64_t m, int64_t n, int z, float* v) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] *= g.scale;
    switch (g.epi) {
        case EPI_STORE:
            store4<T>((T*)g.c + m * g.ldc + n, v);
            break;
        case EPI_STORE_F32:
            store4<float>((float*)g.c + m * g.ldc + n, v);
            break;
        case EPI_PARTIAL:
            store4<float>((float*)g.c + ((int64_t)z * g.M + m) * g.ldc + n, v);
            break;
        case EPI_CROSS: {  // t = acc + b;  x_next = x0 * t + x_l
            float b[4], x0[4], xl[4], xn[4];
            load4<T>((const T*)g.bias + n, b);
            load4<T>((const T*)g.x0 + m * g.ldx + n, x0);
            load4<T>((const T*)g.xl + m * g.ldx + n, xl);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[e] += b[e];
                xn[e] = x0[e] * v[e] + xl[e];
            }
            store4<T>((T*)g.t_out + m * g.ldx + n, v);
            store4<T>((T*)g.c + m * g.ldc + n, xn);
            break;
        }
        case EPI_RESID:      // g_out = g_in + acc
        case EPI_RESID_X0: { // gx0 += g_in + acc
            float gi[4];
            if (g.gin_f32) load4<float>((const float*)g.gin + m * g.ldx + n, gi);
            else load4<T>((const T*)g.gin + m * g.ldx + n, gi);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] += gi[e];
            float* out = (float*)g.c + m * g.ldc + n;
            if (g.epi == EPI_RESID_X0) {
                float o[4];
                load4<float>(out, o);
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] += o[e];
            }
            store4<float>(out, v);
            break;
        }
    }
}

// 8 x 8 bf16 block transpose in registers: in[r] holds row r (8 values along the
// contiguous dimension), out[c] receives column c (8 values along k).
__device__ __forceinline__ void transpose8x8(const u32x4_t* in, u32x4_t* out) {
#pragma unroll
    for (int c2 = 0; c2 < 4; ++c2) {
        uint32_t lo[4], hi[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t a = in[2 * j][c2], b = in[2 * j + 1][c2];
            lo[j] = (a & 0xffffu) | (b << 16);
            hi[j] = (a >> 16) | (b & 0xffff0000u);
        }
        out[2 * c2] = u32x4_t{lo[0], lo[1], lo[2], lo[3]};
        out[2 * c2 + 1] = u32x4_t{hi[0], hi[1], hi[2], hi[3]};
    }
}

// Operand tile loader: ROWS x BK bf16 tile starting at (row0, k0).
template <int ROWS, bool KSTRIDED>
struct TileLoader {
    // K-contiguous: ROWS*BK/8 vectors of 16 bytes, spread over 256 threads.
    // K-strided:    (ROWS/8)*(BK/8) 8x8 blocks; one block per thread.
    static constexpr int NVEC = KSTRIDED ? 8 : (ROWS * BK / 8) / 256;
    u32x4_t r[NVEC > 0 ? NVEC : 1];
    bool active;

    __device__ __forceinline__ void load(const bf16_t* base, int64_t ld, int64_t rows, int64_t K, int64_t row0,
                                         int64_t k0, int tid) {
        if (!KSTRIDED) {
#pragma unroll
            for (int i = 0; i < NVEC; ++i) {
                const int v = tid + 256 * i;
                const int row = v / (BK / 8), kv = v % (BK / 8);
                const int64_t gr = row0 + row, gk = k0 + kv * 8;
                if (gr < rows && gk < K) r[i] = *(const u32x4_t*)(base + gr * ld + gk);
                else r[i] = u32x4_t{0, 0, 0, 0};
            }
        } else {
            constexpr int NB = (ROWS / 8) * (BK / 8);
            active = tid < NB;
            const int kb = tid % (BK / 8), rb = tid / (BK / 8);
            const int64_t gr = row0 + rb * 8;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int64_t gk = k0 + kb * 8 + i;
                if (active && gr < rows && gk < K) r[i] = *(const u32x4_t*)(base + gk * ld + gr);
                else r[i] = u32x4_t{0, 0, 0, 0};
            }
        }
    }

    __device__ __forceinline__ void store(bf16_t* lds, int tid) {
        if (!KSTRIDED) {
#pragma unroll
            for (int i = 0; i < NVEC; ++i) {
                const int v = tid + 256 * i;
                const int row = v / (BK / 8), kv = v % (BK / 8);
                *(u32x4_t*)(lds + row * LDS_LD + kv * 8) = r[i];
            }
        } else if (active) {
            const int kb = tid % (BK / 8), rb = tid / (BK / 8);
            u32x4_t t[8];
            transpose8x8(r, t);
#pragma unroll
            for (int c = 0; c < 8; ++c) *(u32x4_t*)(lds + (rb * 8 + c) * LDS_LD + kb * 8) = t[c];
        }
    }
};

__device__ __forceinline__ int xcd_remap(int id, int n) {
    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of tiles so neighbouring tiles share its L2.
    if (n % 8 != 0) return id;
    return (id % 8) * (n / 8) + id / 8;
}

template <int BM, int BN, bool AKS, bool BKS, typename T>
__global__ __launch_bounds__(256, 2) void k_gemm_mfma(GemmArgs g) {
    constexpr int TM = BM / 32, TN = BN / 32;  // 16x16 tiles per wave
    __shared__ __attribute__((aligned(16))) bf16_t sA[2][BM * LDS_LD];
    __shared__ __attribute__((aligned(16))) bf16_t sB[2][BN * LDS_LD];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int tiles_n = (int)((g.N + BN - 1) / BN);
    const int ntiles = (int)(((g.M + BM - 1) / BM) * tiles_n);
    const int t = xcd_remap(blockIdx.x, ntiles);
    const int64_t m0 = (int64_t)(t / tiles_n) * BM, n0 = (int64_t)(t % tiles_n) * BN;

    // split-K range
    const int z = blockIdx.z;
    const int64_t kchunk = ((g.K + (int64_t)gridDim.z * BK - 1) / ((int64_t)gridDim.z * BK)) * BK;
    const int64_t kbeg = z * kchunk;
    const int64_t kend = kbeg + kchunk < g.K ? kbeg + kchunk : g.K;

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const bf16_t* A = (const bf16_t*)g.a;
    const bf16_t* B = (const bf16_t*)g.b;
    TileLoader<BM, AKS> la;
    TileLoader<BN, BKS> lb;

    if (kbeg < kend) {
        la.load(A, g.lda, g.M, kend, m0, kbeg, tid);
        lb.load(B, g.ldb, g.N, kend, n0, kbeg, tid);
        la.store(sA[0], tid);
        lb.store(sB[0], tid);
    }
    __syncthreads();

    int cur = 0;
    for (int64_t k0 = kbeg; k0 < kend; k0 += BK) {
        const bool more = k0 + BK < kend;
        if (more) {
            la.load(A, g.lda, g.M, kend, m0, k0 + BK, tid);
            lb.load(B, g.ldb, g.N, kend, n0, k0 + BK, tid);
        }
        const bf16_t* a_s = sA[cur];
        const bf16_t* b_s = sB[cur];
#pragma unroll
        for (int ks = 0; ks < BK; ks += 32) {
            bf16x8_t af[TM], bfr[TN];
            const int kk = ks + (lane >> 4) * 8;
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = __builtin_bit_cast(bf16x8_t,
                                           *(const u32x4_t*)(a_s + (wm * (BM / 2) + i * 16 + (lane & 15)) * LDS_LD + kk));
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = __builtin_bit_cast(bf16x8_t,
                                            *(const u32x4_t*)(b_s + (wn * (BN / 2) + j * 16 + (lane & 15)) * LDS_LD + kk));
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
        }
        if (more) {
            la.store(sA[cur ^ 1], tid);
            lb.store(sB[cur ^ 1], tid);
        }
        __syncthreads();
        cur ^= 1;
    }

    // lane holds C[m = tile_m + (lane & 15)][n = tile_n + 4 * (lane >> 4) + e]
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int64_t m = m0 + wm * (BM / 2) + i * 16 + (lane & 15);
        if (m >= g.M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int64_t n = n0 + wn * (BN / 2) + j * 16 + 4 * (lane >> 4);
            if (n >= g.N) continue;
            float v[4] = {acc[i][j].x, acc[i][j].y, acc[i][j].z, acc[i][j].w};
            epilogue4<T>(g, m, n, z, v);
        }
    }
}

// Float VALU GEMM (float-storage models): 64 x 64 tile, 4 x 4 outputs per
// thread (4 consecutive columns), operands addressed through (row, k) strides.
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs g) {
    constexpr int T64 = 64, TK = 16;
    __shared__ float sA[TK][T64 + 1];
    __shared__ float sB[TK][T64 + 1];
    const int tid = threadIdx.x;
    const int tiles_n = (int)((g.N + T64 - 1) / T64);
    const int64_t m0 = (int64_t)(blockIdx.x / tiles_n) * T64, n0 = (int64_t)(blockIdx.x % tiles_n) * T64;
    const int z = blockIdx.z;
    const int64_t kchunk = ((g.K + (int64_t)gridDim.z * TK - 1) / ((int64_t)gridDim.z * TK)) * TK;
    const int64_t kbeg = z * kchunk;
    const int64_t kend = kbeg + kchunk < g.K ? kbeg + kchunk : g.K;
    const float* A = (const float*)g.a;
    const float* B = (const float*)g.b;
    const int64_t a_sr = g.a_kstrided ? 1 : g.lda, a_sk = g.a_kstrided ? g.lda : 1;
    const int64_t b_sr = g.b_kstrided ? 1 : g.ldb, b_sk = g.b_kstrided ? g.ldb : 1;
    const int tr = tid / 16, tc = tid % 16;  // rows tr*4.., cols tc*4..
    float acc[4][4] = {};
    for (int64_t k0 = kbeg; k0 < kend; k0 += TK) {
        for (int e = tid; e < TK * T64; e += 256) {
            const int kk = e / T64, rr = e % T64;
            const int64_t gk = k0 + kk;
            sA[kk][rr] = (m0 + rr < g.M && gk < kend) ? A[(m0 + rr) * a_sr + gk * a_sk] : 0.f;
            sB[kk][rr] = (n0 + rr < g.N && gk < kend) ? B[(n0 + rr) * b_sr + gk * b_sk] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = sA[kk][tr * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = sB[kk][tc * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + tr * 4 + i;
        const int64_t n = n0 + tc * 4;
        if (m < g.M && n < g.N) epilogue4<float>(g, m, n, z, acc[i]);
    }
}

// out[m, n] = scale_out * sum_z part[z, m, n], summed in z order.
__global__ __launch_bounds__(256) void k_splitk_reduce(const float* part, int splits, int64_t MN, float* out) {
    for (int64_t i = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * 4; i < MN;
         i += (int64_t)gridDim.x * blockDim.x * 4) {
        f32x4_t s = *(const f32x4_t*)(part + i);
        for (int z = 1; z < splits; ++z) {
            const f32x4_t p = *(const f32x4_t*)(part + (int64_t)z * MN + i);
            s.x += p.x; s.y += p.y; s.z += p.z; s.w += p.w;
        }
        *(f32x4_t*)(out + i) = s;
    }
}

template <int BM, int BN, typename T>
hipError_t launch_tile(const GemmArgs& g, int splits, hipStream_t s) {
    const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    dim3 grid((unsigned)tiles, 1, (unsigned)splits);
#define RDCN_GEMM(AK, BKS) hipLaunchKernelGGL((k_gemm_mfma<BM, BN, AK, BKS, T>), grid, dim3(256), 0, s, g)
    if (g.a_kstrided) {
        if (g.b_kstrided) RDCN_GEMM(true, true); else RDCN_GEMM(true, false);
    } else {
        if (g.b_kstrided) RDCN_GEMM(false, true); else RDCN_GEMM(false, false);
    }
#undef RDCN_GEMM
    return hipGetLastError();
}

}  // namespace

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, bool bf16, bool allow_split) {
    GemmPlan p;
    if (!bf16) {
        p.bm = p.bn = 64;
    } else {
        const int64_t t128 = ((M + 127) / 128) * ((N + 127) / 128);
        if (t128 >= 240) p.bm = p.bn = 128;
        else p.bm = p.bn = 64;
    }
    const int64_t tiles = ((M + p.bm - 1) / p.bm) * ((N + p.bn - 1) / p.bn);
    p.splits = 1;
    if (allow_split && tiles < 256) {
        int64_t s = (512 + tiles - 1) / tiles;
        const int64_t kmax = K / 256;  // keep >= 4 K steps of 64 per split
        if (s > kmax) s = kmax;
        if (s > 32) s = 32;
        if (s < 1) s = 1;
        p.splits = (int)s;
    }
    return p;
}

hipError_t launch_gemm(const GemmArgs& g, const GemmPlan& p, bool bf16, hipStream_t s) {
    if (g.M == 0 || g.N == 0) return hipSuccess;
    if (!bf16) {
        const int64_t tiles = ((g.M + 63) / 64) * ((g.N + 63) / 64);
        hipLaunchKernelGGL(k_gemm_f32, dim3((unsigned)tiles, 1, (unsigned)p.splits), dim3(256), 0, s, g);
        return hipGetLastError();
    }
    if (p.bm == 128) return launch_tile<128, 128, bf16_t>(g, p.splits, s);
    return launch_tile<64, 64, bf16_t>(g, p.splits, s);
}

hipError_t launch_splitk_reduce(const float* part, int splits, int64_t MN, float* out, hipStream_t s) {
    if (MN == 0) return hipSuccess;
    int64_t blocks = (MN / 4 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)blocks), dim3(256), 0, s, part, splits, MN, out);
    return hipGetLastError();
}

}  // namespace rdcn
