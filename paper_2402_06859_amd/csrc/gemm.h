// GEMM launcher interface (see gemm.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rdcn {

enum GemmEpi {
    EPI_STORE = 0,      // c[m, n] (storage type, or f16 with c_f16) = scale * acc; c2 as c2_kind says
    EPI_STORE_F32 = 1,  // c[m, n] (float) = scale * acc
    EPI_PARTIAL = 2,    // c[z, m, n] (float) = scale * acc   (split-K partials, z = split)
    EPI_CROSS = 3,      // t = scale*acc + bias[n]; c = x0 * t + xl; t_out = t   (storage type;
                        // xl2: lo plane of a hi + lo bf16 x_l; xl_f16: x_l held as f16;
                        // c_f16: c written as f16; c2 as c2_kind says)
    EPI_RESID = 4,      // c (float) = gin + scale * acc
    EPI_RESID_X0 = 5,   // c (float) += gin + scale * acc
    // MLP layers (bf16 storage, A K-contiguous):
    EPI_MLP_FWD = 6,    // c = ReLU(scale*acc + bias[n]) * (rowv ? sigmoid(rowv[m]) : 1);
                        // with c2: an f16 copy of c (c2_kind C2_F16, err needed)
    EPI_MLP_BWD = 7     // v = scale*acc + (colv ? rowv[m] * colv[n] : 0);
                        // act == NULL: c = v;
                        // else c = v * [act[m, n] > 0] * (rowg ? sigmoid(rowg[m]) : 1), and with
                        // rowpart: rowpart[(n0 / BN) * M + m] = sum over the tile's columns of v * act
};

// What an optional second output plane c2 receives (same row stride as c).
enum GemmC2 {
    C2_LO = 0,    // c is bf16 hi = bf16(v), c2 the lo part bf16(v - hi): the pair carries ~16 bits
    C2_BF16 = 1,  // a bf16 copy of v (c holds v as f16)
    C2_F16 = 2    // an f16 copy of v (c holds v in the storage type)
};

// Bit of the device error word set when a value written as f16 is beyond its range.
constexpr int ERR_BIT_F16_RANGE = 2;

struct GemmArgs {
    int64_t M, N, K;
    const void* a;      // A(m, k) = a[m*lda + k], or a[k*lda + m] when a_kstrided
    const void* a2;     // optional second A plane: C = (A + A2) B^T as two passes over K (no split-K)
    int64_t lda;
    const void* b;      // B(n, k) = b[n*ldb + k], or b[k*ldb + n] when b_kstrided
    int64_t ldb;
    bool a_kstrided, b_kstrided;
    bool ops_f16;       // A and B hold f16 values (f16 MFMAs; both K-contiguous, not EPI_MLP_BWD)
    int epi;
    float scale;
    void* c;            // output (see GemmEpi)
    void* c2;           // optional second output plane (see GemmC2)
    int c2_kind;
    bool c_f16;         // EPI_STORE / EPI_CROSS: c is written as f16
    int* err;           // device error word (needed with c_f16 or c2_kind == C2_F16)
    int64_t ldc;
    // cross / residual epilogue operands, row stride ldx
    const void* bias;
    const void* x0;
    const void* xl;
    const void* xl2;    // optional lo plane of x_l
    bool xl_f16;        // x_l is f16
    void* t_out;
    const void* gin;
    bool gin_f32;
    int64_t ldx;
    // MLP epilogue operands (act has row stride ldx)
    const float* rowv;
    const void* colv;
    const float* rowg;
    const void* act;
    float* rowpart;
    int group_m;        // set from GemmPlan::group_m by launch_gemm
};

struct GemmPlan {
    int bm = 128, bn = 128;
    int splits = 1;
    int stages = 3;  // LDS ring depth (2 lets two workgroups share a CU)
    int group_m = 0; // > 1: tiles walked in groups of group_m tile rows, column by column
};

// split_blocks: with split-K allowed, the workgroup count the K split aims for when
// the output tiles alone are fewer than 256 (a product that runs beside other
// kernels does better with fewer, longer splits).
GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, bool bf16, bool allow_split, int split_blocks = 384);
hipError_t launch_gemm(const GemmArgs& g, const GemmPlan& p, bool bf16, hipStream_t s);
// Column tiles of an MLP GEMM under plan p (the rowpart partials per row).
inline int64_t gemm_tiles_n(int64_t N, const GemmPlan& p) { return (N + p.bn - 1) / p.bn; }
hipError_t launch_splitk_reduce(const float* part, int splits, int64_t MN, float* out, hipStream_t s);
// dst = f16(src) for n bf16 values (n % 8 == 0, 16-byte aligned); sets ERR_BIT_F16_RANGE
// in err when a value is beyond the f16 range.
hipError_t launch_bf16_to_f16(const void* src, void* dst, int64_t n, int* err, hipStream_t s);

}  // namespace rdcn
