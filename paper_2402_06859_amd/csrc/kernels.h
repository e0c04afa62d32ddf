// Host-side launchers of the gfx950 kernels (implemented in the .hip files).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rdcn {

struct GatherArgs {
    int64_t batch;
    int32_t F, D, Nd, rows_q;
    uint32_t m;
    uint64_t vocab;
    uint32_t magic, shift;  // 32-bit division by m (valid when vocab <= 2^32)
    int combine;            // 0 = product, 1 = sum
    int hashed;             // 1: hashed front-end (tables [F, 2, rows, D]; every id valid)
    uint64_t seed;          // hash seed
    const void* ids;        // int32 or int64
    const int64_t* offsets; // NULL = single-hot
    const void* q_tables;   // storage-type tables, or int8 codes for the quantized gather
    const void* r_tables;
    const float* q_params;  // quantized gather: (middle, scale) per table row
    const float* r_params;
    const void* dense;
    void* x0;
    int* err;
};
hipError_t launch_qr_gather(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s);
// Same gather from middle-max 8-bit tables (codes in q_tables / r_tables, row parameters in q_params / r_params).
hipError_t launch_qr_gather_q8(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s);
// Middle-max 8-bit row-wise quantization of `rows` table rows of width D.
hipError_t launch_quantize_rows(int64_t rows, int D, const void* tables, int8_t* codes, float* params, bool bf16,
                                hipStream_t s);

}  // namespace rdcn

namespace rdcn {

// bf16 storage: the forward writes o_i, Z_i and the row sums W1_i = sum_j e_ij v_j k_j,
// W2_i = sum_j e_ij k_j of every row to stats ([o | Z | W1 | W2] per sample, row
// stride 4 r) and the backward reads them back.
// H2: optional second plane of h: its f16 value (h2_f16) or the lo part of a bf16
// hi + lo pair; f16 values beyond range set bit 2 of *err.
hipError_t launch_attn_fwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp, void* H,
                           void* H2, bool h2_f16, int64_t ldh, float* stats, int* err, bool bf16, hipStream_t s);
hipError_t launch_attn_bwd(int64_t B, int r, float alpha, float beta, float tau, const void* P, int64_t ldp,
                           const float* stats, const float* GH, int64_t ldg, void* GP, int64_t ldgp, bool bf16,
                           hipStream_t s);

int pointwise_rows_per_block(int64_t B, int64_t d);
hipError_t launch_bwd_pointwise(int64_t B, int64_t d, const void* gin, bool gin_f32, const void* x0, const void* t,
                                float* gx0, bool first, void* gt, float* part, bool bf16, hipStream_t s);
hipError_t launch_colsum(const float* part, int nrb, int64_t d, float* out, hipStream_t s);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);

}  // namespace rdcn
