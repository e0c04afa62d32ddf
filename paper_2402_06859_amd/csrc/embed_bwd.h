// Embedding-backward launcher interface (see embed_bwd.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rdcn {

struct EmbedBwdArgs {
    int64_t batch, nnz, d;
    int32_t F, D, rows_q;
    uint32_t m;
    uint64_t vocab;
    int combine;             // 0 = product, 1 = sum
    int hashed;              // 1: hashed front-end, two (Q, R) pairs per feature and four keys per id
    uint64_t seed;           // hash seed
    const void* ids;
    const int64_t* offsets;  // NULL = single-hot
    const void* q_tables;
    const void* r_tables;
    const float* grad_x0;
    float* grad_q;
    float* grad_r;
    // invariant-divisor multipliers (device_common.h DivMagic) for F, rows_q and m
    uint32_t magic_f, shift_f, magic_q, shift_q, magic_m, shift_m;
};

struct EmbedBwdLayout {
    uint64_t keys0, vals0, keys1, vals1, bag_of, qrow, rrow, hist, sums, carry_head, carry_tail, total;
    int bits, passes, dbits;
};

// (key, occurrence) pairs the embedding backward sorts: two per id, four when hashed
inline int64_t emb_pairs(int64_t nnz, bool hashed) { return (hashed ? 4 : 2) * nnz; }
EmbedBwdLayout embed_bwd_layout(int64_t nnz, int F, int rows_q, int m, int D, bool bags, bool mul, bool hashed);
hipError_t launch_emb_keys(const EmbedBwdArgs& a, bool ids64, void* scratch, hipStream_t s);
hipError_t launch_emb_sort(const EmbedBwdArgs& a, void* scratch, hipStream_t s);
// grad_x0, grad_q and grad_r must be 16-byte aligned (checked by the caller).
hipError_t launch_emb_reduce(const EmbedBwdArgs& a, bool bf16, void* scratch, hipStream_t s);
// One-kernel embedding backward without scratch, for unhashed ids and tables of at most
// 16384 rows (emb_fused_ok); the same sums in the same per-row order of occurrences.
bool emb_fused_ok(int rows_q, int m, int D, bool hashed);
hipError_t launch_emb_fused(const EmbedBwdArgs& a, bool bf16, bool ids64, hipStream_t s);

// Size of the library-owned workspace of qr_embed_backward_static (per device).
constexpr uint64_t EMB_STATIC_SCRATCH_BYTES = 64ull << 20;
// Device address of that workspace on the current device (looked up once per device).
hipError_t emb_static_scratch(void** out);

}  // namespace rdcn
