// QR-hashed embedding gather for gfx950 (forward).
//
// Section "Model Dictionary Compression": an id is split by the remainder-table
// size m into a quotient and a remainder, each indexing a small per-feature
// table, and the two rows are aggregated (sum or elementwise product). Section
// "Residual DCN" / appendix "Feed Ranking Sparse ID features": the looked-up
// embeddings replace one-hot inputs and are concatenated with the dense
// features into x0.
//
// Work split: the output x0 [B, d] is cut into 16-byte vectors (8 bf16 or 4
// floats); one thread produces one vector, and consecutive threads produce
// consecutive vectors of a row, so every store instruction of a wave writes
// one contiguous 1 KiB run of x0. A vector inside an embedding segment loads
// the matching 16 bytes of the quotient row and of the remainder row (the
// tables are small and stay in L2 / MALL), combines in float, pools over the
// bag in bag order, rounds to the storage type and stores. Vectors of the
// dense block are copied.
#include "device_common.h"
#include "kernels.h"

namespace rdcn {

template <typename ID>
__device__ __forceinline__ bool qr_split(ID id_raw, const GatherArgs& a, uint32_t& qi, uint32_t& ri) {
    int64_t id = (int64_t)id_raw;
    if (id < 0 || (uint64_t)id >= a.vocab) return false;
    if (a.vocab <= 0x100000000ull) {
        uint32_t n = (uint32_t)id;
        DivMagic dm{a.magic, a.shift, a.m};
        qi = div_magic(n, dm);
        ri = n - qi * a.m;
    } else {
        uint64_t q = (uint64_t)id / a.m;
        qi = (uint32_t)q;
        ri = (uint32_t)((uint64_t)id - q * a.m);
    }
    return qi < (uint32_t)a.rows_q && ri < a.m;
}

template <typename T, typename ID, bool BAGS>
__global__ __launch_bounds__(256) void k_qr_gather(GatherArgs a) {
#pragma clang fp contract(off)
    constexpr int V = st<T>::vec;
    const int cpf = a.D / V;                        // vectors per embedding segment
    const int cpr = (a.F * a.D + a.Nd) / V;         // vectors per x0 row
    const int emb_vecs = a.F * cpf;
    const int64_t total = a.batch * (int64_t)cpr;
    const T* qt = (const T*)a.q_tables;
    const T* rt = (const T*)a.r_tables;
    const ID* ids = (const ID*)a.ids;
    T* x0 = (T*)a.x0;
    const int64_t d = (int64_t)a.F * a.D + a.Nd;

    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = i / cpr;
        const int c = (int)(i - b * cpr);
        u32x4_t out;
        if (c < emb_vecs) {
            const int f = c / cpf;
            const int cc = c - f * cpf;
            int64_t begin, end;
            if (BAGS) {
                begin = a.offsets[b * a.F + f];
                end = a.offsets[b * a.F + f + 1];
            } else {
                begin = b * a.F + f;
                end = begin + 1;
            }
            float acc[V];
            bool started = false;
            bool bad = false;
            for (int64_t p = begin; p < end; ++p) {
                uint32_t qi, ri;
                if (!qr_split<ID>(ids[p], a, qi, ri)) {
                    bad = true;
                    continue;
                }
                const u32x4_t qw = *(const u32x4_t*)(qt + ((int64_t)f * a.rows_q + qi) * a.D + cc * V);
                const u32x4_t rw = *(const u32x4_t*)(rt + ((int64_t)f * a.m + ri) * a.D + cc * V);
                float qv[V], rv[V];
                st<T>::unpack(qw, qv);
                st<T>::unpack(rw, rv);
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    const float x = a.combine == 0 ? qv[e] * rv[e] : qv[e] + rv[e];
                    acc[e] = started ? acc[e] + x : x;
                }
                started = true;
            }
            if (!started) {
#pragma unroll
                for (int e = 0; e < V; ++e) acc[e] = 0.0f;
            }
            if (bad && cc == 0) atomicOr(a.err, 1);
            out = st<T>::pack(acc);
        } else {
            out = *(const u32x4_t*)((const T*)a.dense + b * a.Nd + (c - emb_vecs) * V);
        }
        *(u32x4_t*)(x0 + b * d + (int64_t)c * V) = out;
    }
}

hipError_t launch_qr_gather(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s) {
    const int V = bf16 ? 8 : 4;
    const int64_t total = a.batch * ((a.F * (int64_t)a.D + a.Nd) / V);
    if (total == 0) return hipSuccess;
    const int threads = 256;
    int64_t blocks = (total + threads - 1) / threads;
    if (blocks > 65536) blocks = 65536;
    const bool bags = a.offsets != nullptr;
#define RDCN_GATHER(T, ID, BG) hipLaunchKernelGGL((k_qr_gather<T, ID, BG>), dim3((unsigned)blocks), dim3(threads), 0, s, a)
    if (bf16) {
        if (ids64) { if (bags) RDCN_GATHER(bf16_t, int64_t, true); else RDCN_GATHER(bf16_t, int64_t, false); }
        else       { if (bags) RDCN_GATHER(bf16_t, int32_t, true); else RDCN_GATHER(bf16_t, int32_t, false); }
    } else {
        if (ids64) { if (bags) RDCN_GATHER(float, int64_t, true); else RDCN_GATHER(float, int64_t, false); }
        else       { if (bags) RDCN_GATHER(float, int32_t, true); else RDCN_GATHER(float, int32_t, false); }
    }
#undef RDCN_GATHER
    return hipGetLastError();
}

}  // namespace rdcn
