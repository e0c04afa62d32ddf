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
// floats). A wave owns 64 consecutive vector columns of x0 and a few rows: lane l
// always produces column c = 64 * blockIdx.x + l, so its feature, the position
// inside the feature's segment (or inside the dense block) and its table offsets
// are fixed, and every store instruction writes one contiguous 1 KiB run of a row.
// The wave first issues the id (or bag-offset) loads of all its rows, then the
// quotient- and remainder-row loads (the tables are small and stay in L2 / MALL),
// and only then combines in float, pools over the bag in bag order, rounds to the
// storage type and stores: the dependent id -> row load chains of its rows are in
// flight together. Vectors of the dense block are copied.
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

constexpr int GATHER_ROWS = 4;  // rows per wave (their loads are issued together)

template <typename T, typename ID, bool BAGS>
__global__ __launch_bounds__(256) void k_qr_gather(GatherArgs a) {
#pragma clang fp contract(off)
    constexpr int V = st<T>::vec;
    const int cpf = a.D / V;                 // vectors per embedding segment
    const int emb_vecs = a.F * cpf;
    const int cpr = emb_vecs + a.Nd / V;     // vectors per x0 row
    const int c = blockIdx.x * 64 + (threadIdx.x & 63);
    if (c >= cpr) return;
    const T* qt = (const T*)a.q_tables;
    const T* rt = (const T*)a.r_tables;
    const ID* ids = (const ID*)a.ids;
    T* x0 = (T*)a.x0;
    const int64_t d = (int64_t)a.F * a.D + a.Nd;
    const bool emb = c < emb_vecs;
    const int f = emb ? c / cpf : 0;
    const int cc = emb ? c - f * cpf : 0;
    const T* qbase = qt + (int64_t)f * a.rows_q * a.D + cc * V;
    const T* rbase = rt + (int64_t)f * a.m * a.D + cc * V;
    const int64_t row_step = (int64_t)gridDim.y * 4 * GATHER_ROWS;
    for (int64_t b0 = ((int64_t)blockIdx.y * 4 + (threadIdx.x >> 6)) * GATHER_ROWS; b0 < a.batch; b0 += row_step) {
        const int nr = a.batch - b0 < GATHER_ROWS ? (int)(a.batch - b0) : GATHER_ROWS;
        u32x4_t out[GATHER_ROWS];
        if (!emb) {
#pragma unroll
            for (int u = 0; u < GATHER_ROWS; ++u)
                if (u < nr) out[u] = *(const u32x4_t*)((const T*)a.dense + (b0 + u) * a.Nd + (c - emb_vecs) * V);
        } else if (!BAGS) {
            ID id[GATHER_ROWS];
#pragma unroll
            for (int u = 0; u < GATHER_ROWS; ++u) id[u] = ids[(b0 + (u < nr ? u : 0)) * a.F + f];
            bool ok[GATHER_ROWS];
            u32x4_t qw[GATHER_ROWS], rw[GATHER_ROWS];
#pragma unroll
            for (int u = 0; u < GATHER_ROWS; ++u) {
                uint32_t qi = 0, ri = 0;
                ok[u] = qr_split<ID>(id[u], a, qi, ri);
                if (!ok[u]) qi = ri = 0;
                qw[u] = *(const u32x4_t*)(qbase + (int64_t)qi * a.D);
                rw[u] = *(const u32x4_t*)(rbase + (int64_t)ri * a.D);
            }
            bool bad = false;
#pragma unroll
            for (int u = 0; u < GATHER_ROWS; ++u) {
                float qv[V], rv[V], acc[V];
                st<T>::unpack(qw[u], qv);
                st<T>::unpack(rw[u], rv);
#pragma unroll
                for (int e = 0; e < V; ++e) acc[e] = ok[u] ? (a.combine == 0 ? qv[e] * rv[e] : qv[e] + rv[e]) : 0.0f;
                out[u] = st<T>::pack(acc);
                bad = bad || (u < nr && !ok[u]);
            }
            if (bad && cc == 0) atomicOr(a.err, 1);
        } else {
            int64_t beg[GATHER_ROWS], end[GATHER_ROWS];
#pragma unroll
            for (int u = 0; u < GATHER_ROWS; ++u) {
                const int64_t bag = (b0 + (u < nr ? u : 0)) * a.F + f;
                beg[u] = a.offsets[bag];
                end[u] = a.offsets[bag + 1];
            }
            bool bad = false;
#pragma unroll
            for (int u = 0; u < GATHER_ROWS; ++u) {
                float acc[V];
                bool started = false;
                for (int64_t p = beg[u]; p < end[u]; ++p) {
                    uint32_t qi, ri;
                    if (!qr_split<ID>(ids[p], a, qi, ri)) {
                        bad = true;
                        continue;
                    }
                    float qv[V], rv[V];
                    st<T>::unpack(*(const u32x4_t*)(qbase + (int64_t)qi * a.D), qv);
                    st<T>::unpack(*(const u32x4_t*)(rbase + (int64_t)ri * a.D), rv);
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
                out[u] = st<T>::pack(acc);
            }
            if (bad && cc == 0) atomicOr(a.err, 1);
        }
#pragma unroll
        for (int u = 0; u < GATHER_ROWS; ++u)
            if (u < nr) *(u32x4_t*)(x0 + (b0 + u) * d + (int64_t)c * V) = out[u];
    }
}

hipError_t launch_qr_gather(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s) {
    const int V = bf16 ? 8 : 4;
    const int64_t cpr = (a.F * (int64_t)a.D + a.Nd) / V;
    if (a.batch == 0 || cpr == 0) return hipSuccess;
    // x: 64-column slices of a row; y: groups of 4 waves x GATHER_ROWS rows (grid-stride beyond)
    int64_t ygroups = (a.batch + 4 * GATHER_ROWS - 1) / (4 * GATHER_ROWS);
    if (ygroups > 65535) ygroups = 65535;
    const dim3 grid((unsigned)((cpr + 63) / 64), (unsigned)ygroups);
    const int threads = 256;
    const bool bags = a.offsets != nullptr;
#define RDCN_GATHER(T, ID, BG) hipLaunchKernelGGL((k_qr_gather<T, ID, BG>), grid, dim3(threads), 0, s, a)
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
