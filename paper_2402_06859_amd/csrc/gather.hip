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
// floats). A wave owns one block of 64 consecutive vector columns of x0 and a few
// rows: lane l always produces column c = 64 * bx + l of its block bx, so its
// feature, the position inside the feature's segment (or inside the dense block) and
// its table offsets are fixed, and every store instruction writes one contiguous
// 1 KiB run of a row. Blocks go to the XCDs in contiguous ranges of column blocks
// (gather_block), so each XCD reads the tables of a few features and keeps them in
// its L2.
// The wave first issues the id (or bag-offset) loads of all its rows, then the
// quotient- and remainder-row loads (the tables are small and stay in L2 / MALL),
// and only then combines in float, pools over the bag in bag order, rounds to the
// storage type and stores: the dependent id -> row load chains of its rows are in
// flight together. A bag (multi-hot feature) is read in chunks of K ids
// (GATHER_BAG_CHUNK), and the next chunk's id loads are issued before this chunk's
// row loads, so a bag of n ids costs about n/K + 1 dependent load latencies rather
// than 2n. With bags a wave sums one bag at a time: K = 1 and one row per wave keep
// the kernel small enough for 8 waves per SIMD, which hides more latency than
// wider chunks at fewer waves. Vectors of the dense block are copied.
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

constexpr int GATHER_ROWS = 2;  // rows per wave (their loads are issued together)
// rows per wave when the features are bags: a wave sums its bags one after another,
// so one bag per wave puts twice as many bags in flight across the chip
constexpr int GATHER_BAG_ROWS = 1;
constexpr int GATHER_BAG_CHUNK = 1;  // ids of a bag whose row loads are issued together

// Table rows in the storage type: a lane's V values are one 16-byte vector.
template <typename T>
struct StorageRows {
    static constexpr int V = st<T>::vec;
    struct Raw {
        u32x4_t w;
    };
    const T* q;  // the lane's columns in row 0 of feature f's quotient table
    const T* r;
    int64_t D;
    __device__ __forceinline__ StorageRows(const GatherArgs& a, int f, int cc)
        : q((const T*)a.q_tables + (int64_t)f * a.rows_q * a.D + cc * V),
          r((const T*)a.r_tables + (int64_t)f * a.m * a.D + cc * V), D(a.D) {}
    __device__ __forceinline__ Raw load_q(uint32_t i) const { return Raw{*(const u32x4_t*)(q + (int64_t)i * D)}; }
    __device__ __forceinline__ Raw load_r(uint32_t i) const { return Raw{*(const u32x4_t*)(r + (int64_t)i * D)}; }
    __device__ __forceinline__ static void values(const Raw& x, float* v) { st<T>::unpack(x.w, v); }
};

// Middle-max 8-bit rows (section "Embedding Table Quantization"): a lane's V codes
// and the row's (middle, scale); value = middle + code * scale with one rounding.
template <typename T>
struct Q8Rows {
    static constexpr int V = st<T>::vec;  // output values per lane (8 for bf16 x0, 4 for float)
    struct Raw {
        uint32_t c[V / 4];
        float2 p;
    };
    const int8_t* q;
    const int8_t* r;
    const float2* qp;
    const float2* rp;
    int64_t D;
    __device__ __forceinline__ Q8Rows(const GatherArgs& a, int f, int cc)
        : q((const int8_t*)a.q_tables + (int64_t)f * a.rows_q * a.D + cc * V),
          r((const int8_t*)a.r_tables + (int64_t)f * a.m * a.D + cc * V),
          qp((const float2*)a.q_params + (int64_t)f * a.rows_q), rp((const float2*)a.r_params + (int64_t)f * a.m),
          D(a.D) {}
    __device__ __forceinline__ static Raw load(const int8_t* codes, const float2* params, uint32_t i, int64_t D) {
        Raw x;
        if (V == 8) {
            const uint2 w = *(const uint2*)(codes + (int64_t)i * D);
            x.c[0] = w.x;
            x.c[V / 4 - 1] = w.y;
        } else {
            x.c[0] = *(const uint32_t*)(codes + (int64_t)i * D);
        }
        x.p = params[i];
        return x;
    }
    __device__ __forceinline__ Raw load_q(uint32_t i) const { return load(q, qp, i, D); }
    __device__ __forceinline__ Raw load_r(uint32_t i) const { return load(r, rp, i, D); }
    __device__ __forceinline__ static void values(const Raw& x, float* v) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int code = (int)(int8_t)((x.c[e / 4] >> (8 * (e % 4))) & 0xffu);
            v[e] = __builtin_fmaf((float)code, x.p.y, x.p.x);
        }
    }
};

// Hashed front-end: the two 32-bit halves of an id's 64-bit hash, each QR-split by m.
__device__ __forceinline__ void hash_split(int64_t id, const GatherArgs& a, uint32_t (&qi)[2], uint32_t (&ri)[2]) {
    const uint64_t h = murmur64a_8((uint64_t)id, a.seed);
    const DivMagic dm{a.magic, a.shift, a.m};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const uint32_t x = (uint32_t)(s ? h >> 32 : h);
        qi[s] = div_magic(x, dm);
        ri[s] = x - qi[s] * a.m;
    }
}

// Workgroup L of the one-dimensional grid of nx column blocks times ny row groups ->
// (column block bx, row group by). Workgroups go round-robin to the 8 XCDs (L % 8).
// Items are listed column block outermost, so a contiguous range of items touches the
// tables of a few features only; each XCD takes an eighth of the ne * ny items of the
// column blocks holding embedding columns as one contiguous range (those tables then
// stay in its L2), followed by an eighth of the items of the dense-only blocks (plain
// copies, far cheaper), so every XCD gets the same share of both kinds. Items left
// over by the two divisions by 8 go to the last workgroups.
__device__ __forceinline__ void gather_block(int L, int ne, int nx, int ny, int& bx, int& by) {
    const int E = ne * ny, Q = (nx - ne) * ny;
    const int eb = E / 8, qb = Q / 8;
    int item;
    if (L < 8 * (eb + qb)) {
        const int k = L % 8, j = L / 8;
        item = j < eb ? k * eb + j : E + k * qb + (j - eb);
    } else {
        const int i = L - 8 * (eb + qb), er = E - 8 * eb;
        item = i < er ? 8 * eb + i : E + 8 * qb + (i - er);
    }
    bx = item / ny;
    by = item - bx * ny;
}

template <typename T, typename ID, bool BAGS, class Rows, bool HASHED>
__global__ __launch_bounds__(256) void k_qr_gather(GatherArgs a, int ny) {
#pragma clang fp contract(off)
    constexpr int RW = BAGS ? GATHER_BAG_ROWS : GATHER_ROWS;
    constexpr int V = st<T>::vec;
    const int cpf = a.D / V;                 // vectors per embedding segment
    const int emb_vecs = a.F * cpf;
    const int cpr = emb_vecs + a.Nd / V;     // vectors per x0 row
    int bx, by;
    gather_block(blockIdx.x, (emb_vecs + 63) / 64, gridDim.x / ny, ny, bx, by);
    const int c = bx * 64 + (threadIdx.x & 63);
    if (c >= cpr) return;
    const ID* ids = (const ID*)a.ids;
    T* x0 = (T*)a.x0;
    const int64_t d = (int64_t)a.F * a.D + a.Nd;
    const bool emb = c < emb_vecs;
    const int f = emb ? c / cpf : 0;
    const int cc = emb ? c - f * cpf : 0;
    // table pair(s) of feature f: pair f, or pairs 2f (low hash half) and 2f + 1 (high)
    const Rows rows(a, HASHED ? 2 * f : f, cc);
    const Rows rows1(a, HASHED ? 2 * f + 1 : f, cc);
    const int64_t row_step = (int64_t)ny * 4 * RW;
    for (int64_t b0 = ((int64_t)by * 4 + (threadIdx.x >> 6)) * RW; b0 < a.batch; b0 += row_step) {
        const int nr = a.batch - b0 < RW ? (int)(a.batch - b0) : RW;
        u32x4_t out[RW];
        if (!emb) {
#pragma unroll
            for (int u = 0; u < RW; ++u)
                if (u < nr) out[u] = *(const u32x4_t*)((const T*)a.dense + (b0 + u) * a.Nd + (c - emb_vecs) * V);
        } else if (!BAGS && HASHED) {
            ID id[RW];
#pragma unroll
            for (int u = 0; u < RW; ++u) id[u] = ids[(b0 + (u < nr ? u : 0)) * a.F + f];
            typename Rows::Raw q0[RW], r0[RW], q1[RW], r1[RW];
#pragma unroll
            for (int u = 0; u < RW; ++u) {
                uint32_t qi[2], ri[2];
                hash_split((int64_t)id[u], a, qi, ri);
                q0[u] = rows.load_q(qi[0]);
                r0[u] = rows.load_r(ri[0]);
                q1[u] = rows1.load_q(qi[1]);
                r1[u] = rows1.load_r(ri[1]);
            }
#pragma unroll
            for (int u = 0; u < RW; ++u) {
                float qa[V], ra[V], qb[V], rb[V], acc[V];
                Rows::values(q0[u], qa);
                Rows::values(r0[u], ra);
                Rows::values(q1[u], qb);
                Rows::values(r1[u], rb);
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    const float e0 = a.combine == 0 ? qa[e] * ra[e] : qa[e] + ra[e];
                    const float e1 = a.combine == 0 ? qb[e] * rb[e] : qb[e] + rb[e];
                    acc[e] = e0 + e1;
                }
                out[u] = st<T>::pack(acc);
            }
        } else if (!BAGS) {
            ID id[RW];
#pragma unroll
            for (int u = 0; u < RW; ++u) id[u] = ids[(b0 + (u < nr ? u : 0)) * a.F + f];
            bool ok[RW];
            typename Rows::Raw qw[RW], rw[RW];
#pragma unroll
            for (int u = 0; u < RW; ++u) {
                uint32_t qi = 0, ri = 0;
                ok[u] = qr_split<ID>(id[u], a, qi, ri);
                if (!ok[u]) qi = ri = 0;
                qw[u] = rows.load_q(qi);
                rw[u] = rows.load_r(ri);
            }
            bool bad = false;
#pragma unroll
            for (int u = 0; u < RW; ++u) {
                float qv[V], rv[V], acc[V];
                Rows::values(qw[u], qv);
                Rows::values(rw[u], rv);
#pragma unroll
                for (int e = 0; e < V; ++e) acc[e] = ok[u] ? (a.combine == 0 ? qv[e] * rv[e] : qv[e] + rv[e]) : 0.0f;
                out[u] = st<T>::pack(acc);
                bad = bad || (u < nr && !ok[u]);
            }
            if (bad && cc == 0) atomicOr(a.err, 1);
        } else {
            int64_t beg[RW], end[RW];
#pragma unroll
            for (int u = 0; u < RW; ++u) {
                const int64_t bag = (b0 + (u < nr ? u : 0)) * a.F + f;
                beg[u] = a.offsets[bag];
                end[u] = u < nr ? a.offsets[bag + 1] : beg[u];
            }
            // a bag is taken in chunks of K ids: the chunk's id loads, then all its row
            // loads, are in flight together; the rows are then added in bag order
            constexpr int K = HASHED ? (GATHER_BAG_CHUNK + 1) / 2 : GATHER_BAG_CHUNK;
            bool bad = false;
#pragma unroll
            for (int u = 0; u < RW; ++u) {
                float acc[V];
#pragma unroll
                for (int e = 0; e < V; ++e) acc[e] = 0.0f;
                bool started = false;
                // the next chunk's ids are loaded before this chunk's rows, so a chunk
                // waits for one row latency rather than an id latency and a row latency
                ID nid[K];
#pragma unroll
                for (int k = 0; k < K; ++k) nid[k] = beg[u] + k < end[u] ? ids[beg[u] + k] : ID(0);
                for (int64_t p0 = beg[u]; p0 < end[u]; p0 += K) {
                    const int n = end[u] - p0 < K ? (int)(end[u] - p0) : K;
                    ID id[K];
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        id[k] = nid[k];
                        if (p0 + K + k < end[u]) nid[k] = ids[p0 + K + k];
                    }
                    if (HASHED) {
                        typename Rows::Raw q0[K], r0[K], q1[K], r1[K];
#pragma unroll
                        for (int k = 0; k < K; ++k)
                            if (k < n) {
                                uint32_t qi[2], ri[2];
                                hash_split((int64_t)id[k], a, qi, ri);
                                q0[k] = rows.load_q(qi[0]);
                                r0[k] = rows.load_r(ri[0]);
                                q1[k] = rows1.load_q(qi[1]);
                                r1[k] = rows1.load_r(ri[1]);
                            }
#pragma unroll
                        for (int k = 0; k < K; ++k)
                            if (k < n) {
                                float qa[V], ra[V], qb[V], rb[V];
                                Rows::values(q0[k], qa);
                                Rows::values(r0[k], ra);
                                Rows::values(q1[k], qb);
                                Rows::values(r1[k], rb);
#pragma unroll
                                for (int e = 0; e < V; ++e) {
                                    const float e0 = a.combine == 0 ? qa[e] * ra[e] : qa[e] + ra[e];
                                    const float e1 = a.combine == 0 ? qb[e] * rb[e] : qb[e] + rb[e];
                                    acc[e] = started ? acc[e] + (e0 + e1) : e0 + e1;
                                }
                                started = true;
                            }
                    } else {
                        bool ok[K];
                        typename Rows::Raw qw[K], rw[K];
#pragma unroll
                        for (int k = 0; k < K; ++k) {
                            uint32_t qi = 0, ri = 0;
                            ok[k] = k < n && qr_split<ID>(id[k], a, qi, ri);
                            bad = bad || (k < n && !ok[k]);
                            if (ok[k]) {
                                qw[k] = rows.load_q(qi);
                                rw[k] = rows.load_r(ri);
                            }
                        }
#pragma unroll
                        for (int k = 0; k < K; ++k)
                            if (ok[k]) {
                                float qv[V], rv[V];
                                Rows::values(qw[k], qv);
                                Rows::values(rw[k], rv);
#pragma unroll
                                for (int e = 0; e < V; ++e) {
                                    const float x = a.combine == 0 ? qv[e] * rv[e] : qv[e] + rv[e];
                                    acc[e] = started ? acc[e] + x : x;
                                }
                                started = true;
                            }
                    }
                }
                if (u < nr) *(u32x4_t*)(x0 + (b0 + u) * d + (int64_t)c * V) = st<T>::pack(acc);
            }
            if (bad && cc == 0) atomicOr(a.err, 1);
            continue;  // each bag's row was stored when its sum was complete
        }
#pragma unroll
        for (int u = 0; u < RW; ++u)
            if (u < nr) *(u32x4_t*)(x0 + (b0 + u) * d + (int64_t)c * V) = out[u];
    }
}

// Middle-max quantization of one row per wave (D <= 256: lane holds columns
// lane + 64 u). Every operation is one IEEE float operation in the order the
// definition writes it (no contraction), rounding to nearest even.
template <typename T>
__global__ __launch_bounds__(256) void k_quantize_rows(int64_t rows, int D, const T* __restrict__ x,
                                                       int8_t* __restrict__ codes, float2* __restrict__ params) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const T* xr = x + row * D;
    float v[4];
    float mn = INFINITY, mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int c = lane + 64 * u;
        v[u] = c < D ? st<T>::load(xr + c) : 0.0f;
        if (c < D) {
            mn = fminf(mn, v[u]);
            mx = fmaxf(mx, v[u]);
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        mn = fminf(mn, __shfl_xor(mn, off));
        mx = fmaxf(mx, __shfl_xor(mx, off));
    }
    mn = __fadd_rn(mn, 0.0f);  // a zero extreme counts as +0
    mx = __fadd_rn(mx, 0.0f);
    const float middle = __fdiv_rn(__fadd_rn(__fmul_rn(mx, 128.0f), __fmul_rn(mn, 127.0f)), 255.0f);
    const float scale = __fdiv_rn(__fsub_rn(mx, mn), 255.0f);
    if (lane == 0) params[row] = make_float2(middle, scale);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int c = lane + 64 * u;
        if (c < D) {
            float q = 0.0f;
            if (scale > 0.0f) q = fminf(fmaxf(__builtin_rintf(__fdiv_rn(__fsub_rn(v[u], middle), scale)), -128.0f), 127.0f);
            codes[row * D + c] = (int8_t)(int)q;
        }
    }
}

template <template <typename> class R>
hipError_t launch_gather_rows(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s) {
    const int V = bf16 ? 8 : 4;
    const int64_t cpr = (a.F * (int64_t)a.D + a.Nd) / V;
    if (a.batch == 0 || cpr == 0) return hipSuccess;
    // nx 64-column slices of a row times ny groups of 4 waves x rw rows (grid-stride
    // beyond), as one dimension
    const bool bags = a.offsets != nullptr;
    const int rw = bags ? GATHER_BAG_ROWS : GATHER_ROWS;
    const int64_t nx = (cpr + 63) / 64;
    int64_t ygroups = (a.batch + 4 * rw - 1) / (4 * rw);
    if (ygroups > 65535) ygroups = 65535;
    if (nx * ygroups > (1 << 24) - 1) ygroups = ((1 << 24) - 1) / nx;  // grid of under 2^32 threads
    if (ygroups < 1) return hipErrorInvalidValue;
    const int ny = (int)ygroups;
    const dim3 grid((unsigned)(nx * ygroups));
    const int threads = 256;
#define RDCN_GATHER(T, ID, BG)                                                                         \
    do {                                                                                               \
        if (a.hashed) hipLaunchKernelGGL((k_qr_gather<T, ID, BG, R<T>, true>), grid, dim3(threads), 0, s, a, ny); \
        else hipLaunchKernelGGL((k_qr_gather<T, ID, BG, R<T>, false>), grid, dim3(threads), 0, s, a, ny);          \
    } while (0)
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

hipError_t launch_qr_gather(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s) {
    return launch_gather_rows<StorageRows>(a, bf16, ids64, s);
}

hipError_t launch_qr_gather_q8(const GatherArgs& a, bool bf16, bool ids64, hipStream_t s) {
    return launch_gather_rows<Q8Rows>(a, bf16, ids64, s);
}

hipError_t launch_quantize_rows(int64_t rows, int D, const void* tables, int8_t* codes, float* params, bool bf16,
                                hipStream_t s) {
    if (rows == 0) return hipSuccess;
    const dim3 grid((unsigned)((rows + 3) / 4));
    if (bf16)
        hipLaunchKernelGGL(k_quantize_rows<bf16_t>, grid, dim3(256), 0, s, rows, D, (const bf16_t*)tables, codes,
                           (float2*)params);
    else
        hipLaunchKernelGGL(k_quantize_rows<float>, grid, dim3(256), 0, s, rows, D, (const float*)tables, codes,
                           (float2*)params);
    return hipGetLastError();
}

}  // namespace rdcn
