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
// Tiling: 64 x 64 and 128 x 128 blocks use 256 threads = 4 waves in a 2 x 2 grid,
// each wave owning a (BM/2) x (BN/2) block of 16 x 16 MFMA tiles
// (v_mfma_f32_16x16x32_bf16); large products use 256 x 256 or 256 x 128 blocks of
// 8 waves with 32 x 32 tiles (v_mfma_f32_32x32x16_bf16). Each K step of 64 is one
// stage of a 2- or 3-stage ring in LDS, filled by direct global-to-LDS loads one or
// two steps ahead of the multiply (a scalar base advanced along K plus per-lane offsets
// computed once per block; a tail stage's positions past K are loaded from a block of
// zeros, so every stage runs the same multiplies); K-strided operands stay [k][m] in LDS and are
// transposed on the way out by ds_read_b64_tr_b16, so no operand is ever
// transposed in memory. The MFMA is issued with B as its first operand, so each
// lane ends up with four consecutive output columns of one row: epilogue loads
// and stores are 8- or 16-byte vectors along the rows of x0, x_l, t and g.
#include <cmath>
#include <type_traits>

#include "device_common.h"
#include "gemm.h"
#include "mlp_common.h"

namespace rdcn {

namespace {

constexpr int BK = 64;

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

// hi = bf16(v), lo = bf16(v - hi): the pair carries about 16 significant bits.
// (float storage has no split; the lo plane is not used there.)
template <typename T>
__device__ __forceinline__ void store_split4(T* hi, T* lo, const float* v);
template <>
__device__ __forceinline__ void store_split4<float>(float* hi, float*, const float* v) {
    store4<float>(hi, v);
}
template <>
__device__ __forceinline__ void store_split4<bf16_t>(bf16_t* hi, bf16_t* lo, const float* v) {
    const uint32_t h0 = f32_to_bf16(v[0]), h1 = f32_to_bf16(v[1]), h2 = f32_to_bf16(v[2]), h3 = f32_to_bf16(v[3]);
    float r[4] = {v[0] - __uint_as_float(h0 << 16), v[1] - __uint_as_float(h1 << 16), v[2] - __uint_as_float(h2 << 16),
                  v[3] - __uint_as_float(h3 << 16)};
    *(uint2*)hi = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
    store4<bf16_t>(lo, r);
}

// Epilogue on four consecutive columns n .. n+3 of row m (n + 3 < N guaranteed).
template <typename T>
__device__ __forceinline__ void epilogue4(const GemmArgs& g, int64_t m, int64_t n, int z, float* v) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] *= g.scale;
    switch (g.epi) {
        case EPI_STORE:
            if (g.c2) store_split4((T*)g.c + m * g.ldc + n, (T*)g.c2 + m * g.ldc + n, v);
            else store4<T>((T*)g.c + m * g.ldc + n, v);
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
            if (g.xl2) {
                float lo[4];
                load4<T>((const T*)g.xl2 + m * g.ldx + n, lo);
#pragma unroll
                for (int e = 0; e < 4; ++e) xl[e] += lo[e];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[e] += b[e];
                xn[e] = x0[e] * v[e] + xl[e];
            }
            store4<T>((T*)g.t_out + m * g.ldx + n, v);
            if (g.c2) store_split4((T*)g.c + m * g.ldc + n, (T*)g.c2 + m * g.ldc + n, xn);
            else store4<T>((T*)g.c + m * g.ldc + n, xn);
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

template <typename T>
__device__ __forceinline__ void load8(const T* p, float* v) {
    load4<T>(p, v);
    load4<T>(p + 4, v + 4);
}
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, float* v) {
    const u32x4_t w = *(const u32x4_t*)p;
    st<bf16_t>::unpack(w, v);
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const float* v) {
    store4<T>(p, v);
    store4<T>(p + 4, v + 4);
}
template <>
__device__ __forceinline__ void store8<bf16_t>(bf16_t* p, const float* v) {
    *(u32x4_t*)p = st<bf16_t>::pack(v);
}
template <typename T>
__device__ __forceinline__ void store_split8(T* hi, T* lo, const float* v) {
    store_split4<T>(hi, lo, v);
    store_split4<T>(hi + 4, lo + 4, v + 4);
}

// Output of eight values v at element offset off of c (and of c2, as c2_kind says).
template <typename T>
__device__ __forceinline__ void store_out8(const GemmArgs& g, int64_t off, const float* v, bool& ovf) {
    if (g.c_f16) *(u32x4_t*)((_Float16*)g.c + off) = pack_f16x8(v, ovf);
    else if (g.c2 && g.c2_kind == C2_LO) {
        store_split8((T*)g.c + off, (T*)g.c2 + off, v);
        return;
    } else store8<T>((T*)g.c + off, v);
    if (!g.c2) return;
    if (g.c2_kind == C2_F16) *(u32x4_t*)((_Float16*)g.c2 + off) = pack_f16x8(v, ovf);
    else store8<bf16_t>((bf16_t*)g.c2 + off, v);
}

// Epilogue on eight consecutive columns n .. n+7 of row m (n + 7 < N guaranteed):
// 16-byte accesses along the rows of x0, x_l, t and g. `ovf` collects f16 range
// overflows of the outputs written as f16.
template <typename T>
__device__ __forceinline__ void epilogue8(const GemmArgs& g, int64_t m, int64_t n, int z, float* v, bool& ovf) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] *= g.scale;
    switch (g.epi) {
        case EPI_STORE:
            store_out8<T>(g, m * g.ldc + n, v, ovf);
            break;
        case EPI_STORE_F32:
            store8<float>((float*)g.c + m * g.ldc + n, v);
            break;
        case EPI_PARTIAL:
            store8<float>((float*)g.c + ((int64_t)z * g.M + m) * g.ldc + n, v);
            break;
        case EPI_CROSS: {
            float b[8], x0[8], xl[8], xn[8];
            load8<T>((const T*)g.bias + n, b);
            load8<T>((const T*)g.x0 + m * g.ldx + n, x0);
            if (g.xl_f16) unpack_f16x8(*(const u32x4_t*)((const _Float16*)g.xl + m * g.ldx + n), xl);
            else load8<T>((const T*)g.xl + m * g.ldx + n, xl);
            if (g.xl2) {
                float lo[8];
                load8<T>((const T*)g.xl2 + m * g.ldx + n, lo);
#pragma unroll
                for (int e = 0; e < 8; ++e) xl[e] += lo[e];
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                v[e] += b[e];
                xn[e] = x0[e] * v[e] + xl[e];
            }
            store8<T>((T*)g.t_out + m * g.ldx + n, v);
            store_out8<T>(g, m * g.ldc + n, xn, ovf);
            break;
        }
        case EPI_RESID:
        case EPI_RESID_X0: {
            float gi[8];
            if (g.gin_f32) load8<float>((const float*)g.gin + m * g.ldx + n, gi);
            else load8<T>((const T*)g.gin + m * g.ldx + n, gi);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += gi[e];
            float* out = (float*)g.c + m * g.ldc + n;
            if (g.epi == EPI_RESID_X0) {
                float o[8];
                load8<float>(out, o);
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] += o[e];
            }
            store8<float>(out, v);
            break;
        }
    }
}

// MLP epilogues on eight consecutive columns n .. n+7 of row m (n + 7 < N); returns
// this thread's share of the row dot product sum(v * act) (EPI_MLP_BWD with act).
// EPI_MLP_FWD with c2 (c2_kind C2_F16) also writes an f16 copy of the activations.
template <typename T>
__device__ __forceinline__ float mlp_epilogue8(const GemmArgs& g, int64_t m, int64_t n, float* v, bool& ovf) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] *= g.scale;
    T* out = (T*)g.c + m * g.ldc + n;
    if (g.epi == EPI_MLP_FWD) {
        float b[8];
        load8<T>((const T*)g.bias + n, b);
        const float gate = g.rowv ? sigmoid_f(g.rowv[m]) : 1.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = relu_f(v[e] + b[e]) * gate;
        store8<T>(out, v);
        if (g.c2) *(u32x4_t*)((_Float16*)g.c2 + m * g.ldc + n) = pack_f16x8(v, ovf);
        return 0.f;
    }
    if (g.colv) {  // the gate's rank-one term
        float cv[8];
        load8<T>((const T*)g.colv + n, cv);
        const float r = g.rowv[m];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = fmaf(r, cv[e], v[e]);
    }
    if (!g.act) {
        store8<T>(out, v);
        return 0.f;
    }
    float a[8];
    load8<T>((const T*)g.act + m * g.ldx + n, a);
    const float rho = g.rowg ? sigmoid_f(g.rowg[m]) : 1.f;
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        dot = fmaf(v[e], a[e], dot);
        v[e] = a[e] > 0.f ? rho * v[e] : 0.f;
    }
    store8<T>(out, v);
    return dot;
}

__device__ __forceinline__ int xcd_remap(int id, int n) {
    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of tiles so neighbouring tiles share its L2. The last
    // n % 8 workgroups keep their own index.
    const int full = n / 8 * 8;
    if (id >= full) return id;
    return (id % 8) * (n / 8) + id / 8;
}

// ---------------------------------------------------------------------------
// LDS layouts (one stage = one KB-deep slice of A and of B; KB = 64 in every launch,
// the layouts also hold for KB = 32):
//  K-contiguous operand, ROWS x KB bf16: row r holds KB/8 chunks of 16 bytes; the
//    chunk of logical k-block kc sits in slot kc ^ kc_swz(r) (((r >> 1) & 7) for KB = 64).
//    Two rows share a 256-byte bank window, so 16 consecutive rows reading the same kc hit 16
//    distinct 16-byte bank groups (ds_read_b128 without conflicts).
//  K-strided operand, 64 k-rows x ROWS bf16 (rows contiguous along m): a k-row
//    holds ROWS/16 chunks of 32 bytes (16 m values); chunk c sits in slot
//    c ^ h(k). MFMA fragments are read with ds_read_b64_tr_b16, which transposes
//    within each 16-lane group: lane (g, j) reads the 4 m values 4(j%4)..+3 of
//    k-row 8g + j/4 (+4 for the second read) and receives the 8 k values of its
//    own m. h(k) spreads the 16 k-rows of one read over all bank groups.
// Loads go straight from global memory into LDS (global_load_lds, 16 bytes per
// lane, lane l writes bytes 16 l .. 16 l + 15 of a 1 KiB block), so the global
// address of each lane is chosen to land in the swizzled position.
// ---------------------------------------------------------------------------
#define LDS_AS __attribute__((address_space(3)))
typedef short s16x4_t __attribute__((ext_vector_type(4)));

// 16-byte direct global-to-LDS load: lane l's 16 bytes land at LDS byte address
// m0 + 16 l. Issued through asm so that the compiler adds no waits of its own:
// every consumer below waits explicitly (wait_vmcnt + s_barrier) for the stage
// it reads. M0 needs one wait state after it is written.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gptr), "s"(lds_base)
                 : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const bf16_t* p) { return (uint32_t)(uintptr_t)((LDS_AS const char*)p); }

// Slot XOR of row r of a K-contiguous operand stage of KB bf16 per row: KB = 64 (8 slots
// of 16 bytes, two rows per 256-byte bank window) or 32 (4 slots, four rows per window);
// 16 consecutive rows reading one slot hit 16 distinct 16-byte bank groups.
template <int KB>
__device__ __forceinline__ int kc_swz(int r) {
    return KB == 64 ? ((r >> 1) & 7) : ((r >> 2) & 3);
}

template <int ROWS>
__device__ __forceinline__ int kstr_swz(int k) {
    // ROWS = 128: 8 slots of 32 B per k-row; ROWS = 256: 16 slots, two 256 B windows per
    // k-row (the XOR spreads the k-rows of one read over all 8 slot positions of a window);
    // ROWS = 64: 4 slots, two k-rows per 256 B window
    return ROWS >= 128 ? (((k & 3) << 1) | ((k >> 3) & 1)) : ((((k >> 1) & 1) << 1) | ((k >> 3) & 1));
}

// 16 zero bytes in device memory: the source of the direct-to-LDS loads of K positions
// past a range, so a tail stage arrives in LDS already zero-padded.
__device__ __align__(16) const uint32_t kZero16[4] = {0u, 0u, 0u, 0u};

// Issue this thread's direct-to-LDS loads of one stage (KB deep) for one operand (NW waves).
// Rows past `rows` re-read the last row (their results are discarded); K positions at
// or past kend read zeros. K-contiguous operands need kend - k0 to be a multiple of 8
// (a 16-byte piece never straddles kend: K is a multiple of 8 for bf16 models).
template <int ROWS, bool KS, int NW, int KB>
__device__ __forceinline__ void stage_load(const bf16_t* __restrict__ base, int64_t ld, int64_t rows, int64_t row0,
                                           int64_t k0, int64_t kend, bf16_t* lds, int wave, int lane) {
    constexpr int NI = ROWS * KB / (512 * NW);  // wave-instructions per thread (1 KiB each)
#pragma unroll
    for (int j = 0; j < NI; ++j) {
        const int blk = wave * NI + j;  // 1 KiB block index within the stage
        int64_t gr, gk;
        if (!KS) {
            constexpr int CPR = KB / 8;    // 16-byte chunks per row
            constexpr int RPB = 64 / CPR;  // rows per 1 KiB block
            const int r = blk * RPB + lane / CPR;
            const int kc = (lane % CPR) ^ kc_swz<KB>(r);
            gr = row0 + r;
            gk = k0 + kc * 8;
            if (gr >= rows) gr = rows - 1;
            const void* src = gk < kend ? (const void*)(base + gr * ld + gk) : (const void*)kZero16;
            dma16(src, lds_addr(lds) + (uint32_t)__builtin_amdgcn_readfirstlane(blk) * 1024u);
        } else {
            constexpr int RPB = ROWS == 256 ? 2 : (ROWS == 128 ? 4 : 8);  // k-rows per 1 KiB block
            constexpr int QPR = 64 / RPB;             // 16-byte pieces per k-row
            const int kr = blk * RPB + lane / QPR;
            const int q = lane % QPR;
            const int c = (q >> 1) ^ kstr_swz<ROWS>(kr);
            gk = k0 + kr;
            gr = row0 + c * 16 + (q & 1) * 8;
            if (gr >= rows) gr = rows - 8;
            const void* src = gk < kend ? (const void*)(base + gk * ld + gr) : (const void*)kZero16;
            dma16(src, lds_addr(lds) + (uint32_t)__builtin_amdgcn_readfirstlane(blk) * 1024u);
        }
    }
}

// The same loads with the address split into a scalar base (wave-uniform, advanced by
// BK along K every step) and a loop-invariant per-lane 32-bit byte offset, computed
// once per block by stage_offsets: no address arithmetic between the barrier and the
// multiplies of a step.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ void dma16_s(uint32_t voff, const void* sbase, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(sbase), "s"(lds_base)
                 : "memory");
}

// Per-lane byte offsets of stage_load's loads relative to element (row_base, k0) of a
// K-contiguous operand ([rows][ld]) or (k0, row_base) of a K-strided one ([K][ld]),
// with rows clamped as stage_load clamps them; row_base <= every clamped row.
template <int ROWS, bool KS, int NW, int KB>
__device__ __forceinline__ void stage_offsets(int64_t ld, int64_t rows, int64_t row0, int64_t row_base, int wave,
                                              int lane, uint32_t (&off)[ROWS * KB / (512 * NW)]) {
    constexpr int NI = ROWS * KB / (512 * NW);
#pragma unroll
    for (int j = 0; j < NI; ++j) {
        const int blk = wave * NI + j;
        if (!KS) {
            constexpr int CPR = KB / 8, RPB = 64 / CPR;
            const int r = blk * RPB + lane / CPR;
            const int kc = (lane % CPR) ^ kc_swz<KB>(r);
            int64_t gr = row0 + r;
            if (gr >= rows) gr = rows - 1;
            off[j] = (uint32_t)(((gr - row_base) * ld + kc * 8) * 2);
        } else {
            constexpr int RPB = ROWS == 256 ? 2 : (ROWS == 128 ? 4 : 8);
            constexpr int QPR = 64 / RPB;
            const int kr = blk * RPB + lane / QPR;
            const int q = lane % QPR;
            const int c = (q >> 1) ^ kstr_swz<ROWS>(kr);
            int64_t gr = row0 + c * 16 + (q & 1) * 8;
            if (gr >= rows) gr = rows - 8;
            off[j] = (uint32_t)((kr * ld + (gr - row_base)) * 2);
        }
    }
}

// MFMA fragment (16 rows x 32 k) of an operand tile at row offset rt, k offset ks.
template <int ROWS, bool KS, int KB>
__device__ __forceinline__ bf16x8_t load_frag(const bf16_t* lds, int rt, int ks, int lane) {
    const int i = lane & 15, g = lane >> 4;
    if (!KS) {
        const int r = rt + i;
        const int kc = ks / 8 + g;
        return __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(lds + r * KB + ((kc ^ kc_swz<KB>(r)) * 8)));
    } else {
        const int c = rt / 16;
        s16x4_t lo, hi;
        {
            const int kr = ks + 8 * g + (i >> 2);
            const int off = kr * ROWS + ((c ^ kstr_swz<ROWS>(kr)) * 16) + (i & 3) * 4;
            lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4_t*)(lds + off));
        }
        {
            const int kr = ks + 8 * g + 4 + (i >> 2);
            const int off = kr * ROWS + ((c ^ kstr_swz<ROWS>(kr)) * 16) + (i & 3) * 4;
            hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4_t*)(lds + off));
        }
        typedef short s16x8_t __attribute__((ext_vector_type(8)));
        const s16x8_t v = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        return __builtin_bit_cast(bf16x8_t, v);
    }
}

// MFMA fragment (32 rows x 16 k) for v_mfma_f32_32x32x16_bf16: lane l holds row
// rt + l % 32 and the 8 k values ks + 8 (l / 32) .. + 7. K-strided operands use the
// same transposing reads as above, each 16-lane group G supplying row chunk
// rt / 16 + (G & 1) and k rows from ks + 8 (G >> 1).
template <int ROWS, bool KS, int KB>
__device__ __forceinline__ bf16x8_t load_frag32(const bf16_t* lds, int rt, int ks, int lane) {
    if (!KS) {
        const int r = rt + (lane & 31);
        const int kc = ks / 8 + (lane >> 5);
        return __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(lds + r * KB + ((kc ^ kc_swz<KB>(r)) * 8)));
    } else {
        const int i = lane & 15, G = lane >> 4;
        const int c = rt / 16 + (G & 1);
        const int kb = ks + 8 * (G >> 1);
        s16x4_t lo, hi;
        {
            const int kr = kb + (i >> 2);
            const int off = kr * ROWS + ((c ^ kstr_swz<ROWS>(kr)) * 16) + (i & 3) * 4;
            lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4_t*)(lds + off));
        }
        {
            const int kr = kb + 4 + (i >> 2);
            const int off = kr * ROWS + ((c ^ kstr_swz<ROWS>(kr)) * 16) + (i & 3) * 4;
            hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4_t*)(lds + off));
        }
        typedef short s16x8_t __attribute__((ext_vector_type(8)));
        const s16x8_t v = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        return __builtin_bit_cast(bf16x8_t, v);
    }
}

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ void wait_vmcnt(int n) {
    // s_waitcnt with vmcnt = n (n <= 63), expcnt and lgkmcnt left at their maxima
    switch (n) {
        case 0: __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8)); break;
        case 2: __builtin_amdgcn_s_waitcnt(2 | (7 << 4) | (15 << 8)); break;
        case 4: __builtin_amdgcn_s_waitcnt(4 | (7 << 4) | (15 << 8)); break;
        case 6: __builtin_amdgcn_s_waitcnt(6 | (7 << 4) | (15 << 8)); break;
        case 8: __builtin_amdgcn_s_waitcnt(8 | (7 << 4) | (15 << 8)); break;
        case 12: __builtin_amdgcn_s_waitcnt(12 | (7 << 4) | (15 << 8)); break;
        case 16: __builtin_amdgcn_s_waitcnt(0 | (1 << 14) | (7 << 4) | (15 << 8)); break;
        default: __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8)); break;
    }
}

__device__ __forceinline__ void wait_lgkm0() {
    // s_waitcnt lgkmcnt(0), vmcnt and expcnt left at their maxima
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));
}

// The two MFMA shapes for bf16 or f16 operands (the same bit patterns either way: the
// LDS layout and fragment reads do not depend on the element type).
template <bool F16>
__device__ __forceinline__ f32x16_t mfma32x32x16(const bf16x8_t& b, const bf16x8_t& a, const f32x16_t& c) {
    if constexpr (F16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8_t, b), __builtin_bit_cast(half8_t, a),
                                                      c, 0, 0, 0);
    else return __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a, c, 0, 0, 0);
}
template <bool F16>
__device__ __forceinline__ f32x4_t mfma16x16x32(const bf16x8_t& b, const bf16x8_t& a, const f32x4_t& c) {
    if constexpr (F16)
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, b), __builtin_bit_cast(half8_t, a),
                                                      c, 0, 0, 0);
    else return __builtin_amdgcn_mfma_f32_16x16x32_bf16(b, a, c, 0, 0, 0);
}

// Block tile BM x BN over WM x WN waves; each wave owns a (BM/WM) x (BN/WN) block of
// MFMA tiles: 16 x 16 (v_mfma_f32_16x16x32_bf16) or, with M32, 32 x 32
// (v_mfma_f32_32x32x16_bf16, twice the flops per clock).
template <int BM, int BN, bool AKS, bool BKS, int ST, int WM, int WN, bool M32, bool F16, int KB>
struct Pipe {
    static constexpr int NW = WM * WN, THREADS = 64 * NW;
    static constexpr int MT = M32 ? 32 : 16;
    static constexpr int TM = BM / WM / MT, TN = BN / WN / MT;  // MFMA tiles per wave
    static constexpr int LOADS = (BM + BN) * KB / (512 * NW);   // load instructions per thread per stage
    static constexpr int STAGE_ELEMS = (BM + BN) * KB;
    using acc_t = typename std::conditional<M32, f32x16_t, f32x4_t>::type;

    static constexpr int NIA = BM * KB / (512 * NW), NIB = BN * KB / (512 * NW);  // loads per thread per stage

    struct Ctx {
        const GemmArgs* g;
        int nk;          // K tiles per A plane
        int ntot;        // nk * planes
        int64_t kbeg, kend, m0, n0;
        int tid;
        bool fast;                  // per-lane offsets fit 32 bits: loads use scalar base + offset
        int64_t abase, bbase;       // first row of each operand the offsets are taken from
        uint32_t aoff[NIA], boff[NIB];
    };

    // Per-block setup of the scalar-base loads.
    __device__ __forceinline__ static void prepare(Ctx& c) {
        const GemmArgs& g = *c.g;
        const int lane = c.tid & 63, wave = c.tid >> 6;
        // K-strided rows clamp to rows - 8, possibly below the block's first row
        c.abase = AKS ? (c.m0 + 8 <= g.M ? c.m0 : (g.M >= 8 ? g.M - 8 : 0)) : c.m0;
        c.bbase = BKS ? (c.n0 + 8 <= g.N ? c.n0 : (g.N >= 8 ? g.N - 8 : 0)) : c.n0;
        // largest offset: a block's rows (or its BK k-rows) times the stride, plus a row
        const double amax = ((AKS ? KB : BM) + 1.0) * (double)g.lda * 2.0 + BM * 2.0;
        const double bmax = ((BKS ? KB : BN) + 1.0) * (double)g.ldb * 2.0 + BN * 2.0;
        c.fast = amax < 2.0e9 && bmax < 2.0e9 && g.M >= 8 && g.N >= 8 && g.K >= 8;
        if (c.fast) {
            stage_offsets<BM, AKS, NW, KB>(g.lda, g.M, c.m0, c.abase, wave, lane, c.aoff);
            stage_offsets<BN, BKS, NW, KB>(g.ldb, g.N, c.n0, c.bbase, wave, lane, c.boff);
        }
    }

    // Loads of tile `t` (clamped to the last tile; planes follow each other) into `buf`.
    __device__ __forceinline__ static void issue(const Ctx& c, int t, bf16_t* buf) {
        const int lane = c.tid & 63, wave = c.tid >> 6;
        if (t > c.ntot - 1) t = c.ntot - 1;
        const int plane = t >= c.nk;
        const int64_t k0 = c.kbeg + (int64_t)(t - plane * c.nk) * KB;
        const bf16_t* a = (const bf16_t*)(plane ? c.g->a2 : c.g->a);
        const bf16_t* b = (const bf16_t*)c.g->b;
        if (c.fast && k0 + KB <= c.kend) {  // a whole stage: no clamp along K
            const void* sa = uniform_ptr(AKS ? a + k0 * c.g->lda + c.abase : a + c.abase * c.g->lda + k0);
            const void* sb = uniform_ptr(BKS ? b + k0 * c.g->ldb + c.bbase : b + c.bbase * c.g->ldb + k0);
            const uint32_t la = lds_addr(buf), lb = lds_addr(buf + BM * KB);
#pragma unroll
            for (int j = 0; j < NIA; ++j)
                dma16_s(c.aoff[j], sa, la + (uint32_t)__builtin_amdgcn_readfirstlane(wave * NIA + j) * 1024u);
#pragma unroll
            for (int j = 0; j < NIB; ++j)
                dma16_s(c.boff[j], sb, lb + (uint32_t)__builtin_amdgcn_readfirstlane(wave * NIB + j) * 1024u);
            return;
        }
        stage_load<BM, AKS, NW, KB>(a, c.g->lda, c.g->M, c.m0, k0, c.kend, buf, wave, lane);
        stage_load<BN, BKS, NW, KB>(b, c.g->ldb, c.g->N, c.n0, k0, c.kend, buf + BM * KB, wave, lane);
    }

    // One step on tile kt held in `cur`; prefetch tile kt + ST - 1 into `nxt`.
    // Every step issues the same number of loads (past the last tile they re-read
    // it), so "all but the newest ST - 2 stages" is a fixed count on every path. A tail
    // tile's positions past the K range arrive as zeros (stage_load), so every step
    // runs the same multiplies.
    __device__ __forceinline__ static void step(const Ctx& c, bf16_t* cur, bf16_t* nxt, int kt,
                                                acc_t (&acc)[TM][TN]) {
        const int lane = c.tid & 63, wave = c.tid >> 6, wm = wave / WN, wn = wave % WN;
        wait_vmcnt(LOADS * (ST - 2));
        __builtin_amdgcn_s_barrier();
        issue(c, kt + ST - 1, nxt);
        if constexpr (M32) {
            // fragments double-buffered: the reads of substep s + 1 are issued before the
            // MFMAs of substep s, so LDS latency hides behind the matrix cores
            bf16x8_t af[2][TM], bfr[2][TN];
            auto frags = [&](int buf, int ks) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    af[buf][i] = load_frag32<BM, AKS, KB>(cur, wm * (BM / WM) + i * 32, ks, lane);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    bfr[buf][j] = load_frag32<BN, BKS, KB>(cur + BM * KB, wn * (BN / WN) + j * 32, ks, lane);
            };
            // (not with a K-strided A and eight accumulator tiles: that variant would spill)
            constexpr bool DB = !(AKS && TM * TN > 4);
            frags(0, 0);
#pragma unroll
            for (int s = 0; s < KB / 16; ++s) {
                if (!DB && s > 0) frags(s & 1, s * 16);
                if (DB && s + 1 < KB / 16) frags((s + 1) & 1, (s + 1) * 16);
                // keep the compiler from sinking those reads below the MFMAs
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] =
                            mfma32x32x16<F16>(bfr[s & 1][j], af[s & 1][i], acc[i][j]);
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
#pragma unroll
            for (int ks = 0; ks < KB; ks += 32) {
                bf16x8_t af[TM], bfr[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) af[i] = load_frag<BM, AKS, KB>(cur, wm * (BM / WM) + i * 16, ks, lane);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    bfr[j] = load_frag<BN, BKS, KB>(cur + BM * KB, wn * (BN / WN) + j * 16, ks, lane);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = mfma16x16x32<F16>(bfr[j], af[i], acc[i][j]);
            }
        }
    }
};

// Epilogue of a BM x BN block through LDS (`smem`, the stage ring of `ring_elems` bf16
// elements, reused once the K loop is done). With 16 x 16 tiles lane holds
// C[m = tile_m + (lane & 15)][n = tile_n + 4 (lane >> 4) + e]; with 32 x 32 tiles
// C[m = tile_m + lane % 32][n = tile_n + 8 q + 4 (lane / 32) + e] in acc[4 q + e]. The
// block is staged row-major, 64 rows at a time, then each thread applies the epilogue
// to 8 consecutive columns of a row.
template <int BM, int BN, int WM, int WN, bool M32, typename T, bool MLP, int THREADS, int RING, typename Acc,
          int TM, int TN>
__device__ __forceinline__ void block_epilogue(const GemmArgs& g, int64_t m0, int64_t n0, int z, Acc (&acc)[TM][TN],
                                               bf16_t* smem, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    bool ovf = false;                      // an output written as f16 overflowed
    constexpr int CH = 64;                 // rows staged per pass
    constexpr int CP = BN + 4;             // float pitch of a staged row
    static_assert(CH * CP * 4 <= RING * 2, "C staging must fit the stage ring");
    float* cs = (float*)smem;
#pragma unroll
    for (int h = 0; h < BM / CH; ++h) {
        __syncthreads();
        if constexpr (M32) {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wm * (BM / WM) + i * 32 + (lane & 31) - h * CH;
                if (row < 0 || row >= CH) continue;
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        *(f32x4_t*)(cs + row * CP + wn * (BN / WN) + j * 32 + 8 * q + 4 * (lane >> 5)) =
                            f32x4_t{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            }
        } else {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wm * (BM / WM) + i * 16 + (lane & 15) - h * CH;
                if (row < 0 || row >= CH) continue;
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    *(f32x4_t*)(cs + row * CP + wn * (BN / WN) + j * 16 + 4 * (lane >> 4)) = acc[i][j];
            }
        }
        __syncthreads();
        for (int q = tid; q < CH * (BN / 8); q += THREADS) {
            const int row = q / (BN / 8), col = (q % (BN / 8)) * 8;
            const int64_t m = m0 + h * CH + row, n = n0 + col;
            if (!MLP) {
                if (m >= g.M || n >= g.N) continue;
                float v[8];
                *(f32x4_t*)v = *(const f32x4_t*)(cs + row * CP + col);
                *(f32x4_t*)(v + 4) = *(const f32x4_t*)(cs + row * CP + col + 4);
                epilogue8<T>(g, m, n, z, v, ovf);
            } else {
                float part = 0.f;
                if (m < g.M && n < g.N) {
                    float v[8];
                    *(f32x4_t*)v = *(const f32x4_t*)(cs + row * CP + col);
                    *(f32x4_t*)(v + 4) = *(const f32x4_t*)(cs + row * CP + col + 4);
                    part = mlp_epilogue8<T>(g, m, n, v, ovf);
                }
                if (g.rowpart) {  // uniform: the BN / 8 threads of one row are an aligned lane group
#pragma unroll
                    for (int o = 1; o < BN / 8; o <<= 1) part += __shfl_xor(part, o);
                    if (col == 0 && m < g.M) g.rowpart[(int64_t)(n0 / BN) * g.M + m] = part;
                }
            }
        }
    }
    if (ovf) atomicOr(g.err, ERR_BIT_F16_RANGE);
}

// C = A B^T with an ST-stage direct-to-LDS pipeline of KB-deep stages (see layouts above).
template <int BM, int BN, bool AKS, bool BKS, int ST, int WM, int WN, bool M32, typename T, bool MLP, bool F16, int KB>
__global__ __launch_bounds__(64 * WM * WN, (ST == 2 && WM * WN == 4) ? 2 : 1)
__attribute__((amdgpu_waves_per_eu(WM * WN == 8 ? 2 : 1, WM * WN == 8 ? 2 : 8))) void k_gemm_mfma(GemmArgs g) {
    using P = Pipe<BM, BN, AKS, BKS, ST, WM, WN, M32, F16, KB>;
    // one buffer: the stage ring during the K loop, the C staging area afterwards
    __shared__ __attribute__((aligned(1024))) bf16_t smem[ST * P::STAGE_ELEMS];

    const int tid = threadIdx.x;
    const int tiles_n = (int)((g.N + BN - 1) / BN);
    const int tiles_m = (int)((g.M + BM - 1) / BM);
    const int t = xcd_remap(blockIdx.x, tiles_m * tiles_n);
    int tm, tn;
    if (g.group_m > 1) {
        // groups of group_m tile rows, walked column by column: the blocks that run
        // together on one XCD share group_m A panels and a few B panels in its L2
        const int per = g.group_m * tiles_n, grp = t / per, first = grp * g.group_m;
        const int rows = tiles_m - first < g.group_m ? tiles_m - first : g.group_m;
        const int r = t - grp * per;
        tm = first + r % rows;
        tn = r / rows;
    } else {
        tm = t / tiles_n;
        tn = t % tiles_n;
    }

    typename P::Ctx c;
    c.g = &g;
    c.tid = tid;
    c.m0 = (int64_t)tm * BM;
    c.n0 = (int64_t)tn * BN;
    const int z = blockIdx.z;
    // split-K ranges are multiples of BK (itself a multiple of every KB)
    const int64_t kchunk = ((g.K + (int64_t)gridDim.z * BK - 1) / ((int64_t)gridDim.z * BK)) * BK;
    c.kbeg = z * kchunk;
    c.kend = c.kbeg + kchunk < g.K ? c.kbeg + kchunk : g.K;
    c.nk = c.kbeg < c.kend ? (int)((c.kend - c.kbeg + KB - 1) / KB) : 0;
    c.ntot = c.nk * (g.a2 ? 2 : 1);
    P::prepare(c);

    typename P::acc_t acc[P::TM][P::TN];
#pragma unroll
    for (int i = 0; i < P::TM; ++i)
#pragma unroll
        for (int j = 0; j < P::TN; ++j)
#pragma unroll
            for (int e = 0; e < (M32 ? 16 : 4); ++e) acc[i][j][e] = 0.f;

    if (c.ntot > 0) {
        // ring of ST stages: step kt multiplies stage kt and fills slot (kt + ST - 1) % ST
        bf16_t* const s0 = smem;
        bf16_t* const s1 = smem + P::STAGE_ELEMS;
        bf16_t* const s2 = smem + (ST >= 3 ? 2 : 0) * P::STAGE_ELEMS;
#pragma unroll
        for (int u = 0; u < ST - 1; ++u) P::issue(c, u, smem + u * P::STAGE_ELEMS);
        if constexpr (ST == 2) {  // unrolled: fixed buffer pointers in each step
            for (int kt = 0; kt < c.ntot; kt += 2) {
                P::step(c, s0, s1, kt, acc);
                if (kt + 1 >= c.ntot) break;
                P::step(c, s1, s0, kt + 1, acc);
            }
        } else if constexpr (ST == 3) {
            for (int kt = 0; kt < c.ntot; kt += 3) {
                P::step(c, s0, s2, kt, acc);
                if (kt + 1 >= c.ntot) break;
                P::step(c, s1, s0, kt + 1, acc);
                if (kt + 2 >= c.ntot) break;
                P::step(c, s2, s1, kt + 2, acc);
            }
        } else {
            int cur = 0;
            for (int kt = 0; kt < c.ntot; ++kt) {
                const int nxt = cur == 0 ? ST - 1 : cur - 1;  // (kt + ST - 1) % ST
                P::step(c, smem + cur * P::STAGE_ELEMS, smem + nxt * P::STAGE_ELEMS, kt, acc);
                cur = cur + 1 == ST ? 0 : cur + 1;
            }
        }
        wait_vmcnt(0);  // the trailing re-read loads land before the workgroup ends
    }

    block_epilogue<BM, BN, WM, WN, M32, T, MLP, P::THREADS, ST * P::STAGE_ELEMS>(g, c.m0, c.n0, z, acc, smem, tid);
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

template <int BM, int BN, int ST, int WM, int WN, bool M32, typename T, int KB = 64>
hipError_t launch_tile(const GemmArgs& g, int splits, hipStream_t s) {
    const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    dim3 grid((unsigned)tiles, 1, (unsigned)splits);
#define RDCN_GEMM(AK, BKS, MLP) \
    hipLaunchKernelGGL((k_gemm_mfma<BM, BN, AK, BKS, ST, WM, WN, M32, T, MLP, false, KB>), grid, dim3(64 * WM * WN), 0, s, g)
    if (g.ops_f16) {
        // f16 operands: the forward products over f16 activations (both K-contiguous;
        // the cross projections and the MLP layers, no split-K for the latter)
        if (g.a_kstrided || g.b_kstrided || g.epi == EPI_MLP_BWD || g.a2) return hipErrorInvalidValue;
        if (g.epi == EPI_MLP_FWD) {
            if (splits != 1) return hipErrorInvalidValue;
            hipLaunchKernelGGL((k_gemm_mfma<BM, BN, false, false, ST, WM, WN, M32, T, true, true, KB>), grid,
                               dim3(64 * WM * WN), 0, s, g);
        } else {
            hipLaunchKernelGGL((k_gemm_mfma<BM, BN, false, false, ST, WM, WN, M32, T, false, true, KB>), grid,
                               dim3(64 * WM * WN), 0, s, g);
        }
    } else if (g.epi == EPI_MLP_FWD || g.epi == EPI_MLP_BWD) {
        // MLP layers: forward (both K-contiguous) and input gradient (B K-strided), no split-K
        if (g.a_kstrided || splits != 1) return hipErrorInvalidValue;
        if (g.b_kstrided) RDCN_GEMM(false, true, true); else RDCN_GEMM(false, false, true);
    } else if (g.a_kstrided) {
        if (g.b_kstrided) RDCN_GEMM(true, true, false); else RDCN_GEMM(true, false, false);
    } else {
        if (g.b_kstrided) RDCN_GEMM(false, true, false); else RDCN_GEMM(false, false, false);
    }
#undef RDCN_GEMM
    return hipGetLastError();
}

}  // namespace

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, bool bf16, bool allow_split, int split_blocks) {
    GemmPlan p;
    if (!bf16) {
        p.bm = p.bn = 64;
    } else {
        const int64_t t128 = ((M + 127) / 128) * ((N + 127) / 128);
        // Weight gradients (split-K allowed) take big tiles, which halve the operand
        // re-reads, and recover parallelism by splitting the batch dimension.
        if (t128 >= 240 || (allow_split && M >= 128 && N >= 128)) p.bm = p.bn = 128;
        else p.bm = p.bn = 64;
    }
    const int64_t tiles = ((M + p.bm - 1) / p.bm) * ((N + p.bn - 1) / p.bn);
    p.splits = 1;
    if (allow_split && tiles < 256) {
        int64_t s = (split_blocks + tiles - 1) / tiles;
        const int64_t kmax = K / 512;  // keep >= 8 K steps of 64 per split
        if (s > kmax) s = kmax;
        if (s > 16) s = 16;
        if (s < 1) s = 1;
        p.splits = (int)s;
    }
    // 128 x 128 tiles: two LDS stages (64 KiB) let two workgroups share a CU, which
    // overlaps one tile's loads and epilogue with the other's multiplies; this beats
    // a third stage (one workgroup per CU) at every K measured.
    p.stages = p.bm == 128 ? 2 : 3;
    // Large products (bound by the MFMA rate rather than by L2 -> LDS loads): eight
    // waves on 256-row blocks with 32 x 32 x 16 MFMAs, which halve the bytes loaded
    // per flop; 256 x 256 blocks when they still cover the chip, else 256 x 128.
    if (bf16 && (double)M * (double)N * (double)K >= 8.0e9) {
        // Per 64-deep K step a block needs max(MFMA time, load time): MFMA at ~3600
        // flop/clk per CU, loads at the ~24 B/clk per CU that L2 -> LDS sustains here.
        // A launch takes ceil(tiles / 256) rounds of that (one block per CU).
        auto cost = [&](int bm, int bn) {
            const double tiles = (double)((M + bm - 1) / bm) * (double)((N + bn - 1) / bn);
            const double mfma = 2.0 * bm * bn * 64 / 3600.0, load = (bm + bn) * 64 * 2 / 24.0;
            return std::ceil(tiles / 256.0) * (mfma > load ? mfma : load);
        };
        const double c256 = cost(256, 256), c128 = cost(256, 128);
        const int64_t t128 = ((M + 255) / 256) * ((N + 127) / 128);
        // Tiles in groups of four tile rows: the 32 blocks an XCD runs at once then
        // read 4 A panels and 8 B panels instead of 1-3 A panels and up to 32 B panels
        // (measured on the large workload's six products: 2-8% faster, none slower).
        if (c256 <= c128) {
            p.bm = p.bn = 256;
            p.splits = 1;
            p.stages = 2;
            p.group_m = 4;
        } else if (t128 >= 128) {
            p.bm = 256;
            p.bn = 128;
            p.splits = 1;
            p.stages = 3;
            p.group_m = 4;
        }
    }
    return p;
}

hipError_t launch_gemm(const GemmArgs& g, const GemmPlan& p, bool bf16, hipStream_t s) {
    if (g.M == 0 || g.N == 0) return hipSuccess;
    if (!bf16 && (g.epi == EPI_MLP_FWD || g.epi == EPI_MLP_BWD)) return hipErrorInvalidValue;
    if (!bf16) {
        const int64_t tiles = ((g.M + 63) / 64) * ((g.N + 63) / 64);
        hipLaunchKernelGGL(k_gemm_f32, dim3((unsigned)tiles, 1, (unsigned)p.splits), dim3(256), 0, s, g);
        return hipGetLastError();
    }
    GemmArgs ga = g;
    ga.group_m = p.group_m;
    if (p.bm == 256) {
        if (p.bn == 256) return launch_tile<256, 256, 2, 2, 4, true, bf16_t>(ga, p.splits, s);
        return launch_tile<256, 128, 3, 4, 2, true, bf16_t>(ga, p.splits, s);
    }
    if (p.bm == 128) {
        if (p.stages == 2) return launch_tile<128, 128, 2, 2, 2, false, bf16_t>(ga, p.splits, s);
        return launch_tile<128, 128, 3, 2, 2, false, bf16_t>(ga, p.splits, s);
    }
    if (p.stages == 2) return launch_tile<64, 64, 2, 2, 2, false, bf16_t>(ga, p.splits, s);
    return launch_tile<64, 64, 3, 2, 2, false, bf16_t>(ga, p.splits, s);
}

// dst = f16(src), 8 values per thread and step; err bit on values beyond the f16 range.
__global__ __launch_bounds__(256) void k_bf16_to_f16(const bf16_t* __restrict__ src, _Float16* __restrict__ dst,
                                                     int64_t n8, int* err) {
    bool ovf = false;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n8; i += (int64_t)gridDim.x * blockDim.x) {
        float v[8];
        st<bf16_t>::unpack(*(const u32x4_t*)(src + 8 * i), v);
        *(u32x4_t*)(dst + 8 * i) = pack_f16x8(v, ovf);
    }
    if (ovf) atomicOr(err, ERR_BIT_F16_RANGE);
}

hipError_t launch_bf16_to_f16(const void* src, void* dst, int64_t n, int* err, hipStream_t s) {
    if (n == 0) return hipSuccess;
    if (n % 8 || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return hipErrorInvalidValue;
    int64_t blocks = (n / 8 + 255) / 256;
    if (blocks > 2048) blocks = 2048;
    hipLaunchKernelGGL(k_bf16_to_f16, dim3((unsigned)blocks), dim3(256), 0, s, (const bf16_t*)src, (_Float16*)dst,
                       n / 8, err);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float* part, int splits, int64_t MN, float* out, hipStream_t s) {
    if (MN == 0) return hipSuccess;
    int64_t blocks = (MN / 4 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)blocks), dim3(256), 0, s, part, splits, MN, out);
    return hipGetLastError();
}

}  // namespace rdcn
