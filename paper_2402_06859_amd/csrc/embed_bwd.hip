// QR embedding backward for gfx950: table gradients from the x0 gradient.
//
// Every valid id occurrence of bag (b, f) with (qi, ri) = (id / m, id mod m)
// (section "Model Dictionary Compression") adds g = dLoss/dx0[b, f*D:(f+1)*D]
// (sum combine) or g * R_f[ri] / g * Q_f[qi] (product combine) to row qi of
// Q_f and row ri of R_f; sum pooling gives each id of a bag the bag's gradient.
//
// Under Zipf-distributed ids a few rows receive a large share of all
// occurrences, so the sum is not formed with atomics. Instead:
//   1. keys: each occurrence gets two keys, its row in the concatenation of
//      all quotient tables followed by all remainder tables; the value is the
//      occurrence index (ids outside [0, V) get a sentinel key that sorts last).
//      With the hashed front-end each feature has two table pairs (one per
//      32-bit half of the id's hash) and an occurrence gets four keys; the value
//      is then occurrence + half * nnz;
//   2. a stable LSD radix sort of (key, occurrence) pairs groups equal rows
//      while keeping occurrence order inside each group;
//   3. a segmented reduction walks the sorted pairs in fixed tiles, one wave
//      per tile, lanes along D, adding contributions in sorted order;
//      a segment that starts and ends inside its tile is written directly
//      (+=), the pieces of a segment that crosses tile boundaries are kept per
//      tile and summed in tile order by a fix-up pass.
// The result is deterministic: each row's contributions are added in
// (b, position-in-bag) order, irrespective of scheduling.
// Unhashed ids with tables of at most 16384 rows take the one-kernel path of
// step 4 instead (no scratch, no global sort).
#include <mutex>

#include "device_common.h"
#include "embed_bwd.h"

namespace rdcn {

namespace {

constexpr int RS_THREADS = 256;
constexpr int RS_ITEMS = 4;
constexpr int RS_TILE = RS_THREADS * RS_ITEMS;  // 1024 pairs per radix tile
constexpr int SEG_TILE = 128;                    // sorted pairs per reduction wave

template <typename ID>
__device__ __forceinline__ bool split_id(ID raw, const EmbedBwdArgs& a, uint32_t& qi, uint32_t& ri) {
    const int64_t id = (int64_t)raw;
    if (id < 0 || (uint64_t)id >= a.vocab) return false;
    if (a.vocab <= 0x100000000ull) {
        qi = div_magic((uint32_t)id, DivMagic{a.magic_m, a.shift_m, a.m});
        ri = (uint32_t)id - qi * a.m;
    } else {
        const uint64_t q = (uint64_t)id / a.m;
        qi = (uint32_t)q;
        ri = (uint32_t)((uint64_t)id - q * a.m);
    }
    return qi < (uint32_t)a.rows_q && ri < a.m;
}

// 1. keys. Single-hot: thread per occurrence o = b*F + f. Bags: thread per bag.
// With the product combine each occurrence also records its quotient and
// remainder rows (the reduction multiplies by the row of the other table).
template <typename ID, bool BAGS, bool MUL, bool HASHED>
__global__ __launch_bounds__(256) void k_emb_keys(EmbedBwdArgs a, uint32_t* __restrict__ keys,
                                                  uint32_t* __restrict__ vals, uint32_t* __restrict__ bag_of,
                                                  uint32_t* __restrict__ qrow, uint32_t* __restrict__ rrow) {
    const ID* ids = (const ID*)a.ids;
    const uint32_t pairs = HASHED ? 2u : 1u;  // table pairs per feature
    const uint32_t sentinel = (uint32_t)a.F * pairs * (a.rows_q + a.m);
    const uint32_t rbase = (uint32_t)a.F * pairs * a.rows_q;
    const int64_t nunits = BAGS ? a.batch * a.F : a.nnz;
    for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nunits;
         u += (int64_t)gridDim.x * blockDim.x) {
        const int f = (int)(u % a.F);
        const int64_t begin = BAGS ? a.offsets[u] : u;
        const int64_t end = BAGS ? a.offsets[u + 1] : u + 1;
        for (int64_t p = begin; p < end && p < a.nnz; ++p) {
            if (HASHED) {  // keys [q of half 0 | r of half 0 | q of half 1 | r of half 1], value p + s * nnz
                const uint64_t h = murmur64a_8((uint64_t)(int64_t)ids[p], a.seed);
                const DivMagic dm{a.magic_m, a.shift_m, a.m};
#pragma unroll
                for (int s = 0; s < 2; ++s) {
                    const uint32_t x = (uint32_t)(s ? h >> 32 : h);
                    const uint32_t qi = div_magic(x, dm), ri = x - qi * a.m;
                    const uint32_t tbl = 2u * (uint32_t)f + (uint32_t)s;
                    const int64_t o = p + s * a.nnz;
                    keys[2 * s * a.nnz + p] = tbl * a.rows_q + qi;
                    keys[(2 * s + 1) * a.nnz + p] = rbase + tbl * a.m + ri;
                    vals[2 * s * a.nnz + p] = (uint32_t)o;
                    vals[(2 * s + 1) * a.nnz + p] = (uint32_t)o;
                    if (MUL) {
                        qrow[o] = qi;
                        rrow[o] = ri;
                    }
                }
                if (BAGS) bag_of[p] = (uint32_t)u;
                continue;
            }
            uint32_t qi = 0, ri = 0, kq = sentinel, kr = sentinel;
            if (split_id<ID>(ids[p], a, qi, ri)) {
                kq = (uint32_t)f * a.rows_q + qi;
                kr = rbase + (uint32_t)f * a.m + ri;
            } else {
                qi = ri = 0;
            }
            keys[p] = kq;
            keys[a.nnz + p] = kr;
            vals[p] = (uint32_t)p;
            vals[a.nnz + p] = (uint32_t)p;
            if (BAGS) bag_of[p] = (uint32_t)u;
            if (MUL) {
                qrow[p] = qi;
                rrow[p] = ri;
            }
        }
    }
}

// 2a. per-tile digit histogram, stored digit-major: hist[digit * ntiles + tile]
constexpr int RS_MAX_BITS = 10;  // digits of up to 10 bits (1024 buckets)
constexpr int RS_BUCKETS = 1 << RS_MAX_BITS;

__global__ __launch_bounds__(RS_THREADS) void k_rs_hist(const uint32_t* __restrict__ keys, uint32_t n, int shift,
                                                        uint32_t mask, uint32_t* __restrict__ hist, int ntiles) {
    __shared__ uint32_t h[RS_BUCKETS];
    for (int d = threadIdx.x; d < RS_BUCKETS; d += RS_THREADS) h[d] = 0;
    __syncthreads();
    const uint32_t base = blockIdx.x * RS_TILE;
#pragma unroll
    for (int i = 0; i < RS_ITEMS; ++i) {
        const uint32_t e = base + i * RS_THREADS + threadIdx.x;
        if (e < n) atomicAdd(&h[(keys[e] >> shift) & mask], 1u);
    }
    __syncthreads();
    for (uint32_t d = threadIdx.x; d <= mask; d += RS_THREADS) hist[(int64_t)d * ntiles + blockIdx.x] = h[d];
}

// Exclusive scan of one value per thread over a 256-thread workgroup.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* sh, uint32_t& total) {
    // 256 threads: wave inclusive scan, then wave totals.
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    if (lane == 63) sh[wave] = x;
    __syncthreads();
    uint32_t wofs = 0;
    for (int w = 0; w < wave; ++w) wofs += sh[w];
    total = sh[0] + sh[1] + sh[2] + sh[3];
    __syncthreads();
    return wofs + x - v;
}

// Exclusive scan of one value per thread over a workgroup of NW waves.
template <int NW>
__device__ __forceinline__ uint32_t block_exclusive_scan_nw(uint32_t v, uint32_t* sh, uint32_t& total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    if (lane == 63) sh[wave] = x;
    __syncthreads();
    uint32_t wofs = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        if (w < wave) wofs += sh[w];
        tot += sh[w];
    }
    total = tot;
    __syncthreads();
    return wofs + x - v;
}

// Per digit d (one workgroup per digit): exclusive prefix over the tiles of
// hist[d][*] in place, 256 tiles per round; digit total into tot[d].
__global__ __launch_bounds__(256) void k_digit_scan(uint32_t* __restrict__ hist, int ntiles,
                                                    uint32_t* __restrict__ tot) {
    __shared__ uint32_t sh[4];
    uint32_t* row = hist + (int64_t)blockIdx.x * ntiles;
    uint32_t run = 0;
    for (int t0 = 0; t0 < ntiles; t0 += 256) {
        const int t = t0 + threadIdx.x;
        const uint32_t v = t < ntiles ? row[t] : 0u;
        uint32_t total;
        const uint32_t ex = block_exclusive_scan(v, sh, total);
        if (t < ntiles) row[t] = run + ex;
        run += total;
    }
    if (threadIdx.x == 0) tot[blockIdx.x] = run;
}

// 2b. stable scatter: items of a tile are ranked in element order (slot-major,
// then thread) with wave ballots; digit bases come from the scanned histogram.
__global__ __launch_bounds__(RS_THREADS) void k_rs_scatter(const uint32_t* __restrict__ kin,
                                                           const uint32_t* __restrict__ vin, uint32_t* __restrict__ kout,
                                                           uint32_t* __restrict__ vout, uint32_t n, int shift, int bits,
                                                           const uint32_t* __restrict__ offs, int ntiles,
                                                           const uint32_t* __restrict__ tot) {
    __shared__ uint32_t base[RS_BUCKETS];
    __shared__ uint32_t wcnt[4][RS_BUCKETS];
    __shared__ uint32_t sh[4];
    const uint32_t mask = (1u << bits) - 1u;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // digit bases: exclusive scan of the digit totals (4 consecutive digits per thread)
    {
        uint32_t v[4], s4 = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t d = threadIdx.x * 4 + e;
            v[e] = d <= mask ? tot[d] : 0u;
            s4 += v[e];
        }
        uint32_t total;
        uint32_t run = block_exclusive_scan(s4, sh, total);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t d = threadIdx.x * 4 + e;
            if (d <= mask) {
                base[d] = run + offs[(int64_t)d * ntiles + blockIdx.x];
                wcnt[0][d] = wcnt[1][d] = wcnt[2][d] = wcnt[3][d] = 0;
            }
            run += v[e];
        }
    }
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int it = 0; it < RS_ITEMS; ++it) {
        const uint32_t e = blockIdx.x * RS_TILE + it * RS_THREADS + threadIdx.x;
        const bool valid = e < n;
        const uint32_t key = valid ? kin[e] : 0u;
        const uint32_t val = valid ? vin[e] : 0u;
        const uint32_t dg = (key >> shift) & mask;
        uint64_t peers = __ballot(valid);
        for (int bb = 0; bb < bits; ++bb) {
            const uint64_t m = __ballot(valid && ((dg >> bb) & 1u));
            peers &= ((dg >> bb) & 1u) ? m : ~m;
        }
        const uint32_t rank = (uint32_t)__popcll(peers & lt);
        if (valid && rank == 0) wcnt[wave][dg] = (uint32_t)__popcll(peers);
        __syncthreads();
        uint32_t pos = 0;
        if (valid) {
            pos = base[dg] + rank;
            for (int w = 0; w < wave; ++w) pos += wcnt[w][dg];
        }
        __syncthreads();
        for (uint32_t d = threadIdx.x; d <= mask; d += RS_THREADS) {
            base[d] += wcnt[0][d] + wcnt[1][d] + wcnt[2][d] + wcnt[3][d];
            wcnt[0][d] = wcnt[1][d] = wcnt[2][d] = wcnt[3][d] = 0;
        }
        if (valid) {
            kout[pos] = key;
            vout[pos] = val;
        }
        __syncthreads();
    }
}

// 3. segmented reduction. A wave takes SEG_TILE consecutive sorted pairs. L lanes
// (a power of two, 4 L >= D) hold one pair's gradient slice, four columns per lane,
// so one wave step covers E = 64 / L pairs; all slices of up to 16 steps are loaded
// before any is summed. Sums run in a fixed order: inside a step a segmented
// inclusive scan over the E pairs (Hillis-Steele, lane shuffles), across steps a
// running carry in front of the step's partial sum.
struct Cols4 {
    float v[4];
};

template <typename T>
struct SegCtx {
    EmbedBwdArgs a;
    const uint32_t* keys;
    const uint32_t* vals;
    const uint32_t* bag_of;  // bags
    const uint32_t* qrow;    // product combine
    const uint32_t* rrow;
    uint32_t n;
    uint32_t sentinel, rbase;

    // loads for the contribution of sorted pair (k, o) to the row of key k, columns
    // c .. c+3: the gradient slice into g and, with the product combine, the other
    // table's row into r (the contribution is g * r). Every load is issued
    // unconditionally (ok = false reads row 0 / occurrence 0; the caller masks the
    // result when it uses it), and nothing writes the loaded registers before that
    // use, so the loads of many pairs are in flight together.
    template <bool MUL, bool BAGS>
    __device__ __forceinline__ void contrib(uint32_t k, uint32_t o, int c, bool ok, Cols4& g, Cols4& r) const {
        const uint32_t kk0 = ok ? k : 0u;
        const bool isq = kk0 < rbase;
        const uint32_t kk = isq ? kk0 : kk0 - rbase;
        // table pair of the key (the feature, or 2 * feature + hash half)
        const uint32_t tbl = isq ? div_magic(kk, DivMagic{a.magic_q, a.shift_q, (uint32_t)a.rows_q})
                                 : div_magic(kk, DivMagic{a.magic_m, a.shift_m, a.m});
        const uint32_t f = a.hashed ? tbl >> 1 : tbl;
        const uint32_t oo = ok ? o : 0u;
        const uint32_t occ = oo >= (uint32_t)a.nnz ? oo - (uint32_t)a.nnz : oo;  // value = occurrence + half * nnz
        const int cc = ok ? c : 0;
        const uint32_t bag = BAGS ? bag_of[occ] : occ;
        const int64_t b = div_magic(bag, DivMagic{a.magic_f, a.shift_f, (uint32_t)a.F});
        const f32x4_t w = *(const f32x4_t*)(a.grad_x0 + b * a.d + (int64_t)f * a.D + cc);
        g = Cols4{{w.x, w.y, w.z, w.w}};
        if (MUL) {
            const T* other = isq ? (const T*)a.r_tables + ((int64_t)tbl * a.m + rrow[oo]) * a.D + cc
                                 : (const T*)a.q_tables + ((int64_t)tbl * a.rows_q + qrow[oo]) * a.D + cc;
#pragma unroll
            for (int e = 0; e < 4; ++e) r.v[e] = st<T>::load(other + e);
        }
    }

    __device__ __forceinline__ float* row_of(uint32_t k) const {
        return k < rbase ? a.grad_q + (int64_t)k * a.D : a.grad_r + (int64_t)(k - rbase) * a.D;
    }
};

// 16-byte column groups (D and d are multiples of 4, the float buffers 16-byte aligned)
__device__ __forceinline__ Cols4 load4(const float* p) {
    const f32x4_t w = *(const f32x4_t*)p;
    return Cols4{{w.x, w.y, w.z, w.w}};
}

__device__ __forceinline__ void store4(float* p, const Cols4& x) {
    *(f32x4_t*)p = f32x4_t{x.v[0], x.v[1], x.v[2], x.v[3]};
}

constexpr uint32_t SEG_PAD = 0xffffffffu;  // key of the slots past the last sorted pair

// Where a finished piece goes: 0 nowhere (padding, ids out of range, or lanes past
// D), 1 the table row (+=), 2 this tile's head carry, 3 its tail carry.
enum { DST_NONE = 0, DST_ROW = 1, DST_HEAD = 2, DST_TAIL = 3 };

template <typename T, int L, bool MUL, bool BAGS>
__global__ __launch_bounds__(256) void k_seg_reduce(SegCtx<T> s, float* __restrict__ carry_head,
                                                    float* __restrict__ carry_tail) {
    constexpr int E = 64 / L;
    constexpr int STEPS = SEG_TILE / E;
    constexpr int U = STEPS < 16 ? STEPS : 16;
    const int lane = threadIdx.x & 63, grp = lane / L, sub = lane % L, c = 4 * sub;
    const uint32_t tile = blockIdx.x * 4 + (threadIdx.x >> 6);
    const uint32_t p0 = tile * SEG_TILE;
    if (p0 >= s.n) return;
    const uint32_t cnt = s.n - p0 < (uint32_t)SEG_TILE ? s.n - p0 : (uint32_t)SEG_TILE;
    const int D = s.a.D;
    const bool colok = c < D;
    const uint32_t first_key = s.keys[p0], last_key = s.keys[p0 + cnt - 1];
    // the first segment started in an earlier tile / the last one goes on in a later tile
    const bool head_cont = p0 > 0 && s.keys[p0 - 1] == first_key;
    const bool tail_cont = p0 + cnt < s.n && s.keys[p0 + cnt] == last_key;
    Cols4 carry = {{0.f, 0.f, 0.f, 0.f}};
    uint32_t carry_key = SEG_PAD;
    for (int s0 = 0; s0 < STEPS; s0 += U) {
        uint32_t key[U], val[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t e = (uint32_t)((s0 + u) * E + grp);
            const uint32_t ec = e < cnt ? e : cnt - 1;
            key[u] = s.keys[p0 + ec];
            val[u] = s.vals[p0 + ec];
            if (e >= cnt) key[u] = SEG_PAD;
        }
        const uint32_t en = (uint32_t)((s0 + U) * E);
        const uint32_t key_after = en < cnt ? s.keys[p0 + en] : SEG_PAD;
        // which pairs end a piece (the next pair has another key, or the tile ends)
        // and where that piece goes; the old table rows of direct writes are loaded
        // together with the gradient slices
        int dst[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t e = (uint32_t)((s0 + u) * E + grp);
            uint32_t knext = __shfl_down(key[u], L);
            const uint32_t k0 = u + 1 < U ? __shfl(key[u + 1 < U ? u + 1 : u], sub) : key_after;
            if (grp == E - 1) knext = k0;
            const uint32_t k = key[u];
            int d = DST_NONE;
            if (k != SEG_PAD && k != s.sentinel && colok && (knext != k || e + 1 == cnt)) {
                if (head_cont && k == first_key) d = DST_HEAD;
                else if (tail_cont && k == last_key) d = DST_TAIL;
                else d = DST_ROW;
            }
            dst[u] = d;
        }
        Cols4 x[U], o4[U], old[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool ok = key[u] != SEG_PAD && key[u] != s.sentinel && colok;
            s.template contrib<MUL, BAGS>(key[u], val[u], c, ok, x[u], o4[u]);
            old[u] = load4(s.row_of(dst[u] == DST_ROW ? key[u] : 0u) + (colok ? c : 0));
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t k = key[u];
            const uint32_t kprev = __shfl_up(k, L);
            bool head = grp == 0 ? k != carry_key : k != kprev;
            const bool ok = k != SEG_PAD && k != s.sentinel && colok;
            Cols4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v.v[e] = ok ? (MUL ? x[u].v[e] * o4[u].v[e] : x[u].v[e]) : 0.f;
#pragma unroll
            for (int off = 1; off < E; off <<= 1) {
                Cols4 y;
#pragma unroll
                for (int e = 0; e < 4; ++e) y.v[e] = __shfl_up(v.v[e], off * L);
                const bool hy = __shfl_up((int)head, off * L) != 0;
                if (grp >= off && !head) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) v.v[e] = y.v[e] + v.v[e];
                }
                if (grp >= off) head = head || hy;
            }
            if (!head) {  // the segment reaches back into the carried one
#pragma unroll
                for (int e = 0; e < 4; ++e) v.v[e] = carry.v[e] + v.v[e];
            }
            if (dst[u] == DST_ROW) {
#pragma unroll
                for (int e = 0; e < 4; ++e) old[u].v[e] += v.v[e];
                store4(s.row_of(k) + c, old[u]);
            } else if (dst[u] == DST_HEAD) {
                store4(carry_head + (int64_t)tile * D + c, v);
            } else if (dst[u] == DST_TAIL) {
                store4(carry_tail + (int64_t)tile * D + c, v);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) carry.v[e] = __shfl(v.v[e], (E - 1) * L + sub);
            carry_key = __shfl(k, (E - 1) * L + sub);
        }
    }
}

// Fix-up: the tile whose last segment starts inside it and continues owns the
// segment. Its wave finds the following tiles that open with the same key 64 at a
// time (one ballot over their first keys), loads their head pieces E tiles per
// step (lanes as in the reduction), and adds them in a fixed order: each lane
// group sums its tiles in tile order, then the groups are added pairwise, and the
// owner's tail piece goes in front.
template <int L>
__global__ __launch_bounds__(256) void k_seg_fixup(const uint32_t* __restrict__ keys, uint32_t n, uint32_t sentinel,
                                                   uint32_t rbase, int D, float* __restrict__ grad_q,
                                                   float* __restrict__ grad_r, const float* __restrict__ carry_head,
                                                   const float* __restrict__ carry_tail) {
    constexpr int E = 64 / L;
    const int lane = threadIdx.x & 63, grp = lane / L, sub = lane % L, c = 4 * sub;
    const uint32_t tile = blockIdx.x * 4 + (threadIdx.x >> 6);
    const uint32_t p0 = tile * SEG_TILE;
    if (p0 >= n) return;
    const uint32_t p1 = p0 + SEG_TILE;
    if (p1 >= n) return;
    const uint32_t k = keys[p1 - 1];
    if (k == sentinel || keys[p1] != k) return;
    // the last piece started before this tile when the whole tile is that segment and it came from before
    if (p0 > 0 && keys[p0] == k && keys[p0 - 1] == k) return;
    const uint32_t ntiles = (n + SEG_TILE - 1) / SEG_TILE;
    Cols4 acc = {{0.f, 0.f, 0.f, 0.f}};
    for (uint32_t base = tile + 1;; base += 64) {
        const uint32_t t = base + lane;
        const bool cont = t < ntiles && keys[t * SEG_TILE] == k;
        const uint64_t mask = __ballot(cont);
        const int run = mask == ~0ull ? 64 : __builtin_ctzll(~mask);  // tiles base .. base+run-1 continue it
        for (int st = 0; st < run; st += E) {
            if (st + grp < run && c < D) {
                const Cols4 x = load4(carry_head + (int64_t)(base + st + grp) * D + c);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc.v[e] += x.v[e];
            }
        }
        if (run < 64) break;
    }
#pragma unroll
    for (int off = 1; off < E; off <<= 1) {  // group g adds group g + off (pairwise tree)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float y = __shfl_down(acc.v[e], off * L);
            if ((grp & (2 * off - 1)) == 0) acc.v[e] += y;
        }
    }
    if (grp == 0 && c < D) {
        Cols4 tot = load4(carry_tail + (int64_t)tile * D + c);
#pragma unroll
        for (int e = 0; e < 4; ++e) tot.v[e] += acc.v[e];
        float* dst = (k < rbase ? grad_q + (int64_t)k * D : grad_r + (int64_t)(k - rbase) * D) + c;
        Cols4 old = load4(dst);
#pragma unroll
        for (int e = 0; e < 4; ++e) old.v[e] += tot.v[e];
        store4(dst, old);
    }
}

// 4. Fused path (unhashed ids, tables of at most FU_ROWS * FU_MAX_SLICES rows):
// one workgroup per (feature, table, row slice) replaces steps 1-3. It walks the
// feature's occurrences in (bag, position) order, CAP at a time, keeps those whose
// row falls in its slice and sorts them by row in LDS (a counting sort over at most
// FU_ROWS rows: each wave ranks its share of the chunk with ballots, a scan over
// the rows gives every (row, wave) run its start). The sorted chunk is split into
// equal parts, one per lane group (L lanes of four columns each, 64 / L groups per
// wave); a group adds its part's contributions one after another, and a segment
// that crosses parts is finished by the group in which it starts, from per-part
// head and tail pieces in LDS, after a barrier. The rows of a slice belong to one workgroup, so
// each chunk's row sums are added straight into the table gradient (+=), chunk after
// chunk. Summation order is fixed by the data: deterministic.
// The workgroups of one feature are given block indices with equal residue mod 8 so
// that they run on one XCD and share its L2 copy of the feature's gradient slab.
constexpr int FU_CAP = 4096;            // occurrences per chunk
constexpr int FU_WAVES = 8;             // waves per workgroup
constexpr int FU_THREADS = 64 * FU_WAVES;
constexpr int FU_ROWS = 4096;           // rows per slice (at most)
constexpr int FU_ROWS_MID = 2048;       // the form with chunks of 2 * FU_CAP occurrences (10240 with bags)
constexpr int FU_ROWS_SMALL = 1024;     // the kernel form for slices of at most this many rows: its
                                        // smaller LDS lets two single-hot workgroups share a CU
constexpr int FU_MAX_SLICES = 16;
constexpr int FU_MAX_TABLE_ROWS = 16384;  // larger tables take the sort path
constexpr int FU_ONE_ROUND = 256;       // workgroups resident at once (one per CU)
constexpr int FU_SPLIT_ROWS = 1024;     // slice rows when the workgroups need several rounds
constexpr int FU_BAGS = 1024;           // bags per block (bag front-end)
constexpr int FU_BPT = FU_BAGS / FU_THREADS;  // bags per thread
constexpr uint32_t FU_SKIP = 0xffffffffu;

struct FusedArgs {
    EmbedBwdArgs a;
    int ids64;
    int slices;                // row slices per table
    uint32_t rps_q, rps_r;     // rows per slice of the quotient / remainder tables
};

// CPL: table columns per lane (4, or 8 when D is a multiple of 8 in the 4096-row
// form: half the lanes per element, so each wave instruction of the ordered sums
// serves twice the elements).
template <typename T, int L, bool MUL, bool BAGS, int ROWS, int CPL, int CAP>
__global__ __launch_bounds__(FU_THREADS) void k_emb_fused(FusedArgs fa) {
    static_assert(CAP == 4096 || CAP == 8192 || CAP == 10240, "chunk of 4096, 8192 or 10240 occurrences");
    // bags with the sum combine: the sums need only each element's bag, so `sorted` carries
    // the bag (below FU_BAGS) instead of the element and no per-element bag array is kept
    constexpr bool BAGDIRECT = BAGS && !MUL;
    static_assert(!BAGDIRECT || FU_BAGS <= 1024, "a bag index takes 10 bits");
    static_assert(BAGDIRECT || CAP != 10240, "10240-occurrence chunks only in the bag-index form");
    constexpr int QW = CAP / FU_WAVES;       // chunk elements per wave
    constexpr int EB = BAGDIRECT ? 10 : CAP == 8192 ? 13 : 12;  // bits of the element (bag) index in `sorted`
    constexpr uint32_t EMASK = (1u << EB) - 1u;
    static_assert(CPL == 4 || CPL == 8, "four or eight columns per lane");
    constexpr int NC = CPL / 4;              // 16-byte column groups per lane
    constexpr int FU_RPT = ROWS / FU_THREADS;  // slice rows per thread in the run-start scan
    constexpr int E = 64 / L;                // lane groups per wave
    constexpr int NP = FU_WAVES * E;         // parts of a sorted chunk, one per lane group
    // elements of a part whose loads are in flight together: twice as many in the bag
    // forms with the sum combine, which run one workgroup per CU and have the registers
    constexpr int U = (BAGS && !MUL && ROWS != FU_ROWS_SMALL ? 16 : 8) / NC;
    __shared__ uint32_t key_e[CAP];       // per chunk element: row << 16 | rank in its wave's run, or FU_SKIP
    __shared__ uint32_t sorted[CAP];      // row << EB | element (bag), in (row, element) order
    __shared__ uint16_t whist[FU_WAVES][ROWS];  // per wave row counts, then run starts (< CAP)
    __shared__ float carry[2][NP][CPL * L];  // per part head / tail pieces
    __shared__ uint16_t bag_e[BAGS && !BAGDIRECT ? CAP : 1];
    __shared__ uint32_t carry_sh;         // 1 + the bag of a chunk's last element (bag-index form)
    __shared__ uint16_t other_e[MUL ? CAP : 1];
    __shared__ uint32_t bstart[BAGS ? FU_BAGS : 1];
    __shared__ int64_t boff[BAGS ? FU_BAGS : 1];
    __shared__ uint32_t sh[FU_WAVES];
    __shared__ uint32_t nkept;

    const EmbedBwdArgs& a = fa.a;
    const int per_f = 2 * fa.slices;
    const int j = (int)(blockIdx.x >> 3);
    const int f = (j / per_f) * 8 + (int)(blockIdx.x & 7);
    if (f >= a.F) return;
    const int sub = j % per_f;
    const bool isq = sub < fa.slices;
    const uint32_t rps = isq ? fa.rps_q : fa.rps_r;
    const uint32_t r0 = (uint32_t)(isq ? sub : sub - fa.slices) * rps;
    const uint32_t rows = isq ? (uint32_t)a.rows_q : a.m;
    if (r0 >= rows) return;
    const uint32_t nr = rows - r0 < rps ? rows - r0 : rps;
    const int nbits = nr > 1 ? 32 - __clz((int)(nr - 1)) : 0;
    const int D = a.D;
    float* gtab = isq ? a.grad_q + ((int64_t)f * a.rows_q + r0) * D : a.grad_r + ((int64_t)f * a.m + r0) * D;
    const T* otab = isq ? (const T*)a.r_tables + (int64_t)f * a.m * D : (const T*)a.q_tables + (int64_t)f * a.rows_q * D;
    const float* gx = a.grad_x0 + (int64_t)f * D;

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int grp = lane / L, sub4 = lane % L, c = CPL * sub4;
    const bool colok = c < D;  // D is a multiple of CPL: a lane's columns are all in range or none
    const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    for (int i = threadIdx.x; i < FU_WAVES * ROWS; i += FU_THREADS) (&whist[0][0])[i] = 0;

    const int64_t step_b = BAGS ? FU_BAGS : CAP;
    for (int64_t b0 = 0; b0 < a.batch;) {
        const uint32_t nb = (uint32_t)(a.batch - b0 < step_b ? a.batch - b0 : step_b);
        uint32_t total = nb;  // occurrences of this block of bags
        uint32_t take = nb;   // bags (samples) taken in this pass
        uint32_t bbeg[FU_BPT], blen[FU_BPT];  // this thread's bags: first occurrence in the pass, length
        if (BAGS) {
            uint32_t len[FU_BPT], s4 = 0;
            int64_t beg[FU_BPT];
#pragma unroll
            for (int k = 0; k < FU_BPT; ++k) {
                const uint32_t t = FU_BPT * threadIdx.x + k;
                len[k] = 0;
                beg[k] = 0;
                if (t < nb) {
                    const int64_t u = (b0 + t) * a.F + f;
                    int64_t s = a.offsets[u], e = a.offsets[u + 1];
                    s = s < 0 ? 0 : (s > a.nnz ? a.nnz : s);
                    e = e < s ? s : (e > a.nnz ? a.nnz : e);
                    beg[k] = s;
                    len[k] = (uint32_t)(e - s);
                }
                s4 += len[k];
            }
            uint32_t run = block_exclusive_scan_nw<FU_WAVES>(s4, sh, total);
            // unless these are the last bags, take only the leading bags that fill whole
            // chunks and leave the rest to the next pass: a partial chunk costs the
            // ranking and placement of a full one (at least one bag is taken)
            if (b0 + nb < a.batch && total > (uint32_t)CAP) {
                const uint32_t limit = total / CAP * CAP;
                uint32_t cnt = 0, end = run;
#pragma unroll
                for (int k = 0; k < FU_BPT; ++k) {
                    end += len[k];
                    cnt += FU_BPT * threadIdx.x + k < nb && end <= limit ? 1u : 0u;
                }
                uint32_t nfit;
                block_exclusive_scan_nw<FU_WAVES>(cnt, sh, nfit);
                take = nfit > 0 ? nfit : 1u;
            }
#pragma unroll
            for (int k = 0; k < FU_BPT; ++k) {
                bstart[FU_BPT * threadIdx.x + k] = run;
                boff[FU_BPT * threadIdx.x + k] = beg[k];
                bbeg[k] = run;
                blen[k] = FU_BPT * threadIdx.x + k < take ? len[k] : 0u;
                run += len[k];
            }
        }
        __syncthreads();
        if (BAGS && take < nb) total = bstart[take];  // the taken bags' occurrences
        uint32_t carry_bag = 0;  // 1 + the bag of the previous chunk's last element
        for (uint32_t c0 = 0; c0 < total; c0 += CAP) {
            const uint32_t n = total - c0 < (uint32_t)CAP ? total - c0 : (uint32_t)CAP;
            // A. rows of this wave's share (all id loads first, then the ranking); the
            // rank of each kept element among the wave's earlier elements of its row
            constexpr int NIT = QW / 64;
            int64_t pv[NIT];
            uint32_t bagv[NIT];
            if (BAGS) {
                // the bag of each element: every non-empty taken bag that starts in the chunk
                // marks its first element with bag + 1 (in key_e, unused until the ranking);
                // bag indices rise with the element, so an element's bag is the last mark at
                // or before it, or before the chunk's first mark the previous chunk's last bag
#pragma unroll
                for (int it = 0; it < NIT; ++it) key_e[wv * QW + it * 64 + lane] = 0u;
                __syncthreads();
#pragma unroll
                for (int k = 0; k < FU_BPT; ++k)
                    if (blen[k] > 0 && bbeg[k] >= c0 && bbeg[k] - c0 < n)
                        key_e[bbeg[k] - c0] = FU_BPT * threadIdx.x + k + 1;
                __syncthreads();
                uint32_t mk[NIT], lmax = 0;
#pragma unroll
                for (int it = 0; it < NIT; ++it) {
                    mk[it] = key_e[wv * QW + it * 64 + lane];
                    lmax = mk[it] > lmax ? mk[it] : lmax;
                }
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const uint32_t y = __shfl_xor(lmax, off);
                    lmax = y > lmax ? y : lmax;
                }
                if (lane == 0) sh[wv] = lmax;
                // the chunk's first element's bag (elements past the chunk end stand in for
                // it, so their loads stay in bounds); read before the ranking reuses key_e
                const uint32_t first_bag = (key_e[0] != 0u ? key_e[0] : carry_bag) - 1u;
                __syncthreads();
                uint32_t cur = carry_bag;  // last mark before this wave's elements
                for (int w = 0; w < wv; ++w) cur = sh[w] > cur ? sh[w] : cur;
#pragma unroll
                for (int it = 0; it < NIT; ++it) {
                    // the last marked lane at or below this one, else the carry
                    const uint64_t upto = __ballot(mk[it] != 0u) & ((2ull << lane) - 1ull);
                    const uint32_t got = __shfl(mk[it], upto ? 63 - __clzll(upto) : 0);
                    const uint32_t bg = upto ? got : cur;
                    if constexpr (BAGDIRECT) {
                        bagv[it] = bg - 1u;
                        if ((uint32_t)(wv * QW + it * 64 + lane) == n - 1) carry_sh = bg;
                    } else {
                        bag_e[wv * QW + it * 64 + lane] = (uint16_t)(bg - 1u);
                    }
                    cur = __builtin_amdgcn_readlane(bg, 63);
                }
                __syncthreads();
                carry_bag = BAGDIRECT ? carry_sh : (uint32_t)bag_e[n - 1] + 1u;
                uint32_t vv[NIT];
#pragma unroll
                for (int it = 0; it < NIT; ++it) {
                    const uint32_t e = (uint32_t)(wv * QW + it * 64 + lane);
                    const uint32_t ee = e < n ? e : 0u;
                    vv[it] = c0 + ee;
                    if constexpr (BAGDIRECT) bagv[it] = e < n ? bagv[it] : first_bag;
                    else bagv[it] = bag_e[ee];
                }
#pragma unroll
                for (int it = 0; it < NIT; ++it) pv[it] = boff[bagv[it]] + (int64_t)(vv[it] - bstart[bagv[it]]);
            } else {
#pragma unroll
                for (int it = 0; it < NIT; ++it) {
                    const uint32_t e = (uint32_t)(wv * QW + it * 64 + lane);
                    pv[it] = (b0 + (e < n ? e : 0u)) * a.F + f;
                    bagv[it] = 0;
                }
            }
            // every load is issued (element 0 stands in past the chunk end), so all are in flight together
            int64_t idv[NIT];
            if (fa.ids64) {
#pragma unroll
                for (int it = 0; it < NIT; ++it) idv[it] = ((const int64_t*)a.ids)[pv[it]];
            } else {
#pragma unroll
                for (int it = 0; it < NIT; ++it) idv[it] = (int64_t)((const int32_t*)a.ids)[pv[it]];
            }
            const DivMagic dm{a.magic_m, a.shift_m, a.m};
#pragma unroll
            for (int it = 0; it < NIT; ++it) {
                const uint32_t e = (uint32_t)(wv * QW + it * 64 + lane);
                // ids below vocab <= rows_q * m <= 2^28 here: the 32-bit split is exact
                const int64_t id = idv[it];
                const uint32_t x = (uint32_t)id;
                const uint32_t qi = div_magic(x, dm), ri = x - qi * a.m;
                const uint32_t r = (isq ? qi : ri) - r0;
                const bool kept = e < n && id >= 0 && (uint64_t)id < a.vocab && qi < (uint32_t)a.rows_q && r < nr;
                const uint32_t row = kept ? r : 0u;
                uint64_t peers = __ballot(kept);
                for (int bb = 0; bb < nbits; ++bb) {
                    const bool bit = (row >> bb) & 1u;
                    const uint64_t m = __ballot(bit);
                    peers &= bit ? m : ~m;
                }
                const uint32_t before = whist[wv][row];
                const uint32_t rank = (uint32_t)__popcll(peers & lt);
                key_e[e] = kept ? (row << 16) | (before + rank) : FU_SKIP;
                if (MUL) other_e[e] = (uint16_t)(isq ? ri : qi);
                if (kept && rank == 0) whist[wv][row] = (uint16_t)(before + (uint32_t)__popcll(peers));
            }
            __syncthreads();
            // B. run starts: rows in order, inside a row the waves in order
            {
                uint32_t cnt[FU_RPT][FU_WAVES], s4 = 0;
#pragma unroll
                for (int k = 0; k < FU_RPT; ++k) {
                    const uint32_t r = FU_RPT * threadIdx.x + k;
#pragma unroll
                    for (int w = 0; w < FU_WAVES; ++w) {
                        cnt[k][w] = r < nr ? whist[w][r] : 0u;
                        s4 += cnt[k][w];
                    }
                }
                uint32_t tot;
                uint32_t run = block_exclusive_scan_nw<FU_WAVES>(s4, sh, tot);
#pragma unroll
                for (int k = 0; k < FU_RPT; ++k) {
                    const uint32_t r = FU_RPT * threadIdx.x + k;
#pragma unroll
                    for (int w = 0; w < FU_WAVES; ++w) {
                        if (r < nr) whist[w][r] = (uint16_t)run;
                        run += cnt[k][w];
                    }
                }
                if (threadIdx.x == 0) nkept = tot;
            }
            __syncthreads();
            // C. placement
#pragma unroll
            for (int it = 0; it < NIT; ++it) {
                const uint32_t e = (uint32_t)(wv * QW + it * 64 + lane);
                const uint32_t kv = key_e[e];
                if (kv != FU_SKIP) {
                    const uint32_t row = kv >> 16;
                    sorted[whist[wv][row] + (kv & 0xffffu)] = (row << EB) | (BAGDIRECT ? bagv[it] : e);
                }
            }
            __syncthreads();
            for (int i = threadIdx.x; i < FU_WAVES * ROWS; i += FU_THREADS) (&whist[0][0])[i] = 0;
            // D. sums in sorted order: lane group g of wave w takes part P = w * E + g, an
            // equal share of the sorted chunk, and adds its elements one after another
            const uint32_t nk = nkept;
            const int P = wv * E + grp;
            const uint32_t lo = (uint32_t)(((uint64_t)nk * P) / NP), hi = (uint32_t)(((uint64_t)nk * (P + 1)) / NP);
            uint32_t first_key = SEG_PAD, last_key = SEG_PAD;
            bool head_cont = false, tail_cont = false;
            if (lo < hi) {
                first_key = sorted[lo] >> EB;
                last_key = sorted[hi - 1] >> EB;
                head_cont = lo > 0 && (sorted[lo - 1] >> EB) == first_key;
                tail_cont = hi < nk && (sorted[hi] >> EB) == last_key;
            }
            const uint32_t cnt = hi - lo;
            const uint32_t cmax = (nk + NP - 1) / NP;  // longest part (uniform loop bound)
            Cols4 acc[NC];
#pragma unroll
            for (int h = 0; h < NC; ++h) acc[h] = Cols4{{0.f, 0.f, 0.f, 0.f}};
            uint32_t acc_key = SEG_PAD;
            for (uint32_t s0 = 0; s0 < cmax; s0 += U) {
                uint32_t key[U], el[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t i = s0 + u;
                    const uint32_t v = i < cnt ? sorted[lo + i] : 0u;
                    key[u] = i < cnt ? v >> EB : SEG_PAD;
                    el[u] = v & EMASK;
                }
                const uint32_t key_after = s0 + U < cnt ? sorted[lo + s0 + U] >> EB : SEG_PAD;
                // where each segment that ends here goes: the table row, or this part's head /
                // tail piece when the segment runs on into the previous / next part
                int dst[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t k = key[u];
                    const uint32_t knext = u + 1 < U ? key[u + 1 < U ? u + 1 : u] : key_after;
                    int d = DST_NONE;
                    if (k != SEG_PAD && colok && knext != k) {
                        if (head_cont && k == first_key) d = DST_HEAD;
                        else if (tail_cont && k == last_key) d = DST_TAIL;
                        else d = DST_ROW;
                    }
                    dst[u] = d;
                }
                // all loads first (padding lanes read bag b0 / row 0 and are masked when used):
                // a load's registers are not written again before use, so none waits for another
                Cols4 x[U][NC], o4[U][NC], old[U][NC];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const bool ok = key[u] != SEG_PAD && colok;
                    const int cc = colok ? c : 0;
                    const uint32_t ee = ok ? el[u] : 0u;
                    const int64_t b = b0 + (ok ? (BAGS && !BAGDIRECT ? (int64_t)bag_e[ee] : (int64_t)ee) : 0);
#pragma unroll
                    for (int h = 0; h < NC; ++h) x[u][h] = load4(gx + b * a.d + cc + 4 * h);
                    if (MUL) {
                        const T* o = otab + (int64_t)(ok ? other_e[ee] : 0u) * D + cc;
#pragma unroll
                        for (int h = 0; h < NC; ++h)
#pragma unroll
                            for (int q = 0; q < 4; ++q) o4[u][h].v[q] = st<T>::load(o + 4 * h + q);
                    }
                    // the table row is loaded only where a segment ends (in the forms
                    // with one workgroup per CU: the branch costs registers)
                    if (ROWS == FU_ROWS_SMALL || dst[u] == DST_ROW) {
                        const float* orow = gtab + (int64_t)(dst[u] == DST_ROW ? key[u] : 0u) * D + cc;
#pragma unroll
                        for (int h = 0; h < NC; ++h) old[u][h] = load4(orow + 4 * h);
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint32_t k = key[u];
                    const bool cont = k == acc_key;
                    // padding elements past the part's end and lanes past the row width add
                    // stand-in values, but their sums are never stored or carried
#pragma unroll
                    for (int h = 0; h < NC; ++h)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const float v = MUL ? x[u][h].v[q] * o4[u][h].v[q] : x[u][h].v[q];
                            acc[h].v[q] = cont ? acc[h].v[q] + v : v;
                        }
                    acc_key = k;
                    if (dst[u] == DST_ROW) {
#pragma unroll
                        for (int h = 0; h < NC; ++h) {
#pragma unroll
                            for (int q = 0; q < 4; ++q) old[u][h].v[q] += acc[h].v[q];
                            store4(gtab + (int64_t)k * D + c + 4 * h, old[u][h]);
                        }
                    } else if (dst[u] != DST_NONE) {
                        float* cp = &carry[dst[u] == DST_HEAD ? 0 : 1][P][c];
#pragma unroll
                        for (int h = 0; h < NC; ++h)
#pragma unroll
                            for (int q = 0; q < 4; ++q) cp[4 * h + q] = acc[h].v[q];
                    }
                }
            }
            __syncthreads();
            // E. a segment that runs on into later parts is finished by the part where it
            // starts: its tail piece, then the head pieces of the parts it covers, in order
            if (lo < hi && tail_cont && !(head_cont && first_key == last_key) && colok) {
                float tot[CPL];
#pragma unroll
                for (int q = 0; q < CPL; ++q) tot[q] = carry[1][P][c + q];
                for (int p2 = P + 1; p2 < NP; ++p2) {
                    const uint32_t lo2 = (uint32_t)(((uint64_t)nk * p2) / NP);
                    const uint32_t hi2 = (uint32_t)(((uint64_t)nk * (p2 + 1)) / NP);
                    if (lo2 == hi2) continue;
                    if ((sorted[lo2] >> EB) != last_key) break;
#pragma unroll
                    for (int q = 0; q < CPL; ++q) tot[q] += carry[0][p2][c + q];
                    if ((sorted[hi2 - 1] >> EB) != last_key) break;
                }
                float* dstp = gtab + (int64_t)last_key * D + c;
#pragma unroll
                for (int h = 0; h < NC; ++h) {
                    Cols4 old = load4(dstp + 4 * h);
#pragma unroll
                    for (int q = 0; q < 4; ++q) old.v[q] += tot[4 * h + q];
                    store4(dstp + 4 * h, old);
                }
            }
            // no barrier: E reads `sorted` and `carry`, which the next chunk writes only
            // after its first barrier, and that barrier also orders E's row update before
            // the next chunk's updates of the same rows
        }
        b0 += take;
    }
}

struct RedPtrs {
    const uint32_t *keys, *vals, *bag_of, *qrow, *rrow;
    float *carry_head, *carry_tail;
};

template <typename T, int L, bool MUL, bool BAGS>
hipError_t launch_reduce(const EmbedBwdArgs& a, const RedPtrs& p, uint32_t n, hipStream_t st) {
    SegCtx<T> s;
    s.a = a;
    s.keys = p.keys;
    s.vals = p.vals;
    s.bag_of = p.bag_of;
    s.qrow = p.qrow;
    s.rrow = p.rrow;
    s.n = n;
    s.sentinel = (uint32_t)a.F * (a.hashed ? 2u : 1u) * (a.rows_q + a.m);
    s.rbase = (uint32_t)a.F * (a.hashed ? 2u : 1u) * a.rows_q;
    const uint32_t ntiles = (n + SEG_TILE - 1) / SEG_TILE;
    const unsigned blocks = (ntiles + 3) / 4;
    hipLaunchKernelGGL((k_seg_reduce<T, L, MUL, BAGS>), dim3(blocks), dim3(256), 0, st, s, p.carry_head,
                       p.carry_tail);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_seg_fixup<L>), dim3(blocks), dim3(256), 0, st, p.keys, n, s.sentinel, s.rbase, a.D,
                       a.grad_q, a.grad_r, p.carry_head, p.carry_tail);
    return hipGetLastError();
}

// lanes per pair (4 columns each) for table width D <= 256
template <typename T, bool MUL, bool BAGS>
hipError_t launch_reduce_d(const EmbedBwdArgs& a, const RedPtrs& p, uint32_t n, hipStream_t st) {
    const int q = (a.D + 3) / 4;
    if (q <= 4) return launch_reduce<T, 4, MUL, BAGS>(a, p, n, st);
    if (q <= 8) return launch_reduce<T, 8, MUL, BAGS>(a, p, n, st);
    if (q <= 16) return launch_reduce<T, 16, MUL, BAGS>(a, p, n, st);
    if (q <= 32) return launch_reduce<T, 32, MUL, BAGS>(a, p, n, st);
    return launch_reduce<T, 64, MUL, BAGS>(a, p, n, st);
}

template <typename T, bool MUL, bool BAGS, int ROWS, int CPL, int CAP = FU_CAP>
hipError_t launch_fused_rows(const FusedArgs& fa, unsigned blocks, hipStream_t st) {
    const int q = (fa.a.D + CPL - 1) / CPL;  // lanes per element needed
#define RDCN_FUSED(L) \
    hipLaunchKernelGGL((k_emb_fused<T, L, MUL, BAGS, ROWS, CPL, CAP>), dim3(blocks), dim3(FU_THREADS), 0, st, fa)
    if (q <= 4) RDCN_FUSED(4);
    else if (q <= 8) RDCN_FUSED(8);
    else if (q <= 16) RDCN_FUSED(16);
    else if (q <= 32) RDCN_FUSED(32);
    else RDCN_FUSED(64);
#undef RDCN_FUSED
    return hipGetLastError();
}

template <typename T, bool MUL, bool BAGS>
hipError_t launch_fused_d(const FusedArgs& fa, unsigned blocks, hipStream_t st) {
    const uint32_t rps = fa.rps_q > fa.rps_r ? fa.rps_q : fa.rps_r;
    if (rps <= (uint32_t)FU_ROWS_SMALL) return launch_fused_rows<T, MUL, BAGS, FU_ROWS_SMALL, 4>(fa, blocks, st);
    // slices of up to 2048 rows without the product combine: chunks of 8192 occurrences
    // (10240 with bags, whose sorted entries carry the bag and need no per-element bag
    // array), so each reached row of the slice is read and written less often
    if constexpr (!MUL)
        if (rps <= (uint32_t)FU_ROWS_MID && fa.a.D % 8 == 0)
            return launch_fused_rows<T, MUL, BAGS, FU_ROWS_MID, 8, BAGS ? 10240 : 2 * FU_CAP>(fa, blocks, st);
    if (fa.a.D % 8 == 0) return launch_fused_rows<T, MUL, BAGS, FU_ROWS, 8>(fa, blocks, st);
    return launch_fused_rows<T, MUL, BAGS, FU_ROWS, 4>(fa, blocks, st);
}

inline int key_bits(uint32_t maxkey) {
    int b = 1;
    while (b < 32 && (maxkey >> b) != 0) ++b;
    return b;
}

}  // namespace

EmbedBwdLayout embed_bwd_layout(int64_t nnz, int F, int rows_q, int m, int D, bool bags, bool mul, bool hashed) {
    EmbedBwdLayout L;
    const uint64_t n = (uint64_t)emb_pairs(nnz, hashed);
    const uint64_t ntiles = (n + RS_TILE - 1) / RS_TILE;
    const int bits = key_bits((uint32_t)F * (hashed ? 2u : 1u) * (uint32_t)(rows_q + m));
    const int passes = (bits + RS_MAX_BITS - 1) / RS_MAX_BITS;
    const int dbits = (bits + passes - 1) / passes;
    const uint64_t hist = ((uint64_t)1 << dbits) * (ntiles ? ntiles : 1);
    const uint64_t sums = RS_BUCKETS;  // digit totals of one pass
    const uint64_t segtiles = (n + SEG_TILE - 1) / SEG_TILE + 1;
    auto al = [](uint64_t x) { return (x + 255) & ~(uint64_t)255; };
    uint64_t off = 0;
    L.keys0 = off; off += al(4 * n);
    L.vals0 = off; off += al(4 * n);
    L.keys1 = off; off += al(4 * n);
    L.vals1 = off; off += al(4 * n);
    L.bag_of = off; off += bags ? al(4 * (uint64_t)nnz) : 0;
    L.qrow = off; off += mul ? al(4 * (hashed ? 2 : 1) * (uint64_t)nnz) : 0;  // per (occurrence, half)
    L.rrow = off; off += mul ? al(4 * (hashed ? 2 : 1) * (uint64_t)nnz) : 0;
    L.hist = off; off += al(4 * hist);
    L.sums = off; off += al(4 * sums);
    L.carry_head = off; off += al(4 * segtiles * (uint64_t)D);
    L.carry_tail = off; off += al(4 * segtiles * (uint64_t)D);
    L.total = off;
    L.bits = bits;
    L.passes = passes;
    L.dbits = dbits;
    return L;
}

struct EmbPtrs {
    uint32_t* keys[2];
    uint32_t* vals[2];
    uint32_t* bag_of;
    uint32_t *qrow, *rrow;
    uint32_t* hist;
    uint32_t* sums;
    float* carry_head;
    float* carry_tail;
    EmbedBwdLayout L;
};

static EmbPtrs emb_ptrs(const EmbedBwdArgs& a, void* scratch) {
    EmbPtrs p;
    const bool bags = a.offsets != nullptr;
    const bool mul = a.combine == 0;
    p.L = embed_bwd_layout(a.nnz, a.F, a.rows_q, a.m, a.D, bags, mul, a.hashed != 0);
    char* base = (char*)scratch;
    p.keys[0] = (uint32_t*)(base + p.L.keys0);
    p.keys[1] = (uint32_t*)(base + p.L.keys1);
    p.vals[0] = (uint32_t*)(base + p.L.vals0);
    p.vals[1] = (uint32_t*)(base + p.L.vals1);
    p.bag_of = bags ? (uint32_t*)(base + p.L.bag_of) : nullptr;
    p.qrow = mul ? (uint32_t*)(base + p.L.qrow) : nullptr;
    p.rrow = mul ? (uint32_t*)(base + p.L.rrow) : nullptr;
    p.hist = (uint32_t*)(base + p.L.hist);
    p.sums = (uint32_t*)(base + p.L.sums);
    p.carry_head = (float*)(base + p.L.carry_head);
    p.carry_tail = (float*)(base + p.L.carry_tail);
    return p;
}

hipError_t launch_emb_keys(const EmbedBwdArgs& a, bool ids64, void* scratch, hipStream_t st) {
    if (a.nnz == 0 || a.F == 0) return hipSuccess;
    const EmbPtrs P = emb_ptrs(a, scratch);
    const bool bags = a.offsets != nullptr;
    const int64_t units = bags ? a.batch * a.F : a.nnz;
    int64_t blocks = (units + 255) / 256;
    if (blocks > 65536) blocks = 65536;
#define RDCN_KEYS(ID, BG, MU)                                                                                   \
    do {                                                                                                        \
        if (a.hashed)                                                                                           \
            hipLaunchKernelGGL((k_emb_keys<ID, BG, MU, true>), dim3((unsigned)blocks), dim3(256), 0, st, a,     \
                               P.keys[0], P.vals[0], P.bag_of, P.qrow, P.rrow);                                 \
        else                                                                                                    \
            hipLaunchKernelGGL((k_emb_keys<ID, BG, MU, false>), dim3((unsigned)blocks), dim3(256), 0, st, a,    \
                               P.keys[0], P.vals[0], P.bag_of, P.qrow, P.rrow);                                 \
    } while (0)
#define RDCN_KEYS_M(ID, BG) do { if (a.combine == 0) RDCN_KEYS(ID, BG, true); else RDCN_KEYS(ID, BG, false); } while (0)
    if (ids64) { if (bags) RDCN_KEYS_M(int64_t, true); else RDCN_KEYS_M(int64_t, false); }
    else       { if (bags) RDCN_KEYS_M(int32_t, true); else RDCN_KEYS_M(int32_t, false); }
#undef RDCN_KEYS_M
#undef RDCN_KEYS
    return hipGetLastError();
}

// The sorted pairs end in buffer (passes % 2).
hipError_t launch_emb_sort(const EmbedBwdArgs& a, void* scratch, hipStream_t st) {
    if (a.nnz == 0 || a.F == 0) return hipSuccess;
    const EmbPtrs P = emb_ptrs(a, scratch);
    const uint32_t n = (uint32_t)emb_pairs(a.nnz, a.hashed != 0);
    const int ntiles = (int)((n + RS_TILE - 1) / RS_TILE);
    int cur = 0;
    for (int pass = 0; pass < P.L.passes; ++pass) {
        const int shift = pass * P.L.dbits;
        const int bits = P.L.bits - shift < P.L.dbits ? P.L.bits - shift : P.L.dbits;
        const uint32_t mask = (1u << bits) - 1u;
        hipLaunchKernelGGL(k_rs_hist, dim3(ntiles), dim3(RS_THREADS), 0, st, P.keys[cur], n, shift, mask, P.hist,
                           ntiles);
        const int ndig = (int)(mask + 1);
        hipLaunchKernelGGL(k_digit_scan, dim3(ndig), dim3(256), 0, st, P.hist, ntiles, P.sums);
        hipLaunchKernelGGL(k_rs_scatter, dim3(ntiles), dim3(RS_THREADS), 0, st, P.keys[cur], P.vals[cur],
                           P.keys[cur ^ 1], P.vals[cur ^ 1], n, shift, bits, P.hist, ntiles, P.sums);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        cur ^= 1;
    }
    return hipSuccess;
}

hipError_t launch_emb_reduce(const EmbedBwdArgs& a, bool bf16, void* scratch, hipStream_t st) {
    if (a.nnz == 0 || a.F == 0) return hipSuccess;
    const EmbPtrs P = emb_ptrs(a, scratch);
    const uint32_t n = (uint32_t)emb_pairs(a.nnz, a.hashed != 0);
    const int cur = P.L.passes & 1;
    const RedPtrs rp = {P.keys[cur], P.vals[cur], P.bag_of, P.qrow, P.rrow, P.carry_head, P.carry_tail};
    const bool mul = a.combine == 0, bags = a.offsets != nullptr;
#define RDCN_RED(T) do {                                                  \
        if (mul) return bags ? launch_reduce_d<T, true, true>(a, rp, n, st) : launch_reduce_d<T, true, false>(a, rp, n, st); \
        return bags ? launch_reduce_d<T, false, true>(a, rp, n, st) : launch_reduce_d<T, false, false>(a, rp, n, st);      \
    } while (0)
    if (bf16) RDCN_RED(bf16_t);
    RDCN_RED(float);
#undef RDCN_RED
}

bool emb_fused_ok(int rows_q, int m, int D, bool hashed) {
    return !hashed && D > 0 && D <= 256 && rows_q > 0 && m > 0 && rows_q <= FU_MAX_TABLE_ROWS &&
           m <= FU_MAX_TABLE_ROWS;
}

hipError_t launch_emb_fused(const EmbedBwdArgs& a, bool bf16, bool ids64, hipStream_t st) {
    if (a.nnz == 0 || a.F == 0 || a.batch == 0) return hipSuccess;
    if (!emb_fused_ok(a.rows_q, (int)a.m, a.D, a.hashed != 0)) return hipErrorInvalidValue;
    FusedArgs fa;
    fa.a = a;
    fa.ids64 = ids64 ? 1 : 0;
    const int rmax = a.rows_q > (int)a.m ? a.rows_q : (int)a.m;
    // Every workgroup walks all of its feature's occurrences, so its time hardly
    // depends on how many rows its slice has. When the smallest slice count (slices of
    // up to FU_ROWS rows) keeps all workgroups resident at once (one per CU), take the
    // most slices that still do; otherwise slices of FU_SPLIT_ROWS rows, which keep
    // each of the several rounds short (µs, small / feed / multihot / large:
    // 36 / 218 / 1634 / 1426 this way, against 36 / 247 / 2126 / 1424 with slices
    // of at most 1024 rows everywhere and 46 / 219 / 2294 / 1550 with the fewest slices).
    const int per_slice = 2 * a.F;  // workgroups per slice index (two tables per feature)
    int S = (rmax + FU_ROWS - 1) / FU_ROWS;
    if (per_slice * S <= FU_ONE_ROUND) {
        const int fit = FU_ONE_ROUND / per_slice;
        if (fit > S) S = fit;
    } else {
        const int split = (rmax + FU_SPLIT_ROWS - 1) / FU_SPLIT_ROWS;
        if (split > S) S = split;
    }
    if (S > FU_MAX_SLICES) S = FU_MAX_SLICES;
    if (S > rmax) S = rmax;
    fa.slices = S;
    fa.rps_q = (uint32_t)((a.rows_q + S - 1) / S);
    fa.rps_r = (a.m + (uint32_t)S - 1) / (uint32_t)S;
    const unsigned blocks = 8u * (unsigned)((a.F + 7) / 8) * 2u * (unsigned)S;
    const bool mul = a.combine == 0, bags = a.offsets != nullptr;
#define RDCN_FU(T)                                                                                           \
    do {                                                                                                     \
        if (mul) return bags ? launch_fused_d<T, true, true>(fa, blocks, st) : launch_fused_d<T, true, false>(fa, blocks, st); \
        return bags ? launch_fused_d<T, false, true>(fa, blocks, st) : launch_fused_d<T, false, false>(fa, blocks, st);       \
    } while (0)
    if (bf16) RDCN_FU(bf16_t);
    RDCN_FU(float);
#undef RDCN_FU
}

// ---------------------------------------------------------------------------
// Workspace of the allocation-free embedding backward (qr_embed_backward_static):
// a file-scope device array, one copy on every GPU the library runs on, held until
// the process ends. Its name is a host-side stand-in in host code; kernels get the
// device address that hipGetSymbolAddress returns for the current device.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[EMB_STATIC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};
}  // namespace

hipError_t emb_static_scratch(void** out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace rdcn
