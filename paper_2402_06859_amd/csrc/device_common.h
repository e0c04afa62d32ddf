// Device-side helpers shared by the gfx950 kernels of librdcn.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rdcn {

typedef uint16_t bf16_t;  // raw bfloat16 bits
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint32_t raw16) { return __uint_as_float(raw16 << 16); }

// Values at or beyond this magnitude round to infinity when converted to f16.
constexpr float F16_OVERFLOW = 65520.f;

// 8 floats -> one 16-byte vector of 8 f16 (round to nearest, ties to even); `ovf` is
// set when a value is beyond the f16 range (it becomes infinity).
__device__ __forceinline__ u32x4_t pack_f16x8(const float* v, bool& ovf) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const half2_t p = {(_Float16)v[2 * i], (_Float16)v[2 * i + 1]};
        w[i] = __builtin_bit_cast(uint32_t, p);
    }
    // one test on the largest magnitude (fmaxf passes over NaN, which is not flagged)
    const float mx = fmaxf(fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))),
                           fmaxf(fmaxf(fabsf(v[4]), fabsf(v[5])), fmaxf(fabsf(v[6]), fabsf(v[7]))));
    ovf |= mx >= F16_OVERFLOW;
    return u32x4_t{w[0], w[1], w[2], w[3]};
}

__device__ __forceinline__ void unpack_f16x8(const u32x4_t& w, float* v) {
    const uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const half2_t p = __builtin_bit_cast(half2_t, x[i]);
        v[2 * i] = (float)p.x;
        v[2 * i + 1] = (float)p.y;
    }
}

// Two floats -> one word holding (lo, hi) bfloat16 values: gfx950's packed conversion
// (v_cvt_pk_bf16_f32), one instruction for both. It rounds as the wave's float mode
// says, and every kernel here runs with round to nearest, ties to even, and float
// denormals kept, so the result is the nearest bfloat16 with ties to even for every
// finite input (denormals and overflow to infinity included); NaN stays NaN.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t p = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, p);
}

// float -> bfloat16 bits (as pack_bf16x2).
__device__ __forceinline__ uint32_t f32_to_bf16(float x) { return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x); }

// Storage-type traits: T is float or bf16_t.
template <typename T> struct st;
template <> struct st<float> {
    static constexpr int vec = 4;  // elements per 16-byte vector
    __device__ static __forceinline__ float round(float v) { return v; }  // the value a store keeps
    __device__ static __forceinline__ float load(const float* p) { return *p; }
    __device__ static __forceinline__ void store(float* p, float v) { *p = v; }
    // 16-byte vector <-> 4 floats
    __device__ static __forceinline__ void unpack(const u32x4_t& w, float* v) {
        v[0] = __uint_as_float(w.x); v[1] = __uint_as_float(w.y);
        v[2] = __uint_as_float(w.z); v[3] = __uint_as_float(w.w);
    }
    __device__ static __forceinline__ u32x4_t pack(const float* v) {
        return u32x4_t{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
    }
};
template <> struct st<bf16_t> {
    static constexpr int vec = 8;
    __device__ static __forceinline__ float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
    __device__ static __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
    __device__ static __forceinline__ void store(bf16_t* p, float v) { *p = (bf16_t)f32_to_bf16(v); }
    __device__ static __forceinline__ void unpack(const u32x4_t& w, float* v) {
        v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xffff0000u);
        v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xffff0000u);
        v[4] = __uint_as_float(w.z << 16); v[5] = __uint_as_float(w.z & 0xffff0000u);
        v[6] = __uint_as_float(w.w << 16); v[7] = __uint_as_float(w.w & 0xffff0000u);
    }
    __device__ static __forceinline__ u32x4_t pack(const float* v) {
        return u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                       pack_bf16x2(v[6], v[7])};
    }
};

// Unsigned 32-bit division by an invariant divisor m >= 1 (Granlund & Montgomery,
// "Division by invariant integers using multiplication", 1994, unsigned case):
//   t = mulhi(magic, n);  q = (t + ((n - t) >> 1)) >> shift_minus_1   (m > 1)
struct DivMagic {
    uint32_t magic;
    uint32_t shift;  // l - 1 where l = ceil(log2 m); unused when m == 1
    uint32_t m;
};
__device__ __forceinline__ uint32_t div_magic(uint32_t n, const DivMagic& dm) {
    if (dm.m == 1) return n;
    uint32_t t = __umulhi(dm.magic, n);
    return (t + ((n - t) >> 1)) >> dm.shift;
}

// MurmurHash64A (Austin Appleby, MurmurHash2 family) of one 8-byte key, from the
// published description: the key's little-endian bytes are one block.
__device__ __forceinline__ uint64_t murmur64a_8(uint64_t key, uint64_t seed) {
    const uint64_t m = 0xc6a4a7935bd1e995ull;
    uint64_t h = seed ^ (8ull * m);
    uint64_t k = key * m;
    k ^= k >> 47;
    k *= m;
    h ^= k;
    h *= m;
    h ^= h >> 47;
    h *= m;
    h ^= h >> 47;
    return h;
}

}  // namespace rdcn
