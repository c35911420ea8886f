// common.hpp -- device helpers shared by the ELSAA HIP kernels (gfx950 only).
//
// Matrix-core convention used by every kernel (v_mfma_f32_16x16x32_bf16 and,
// for float32 storage, eight v_mfma_f32_16x16x4_f32 per 32-wide k-step):
//   * a "k-step" contracts 32 values of k; lane l (0..63) holds, for both
//     operands, the 8 k-slots 8*(l/16) + j (j = 0..7) of row / column l%16;
//   * the accumulator tile is 16x16 float32: lane l holds rows 4*(l/16)+i
//     (i = 0..3) of column l%16.
// Which physical k each slot maps to does not matter as long as A and B use
// the same slot order, which is how all kernels build their fragments.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace elsaa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Storage traits: element type in HBM / LDS and the 8-slot operand fragment.
struct BF16 {
    using store_t = uint16_t;
    using frag_t = bf16x8;
    static constexpr int bytes = 2;
    __device__ static __forceinline__ float load(store_t v) { return bf16_to_f32(v); }
    __device__ static __forceinline__ store_t store(float v) { return f32_to_bf16(v); }
    __device__ static __forceinline__ f32x4 mma(frag_t a, frag_t b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    // 8 contiguous elements (16-byte aligned)
    __device__ static __forceinline__ frag_t ld8(const store_t* p) { return *(const frag_t*)p; }
    // elements p0[0..3] then p1[0..3] (8-byte aligned each)
    __device__ static __forceinline__ frag_t ld44(const store_t* p0, const store_t* p1)
    {
        bf16x4 a = *(const bf16x4*)p0, b = *(const bf16x4*)p1;
        return frag_t{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    }
    __device__ static __forceinline__ frag_t pack(const float* v)
    {
        frag_t f;
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = (__bf16)v[j];
        return f;
    }
    // v = hi + lo to about 2^-16 relative (both bf16): float32-accurate operand
    static constexpr bool kSplit = true;
    __device__ static __forceinline__ void split(const float* v, frag_t& hi, frag_t& lo)
    {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint16_t h = f32_to_bf16(v[j]);
            hi[j] = __builtin_bit_cast(__bf16, h);
            lo[j] = __builtin_bit_cast(__bf16, f32_to_bf16(v[j] - bf16_to_f32(h)));
        }
    }
};

struct F32 {
    using store_t = float;
    using frag_t = f32x8;
    static constexpr int bytes = 4;
    __device__ static __forceinline__ float load(store_t v) { return v; }
    __device__ static __forceinline__ store_t store(float v) { return v; }
    __device__ static __forceinline__ f32x4 mma(frag_t a, frag_t b, f32x4 c)
    {
#pragma unroll
        for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
        return c;
    }
    __device__ static __forceinline__ frag_t ld8(const store_t* p)
    {
        f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
        return frag_t{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    }
    __device__ static __forceinline__ frag_t ld44(const store_t* p0, const store_t* p1)
    {
        f32x4 a = *(const f32x4*)p0, b = *(const f32x4*)p1;
        return frag_t{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    }
    __device__ static __forceinline__ frag_t pack(const float* v)
    {
        frag_t f;
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = v[j];
        return f;
    }
    static constexpr bool kSplit = false;   // float32 operands are exact
    __device__ static __forceinline__ void split(const float* v, frag_t& hi, frag_t& lo)
    {
        hi = pack(v);
        lo = hi;
    }
};

// (a_hi + a_lo) x b: product with the A operand kept in float32 accuracy
template <class T>
__device__ __forceinline__ f32x4 mma_split_a(const float* a, typename T::frag_t b, f32x4 c)
{
    typename T::frag_t hi, lo;
    T::split(a, hi, lo);
    c = T::mma(hi, b, c);
    if (T::kSplit) c = T::mma(lo, b, c);
    return c;
}

// a x (b_hi + b_lo): product with an operand kept in float32 accuracy
template <class T>
__device__ __forceinline__ f32x4 mma_split(typename T::frag_t a, const float* b, f32x4 c)
{
    typename T::frag_t hi, lo;
    T::split(b, hi, lo);
    c = T::mma(a, hi, c);
    if (T::kSplit) c = T::mma(a, lo, c);
    return c;
}

// Four consecutive outputs of one row in the storage dtype, one store.
template <class T>
__device__ __forceinline__ void store4(typename T::store_t* p, f32x4 v)
{
    if constexpr (T::bytes == 2) {
        const uint32_t lo = (uint32_t)T::store(v[0]) | ((uint32_t)T::store(v[1]) << 16);
        const uint32_t hi = (uint32_t)T::store(v[2]) | ((uint32_t)T::store(v[3]) << 16);
        *(uint2*)p = make_uint2(lo, hi);
    } else {
        *(f32x4*)p = v;
    }
}

// Four consecutive elements of the storage dtype as float32, one load.
template <class T>
__device__ __forceinline__ f32x4 load4(const typename T::store_t* p)
{
    if constexpr (T::bytes == 2) {
        const uint2 v = *(const uint2*)p;
        return f32x4{bf16_to_f32(v.x & 0xffffu), bf16_to_f32(v.x >> 16), bf16_to_f32(v.y & 0xffffu),
                     bf16_to_f32(v.y >> 16)};
    } else {
        return *(const f32x4*)p;
    }
}

// Four consecutive storage-dtype elements loaded as they are (no conversion,
// so a load issued early is not waited for until its value is used), and
// their float32 values.
template <class T> struct Raw4 {
    using type = f32x4;
    __device__ static __forceinline__ type ld(const typename T::store_t* p) { return *(const f32x4*)p; }
    __device__ static __forceinline__ f32x4 val(type v) { return v; }
};
template <> struct Raw4<BF16> {
    using type = uint2;
    __device__ static __forceinline__ type ld(const uint16_t* p) { return *(const uint2*)p; }
    __device__ static __forceinline__ f32x4 val(type v)
    {
        return f32x4{bf16_to_f32(v.x & 0xffffu), bf16_to_f32(v.x >> 16), bf16_to_f32(v.y & 0xffffu),
                     bf16_to_f32(v.y >> 16)};
    }
};

// x[e] += the 8 storage-dtype elements at p (16-byte aligned in bf16).
template <class T>
__device__ __forceinline__ void add8(const typename T::store_t* p, float (&x)[8])
{
    if constexpr (T::bytes == 2) {
        const uint4 v = *(const uint4*)p;
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] += bf16_to_f32(u[i] & 0xffffu);
            x[2 * i + 1] += bf16_to_f32(u[i] >> 16);
        }
    } else {
        const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] += a[i];
            x[4 + i] += b[i];
        }
    }
}

// 8 consecutive elements of the storage dtype from float32, one 16-byte
// store in bf16.
template <class T>
__device__ __forceinline__ void store8(typename T::store_t* p, const float (&x)[8])
{
    if constexpr (T::bytes == 2) {
        uint32_t u[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) u[i] = (uint32_t)T::store(x[2 * i]) | ((uint32_t)T::store(x[2 * i + 1]) << 16);
        *(uint4*)p = make_uint4(u[0], u[1], u[2], u[3]);
    } else {
        *(f32x4*)p = f32x4{x[0], x[1], x[2], x[3]};
        *(f32x4*)(p + 4) = f32x4{x[4], x[5], x[6], x[7]};
    }
}

// Eight consecutive storage-dtype elements loaded as they are (16 bytes in
// bf16), and their float32 values.
template <class T> struct Raw8 {
    struct type { f32x4 a, b; };
    __device__ static __forceinline__ type ld(const typename T::store_t* p)
    {
        return type{*(const f32x4*)p, *(const f32x4*)(p + 4)};
    }
    __device__ static __forceinline__ void val(type v, float (&x)[8])
    {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = v.a[i];
            x[4 + i] = v.b[i];
        }
    }
};
template <> struct Raw8<BF16> {
    using type = uint4;
    __device__ static __forceinline__ type ld(const uint16_t* p) { return *(const uint4*)p; }
    __device__ static __forceinline__ void val(type v, float (&x)[8])
    {
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] = bf16_to_f32(u[i] & 0xffffu);
            x[2 * i + 1] = bf16_to_f32(u[i] >> 16);
        }
    }
};

// 16-byte global load / store of raw bytes.
__device__ __forceinline__ uint4 ldg16(const void* p) { return *(const uint4*)p; }
__device__ __forceinline__ void stg16(void* p, uint4 v) { *(uint4*)p = v; }

// The values of lanes l & ~16 (lo) and l | 16 (hi) in every lane l, from one
// gfx950 v_permlane16_swap of v with itself (no LDS traffic); xpair32 does the
// same for lane bit 5.
struct LanePair {
    float lo, hi;
};
__device__ __forceinline__ LanePair xpair16(float v)
{
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ LanePair xpair32(float v)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}

// out[r] = v of lane (l % 16) + 16 r, for every lane l (three exchanges).
__device__ __forceinline__ void gather16x4(float v, float (&out)[4])
{
    const LanePair a = xpair16(v);                  // rows 2s, 2s + 1 of this lane's half s
    const LanePair b0 = xpair32(a.lo), b1 = xpair32(a.hi);
    out[0] = b0.lo;
    out[1] = b1.lo;
    out[2] = b0.hi;
    out[3] = b1.hi;
}

__device__ __forceinline__ float wave_max16(float v)   // max over lanes l, l^16, l^32, l^48
{
    const LanePair a = xpair16(v);
    const LanePair b = xpair32(fmaxf(a.lo, a.hi));
    return fmaxf(b.lo, b.hi);
}

__device__ __forceinline__ float wave_sum16(float v)   // sum over lanes l, l^16, l^32, l^48
{
    const LanePair a = xpair16(v);
    const LanePair b = xpair32(a.lo + a.hi);
    return b.lo + b.hi;
}

__device__ __forceinline__ float row_sum16(float v)    // sum over the 16 lanes of a row group
{
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 4);
    v += __shfl_xor(v, 8);
    return v;
}

// Transposed LDS read of 16-bit data (ds_read_b64_tr_b16, gfx950).  Within
// each group of 16 lanes, lane s supplies the LDS address of 4 contiguous
// elements; lane i receives element i % 4 of the pieces supplied by lanes
// i / 4 + 4 j, j = 0..3.  When lane s points at row kb + s / 4, columns
// c0 + 4 (s % 4) of a tile stored [k][c] (c contiguous), lane i receives
// column c0 + i at rows kb .. kb + 3: four consecutive k of one operand row.
__device__ __forceinline__ bf16x4 lds_read_tr4(const uint16_t* p)
{
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
    return __builtin_bit_cast(bf16x4, v);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Row order of a 64-row tile fed through four 16-row score sub-tiles so that
// the accumulators can be reused as a 32-wide k-step operand: register i of
// sub-tile s in lane group g holds tile row key_of(s, g, i), and sub-tiles
// 2m, 2m+1 together give lane group g the rows 32m + 8g .. 32m + 8g + 7.
__device__ __forceinline__ int key_of(int s, int g, int i) { return 32 * (s >> 1) + 8 * g + 4 * (s & 1) + i; }
// Tile row fed to operand row rho of sub-tile s (the inverse of key_of).
__device__ __forceinline__ int krow_of(int s, int rho) { return 32 * (s >> 1) + 8 * (rho >> 2) + 4 * (s & 1) + (rho & 3); }

}  // namespace elsaa
