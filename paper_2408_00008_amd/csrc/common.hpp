// Device-side helpers shared by the gfx950 kernels of libmoe.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef uint16_t bf16_t;  // raw bfloat16 bits in memory
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_t b)
{
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bfloat16, round to nearest even (gfx950's v_cvt_pk_bf16_f32; NaN
// stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f)
{
    return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    bf16x2_t v;
    v[0] = static_cast<__bf16>(lo);
    v[1] = static_cast<__bf16>(hi);
    return __builtin_bit_cast(uint32_t, v);
}

// silu(z) = z / (1 + exp(-z)) with the hardware exp2 and reciprocal (a few
// ulp in f32; the result is rounded to bf16).  Large negative z: exp -> inf,
// reciprocal -> 0, silu -> -0.
__device__ __forceinline__ float silu(float z)
{
    return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

// 16x16x32 bf16 MFMA, f32 accumulate (gfx950).  Operand A: lane l holds row
// (l % 16), reduction elements 8*(l/16) .. +7; operand B: lane l holds column
// (l % 16), the same reduction elements.  Result: lane l, element i holds
// D[4*(l/16) + i][l % 16].
__device__ __forceinline__ floatx4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const floatx4& c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 32x32x16 bf16 MFMA, f32 accumulate (gfx950).  Operand A: lane l holds row
// (l % 32), reduction elements 8*(l/32) .. +7; operand B: lane l holds column
// (l % 32), the same reduction elements.  Result: lane l, element 4*q + i
// holds D[8*q + 4*(l/32) + i][l % 32].
__device__ __forceinline__ floatx16 mfma32x32x16(const bf16x8& a, const bf16x8& b, const floatx16& c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v)
{
    return __builtin_bit_cast(bf16x8, v);
}

// Eight OCP FP8 E4M3 values (the bytes of lo, then of hi, in memory order) ->
// bf16x8.  Exact: every E4M3 value is a bfloat16 value.  The packed
// conversion results are taken as whole words.
__device__ __forceinline__ bf16x8 e4m3x8_to_bf16(uint32_t lo, uint32_t hi)
{
    uint4 r;
    r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, false));
    r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, true));
    r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, false));
    r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, true));
    return __builtin_bit_cast(bf16x8, r);
}

__device__ __forceinline__ uint4 ldg16(const void* p)
{
    return *reinterpret_cast<const uint4*>(p);
}

template <typename T>
__device__ __forceinline__ T wave_shfl_xor(T v, int mask)
{
    return __shfl_xor(v, mask, 64);
}

// Parts of the tiled down GEMM's reduction (used by that kernel and by the
// kernel that folds a heavy expert's parts back together).  The persistent
// workgroups of an XCD take its items in rounds, so the layer costs
// ceil(share / workgroups) rounds of one item; with a few hundred 256 x 256 tiles over 256 CUs the
// last round is mostly idle (560 tiles: 3 rounds for 2.2 rounds of work).
// Cutting every tile's reduction into S parts gives S times as many items of
// 1/S of the steps, which evens out the rounds, at the price of a start-up
// and an output store per item and S - 1 more f32 slices for the combine to
// read.  Cost in thousandths of a reduction step (one step = 64 elements of
// the reduction, ~1.5 us on the 4096 x 14336 shapes): per item 1000 nk / S +
// 6000, per extra slice A * N / 1800 (its read at ~5 TB/s).  Integer
// arithmetic, so every kernel that evaluates it gets the same answer.
__device__ __forceinline__ int down_parts(int total, int per_xcd, int nk, int64_t A, int N, int smax)
{
    int best = 1;
    int64_t best_cost = INT64_MAX;
    const int64_t slice_cost = A * N / 1800;
    for (int s = 1; s <= smax && s <= nk; s *= 2) {
        const int64_t share = ((int64_t)total * s + 7) / 8;
        const int64_t rounds = (share + per_xcd - 1) / per_xcd;
        const int64_t cost = rounds * (1000LL * nk / s + 6000) + (s - 1) * slice_cost;
        if (cost < best_cost) {
            best_cost = cost;
            best = s;
        }
    }
    return best;
}

}  // namespace moe
