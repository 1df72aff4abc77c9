// Shared device helpers of the gfx950 YOSO kernels (internal header).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace yoso {

constexpr int D = 64;  // head dimension supported by the kernels

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Exact widening of bf16 bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Load 8 consecutive elements of a row (fp32 or bf16 storage) as fp32.
// `p` must be 16-byte aligned for fp32 and 16-byte aligned for bf16.
template <bool BF16>
__device__ __forceinline__ void load8(const void *base, int64_t elem_off, float out[8]) {
    if constexpr (BF16) {
        const uint4 w = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(base) + elem_off);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            out[2 * i] = __uint_as_float(ws[i] << 16);
            out[2 * i + 1] = __uint_as_float(ws[i] & 0xFFFF0000u);
        }
    } else {
        const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(base) + elem_off);
        const float4 a = p[0], b = p[1];
        out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
        out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
    }
}

// Load one element (fp32 or bf16 storage) as fp32.
template <bool BF16>
__device__ __forceinline__ float load1(const void *base, int64_t elem_off) {
    if constexpr (BF16)
        return bf16_to_f32(static_cast<const uint16_t *>(base)[elem_off]);
    else
        return static_cast<const float *>(base)[elem_off];
}

// Split fp32 values into an fp16 pair (hi + lo) after multiplying by `scale`
// (a power of two, so the scaling is exact).  hi + lo carries about 22
// significant bits: enough that the three MFMA products hi*hi, hi*lo, lo*hi
// reproduce an fp32 dot product to ~1e-6 relative.
// The scaled value passes through an empty asm operand, so that hi and lo are
// both derived from the one fp32 register s.  Left visible, the product that
// produced s gets fused into the conversions (v_fma_mixlo_f16 rounds the exact
// product to fp16 once) for one use of hi while the kept hi is rounded to fp32
// first; where the two roundings differ (an fp32 result on an fp16 tie), lo
// compensates the wrong hi and hi + lo is off by one fp16 ulp.
__device__ __forceinline__ void split8(const float v[8], float scale, half8 &hi, half8 &lo) {
#pragma clang fp contract(off)
#pragma unroll
    for (int i = 0; i < 8; i++) {
        float s = v[i] * scale;
        asm volatile("" : "+v"(s));
        const _Float16 h = static_cast<_Float16>(s);
        hi[i] = h;
        lo[i] = static_cast<_Float16>(s - static_cast<float>(h));
    }
}

__device__ __forceinline__ void split4(const float v[4], float scale, half4 &hi, half4 &lo) {
#pragma clang fp contract(off)
#pragma unroll
    for (int i = 0; i < 4; i++) {
        float s = v[i] * scale;
        asm volatile("" : "+v"(s));
        const _Float16 h = static_cast<_Float16>(s);
        hi[i] = h;
        lo[i] = static_cast<_Float16>(s - static_cast<float>(h));
    }
}

// split4 for a power-of-two `scale`: v * scale is exact, so rounding the product to
// fp16 once or through fp32 gives the same hi, and the operand barrier is not needed.
__device__ __forceinline__ void split4_pow2(const float v[4], float scale, half4 &hi, half4 &lo) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const float s = v[i] * scale;
        const _Float16 h = static_cast<_Float16>(s);
        hi[i] = h;
        lo[i] = static_cast<_Float16>(s - static_cast<float>(h));
    }
}

// Load a T at `byte_off` bytes past `base` (a wave-uniform pointer): keeps the
// per-lane part of the address in one 32-bit register.
template <typename T>
__device__ __forceinline__ T ld(const void *base, uint32_t byte_off) {
    return *reinterpret_cast<const T *>(static_cast<const char *>(base) + byte_off);
}

// Three-product fp16 emulation of an fp32 MFMA step: acc += a*b.
__device__ __forceinline__ floatx4 mfma3_16x16x32(const half8 &ah, const half8 &al, const half8 &bh,
                                                  const half8 &bl, floatx4 acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bh, acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ floatx4 mfma3_16x16x16(const half4 &ah, const half4 &al, const half4 &bh,
                                                  const half4 &bl, floatx4 acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(ah, bh, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(ah, bl, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(al, bh, acc, 0, 0, 0);
    return acc;
}

// ---- cross-lane sums without LDS traffic (DPP and the gfx950 permlane swaps)
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Butterfly sum over aligned groups of W lanes (W a power of two, 1 <= W <= 64):
// every lane of a group ends with the group's total.  Must run with all lanes
// of each group active.  Steps: xor 1 and xor 2 (quad_perm), the other quad of
// a half-row (row_half_mirror), the other half-row (row_mirror), the other row
// of a row pair (permlane16_swap), the other half of the wave (permlane32_swap).
__device__ __forceinline__ float group_sum(float x, int W) {
    if (W >= 2) x += dpp_mov<0xB1>(x);   // quad_perm [1,0,3,2]
    if (W >= 4) x += dpp_mov<0x4E>(x);   // quad_perm [2,3,0,1]
    if (W >= 8) x += dpp_mov<0x141>(x);  // row_half_mirror
    if (W >= 16) x += dpp_mov<0x140>(x); // row_mirror
    if (W >= 32) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    if (W >= 64) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    return x;
}

// Maximum over the whole wave (every lane gets it).
__device__ __forceinline__ float wave_max(float x) {
    x = fmaxf(x, dpp_mov<0xB1>(x));
    x = fmaxf(x, dpp_mov<0x4E>(x));
    x = fmaxf(x, dpp_mov<0x141>(x));
    x = fmaxf(x, dpp_mov<0x140>(x));
    {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    return x;
}

// Exponent e with amax < 2^e (amax >= 0 finite; 0 for amax == 0), clamped to
// [-60, 60] so that scales 2^(13 - e) stay normal floats.
__device__ __forceinline__ int pow2_above(float amax) {
    int e = 0;
    if (amax > 0.f) frexpf(amax, &e);  // amax = f 2^e, f in [0.5, 1)
    return min(max(e, -60), 60);
}

// Workgroups are dispatched to the 8 XCDs round-robin (id % 8).  Remap so that
// consecutive logical ids land on the same XCD and share its L2; the mapping is
// a bijection on [0, n) for any n.
__device__ __forceinline__ int64_t xcd_remap(int64_t id, int64_t n) {
    constexpr int64_t X = 8;
    const int64_t q = n / X, r = n % X;
    const int64_t x = id % X, i = id / X;
    return x * q + (x < r ? x : r) + i;
}

}  // namespace yoso
