// Device-side FP8 arithmetic shared by the kernels of libfp8lin.so: format
// parameters (Table 7), the Eq. 3 bias from an amax bit pattern, magnitude
// reductions, and the exact scale + saturating round-to-nearest-even cast of
// Sec. 2.1 Eq. 1 / App. A.  Internal, not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8lin.h"

namespace fp8lin {
namespace {

// ---------------------------------------------------------------- formats
// Largest finite value f_M * 2^kMaxExp, with f_M = 1.75 (kMantMax 0x600000 as
// fp32 mantissa bits) or 1.875 (0x700000).
// OCP FP8 (Table 7 rows "(b)"): converted by the hardware.
// The paper's formats (rows "(a)": E4 bias 8, max 240; E5 bias 16, max 57344;
// one NaN code 0x80, no infinity, no -0): every code finite in both families
// decodes in (a) to half its OCP value, so the (a) code of x at bias b is the
// OCP code of x * 2^(b + 1) (kShift), except where (a) has values above the OCP
// maximum, for -0 (0x00 in (a)) and for NaN (0x80 in (a)).
template <int FMT> struct Fmt;
template <> struct Fmt<FP8_E4M3> {
    static constexpr int kMaxExp = 8;  // max finite = 1.75 * 2^8 = 448
    static constexpr uint32_t kMantMax = 0x600000u;
    static constexpr float kMax = 448.0f;  // hardware clip (OCP maximum)
    static constexpr int kShift = 0, kHw = FP8_E4M3;
    static constexpr bool kPaper = false;
};
template <> struct Fmt<FP8_E5M2> {
    static constexpr int kMaxExp = 15;  // max finite = 1.75 * 2^15 = 57344
    static constexpr uint32_t kMantMax = 0x600000u;
    static constexpr float kMax = 57344.0f;
    static constexpr int kShift = 0, kHw = FP8_E5M2;
    static constexpr bool kPaper = false;
};
template <> struct Fmt<FP8_E4_A> {
    static constexpr int kMaxExp = 7;  // max finite = 1.875 * 2^7 = 240
    static constexpr uint32_t kMantMax = 0x700000u;
    static constexpr float kMax = 448.0f;
    static constexpr int kShift = 1, kHw = FP8_E4M3;
    static constexpr bool kPaper = true;
};
template <> struct Fmt<FP8_E5_A> {
    static constexpr int kMaxExp = 15;  // max finite = 1.75 * 2^15 = 57344
    static constexpr uint32_t kMantMax = 0x600000u;
    static constexpr float kMax = 57344.0f;
    static constexpr int kShift = 1, kHw = FP8_E5M2;
    static constexpr bool kPaper = true;
};

constexpr int kBiasClamp = 512;  // beyond this every input saturates or flushes

// Eq. 3 on the fp32 bit pattern of the amax: with amax = 1.f_a * 2^ea and
// max_num = f_M * 2^eM, floor(log2(max_num / amax)) = eM - ea - [1.f_a > f_M].
template <int FMT>
__device__ __forceinline__ int32_t bias_of(uint32_t u, int32_t margin, uint32_t* fl) {
    u &= 0x7FFFFFFFu;
    if (u >= 0x7F800000u) { *fl = FP8_FLAG_NONFINITE; return 0; }
    if (u == 0u) { *fl = FP8_FLAG_ZERO; return 0; }
    *fl = 0u;
    int e = (int)(u >> 23);
    uint32_t mant = u & 0x7FFFFFu;
    int ea;
    if (e == 0) {  // subnormal amax: normalise the mantissa
        const int p = 31 - __builtin_clz(mant);
        ea = p - 149;
        mant = (mant << (23 - p)) & 0x7FFFFFu;
    } else {
        ea = e - 127;
    }
    const int b = Fmt<FMT>::kMaxExp - ea - (mant > Fmt<FMT>::kMantMax ? 1 : 0);
    return b - margin;
}

// ---------------------------------------------------------------- amax
// The amax of a tensor holding a NaN is NaN; its fp32 pattern is the canonical
// quiet NaN 0x7FC00000 whatever the payloads of the input NaNs.  Mapping every
// contribution before it is folded into a maximum keeps the fold exact: the
// canonical NaN pattern exceeds every finite or infinite magnitude pattern.
__device__ __forceinline__ uint32_t canon_amax(uint32_t a32) {
    return a32 > 0x7F800000u ? 0x7FC00000u : a32;
}

typedef unsigned short us2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, 64));
    return v;
}

__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* red) {
    v = wave_max(v);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) red[w] = v;
    __syncthreads();
    uint32_t r = 0;
    if (threadIdx.x == 0) {
        for (int i = 0; i < (int)(blockDim.x >> 6); ++i) r = max(r, red[i]);
    }
    return r;  // valid in thread 0
}

// Largest of p[threadIdx.x], p[threadIdx.x + NT], ... below n (this thread's
// share of a block-wide maximum over n words), eight independent loads at a
// time: a plain strided loop waits for each load before issuing the next.
template <int NT>
__device__ __forceinline__ uint32_t strided_max(const uint32_t* __restrict__ p, int n) {
    uint32_t m = 0;
    int i = threadIdx.x;
    for (; i + 7 * NT < n; i += 8 * NT) {
        uint32_t v[8];
#pragma unroll
        for (int l = 0; l < 8; ++l) v[l] = p[i + l * NT];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int l = 0; l < 8; ++l) m = max(m, v[l]);
    }
    // the rest: unconditional loads of in-range words (a guarded load compiles
    // to a branch and a wait per load), masked afterwards
    if (n > 0) {
        uint32_t v[8];
#pragma unroll
        for (int l = 0; l < 8; ++l) v[l] = p[min(i + l * NT, n - 1)];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int l = 0; l < 8; ++l) m = max(m, i + l * NT < n ? v[l] : 0u);
    }
    return m;
}

__device__ __forceinline__ us2 fold_bf16(us2 m, uint4 v) {
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.x & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.y & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.z & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.w & 0x7FFF7FFFu));
    return m;
}

__device__ __forceinline__ uint32_t fold_f32(uint32_t m, uint4 v) {
    m = max(m, v.x & 0x7FFFFFFFu);
    m = max(m, v.y & 0x7FFFFFFFu);
    m = max(m, v.z & 0x7FFFFFFFu);
    m = max(m, v.w & 0x7FFFFFFFu);
    return m;
}

// Sign-cleared pattern of element i (bf16: 16-bit pattern; fp32: 31 bits).
template <int DT>
__device__ __forceinline__ uint32_t elem_mag(const void* x, int64_t i) {
    if (DT == FP8_DT_BF16) return ((const uint16_t*)x)[i] & 0x7FFFu;
    return ((const uint32_t*)x)[i] & 0x7FFFFFFFu;
}

// ---------------------------------------------------------------- cast
// Two scaled, clipped values -> two codes in the low (HI = false) or high
// half of `old`, by the hardware converter of the format's OCP counterpart.
template <int FMT, bool HI>
__device__ __forceinline__ uint32_t cvt2(float a, float b, uint32_t old) {
    if (Fmt<FMT>::kHw == FP8_E4M3) return __builtin_amdgcn_cvt_pk_fp8_f32(a, b, old, HI);
    return __builtin_amdgcn_cvt_pk_bf8_f32(a, b, old, HI);
}

// x * 2^(b + kShift): exact (a power-of-two scale).
template <int FMT>
__device__ __forceinline__ float scaled(float f, int b) { return ldexpf(f, b + Fmt<FMT>::kShift); }

// Clip to the OCP maximum before the hardware conversion (App. A: overflow
// clips to the maximum, infinities included).
template <int FMT>
__device__ __forceinline__ float clip(float y) {
    return __builtin_amdgcn_fmed3f(y, -Fmt<FMT>::kMax, Fmt<FMT>::kMax);
}

// (a) formats, |y| (scaled by 2^(b+1)) above the OCP maximum: magnitude code
// among the (a) codes beyond it, to nearest with ties to the even mantissa,
// clipping at the (a) maximum.  E4: 0x7E = 448 and 0x7F = 480 in these units.
// E5: 0x7B = 57344, 0x7C..0x7F = 65536, 81920, 98304, 114688.
template <int FMT>
__device__ __forceinline__ uint32_t top_code(float a) {
    if (FMT == FP8_E4_A) return a > 464.0f ? 0x7Fu : 0x7Eu;
    return a < 61440.0f ? 0x7Bu : a <= 73728.0f ? 0x7Cu : a < 90112.0f ? 0x7Du : a <= 106496.0f ? 0x7Eu : 0x7Fu;
}

// (a) formats: fix-ups of four hardware codes for the scaled values y[4]
// (before the NaN patch): -0 (0x80) becomes 0x00, values beyond the OCP
// maximum get their (a) code.  OCP formats: unchanged.
template <int FMT>
__device__ __forceinline__ uint32_t paper_fix(uint32_t c, const float y[4]) {
    if (!Fmt<FMT>::kPaper) return c;
    const uint32_t v = c ^ 0x80808080u;  // bytes that were 0x80 are now 0
    const uint32_t z = ~(((v & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | v) & 0x80808080u;
    c &= ~((z >> 7) * 0xFFu);
    const float m = fmaxf(fmaxf(fabsf(y[0]), fabsf(y[1])), fmaxf(fabsf(y[2]), fabsf(y[3])));
    if (__builtin_expect(m > Fmt<FMT>::kMax, 0)) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = fabsf(y[e]);
            if (a > Fmt<FMT>::kMax)
                c = (c & ~(0xFFu << (8 * e))) | ((top_code<FMT>(a) | (y[e] < 0.0f ? 0x80u : 0u)) << (8 * e));
        }
    }
    return c;
}

// Four scaled values -> four codes, before the NaN patch.
template <int FMT>
__device__ __forceinline__ uint32_t cast4(const float y[4]) {
    const uint32_t c = cvt2<FMT, false>(clip<FMT>(y[0]), clip<FMT>(y[1]), 0u);
    return paper_fix<FMT>(cvt2<FMT, true>(clip<FMT>(y[2]), clip<FMT>(y[3]), c), y);
}

// Four bf16 values (two packed words) -> four codes, before the NaN patch.
template <int FMT>
__device__ __forceinline__ uint32_t cast4_bf16(uint32_t w0, uint32_t w1, int b) {
    const float y[4] = {scaled<FMT>(__uint_as_float(w0 << 16), b), scaled<FMT>(__uint_as_float(w0 & 0xFFFF0000u), b),
                        scaled<FMT>(__uint_as_float(w1 << 16), b), scaled<FMT>(__uint_as_float(w1 & 0xFFFF0000u), b)};
    return cast4<FMT>(y);
}

template <int FMT>
__device__ __forceinline__ uint32_t cast4_f32(uint4 v, int b) {
    const float y[4] = {scaled<FMT>(__uint_as_float(v.x), b), scaled<FMT>(__uint_as_float(v.y), b),
                        scaled<FMT>(__uint_as_float(v.z), b), scaled<FMT>(__uint_as_float(v.w), b)};
    return cast4<FMT>(y);
}

// NaN code: 0x7F with the input's sign (OCP), 0x80 (the paper's formats).
template <int FMT>
__device__ __forceinline__ uint32_t nan_code(uint32_t key) {
    return Fmt<FMT>::kPaper ? 0x80u : (0x7Fu | ((key >> 8) & 0x80u));
}

// Re-encode NaN inputs.  hs[e] is input e as a bf16 pattern or as the top
// half of an fp32 pattern with the low half folded into bit 0 (only the NaN
// test reads it).
template <int FMT>
__device__ __forceinline__ uint32_t nan_patch(uint32_t c, const uint32_t hs[4]) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if ((hs[e] & 0x7FFFu) > 0x7F80u) c = (c & ~(0xFFu << (8 * e))) | (nan_code<FMT>(hs[e]) << (8 * e));
    return c;
}

// Packed test: does one of the four bf16 values in w0, w1 have a NaN pattern?
__device__ __forceinline__ bool any_nan_bf16(uint32_t w0, uint32_t w1) {
    return ((((w0 & 0x7FFF7FFFu) + 0x007F007Fu) | ((w1 & 0x7FFF7FFFu) + 0x007F007Fu)) & 0x80008000u) != 0u;
}

__device__ __forceinline__ uint32_t f32_key(uint32_t u) {  // fp32 pattern -> NaN-test key
    return (u >> 16) | ((u & 0xFFFFu) ? 1u : 0u);
}

template <int DT, int FMT>
__device__ __forceinline__ uint32_t cast1(const void* x, int64_t idx, int b) {
    uint32_t key;
    float f;
    if (DT == FP8_DT_BF16) {
        key = ((const uint16_t*)x)[idx];
        f = __uint_as_float(key << 16);
    } else {
        const uint32_t u = ((const uint32_t*)x)[idx];
        key = f32_key(u);
        f = __uint_as_float(u);
    }
    const float y[4] = {scaled<FMT>(f, b), 0.0f, 0.0f, 0.0f};
    uint32_t c = cast4<FMT>(y) & 0xFFu;
    if ((key & 0x7FFFu) > 0x7F80u) c = nan_code<FMT>(key);
    return c;
}

// 16-byte load of input data read once per pass, with the non-temporal hint
// (streaming reads from HBM run about 7-10 % faster with it).
__device__ __forceinline__ uint4 ld_stream(const void* p) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Two fp32 -> two bf16 (round to nearest even, v_cvt_pk_bf16_f32) in one word.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// Biases beyond this saturate or flush every input; casts clamp to it.
__device__ __forceinline__ int clamp_bias(int32_t b) { return max(-kBiasClamp, min(kBiasClamp, b)); }

}  // namespace
}  // namespace fp8lin
