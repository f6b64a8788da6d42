// Per-tensor amax, scaling bias (Sec. 2.3 Eq. 3) and scale-and-cast to FP8
// (Sec. 2.1 Eq. 1) for gfx950.
//
// amax: the absolute maximum is taken as the integer maximum of the
// sign-cleared bit patterns.  For finite values the order of the patterns is
// the order of the magnitudes, NaN patterns sort above infinity, and -0
// clears to 0, so the result is exact and independent of the reduction order.
// Pass 1 reduces to one partial per workgroup (coalesced 16-byte loads, packed
// 16-bit max for bf16); pass 2 (one workgroup) reduces the partials and turns
// the amax into the bias with integer arithmetic.
//
// cast: x * 2^b is formed exactly on the exponent field (no floating-point
// multiply), then rounded to the FP8 grid with round-to-nearest-even in
// integer arithmetic and clipped to the largest finite code.  The optional
// transposed copy goes through a 128 x 64 byte LDS tile so that both outputs
// are written with wide, coalesced stores.
#include "fp8lin_internal.h"

namespace fp8lin {
namespace {

// ---------------------------------------------------------------- formats
// OCP FP8 (Table 7 rows "(b)").  kM: mantissa bits, kEmin: exponent of the
// smallest normal, kMaxCode: code of the largest finite value.
template <int FMT> struct Fmt;
template <> struct Fmt<FP8_E4M3> {
    static constexpr int kM = 3, kEmin = -6, kMaxCode = 0x7E;
    static constexpr int kMaxExp = 8;  // max finite = 1.75 * 2^8 = 448
};
template <> struct Fmt<FP8_E5M2> {
    static constexpr int kM = 2, kEmin = -14, kMaxCode = 0x7B;
    static constexpr int kMaxExp = 15;  // max finite = 1.75 * 2^15 = 57344
};

constexpr int kBiasClamp = 512;  // beyond this every input saturates or flushes

// Encode |value| = sig * 2^(E - (kSig - 1)), sig in [2^(kSig-1), 2^kSig), into the
// magnitude bits of an FP8 code, rounding to nearest even and clipping.
//   Ec = max(E, kEmin) is the exponent whose quantum 2^(Ec - kM) applies;
//   n  = round(|value| / 2^(Ec - kM)); code = ((Ec - kEmin) << kM) + n.
// A round-up that reaches 2^(kM+1) carries into the next binade by itself.
template <int FMT, int kSig>
__device__ __forceinline__ uint32_t encode_mag(uint32_t sig, int E) {
    using F = Fmt<FMT>;
    const int Ec = max(E, F::kEmin);
    const int sh = min((kSig - 1 - F::kM) + (Ec - E), kSig + 2);
    const uint32_t n = (sig + (1u << (sh - 1)) - 1u + ((sig >> sh) & 1u)) >> sh;
    const int code = ((Ec - F::kEmin) << F::kM) + (int)n;
    return (uint32_t)min(code, F::kMaxCode);
}

// bf16 bit pattern (low 16 bits of h) scaled by 2^b -> FP8 code.
template <int FMT>
__device__ __forceinline__ uint32_t enc_bf16(uint32_t h, int b) {
    const uint32_t s = (h >> 8) & 0x80u;
    const uint32_t a = h & 0x7FFFu;
    const int e = (int)(a >> 7);
    const uint32_t m = a & 0x7Fu;
    const int p = 31 - __builtin_clz(m | 1u);          // top bit of a subnormal mantissa
    const bool sub = (e == 0);
    const int E = (sub ? p - 133 : e - 127) + b;
    const uint32_t sig = sub ? (m << (7 - p)) : (m | 0x80u);
    uint32_t c = encode_mag<FMT, 8>(sig, E);
    c = (a == 0u) ? 0u : c;
    c = (a >= 0x7F80u) ? ((a == 0x7F80u) ? (uint32_t)Fmt<FMT>::kMaxCode : 0x7Fu) : c;
    return c | s;
}

// fp32 bit pattern scaled by 2^b -> FP8 code.
template <int FMT>
__device__ __forceinline__ uint32_t enc_f32(uint32_t u, int b) {
    const uint32_t s = (u >> 24) & 0x80u;
    const uint32_t a = u & 0x7FFFFFFFu;
    const int e = (int)(a >> 23);
    const uint32_t m = a & 0x7FFFFFu;
    const int p = 31 - __builtin_clz(m | 1u);
    const bool sub = (e == 0);
    const int E = (sub ? p - 149 : e - 127) + b;
    const uint32_t sig = sub ? (m << (23 - p)) : (m | 0x800000u);
    uint32_t c = encode_mag<FMT, 24>(sig, E);
    c = (a == 0u) ? 0u : c;
    c = (a >= 0x7F800000u) ? ((a == 0x7F800000u) ? (uint32_t)Fmt<FMT>::kMaxCode : 0x7Fu) : c;
    return c | s;
}

// Eq. 3 on the fp32 bit pattern of the amax: with amax = 1.f_a * 2^ea and
// max_num = 1.75 * 2^eM, floor(log2(max_num / amax)) = eM - ea - [1.f_a > 1.75].
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
    const int b = Fmt<FMT>::kMaxExp - ea - (mant > 0x600000u ? 1 : 0);
    return b - margin;
}

// ---------------------------------------------------------------- amax
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

template <int DT>
__global__ __launch_bounds__(kAmaxThreads) void amax_partial_kernel(const void* __restrict__ x,
                                                                   int64_t n, int vec,
                                                                   uint32_t* __restrict__ partial) {
    __shared__ uint32_t red[kAmaxThreads / 64];
    const int64_t tid = (int64_t)blockIdx.x * kAmaxThreads + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * kAmaxThreads;
    uint32_t m = 0;
    int64_t tail0 = 0;
    if (vec) {
        constexpr int per = DT == FP8_DT_BF16 ? 8 : 4;
        const uint4* __restrict__ p = (const uint4*)x;
        const int64_t nv = n / per;
        tail0 = nv * per;
        int64_t i = tid;
        if (DT == FP8_DT_BF16) {
            us2 mm = {0, 0};
            for (; i + 3 * nth < nv; i += 4 * nth) {
                const uint4 a = p[i], b = p[i + nth], c = p[i + 2 * nth], d = p[i + 3 * nth];
                mm = fold_bf16(mm, a);
                mm = fold_bf16(mm, b);
                mm = fold_bf16(mm, c);
                mm = fold_bf16(mm, d);
            }
            for (; i < nv; i += nth) mm = fold_bf16(mm, p[i]);
            m = max((uint32_t)mm.x, (uint32_t)mm.y);
        } else {
            for (; i + 3 * nth < nv; i += 4 * nth) {
                const uint4 a = p[i], b = p[i + nth], c = p[i + 2 * nth], d = p[i + 3 * nth];
                m = fold_f32(m, a);
                m = fold_f32(m, b);
                m = fold_f32(m, c);
                m = fold_f32(m, d);
            }
            for (; i < nv; i += nth) m = fold_f32(m, p[i]);
        }
    }
    for (int64_t j = tail0 + tid; j < n; j += nth) m = max(m, elem_mag<DT>(x, j));
    m = block_max(m, red);
    if (threadIdx.x == 0) partial[blockIdx.x] = m;
}

template <int DT, int FMT>
__global__ __launch_bounds__(kAmaxThreads) void amax_finalize_kernel(
    const uint32_t* __restrict__ partial, int nparts, int32_t margin, int32_t* __restrict__ bias,
    uint32_t* __restrict__ amax_bits, uint32_t* __restrict__ flags) {
    __shared__ uint32_t red[kAmaxThreads / 64];
    uint32_t m = 0;
    for (int i = threadIdx.x; i < nparts; i += kAmaxThreads) m = max(m, partial[i]);
    m = block_max(m, red);
    if (threadIdx.x == 0) {
        const uint32_t a32 = DT == FP8_DT_BF16 ? (m << 16) : m;
        uint32_t fl;
        const int32_t b = bias_of<FMT>(a32, margin, &fl);
        *bias = b;
        if (amax_bits) *amax_bits = a32;
        if (flags) *flags = fl;
    }
}

template <int FMT>
__global__ void bias_from_amax_kernel(const uint32_t* __restrict__ amax_bits, int32_t margin,
                                      int32_t* __restrict__ bias, uint32_t* __restrict__ flags) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        uint32_t fl;
        *bias = bias_of<FMT>(*amax_bits, margin, &fl);
        if (flags) *flags = fl;
    }
}

// ---------------------------------------------------------------- cast
// Workgroup tile: 64 rows x 128 columns, 256 threads.  Lane l of wave w owns
// rows r0 .. r0+3 (r0 = 16 w + 4 (l / 16)) and columns c0 .. c0+7
// (c0 = 8 (l % 16)): each of its four row loads is one 16-byte (bf16) or two
// 16-byte (fp32) accesses, and 16 lanes cover 256 contiguous bytes of a row.
constexpr int kCastRows = 64, kCastCols = 128, kCastThreads = 256;

// Byte j of a 32-bit word.
__device__ __forceinline__ uint32_t byte_of(uint32_t w, int j) { return (w >> (8 * j)) & 0xFFu; }

template <int DT, int FMT>
__global__ __launch_bounds__(kCastThreads) void cast_kernel(
    const void* __restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    const int32_t* __restrict__ bias_p, uint8_t* __restrict__ q, int64_t ldq,
    uint8_t* __restrict__ qT, int64_t ldqT, int64_t tiles_c, int vec_in, int vec_q, int vec_qT) {
    // Transposed tile: 128 columns x 64 rows of codes; the 16-byte row chunk
    // index is XOR-swizzled with the column block to spread LDS banks.
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int chunk = lane & 15, g = lane >> 4;
    const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x % tiles_c;
    const int64_t R0 = tr * kCastRows, C0 = tc * kCastCols;
    const int lr = w * 16 + g * 4, lc = chunk * 8;  // local row / column of this lane
    const int64_t r0 = R0 + lr, c0 = C0 + lc;
    const int b = max(-kBiasClamp, min(kBiasClamp, *bias_p));

    uint32_t lo[4], hi[4];  // codes of columns c0..c0+3 and c0+4..c0+7, per row
    const bool full = vec_in && (r0 + 4 <= rows) && (c0 + 8 <= cols);
    if (full) {
        if (DT == FP8_DT_BF16) {
            uint4 v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                v[i] = *(const uint4*)((const uint16_t*)x + (r0 + i) * ldx + c0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t e0 = enc_bf16<FMT>(v[i].x & 0xFFFFu, b), e1 = enc_bf16<FMT>(v[i].x >> 16, b);
                const uint32_t e2 = enc_bf16<FMT>(v[i].y & 0xFFFFu, b), e3 = enc_bf16<FMT>(v[i].y >> 16, b);
                const uint32_t e4 = enc_bf16<FMT>(v[i].z & 0xFFFFu, b), e5 = enc_bf16<FMT>(v[i].z >> 16, b);
                const uint32_t e6 = enc_bf16<FMT>(v[i].w & 0xFFFFu, b), e7 = enc_bf16<FMT>(v[i].w >> 16, b);
                lo[i] = e0 | (e1 << 8) | (e2 << 16) | (e3 << 24);
                hi[i] = e4 | (e5 << 8) | (e6 << 16) | (e7 << 24);
            }
        } else {
            uint4 v[4][2];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint4* p = (const uint4*)((const uint32_t*)x + (r0 + i) * ldx + c0);
                v[i][0] = p[0];
                v[i][1] = p[1];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                lo[i] = enc_f32<FMT>(v[i][0].x, b) | (enc_f32<FMT>(v[i][0].y, b) << 8) |
                        (enc_f32<FMT>(v[i][0].z, b) << 16) | (enc_f32<FMT>(v[i][0].w, b) << 24);
                hi[i] = enc_f32<FMT>(v[i][1].x, b) | (enc_f32<FMT>(v[i][1].y, b) << 8) |
                        (enc_f32<FMT>(v[i][1].z, b) << 16) | (enc_f32<FMT>(v[i][1].w, b) << 24);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t wlo = 0, whi = 0;
            for (int j = 0; j < 8; ++j) {
                const int64_t r = r0 + i, c = c0 + j;
                uint32_t code = 0;
                if (r < rows && c < cols) {
                    if (DT == FP8_DT_BF16)
                        code = enc_bf16<FMT>(((const uint16_t*)x)[r * ldx + c], b);
                    else
                        code = enc_f32<FMT>(((const uint32_t*)x)[r * ldx + c], b);
                }
                if (j < 4) wlo |= code << (8 * j); else whi |= code << (8 * (j - 4));
            }
            lo[i] = wlo;
            hi[i] = whi;
        }
    }

    if (q) {
        if (full && vec_q) {
#pragma unroll
            for (int i = 0; i < 4; ++i) *(uint2*)(q + (r0 + i) * ldq + c0) = make_uint2(lo[i], hi[i]);
        } else {
            for (int i = 0; i < 4; ++i)
                for (int j = 0; j < 8; ++j) {
                    const int64_t r = r0 + i, c = c0 + j;
                    if (r < rows && c < cols)
                        q[r * ldq + c] = (uint8_t)byte_of(j < 4 ? lo[i] : hi[i], j & 3);
                }
        }
    }

    if (qT) {
        // Column j of this lane's 4x8 block, rows r0..r0+3, as one word.
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t* src = j < 4 ? lo : hi;
            const int jj = j & 3;
            const uint32_t col = byte_of(src[0], jj) | (byte_of(src[1], jj) << 8) |
                                 (byte_of(src[2], jj) << 16) | (byte_of(src[3], jj) << 24);
            const int cl = lc + j;
            const int off = cl * kCastRows + (((w ^ (cl >> 3)) & 3) << 4) + g * 4;
            *(uint32_t*)(tile + off) = col;
        }
        __syncthreads();
        // 128 transposed rows x 4 chunks of 16 bytes = 512 chunks, two per thread.
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = threadIdx.x + h * kCastThreads;
            const int cl = idx >> 2, qq = idx & 3;
            const int64_t c = C0 + cl;
            const int64_t rr = R0 + qq * 16;
            if (c >= cols || rr >= rows) continue;
            const uint4 v = *(const uint4*)(tile + cl * kCastRows + (((qq ^ (cl >> 3)) & 3) << 4));
            uint8_t* dst = qT + c * ldqT + rr;
            if (vec_qT && rr + 16 <= rows) {
                *(uint4*)dst = v;
            } else {
                const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
                for (int t = 0; t < 16 && rr + t < rows; ++t) dst[t] = (uint8_t)byte_of(wv[t >> 2], t & 3);
            }
        }
    }
}

template <int DT, int FMT>
void launch_cast_t(const void* x, int64_t rows, int64_t cols, int64_t ldx, const int32_t* bias,
                   uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT, hipStream_t s) {
    const int64_t tiles_r = (rows + kCastRows - 1) / kCastRows;
    const int64_t tiles_c = (cols + kCastCols - 1) / kCastCols;
    const int esz = DT == FP8_DT_BF16 ? 2 : 4;
    const int vec_in = ((uintptr_t)x % 16 == 0) && ((ldx * esz) % 16 == 0);
    const int vec_q = q && ((uintptr_t)q % 8 == 0) && (ldq % 8 == 0);
    const int vec_qT = qT && ((uintptr_t)qT % 16 == 0) && (ldqT % 16 == 0);
    hipLaunchKernelGGL((cast_kernel<DT, FMT>), dim3((unsigned)(tiles_r * tiles_c)), dim3(kCastThreads), 0,
                       s, x, rows, cols, ldx, bias, q, ldq, qT, ldqT, tiles_c, vec_in, vec_q, vec_qT);
}

}  // namespace

int amax_blocks(int64_t n) {
    const int64_t per_block = (int64_t)kAmaxThreads * 8 * 4;  // 4 vectors of 8 bf16 per thread
    int64_t nb = (n + per_block - 1) / per_block;
    if (nb < 1) nb = 1;
    if (nb > kAmaxMaxBlocks) nb = kAmaxMaxBlocks;
    return (int)nb;
}

int32_t launch_scale_bias(const void* x, int dt, int64_t n, int fmt, int32_t margin, int32_t* bias,
                          uint32_t* amax_bits, uint32_t* flags, uint32_t* partials, hipStream_t s) {
    // n == 0: no partials; the finalize pass sees an amax of 0.
    const int nb = n > 0 ? amax_blocks(n) : 0;
    const int vec = ((uintptr_t)x % 16 == 0) ? 1 : 0;
    if (nb > 0 && dt == FP8_DT_BF16)
        hipLaunchKernelGGL(amax_partial_kernel<FP8_DT_BF16>, dim3(nb), dim3(kAmaxThreads), 0, s, x, n, vec, partials);
    else if (nb > 0)
        hipLaunchKernelGGL(amax_partial_kernel<FP8_DT_F32>, dim3(nb), dim3(kAmaxThreads), 0, s, x, n, vec, partials);
    if (dt == FP8_DT_BF16 && fmt == FP8_E4M3)
        hipLaunchKernelGGL((amax_finalize_kernel<FP8_DT_BF16, FP8_E4M3>), dim3(1), dim3(kAmaxThreads), 0, s, partials, nb, margin, bias, amax_bits, flags);
    else if (dt == FP8_DT_BF16)
        hipLaunchKernelGGL((amax_finalize_kernel<FP8_DT_BF16, FP8_E5M2>), dim3(1), dim3(kAmaxThreads), 0, s, partials, nb, margin, bias, amax_bits, flags);
    else if (fmt == FP8_E4M3)
        hipLaunchKernelGGL((amax_finalize_kernel<FP8_DT_F32, FP8_E4M3>), dim3(1), dim3(kAmaxThreads), 0, s, partials, nb, margin, bias, amax_bits, flags);
    else
        hipLaunchKernelGGL((amax_finalize_kernel<FP8_DT_F32, FP8_E5M2>), dim3(1), dim3(kAmaxThreads), 0, s, partials, nb, margin, bias, amax_bits, flags);
    return hip_status();
}

int32_t launch_bias_from_amax(const uint32_t* amax_bits, int fmt, int32_t margin, int32_t* bias,
                              uint32_t* flags, hipStream_t s) {
    if (fmt == FP8_E4M3)
        hipLaunchKernelGGL(bias_from_amax_kernel<FP8_E4M3>, dim3(1), dim3(64), 0, s, amax_bits, margin, bias, flags);
    else
        hipLaunchKernelGGL(bias_from_amax_kernel<FP8_E5M2>, dim3(1), dim3(64), 0, s, amax_bits, margin, bias, flags);
    return hip_status();
}

int32_t launch_cast(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                    const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                    hipStream_t s) {
    if (dt == FP8_DT_BF16 && fmt == FP8_E4M3)
        launch_cast_t<FP8_DT_BF16, FP8_E4M3>(x, rows, cols, ldx, bias, q, ldq, qT, ldqT, s);
    else if (dt == FP8_DT_BF16)
        launch_cast_t<FP8_DT_BF16, FP8_E5M2>(x, rows, cols, ldx, bias, q, ldq, qT, ldqT, s);
    else if (fmt == FP8_E4M3)
        launch_cast_t<FP8_DT_F32, FP8_E4M3>(x, rows, cols, ldx, bias, q, ldq, qT, ldqT, s);
    else
        launch_cast_t<FP8_DT_F32, FP8_E5M2>(x, rows, cols, ldx, bias, q, ldq, qT, ldqT, s);
    return hip_status();
}

}  // namespace fp8lin
