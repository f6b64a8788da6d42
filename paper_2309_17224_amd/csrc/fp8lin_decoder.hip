// The higher-precision layers of the Llama 2 decoder layer around its four
// FP8 linears (App. E: the QKV projection, the attention output projection
// and the two feed-forward layers are FP8; everything else stays in higher
// precision): RMSNorm with the residual add, rotary embeddings, causal
// grouped-query attention, SwiGLU, and the residual add, for gfx950, in bf16
// with fp32 arithmetic.
//
// Where an FP8 linear consumes a tensor (the outputs of the two RMSNorms, of
// the attention and of SwiGLU), its FP8-AMAX quantise (Sec. 2.3 Eq. 3 bias,
// Sec. 2.1 Eq. 1 cast) is fused into the kernel that produces it: that kernel
// casts its bf16 output with a predicted bias (the previous call's) and writes
// its workgroup maxima; the check kernel of fp8_quantise then computes the
// exact bias from the maxima and re-casts from the bf16 output only if the
// prediction was wrong.  The codes are therefore always those of the exact
// bias (Sec. 3: the amax needs a pass over the tensor before any element can
// be cast; the producer takes it while the tensor is still in registers).
//
// Every output is rounded once to bf16, to nearest even.
#include "fp8lin_fp8.h"
#include "fp8lin_internal.h"

using namespace fp8lin;

namespace {

constexpr int kThreads = 256;
constexpr int kGluePartsMax = 2048;          // workgroups of the grid-stride glue kernels
constexpr int32_t kNoPrediction = INT32_MIN;  // never equal to a clamped bias

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint4 ld16(const void* p) { return *(const uint4*)p; }
__device__ __forceinline__ void st16(void* p, uint4 v) { *(uint4*)p = v; }

// Eight bf16 values (four packed words) -> eight codes with bias b; NaN
// inputs are re-encoded as the casts do.
template <int FMT>
__device__ __forceinline__ uint2 codes8(uint4 v, int b) {
    uint32_t lo = cast4_bf16<FMT>(v.x, v.y, b), hi = cast4_bf16<FMT>(v.z, v.w, b);
    if (__builtin_expect(any_nan_bf16(v.x, v.y) || any_nan_bf16(v.z, v.w), 0)) {
        const uint32_t h0[4] = {v.x & 0xFFFFu, v.x >> 16, v.y & 0xFFFFu, v.y >> 16};
        const uint32_t h1[4] = {v.z & 0xFFFFu, v.z >> 16, v.w & 0xFFFFu, v.w >> 16};
        lo = nan_patch<FMT>(lo, h0);
        hi = nan_patch<FMT>(hi, h1);
    }
    return make_uint2(lo, hi);
}

// Largest magnitude pattern of eight bf16 values.
__device__ __forceinline__ uint32_t mag8(uint4 v) {
    us2 m = {0, 0};
    m = fold_bf16(m, v);
    return max((uint32_t)m.x, (uint32_t)m.y);
}

// The bias the fused cast uses: the prediction, clamped as the casts clamp.
// Block 0 records it for the check kernel (kNoPrediction without one, which
// makes the check kernel cast every element).
__device__ __forceinline__ int fused_bias(const int32_t* pred, int32_t* used) {
    const int b = pred ? clamp_bias(*pred) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *used = pred ? b : kNoPrediction;
    return b;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// ------------------------------------------------------------- residual add
// out = round(a + b).  The fp32 sum of two bf16 values is exact unless their
// exponents differ by more than 16, and then the smaller is far below half a
// bf16 quantum of the larger: the result is the correctly rounded sum.
__device__ __forceinline__ uint4 add8(uint4 a, uint4 b) {
    uint4 r;
    r.x = pack_bf16x2(lo_f(a.x) + lo_f(b.x), hi_f(a.x) + hi_f(b.x));
    r.y = pack_bf16x2(lo_f(a.y) + lo_f(b.y), hi_f(a.y) + hi_f(b.y));
    r.z = pack_bf16x2(lo_f(a.z) + lo_f(b.z), hi_f(a.z) + hi_f(b.z));
    r.w = pack_bf16x2(lo_f(a.w) + lo_f(b.w), hi_f(a.w) + hi_f(b.w));
    return r;
}

__global__ __launch_bounds__(kThreads) void add_kernel(const uint16_t* __restrict__ a, const uint16_t* __restrict__ b,
                                                       uint16_t* __restrict__ out, int64_t n8) {
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n8; i += (int64_t)gridDim.x * kThreads)
        st16(out + 8 * i, add8(ld_stream(a + 8 * i), ld_stream(b + 8 * i)));
}

// ------------------------------------------------------------- RMSNorm
// One workgroup per row.  h = x (+ res), rounded; y = h / sqrt(mean(h^2) + eps)
// * g.  The sum of squares is taken in fp32 in a fixed order (each lane its
// elements in order, then a fixed reduction tree).  Rows of up to
// 8 x 8 x kThreads columns are held in registers (all loads issued at once,
// one read of the row); longer rows are read twice, the second time from L2.
template <bool RES>
__device__ __forceinline__ uint4 row_h8(const uint16_t* x, const uint16_t* res) {
    const uint4 v = ld16(x);
    return RES ? add8(v, ld16(res)) : v;
}

__device__ __forceinline__ float sumsq8(uint4 v, float s) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float a = lo_f(w[k]), b = hi_f(w[k]);
        s += a * a;
        s += b * b;
    }
    return s;
}

// CH: 16-byte chunks of the row each lane holds in registers (4 for rows of
// up to 8192 columns, so that more workgroups fit on a compute unit; 8 up to
// 16384).
template <bool RES, bool QUANT, int FMT, int CH>
__global__ __launch_bounds__(kThreads) void rmsnorm_kernel(
    const uint16_t* __restrict__ x, int64_t ldx, const uint16_t* __restrict__ res, int64_t ldr,
    const uint16_t* __restrict__ g, int64_t cols, float eps, uint16_t* __restrict__ h, int64_t ldh,
    uint16_t* __restrict__ y, int64_t ldy, const int32_t* __restrict__ pred, int32_t* __restrict__ used,
    uint32_t* __restrict__ parts, uint8_t* __restrict__ q, int64_t ldq) {
    __shared__ float red[kThreads / 64];
    __shared__ uint32_t redm[kThreads / 64];
    const int64_t r = blockIdx.x;
    const uint16_t* xr = x + r * ldx;
    const uint16_t* rr = RES ? res + r * ldr : nullptr;
    constexpr int kChunks = CH;
    const bool in_regs = cols <= (int64_t)8 * kThreads * kChunks;
    uint4 hr[kChunks], gr[kChunks];
    float ss = 0.0f;
    if (in_regs) {
        // unconditional loads (the last chunk of the row is in bounds: cols is
        // a nonzero multiple of 8), chunks past the end zeroed afterwards
#pragma unroll
        for (int k = 0; k < kChunks; ++k) {
            const int64_t c = min((int64_t)8 * (threadIdx.x + kThreads * k), cols - 8);
            hr[k] = row_h8<RES>(xr + c, rr + c);
        }
#pragma unroll
        for (int k = 0; k < kChunks; ++k) gr[k] = ld16(g + min((int64_t)8 * (threadIdx.x + kThreads * k), cols - 8));
#pragma unroll
        for (int k = 0; k < kChunks; ++k) {
            if (8 * (threadIdx.x + kThreads * k) >= cols) hr[k] = make_uint4(0u, 0u, 0u, 0u);
            ss = sumsq8(hr[k], ss);
        }
    } else {
        for (int64_t c = 8 * threadIdx.x; c < cols; c += 8 * kThreads) ss = sumsq8(row_h8<RES>(xr + c, rr + c), ss);
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float total = (red[0] + red[1]) + (red[2] + red[3]);
    const float rstd = 1.0f / sqrtf(total / (float)cols + eps);

    const bool cast = QUANT && pred;
    const int b = QUANT ? fused_bias(pred, used) : 0;
    uint32_t mag = 0;
#pragma unroll
    for (int k = 0; k < kChunks; ++k) {
        const int64_t c = (int64_t)8 * (threadIdx.x + kThreads * k);
        if (!in_regs || c >= cols) break;
        const uint4 hv = hr[k], gv = gr[k];
        if (h) st16(h + r * ldh + c, hv);
        uint4 yv;
        yv.x = pack_bf16x2(lo_f(hv.x) * rstd * lo_f(gv.x), hi_f(hv.x) * rstd * hi_f(gv.x));
        yv.y = pack_bf16x2(lo_f(hv.y) * rstd * lo_f(gv.y), hi_f(hv.y) * rstd * hi_f(gv.y));
        yv.z = pack_bf16x2(lo_f(hv.z) * rstd * lo_f(gv.z), hi_f(hv.z) * rstd * hi_f(gv.z));
        yv.w = pack_bf16x2(lo_f(hv.w) * rstd * lo_f(gv.w), hi_f(hv.w) * rstd * hi_f(gv.w));
        st16(y + r * ldy + c, yv);
        if (QUANT) {
            mag = max(mag, mag8(yv));
            if (cast) *(uint2*)(q + r * ldq + c) = codes8<FMT>(yv, b);
        }
    }
    for (int64_t c = 8 * threadIdx.x; !in_regs && c < cols; c += 8 * kThreads) {
        const uint4 hv = row_h8<RES>(xr + c, rr + c);
        if (h) st16(h + r * ldh + c, hv);
        const uint4 gv = ld16(g + c);
        uint4 yv;
        yv.x = pack_bf16x2(lo_f(hv.x) * rstd * lo_f(gv.x), hi_f(hv.x) * rstd * hi_f(gv.x));
        yv.y = pack_bf16x2(lo_f(hv.y) * rstd * lo_f(gv.y), hi_f(hv.y) * rstd * hi_f(gv.y));
        yv.z = pack_bf16x2(lo_f(hv.z) * rstd * lo_f(gv.z), hi_f(hv.z) * rstd * hi_f(gv.z));
        yv.w = pack_bf16x2(lo_f(hv.w) * rstd * lo_f(gv.w), hi_f(hv.w) * rstd * hi_f(gv.w));
        st16(y + r * ldy + c, yv);
        if (QUANT) {
            mag = max(mag, mag8(yv));
            if (cast) *(uint2*)(q + r * ldq + c) = codes8<FMT>(yv, b);
        }
    }
    if (QUANT) {
        const uint32_t bm = block_max(mag, redm);
        if (threadIdx.x == 0) parts[r] = bm;
    }
}

// ------------------------------------------------------------- rotary embedding
// Table of (cos, sin) of pos * theta^(-2i/d_head), evaluated in fp64 and
// rounded to fp32: [seq_len, d_head / 2].
__global__ void rope_table_kernel(int64_t seq_len, int half, double theta, float2* __restrict__ tab) {
    const int64_t n = seq_len * half;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = i / half;
        const int k = (int)(i % half);
        const double ang = (double)p * pow(theta, -(double)k / (double)half);
        double s, c;
        sincos(ang, &s, &c);
        tab[i] = make_float2((float)c, (float)s);
    }
}

// In place on nheads consecutive heads of d_head = 2 * half columns: element
// i < half of a head pairs with element i + half; row r is at position
// r mod seq_len.  Each lane rotates eight pairs.
__global__ __launch_bounds__(kThreads) void rope_kernel(uint16_t* __restrict__ x, int64_t rows, int64_t ld,
                                                        int nheads, int half, int64_t seq_len,
                                                        const float2* __restrict__ tab) {
    const int per_head = half / 8;
    const int64_t per_row = (int64_t)nheads * per_head;
    const int64_t n = rows * per_row;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
        const int64_t r = i / per_row;
        const int rem = (int)(i % per_row);
        const int hh = rem / per_head, k0 = (rem % per_head) * 8;
        uint16_t* p = x + r * ld + (int64_t)hh * 2 * half + k0;
        const uint4 a = ld16(p), b = ld16(p + half);
        const float2* t = tab + (r % seq_len) * half + k0;
        const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
        uint32_t o1[4], o2[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float2 t0 = t[2 * k], t1 = t[2 * k + 1];
            const float a0 = lo_f(aw[k]), a1 = hi_f(aw[k]), b0 = lo_f(bw[k]), b1 = hi_f(bw[k]);
            o1[k] = pack_bf16x2(a0 * t0.x - b0 * t0.y, a1 * t1.x - b1 * t1.y);
            o2[k] = pack_bf16x2(b0 * t0.x + a0 * t0.y, b1 * t1.x + a1 * t1.y);
        }
        st16(p, make_uint4(o1[0], o1[1], o1[2], o1[3]));
        st16(p + half, make_uint4(o2[0], o2[1], o2[2], o2[3]));
    }
}

// ------------------------------------------------------------- SwiGLU
// a = g * sigmoid(g) * u over the fused gate+up output (gate columns
// [0, ffn), up columns [ffn, 2 ffn)); grid-stride, eight outputs per lane.
template <bool QUANT, int FMT>
__global__ __launch_bounds__(kThreads) void swiglu_kernel(
    const uint16_t* __restrict__ gu, int64_t ldgu, int64_t rows, int64_t ffn, uint16_t* __restrict__ a,
    int64_t lda, const int32_t* __restrict__ pred, int32_t* __restrict__ used, uint32_t* __restrict__ parts,
    uint8_t* __restrict__ q, int64_t ldq) {
    __shared__ uint32_t redm[kThreads / 64];
    const bool cast = QUANT && pred;
    const int b = QUANT ? fused_bias(pred, used) : 0;
    const int64_t per_row = ffn / 8;
    const int64_t n = rows * per_row;
    uint32_t mag = 0;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
        const int64_t r = i / per_row, c = (i % per_row) * 8;
        const uint4 gv = ld_stream(gu + r * ldgu + c), uv = ld_stream(gu + r * ldgu + ffn + c);
        const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w}, uw[4] = {uv.x, uv.y, uv.z, uv.w};
        uint32_t ow[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float g0 = lo_f(gw[k]), g1 = hi_f(gw[k]);
            ow[k] = pack_bf16x2(g0 / (1.0f + expf(-g0)) * lo_f(uw[k]), g1 / (1.0f + expf(-g1)) * hi_f(uw[k]));
        }
        const uint4 av = make_uint4(ow[0], ow[1], ow[2], ow[3]);
        st16(a + r * lda + c, av);
        if (QUANT) {
            mag = max(mag, mag8(av));
            if (cast) *(uint2*)(q + r * ldq + c) = codes8<FMT>(av, b);
        }
    }
    if (QUANT) {
        const uint32_t bm = block_max(mag, redm);
        if (threadIdx.x == 0) parts[blockIdx.x] = bm;
    }
}

// ------------------------------------------------------------- attention
// Causal softmax attention for head dimension 128, one workgroup of 4 waves
// per (query head, sequence, block of 128 queries); wave w owns queries
// 32 w .. 32 w + 31 of the block as two tiles of 16.  Keys and values stream
// through LDS in blocks of 64 (double buffered; the next block's copies into
// LDS are issued before the current block's matrix work).  Everything runs on
// v_mfma_f32_16x16x32_bf16 in transposed form, so that no fragment needs a
// shuffle between the two products:
//   S^T = K . Q^T: A = key rows from LDS, B = query rows kept in registers;
//                  each lane holds S^T[4 keys][1 query] per 16 x 16 tile;
//   O^T += V^T . P^T: B = the probabilities straight from the S^T registers
//                  (keys 4g..4g+3 and 16+4g..16+4g+3 of a 32-key slice for
//                  lane group g), A = V^T fragments taken from the row-major
//                  LDS copy of V by gfx950's transposing LDS read
//                  (ds_read_b64_tr_b16), which hands each lane one column of
//                  four consecutive keys, in the key order of P.
// Online softmax in fp32 with base-2 exponentials (the scale log2(e) /
// sqrt(128) folded into the exponent's FMA); the exponent offset follows the
// running maximum lazily (moved only when it is exceeded by 8 in log2 units,
// so the probabilities stay below 256 and O is rarely rescaled); P is rounded
// to bf16 for the second product; the row sums are kept per lane and reduced
// once at the end.  A query row that sees no key of a block (above the
// diagonal) gets maximum -inf there, no rescale and zero weights.
constexpr int kHd = 128, kBq = 128, kBk = 64;
constexpr int kKvBytes = kBk * kHd * 2;  // one K or V block in LDS: 16 KiB

struct AttnArgs {
    const uint16_t* qkv;
    int64_t ld, rows, seq_len;
    int nh, nkv, nqb, nseq;
    float scale_log2;
    uint16_t* o;
    int64_t ldo;
    const int32_t* pred;
    int32_t* used;
    uint32_t* parts;
    uint8_t* q8;
    int64_t ldq;
};

__device__ __forceinline__ f4_t mfma_bf16(u32x4 a, u32x4 b, f4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 ldg16(const uint16_t* p) { return *(const u32x4*)p; }

// 32-bit LDS address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr32(const void* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4 with
// a wave-uniform 64-bit base and a 32-bit lane byte offset): lane i's bytes
// land at lds_dst + 16 i.  Issued from inline assembly, so the compiler does
// not track it: the caller waits (s_waitcnt vmcnt) before the data is read.
__device__ __forceinline__ void lds_copy16(const void* sbase, uint32_t voff, uint32_t lds_dst) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(lds_dst), "v"(voff), "s"(sbase)
                 : "memory");
}

// Maximum / sum over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four lanes that hold
// one query's scores) with VALU lane swaps: swapping a value with itself
// between rows 0-1 and 2-3 of 16 lanes (then between the two halves of the
// wave) leaves each lane holding its own value and its partner's, in some
// order, which a symmetric operation does not see.
__device__ __forceinline__ float quad_max(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float quad_sum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Physical 16-byte chunk of logical chunk c in LDS row `key` of a V block:
// c ^ v_swz(key), which moves whole 32-byte chunk pairs.  A transposing read
// (below) takes 32 contiguous bytes of each of 8 consecutive keys per half
// wave; keys differing in bits 0-2 then sit in different pairs, so each half
// wave reads all 64 banks once.
__device__ __forceinline__ int v_swz(int key) { return 2 * (key & 7); }

// ds_read_b64_tr_b16: within each group of 16 lanes, lane 4a + b receives
// element b of the 8-byte chunks addressed by lanes a, 4 + a, 8 + a and
// 12 + a (measured on gfx950 with index patterns).
typedef short v4s_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr16(const uint8_t* p) {
    const v4s_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s_t*)p);
    return __builtin_bit_cast(uint2, r);
}

template <bool QUANT, int FMT>
__global__ __launch_bounds__(kThreads, 2) void attention_kernel(AttnArgs p) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[4 * kKvBytes];  // K0 V0 K1 V1; output staging
    __shared__ uint32_t redm[kThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g = lane >> 4;

    // Workgroup -> (head, sequence, query block), heaviest query blocks first.
    // Workgroups are dealt round-robin to the 8 XCDs; with n_heads a multiple
    // of 8, heads h .. h + n_heads/8 - 1 (which share key/value heads) land on
    // one XCD and its L2.
    const int bid = blockIdx.x;
    const int hi = bid % p.nh;
    const int h = (p.nh % 8 == 0) ? (hi % 8) * (p.nh / 8) + hi / 8 : hi;
    const int t = bid / p.nh;
    const int qb = p.nqb - 1 - t / p.nseq;
    const int64_t s0 = (int64_t)(t % p.nseq) * p.seq_len;
    // Positions within the sequence (32-bit): queries q0 .., keys 0 .. kend-1.
    const int slen = (int)(s0 + p.seq_len < p.rows ? p.seq_len : p.rows - s0);
    const int q0 = qb * kBq;

    const bool cast = QUANT && p.pred;
    const int bq = QUANT ? fused_bias(p.pred, p.used) : 0;
    if (q0 >= slen) {  // a block past the end of a short last sequence
        if (QUANT && tid == 0) p.parts[bid] = 0u;
        return;
    }
    const int hk = h / (p.nh / p.nkv);
    const uint16_t* Qg = p.qkv + s0 * p.ld + (int64_t)h * kHd;
    const uint16_t* Kg = p.qkv + s0 * p.ld + (int64_t)(p.nh + hk) * kHd;
    const uint16_t* Vg = p.qkv + s0 * p.ld + (int64_t)(p.nh + p.nkv + hk) * kHd;
    const int kend = q0 + kBq < slen ? q0 + kBq : slen;
    const int nkb = (kend + kBk - 1) / kBk;
    const int wq0 = q0 + 32 * w;

    // Query fragments (B operand of S^T = K . Q^T): Q[q][32 ds + 8 g .. + 7];
    // rows past the end read the last row (their outputs are not stored).
    u32x4 qf[2][4];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const int row = min(wq0 + 16 * qt + l16, slen - 1);
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) qf[qt][ds] = ldg16(Qg + (int64_t)row * p.ld + 32 * ds + 8 * g);
    }

    // Staging: K and V go straight to LDS (global_load_lds_dwordx4), wave w
    // copying keys 16 w .. 16 w + 15 of each (4 copies of 4 rows; lane l: key
    // 16 w + 4 j + l/16, physical chunk l%16, which holds logical chunk
    // (l%16) ^ (key mod 16) for K and (l%16) ^ v_swz(key) for V).  Both are
    // rows of 256 bytes, one per key.  Rows past kend read row kend-1 (a
    // finite copy; those keys are masked).  Full blocks: a wave-uniform block
    // base plus per-lane 32-bit offsets; the last, partial block clamps each
    // row.
    const int ld = (int)p.ld;
    const int wu = __builtin_amdgcn_readfirstlane(w);
    int kkey[4];
    uint32_t kboff[4], vboff[4];  // byte offsets of this lane's K and V copies in a full block
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        kkey[j] = 16 * wu + 4 * j + (lane >> 4);
        kboff[j] = (uint32_t)(kkey[j] * ld + 8 * ((lane & 15) ^ (kkey[j] & 15))) * 2u;
        vboff[j] = (uint32_t)(kkey[j] * ld + 8 * ((lane & 15) ^ v_swz(kkey[j]))) * 2u;
    }
    // One block of K (V = false) or V into buffer buf.
    auto copy_kv = [&](int kb, int buf, bool V) {
        const int kbase = kb * kBk;
        const uint16_t* src = (V ? Vg : Kg) + (int64_t)kbase * p.ld;
        const uint32_t dst = lds_addr32(lds + buf * 2 * kKvBytes + (V ? kKvBytes : 0)) + (16 * wu) * 256;
        if (kbase + kBk <= kend) {
#pragma unroll
            for (int j = 0; j < 4; ++j) lds_copy16(src, V ? vboff[j] : kboff[j], dst + j * 1024);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = min(kbase + kkey[j], kend - 1) - kbase;
                const int c = (lane & 15) ^ (V ? v_swz(kkey[j]) : (kkey[j] & 15));
                lds_copy16(src, (uint32_t)(row * ld + 8 * c) * 2u, dst + j * 1024);
            }
        }
    };

    f4_t o[8][2];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
        for (int qt = 0; qt < 2; ++qt) o[dt][qt] = f4_t{0.f, 0.f, 0.f, 0.f};
    // Running maximum of the raw scores and per-lane partial row sums.
    float mrun[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f};
    const float c2 = p.scale_log2;
    const float lazy = 8.0f / c2;  // 2^8 in probability, in units of raw scores

    copy_kv(0, 0, false);
    copy_kv(0, 0, true);
    // Every load of the prologue (the query fragments and the K and V copies
    // included) has landed: the loop's waits then only cover the loads issued
    // inside the loop.
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
        const int buf = kb & 1;
        // The next block's copies into the other buffer, which every wave
        // finished reading before the last barrier.
        if (kb + 1 < nkb) {
            copy_kv(kb + 1, buf ^ 1, false);
            copy_kv(kb + 1, buf ^ 1, true);
        }
        const int kbase = kb * kBk;
        // Every wave runs every block: one entirely above a wave's diagonal
        // (at most 2 of 4 waves, in the last block) is masked to zero weight,
        // which costs less than the accumulator copies a skip branch makes
        // the compiler insert.
        {
            const uint8_t* Kl = lds + buf * 2 * kKvBytes;
            const uint8_t* Vl = Kl + kKvBytes;
            f4_t s[4][2];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt)
                for (int qt = 0; qt < 2; ++qt) s[kt][qt] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ds = 0; ds < 4; ++ds)
#pragma unroll
                for (int kt = 0; kt < 4; ++kt) {
                    const int key = kt * 16 + l16;
                    const u32x4 kf = *(const u32x4*)(Kl + key * 256 + (((4 * ds + g) ^ (key & 15)) << 4));
                    s[kt][0] = mfma_bf16(kf, qf[0][ds], s[kt][0]);
                    s[kt][1] = mfma_bf16(kf, qf[1][ds], s[kt][1]);
                }
            // keys above a query's position, or past the end: -inf (wave-uniform test)
            if (kbase + kBk - 1 > wq0 || kbase + kBk > kend) {
#pragma unroll
                for (int qt = 0; qt < 2; ++qt) {
                    const int q = wq0 + 16 * qt + l16;
#pragma unroll
                    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int key = kbase + kt * 16 + 4 * g + i;
                            s[kt][qt][i] = (key > q || key >= kend) ? -INFINITY : s[kt][qt][i];
                        }
                }
            }
            u32x4 pf[2][2];
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) {
                float mx = -INFINITY;
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[kt][qt][i]);
                mx = quad_max(mx);
                // The exponent offset moves only when a score exceeds it by
                // more than 2^8 in probability (the first block always): the
                // probabilities stay below 256, and the rescale of the sums
                // and of O by alpha is rare.
                const bool grow = mx > mrun[qt] + lazy;
                if (__any(grow)) {
                    const float mnew = grow ? mx : mrun[qt];
                    const float alpha = __builtin_amdgcn_exp2f((mrun[qt] - mnew) * c2);
                    mrun[qt] = mnew;
                    lsum[qt] *= alpha;
#pragma unroll
                    for (int dt = 0; dt < 8; ++dt) o[dt][qt] *= alpha;
                }
                const float mnew = mrun[qt];
                const float moff = -mnew * c2;
                float pr[4][4];
                float ls = lsum[qt];
#pragma unroll
                for (int kt = 0; kt < 4; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        pr[kt][i] = __builtin_amdgcn_exp2f(fmaf(s[kt][qt][i], c2, moff));
                        ls += pr[kt][i];
                    }
                lsum[qt] = ls;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
                    pf[qt][ks] = u32x4{pack_bf16x2(pr[2 * ks][0], pr[2 * ks][1]), pack_bf16x2(pr[2 * ks][2], pr[2 * ks][3]),
                                       pack_bf16x2(pr[2 * ks + 1][0], pr[2 * ks + 1][1]),
                                       pack_bf16x2(pr[2 * ks + 1][2], pr[2 * ks + 1][3])};
            }
            // key slices outer: successive products into one accumulator are
            // 16 instructions apart
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) {
                    // lane (g, j) addresses key 32 ks + 16 t + 4 g + j/4,
                    // columns 16 dt + 4 (j%4) .. + 3, and receives column
                    // 16 dt + j of keys 32 ks + 16 t + 4 g + 0..3
                    u32x4 vf;
#pragma unroll
                    for (int t = 0; t < 2; ++t) {
                        const int key = 32 * ks + 16 * t + 4 * g + (l16 >> 2);
                        const int c = 2 * dt + ((l16 & 3) >> 1);
                        const uint2 u = lds_read_tr16(Vl + key * 256 + ((c ^ v_swz(key)) << 4) + 8 * (l16 & 1));
                        vf[2 * t] = u.x;
                        vf[2 * t + 1] = u.y;
                    }
                    o[dt][0] = mfma_bf16(vf, pf[0][ks], o[dt][0]);
                    o[dt][1] = mfma_bf16(vf, pf[1][ks], o[dt][1]);
                }
            }
        }
        // this wave's K and V copies into the other buffer (not tracked by
        // the compiler) have landed before the barrier
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }

    // O[q][d] = O^T[d][q] / l[q]: staged in LDS as rows of 256 bytes (16-byte
    // chunk c of query row r at chunk c ^ (r mod 16)), then stored as whole
    // 256-byte rows of this head, cast with the fused bias on the way.
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const float inv = 1.0f / quad_sum(lsum[qt]);
        const int r = 32 * w + 16 * qt + l16;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const f4_t v = o[dt][qt];
            const int c = 2 * dt + (g >> 1);
            *(uint2*)(lds + r * 256 + ((c ^ (r & 15)) << 4) + 8 * (g & 1)) =
                make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
        }
    }
    __syncthreads();
    uint32_t mag = 0;
    uint16_t* Og = p.o + s0 * p.ldo + (int64_t)h * kHd;
    uint8_t* Q8 = QUANT ? p.q8 + s0 * p.ldq + (int64_t)h * kHd : nullptr;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int idx = tid + kThreads * j;
        const int r = idx >> 4, c = idx & 15;
        const int q = q0 + r;
        if (q >= slen) continue;
        const uint4 v = *(const uint4*)(lds + r * 256 + ((c ^ (r & 15)) << 4));
        st16(Og + (int64_t)q * p.ldo + 8 * c, v);
        if (QUANT) {
            mag = max(mag, mag8(v));
            if (cast) *(uint2*)(Q8 + (int64_t)q * p.ldq + 8 * c) = codes8<FMT>(v, bq);
        }
    }
    if (QUANT) {
        const uint32_t bm = block_max(mag, redm);
        if (tid == 0) p.parts[bid] = bm;
    }
}

// ------------------------------------------------------------- host side
template <int V> using IC = std::integral_constant<int, V>;

template <typename Fn>
void with_fmt(int fmt, Fn&& fn) {
    switch (fmt) {
        case FP8_E4M3: fn(IC<FP8_E4M3>{}); break;
        case FP8_E5M2: fn(IC<FP8_E5M2>{}); break;
        case FP8_E4_A: fn(IC<FP8_E4_A>{}); break;
        default: fn(IC<FP8_E5_A>{}); break;
    }
}

int glue_grid(int64_t items) {
    const int64_t b = (items + kThreads - 1) / kThreads;
    return (int)(b < 1 ? 1 : b > kGluePartsMax ? kGluePartsMax : b);
}

// Finish a fused quantise: exact bias from the parts, recast if mispredicted.
int32_t quant_finish(const uint16_t* y, int64_t rows, int64_t cols, int64_t ldy, const FusedQuant& fq, int nparts,
                     hipStream_t s) {
    return launch_quant_check(y, FP8_DT_BF16, rows, cols, ldy, fq.fmt, fq.margin, fq.ws + 1, nparts,
                              (const int32_t*)fq.ws, fq.bias, fq.amax_bits, fq.flags, fq.q, fq.ldq, nullptr, 0, s);
}

}  // namespace

namespace fp8lin {

int64_t glue_parts_rmsnorm(int64_t rows) { return rows; }
int64_t glue_parts_swiglu() { return kGluePartsMax; }
int64_t glue_parts_attention(int64_t rows, int64_t seq_len, int nh) {
    const int64_t nseq = (rows + seq_len - 1) / seq_len;
    const int64_t nqb = ((seq_len < rows ? seq_len : rows) + kBq - 1) / kBq;
    return nseq * nqb * nh;
}

int32_t launch_residual_add(const uint16_t* a, const uint16_t* b, uint16_t* out, int64_t n, hipStream_t s) {
    const int64_t n8 = n / 8;
    hipLaunchKernelGGL(add_kernel, dim3(glue_grid(n8)), dim3(kThreads), 0, s, a, b, out, n8);
    return hip_status();
}

int32_t launch_rmsnorm(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr, const uint16_t* g,
                       int64_t rows, int64_t cols, float eps, uint16_t* h, int64_t ldh, uint16_t* y, int64_t ldy,
                       const FusedQuant* fq, hipStream_t s) {
    const bool quant = fq && fq->q;
    const int32_t* pred = quant ? fq->pred : nullptr;
    int32_t* used = quant ? (int32_t*)fq->ws : nullptr;
    uint32_t* parts = quant ? fq->ws + 1 : nullptr;
    uint8_t* q = quant ? fq->q : nullptr;
    const int64_t ldq = quant ? fq->ldq : 0;
    auto go = [&](auto R, auto Q, auto F) {
        constexpr bool kR = decltype(R)::value != 0, kQ = decltype(Q)::value != 0;
        constexpr int kF = decltype(F)::value;
        if (cols <= (int64_t)8 * kThreads * 4)
            hipLaunchKernelGGL((rmsnorm_kernel<kR, kQ, kF, 4>), dim3((unsigned)rows), dim3(kThreads), 0, s, x, ldx, res,
                               ldr, g, cols, eps, h, ldh, y, ldy, pred, used, parts, q, ldq);
        else
            hipLaunchKernelGGL((rmsnorm_kernel<kR, kQ, kF, 8>), dim3((unsigned)rows), dim3(kThreads), 0, s, x, ldx, res,
                               ldr, g, cols, eps, h, ldh, y, ldy, pred, used, parts, q, ldq);
    };
    with_fmt(quant ? fq->fmt : FP8_E4M3, [&](auto F) {
        if (res) {
            if (quant) go(IC<1>{}, IC<1>{}, F); else go(IC<1>{}, IC<0>{}, F);
        } else {
            if (quant) go(IC<0>{}, IC<1>{}, F); else go(IC<0>{}, IC<0>{}, F);
        }
    });
    int32_t st = hip_status();
    if (st == FP8_OK && quant) st = quant_finish(y, rows, cols, ldy, *fq, (int)rows, s);
    return st;
}

int32_t launch_rope_table(int64_t seq_len, int d_head, double theta, float* table, hipStream_t s) {
    const int half = d_head / 2;
    hipLaunchKernelGGL(rope_table_kernel, dim3(glue_grid(seq_len * half)), dim3(kThreads), 0, s, seq_len, half, theta,
                       (float2*)table);
    return hip_status();
}

int32_t launch_rope(uint16_t* x, int64_t rows, int64_t ld, int nheads, int d_head, int64_t seq_len,
                    const float* table, hipStream_t s) {
    const int half = d_head / 2;
    hipLaunchKernelGGL(rope_kernel, dim3(glue_grid(rows * nheads * (half / 8))), dim3(kThreads), 0, s, x, rows, ld,
                       nheads, half, seq_len, (const float2*)table);
    return hip_status();
}

int32_t launch_swiglu(const uint16_t* gu, int64_t ldgu, int64_t rows, int64_t ffn, uint16_t* a, int64_t lda,
                      const FusedQuant* fq, hipStream_t s) {
    const bool quant = fq && fq->q;
    const int grid = glue_grid(rows * (ffn / 8));
    with_fmt(quant ? fq->fmt : FP8_E4M3, [&](auto F) {
        if (quant)
            hipLaunchKernelGGL((swiglu_kernel<true, decltype(F)::value>), dim3(grid), dim3(kThreads), 0, s, gu, ldgu,
                               rows, ffn, a, lda, fq->pred, (int32_t*)fq->ws, fq->ws + 1, fq->q, fq->ldq);
        else
            hipLaunchKernelGGL((swiglu_kernel<false, decltype(F)::value>), dim3(grid), dim3(kThreads), 0, s, gu, ldgu,
                               rows, ffn, a, lda, nullptr, nullptr, nullptr, nullptr, (int64_t)0);
    });
    int32_t st = hip_status();
    if (st == FP8_OK && quant) st = quant_finish(a, rows, ffn, lda, *fq, grid, s);
    return st;
}

int32_t launch_attention(const uint16_t* qkv, int64_t rows, int64_t ld, int64_t seq_len, int nh, int nkv,
                         uint16_t* o, int64_t ldo, const FusedQuant* fq, hipStream_t s) {
    const bool quant = fq && fq->q;
    AttnArgs a;
    a.qkv = qkv;
    a.ld = ld;
    a.rows = rows;
    a.seq_len = seq_len;
    a.nh = nh;
    a.nkv = nkv;
    a.nseq = (int)((rows + seq_len - 1) / seq_len);
    a.nqb = (int)(((seq_len < rows ? seq_len : rows) + kBq - 1) / kBq);
    a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)kHd));
    a.o = o;
    a.ldo = ldo;
    a.pred = quant ? fq->pred : nullptr;
    a.used = quant ? (int32_t*)fq->ws : nullptr;
    a.parts = quant ? fq->ws + 1 : nullptr;
    a.q8 = quant ? fq->q : nullptr;
    a.ldq = quant ? fq->ldq : 0;
    const int64_t nblk = glue_parts_attention(rows, seq_len, nh);
    with_fmt(quant ? fq->fmt : FP8_E4M3, [&](auto F) {
        if (quant)
            hipLaunchKernelGGL((attention_kernel<true, decltype(F)::value>), dim3((unsigned)nblk), dim3(kThreads), 0,
                               s, a);
        else
            hipLaunchKernelGGL((attention_kernel<false, decltype(F)::value>), dim3((unsigned)nblk), dim3(kThreads), 0,
                               s, a);
    });
    int32_t st = hip_status();
    if (st == FP8_OK && quant) st = quant_finish(o, rows, (int64_t)nh * kHd, ldo, *fq, (int)nblk, s);
    return st;
}

}  // namespace fp8lin
