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
// cast: x * 2^b is formed with v_ldexp_f32, which is exact for every bf16 /
// fp32 x (a power-of-two scale; results below the fp32 normal range are far
// below half the smallest FP8 subnormal and become signed zeros either way),
// clipped to +-max_num with v_med3_f32 (App. A: overflow clips to the
// maximum; infinities included), and converted two at a time by
// v_cvt_pk_fp8_f32 / v_cvt_pk_bf8_f32, which round to nearest even and keep
// subnormals.  The converters encode NaN inputs as 0xFF / 0xFE and overflow
// as NaN or infinity; the clip removes the overflow case and NaN inputs,
// detected with a packed integer test, are re-encoded as 0x7F with their sign.
// The transposed copy goes through a 128 x 128 byte LDS tile so that both
// outputs leave as coalesced stores (whole 128-byte lines for the transpose).
#include <type_traits>

#include "fp8lin_fp8.h"
#include "fp8lin_internal.h"

namespace fp8lin {
namespace {

// Each workgroup reads one contiguous range of 16-byte vectors (a multiple of
// 4 KiB, so ranges start on DRAM-page-friendly boundaries) with eight
// non-temporal loads in flight per lane: a range per workgroup keeps every
// HBM channel streaming through whole pages, which reads measurably faster
// than a grid-stride sweep (about 7 vs 5.5 TB/s on a 2 GiB buffer).
template <int DT>
__global__ __launch_bounds__(kAmaxThreads) void amax_partial_kernel(const void* __restrict__ x,
                                                                   int64_t n, int vec,
                                                                   uint32_t* __restrict__ partial) {
    __shared__ uint32_t red[kAmaxThreads / 64];
    constexpr int kL = 8;
    uint32_t m = 0;
    int64_t tail0 = 0;
    if (vec) {
        constexpr int per = DT == FP8_DT_BF16 ? 8 : 4;
        const uint4* __restrict__ p = (const uint4*)x;
        const int64_t nv = n / per;
        tail0 = nv * per;
        const int64_t chunk = ((nv + gridDim.x - 1) / gridDim.x + 255) & ~(int64_t)255;
        const int64_t b0 = min(nv, (int64_t)blockIdx.x * chunk), b1 = min(nv, b0 + chunk);
        int64_t i = b0 + threadIdx.x;
        us2 mm = {0, 0};
        auto fold = [&](const uint4& v) {
            if (DT == FP8_DT_BF16) mm = fold_bf16(mm, v);
            else m = fold_f32(m, v);
        };
        for (; i + (kL - 1) * kAmaxThreads < b1; i += kL * kAmaxThreads) {
            uint4 v[kL];
#pragma unroll
            for (int l = 0; l < kL; ++l) v[l] = ld_stream(p + i + l * kAmaxThreads);
            // all kL loads issue before the first use (the scheduler would
            // otherwise start folding the first one and wait for it alone)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int l = 0; l < kL; ++l) fold(v[l]);
        }
        // fewer than kL vectors of this lane left: unconditional loads of
        // in-range vectors (a guarded load compiles to a branch and a wait per
        // load), those past the range replaced by zero, neutral for the maximum
        if (b1 > b0) {
            uint4 v[kL];
#pragma unroll
            for (int l = 0; l < kL; ++l) v[l] = ld_stream(p + min(i + l * kAmaxThreads, b1 - 1));
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int l = 0; l < kL; ++l)
                if (i + l * kAmaxThreads >= b1) v[l] = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
            for (int l = 0; l < kL; ++l) fold(v[l]);
        }
        if (DT == FP8_DT_BF16) m = max((uint32_t)mm.x, (uint32_t)mm.y);
    }
    // elements past the last whole vector (or every element when x is not
    // 16-byte aligned), strided over the whole grid
    const int64_t tid = (int64_t)blockIdx.x * kAmaxThreads + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * kAmaxThreads;
    for (int64_t j = tail0 + tid; j < n; j += nth) m = max(m, elem_mag<DT>(x, j));
    m = block_max(m, red);
    if (threadIdx.x == 0) partial[blockIdx.x] = m;
}

template <int DT, int FMT>
__global__ __launch_bounds__(kAmaxThreads) void amax_finalize_kernel(
    const uint32_t* __restrict__ partial, int nparts, int32_t margin, int32_t* __restrict__ bias,
    uint32_t* __restrict__ amax_bits, uint32_t* __restrict__ flags) {
    __shared__ uint32_t red[kAmaxThreads / 64];
    uint32_t m = strided_max<kAmaxThreads>(partial, nparts);
    m = block_max(m, red);
    if (threadIdx.x == 0) {
        const uint32_t a32 = canon_amax(DT == FP8_DT_BF16 ? (m << 16) : m);
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

// Workgroup tile: 128 rows x 128 columns, 256 threads.  Lane l of wave w owns
// rows r0 .. r0+7 (r0 = 8 (4 w + l / 16)) and columns c0 .. c0+7
// (c0 = 8 (l % 16)): each of its row loads is one 16-byte (bf16) or two
// 16-byte (fp32) accesses, 16 lanes covering 256 (512) contiguous bytes.
constexpr int kCastRows = 128, kCastCols = 128, kCastThreads = 256, kRpt = 8;

__device__ __forceinline__ uint32_t byte_of(uint32_t w, int j) { return (w >> (8 * j)) & 0xFFu; }

// One 128 x 128 tile (tile row tr, tile column tc) of the cast with bias b:
// codes to q (if given) and transposed codes to qT (if given).  With MAX, the
// largest magnitude pattern of the tile's elements (bf16: 15 bits, fp32: 31
// bits; 0 past the edges) is returned, valid in every thread after a block
// reduction by the caller.  Every thread of the block must call it (it
// synchronises through the LDS tile), and it leaves the LDS tile free for
// the next call.
// With ROWB, row r is cast with its own bias rowb[r] (clamped) instead of b.
template <int DT, int FMT, bool MAX, bool ROWB = false>
__device__ __forceinline__ uint32_t cast_tile(const void* __restrict__ x, int64_t rows, int64_t cols,
                                              int64_t ldx, int b, uint8_t* __restrict__ q, int64_t ldq,
                                              uint8_t* __restrict__ qT, int64_t ldqT, int64_t tr,
                                              int64_t tc, int vec_in, int vec_q, int vec_qT,
                                              uint8_t* __restrict__ tile,
                                              const int32_t* __restrict__ rowb = nullptr) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int chunk = lane & 15, g = lane >> 4;
    const int64_t R0 = tr * kCastRows, C0 = tc * kCastCols;
    const int lr = (w * 4 + g) * kRpt, lc = chunk * 8;
    const int64_t r0 = R0 + lr, c0 = C0 + lc;
    int bi[kRpt];  // bias of each of this lane's rows
#pragma unroll
    for (int i = 0; i < kRpt; ++i) bi[i] = ROWB ? (r0 + i < rows ? clamp_bias(rowb[r0 + i]) : 0) : b;

    uint32_t lo[kRpt], hi[kRpt];  // codes of columns c0..c0+3 and c0+4..c0+7, per row
    uint32_t mag = 0;
    const bool full = vec_in && (r0 + kRpt <= rows) && (c0 + 8 <= cols);
    if (full) {
        if (DT == FP8_DT_BF16) {
            uint4 v[kRpt];
#pragma unroll
            for (int i = 0; i < kRpt; ++i) v[i] = ld_stream((const uint16_t*)x + (r0 + i) * ldx + c0);
            if (MAX) {
                us2 mm = {0, 0};
#pragma unroll
                for (int i = 0; i < kRpt; ++i) mm = fold_bf16(mm, v[i]);
                mag = max((uint32_t)mm.x, (uint32_t)mm.y);
            }
#pragma unroll
            for (int i = 0; i < kRpt; ++i) {
                lo[i] = cast4_bf16<FMT>(v[i].x, v[i].y, bi[i]);
                hi[i] = cast4_bf16<FMT>(v[i].z, v[i].w, bi[i]);
                if (__builtin_expect(any_nan_bf16(v[i].x, v[i].y) || any_nan_bf16(v[i].z, v[i].w), 0)) {
                    const uint32_t h0[4] = {v[i].x & 0xFFFFu, v[i].x >> 16, v[i].y & 0xFFFFu, v[i].y >> 16};
                    const uint32_t h1[4] = {v[i].z & 0xFFFFu, v[i].z >> 16, v[i].w & 0xFFFFu, v[i].w >> 16};
                    lo[i] = nan_patch<FMT>(lo[i], h0);
                    hi[i] = nan_patch<FMT>(hi[i], h1);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < kRpt; ++i) {
                const uint4* p = (const uint4*)((const uint32_t*)x + (r0 + i) * ldx + c0);
                const uint4 a = ld_stream(p), bb = ld_stream(p + 1);
                if (MAX) mag = fold_f32(fold_f32(mag, a), bb);
                lo[i] = cast4_f32<FMT>(a, bi[i]);
                hi[i] = cast4_f32<FMT>(bb, bi[i]);
                const uint32_t m = (a.x | a.y | a.z | a.w | bb.x | bb.y | bb.z | bb.w) & 0x7F800000u;
                if (__builtin_expect(m == 0x7F800000u, 0)) {  // some exponent field may be all ones
                    const uint32_t h0[4] = {f32_key(a.x), f32_key(a.y), f32_key(a.z), f32_key(a.w)};
                    const uint32_t h1[4] = {f32_key(bb.x), f32_key(bb.y), f32_key(bb.z), f32_key(bb.w)};
                    lo[i] = nan_patch<FMT>(lo[i], h0);
                    hi[i] = nan_patch<FMT>(hi[i], h1);
                }
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < kRpt; ++i) {
            uint32_t wlo = 0, whi = 0;
            for (int j = 0; j < 8; ++j) {
                const int64_t r = r0 + i, c = c0 + j;
                uint32_t code = 0u;
                if (r < rows && c < cols) {
                    code = cast1<DT, FMT>(x, r * ldx + c, bi[i]);
                    if (MAX) mag = max(mag, elem_mag<DT>(x, r * ldx + c));
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
            for (int i = 0; i < kRpt; ++i) *(uint2*)(q + (r0 + i) * ldq + c0) = make_uint2(lo[i], hi[i]);
        } else {
            for (int i = 0; i < kRpt; ++i)
                for (int j = 0; j < 8; ++j) {
                    const int64_t r = r0 + i, c = c0 + j;
                    if (r < rows && c < cols) q[r * ldq + c] = (uint8_t)byte_of(j < 4 ? lo[i] : hi[i], j & 3);
                }
        }
    }

    if (qT) {
        // Column c0 + j of this lane's 8x8 block, rows r0..r0+7, as 8 bytes at
        // row offset lr of transposed row lc + j; 16-byte chunks of a
        // transposed row are XOR-swizzled with the column block.
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t* src = j < 4 ? lo : hi;
            const int jj = j & 3;
            const uint32_t w0 = byte_of(src[0], jj) | (byte_of(src[1], jj) << 8) | (byte_of(src[2], jj) << 16) |
                                (byte_of(src[3], jj) << 24);
            const uint32_t w1 = byte_of(src[4], jj) | (byte_of(src[5], jj) << 8) | (byte_of(src[6], jj) << 16) |
                                (byte_of(src[7], jj) << 24);
            const int cl = lc + j;
            const int off = cl * kCastRows + ((((lr >> 4) ^ (cl >> 3)) & 7) << 4) + (lr & 15);
            *(uint2*)(tile + off) = make_uint2(w0, w1);
        }
        __syncthreads();
        // 128 transposed rows x 8 chunks of 16 bytes = 1024 chunks, four per thread.
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const int idx = threadIdx.x + h * kCastThreads;
            const int cl = idx >> 3, qq = idx & 7;
            const int64_t c = C0 + cl;
            const int64_t rr = R0 + qq * 16;
            if (c >= cols || rr >= rows) continue;
            const uint4 v = *(const uint4*)(tile + cl * kCastRows + (((qq ^ (cl >> 3)) & 7) << 4));
            uint8_t* dst = qT + c * ldqT + rr;
            if (vec_qT && rr + 16 <= rows) {
                *(uint4*)dst = v;
            } else {
                const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
                for (int t = 0; t < 16 && rr + t < rows; ++t) dst[t] = (uint8_t)byte_of(wv[t >> 2], t & 3);
            }
        }
        __syncthreads();  // the tile may be rewritten by the next call
    }
    return mag;
}


template <int DT, int FMT>
__global__ __launch_bounds__(kCastThreads) void cast_kernel(
    const void* __restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    const int32_t* __restrict__ bias_p, uint8_t* __restrict__ q, int64_t ldq,
    uint8_t* __restrict__ qT, int64_t ldqT, int64_t tiles_c, int vec_in, int vec_q, int vec_qT) {
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];
    const int b = clamp_bias(*bias_p);
    cast_tile<DT, FMT, false>(x, rows, cols, ldx, b, q, ldq, qT, ldqT, blockIdx.x / tiles_c,
                              blockIdx.x % tiles_c, vec_in, vec_q, vec_qT, tile);
}

// ------------------------------------------------- quantise: amax + bias + cast
// Pass 1 (quant_pass1_kernel), one workgroup per tile: the largest magnitude
// pattern of the tile goes to parts[tile]; with CAST the tile is also cast with
// the predicted bias (clamped), which block 0 records in *used.
// Pass 2 (quant_pass2_kernel): every workgroup reduces parts[] and evaluates
// Eq. 3; block 0 writes bias, amax and flags.  If pass 1 did not cast, or cast
// with a bias other than the exact one, the workgroups recast all ncast tiles
// (grid-stride) with the exact bias; otherwise the codes of pass 1 are already
// those of the exact bias and nothing more is written.  parts[] may come from
// another producer of the same tensor (a matmul epilogue) with its own tiling.
template <int DT, int FMT, bool CAST>
__global__ __launch_bounds__(kCastThreads) void quant_pass1_kernel(
    const void* __restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    const int32_t* __restrict__ bias_pred, int32_t* __restrict__ used, uint32_t* __restrict__ parts,
    uint8_t* __restrict__ q, int64_t ldq, uint8_t* __restrict__ qT, int64_t ldqT, int64_t tiles_c,
    int vec_in, int vec_q, int vec_qT) {
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];
    __shared__ uint32_t red[kCastThreads / 64];
    int b = 0;
    if (CAST) {
        b = clamp_bias(*bias_pred);
        if (blockIdx.x == 0 && threadIdx.x == 0) *used = b;
    }
    const uint32_t m = cast_tile<DT, FMT, true>(x, rows, cols, ldx, b, CAST ? q : nullptr, ldq,
                                                CAST ? qT : nullptr, ldqT, blockIdx.x / tiles_c,
                                                blockIdx.x % tiles_c, vec_in, vec_q, vec_qT, tile);
    const uint32_t bm = block_max(m, red);
    if (threadIdx.x == 0) parts[blockIdx.x] = bm;
}

// Pass 2 of one tensor as workgroup bid of nb: see quant_pass2_kernel.
template <int DT, int FMT>
__device__ __forceinline__ void quant_pass2_body(
    int bid, int nb, uint8_t* tile, uint32_t* red, uint32_t& amax_s, const void* __restrict__ x,
    int64_t rows, int64_t cols, int64_t ldx, const uint32_t* __restrict__ parts, int nparts,
    const int32_t* __restrict__ used, int have_used, int32_t margin, int32_t* __restrict__ bias,
    uint32_t* __restrict__ amax_bits, uint32_t* __restrict__ flags, uint8_t* __restrict__ q, int64_t ldq,
    uint8_t* __restrict__ qT, int64_t ldqT, int64_t tiles_c, int64_t ncast, int vec_in, int vec_q,
    int vec_qT) {
    uint32_t m = strided_max<kCastThreads>(parts, nparts);
    m = block_max(m, red);
    if (threadIdx.x == 0) amax_s = m;
    __syncthreads();
    const uint32_t a32 = canon_amax(DT == FP8_DT_BF16 ? (amax_s << 16) : amax_s);
    uint32_t fl;
    const int32_t bx = bias_of<FMT>(a32, margin, &fl);
    if (bid == 0 && threadIdx.x == 0) {
        *bias = bx;
        if (amax_bits) *amax_bits = a32;
        if (flags) *flags = fl;
    }
    const int b = clamp_bias(bx);
    if (have_used && *used == b) return;  // pass 1 already wrote these codes
    for (int64_t t = bid; t < ncast; t += nb)
        cast_tile<DT, FMT, false>(x, rows, cols, ldx, b, q, ldq, qT, ldqT, t / tiles_c, t % tiles_c,
                                  vec_in, vec_q, vec_qT, tile);
}

template <int DT, int FMT>
__global__ __launch_bounds__(kCastThreads) void quant_pass2_kernel(
    const void* __restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    const uint32_t* __restrict__ parts, int nparts, const int32_t* __restrict__ used, int have_used,
    int32_t margin, int32_t* __restrict__ bias, uint32_t* __restrict__ amax_bits,
    uint32_t* __restrict__ flags, uint8_t* __restrict__ q, int64_t ldq, uint8_t* __restrict__ qT,
    int64_t ldqT, int64_t tiles_c, int64_t ncast, int vec_in, int vec_q, int vec_qT) {
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];
    __shared__ uint32_t red[kCastThreads / 64];
    __shared__ uint32_t amax_s;
    quant_pass2_body<DT, FMT>(blockIdx.x, gridDim.x, tile, red, amax_s, x, rows, cols, ldx, parts, nparts, used,
                              have_used, margin, bias, amax_bits, flags, q, ldq, qT, ldqT, tiles_c, ncast,
                              vec_in, vec_q, vec_qT);
}

// ------------------------------------------------ delayed scaling
// The second launch of fp8_quantise_delayed (one workgroup): the tensor's amax
// from the tile maxima of pass 1 (cast with the bias in *bias, recorded in
// *used), whether those codes clipped (amax * 2^used > max_num, i.e. used is
// above the tensor's own Eq. 3 bias), the amax appended to the history ring
// at *count % hlen, and the bias of the next call: Eq. 3 of the largest amax
// in the history, minus the margin.  History words are amax bit patterns with
// the sign clear (canonical NaN 0x7FC00000 largest), so their integer maximum
// is the largest amax.  Slot *count % hlen is left out of the history
// reduction and replaced by this tensor's amax, so no thread reads the word
// thread 0 writes.
template <int DT, int FMT>
__global__ __launch_bounds__(kCastThreads) void quant_delayed_finish_kernel(
    const uint32_t* __restrict__ parts, int nparts, const int32_t* __restrict__ used, int32_t margin,
    uint32_t* __restrict__ history, int hlen, uint32_t* __restrict__ count, int32_t* __restrict__ bias,
    uint32_t* __restrict__ amax_bits, uint32_t* __restrict__ flags) {
    __shared__ uint32_t red[kCastThreads / 64];
    __shared__ uint32_t slot_s;
    uint32_t m = strided_max<kCastThreads>(parts, nparts);
    m = block_max(m, red);
    if (threadIdx.x == 0) slot_s = *count;
    __syncthreads();
    const uint32_t c = slot_s;
    const int slot = (int)(c % (uint32_t)hlen);
    uint32_t h = 0;
    for (int i = threadIdx.x; i < hlen; i += kCastThreads)
        if (i != slot) h = max(h, history[i]);
    __syncthreads();  // red[] is reused
    h = block_max(h, red);
    if (threadIdx.x == 0) {
        const uint32_t a32 = canon_amax(DT == FP8_DT_BF16 ? (m << 16) : m);
        uint32_t fl;
        const int32_t own = bias_of<FMT>(a32, 0, &fl);
        if (fl == 0u && nparts > 0 && *used > own) fl = FP8_FLAG_SATURATED;
        history[slot] = a32;
        *count = c + 1u;
        uint32_t fl_next;
        *bias = bias_of<FMT>(max(h, a32), margin, &fl_next);
        if (amax_bits) *amax_bits = a32;
        if (flags) *flags = fl;
    }
}

// ------------------------------------------------ quantise several tensors
// fp8_quantise of up to kQBatch tensors of one element type and format in one
// pass-1 launch and one pass-2 launch: workgroups [t0[i], t0[i+1]) of pass 1
// are tensor i's tiles, workgroups [p0[i], p0[i+1]) of pass 2 its finishing
// workgroups; each tensor keeps its own workspace (used word + tile maxima),
// so the bits are those of separate calls.
struct QBatch {
    int n;
    int64_t t0[kQBatch + 1], p0[kQBatch + 1];
    const void* x[kQBatch];
    int64_t rows[kQBatch], cols[kQBatch], ldx[kQBatch], tiles_c[kQBatch];
    const int32_t* pred[kQBatch];
    int32_t* bias[kQBatch];
    uint32_t* amax[kQBatch];
    uint32_t* flags[kQBatch];
    uint8_t* q[kQBatch];
    int64_t ldq[kQBatch];
    uint8_t* qT[kQBatch];
    int64_t ldqT[kQBatch];
    uint32_t* ws[kQBatch];
    int vec_in[kQBatch], vec_q[kQBatch], vec_qT[kQBatch];
};

__device__ __forceinline__ int batch_slot(const int64_t* start, int n, int64_t b) {
    int i = 0;
    while (i + 1 < n && b >= start[i + 1]) ++i;
    return i;
}

template <int DT, int FMT, bool CAST>
__global__ __launch_bounds__(kCastThreads) void quant_pass1_batch_kernel(QBatch qb) {
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];
    __shared__ uint32_t red[kCastThreads / 64];
    const int i = batch_slot(qb.t0, qb.n, blockIdx.x);
    const int64_t t = (int64_t)blockIdx.x - qb.t0[i];
    int b = 0;
    if (CAST) {
        b = clamp_bias(*qb.pred[i]);
        if (t == 0 && threadIdx.x == 0) *(int32_t*)qb.ws[i] = b;
    }
    const uint32_t m = cast_tile<DT, FMT, true>(qb.x[i], qb.rows[i], qb.cols[i], qb.ldx[i], b, CAST ? qb.q[i] : nullptr,
                                                qb.ldq[i], CAST ? qb.qT[i] : nullptr, qb.ldqT[i], t / qb.tiles_c[i],
                                                t % qb.tiles_c[i], qb.vec_in[i], qb.vec_q[i], qb.vec_qT[i], tile);
    const uint32_t bm = block_max(m, red);
    if (threadIdx.x == 0) qb.ws[i][1 + t] = bm;
}

template <int DT, int FMT>
__global__ __launch_bounds__(kCastThreads) void quant_pass2_batch_kernel(QBatch qb, int32_t margin, int have_used) {
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];
    __shared__ uint32_t red[kCastThreads / 64];
    __shared__ uint32_t amax_s;
    const int i = batch_slot(qb.p0, qb.n, blockIdx.x);
    const int64_t ntiles = qb.t0[i + 1] - qb.t0[i];
    quant_pass2_body<DT, FMT>((int)(blockIdx.x - qb.p0[i]), (int)(qb.p0[i + 1] - qb.p0[i]), tile, red, amax_s,
                              qb.x[i], qb.rows[i], qb.cols[i], qb.ldx[i], qb.ws[i] + 1, (int)ntiles,
                              (const int32_t*)qb.ws[i], have_used, margin, qb.bias[i], qb.amax[i], qb.flags[i],
                              qb.q[i], qb.ldq[i], qb.qT[i], qb.ldqT[i], qb.tiles_c[i], ntiles, qb.vec_in[i],
                              qb.vec_q[i], qb.vec_qT[i]);
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

constexpr int kQuantPass2MaxBlocks = 1024;

template <int DT, int FMT>
void launch_quantise_t(const void* x, int64_t rows, int64_t cols, int64_t ldx, int32_t margin,
                       const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits, uint32_t* flags,
                       uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT, uint32_t* ws,
                       hipStream_t s) {
    const int64_t tiles_r = (rows + kCastRows - 1) / kCastRows;
    const int64_t tiles_c = (cols + kCastCols - 1) / kCastCols;
    const int64_t ntiles = tiles_r * tiles_c;
    const int esz = DT == FP8_DT_BF16 ? 2 : 4;
    const int vec_in = ((uintptr_t)x % 16 == 0) && ((ldx * esz) % 16 == 0);
    const int vec_q = q && ((uintptr_t)q % 8 == 0) && (ldq % 8 == 0);
    const int vec_qT = qT && ((uintptr_t)qT % 16 == 0) && (ldqT % 16 == 0);
    int32_t* used = (int32_t*)ws;
    uint32_t* parts = ws + 1;
    if (bias_pred)
        hipLaunchKernelGGL((quant_pass1_kernel<DT, FMT, true>), dim3((unsigned)ntiles), dim3(kCastThreads), 0, s,
                           x, rows, cols, ldx, bias_pred, used, parts, q, ldq, qT, ldqT, tiles_c, vec_in,
                           vec_q, vec_qT);
    else
        hipLaunchKernelGGL((quant_pass1_kernel<DT, FMT, false>), dim3((unsigned)ntiles), dim3(kCastThreads), 0, s,
                           x, rows, cols, ldx, bias_pred, used, parts, q, ldq, qT, ldqT, tiles_c, vec_in,
                           vec_q, vec_qT);
    const int nb2 = (int)(ntiles < kQuantPass2MaxBlocks ? ntiles : kQuantPass2MaxBlocks);
    hipLaunchKernelGGL((quant_pass2_kernel<DT, FMT>), dim3(nb2), dim3(kCastThreads), 0, s, x, rows, cols, ldx,
                       parts, (int)ntiles, used, bias_pred ? 1 : 0, margin, bias, amax_bits, flags, q, ldq,
                       qT, ldqT, tiles_c, ntiles, vec_in, vec_q, vec_qT);
}

template <int DT, int FMT>
void launch_quantise_batch_t(int n, const QuantDesc* d, int32_t margin, hipStream_t s) {
    QBatch qb{};
    qb.n = n;
    const int esz = DT == FP8_DT_BF16 ? 2 : 4;
    bool pred = false;
    for (int i = 0; i < n; ++i) {
        const int64_t tiles_c = (d[i].cols + kCastCols - 1) / kCastCols;
        const int64_t ntiles = ((d[i].rows + kCastRows - 1) / kCastRows) * tiles_c;
        qb.t0[i + 1] = qb.t0[i] + ntiles;
        qb.p0[i + 1] = qb.p0[i] + (ntiles < kQuantPass2MaxBlocks ? ntiles : kQuantPass2MaxBlocks);
        qb.x[i] = d[i].x;
        qb.rows[i] = d[i].rows;
        qb.cols[i] = d[i].cols;
        qb.ldx[i] = d[i].ldx;
        qb.tiles_c[i] = tiles_c;
        qb.pred[i] = d[i].pred;
        qb.bias[i] = d[i].bias;
        qb.amax[i] = d[i].amax;
        qb.flags[i] = d[i].flags;
        qb.q[i] = d[i].q;
        qb.ldq[i] = d[i].ldq;
        qb.qT[i] = d[i].qT;
        qb.ldqT[i] = d[i].ldqT;
        qb.ws[i] = d[i].ws;
        qb.vec_in[i] = ((uintptr_t)d[i].x % 16 == 0) && ((d[i].ldx * esz) % 16 == 0);
        qb.vec_q[i] = d[i].q && ((uintptr_t)d[i].q % 8 == 0) && (d[i].ldq % 8 == 0);
        qb.vec_qT[i] = d[i].qT && ((uintptr_t)d[i].qT % 16 == 0) && (d[i].ldqT % 16 == 0);
        pred = d[i].pred != nullptr;
    }
    if (pred)
        hipLaunchKernelGGL((quant_pass1_batch_kernel<DT, FMT, true>), dim3((unsigned)qb.t0[n]), dim3(kCastThreads), 0,
                           s, qb);
    else
        hipLaunchKernelGGL((quant_pass1_batch_kernel<DT, FMT, false>), dim3((unsigned)qb.t0[n]), dim3(kCastThreads),
                           0, s, qb);
    hipLaunchKernelGGL((quant_pass2_batch_kernel<DT, FMT>), dim3((unsigned)qb.p0[n]), dim3(kCastThreads), 0, s, qb,
                       margin, pred ? 1 : 0);
}

template <int DT, int FMT>
void launch_quant_check_t(const void* x, int64_t rows, int64_t cols, int64_t ldx, int32_t margin,
                          const uint32_t* parts, int nparts, const int32_t* used, int32_t* bias,
                          uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT,
                          int64_t ldqT, hipStream_t s) {
    const int64_t tiles_c = (cols + kCastCols - 1) / kCastCols;
    const int64_t ncast = ((rows + kCastRows - 1) / kCastRows) * tiles_c;
    const int esz = DT == FP8_DT_BF16 ? 2 : 4;
    const int vec_in = ((uintptr_t)x % 16 == 0) && ((ldx * esz) % 16 == 0);
    const int vec_q = q && ((uintptr_t)q % 8 == 0) && (ldq % 8 == 0);
    const int vec_qT = qT && ((uintptr_t)qT % 16 == 0) && (ldqT % 16 == 0);
    const int nb2 = (int)(ncast < kQuantPass2MaxBlocks ? ncast : kQuantPass2MaxBlocks);
    hipLaunchKernelGGL((quant_pass2_kernel<DT, FMT>), dim3(nb2), dim3(kCastThreads), 0, s, x, rows, cols, ldx,
                       parts, nparts, used, 1, margin, bias, amax_bits, flags, q, ldq, qT, ldqT, tiles_c, ncast,
                       vec_in, vec_q, vec_qT);
}

template <int DT, int FMT>
void launch_quantise_delayed_t(const void* x, int64_t rows, int64_t cols, int64_t ldx, int32_t margin, int32_t* bias,
                               uint32_t* history, int hlen, uint32_t* count, uint32_t* amax_bits, uint32_t* flags,
                               uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT, uint32_t* ws, hipStream_t s) {
    const int64_t tiles_r = (rows + kCastRows - 1) / kCastRows;
    const int64_t tiles_c = (cols + kCastCols - 1) / kCastCols;
    const int64_t ntiles = tiles_r * tiles_c;
    int32_t* used = (int32_t*)ws;
    uint32_t* parts = ws + 1;
    if (ntiles > 0) {
        const int esz = DT == FP8_DT_BF16 ? 2 : 4;
        const int vec_in = ((uintptr_t)x % 16 == 0) && ((ldx * esz) % 16 == 0);
        const int vec_q = q && ((uintptr_t)q % 8 == 0) && (ldq % 8 == 0);
        const int vec_qT = qT && ((uintptr_t)qT % 16 == 0) && (ldqT % 16 == 0);
        hipLaunchKernelGGL((quant_pass1_kernel<DT, FMT, true>), dim3((unsigned)ntiles), dim3(kCastThreads), 0, s, x,
                           rows, cols, ldx, bias, used, parts, q, ldq, qT, ldqT, tiles_c, vec_in, vec_q, vec_qT);
    }
    hipLaunchKernelGGL((quant_delayed_finish_kernel<DT, FMT>), dim3(1), dim3(kCastThreads), 0, s, parts, (int)ntiles,
                       used, margin, history, hlen, count, bias, amax_bits, flags);
}

// Host dispatch of (element type, format) to kernel template arguments.
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

template <typename Fn>
void with_dt_fmt(int dt, int fmt, Fn&& fn) {
    if (dt == FP8_DT_BF16)
        with_fmt(fmt, [&](auto F) { fn(IC<FP8_DT_BF16>{}, F); });
    else
        with_fmt(fmt, [&](auto F) { fn(IC<FP8_DT_F32>{}, F); });
}


// ------------------------------------------- segments: one bias per row group
// Segment s holds rows offsets[s] <= r < offsets[s + 1] (one data sample or
// micro-batch).  seg_of(r) is the largest s < nseg with offsets[s] <= r (0 if
// none), so every index stays in [0, nseg) whatever the offsets hold: invalid
// offsets give unspecified biases, never an access out of bounds.
__device__ __forceinline__ int seg_of(const int32_t* __restrict__ off, int nseg, int64_t r) {
    int lo = 0, hi = nseg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((int64_t)off[mid] <= r) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__global__ void fill_words_kernel(uint32_t* __restrict__ p, int64_t n, uint32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// Largest magnitude pattern per segment.  A workgroup of 4 waves takes
// kSegRows consecutive rows, a wave one row at a time (16-byte loads across
// the row); the row maxima are folded by runs of rows of one segment, one
// atomic max per run.
constexpr int kSegRows = 4, kSegThreads = 256;  // one row per wave: a few thousand rows fill the chip

template <int DT>
__global__ __launch_bounds__(kSegThreads) void seg_amax_kernel(const void* __restrict__ x, int64_t rows,
                                                               int64_t cols, int64_t ldx,
                                                               const int32_t* __restrict__ off, int nseg,
                                                               uint32_t* __restrict__ amax, int vec_in) {
    __shared__ uint32_t rmax[kSegRows];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t rb = (int64_t)blockIdx.x * kSegRows;
    constexpr int kPer = DT == FP8_DT_BF16 ? 8 : 4;  // elements per 16 bytes
    for (int i = w; i < kSegRows; i += kSegThreads / 64) {
        const int64_t r = rb + i;
        uint32_t m = 0;
        if (r < rows) {
            if (vec_in) {
                for (int64_t c = (int64_t)lane * kPer; c < cols; c += 64 * kPer) {
                    const uint4 v = *(const uint4*)((const char*)x + (r * ldx + c) * (DT == FP8_DT_BF16 ? 2 : 4));
                    if (DT == FP8_DT_BF16) {
                        us2 mm = fold_bf16(us2{0, 0}, v);
                        m = max(m, (uint32_t)max(mm.x, mm.y));
                    } else {
                        m = fold_f32(m, v);
                    }
                }
            } else {
                for (int64_t c = lane; c < cols; c += 64) m = max(m, elem_mag<DT>(x, r * ldx + c));
            }
        }
        m = wave_max(m);
        if (lane == 0) rmax[i] = m;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const int n = (int)min((int64_t)kSegRows, rows - rb);
        int s = seg_of(off, nseg, rb);
        uint32_t run = 0;
        for (int i = 0; i < n; ++i) {
            const int si = seg_of(off, nseg, rb + i);
            if (si != s) {
                atomicMax(amax + s, canon_amax(DT == FP8_DT_BF16 ? run << 16 : run));
                s = si;
                run = 0;
            }
            run = max(run, rmax[i]);
        }
        if (n > 0) atomicMax(amax + s, canon_amax(DT == FP8_DT_BF16 ? run << 16 : run));
    }
}

// Eq. 3 per segment, and its bias expanded to every row of the segment.
template <int FMT>
__global__ void seg_bias_kernel(const uint32_t* __restrict__ amax, const int32_t* __restrict__ off, int nseg,
                                int64_t rows, int32_t margin, int32_t* __restrict__ bias,
                                uint32_t* __restrict__ flags, int32_t* __restrict__ rowb) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < nseg) {
        uint32_t fl;
        bias[i] = bias_of<FMT>(amax[i], margin, &fl);
        if (flags) flags[i] = fl;
    }
    if (i < rows) {
        uint32_t fl;
        rowb[i] = bias_of<FMT>(amax[seg_of(off, nseg, i)], margin, &fl);
    }
}

template <int DT, int FMT>
__global__ __launch_bounds__(kCastThreads) void cast_rows_kernel(
    const void* __restrict__ x, int64_t rows, int64_t cols, int64_t ldx, const int32_t* __restrict__ rowb,
    uint8_t* __restrict__ q, int64_t ldq, uint8_t* __restrict__ qT, int64_t ldqT, int64_t tiles_c, int vec_in,
    int vec_q, int vec_qT) {
    __shared__ __attribute__((aligned(16))) uint8_t tile[kCastCols * kCastRows];
    cast_tile<DT, FMT, false, true>(x, rows, cols, ldx, 0, q, ldq, qT, ldqT, blockIdx.x / tiles_c,
                                    blockIdx.x % tiles_c, vec_in, vec_q, vec_qT, tile, rowb);
}

template <int DT, int FMT>
void launch_quantise_segments_t(const void* x, int64_t rows, int64_t cols, int64_t ldx, int32_t margin,
                                const int32_t* off, int nseg, int32_t* bias, uint32_t* amax, uint32_t* flags,
                                int32_t* rowb, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT, hipStream_t s) {
    const int esz = DT == FP8_DT_BF16 ? 2 : 4;
    hipLaunchKernelGGL(fill_words_kernel, dim3((unsigned)std::min<int64_t>(((int64_t)nseg + 255) / 256, 1024)), dim3(256), 0, s,
                       amax, (int64_t)nseg, 0u);
    if (rows > 0 && cols > 0) {
        const int vec_in = ((uintptr_t)x % 16 == 0) && ((ldx * esz) % 16 == 0) && ((cols * esz) % 16 == 0);
        hipLaunchKernelGGL((seg_amax_kernel<DT>), dim3((unsigned)((rows + kSegRows - 1) / kSegRows)),
                           dim3(kSegThreads), 0, s, x, rows, cols, ldx, off, nseg, amax, vec_in);
    }
    const int64_t nb = (std::max(rows, (int64_t)nseg) + 255) / 256;
    hipLaunchKernelGGL((seg_bias_kernel<FMT>), dim3((unsigned)nb), dim3(256), 0, s, amax, off, nseg, rows, margin,
                       bias, flags, rowb);
    if (rows > 0 && cols > 0 && (q || qT)) {
        const int64_t tiles_r = (rows + kCastRows - 1) / kCastRows, tiles_c = (cols + kCastCols - 1) / kCastCols;
        const int vec_in = ((uintptr_t)x % 16 == 0) && ((ldx * esz) % 16 == 0);
        const int vec_q = q && ((uintptr_t)q % 8 == 0) && (ldq % 8 == 0);
        const int vec_qT = qT && ((uintptr_t)qT % 16 == 0) && (ldqT % 16 == 0);
        hipLaunchKernelGGL((cast_rows_kernel<DT, FMT>), dim3((unsigned)(tiles_r * tiles_c)), dim3(kCastThreads), 0, s,
                           x, rows, cols, ldx, rowb, q, ldq, qT, ldqT, tiles_c, vec_in, vec_q, vec_qT);
    }
}

// Statistical mode of n biases (most frequent value; the smallest of equally
// frequent ones), appended to a ring buffer: ring[*count % capacity] = mode,
// then *count += 1.  One workgroup; biases outside [-kModeRange, kModeRange)
// are counted at the nearest end of that range.
constexpr int kModeRange = 1024;

__global__ __launch_bounds__(256) void bias_mode_kernel(const int32_t* __restrict__ b, int64_t n,
                                                        int32_t* __restrict__ ring, int64_t capacity,
                                                        uint32_t* __restrict__ count) {
    __shared__ uint32_t hist[2 * kModeRange];
    __shared__ uint64_t best[256];
    for (int i = threadIdx.x; i < 2 * kModeRange; i += 256) hist[i] = 0;
    __syncthreads();
    for (int64_t i = threadIdx.x; i < n; i += 256) {
        const int v = max(-kModeRange, min(kModeRange - 1, b[i]));
        atomicAdd(&hist[v + kModeRange], 1u);
    }
    __syncthreads();
    // key: count in the high bits, (2 kModeRange - 1 - bin) in the low 11, so
    // that the largest key is the most frequent bin, and among equals the lowest
    uint64_t k = 0;
    for (int i = threadIdx.x; i < 2 * kModeRange; i += 256)
        if (hist[i]) k = max(k, ((uint64_t)hist[i] << 11) | (uint64_t)(2 * kModeRange - 1 - i));
    best[threadIdx.x] = k;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (threadIdx.x < off) best[threadIdx.x] = max(best[threadIdx.x], best[threadIdx.x + off]);
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const int bin = 2 * kModeRange - 1 - (int)(best[0] & 0x7FFull);
        const uint32_t c = *count;
        ring[c % (uint64_t)capacity] = bin - kModeRange;
        *count = c + 1;
    }
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
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        hipLaunchKernelGGL((amax_finalize_kernel<decltype(D)::value, decltype(F)::value>), dim3(1), dim3(kAmaxThreads), 0,
                           s, partials, nb, margin, bias, amax_bits, flags);
    });
    return hip_status();
}

int32_t launch_bias_from_amax(const uint32_t* amax_bits, int fmt, int32_t margin, int32_t* bias,
                              uint32_t* flags, hipStream_t s) {
    with_fmt(fmt, [&](auto F) {
        hipLaunchKernelGGL(bias_from_amax_kernel<decltype(F)::value>, dim3(1), dim3(64), 0, s, amax_bits, margin, bias, flags);
    });
    return hip_status();
}

int32_t launch_cast(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                    const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                    hipStream_t s) {
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        launch_cast_t<decltype(D)::value, decltype(F)::value>(x, rows, cols, ldx, bias, q, ldq, qT, ldqT, s);
    });
    return hip_status();
}

int32_t launch_quant_check(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                           int32_t margin, const uint32_t* parts, int nparts, const int32_t* used,
                           int32_t* bias, uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq,
                           uint8_t* qT, int64_t ldqT, hipStream_t s) {
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        launch_quant_check_t<decltype(D)::value, decltype(F)::value>(x, rows, cols, ldx, margin, parts, nparts, used,
                                                                     bias, amax_bits, flags, q, ldq, qT, ldqT, s);
    });
    return hip_status();
}

int32_t launch_quantise_delayed(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                                int32_t margin, int32_t* bias, uint32_t* history, int hlen, uint32_t* count,
                                uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT,
                                int64_t ldqT, uint32_t* ws, hipStream_t s) {
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        launch_quantise_delayed_t<decltype(D)::value, decltype(F)::value>(x, rows, cols, ldx, margin, bias, history,
                                                                          hlen, count, amax_bits, flags, q, ldq, qT,
                                                                          ldqT, ws, s);
    });
    return hip_status();
}

int64_t quantise_ws_words(int64_t rows, int64_t cols) {
    const int64_t tiles = ((rows + kCastRows - 1) / kCastRows) * ((cols + kCastCols - 1) / kCastCols);
    return 1 + tiles;
}

int64_t quantise_tiles_upto(int64_t rows, int64_t cols, int64_t limit) {
    const int64_t tr = (rows + kCastRows - 1) / kCastRows, tc = (cols + kCastCols - 1) / kCastCols;
    if (tr == 0 || tc == 0) return 0;
    if (tr > limit / tc) return -1;
    return tr * tc;
}

int32_t launch_quantise(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                        int32_t margin, const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits,
                        uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                        uint32_t* ws, hipStream_t s) {
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        launch_quantise_t<decltype(D)::value, decltype(F)::value>(x, rows, cols, ldx, margin, bias_pred, bias, amax_bits,
                                                                  flags, q, ldq, qT, ldqT, ws, s);
    });
    return hip_status();
}

int32_t launch_quantise_batch(int n, const QuantDesc* d, int dt, int fmt, int32_t margin, hipStream_t s) {
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        launch_quantise_batch_t<decltype(D)::value, decltype(F)::value>(n, d, margin, s);
    });
    return hip_status();
}

int32_t launch_quantise_segments(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                                 int32_t margin, const int32_t* offsets, int nseg, int32_t* bias, uint32_t* amax_bits,
                                 uint32_t* flags, int32_t* row_bias, uint8_t* q, int64_t ldq, uint8_t* qT,
                                 int64_t ldqT, hipStream_t s) {
    with_dt_fmt(dt, fmt, [&](auto D, auto F) {
        launch_quantise_segments_t<decltype(D)::value, decltype(F)::value>(
            x, rows, cols, ldx, margin, offsets, nseg, bias, amax_bits, flags, row_bias, q, ldq, qT, ldqT, s);
    });
    return hip_status();
}

int32_t launch_bias_mode(const int32_t* bias, int64_t n, int32_t* ring, int64_t capacity, uint32_t* count,
                         hipStream_t s) {
    hipLaunchKernelGGL(bias_mode_kernel, dim3(1), dim3(256), 0, s, bias, n, ring, capacity, count);
    return hip_status();
}

}  // namespace fp8lin
