// FP8 x FP8 -> fp32 matmul with the unscale 2^-(b_a + b_b) fused into the
// epilogue (Sec. 2 and 2.2; Eq. 2), for gfx950 matrix cores.
//
// C[m, n] = 2^-(ba + bb) * sum_k A[m, k] * B[n, k]   ("NT": both operands
// are contiguous along the contraction index).  The forward pass, the
// grad-input and the grad-weight products of the linear layer are all of
// this form once the casts have written the transposed copies they need.
//
// Main kernel (K a multiple of 128, 16-byte aligned operands):
//  * 256 x 256 output tile per workgroup of 8 waves, two per SIMD (wave w
//    runs on SIMD w % 4).  Each wave owns a 64 x 128 sub-tile = 4 x 8 blocks
//    of v_mfma_f32_16x16x128_f8f6f4; the two waves of a SIMD own the two
//    halves of one 128 x 128 quadrant.
//  * K advances 128 bytes at a time; both operand tiles (256 rows x 128 B)
//    go HBM/L2 -> LDS with global_load_lds_dwordx4 (no VGPR staging): A into
//    two stages, B into three (all 160 KiB of LDS).
//  * The copies are slow to issue (the L1 holds only so many outstanding
//    fills): group 0 copies the A tiles and group 1 the B tiles, each in its
//    own load phase, so both load phases share the cost.
//  * The two waves of a SIMD alternate between an MFMA phase and a load
//    phase, the phases separated by workgroup barriers: while one issues its
//    32 MFMAs of step k, the other reads all its fragments of its next step
//    into registers and issues the copies of its operand for a later step.
//    The matrix core of each SIMD is fed by one wave at a time, and the
//    cost of issuing vector-memory and LDS instructions falls on the wave
//    that is not feeding it (see the main loop).
//  * LDS rows are 128 B; the 16-byte chunk index is XOR-swizzled with the row
//    (chunk ^ chunk_swz(row), below) by choosing which global chunk each lane
//    fetches.  The LDS has 64 four-byte banks (16 groups of 16 bytes) and
//    serves a ds_read_b128 in four phases of 16 lanes: lane bit 5 and the
//    parity of lane bits 2, 3 and 4 select the phase (measured on gfx950 with
//    a sweep of address patterns; lanes 0-15 are NOT one phase).  The swizzle
//    gives the 16 lanes of every phase of a fragment read distinct bank groups.
//  * A fragment of the 16x16x128 MFMA is 32 bytes per lane: row (lane % 16),
//    32 consecutive k of group (lane / 16).  The matrix core pairs the same
//    register bytes of both operands, so any k order that is the same for
//    both operands gives the same dot products.
//  * The MFMA gets the B fragment as its first operand, so each lane's four
//    accumulators are four consecutive n of one m: the epilogue writes 8 B
//    (bf16) or 16 B (fp32) per lane.
//  * Workgroup -> tile mapping: workgroups are dealt round-robin to the 8
//    XCDs; the remap gives each XCD a contiguous range of tiles, walked in
//    groups of 8 tile-rows, so tiles sharing operand panels meet in the same
//    L2.
// Decode kernel (M <= 32): weight-streaming split-K, see below.
// Fallback kernel (K not a multiple of 128, or K >= 2^22): 64 x 64 tiles,
// 16-byte loads when K is a multiple of 16 and byte loads otherwise, with
// bounds checks and zero fill, same MFMA and epilogue.
#include "fp8lin_fp8.h"
#include "fp8lin_internal.h"

namespace fp8lin {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

// MFMA operand format selectors: 0 = fp8 (E4M3), 1 = bf8 (E5M2).
template <int F0, int F1>
__device__ __forceinline__ v4f mfma16(v8i a, v8i b, v4f c) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, F0, F1, 0, 0, 0, 0);
}

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, 64));
    return v;
}

// 32-bit LDS address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// Wait until every LDS read of this wave has returned its data.
__device__ __forceinline__ void wait_lgkmcnt0() { asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory"); }

// Workgroup barrier with no memory fence: the main loop orders its LDS
// traffic itself (wait_vmcnt for the copies, wait_lgkmcnt0 for the reads).
__device__ __forceinline__ void ws_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// The two 16-byte pieces of an MFMA operand fragment, as one 8-register vector.
__device__ __forceinline__ v8i ld_frag(const uint8_t* p, int fo0, int fo1) {
    const uint4 p0 = *(const uint4*)(p + fo0);
    const uint4 p1 = *(const uint4*)(p + fo1);
    return v8i{(int)p0.x, (int)p0.y, (int)p0.z, (int)p0.w, (int)p1.x, (int)p1.y, (int)p1.z, (int)p1.w};
}

// Physical 16-byte chunk of logical chunk c in LDS operand row r is
// c ^ chunk_swz(r).  A fragment read has lane l on row r = l % 16 (row bit 0
// picks the half of a 256-byte bank line) and logical chunk 2 (l / 16) + piece.
// Within one phase (fixed lane bit 5 and parity of lane bits 2..4) the map
// (r1, r2, r3) -> (r1 ^ piece, parity ^ r3, bit 5 ^ r2) of the three chunk bits
// is one-to-one, so the 16 lanes hit 16 distinct bank groups.
__device__ __forceinline__ int chunk_swz(int r) { return ((r >> 1) & 1) | (((r >> 2) & 1) << 2); }

// Contiguous tile ranges per XCD, then grouped row-major order inside.
__device__ __forceinline__ void tile_of(int b, int nb, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int x = b & 7, l = b >> 3;
    const int per = nb >> 3, rem = nb & 7;
    const int t = x * per + min(x, rem) + l;
    constexpr int G = 8;
    const int group = G * tiles_n;
    const int gid = t / group;
    const int first = gid * G;
    const int gm = min(tiles_m - first, G);
    const int r = t - gid * group;
    tm = first + r % gm;
    tn = r / gm;
}

// Store 4 consecutive outputs of row m starting at column n (unscaled by
// 2^-sh); returns the largest output magnitude pattern (as fp32 bits).
template <int OUT_DT>
__device__ __forceinline__ uint32_t store4(void* C, int64_t ldc, int64_t m, int64_t n, int64_t M,
                                           int64_t N, v4f acc, int sh, bool vec) {
    float y[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) y[v] = ldexpf(acc[v], sh);
    uint32_t mx = 0;
    if (OUT_DT == FP8_DT_BF16) {
        uint32_t h[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            h[v] = f32_to_bf16_rne(y[v]);
            mx = max(mx, (h[v] & 0x7FFFu) << 16);
        }
        if (m < M) {
            uint16_t* p = (uint16_t*)C + m * ldc + n;
            if (vec && n + 3 < N) {
                *(uint2*)p = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
            } else {
                for (int v = 0; v < 4; ++v)
                    if (n + v < N) p[v] = (uint16_t)h[v];
            }
        }
    } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) mx = max(mx, __float_as_uint(y[v]) & 0x7FFFFFFFu);
        if (m < M) {
            float* p = (float*)C + m * ldc + n;
            if (vec && n + 3 < N) {
                *(float4*)p = make_float4(y[0], y[1], y[2], y[3]);
            } else {
                for (int v = 0; v < 4; ++v)
                    if (n + v < N) p[v] = y[v];
            }
        }
    }
    return m < M ? mx : 0u;
}

// Unscale exponent of output row m (of M): -(ba + bb), with ba of row m when
// ba_rows (per-row activation biases, one per data sample or segment).
__device__ __forceinline__ int row_shift(const int32_t* ba_p, int ba_rows, int bb, int64_t m, int64_t M) {
    return -((ba_rows ? ba_p[min(m, M - 1)] : ba_p[0]) + bb);
}

// ------------------------------------------------------------ main kernel
constexpr int kBM = 256, kBN = 256, kBK = 128, kThreads = 256;
constexpr int kMainThreads = 512;      // 8 waves: two groups of four
constexpr int kTileBytes = kBM * kBK;  // one operand tile, 32 KiB

// Direct L2 -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4, the
// form with a wave-uniform 64-bit base in SGPRs and a 32-bit lane offset):
// lane i's 16 bytes land at lds_row + 16 i; lds_row must be wave-uniform.
// The instruction is issued from inline assembly so that the compiler does
// not treat every later LDS read as dependent on it (it cannot tell the two
// halves of the double buffer apart and would wait for the prefetch before
// each read); completion is tracked with wait_vmcnt.
__device__ __forceinline__ void lds_dma16_s(const uint8_t* sbase, uint32_t voff, uint32_t lds_row) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(lds_row), "v"(voff), "s"(sbase)
                 : "memory");
}

// The same copy with the non-temporal hint (a stream read once).
__device__ __forceinline__ void lds_dma16_nt(const uint8_t* sbase, uint32_t voff, uint32_t lds_row) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
                 :
                 : "s"(lds_row), "v"(voff), "s"(sbase)
                 : "memory");
}

__device__ __forceinline__ int bq_used(const int32_t* pred) { return clamp_bias(*pred); }

// 16-byte store of matmul output with the non-temporal hint: the output is not
// read again by this kernel and should not displace cached operands.
__device__ __forceinline__ void st_stream(void* p, uint4 v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, (u32x4*)p);
}

// Epilogue staging rows (bytes): 32 output rows of a wave per pass; the
// codes of the fused quantise (256 x 256 bytes) follow the bf16 staging area.
constexpr int kEpRowBf16 = 128 * 2 + 16, kEpRowF32 = 128 * 4 + 16;
constexpr int kEpBf16Bytes = 8 * 32 * kEpRowBf16, kEpF32Bytes = 8 * 32 * kEpRowF32;
constexpr int kCodesOff = kEpBf16Bytes;
constexpr int kEpBytes = kCodesOff + kBM * kBN > kEpF32Bytes ? kCodesOff + kBM * kBN : kEpF32Bytes;
// Main loop: two A stages and three B stages (B tiles are copied two steps
// ahead, see gemm_tile); the epilogue reuses the space, and the workgroup's
// amax words sit in its last 64 bytes, past every epilogue staging area.
constexpr int kSmemBytes = 2 * kTileBytes + 3 * kBN * kBK;
constexpr int kWmxOff = kSmemBytes - 64;
static_assert(kEpBytes <= kWmxOff && kSmemBytes <= 160 * 1024, "LDS budget");
static_assert(kCodesOff % 16 == 0, "codes staging alignment");

// Output codes of the fused quantise (QF >= 0, bf16 output only): Y8 [M, N]
// and optionally Y8T [N, M] in format QF, cast with a predicted bias; the
// tile maxima and the prediction used go to a workspace for the exact-bias
// check (see launch_gemm_nt_quantise).
struct QuantOut {
    const int32_t* pred;  // predicted bias (device)
    int32_t* used;        // out: the clamped prediction the codes were cast with
    uint32_t* parts;      // out: per-workgroup largest |Y| pattern (bf16 bits)
    uint8_t* y8;
    int64_t ldy8;
    uint8_t* y8t;  // may be null
    int64_t ldy8t;
    int vec8, vec8t;  // 16-byte stores allowed
};

// Eq. 3 bias of the output taken in the same launch (ws != nullptr): every
// workgroup folds its largest |Y| pattern into ws[0] and then counts itself
// in ws[1]; the last one to count takes the total, writes amax, bias and
// flags, and leaves both words zero for the next call.
struct BiasOut {
    int32_t* bias;
    uint32_t* flags;  // may be null
    uint32_t* ws;     // [0] running maximum, [1] finished workgroups; zero between calls
    int fmt;
    int32_t margin;
};

__device__ __forceinline__ int32_t bias_of_fmt(int fmt, uint32_t a, int32_t margin, uint32_t* fl) {
    switch (fmt) {
        case FP8_E4M3: return bias_of<FP8_E4M3>(a, margin, fl);
        case FP8_E5M2: return bias_of<FP8_E5M2>(a, margin, fl);
        case FP8_E4_A: return bias_of<FP8_E4_A>(a, margin, fl);
        default: return bias_of<FP8_E5_A>(a, margin, fl);
    }
}

// One output tile of 256 rows x TN columns (TN = 64..256; each wave owns 64
// rows x TN/2 columns), tile number bid of nb in this workgroup's share of the
// launch, over columns [col0, col0 + tiles_n TN) of C.  The last workgroup of
// the launch takes the bias when bo.ws is set.
template <int FA, int FB, int OUT_DT, bool AMAX, int QF, int TN>
__device__ __forceinline__ void gemm_tile(
    uint8_t* __restrict__ smem, int bid, int nb, const uint8_t* __restrict__ A, const uint8_t* __restrict__ B,
    const int32_t* __restrict__ ba_p, const int32_t* __restrict__ bb_p, void* __restrict__ C, int M, int N, int K,
    int tiles_m, int tiles_n, int col0, int vec_out, uint32_t* __restrict__ amax_out, const QuantOut& qo,
    const BiasOut& bo, int ba_rows) {
    static_assert(QF < 0 || OUT_DT == FP8_DT_BF16, "fused quantise is for bf16 outputs");
    static_assert(QF < 0 || TN == 256, "fused quantise stages whole 256 x 256 tiles");
    static_assert(TN % 64 == 0 && TN >= 64 && TN <= 256, "tile width");
    constexpr int kNbw = TN / 32;                  // 16-column blocks per wave, B copies per loader wave
    constexpr int kBStage = TN * kBK;              // one B tile in LDS
    constexpr int kNf = 4 + kNbw;                  // fragment pieces a wave reads per step
    constexpr int kNc = 8 + kNbw;                  // copies a loader wave issues per stage

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // group (0: waves 0-3, 1: waves 4-7) and quadrant; wave-uniform
    const int g = __builtin_amdgcn_readfirstlane(w >> 2), sq = __builtin_amdgcn_readfirstlane(w & 3);
    int tm, tn;
    tile_of(bid, nb, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * kBM, n0 = col0 + tn * TN;

    // Loader (group 0): wave sq fills rows [64 sq, 64 sq + 64) of the A tile
    // and [TN/4 sq, TN/4 (sq + 1)) of the B tile, 8 rows per copy (voff[0..7]
    // for A, voff[8..] for B); lane -> row r = (first row) + 8 i + lane / 8 and
    // physical chunk lane % 8, which holds logical chunk (lane % 8) ^
    // chunk_swz(r).  Rows past the matrix edge re-read the last row (their
    // outputs are not stored).  Offsets are relative to the tile's first row,
    // so they fit 32 bits for K < 2^22.
    const int lrow = lane >> 3;
    uint32_t voff[kNc];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = sq * 64 + i * 8 + lrow;
        voff[i] = (uint32_t)((min(m0 + r, M - 1) - m0) * K + ((lane & 7) ^ chunk_swz(r)) * 16);
    }
#pragma unroll
    for (int i = 0; i < kNbw; ++i) {
        const int r = sq * (TN / 4) + i * 8 + lrow;
        voff[8 + i] = (uint32_t)((min(n0 + r, N - 1) - n0) * K + ((lane & 7) ^ chunk_swz(r)) * 16);
    }
    const uint8_t* baseA = A + (int64_t)m0 * K;
    const uint8_t* baseB = B + (int64_t)n0 * K;
    // LDS addresses of this wave's first loader rows (wave-uniform); copy d
    // < 8 fills A row group d, copy d >= 8 B row group d - 8.
    // LDS: A stages 0 and 1 at s * kTileBytes, B stages 0, 1 and 2 after them.
    const uint32_t lds_a = __builtin_amdgcn_readfirstlane(lds_addr(smem) + sq * 64 * kBK);
    const uint32_t lds_b = __builtin_amdgcn_readfirstlane(lds_addr(smem) + 2 * kTileBytes + sq * (TN / 4) * kBK);
    auto dma = [&](int d, int stage, int k0) {  // stage: of A for d < 8, of B for d >= 8
        lds_dma16_s((d >= 8 ? baseB : baseA) + k0, voff[d],
                    d >= 8 ? lds_b + (d - 8) * 8 * kBK + stage * kBStage : lds_a + d * 8 * kBK + stage * kTileBytes);
    };

    // this wave's sub-tile: rows [wr0, wr0 + 64), columns [wc0, wc0 + TN/2) of the tile
    const int wr0 = (sq >> 1) * 128 + g * 64, wc0 = (sq & 1) * (TN / 2);
    const int frow = lane & 15, fg = lane >> 4;
    // byte offsets (within a 16-row block) of this lane's two fragment pieces
    const int fo0 = frow * kBK + (((2 * fg) ^ chunk_swz(frow)) << 4);
    const int fo1 = frow * kBK + (((2 * fg + 1) ^ chunk_swz(frow)) << 4);

    v4f acc[4][kNbw];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < kNbw; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // Ping-pong pipeline.  Phases are separated by workgroup barriers; in
    // every phase one group issues MFMAs and the other loads:
    //   phase 1:        group 0 loads fragments of step 0
    //   phase 2k + 2:   group 0 MFMAs of step k,   group 1 loads step k
    //   phase 2k + 3:   group 0 loads step k + 1,  group 1 MFMAs of step k
    // A load phase reads all kNf fragment pieces of the wave's next step and
    // waits for them before the barrier.  A tile k sits in A stage k % 2, B
    // tile k in B stage k % 3.  Group 0 copies A tile k + 1 in its load phase
    // of step k (after both groups have read A tile k - 1 from that stage) and
    // waits for the copies at the end of its next MFMA phase.  Group 1 copies
    // B tile k + 2 in its load phase of step k (B tile k - 1 has been read by
    // then) and, before that phase's barrier, waits for B tile k + 1 — issued
    // one load phase earlier — but not for the copies it has just issued.
    // Steps 0 and 1 are copied before phase 1.  Every wave passes 2 nk + 1
    // barriers (group 1 passes one before its first load phase and none after
    // its last MFMA phase), so the groups stay in step.
    const int nk = K / kBK;
    if (nk > 0) {
        if (g == 0) {
#pragma unroll
            for (int d = 0; d < 8; ++d) dma(d, 0, 0);
            if (nk > 1) {
#pragma unroll
                for (int d = 0; d < 8; ++d) dma(d, 1, kBK);
                wait_vmcnt<8>();
            } else {
                wait_vmcnt<0>();
            }
        } else {
#pragma unroll
            for (int d = 8; d < kNc; ++d) dma(d, 0, 0);
            if (nk > 1) {
#pragma unroll
                for (int d = 8; d < kNc; ++d) dma(d, 1, kBK);
                wait_vmcnt<kNbw>();
            } else {
                wait_vmcnt<0>();
            }
        }
        ws_barrier();
        if (g == 1) ws_barrier();
    }
    v8i af[4], bf[kNbw];
    int bs = 0;  // k % 3: the B stage of step k
    for (int kt = 0; kt < nk; ++kt) {
        const uint8_t* sa = smem + (kt & 1) * kTileBytes + wr0 * kBK;
        const uint8_t* sb = smem + 2 * kTileBytes + bs * kBStage + wc0 * kBK;
        if (g == 0 && kt >= 1 && kt + 1 < nk) {
            // A tile of step kt + 1, the copies spread over the fragment reads
            const int st = (kt + 1) & 1, k1 = (kt + 1) * kBK;
#pragma unroll
            for (int q = 0; q < kNf; ++q) {
                if (q < 4) af[q] = ld_frag(sa + q * 16 * kBK, fo0, fo1);
                else bf[q - 4] = ld_frag(sb + (q - 4) * 16 * kBK, fo0, fo1);
                if (q < 8) dma(q, st, k1);
            }
#pragma unroll
            for (int d = kNf; d < 8; ++d) dma(d, st, k1);
        } else if (g == 1 && kt + 2 < nk) {
            // B tile of step kt + 2 into the stage B tile kt - 1 used
            const int st = bs == 0 ? 2 : bs - 1, k2 = (kt + 2) * kBK;
#pragma unroll
            for (int q = 0; q < kNf; ++q) {
                if (q < 4) af[q] = ld_frag(sa + q * 16 * kBK, fo0, fo1);
                else bf[q - 4] = ld_frag(sb + (q - 4) * 16 * kBK, fo0, fo1);
                if (q < kNbw) dma(8 + q, st, k2);
            }
        } else {
#pragma unroll
            for (int q = 0; q < kNf; ++q) {
                if (q < 4) af[q] = ld_frag(sa + q * 16 * kBK, fo0, fo1);
                else bf[q - 4] = ld_frag(sb + (q - 4) * 16 * kBK, fo0, fo1);
            }
        }
        if (g == 1) {  // B tile kt + 1 has landed (the copies just issued need not have)
            if (kt + 2 < nk) wait_vmcnt<kNbw>();
            else wait_vmcnt<0>();
        }
        bs = bs == 2 ? 0 : bs + 1;
        wait_lgkmcnt0();
        ws_barrier();
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < kNbw; ++j) {
                acc[i][j] = mfma16<FB, FA>(bf[j], af[i], acc[i][j]);
                __builtin_amdgcn_sched_barrier(0);
            }
        if (g == 0) {
            wait_vmcnt<0>();
            ws_barrier();
        } else if (kt + 1 < nk) {
            ws_barrier();
        }
    }

    // Epilogue: y = 2^-(ba + bb) acc (exact ldexp), rounded once to the output
    // type, staged through LDS 32 rows at a time per wave so that every global
    // store writes 16-byte pieces of whole 256-byte (bf16) or 512-byte (fp32)
    // row runs.  Staging reads map one LDS read phase (lane bit 5 and the
    // parity of lane bits 2..4) to one row, so they are free of bank conflicts.
    // The last barrier of the main loop follows every read of the operand
    // tiles, so group 0 stages and stores its outputs while group 1 issues its
    // last MFMAs.
    int shr[4];  // unscale exponent of this lane's rows wr0 + 16 i + frow
#pragma unroll
    for (int i = 0; i < 4; ++i) shr[i] = row_shift(ba_p, ba_rows, *bb_p, (int64_t)m0 + wr0 + i * 16 + frow, M);
    const int prow = 2 * (lane >> 5) + (((lane >> 2) ^ (lane >> 3) ^ (lane >> 4)) & 1);
    uint32_t mx = 0;
    if (OUT_DT == FP8_DT_BF16) {
        uint8_t* ep = smem + w * 32 * kEpRowBf16;
        typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
        u16x2 m2 = {0, 0};
        // Fused quantise: the codes of the tile, row-major, after the staging
        // rows (row r = 256 bytes; 16-byte chunk c stored at chunk c ^ (r % 16)).
        uint8_t* cs = smem + kCodesOff;
        int bq = 0;
        uint32_t codes[4][8];
        if (QF >= 0) bq = clamp_bias(*qo.pred);
#pragma unroll
        for (int i2 = 0; i2 < 2; ++i2) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * i2 + ii;
#pragma unroll
                for (int j = 0; j < kNbw; ++j) {
                    const uint32_t lo = pack_bf16x2(ldexpf(acc[i][j][0], shr[i]), ldexpf(acc[i][j][1], shr[i]));
                    const uint32_t hi = pack_bf16x2(ldexpf(acc[i][j][2], shr[i]), ldexpf(acc[i][j][3], shr[i]));
                    if (AMAX || QF >= 0) {
                        m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(u16x2, lo & 0x7FFF7FFFu));
                        m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(u16x2, hi & 0x7FFF7FFFu));
                    }
                    if (QF >= 0) {
                        uint32_t c4 = cast4_bf16<QF < 0 ? 0 : QF>(lo, hi, bq);
                        if (__builtin_expect(any_nan_bf16(lo, hi), 0)) {
                            const uint32_t hs[4] = {lo & 0xFFFFu, lo >> 16, hi & 0xFFFFu, hi >> 16};
                            c4 = nan_patch<QF < 0 ? 0 : QF>(c4, hs);
                        }
                        codes[i][j] = c4;
                        const int r = wr0 + i * 16 + frow, col = wc0 + j * 16 + 4 * fg;
                        *(uint32_t*)(cs + r * 256 + ((((col >> 4) ^ r) & 15) << 4) + (col & 15)) = c4;
                    }
                    *(uint2*)(ep + (ii * 16 + frow) * kEpRowBf16 + (j * 16 + 4 * fg) * 2) = make_uint2(lo, hi);
                }
            }
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int row = 4 * t + prow, c16 = lane & 15;
                const uint4 v = *(const uint4*)(ep + row * kEpRowBf16 + c16 * 16);
                const int64_t m = m0 + wr0 + i2 * 32 + row, n = n0 + wc0 + c16 * 8;
                if (m < M && c16 < TN / 16) {
                    uint16_t* p = (uint16_t*)C + m * N + n;
                    if (vec_out && n + 8 <= N) {
                        st_stream(p, v);
                    } else {
                        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
                        for (int e = 0; e < 8 && n + e < N; ++e) p[e] = (uint16_t)(wv[e >> 1] >> (16 * (e & 1)));
                    }
                }
            }
        }
        mx = (uint32_t)max(m2.x, m2.y) << 16;
        if (QF >= 0) {
            // Y8 rows from the staged codes: 4096 chunks of 16 bytes, 8 per thread.
            __syncthreads();
#pragma unroll
            for (int h = 0; h < 8; ++h) {
                const int idx = threadIdx.x + h * kMainThreads, r = idx >> 4, c = idx & 15;
                const uint4 v = *(const uint4*)(cs + r * 256 + (((c ^ r) & 15) << 4));
                const int64_t m = m0 + r, n = n0 + c * 16;
                if (m < M && n < N) {
                    uint8_t* p = qo.y8 + m * qo.ldy8 + n;
                    if (qo.vec8 && n + 16 <= N) {
                        *(uint4*)p = v;
                    } else {
                        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
                        for (int e = 0; e < 16 && n + e < N; ++e) p[e] = (uint8_t)(wv[e >> 2] >> (8 * (e & 3)));
                    }
                }
            }
            if (qo.y8t) {
                // Y8T: restage the codes column-major (column c = 256 bytes of
                // rows; chunk q of column c stored at chunk q ^ (c % 16)).
                __syncthreads();
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int r = wr0 + i * 16 + frow, col0 = wc0 + j * 16 + 4 * fg;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int c = col0 + e;
                            cs[c * 256 + ((((r >> 4) ^ c) & 15) << 4) + (r & 15)] = (uint8_t)(codes[i][j] >> (8 * e));
                        }
                    }
                __syncthreads();
#pragma unroll
                for (int h = 0; h < 8; ++h) {
                    const int idx = threadIdx.x + h * kMainThreads, c = idx >> 4, q = idx & 15;
                    const uint4 v = *(const uint4*)(cs + c * 256 + (((q ^ c) & 15) << 4));
                    const int64_t n = n0 + c, m = m0 + q * 16;
                    if (n < N && m < M) {
                        uint8_t* p = qo.y8t + n * qo.ldy8t + m;
                        if (qo.vec8t && m + 16 <= M) {
                            *(uint4*)p = v;
                        } else {
                            const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
                            for (int e = 0; e < 16 && m + e < M; ++e) p[e] = (uint8_t)(wv[e >> 2] >> (8 * (e & 3)));
                        }
                    }
                }
            }
        }
    } else {
        uint8_t* ep = smem + w * 32 * kEpRowF32;
#pragma unroll
        for (int i2 = 0; i2 < 2; ++i2) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * i2 + ii;
#pragma unroll
                for (int j = 0; j < kNbw; ++j) {
                    float y[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        y[v] = ldexpf(acc[i][j][v], shr[i]);
                        if (AMAX) mx = max(mx, __float_as_uint(y[v]) & 0x7FFFFFFFu);
                    }
                    *(float4*)(ep + (ii * 16 + frow) * kEpRowF32 + (j * 16 + 4 * fg) * 4) =
                        make_float4(y[0], y[1], y[2], y[3]);
                }
            }
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int row = 2 * t + (lane >> 5), c32 = lane & 31;
                const float4 v = *(const float4*)(ep + row * kEpRowF32 + c32 * 16);
                const int64_t m = m0 + wr0 + i2 * 32 + row, n = n0 + wc0 + c32 * 4;
                if (m < M && c32 < TN / 8) {
                    float* p = (float*)C + m * N + n;
                    if (vec_out && n + 4 <= N) {
                        st_stream(p, make_uint4(__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)));
                    } else {
                        const float fv[4] = {v.x, v.y, v.z, v.w};
                        for (int e = 0; e < 4 && n + e < N; ++e) p[e] = fv[e];
                    }
                }
            }
        }
    }
    if (AMAX || QF >= 0) {
        // The workgroup's largest |Y| pattern: one global atomic per workgroup
        // (the waves of all resident workgroups finish together, and atomics
        // on one word from every wave would queue behind each other).  Rows
        // and columns past the edge computed clamped copies of real ones, so
        // including them cannot change the maximum.
        uint32_t* wmx = (uint32_t*)(smem + kWmxOff);
        const uint32_t wv = wave_max_u32(mx);
        if (lane == 0) wmx[w] = wv;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t b = 0;
#pragma unroll
            for (int v = 0; v < kMainThreads / 64; ++v) b = max(b, wmx[v]);
            const uint32_t bc = canon_amax(b);  // the fold and the atomics take canonical NaNs
            if (AMAX && !bo.ws) atomicMax(amax_out, bc);
            if (AMAX && bo.ws) {
                // The fold is a returning device-scope atomic whose result is
                // consumed by an asm statement that also clobbers memory: the
                // compiler cannot move the count above it, and the hardware
                // has performed the fold (the wait for its return) before the
                // count is issued.  The workgroup that counts last therefore
                // finds every fold in ws[0].  A release/acquire count would
                // say the same in the language's terms, but at agent scope
                // its release writes back the XCD's L2 in every workgroup's
                // epilogue (2-6 % slower on launches of several rounds).
                const uint32_t prev = __hip_atomic_fetch_max(bo.ws, bc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                asm volatile("; fold returned %0" : : "v"(prev) : "memory");
                const uint32_t done = __hip_atomic_fetch_add(bo.ws + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (done == gridDim.x - 1) {
                    const uint32_t a = __hip_atomic_exchange(bo.ws, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(bo.ws + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    uint32_t fl;
                    *bo.bias = bias_of_fmt(bo.fmt, a, bo.margin, &fl);
                    if (amax_out) *amax_out = a;
                    if (bo.flags) *bo.flags = fl;
                }
            }
            if (QF >= 0) {  // bf16 magnitude pattern
                qo.parts[blockIdx.x] = b >> 16;
                if (blockIdx.x == 0) *qo.used = bq_used(qo.pred);
            }
        }
    }
}

// The 256-row kernel.  Workgroups below g1 take 256 x 256 tiles (tiles_m x
// tiles_n of them); with TN2 > 0 the rest take tiles TN2 wide over the
// columns after them (tiles_m x tiles_n2), a last round of narrower tiles
// instead of a partial round of full ones (see narrow_split).  g1 is a whole
// number of rounds of 8 workgroups per XCD, so both parts keep their XCD
// layout.
template <int FA, int FB, int OUT_DT, bool AMAX, int QF = -1, int TN2 = 0>
__global__ __launch_bounds__(kMainThreads) void gemm_nt_256(
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ B, const int32_t* __restrict__ ba_p,
    const int32_t* __restrict__ bb_p, void* __restrict__ C, int M, int N, int K, int tiles_m,
    int tiles_n, int vec_out, uint32_t* __restrict__ amax_out, QuantOut qo, BiasOut bo, int ba_rows,
    int g1, int tiles_n2) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmemBytes];
    const int b = blockIdx.x;
    if (TN2 == 0 || b < g1)
        gemm_tile<FA, FB, OUT_DT, AMAX, QF, 256>(smem, b, TN2 == 0 ? (int)gridDim.x : g1, A, B, ba_p, bb_p, C, M, N,
                                                 K, tiles_m, tiles_n, 0, vec_out, amax_out, qo, bo, ba_rows);
    else
        gemm_tile<FA, FB, OUT_DT, AMAX, -1, (TN2 > 0 ? TN2 : 256)>(smem, b - g1, (int)gridDim.x - g1, A, B, ba_p,
                                                                   bb_p, C, M, N, K, tiles_m, tiles_n2, tiles_n * kBN,
                                                                   vec_out, amax_out, qo, bo, ba_rows);
}

// ------------------------------------------------------------ fallback kernel
constexpr int kSBM = 64, kSBN = 64;

template <int FA, int FB, int OUT_DT, bool AMAX>
__global__ __launch_bounds__(kThreads) void gemm_nt_small(
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ B, const int32_t* __restrict__ ba_p,
    const int32_t* __restrict__ bb_p, void* __restrict__ C, int64_t M, int64_t N, int64_t K,
    int64_t tiles_n, int vec_out, uint32_t* __restrict__ amax_out, int ba_rows) {
    __shared__ __attribute__((aligned(16))) uint8_t sa[kSBM * kBK];
    __shared__ __attribute__((aligned(16))) uint8_t sb[kSBN * kBK];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t m0 = (blockIdx.x / tiles_n) * kSBM, n0 = (blockIdx.x % tiles_n) * kSBN;
    // loader: thread -> row (tid / 4), logical chunks 2 (tid % 4), +1
    const int lr = threadIdx.x >> 2, lq = threadIdx.x & 3;
    const int wm = w >> 1, wn = w & 1;
    const int frow = lane & 15, fg = lane >> 4;
    const int fo0 = frow * kBK + (((2 * fg) ^ chunk_swz(frow)) << 4);
    const int fo1 = frow * kBK + (((2 * fg + 1) ^ chunk_swz(frow)) << 4);

    v4f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // K a multiple of 16 with 16-byte aligned operands: every row starts on a
    // 16-byte boundary and each 16-byte chunk lies wholly inside or wholly
    // past the row, so chunks are loaded whole (zero past the row end).
    const bool v16 = (K & 15) == 0 && (((uintptr_t)A | (uintptr_t)B) & 15) == 0;
    for (int64_t k0 = 0; k0 < K; k0 += kBK) {
#pragma unroll
        for (int op = 0; op < 2; ++op) {
            const uint8_t* src = op == 0 ? A : B;
            const int64_t r = (op == 0 ? m0 : n0) + lr;
            const int64_t rmax = op == 0 ? M : N;
            uint8_t* dst = op == 0 ? sa : sb;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int c = 2 * lq + h;  // logical 16-byte chunk
                uint4 v = make_uint4(0, 0, 0, 0);
                if (v16) {
                    const int64_t k = k0 + c * 16;
                    if (r < rmax && k < K) v = *(const uint4*)(src + r * K + k);
                } else {
                    uint32_t wv[4] = {0, 0, 0, 0};
                    for (int t = 0; t < 16; ++t) {
                        const int64_t k = k0 + c * 16 + t;
                        uint32_t byte = 0;
                        if (r < rmax && k < K) byte = src[r * K + k];
                        wv[t >> 2] |= byte << (8 * (t & 3));
                    }
                    v = make_uint4(wv[0], wv[1], wv[2], wv[3]);
                }
                *(uint4*)(dst + lr * kBK + ((c ^ chunk_swz(lr)) << 4)) = v;
            }
        }
        __syncthreads();
        v8i bf[2], af[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const uint8_t* p = sb + (wn * 32 + j * 16) * kBK;
            const uint4 p0 = *(const uint4*)(p + fo0), p1 = *(const uint4*)(p + fo1);
            bf[j] = v8i{(int)p0.x, (int)p0.y, (int)p0.z, (int)p0.w, (int)p1.x, (int)p1.y, (int)p1.z, (int)p1.w};
            const uint8_t* q = sa + (wm * 32 + j * 16) * kBK;
            const uint4 q0 = *(const uint4*)(q + fo0), q1 = *(const uint4*)(q + fo1);
            af[j] = v8i{(int)q0.x, (int)q0.y, (int)q0.z, (int)q0.w, (int)q1.x, (int)q1.y, (int)q1.z, (int)q1.w};
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = mfma16<FB, FA>(bf[j], af[i], acc[i][j]);
        __syncthreads();
    }

    uint32_t mx = 0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t m = m0 + wm * 32 + i * 16 + frow;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 32 + j * 16 + fg * 4;
            if (n < N) mx = max(mx, store4<OUT_DT>(C, N, m, n, M, N, acc[i][j], row_shift(ba_p, ba_rows, *bb_p, m, M), vec_out != 0));
        }
    }
    if (AMAX) {
        mx = wave_max_u32(mx);
        if (lane == 0) atomicMax(amax_out, canon_amax(mx));
    }
}


// ------------------------------------------------------------ decode kernel
// M <= 32 (token-by-token inference): the product is bound by streaming B
// (the FP8 weight, N x K bytes) from HBM once.  A workgroup of kDecWaves
// waves owns NB 16-column blocks; wave w takes a contiguous slice of the K
// range, reads its operand fragments straight from global memory into
// registers (three 128-byte k-steps in flight), and the partial sums of the
// waves are added in LDS in a fixed order, so the result does not depend on
// timing.

__device__ __forceinline__ v8i ld_frag_g(const uint8_t* p) {
    const uint4 p0 = *(const uint4*)p;
    const uint4 p1 = *(const uint4*)(p + 16);
    return v8i{(int)p0.x, (int)p0.y, (int)p0.z, (int)p0.w, (int)p1.x, (int)p1.y, (int)p1.z, (int)p1.w};
}

// The same with the non-temporal hint, for the weight stream: each weight
// byte is read once per call, and keeping it out of the caches leaves them to
// the activation rows every workgroup shares (+38 % weight bandwidth on the
// Llama-2-70B decode shapes with cold caches).
__device__ __forceinline__ v8i ld_frag_stream(const uint8_t* p) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 p0 = __builtin_nontemporal_load((const u32x4*)p);
    const u32x4 p1 = __builtin_nontemporal_load((const u32x4*)(p + 16));
    return v8i{(int)p0.x, (int)p0.y, (int)p0.z, (int)p0.w, (int)p1.x, (int)p1.y, (int)p1.z, (int)p1.w};
}

// NB: 16-column blocks per workgroup; kDecWaves: waves splitting the K range.
template <int FA, int FB, int OUT_DT, bool AMAX, int MB, int NB, int kDecWaves>
__global__ __launch_bounds__(kDecWaves * 64) void gemm_nt_decode(
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ B, const int32_t* __restrict__ ba_p,
    const int32_t* __restrict__ bb_p, void* __restrict__ C, int M, int N, int K, int vec_out,
    uint32_t* __restrict__ amax_out, int ba_rows) {
    __shared__ __attribute__((aligned(16))) float red[kDecWaves][MB][NB][64][4];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int n0 = blockIdx.x * NB * 16;
    const int frow = lane & 15, fg = lane >> 4;
    // fragment sources: row (lane % 16) of each 16-row block, 32 bytes at
    // k-offset 32 (lane / 16) of every 128-byte step
    const uint8_t* pa[MB];
    const uint8_t* pb[NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) pa[mb] = A + (int64_t)min(mb * 16 + frow, M - 1) * K + fg * 32;
#pragma unroll
    for (int j = 0; j < NB; ++j) pb[j] = B + (int64_t)min(n0 + j * 16 + frow, N - 1) * K + fg * 32;
    const int nkc = K / kBK;
    const int c0 = (int)((int64_t)nkc * w / kDecWaves), c1 = (int)((int64_t)nkc * (w + 1) / kDecWaves);

    v4f acc[MB][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[mb][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // three k-steps in flight
    v8i xa[3][MB], wb[3][NB];
    auto load = [&](int slot, int c) {
        const int64_t k0 = (int64_t)c * kBK;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) xa[slot][mb] = ld_frag_g(pa[mb] + k0);
#pragma unroll
        for (int j = 0; j < NB; ++j) wb[slot][j] = ld_frag_stream(pb[j] + k0);
    };
    auto step = [&](int slot) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < NB; ++j) acc[mb][j] = mfma16<FB, FA>(wb[slot][j], xa[slot][mb], acc[mb][j]);
    };
    if (c0 < c1) load(0, c0);
    if (c0 + 1 < c1) load(1, c0 + 1);
    for (int c = c0; c < c1; c += 3) {
        if (c + 2 < c1) load(2, c + 2);
        step(0);
        if (c + 1 < c1) {
            if (c + 3 < c1) load(0, c + 3);
            step(1);
        }
        if (c + 2 < c1) {
            if (c + 4 < c1) load(1, c + 4);
            step(2);
        }
    }

#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < NB; ++j) *(v4f*)red[w][mb][j][lane] = acc[mb][j];
    __syncthreads();
    uint32_t mx = 0;
    for (int slot = threadIdx.x; slot < MB * NB * 64; slot += kDecWaves * 64) {
        const int mb = slot / (NB * 64), j = (slot / 64) % NB, l = slot & 63;
        v4f sum = *(const v4f*)red[0][mb][j][l];
#pragma unroll
        for (int ww = 1; ww < kDecWaves; ++ww) sum += *(const v4f*)red[ww][mb][j][l];
        const int64_t m = mb * 16 + (l & 15);
        const int64_t n = n0 + j * 16 + (l >> 4) * 4;
        if (n < N) mx = max(mx, store4<OUT_DT>(C, N, m, n, M, N, sum, row_shift(ba_p, ba_rows, *bb_p, m, M), vec_out != 0));
    }
    if (AMAX) {
        mx = wave_max_u32(mx);
        if (lane == 0) atomicMax(amax_out, canon_amax(mx));
    }
}

// Staged decode kernel (M <= 16, K a multiple of 512): the same product with
// the weight rows streamed through LDS.  A load instruction that feeds an MFMA
// fragment straight from memory touches 16 weight rows K bytes apart, 64 bytes
// each; here a workgroup copies its BR weight rows (one contiguous block of
// memory) and the 16 activation rows 512 bytes of k at a time with
// global_load_lds_dwordx4, each instruction reading 512-byte runs of two
// rows, three stages in flight, and the waves read the fragments from LDS.
// Chunk c of LDS row r (16 bytes) is stored at chunk c ^ (r % 16): the 16
// lanes of every ds_read_b128 phase (lane bit 5 and the parity of lane bits
// 2..4 fixed; see the main kernel) then hit 16 distinct bank groups.
// BR = 64: each wave one 16-row block, all k-steps.  BR = 32: waves w and w + 2
// share block w % 2, each half of every stage's k-steps, added in a fixed order.
constexpr int kDlKC = 512, kDlBuf = 3;

template <int FA, int FB, int OUT_DT, bool AMAX, int BR>
__global__ __launch_bounds__(256) void gemm_nt_decode_lds(
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ B, const int32_t* __restrict__ ba_p,
    const int32_t* __restrict__ bb_p, void* __restrict__ C, int M, int N, int K, int vec_out,
    uint32_t* __restrict__ amax_out, int ba_rows) {
    constexpr int kRows = BR + 16, kStage = kRows * kDlKC, kCpr = kDlKC / 16;
    constexpr int kNi = kRows / 2;  // copies per stage, two rows each
    static_assert(kNi % 4 == 0, "copies split over four waves");
    constexpr int kNiw = kNi / 4;
    constexpr int kNbb = BR / 16, kWpb = 4 / kNbb, kKs = kDlKC / 128 / kWpb;
    __shared__ __attribute__((aligned(1024))) uint8_t sm[kDlBuf * kStage];
    __shared__ __attribute__((aligned(16))) float red[4][64][4];
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n0 = blockIdx.x * BR;
    // copy t of this wave: LDS rows 2d, 2d + 1 (d = kNiw w + t); rows < BR are
    // weight rows n0 + r (clamped to N - 1), the rest activation rows (clamped
    // to M - 1); lane -> row 2d + lane / 32, physical chunk lane % 32
    uint32_t voff[kNiw];
#pragma unroll
    for (int t = 0; t < kNiw; ++t) {
        const int d = w * kNiw + t, r = 2 * d + (lane >> 5), c = (lane & 31) ^ (r & 15);
        voff[t] = r < BR ? (uint32_t)((min(n0 + r, N - 1) - n0) * K + c * 16)
                         : (uint32_t)(min(r - BR, M - 1) * K + c * 16);
    }
    const uint8_t* bbase = B + (int64_t)n0 * K;
    const uint32_t lds0 = lds_addr(sm);
    auto issue = [&](int st) {
        const int buf = st % kDlBuf;
#pragma unroll
        for (int t = 0; t < kNiw; ++t) {
            const int d = w * kNiw + t;
            const uint32_t dst = __builtin_amdgcn_readfirstlane(lds0 + buf * kStage + d * 2 * kDlKC);
            if (2 * d < BR) lds_dma16_nt(bbase + (int64_t)st * kDlKC, voff[t], dst);
            else lds_dma16_s(A + (int64_t)st * kDlKC, voff[t], dst);
        }
    };
    const int frow = lane & 15, fg = lane >> 4;
    const int j = w % kNbb, h = w / kNbb;
    const int rb = 16 * j + frow, ra = BR + frow;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    const int nst = K / kDlKC;
#pragma unroll
    for (int st = 0; st < kDlBuf - 1; ++st)
        if (st < nst) issue(st);
    for (int st = 0; st < nst; ++st) {
        // stage st has landed once only the next stage's copies may be pending
        if (st + 1 < nst) wait_vmcnt<kNiw>();
        else wait_vmcnt<0>();
        ws_barrier();
        // the buffer of stage st - 1, which every wave has finished reading
        if (st + kDlBuf - 1 < nst) issue(st + kDlBuf - 1);
        const uint8_t* sb = sm + (st % kDlBuf) * kStage;
#pragma unroll
        for (int q = 0; q < kKs; ++q) {
            const int c0 = (h * kKs + q) * 8 + 2 * fg;
            const v8i bf = ld_frag(sb + rb * kDlKC, 16 * (c0 ^ (rb & 15)), 16 * ((c0 + 1) ^ (rb & 15)));
            const v8i af = ld_frag(sb + ra * kDlKC, 16 * (c0 ^ (ra & 15)), 16 * ((c0 + 1) ^ (ra & 15)));
            acc = mfma16<FB, FA>(bf, af, acc);
        }
    }
    *(v4f*)red[w][lane] = acc;
    __syncthreads();
    uint32_t mx = 0;
    if (w < kNbb) {
        v4f sum = *(const v4f*)red[w][lane];
#pragma unroll
        for (int hh = 1; hh < kWpb; ++hh) sum += *(const v4f*)red[w + hh * kNbb][lane];
        const int64_t m = lane & 15, n = n0 + w * 16 + (lane >> 4) * 4;
        if (n < N) mx = store4<OUT_DT>(C, N, m, n, M, N, sum, row_shift(ba_p, ba_rows, *bb_p, m, M), vec_out != 0);
    }
    if (AMAX) {
        mx = wave_max_u32(mx);
        if (lane == 0) atomicMax(amax_out, canon_amax(mx));
    }
}

template <int FA, int FB, int OUT_DT, bool AMAX, int MB>
void launch_decode(const uint8_t* A, const int32_t* ba, const uint8_t* B, const int32_t* bb, void* C,
                   int M, int N, int K, int vec_out, uint32_t* amax, int ba_rows, hipStream_t s) {
    // 32 output columns per workgroup of 4 waves, each wave a quarter of the
    // K range (the best of 1-8 column blocks x 4-16 waves on the Llama-2-70B
    // decode shapes)
    const int nblk = (N + 31) / 32;
    hipLaunchKernelGGL((gemm_nt_decode<FA, FB, OUT_DT, AMAX, MB, 2, 4>), dim3(nblk), dim3(4 * 64), 0, s, A, B, ba,
                       bb, C, M, N, K, vec_out, amax, ba_rows);
}

__global__ void fill_u32_kernel(uint32_t* p, uint32_t v) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *p = v;
}

// The LDS-staged kernels need K a multiple of 128, 16-byte aligned operands
// and 32-bit offsets within a tile.
bool fast_path(const uint8_t* A, const uint8_t* B, int64_t M, int64_t N, int64_t K) {
    return (K % kBK == 0) && ((uintptr_t)A % 16 == 0) && ((uintptr_t)B % 16 == 0) && M <= INT32_MAX &&
           N <= INT32_MAX && K < (1 << 22);
}

// Workgroups of the 256-row kernel that run at once (one per CU of gfx950).
constexpr int kRound = 256;

// Columns of 256-wide tiles taken in whole rounds of kRound workgroups, and
// the rest in one round of narrower tiles: with all 256-wide, a last partial
// round costs as much as a full one.  E.g. 4096 x 11008 (16 x 43 tiles):
// two rounds over the first 8192 columns, then 240 tiles 192 wide (0.75 of
// the work each) over the last 2816.  Every output is still computed by one
// workgroup over the whole K in the same order, so the bits do not change.
// ndp: 256-wide tile columns; tw, tn2: width and count of the narrow ones
// (tw = 0: no narrow launch).
void narrow_split(int tiles_m, int tiles_n, int64_t N, int& ndp, int& tw, int& tn2) {
    ndp = tiles_n;
    tw = 0;
    tn2 = 0;
    const int64_t T = (int64_t)tiles_m * tiles_n;
    if (T % kRound == 0 || tiles_m > kRound) return;
    int gcd = kRound, b = tiles_m;
    while (b) {
        const int t = gcd % b;
        gcd = b;
        b = t;
    }
    const int step = kRound / gcd;  // tile columns per whole number of rounds
    const int c = tiles_n / step * step;
    const int64_t nrem = N - (int64_t)c * kBN;
    for (int w : {64, 128, 192}) {
        const int64_t strips = (nrem + w - 1) / w;
        if (tiles_m * strips <= kRound) {
            ndp = c;
            tw = w;
            tn2 = (int)strips;
            return;
        }
    }
}

// bo.ws != nullptr only where the 256-row kernel runs (fast_path, M > 32).
template <int FA, int FB, int OUT_DT, bool AMAX>
void launch_t(const uint8_t* A, const int32_t* ba, const uint8_t* B, const int32_t* bb, void* C,
              int64_t M, int64_t N, int64_t K, uint32_t* amax, const BiasOut& bo, int ba_rows, hipStream_t s) {
    const int esz = OUT_DT == FP8_DT_BF16 ? 2 : 4;
    const int vec_out = ((uintptr_t)C % (4 * esz) == 0) && (N % 4 == 0);
    const bool fast = fast_path(A, B, M, N, K);
    if (fast && M <= 16 && K % kDlKC == 0) {
        // 64 weight rows per workgroup unless that leaves fewer than 256
        // workgroups streaming long rows (measured on the Llama-2-70B shapes)
        if (N >= 64 * 256 || K <= 8192)
            hipLaunchKernelGGL((gemm_nt_decode_lds<FA, FB, OUT_DT, AMAX, 64>), dim3((unsigned)((N + 63) / 64)), dim3(256),
                               0, s, A, B, ba, bb, C, (int)M, (int)N, (int)K, vec_out, amax, ba_rows);
        else
            hipLaunchKernelGGL((gemm_nt_decode_lds<FA, FB, OUT_DT, AMAX, 32>), dim3((unsigned)((N + 31) / 32)), dim3(256),
                               0, s, A, B, ba, bb, C, (int)M, (int)N, (int)K, vec_out, amax, ba_rows);
    } else if (fast && M <= 32) {
        if (M <= 16) launch_decode<FA, FB, OUT_DT, AMAX, 1>(A, ba, B, bb, C, (int)M, (int)N, (int)K, vec_out, amax, ba_rows, s);
        else launch_decode<FA, FB, OUT_DT, AMAX, 2>(A, ba, B, bb, C, (int)M, (int)N, (int)K, vec_out, amax, ba_rows, s);
    } else if (fast) {
        const int tiles_m = (int)((M + kBM - 1) / kBM), tiles_n = (int)((N + kBN - 1) / kBN);
        const int vec16 = ((uintptr_t)C % 16 == 0) && ((N * esz) % 16 == 0);
        int ndp, tw, tn2;
        narrow_split(tiles_m, tiles_n, N, ndp, tw, tn2);
        const int g1 = tiles_m * ndp, grid = g1 + tiles_m * tn2;
#define FP8LIN_GEMM256(TW)                                                                                         \
    hipLaunchKernelGGL((gemm_nt_256<FA, FB, OUT_DT, AMAX, -1, TW>), dim3(grid), dim3(kMainThreads), 0, s, A, B, ba, \
                       bb, C, (int)M, (int)N, (int)K, tiles_m, ndp, vec16, amax, QuantOut{}, bo, ba_rows, g1, tn2)
        if (tw == 64) FP8LIN_GEMM256(64);
        else if (tw == 128) FP8LIN_GEMM256(128);
        else if (tw == 192) FP8LIN_GEMM256(192);
        else FP8LIN_GEMM256(0);
#undef FP8LIN_GEMM256
    } else {
        const int64_t tiles_m = (M + kSBM - 1) / kSBM, tiles_n = (N + kSBN - 1) / kSBN;
        hipLaunchKernelGGL((gemm_nt_small<FA, FB, OUT_DT, AMAX>), dim3((unsigned)(tiles_m * tiles_n)),
                           dim3(kThreads), 0, s, A, B, ba, bb, C, M, N, K, tiles_n, vec_out, amax, ba_rows);
    }
}

// with_amax: epilogue amax (into *amax, or folded into bo.ws).
template <int FA, int FB>
void dispatch_out(const uint8_t* A, const int32_t* ba, const uint8_t* B, const int32_t* bb, void* C,
                  int out_dt, int64_t M, int64_t N, int64_t K, bool with_amax, uint32_t* amax,
                  const BiasOut& bo, int ba_rows, hipStream_t s) {
    if (out_dt == FP8_DT_BF16) {
        if (with_amax) launch_t<FA, FB, FP8_DT_BF16, true>(A, ba, B, bb, C, M, N, K, amax, bo, ba_rows, s);
        else launch_t<FA, FB, FP8_DT_BF16, false>(A, ba, B, bb, C, M, N, K, amax, bo, ba_rows, s);
    } else {
        if (with_amax) launch_t<FA, FB, FP8_DT_F32, true>(A, ba, B, bb, C, M, N, K, amax, bo, ba_rows, s);
        else launch_t<FA, FB, FP8_DT_F32, false>(A, ba, B, bb, C, M, N, K, amax, bo, ba_rows, s);
    }
}

void dispatch_fmts(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb, const int32_t* bb,
                   void* C, int out_dt, int64_t M, int64_t N, int64_t K, bool with_amax, uint32_t* amax,
                   const BiasOut& bo, int ba_rows, hipStream_t s) {
    if (fa == FP8_E4M3 && fb == FP8_E4M3)
        dispatch_out<FP8_E4M3, FP8_E4M3>(A, ba, B, bb, C, out_dt, M, N, K, with_amax, amax, bo, ba_rows, s);
    else if (fa == FP8_E5M2 && fb == FP8_E4M3)
        dispatch_out<FP8_E5M2, FP8_E4M3>(A, ba, B, bb, C, out_dt, M, N, K, with_amax, amax, bo, ba_rows, s);
    else if (fa == FP8_E4M3 && fb == FP8_E5M2)
        dispatch_out<FP8_E4M3, FP8_E5M2>(A, ba, B, bb, C, out_dt, M, N, K, with_amax, amax, bo, ba_rows, s);
    else
        dispatch_out<FP8_E5M2, FP8_E5M2>(A, ba, B, bb, C, out_dt, M, N, K, with_amax, amax, bo, ba_rows, s);
}

template <int FA, int FB, int QF>
void launch_fused_t(const uint8_t* A, const int32_t* ba, const uint8_t* B, const int32_t* bb, void* C,
                    int64_t M, int64_t N, int64_t K, const QuantOut& qo, hipStream_t s) {
    const int tiles_m = (int)((M + kBM - 1) / kBM), tiles_n = (int)((N + kBN - 1) / kBN);
    const int vec16 = ((uintptr_t)C % 16 == 0) && ((N * 2) % 16 == 0);
    hipLaunchKernelGGL((gemm_nt_256<FA, FB, FP8_DT_BF16, false, QF>), dim3(tiles_m * tiles_n), dim3(kMainThreads), 0,
                       s, A, B, ba, bb, C, (int)M, (int)N, (int)K, tiles_m, tiles_n, vec16, nullptr, qo, BiasOut{}, 0,
                       tiles_m * tiles_n, 0);
}

template <int FA, int FB>
void fused_fmt(int qfmt, const uint8_t* A, const int32_t* ba, const uint8_t* B, const int32_t* bb, void* C,
               int64_t M, int64_t N, int64_t K, const QuantOut& qo, hipStream_t s) {
    switch (qfmt) {
        case FP8_E4M3: launch_fused_t<FA, FB, FP8_E4M3>(A, ba, B, bb, C, M, N, K, qo, s); break;
        case FP8_E5M2: launch_fused_t<FA, FB, FP8_E5M2>(A, ba, B, bb, C, M, N, K, qo, s); break;
        case FP8_E4_A: launch_fused_t<FA, FB, FP8_E4_A>(A, ba, B, bb, C, M, N, K, qo, s); break;
        default: launch_fused_t<FA, FB, FP8_E5_A>(A, ba, B, bb, C, M, N, K, qo, s); break;
    }
}

}  // namespace

int64_t gemm_quantise_ws_words(int64_t M, int64_t N) {
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
    const int64_t q = quantise_ws_words(M, N);
    return 1 + tiles > q ? 1 + tiles : q;
}

int32_t launch_gemm_nt_quantise(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb,
                                const int32_t* bb, void* C, int64_t M, int64_t N, int64_t K, int qfmt,
                                int32_t margin, const int32_t* pred, int32_t* bias, uint32_t* amax_bits,
                                uint32_t* flags, uint8_t* y8, int64_t ldy8, uint8_t* y8t, int64_t ldy8t,
                                uint32_t* ws, hipStream_t s) {
    const bool fused = pred && fast_path(A, B, M, N, K) && M > 32 && (fa == FP8_E4M3 || fa == FP8_E5M2) &&
                       fb == FP8_E4M3;
    if (!fused) {  // matmul, then the quantise of its output (same bits, more passes)
        const int32_t st = launch_gemm_nt(A, fa, ba, B, fb, bb, C, FP8_DT_BF16, M, N, K, nullptr, s);
        if (st != FP8_OK) return st;
        return launch_quantise(C, FP8_DT_BF16, M, N, N, qfmt, margin, pred, bias, amax_bits, flags, y8, ldy8, y8t,
                               ldy8t, ws, s);
    }
    QuantOut qo;
    qo.pred = pred;
    qo.used = (int32_t*)ws;
    qo.parts = ws + 1;
    qo.y8 = y8;
    qo.ldy8 = ldy8;
    qo.y8t = y8t;
    qo.ldy8t = ldy8t;
    qo.vec8 = ((uintptr_t)y8 % 16 == 0) && (ldy8 % 16 == 0);
    qo.vec8t = y8t && ((uintptr_t)y8t % 16 == 0) && (ldy8t % 16 == 0);
    if (fa == FP8_E4M3)
        fused_fmt<FP8_E4M3, FP8_E4M3>(qfmt, A, ba, B, bb, C, M, N, K, qo, s);
    else
        fused_fmt<FP8_E5M2, FP8_E4M3>(qfmt, A, ba, B, bb, C, M, N, K, qo, s);
    const int tiles = (int)(((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN));
    const int32_t st = hip_status();
    if (st != FP8_OK) return st;
    return launch_quant_check(C, FP8_DT_BF16, M, N, N, qfmt, margin, ws + 1, tiles, (int32_t*)ws, bias, amax_bits,
                              flags, y8, ldy8, y8t, ldy8t, s);
}

int32_t launch_fill_u32(uint32_t* p, uint32_t v, hipStream_t s) {
    hipLaunchKernelGGL(fill_u32_kernel, dim3(1), dim3(64), 0, s, p, v);
    return hip_status();
}

int32_t launch_gemm_nt(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb,
                       const int32_t* bb, void* C, int out_dt, int64_t M, int64_t N, int64_t K,
                       uint32_t* amax_bits, hipStream_t s, int ba_rows) {
    if (amax_bits) hipLaunchKernelGGL(fill_u32_kernel, dim3(1), dim3(64), 0, s, amax_bits, 0u);
    dispatch_fmts(A, fa, ba, B, fb, bb, C, out_dt, M, N, K, amax_bits != nullptr, amax_bits, BiasOut{}, ba_rows, s);
    return hip_status();
}

int32_t launch_gemm_nt_bias(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb,
                            const int32_t* bb, void* C, int out_dt, int64_t M, int64_t N, int64_t K, int bfmt,
                            int32_t margin, int32_t* bias, uint32_t* amax_bits, uint32_t* flags, uint32_t* ws,
                            hipStream_t s, int ba_rows) {
    if (fast_path(A, B, M, N, K) && M > 32) {
        dispatch_fmts(A, fa, ba, B, fb, bb, C, out_dt, M, N, K, true, amax_bits, BiasOut{bias, flags, ws, bfmt, margin},
                      ba_rows, s);
        return hip_status();
    }
    // decode and fallback kernels: amax with atomics into a zeroed word (ws[0]
    // if no amax output is wanted, zeroed again afterwards), then the bias
    uint32_t* acc = amax_bits ? amax_bits : ws;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(1), dim3(64), 0, s, acc, 0u);
    dispatch_fmts(A, fa, ba, B, fb, bb, C, out_dt, M, N, K, true, acc, BiasOut{}, ba_rows, s);
    int32_t st = hip_status();
    if (st != FP8_OK) return st;
    st = launch_bias_from_amax(acc, bfmt, margin, bias, flags, s);
    if (st != FP8_OK || acc != ws) return st;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(1), dim3(64), 0, s, ws, 0u);
    return hip_status();
}

}  // namespace fp8lin
