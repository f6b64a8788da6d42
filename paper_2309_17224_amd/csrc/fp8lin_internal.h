// Internal declarations shared by the translation units of libfp8lin.so.
// Not part of the ABI: the public interface is include/fp8lin.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fp8lin.h"

namespace fp8lin {

// Threads and block cap of the amax reduction: one fp32 partial per block.
constexpr int kAmaxThreads = 256;
constexpr int kAmaxMaxBlocks = 2048;

int amax_blocks(int64_t n);

int32_t launch_scale_bias(const void* x, int dt, int64_t n, int fmt, int32_t margin, int32_t* bias,
                          uint32_t* amax_bits, uint32_t* flags, uint32_t* partials,
                          hipStream_t s);
int32_t launch_bias_from_amax(const uint32_t* amax_bits, int fmt, int32_t margin, int32_t* bias,
                              uint32_t* flags, hipStream_t s);
int32_t launch_cast(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                    const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                    hipStream_t s);

// amax + bias + cast of a rows x cols tensor (two kernels); ws holds
// quantise_ws_words(rows, cols) uint32 words.
int64_t quantise_ws_words(int64_t rows, int64_t cols);
// Number of quantise tiles of a rows x cols tensor, or -1 when it exceeds
// limit (computed without overflow for any sizes below 2^62).
int64_t quantise_tiles_upto(int64_t rows, int64_t cols, int64_t limit);

// fp8_quantise of several tensors of one type and format (checked arguments).
constexpr int kQBatch = FP8_QUANTISE_BATCH_MAX;
struct QuantDesc {
    const void* x;
    int64_t rows, cols, ldx;
    const int32_t* pred;
    int32_t* bias;
    uint32_t* amax;
    uint32_t* flags;
    uint8_t* q;
    int64_t ldq;
    uint8_t* qT;
    int64_t ldqT;
    uint32_t* ws;
};
int32_t launch_quantise_batch(int n, const QuantDesc* d, int dt, int fmt, int32_t margin, hipStream_t s);
int32_t launch_quantise(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                        int32_t margin, const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits,
                        uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                        uint32_t* ws, hipStream_t s);

// Delayed scaling: cast with *bias (one pass over x), then a one-workgroup
// kernel appends the tensor's amax to history[*count % hlen], increments
// *count and writes the next call's bias into *bias.  ws as launch_quantise.
int32_t launch_quantise_delayed(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                                int32_t margin, int32_t* bias, uint32_t* history, int hlen, uint32_t* count,
                                uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT,
                                int64_t ldqT, uint32_t* ws, hipStream_t s);

// The exact-bias check and recast of fp8_quantise's second pass for a tensor
// x whose per-tile maxima (nparts of them, any tiling) and the prediction its
// codes were cast with (*used) were written by another kernel.
int32_t launch_quant_check(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                           int32_t margin, const uint32_t* parts, int nparts, const int32_t* used,
                           int32_t* bias, uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq,
                           uint8_t* qT, int64_t ldqT, hipStream_t s);

// Matmul with bf16 output C whose epilogue also casts C to format qfmt with
// the predicted bias *pred and writes y8 (and y8t if non-null), followed by
// the exact-bias check: the same bits as launch_gemm_nt followed by
// launch_quantise.  ws holds gemm_quantise_ws_words(M, N) uint32 words.
int64_t gemm_quantise_ws_words(int64_t M, int64_t N);
int32_t launch_gemm_nt_quantise(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb,
                                const int32_t* bb, void* C, int64_t M, int64_t N, int64_t K, int qfmt,
                                int32_t margin, const int32_t* pred, int32_t* bias, uint32_t* amax_bits,
                                uint32_t* flags, uint8_t* y8, int64_t ldy8, uint8_t* y8t, int64_t ldy8t,
                                uint32_t* ws, hipStream_t s);

// C[m, n] = 2^-(*ba + *bb) * sum_k A[m, k] * B[n, k]; A [M, K] (format fa),
// B [N, K] (format fb), both dense; C [M, N] dense of type out_dt.  With
// ba_rows, ba holds one bias per row of A: 2^-(ba[m] + *bb).
int32_t launch_gemm_nt(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb,
                       const int32_t* bb, void* C, int out_dt, int64_t M, int64_t N, int64_t K,
                       uint32_t* amax_bits, hipStream_t s, int ba_rows = 0);

// Per row segment of x (rows offsets[s] .. offsets[s+1]-1): amax, Eq. 3 bias
// and flags into [nseg] arrays, the bias of every row into row_bias [rows],
// and the cast of each row with its segment's bias.
int32_t launch_quantise_segments(const void* x, int dt, int64_t rows, int64_t cols, int64_t ldx, int fmt,
                                 int32_t margin, const int32_t* offsets, int nseg, int32_t* bias, uint32_t* amax_bits,
                                 uint32_t* flags, int32_t* row_bias, uint8_t* q, int64_t ldq, uint8_t* qT,
                                 int64_t ldqT, hipStream_t s);

// Mode of n biases appended to ring[*count % capacity]; *count += 1.
int32_t launch_bias_mode(const int32_t* bias, int64_t n, int32_t* ring, int64_t capacity, uint32_t* count,
                         hipStream_t s);

// launch_gemm_nt with the epilogue amax of C turned into the Eq. 3 bias for
// format bfmt in the same launch (256 x 256 kernel: the last workgroup to
// finish computes it from a running maximum in ws[0..1], which must be zero
// and is left zero); other kernels: amax with atomics, then the bias kernel.
// amax_bits and flags may be null.
int32_t launch_gemm_nt_bias(const uint8_t* A, int fa, const int32_t* ba, const uint8_t* B, int fb,
                            const int32_t* bb, void* C, int out_dt, int64_t M, int64_t N, int64_t K, int bfmt,
                            int32_t margin, int32_t* bias, uint32_t* amax_bits, uint32_t* flags, uint32_t* ws,
                            hipStream_t s, int ba_rows = 0);

// ---- decoder-layer glue (fp8lin_decoder.hip)
// The FP8-AMAX quantise fused into a glue kernel's bf16 output: codes cast
// with the prediction (if any), then the exact-bias check and recast.
struct FusedQuant {
    int fmt;
    int32_t margin;
    const int32_t* pred;  // predicted bias (device) or null
    int32_t* bias;
    uint32_t* amax_bits;  // may be null
    uint32_t* flags;      // may be null
    uint8_t* q;           // codes [rows, cols], row stride ldq; null: no quantise
    int64_t ldq;
    uint32_t* ws;         // word 0: the bias the codes were cast with; then one maximum per workgroup
};

// Workgroup maxima each glue kernel writes (workspace words beyond the first).
int64_t glue_parts_rmsnorm(int64_t rows);
int64_t glue_parts_swiglu();
int64_t glue_parts_attention(int64_t rows, int64_t seq_len, int nh);

int32_t launch_residual_add(const uint16_t* a, const uint16_t* b, uint16_t* out, int64_t n, hipStream_t s);
int32_t launch_rmsnorm(const uint16_t* x, int64_t ldx, const uint16_t* res, int64_t ldr, const uint16_t* g,
                       int64_t rows, int64_t cols, float eps, uint16_t* h, int64_t ldh, uint16_t* y, int64_t ldy,
                       const FusedQuant* fq, hipStream_t s);
int32_t launch_rope_table(int64_t seq_len, int d_head, double theta, float* table, hipStream_t s);
int32_t launch_rope(uint16_t* x, int64_t rows, int64_t ld, int nheads, int d_head, int64_t seq_len,
                    const float* table, hipStream_t s);
int32_t launch_swiglu(const uint16_t* gu, int64_t ldgu, int64_t rows, int64_t ffn, uint16_t* a, int64_t lda,
                      const FusedQuant* fq, hipStream_t s);
int32_t launch_attention(const uint16_t* qkv, int64_t rows, int64_t ld, int64_t seq_len, int nh, int nkv,
                         uint16_t* o, int64_t ldo, const FusedQuant* fq, hipStream_t s);

// *p = v on the stream (one word).
int32_t launch_fill_u32(uint32_t* p, uint32_t v, hipStream_t s);

inline int32_t hip_status() { return hipGetLastError() == hipSuccess ? FP8_OK : FP8_EHIP; }

}  // namespace fp8lin
