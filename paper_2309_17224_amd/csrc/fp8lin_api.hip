// C entry points of libfp8lin.so (declared and documented in fp8lin.h).
// Each call checks its arguments on the host, then enqueues kernels on the
// caller's stream; nothing is allocated, kept or synchronised.
#include <mutex>

#include "fp8lin_internal.h"

using namespace fp8lin;

namespace {

constexpr int64_t kMaxDim = (int64_t)1 << 40;

bool fmt_ok(int32_t f) { return f == FP8_E4M3 || f == FP8_E5M2 || f == FP8_E4_A || f == FP8_E5_A; }
bool dt_ok(int32_t d) { return d == FP8_DT_BF16 || d == FP8_DT_F32; }
int esize(int32_t d) { return d == FP8_DT_BF16 ? 2 : 4; }
bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }
hipStream_t as_stream(void* s) { return (hipStream_t)s; }
bool a16(const void* p) { return aligned(p, 16); }

int32_t cast_common(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                    const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                    int fmt, void* stream) {
    if (!dt_ok(dt) || !fmt_ok(fmt) || rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return FP8_EINVAL;
    if (rows == 0 || cols == 0) return FP8_OK;
    if (!x || !bias || (!q && !qT)) return FP8_EINVAL;
    if (!aligned(x, esize(dt)) || !aligned(bias, 4)) return FP8_EINVAL;
    if (ldx < cols || (q && ldq < cols) || (qT && ldqT < rows)) return FP8_EINVAL;
    if (quantise_tiles_upto(rows, cols, INT32_MAX) < 0) return FP8_ENOTSUP;  // one workgroup per 128 x 128 tile
    return launch_cast(x, dt, rows, cols, ldx, fmt, bias, q, ldq, qT, ldqT, as_stream(stream));
}

// Matmul operands (FP8 codes) start on 16-byte boundaries when K > 0.
bool operands_ok(const uint8_t* a, const uint8_t* b, int64_t K) { return K == 0 || (a16(a) && a16(b)); }

int32_t gemm_common(const uint8_t* a, int fa, const int32_t* ba, const uint8_t* b, int fb,
                    const int32_t* bb, void* c, int32_t c_dt, int64_t M, int64_t N, int64_t K,
                    uint32_t* amax, void* stream) {
    if (!dt_ok(c_dt) || M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim)
        return FP8_EINVAL;
    if (amax && !aligned(amax, 4)) return FP8_EINVAL;
    if (M == 0 || N == 0)  // no output: its amax is 0
        return amax ? launch_fill_u32(amax, 0u, as_stream(stream)) : FP8_OK;
    if (!c || !ba || !bb || (K > 0 && (!a || !b))) return FP8_EINVAL;
    if (!aligned(c, esize(c_dt)) || !aligned(ba, 4) || !aligned(bb, 4)) return FP8_EINVAL;
    if (!operands_ok(a, b, K)) return FP8_EINVAL;
    if (M > INT32_MAX || N > INT32_MAX) return FP8_ENOTSUP;
    return launch_gemm_nt(a, fa, ba, b, fb, bb, c, c_dt, M, N, K, amax, as_stream(stream));
}


// ---- decoder-layer glue: shared checks
bool rows_ok(int64_t ld, int64_t cols) { return ld >= cols && ld % 8 == 0; }

// Checks the arguments of a fused quantise and fills *fq; q == NULL means no
// quantise (the other arguments are then ignored).  need_words: workspace
// words the op needs.
int32_t glue_quant(int32_t fmt, int32_t margin, const int32_t* pred, int32_t* bias, uint32_t* amax_bits,
                   uint32_t* flags, uint8_t* q, int64_t ldq, int64_t cols, void* ws, size_t ws_bytes,
                   int64_t need_words, FusedQuant* fq) {
    fq->q = nullptr;
    if (!q) return FP8_OK;
    if (!fmt_ok(fmt) || margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN) return FP8_EINVAL;
    if (!bias || !aligned(bias, 4) || (pred && !aligned(pred, 4))) return FP8_EINVAL;
    if ((amax_bits && !aligned(amax_bits, 4)) || (flags && !aligned(flags, 4))) return FP8_EINVAL;
    if (!aligned(q, 8) || !rows_ok(ldq, cols)) return FP8_EINVAL;
    if (!ws || !aligned(ws, 4) || ws_bytes < (size_t)need_words * sizeof(uint32_t)) return FP8_EINVAL;
    if (need_words - 1 > INT32_MAX) return FP8_ENOTSUP;
    fq->fmt = fmt;
    fq->margin = margin;
    fq->pred = pred;
    fq->bias = bias;
    fq->amax_bits = amax_bits;
    fq->flags = flags;
    fq->q = q;
    fq->ldq = ldq;
    fq->ws = (uint32_t*)ws;
    return FP8_OK;
}

// An empty output with a quantise: amax 0, bias 0 and the zero flag.
int32_t glue_empty(int32_t fmt, int32_t margin, int32_t* bias, uint32_t* amax_bits, uint32_t* flags, uint8_t* q,
                   void* stream) {
    if (!q) return FP8_OK;
    if (!fmt_ok(fmt) || margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN || !bias || !aligned(bias, 4))
        return FP8_EINVAL;
    if ((amax_bits && !aligned(amax_bits, 4)) || (flags && !aligned(flags, 4))) return FP8_EINVAL;
    return launch_scale_bias(nullptr, FP8_DT_BF16, 0, fmt, margin, bias, amax_bits, flags, nullptr, as_stream(stream));
}

}  // namespace

extern "C" {

const char* fp8_status_string(int32_t status) {
    switch (status) {
        case FP8_OK: return "ok";
        case FP8_EINVAL: return "invalid argument";
        case FP8_ENOTSUP: return "unsupported argument combination";
        case FP8_EHIP: return "HIP launch error";
        default: return "unknown status";
    }
}

int32_t fp8_abi_version(void) { return 1; }

size_t fp8_scale_bias_ws_bytes(int64_t n) {
    if (n <= 0) return 0;
    return (size_t)amax_blocks(n) * sizeof(uint32_t);
}

int32_t fp8_scale_bias(const void* x, int32_t dt, int64_t n, int32_t fmt, int32_t margin,
                       int32_t* bias, uint32_t* amax_bits, uint32_t* flags, void* ws,
                       size_t ws_bytes, void* stream) {
    if (!dt_ok(dt) || !fmt_ok(fmt) || n < 0 || n > kMaxDim * 64) return FP8_EINVAL;
    if (margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN) return FP8_EINVAL;
    if (!bias || !aligned(bias, 4)) return FP8_EINVAL;
    if ((amax_bits && !aligned(amax_bits, 4)) || (flags && !aligned(flags, 4))) return FP8_EINVAL;
    if (n > 0) {  // an empty tensor has amax 0: no input or workspace is read
        if (!x || !aligned(x, esize(dt))) return FP8_EINVAL;
        if (!ws || !aligned(ws, 4) || ws_bytes < fp8_scale_bias_ws_bytes(n)) return FP8_EINVAL;
    }
    return launch_scale_bias(x, dt, n, fmt, margin, bias, amax_bits, flags, (uint32_t*)ws,
                             as_stream(stream));
}

int32_t fp8_cast(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx, int32_t fmt,
                 const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                 void* stream) {
    return cast_common(x, dt, rows, cols, ldx, bias, q, ldq, qT, ldqT, fmt, stream);
}

size_t fp8_quantise_ws_bytes(int64_t rows, int64_t cols) {
    if (rows <= 0 || cols <= 0 || rows > kMaxDim || cols > kMaxDim) return 0;
    if (quantise_tiles_upto(rows, cols, INT32_MAX) < 0) return SIZE_MAX;  // beyond what a call accepts
    return (size_t)quantise_ws_words(rows, cols) * sizeof(uint32_t);
}

}  // extern "C"

namespace {
// Checks of fp8_quantise's arguments other than the workspace; *empty is set
// when there is nothing to cast (rows == 0 or cols == 0).
int32_t quantise_checks(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx, int32_t fmt,
                        int32_t margin, const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits,
                        uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT, bool* empty) {
    *empty = false;
    if (!dt_ok(dt) || !fmt_ok(fmt) || rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim)
        return FP8_EINVAL;
    if (margin > FP8_MAX_MARGIN || margin < -FP8_MAX_MARGIN) return FP8_EINVAL;
    if (!bias || !aligned(bias, 4)) return FP8_EINVAL;
    if ((amax_bits && !aligned(amax_bits, 4)) || (flags && !aligned(flags, 4))) return FP8_EINVAL;
    if (bias_pred && !aligned(bias_pred, 4)) return FP8_EINVAL;
    if (rows == 0 || cols == 0) {
        *empty = true;
        return FP8_OK;
    }
    if (!x || (!q && !qT)) return FP8_EINVAL;
    if (!aligned(x, esize(dt))) return FP8_EINVAL;
    if (ldx < cols || (q && ldq < cols) || (qT && ldqT < rows)) return FP8_EINVAL;
    if (quantise_tiles_upto(rows, cols, INT32_MAX) < 0) return FP8_ENOTSUP;
    return FP8_OK;
}
}  // namespace

extern "C" {

int32_t fp8_quantise(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                     int32_t fmt, int32_t margin, const int32_t* bias_pred, int32_t* bias,
                     uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT,
                     int64_t ldqT, void* ws, size_t ws_bytes, void* stream) {
    bool empty;
    const int32_t st = quantise_checks(x, dt, rows, cols, ldx, fmt, margin, bias_pred, bias, amax_bits, flags, q,
                                       ldq, qT, ldqT, &empty);
    if (st != FP8_OK) return st;
    if (empty)  // amax 0: bias 0 and the zero flag, nothing to cast
        return launch_scale_bias(x, dt, 0, fmt, margin, bias, amax_bits, flags, nullptr, as_stream(stream));
    if (!ws || !aligned(ws, 4) || ws_bytes < fp8_quantise_ws_bytes(rows, cols)) return FP8_EINVAL;
    return launch_quantise(x, dt, rows, cols, ldx, fmt, margin, bias_pred, bias, amax_bits, flags,
                           q, ldq, qT, ldqT, (uint32_t*)ws, as_stream(stream));
}

}  // extern "C"

// ---- fp8_quantise without a caller workspace (fp8_quantise_noalloc)
// The quantise's scratch words (the prediction the codes were cast with, one
// maximum per 128 x 128 tile) live in this file-scope device array; every GPU
// the library runs on holds its own copy until the process ends.  Host code
// never uses the array's name as an address: each device's address comes
// from hipGetSymbolAddress, taken once with that device current.
static __device__ __align__(256) uint32_t scratch[FP8_NOALLOC_SCRATCH_BYTES / sizeof(uint32_t)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint32_t* g_scratch_ptr[kMaxDevices];  // per device; null until resolved

// Device address of the current device's scratch array.
int32_t current_scratch(uint32_t** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FP8_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FP8_EHIP;
        g_scratch_ptr[dev] = (uint32_t*)p;
    }
    *out = g_scratch_ptr[dev];
    return FP8_OK;
}
}  // namespace

extern "C" {

int32_t fp8_quantise_noalloc(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx, int32_t fmt,
                             int32_t margin, const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits,
                             uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT, void* stream) {
    bool empty;
    const int32_t st = quantise_checks(x, dt, rows, cols, ldx, fmt, margin, bias_pred, bias, amax_bits, flags, q,
                                       ldq, qT, ldqT, &empty);
    if (st != FP8_OK) return st;
    if (empty) return launch_scale_bias(x, dt, 0, fmt, margin, bias, amax_bits, flags, nullptr, as_stream(stream));
    if (quantise_tiles_upto(rows, cols, FP8_NOALLOC_MAX_TILES) < 0) return FP8_EINVAL;
    int cur = -1;
    hipDevice_t sdev = -1;
    if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(as_stream(stream), &sdev) != hipSuccess)
        return FP8_EHIP;
    if (sdev != cur) return FP8_EINVAL;  // the scratch address is the current device's
    uint32_t* ws = nullptr;
    const int32_t sst = current_scratch(&ws);
    if (sst != FP8_OK) return sst;
    return launch_quantise(x, dt, rows, cols, ldx, fmt, margin, bias_pred, bias, amax_bits, flags, q, ldq, qT, ldqT,
                           ws, as_stream(stream));
}

int32_t fp8_quantise_delayed(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx, int32_t fmt,
                             int32_t margin, int32_t* bias, uint32_t* history, int64_t history_len, uint32_t* count,
                             uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                             void* ws, size_t ws_bytes, void* stream) {
    bool empty;
    const int32_t st = quantise_checks(x, dt, rows, cols, ldx, fmt, margin, nullptr, bias, amax_bits, flags, q, ldq,
                                       qT, ldqT, &empty);
    if (st != FP8_OK) return st;
    if (history_len < 1 || history_len > 65536 || !history || !aligned(history, 4) || !count || !aligned(count, 4))
        return FP8_EINVAL;
    if (!ws || !aligned(ws, 4)) return FP8_EINVAL;
    if (!empty && ws_bytes < fp8_quantise_ws_bytes(rows, cols)) return FP8_EINVAL;
    if (empty && ws_bytes < sizeof(uint32_t)) return FP8_EINVAL;
    return launch_quantise_delayed(x, dt, empty ? 0 : rows, empty ? 0 : cols, ldx, fmt, margin, bias, history,
                                   (int)history_len, count, amax_bits, flags, q, ldq, qT, ldqT, (uint32_t*)ws,
                                   as_stream(stream));
}

int32_t fp8_quantise_batch(int32_t n, const fp8_quantise_args* t, int32_t dt, int32_t fmt, int32_t margin,
                           void* stream) {
    if (n == 0) return FP8_OK;
    if (n < 0 || n > FP8_QUANTISE_BATCH_MAX || !t) return FP8_EINVAL;
    if (!dt_ok(dt) || !fmt_ok(fmt) || margin > FP8_MAX_MARGIN || margin < -FP8_MAX_MARGIN) return FP8_EINVAL;
    QuantDesc d[kQBatch];
    int m = 0, npred = 0;
    int64_t tiles = 0;
    for (int i = 0; i < n; ++i) {
        const fp8_quantise_args& a = t[i];
        if (a.rows < 0 || a.cols < 0 || a.rows > kMaxDim || a.cols > kMaxDim) return FP8_EINVAL;
        if (!a.bias || !aligned(a.bias, 4)) return FP8_EINVAL;
        if ((a.amax_bits && !aligned(a.amax_bits, 4)) || (a.flags && !aligned(a.flags, 4))) return FP8_EINVAL;
        if (a.bias_pred && !aligned(a.bias_pred, 4)) return FP8_EINVAL;
        if (a.rows == 0 || a.cols == 0) continue;  // handled below, like fp8_quantise
        if (!a.x || (!a.q && !a.qT) || !a.ws) return FP8_EINVAL;
        if (!aligned(a.x, esize(dt)) || !aligned(a.ws, 4)) return FP8_EINVAL;
        if (a.ldx < a.cols || (a.q && a.ldq < a.cols) || (a.qT && a.ldqT < a.rows)) return FP8_EINVAL;
        if (a.ws_bytes < fp8_quantise_ws_bytes(a.rows, a.cols)) return FP8_EINVAL;
        const int64_t nt = quantise_tiles_upto(a.rows, a.cols, INT32_MAX);
        if (nt < 0) return FP8_ENOTSUP;
        tiles += nt;
        npred += a.bias_pred ? 1 : 0;
        d[m++] = QuantDesc{a.x, a.rows, a.cols, a.ldx, a.bias_pred, a.bias, a.amax_bits, a.flags,
                           a.q, a.ldq, a.qT, a.ldqT, (uint32_t*)a.ws};
    }
    if (npred != 0 && npred != m) return FP8_EINVAL;
    if (tiles > INT32_MAX) return FP8_ENOTSUP;
    for (int i = 0; i < n; ++i) {
        const fp8_quantise_args& a = t[i];
        if (a.rows == 0 || a.cols == 0) {
            const int32_t st = launch_scale_bias(a.x, dt, 0, fmt, margin, a.bias, a.amax_bits, a.flags, nullptr,
                                                 as_stream(stream));
            if (st != FP8_OK) return st;
        }
    }
    return m > 0 ? launch_quantise_batch(m, d, dt, fmt, margin, as_stream(stream)) : FP8_OK;
}

int32_t fp8_bias_from_amax(const uint32_t* amax_bits, int32_t fmt, int32_t margin, int32_t* bias,
                           uint32_t* flags, void* stream) {
    if (!fmt_ok(fmt) || margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN) return FP8_EINVAL;
    if (!amax_bits || !bias || !aligned(amax_bits, 4) || !aligned(bias, 4)) return FP8_EINVAL;
    if (flags && !aligned(flags, 4)) return FP8_EINVAL;
    return launch_bias_from_amax(amax_bits, fmt, margin, bias, flags, as_stream(stream));
}

int32_t fp8_cast_e4(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                    const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                    void* stream) {
    return cast_common(x, dt, rows, cols, ldx, bias, q, ldq, qT, ldqT, FP8_E4M3, stream);
}

int32_t fp8_cast_e5(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                    const int32_t* bias, uint8_t* q, int64_t ldq, uint8_t* qT, int64_t ldqT,
                    void* stream) {
    return cast_common(x, dt, rows, cols, ldx, bias, q, ldq, qT, ldqT, FP8_E5M2, stream);
}

int32_t fp8_linear_fwd(const uint8_t* x8, const int32_t* bx, const uint8_t* w8t, const int32_t* bw,
                       void* y, int32_t y_dt, int64_t M, int64_t N, int64_t K,
                       uint32_t* y_amax_bits, void* stream) {
    return gemm_common(x8, FP8_E4M3, bx, w8t, FP8_E4M3, bw, y, y_dt, M, N, K, y_amax_bits, stream);
}

int32_t fp8_linear_bwd_dx(const uint8_t* dy8, const int32_t* bg, const uint8_t* w8,
                          const int32_t* bw, void* dx, int32_t dx_dt, int64_t M, int64_t N,
                          int64_t K, uint32_t* dx_amax_bits, void* stream) {
    // dX [M, K] = dY8 [M, N] . W8 [K, N]^T: contraction over N.
    return gemm_common(dy8, FP8_E5M2, bg, w8, FP8_E4M3, bw, dx, dx_dt, M, K, N, dx_amax_bits, stream);
}

int32_t fp8_linear_bwd_dw(const uint8_t* x8t, const int32_t* bx, const uint8_t* dy8t,
                          const int32_t* bg, void* dw, int32_t dw_dt, int64_t M, int64_t N,
                          int64_t K, void* stream) {
    // dW [K, N] = X8T [K, M] . dY8T [N, M]^T: contraction over M.
    return gemm_common(x8t, FP8_E4M3, bx, dy8t, FP8_E5M2, bg, dw, dw_dt, K, N, M, nullptr, stream);
}

size_t fp8_linear_bias_ws_bytes(void) { return 2 * sizeof(uint32_t); }

namespace {
// C [rows, cols] = 2^-(*ba + *bb) A [rows, kc] . B [cols, kc]^T with the Eq. 3
// bias of C taken in the same launch (see fp8_linear_fwd_bias).
int32_t gemm_bias_common(const uint8_t* a, int fa, const int32_t* ba, const uint8_t* b, int fb,
                         const int32_t* bb, void* c, int32_t c_dt, int64_t rows, int64_t cols, int64_t kc,
                         int32_t fmt, int32_t margin, int32_t* bias, uint32_t* amax_bits, uint32_t* flags,
                         void* ws, size_t ws_bytes, void* stream) {
    if (!dt_ok(c_dt) || !fmt_ok(fmt) || rows < 0 || cols < 0 || kc < 0 || rows > kMaxDim || cols > kMaxDim ||
        kc > kMaxDim)
        return FP8_EINVAL;
    if (margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN) return FP8_EINVAL;
    if (!bias || !aligned(bias, 4)) return FP8_EINVAL;
    if ((amax_bits && !aligned(amax_bits, 4)) || (flags && !aligned(flags, 4))) return FP8_EINVAL;
    if (!ws || !aligned(ws, 4) || ws_bytes < fp8_linear_bias_ws_bytes()) return FP8_EINVAL;
    if (rows == 0 || cols == 0)  // an empty output has amax 0
        return launch_scale_bias(nullptr, FP8_DT_BF16, 0, fmt, margin, bias, amax_bits, flags, nullptr,
                                 as_stream(stream));
    if (!c || !ba || !bb || (kc > 0 && (!a || !b))) return FP8_EINVAL;
    if (!aligned(c, esize(c_dt)) || !aligned(ba, 4) || !aligned(bb, 4)) return FP8_EINVAL;
    if (!operands_ok(a, b, kc)) return FP8_EINVAL;
    if (rows > INT32_MAX || cols > INT32_MAX) return FP8_ENOTSUP;
    return launch_gemm_nt_bias(a, fa, ba, b, fb, bb, c, c_dt, rows, cols, kc, fmt, margin, bias, amax_bits, flags,
                               (uint32_t*)ws, as_stream(stream));
}
}  // namespace

int32_t fp8_linear_fwd_bias(const uint8_t* x8, const int32_t* bx, const uint8_t* w8t, const int32_t* bw,
                            void* y, int32_t y_dt, int64_t M, int64_t N, int64_t K, int32_t y_fmt,
                            int32_t margin, int32_t* y_bias, uint32_t* y_amax_bits, uint32_t* y_flags,
                            void* ws, size_t ws_bytes, void* stream) {
    return gemm_bias_common(x8, FP8_E4M3, bx, w8t, FP8_E4M3, bw, y, y_dt, M, N, K, y_fmt, margin, y_bias,
                            y_amax_bits, y_flags, ws, ws_bytes, stream);
}

int32_t fp8_linear_bwd_dx_bias(const uint8_t* dy8, const int32_t* bg, const uint8_t* w8, const int32_t* bw,
                               void* dx, int32_t dx_dt, int64_t M, int64_t N, int64_t K, int32_t dx_fmt,
                               int32_t margin, int32_t* dx_bias, uint32_t* dx_amax_bits, uint32_t* dx_flags,
                               void* ws, size_t ws_bytes, void* stream) {
    // dX [M, K] = dY8 [M, N] . W8 [K, N]^T: contraction over N.
    return gemm_bias_common(dy8, FP8_E5M2, bg, w8, FP8_E4M3, bw, dx, dx_dt, M, K, N, dx_fmt, margin, dx_bias,
                            dx_amax_bits, dx_flags, ws, ws_bytes, stream);
}

size_t fp8_linear_quantise_ws_bytes(int64_t M, int64_t N) {
    if (M <= 0 || N <= 0 || M > kMaxDim || N > kMaxDim) return 0;
    return (size_t)gemm_quantise_ws_words(M, N) * sizeof(uint32_t);
}

namespace {
// C [rows, cols] (bf16) = 2^-(*ba + *bb) A [rows, kc] . B [cols, kc]^T, then
// its bias and codes (see fp8_linear_fwd_quantise).
int32_t gemm_quantise_common(const uint8_t* a, int fa, const int32_t* ba, const uint8_t* b,
                             const int32_t* bb, void* c, int64_t rows, int64_t cols, int64_t kc,
                             int32_t fmt, int32_t margin, const int32_t* pred, int32_t* bias,
                             uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, uint8_t* qT,
                             int64_t ldqT, void* ws, size_t ws_bytes, void* stream) {
    if (!fmt_ok(fmt) || rows < 0 || cols < 0 || kc < 0 || rows > kMaxDim || cols > kMaxDim || kc > kMaxDim)
        return FP8_EINVAL;
    if (margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN) return FP8_EINVAL;
    if (!bias || !aligned(bias, 4) || (pred && !aligned(pred, 4))) return FP8_EINVAL;
    if ((amax_bits && !aligned(amax_bits, 4)) || (flags && !aligned(flags, 4))) return FP8_EINVAL;
    if (rows == 0 || cols == 0)
        return launch_scale_bias(nullptr, FP8_DT_BF16, 0, fmt, margin, bias, amax_bits, flags, nullptr,
                                 as_stream(stream));
    if (!c || !ba || !bb || !q || (kc > 0 && (!a || !b)) || !ws) return FP8_EINVAL;
    if (!aligned(c, 2) || !aligned(ba, 4) || !aligned(bb, 4) || !aligned(ws, 4)) return FP8_EINVAL;
    if (!operands_ok(a, b, kc)) return FP8_EINVAL;
    if (ldq < cols || (qT && ldqT < rows)) return FP8_EINVAL;
    if (ws_bytes < fp8_linear_quantise_ws_bytes(rows, cols)) return FP8_EINVAL;
    if (rows > INT32_MAX || cols > INT32_MAX) return FP8_ENOTSUP;
    return launch_gemm_nt_quantise(a, fa, ba, b, FP8_E4M3, bb, c, rows, cols, kc, fmt, margin, pred, bias,
                                   amax_bits, flags, q, ldq, qT, ldqT, (uint32_t*)ws, as_stream(stream));
}
}  // namespace

int32_t fp8_linear_fwd_quantise(const uint8_t* x8, const int32_t* bx, const uint8_t* w8t,
                                const int32_t* bw, void* y, int64_t M, int64_t N, int64_t K,
                                int32_t y_fmt, int32_t margin, const int32_t* y_bias_pred,
                                int32_t* y_bias, uint32_t* y_amax_bits, uint32_t* y_flags,
                                uint8_t* y8, int64_t ldy8, uint8_t* y8t, int64_t ldy8t, void* ws,
                                size_t ws_bytes, void* stream) {
    return gemm_quantise_common(x8, FP8_E4M3, bx, w8t, bw, y, M, N, K, y_fmt, margin, y_bias_pred,
                                y_bias, y_amax_bits, y_flags, y8, ldy8, y8t, ldy8t, ws, ws_bytes,
                                stream);
}

int32_t fp8_linear_bwd_dx_quantise(const uint8_t* dy8, const int32_t* bg, const uint8_t* w8,
                                   const int32_t* bw, void* dx, int64_t M, int64_t N, int64_t K,
                                   int32_t dx_fmt, int32_t margin, const int32_t* dx_bias_pred,
                                   int32_t* dx_bias, uint32_t* dx_amax_bits, uint32_t* dx_flags,
                                   uint8_t* dx8, int64_t lddx8, uint8_t* dx8t, int64_t lddx8t,
                                   void* ws, size_t ws_bytes, void* stream) {
    // dX [M, K] = dY8 [M, N] . W8 [K, N]^T: contraction over N.
    return gemm_quantise_common(dy8, FP8_E5M2, bg, w8, bw, dx, M, K, N, dx_fmt, margin, dx_bias_pred,
                                dx_bias, dx_amax_bits, dx_flags, dx8, lddx8, dx8t, lddx8t, ws, ws_bytes,
                                stream);
}

int32_t fp8_quantise_segments(const void* x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx, int32_t fmt,
                              int32_t margin, const int32_t* offsets, int64_t nseg, int32_t* bias,
                              uint32_t* amax_bits, uint32_t* flags, int32_t* row_bias, uint8_t* q, int64_t ldq,
                              uint8_t* qT, int64_t ldqT, void* stream) {
    if (!dt_ok(dt) || !fmt_ok(fmt) || rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return FP8_EINVAL;
    if (margin < -FP8_MAX_MARGIN || margin > FP8_MAX_MARGIN) return FP8_EINVAL;
    if (nseg < 1 || nseg > INT32_MAX) return FP8_EINVAL;
    if (!offsets || !bias || !amax_bits || !aligned(offsets, 4) || !aligned(bias, 4) || !aligned(amax_bits, 4))
        return FP8_EINVAL;
    if (flags && !aligned(flags, 4)) return FP8_EINVAL;
    if (rows > 0 && (!row_bias || !aligned(row_bias, 4))) return FP8_EINVAL;
    if (rows > 0 && cols > 0) {
        if (!x || !aligned(x, esize(dt)) || ldx < cols) return FP8_EINVAL;
        if ((q && ldq < cols) || (qT && ldqT < rows)) return FP8_EINVAL;
    }
    return launch_quantise_segments(x, dt, rows, cols, ldx, fmt, margin, offsets, (int)nseg, bias, amax_bits, flags,
                                    row_bias, q, ldq, qT, ldqT, as_stream(stream));
}

int32_t fp8_linear_fwd_rows(const uint8_t* x8, const int32_t* bx_rows, const uint8_t* w8t, const int32_t* bw,
                            void* y, int32_t y_dt, int64_t M, int64_t N, int64_t K, uint32_t* y_amax_bits,
                            void* stream) {
    if (!dt_ok(y_dt) || M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return FP8_EINVAL;
    if (y_amax_bits && !aligned(y_amax_bits, 4)) return FP8_EINVAL;
    if (M == 0 || N == 0)  // no output: its amax is 0
        return y_amax_bits ? launch_fill_u32(y_amax_bits, 0u, as_stream(stream)) : FP8_OK;
    if (!y || !bx_rows || !bw || (K > 0 && (!x8 || !w8t))) return FP8_EINVAL;
    if (!aligned(y, esize(y_dt)) || !aligned(bx_rows, 4) || !aligned(bw, 4)) return FP8_EINVAL;
    if (!operands_ok(x8, w8t, K)) return FP8_EINVAL;
    if (M > INT32_MAX || N > INT32_MAX) return FP8_ENOTSUP;
    return launch_gemm_nt(x8, FP8_E4M3, bx_rows, w8t, FP8_E4M3, bw, y, y_dt, M, N, K, y_amax_bits,
                          as_stream(stream), 1);
}

int32_t fp8_bias_mode(const int32_t* bias, int64_t n, int32_t* ring, int64_t capacity, uint32_t* count,
                      void* stream) {
    if (n < 0 || capacity < 1 || !ring || !count || !aligned(ring, 4) || !aligned(count, 4)) return FP8_EINVAL;
    if (n == 0) return FP8_OK;
    if (!bias || !aligned(bias, 4)) return FP8_EINVAL;
    return launch_bias_mode(bias, n, ring, capacity, count, as_stream(stream));
}

int32_t ptq_quantise_weights(const void* w, int32_t dt, int64_t K, int64_t N, uint8_t* w8,
                             uint8_t* w8t, int32_t* bw, uint32_t* flags, void* ws, size_t ws_bytes,
                             void* stream) {
    if (!dt_ok(dt) || K < 0 || N < 0 || K > kMaxDim || N > kMaxDim) return FP8_EINVAL;
    if (N > 0 && K > kMaxDim * 64 / N) return FP8_EINVAL;  // K * N beyond what fp8_scale_bias accepts
    if (!bw || (!w8 && !w8t)) return FP8_EINVAL;
    int32_t st = fp8_scale_bias(w, dt, K * N, FP8_E4M3, 0, bw, nullptr, flags, ws, ws_bytes, stream);
    if (st != FP8_OK || K == 0 || N == 0) return st;
    return cast_common(w, dt, K, N, N, bw, w8, N, w8t, K, FP8_E4M3, stream);
}

// ---- decoder-layer glue (App. E)
size_t llama_rmsnorm_ws_bytes(int64_t rows) {
    if (rows <= 0 || rows > kMaxDim) return 0;
    return (size_t)(1 + glue_parts_rmsnorm(rows)) * sizeof(uint32_t);
}

int32_t llama_rmsnorm_quantise(const void* x, int64_t ldx, const void* res, int64_t ldr, const void* g, int64_t rows,
                               int64_t cols, float eps, void* h, int64_t ldh, void* y, int64_t ldy, int32_t fmt,
                               int32_t margin, const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits,
                               uint32_t* flags, uint8_t* q, int64_t ldq, void* ws, size_t ws_bytes, void* stream) {
    if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return FP8_EINVAL;
    if (!(eps >= 0.0f) || eps > 3.0e38f) return FP8_EINVAL;
    FusedQuant fq;
    if (rows == 0 || cols == 0) return glue_empty(fmt, margin, bias, amax_bits, flags, q, stream);
    if (!x || !g || !y || !a16(x) || !a16(g) || !a16(y) || cols % 8) return FP8_EINVAL;
    if (!rows_ok(ldx, cols) || !rows_ok(ldy, cols)) return FP8_EINVAL;
    if (res && (!a16(res) || !rows_ok(ldr, cols))) return FP8_EINVAL;
    if (h && (!a16(h) || !rows_ok(ldh, cols))) return FP8_EINVAL;
    if (rows > INT32_MAX) return FP8_ENOTSUP;
    const int32_t st = glue_quant(fmt, margin, bias_pred, bias, amax_bits, flags, q, ldq, cols, ws, ws_bytes,
                                  1 + glue_parts_rmsnorm(rows), &fq);
    if (st != FP8_OK) return st;
    return launch_rmsnorm((const uint16_t*)x, ldx, (const uint16_t*)res, ldr, (const uint16_t*)g, rows, cols, eps,
                          (uint16_t*)h, ldh, (uint16_t*)y, ldy, &fq, as_stream(stream));
}

int32_t llama_rope_table(int64_t seq_len, int32_t d_head, double theta, float* table, void* stream) {
    if (seq_len < 1 || seq_len > kMaxDim || d_head < 16 || d_head % 16 || d_head > 4096) return FP8_EINVAL;
    if (!(theta > 0.0) || theta > 1e300 || !table || !aligned(table, 8)) return FP8_EINVAL;
    return launch_rope_table(seq_len, d_head, theta, table, as_stream(stream));
}

int32_t llama_rope(void* x, int64_t rows, int64_t ld, int32_t n_heads, int32_t d_head, int64_t seq_len,
                   const float* table, void* stream) {
    if (rows < 0 || rows > kMaxDim || n_heads < 0 || seq_len < 1 || seq_len > kMaxDim) return FP8_EINVAL;
    if (d_head < 16 || d_head % 16 || d_head > 4096) return FP8_EINVAL;
    if (rows == 0 || n_heads == 0) return FP8_OK;
    if (!x || !a16(x) || !rows_ok(ld, (int64_t)n_heads * d_head) || !table || !aligned(table, 8)) return FP8_EINVAL;
    return launch_rope((uint16_t*)x, rows, ld, n_heads, d_head, seq_len, table, as_stream(stream));
}

size_t llama_attention_ws_bytes(int64_t rows, int64_t seq_len, int32_t n_heads) {
    if (rows <= 0 || seq_len < 1 || n_heads < 1 || rows > kMaxDim || seq_len > kMaxDim) return 0;
    return (size_t)(1 + glue_parts_attention(rows, seq_len, n_heads)) * sizeof(uint32_t);
}

int32_t llama_attention(const void* qkv, int64_t rows, int64_t ld, int64_t seq_len, int32_t n_heads,
                        int32_t n_kv_heads, int32_t d_head, void* o, int64_t ldo, int32_t fmt, int32_t margin,
                        const int32_t* bias_pred, int32_t* bias, uint32_t* amax_bits, uint32_t* flags, uint8_t* q,
                        int64_t ldq, void* ws, size_t ws_bytes, void* stream) {
    if (rows < 0 || rows > kMaxDim || seq_len < 1 || seq_len > kMaxDim) return FP8_EINVAL;
    if (n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads) return FP8_EINVAL;
    if (d_head != 128) return FP8_ENOTSUP;
    FusedQuant fq;
    if (rows == 0) return glue_empty(fmt, margin, bias, amax_bits, flags, q, stream);
    const int64_t cols = (int64_t)n_heads * d_head;
    if (!qkv || !o || !a16(qkv) || !a16(o)) return FP8_EINVAL;
    if (!rows_ok(ld, (int64_t)(n_heads + 2 * n_kv_heads) * d_head) || !rows_ok(ldo, cols)) return FP8_EINVAL;
    if (glue_parts_attention(rows, seq_len, n_heads) > INT32_MAX) return FP8_ENOTSUP;
    if ((seq_len < rows ? seq_len : rows) > ((int64_t)1 << 30)) return FP8_ENOTSUP;  // positions are 32-bit
    if (ld > ((int64_t)1 << 24)) return FP8_ENOTSUP;  // 32-bit offsets within a block of 64 rows
    const int32_t st = glue_quant(fmt, margin, bias_pred, bias, amax_bits, flags, q, ldq, cols, ws, ws_bytes,
                                  1 + glue_parts_attention(rows, seq_len, n_heads), &fq);
    if (st != FP8_OK) return st;
    return launch_attention((const uint16_t*)qkv, rows, ld, seq_len, n_heads, n_kv_heads, (uint16_t*)o, ldo, &fq,
                            as_stream(stream));
}

size_t llama_swiglu_ws_bytes(void) { return (size_t)(1 + glue_parts_swiglu()) * sizeof(uint32_t); }

int32_t llama_swiglu_quantise(const void* gu, int64_t ldgu, int64_t rows, int64_t ffn, void* a, int64_t lda,
                              int32_t fmt, int32_t margin, const int32_t* bias_pred, int32_t* bias,
                              uint32_t* amax_bits, uint32_t* flags, uint8_t* q, int64_t ldq, void* ws,
                              size_t ws_bytes, void* stream) {
    if (rows < 0 || ffn < 0 || rows > kMaxDim || ffn > kMaxDim) return FP8_EINVAL;
    FusedQuant fq;
    if (rows == 0 || ffn == 0) return glue_empty(fmt, margin, bias, amax_bits, flags, q, stream);
    if (!gu || !a || !a16(gu) || !a16(a) || ffn % 8) return FP8_EINVAL;
    if (!rows_ok(ldgu, 2 * ffn) || !rows_ok(lda, ffn)) return FP8_EINVAL;
    const int32_t st = glue_quant(fmt, margin, bias_pred, bias, amax_bits, flags, q, ldq, ffn, ws, ws_bytes,
                                  1 + glue_parts_swiglu(), &fq);
    if (st != FP8_OK) return st;
    return launch_swiglu((const uint16_t*)gu, ldgu, rows, ffn, (uint16_t*)a, lda, &fq, as_stream(stream));
}

int32_t llama_residual_add(const void* a, const void* b, void* out, int64_t n, void* stream) {
    if (n < 0 || n > kMaxDim * 64 || n % 8) return FP8_EINVAL;
    if (n == 0) return FP8_OK;
    if (!a || !b || !out || !a16(a) || !a16(b) || !a16(out)) return FP8_EINVAL;
    return launch_residual_add((const uint16_t*)a, (const uint16_t*)b, (uint16_t*)out, n, as_stream(stream));
}

}  // extern "C"
