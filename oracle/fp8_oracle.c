/*
 * fp8_oracle.c -- CPU oracle for the FP8 linear layer with per-tensor
 * power-of-two scaling biases (Perez et al., "Training and inference of large
 * language models using 8-bit floating point", arXiv 2309.17224).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * statement of what the GPU path computes.  Only the test-suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load it.  It shares no
 * code, header or table with the HIP library: it includes nothing but the C
 * standard library and derives every constant it uses from the format
 * definitions below.
 *
 * Every routine takes host pointers and runs synchronously.  Floating-point
 * arithmetic is done in double precision (fp64).
 *
 * Paper passages followed (section / equation / table of the paper):
 *   formats       App. A Eq. 4 and Table 7, App. B (special values)
 *   amax, bias    Sec. 2.3 Eq. 3 (FP8-AMAX), Sec. 3 (granularity), Sec. 3.2 (margin)
 *   scale, cast   Sec. 2.1 Eq. 1 (bias added to the exponent = x * 2^b),
 *                 App. A (overflow is clipped to the maximum)
 *   matmul        Sec. 2 / Sec. 2.2 (FP8 inputs, higher-precision accumulation),
 *                 Sec. 2.1 Eq. 2 (unscale by -(b_w + b_x))
 *   PTQ           Sec. 3.1 (weight bias computed once at checkpoint load)
 *
 * Readings where the paper is silent (each one is listed with its reason in
 * the design notes of the repository):
 *   - the formats consumed by the matrix cores are the OCP ones, which are the
 *     "(b)" rows of Table 7; the paper's default "(a)" rows are implemented
 *     here as well, for comparison only;
 *   - rounding of the cast is round-to-nearest, ties to the even code;
 *   - values beyond the largest finite number (including infinities) clip to
 *     that number with their sign; NaN becomes the canonical NaN code;
 *   - amax of a tensor holding a NaN is NaN; -0 counts as 0;
 *   - a non-finite amax gives bias 0 and sets flag bit 0, a zero amax gives
 *     bias 0 and sets flag bit 1;
 *   - the margin is subtracted from the floor of Eq. 3;
 *   - matmul output is rounded once, from the fp64 sum, to fp32 or bf16.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---- identifiers (the oracle's own; same numeric meaning as the library) */
enum { ORC_E4M3 = 0, ORC_E5M2 = 1, ORC_E4_A = 2, ORC_E5_A = 3 };
enum { ORC_BF16 = 0, ORC_F32 = 1 };
enum { ORC_FLAG_NONFINITE = 1u, ORC_FLAG_ZERO = 2u };

/* ---- FP8 formats (Table 7 and App. B) ------------------------------------
 * A code is sign | exponent field (E bits) | mantissa field (M bits).
 * Normal value:    (-1)^s * (1 + m / 2^M) * 2^(e - bias)
 * Subnormal (e=0): (-1)^s * (m / 2^M) * 2^(1 - bias)
 * Special values differ between the proposals (App. B):
 *   E4 (b): only the all-ones exponent+mantissa pattern is NaN, no infinity.
 *   E5 (b): IEEE-like, all-ones exponent = infinity (m = 0) or NaN (m != 0).
 *   (a) formats: the negative-zero code 0x80 is the single NaN/inf code. */
typedef struct {
    int ebits, mbits, bias;
    int special; /* 0: E4(b) rule, 1: IEEE rule, 2: negative-zero rule */
} fmt_desc;

static const fmt_desc FMTS[4] = {
    {4, 3, 7, 0},  /* ORC_E4M3 = E4 (b) */
    {5, 2, 15, 1}, /* ORC_E5M2 = E5 (b) */
    {4, 3, 8, 2},  /* ORC_E4_A = E4 (a) */
    {5, 2, 16, 2}, /* ORC_E5_A = E5 (a) */
};

static int fmt_ok(int fmt) { return fmt >= 0 && fmt < 4; }

double oracle_fp8_decode(int fmt, int code)
{
    if (!fmt_ok(fmt) || code < 0 || code > 255)
        return NAN;
    const fmt_desc *f = &FMTS[fmt];
    int s = (code >> 7) & 1;
    int e = (code >> f->mbits) & ((1 << f->ebits) - 1);
    int m = code & ((1 << f->mbits) - 1);
    int emax_field = (1 << f->ebits) - 1;
    if (f->special == 0 && e == emax_field && m == (1 << f->mbits) - 1)
        return NAN;
    if (f->special == 1 && e == emax_field)
        return m == 0 ? (s ? -INFINITY : INFINITY) : NAN;
    if (f->special == 2 && code == 0x80)
        return NAN;
    double mag;
    if (e == 0)
        mag = ldexp((double)m, 1 - f->bias - f->mbits);
    else
        mag = ldexp((double)((1 << f->mbits) + m), e - f->bias - f->mbits);
    return s ? -mag : mag;
}

/* Largest finite value of the format: found by looking at every code. */
double oracle_fp8_max_num(int fmt)
{
    double best = 0.0;
    for (int c = 0; c < 256; ++c) {
        double v = oracle_fp8_decode(fmt, c);
        if (isfinite(v) && v > best)
            best = v;
    }
    return best;
}

static int max_code(int fmt)
{
    double mx = oracle_fp8_max_num(fmt);
    for (int c = 0; c < 128; ++c)
        if (oracle_fp8_decode(fmt, c) == mx)
            return c;
    return 0;
}

/* Encode a real number (given exactly as a double) into the format:
 * NaN -> canonical NaN; |v| >= max -> +-max (clipping, App. A);
 * otherwise the nearest representable magnitude, ties to the even code.
 * The nearest value is found by looking at every non-negative code.  The
 * distances |a - value| are exact except when a and the value are more than
 * ~29 binades apart, where the comparison is decided by orders of magnitude
 * and no tie can arise. */
int oracle_fp8_encode(int fmt, double v)
{
    if (!fmt_ok(fmt))
        return -1;
    const fmt_desc *f = &FMTS[fmt];
    int neg = signbit(v) ? 1 : 0;
    if (isnan(v))
        return f->special == 2 ? 0x80 : (0x7F | (neg << 7));
    double a = fabs(v);
    double mx = oracle_fp8_max_num(fmt);
    int best;
    if (a >= mx) {
        best = max_code(fmt);
    } else {
        best = 0;
        double bestd = INFINITY;
        for (int c = 0; c < 128; ++c) {
            double val = oracle_fp8_decode(fmt, c);
            if (!isfinite(val))
                continue;
            double d = fabs(a - val);
            if (d < bestd || (d == bestd && (c & 1) == 0)) {
                best = c;
                bestd = d;
            }
        }
    }
    if (neg) {
        if (f->special == 2 && best == 0)
            return 0; /* (a) formats have no negative zero */
        return best | 0x80;
    }
    return best;
}

/* ---- table of decoded values, filled once (speeds up the scans only) ---- */
static double DEC[4][256];
static double MAXN[4];
static int MAXC[4];
static int tables_ready = 0;

static void init_tables(void)
{
    if (tables_ready)
        return;
#ifdef _OPENMP
#pragma omp critical(oracle_tables)
#endif
    {
        if (!tables_ready) {
            for (int f = 0; f < 4; ++f) {
                for (int c = 0; c < 256; ++c)
                    DEC[f][c] = oracle_fp8_decode(f, c);
                MAXN[f] = oracle_fp8_max_num(f);
                MAXC[f] = max_code(f);
            }
            tables_ready = 1;
        }
    }
}

/* Same rule as oracle_fp8_encode, reading the decoded values from the table. */
static uint8_t encode_tab(int fmt, double v)
{
    const fmt_desc *f = &FMTS[fmt];
    int neg = signbit(v) ? 1 : 0;
    if (isnan(v))
        return (uint8_t)(f->special == 2 ? 0x80 : (0x7F | (neg << 7)));
    double a = fabs(v);
    int best;
    if (a >= MAXN[fmt]) {
        best = MAXC[fmt];
    } else {
        best = 0;
        double bestd = INFINITY;
        for (int c = 0; c < 128; ++c) {
            double val = DEC[fmt][c];
            if (!isfinite(val))
                continue;
            double d = fabs(a - val);
            if (d < bestd || (d == bestd && (c & 1) == 0)) {
                best = c;
                bestd = d;
            }
        }
    }
    if (neg) {
        if (f->special == 2 && best == 0)
            return 0;
        return (uint8_t)(best | 0x80);
    }
    return (uint8_t)best;
}

/* ---- higher-precision inputs (Table 7: BF16 is the top half of FP32) ---- */
static double load_hp(const void *x, int dt, int64_t i)
{
    float f;
    if (dt == ORC_BF16) {
        uint32_t u = (uint32_t)((const uint16_t *)x)[i] << 16;
        memcpy(&f, &u, 4);
    } else {
        memcpy(&f, (const uint32_t *)x + i, 4);
    }
    return (double)f;
}

static uint32_t f32_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return u;
}

/* ---- amax: max |x_i| over the whole tensor (Eq. 3) ----------------------
 * Returned as the fp32 bit pattern of the amax (exact: inputs are bf16/fp32).
 * A NaN anywhere gives the canonical NaN 0x7FC00000. */
void oracle_amax(const void *x, int dt, int64_t n, uint32_t *amax_bits)
{
    double m = 0.0;
    int nan_seen = 0;
    for (int64_t i = 0; i < n; ++i) {
        double v = load_hp(x, dt, i);
        if (isnan(v)) {
            nan_seen = 1;
            continue;
        }
        double a = fabs(v);
        if (a > m)
            m = a;
    }
    *amax_bits = nan_seen ? 0x7FC00000u : f32_bits((float)m);
}

/* ---- scaling bias (Eq. 3) ------------------------------------------------
 * bias = floor(log2(max_num / amax)) - margin, evaluated exactly:
 * with amax = fa * 2^ea and max_num = fm * 2^em (frexp, fa, fm in [0.5, 1)),
 * log2(max_num / amax) = (em - ea) + log2(fm / fa) with fm / fa in (0.5, 2),
 * so the floor is (em - ea) when fm >= fa and (em - ea - 1) otherwise. */
int32_t oracle_bias_from_amax(uint32_t amax_bits, int fmt, int32_t margin, uint32_t *flags)
{
    init_tables();
    float af;
    memcpy(&af, &amax_bits, 4);
    double amax = fabs((double)af);
    if (!isfinite(amax)) {
        if (flags)
            *flags |= ORC_FLAG_NONFINITE;
        return 0;
    }
    if (amax == 0.0) {
        if (flags)
            *flags |= ORC_FLAG_ZERO;
        return 0;
    }
    int ea, em;
    double fa = frexp(amax, &ea);
    double fm = frexp(MAXN[fmt], &em);
    int32_t b = (em - ea) - (fm >= fa ? 0 : 1);
    return b - margin;
}

/* amax followed by the bias: the compute_bias step of the training and
 * inference procedures (Sec. 2.3, Sec. 3). */
int32_t oracle_fp8_scale_bias(const void *x, int dt, int64_t n, int fmt, int32_t margin,
                              int32_t *bias, uint32_t *amax_bits, uint32_t *flags)
{
    if (!fmt_ok(fmt) || (dt != ORC_BF16 && dt != ORC_F32) || n < 0)
        return 1;
    uint32_t a;
    oracle_amax(x, dt, n, &a);
    if (amax_bits)
        *amax_bits = a;
    *bias = oracle_bias_from_amax(a, fmt, margin, flags);
    return 0;
}

/* ---- scale then cast (Eq. 1): q = encode(x * 2^bias) ----------------------
 * x * 2^bias is exact in fp64 for every bf16/fp32 x and every bias the
 * library accepts.  q is [rows, cols] with row stride ldq; if qT is given it
 * receives the same codes transposed, [cols, rows] with row stride ldqT. */
int32_t oracle_fp8_cast(const void *x, int dt, int64_t rows, int64_t cols, int64_t ldx,
                        int fmt, int32_t bias, uint8_t *q, int64_t ldq,
                        uint8_t *qT, int64_t ldqT)
{
    if (!fmt_ok(fmt) || (dt != ORC_BF16 && dt != ORC_F32) || rows < 0 || cols < 0)
        return 1;
    init_tables();
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t c = 0; c < cols; ++c) {
            double v = ldexp(load_hp(x, dt, r * ldx + c), bias);
            uint8_t code = encode_tab(fmt, v);
            if (q)
                q[r * ldq + c] = code;
            if (qT)
                qT[c * ldqT + r] = code;
        }
    }
    return 0;
}

/* ---- rounding of an fp64 value to fp32 / bf16, once, ties to even -------
 * p significant bits, smallest normal exponent emin, largest exponent emax. */
static double round_to_format(double y, int p, int emin, int emax)
{
    if (!isfinite(y) || y == 0.0)
        return y;
    double a = fabs(y);
    int e;
    frexp(a, &e);          /* a = f * 2^e, f in [0.5, 1): floor(log2 a) = e - 1 */
    int ex = e - 1;
    if (ex < emin)
        ex = emin;             /* subnormal range keeps the smallest quantum */
    double quantum = ldexp(1.0, ex - (p - 1));
    double r = nearbyint(a / quantum) * quantum; /* default mode: ties to even */
    if (r >= ldexp(1.0, emax + 1))
        r = INFINITY;
    return y < 0 ? -r : r;
}

static void store_out(void *out, int out_dt, int64_t idx, double y)
{
    if (out_dt == ORC_F32) {
        float f = (float)round_to_format(y, 24, -126, 127);
        ((float *)out)[idx] = f;
    } else {
        double r = round_to_format(y, 8, -126, 127);
        float f = (float)r; /* exact: r has at most 8 significant bits */
        uint32_t u = isnan(y) ? 0x7FC00000u : f32_bits(f);
        ((uint16_t *)out)[idx] = (uint16_t)(u >> 16);
    }
}

/* ---- FP8 matmul with fp64 accumulation and unscale (Eq. 2) ---------------
 * out[r, j] = round_out( 2^-(ba + bb) * sum_k dec(A[i, k]) * dec(B[j, k]) )
 * Both operands are stored with the contraction index contiguous ("NT"):
 * A is [M, K] with row stride lda, B is [N, K] with row stride ldb.
 * If rows is given, output row r is computed from A row rows[r] (used to
 * sample a few rows of a large product); otherwise i = r.
 * out is [M, N] with row stride ldo, fp32 or bf16. */
int32_t oracle_gemm_nt(const uint8_t *a, int fmt_a, int32_t ba, int64_t lda,
                       const uint8_t *b, int fmt_b, int32_t bb, int64_t ldb,
                       int64_t M, int64_t N, int64_t K, const int64_t *rows,
                       void *out, int out_dt, int64_t ldo)
{
    if (!fmt_ok(fmt_a) || !fmt_ok(fmt_b) || M < 0 || N < 0 || K < 0)
        return 1;
    init_tables();
    const double *da = DEC[fmt_a];
    const double *db = DEC[fmt_b];
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int64_t r = 0; r < M; ++r) {
        int64_t i = rows ? rows[r] : r;
        const uint8_t *ar = a + i * lda;
        for (int64_t j = 0; j < N; ++j) {
            const uint8_t *br = b + j * ldb;
            double s = 0.0;
            for (int64_t k = 0; k < K; ++k)
                s += da[ar[k]] * db[br[k]];
            store_out(out, out_dt, r * ldo + j, ldexp(s, -(ba + bb)));
        }
    }
    return 0;
}

/* ---- post-training quantisation of one weight (Sec. 3.1) ----------------
 * W is [K, N]; W8 gets the E4 codes in the same layout, W8T (optional) the
 * transposed codes [N, K]; the bias is computed once from the whole tensor. */
int32_t oracle_ptq_quantise_weights(const void *w, int dt, int64_t K, int64_t N,
                                    uint8_t *w8, uint8_t *w8t, int32_t *bw, uint32_t *flags)
{
    int32_t st = oracle_fp8_scale_bias(w, dt, K * N, ORC_E4M3, 0, bw, NULL, flags);
    if (st)
        return st;
    return oracle_fp8_cast(w, dt, K, N, N, ORC_E4M3, *bw, w8, N, w8t, K);
}

/* ---- misc ---------------------------------------------------------------- */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Decode one bf16 pattern (used by tests that build bf16 inputs by hand). */
double oracle_bf16_to_double(uint16_t h)
{
    return load_hp(&h, ORC_BF16, 0);
}

/* Round an fp64 value to the bf16 bit pattern, once, ties to even. */
uint16_t oracle_round_bf16(double y)
{
    uint16_t h;
    store_out(&h, ORC_BF16, 0, y);
    return h;
}
