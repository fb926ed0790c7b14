/*
 * reqat_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU statement of what the microscaled-FP4
 * linear layer computes: E2M1 element codes with per-block scales (MXFP4 and
 * NVFP4), the quantize-dequantize ("fake-quant") output, and the block-scaled
 * FP4 x FP4 product.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this file's library.  It shares no
 * code, header, table or constant with the GPU library, and the GPU library
 * never calls it.
 *
 * Formats follow the ReQAT paper, App. A ("Microscaling Formats",
 * Tab. mx_configs) and the E2M1 layout named in its Sec. 1 (Introduction):
 *   MXFP4: E2M1 elements, E8M0 block scale, block of 32, no global scale.
 *   NVFP4: E2M1 elements, E4M3 block scale, block of 16, FP32 global scale.
 * The paper states no rounding, scale-selection or layout rule; the readings
 * used here are listed with each function (and in the design notes):
 *   - blocks run along the contiguous (reduction) dimension;
 *   - element rounding is round-to-nearest, ties to the even code, of the
 *     exact quotient |x| / (block scale * global scale), saturating at 6;
 *   - the block scale is the SMALLEST representable scale with
 *     block_absmax <= 6 * scale * global  ("ceil" rule), so no element clips;
 *   - the computed NVFP4 global scale is the smallest power of two 2^k,
 *     k >= -126, with tensor_absmax <= 6 * 448 * 2^k;
 *   - a block holding NaN or Inf gets a NaN scale and zero codes;
 *   - codes are packed two per byte, element 2i in bits 3:0.
 * Arithmetic is FP64 throughout.  Every rounding decision compares |x| with
 * a product of at most 31 significant bits, exact in FP64, so each decision is
 * that of exact real arithmetic.  The product reference is not exact in
 * general: a dequantized value code * s * g carries up to 30 significant bits
 * under a caller-given g (6 under a power-of-two g), so a product of two of
 * them may need 60 bits and is rounded once in FP64, and the sums over K are
 * rounded in FP64 too; both are many orders of magnitude below the 1e-3
 * tolerance the product is checked against.
 *
 * Parity status: every function here is pinned by a CPU test against an
 * independent statement (brute-force nearest search, torch's float8 and
 * bfloat16 conversions, closed forms, numpy matmul).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define ORC_FMT_NVFP4 0
#define ORC_FMT_MXFP4 1

/* ---------- element and scale formats (App. A, Tab. mx_configs) ---------- */

/* E2M1: sign bit 3, exponent bits 2:1 (bias 1), mantissa bit 0.
 * Exponent field 0 is subnormal: value = 0.5 * mantissa. */
double orc_e2m1_value(uint8_t code)
{
    int s = (code >> 3) & 1, e = (code >> 1) & 3, m = code & 1;
    double mag = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);
    return s ? -mag : mag;
}

/* E4M3 as in the OCP FP8 "E4M3FN" encoding: bias 7, no infinities,
 * S.1111.111 is NaN, largest finite 448, smallest subnormal 2^-9. */
double orc_e4m3_value(uint8_t b)
{
    int s = b >> 7, e = (b >> 3) & 15, m = b & 7;
    double mag;
    if (e == 15 && m == 7) return NAN;
    mag = (e == 0) ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
    return s ? -mag : mag;
}

/* E8M0: an exponent only, value 2^(b - 127); 0xFF is NaN. */
double orc_e8m0_value(uint8_t b)
{
    if (b == 0xFF) return NAN;
    return ldexp(1.0, (int)b - 127);
}

/* bfloat16 bit pattern -> value (exact). */
double orc_bf16_value(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round a double to bfloat16, nearest with ties to even, with gradual
 * underflow and overflow to infinity.  Written from the IEEE-754 definition:
 * find the two neighbouring bfloat16 values and pick the nearer one. */
uint16_t orc_bf16_from_double(double v)
{
    uint16_t sign;
    double a, q, lo, r;
    int ex;
    if (isnan(v)) return 0x7FC0;
    sign = signbit(v) ? 0x8000 : 0x0000;
    a = fabs(v);
    if (a == 0.0) return sign;
    /* bfloat16: 8 significant bits, exponent range of binary32.  The spacing
     * of representable values around a is 2^(max(floor(log2 a), -126) - 7). */
    frexp(a, &ex);               /* a = f * 2^ex, f in [0.5, 1) */
    ex -= 1;                     /* a in [2^ex, 2^(ex+1)) */
    if (ex < -126) ex = -126;
    q = ldexp(1.0, ex - 7);      /* spacing */
    lo = floor(a / q);           /* exact: a/q is a scaling by a power of two */
    r = a / q - lo;              /* exact */
    if (r > 0.5 || (r == 0.5 && fmod(lo, 2.0) != 0.0)) lo += 1.0;
    a = lo * q;
    if (a >= ldexp(1.0, 128)) return sign | 0x7F80;   /* overflow -> inf */
    {
        float f = (float)a;      /* exact: a has at most 8 significant bits */
        uint32_t u;
        memcpy(&u, &f, 4);
        return sign | (uint16_t)((u >> 16) & 0x7FFF);
    }
}

/* ---------- scale rules ---------- */

/* MXFP4 block scale, "ceil" reading: the smallest e in [-127, 127] with
 * amax <= 6 * 2^e.  Closed form: with amax = 1.f * 2^E, 6 * 2^(E-2) = 1.5 * 2^E,
 * so e = E - 2 when 1.f <= 1.5 and E - 1 otherwise.  Returns the E8M0 byte. */
uint8_t orc_mx_scale_byte(double amax)
{
    int ex, e;
    double f;
    if (isnan(amax) || isinf(amax)) return 0xFF;
    if (amax == 0.0) return 0x00;
    f = frexp(amax, &ex);        /* amax = f * 2^ex, f in [0.5,1); 1.f = 2f, E = ex-1 */
    e = (2.0 * f <= 1.5) ? (ex - 1) - 2 : (ex - 1) - 1;
    if (e < -127) e = -127;
    if (e > 127) e = 127;
    return (uint8_t)(e + 127);
}

/* NVFP4 computed global scale: g = 2^k with k the smallest integer >= -126
 * such that amax <= 6 * 448 * 2^k = 2688 * 2^k.  2688 = 1.3125 * 2^11, so with
 * amax = 1.f * 2^E, k = E - 11 when 1.f <= 1.3125, else E - 10.  A tensor with
 * no nonzero finite value gets g = 1. */
float orc_nv_global_scale(double amax)
{
    int ex, k;
    double f;
    if (!(amax > 0.0) || isinf(amax)) return 1.0f;
    f = frexp(amax, &ex);
    k = (2.0 * f <= 1.3125) ? (ex - 1) - 11 : (ex - 1) - 10;
    if (k < -126) k = -126;
    return (float)ldexp(1.0, k);
}

/* Ascending table of the 126 positive finite E4M3 values and their bytes. */
static double e4m3_pos_val[126];
static uint8_t e4m3_pos_byte[126];
static int e4m3_ready = 0;
static void e4m3_init(void)
{
    int n = 0, b;
    if (e4m3_ready) return;
    for (b = 0x01; b <= 0x7E; b++) {       /* positive bytes are monotone in value */
        e4m3_pos_val[n] = orc_e4m3_value((uint8_t)b);
        e4m3_pos_byte[n] = (uint8_t)b;
        n++;
    }
    e4m3_ready = 1;
}

/* NVFP4 block scale, "ceil" reading: the smallest positive finite E4M3 value
 * s with amax <= 6 * s * g.  amax == 0 gives byte 0x00.  When even s = 448 is
 * too small (only possible with a caller-chosen g), 448 is used and the
 * elements saturate.
 * Computed as the first E4M3 value >= q = amax / (6 g).  The FP64 quotient is
 * within 2^-53 (relative) of the true one, while the true quotient is either
 * exactly an E4M3 value v (then FP64 returns v exactly) or at least 2^-31 away
 * from every such v (amax has 8 significant bits and 6 v g at most 30), so the
 * search on the rounded quotient finds the same value as on the true one. */
uint8_t orc_nv_scale_byte(double amax, double g)
{
    int i;
    double q;
    if (isnan(amax) || isinf(amax)) return 0x7F;
    if (amax == 0.0) return 0x00;
    e4m3_init();
    q = amax / (6.0 * g);
    for (i = 0; i < 126 && e4m3_pos_val[i] < q; i++) {}
    if (i >= 126) return 0x7E;  /* above 448: saturate */
    return e4m3_pos_byte[i];
}

/* ---------- element rounding ---------- */

/* E2M1 magnitude code of |x| / S, round to nearest with ties to the even code,
 * saturating at 6.  Decided by exact comparisons of |x| with the midpoints
 * between neighbouring grid values times S (each product exact in FP64). */
static int e2m1_mag_code(double ax, double S)
{
    static const double mid[7] = {0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0};
    int i;
    for (i = 0; i < 7; i++) {
        double t = mid[i] * S;
        if (ax < t) return i;
        if (ax == t) return (i % 2 == 0) ? i : i + 1;   /* tie: the even code */
    }
    return 7;
}

/* Full E2M1 code (sign copied from x, also for magnitude 0). */
uint8_t orc_e2m1_encode(double x, double S)
{
    int m = (S > 0.0) ? e2m1_mag_code(fabs(x), S) : 0;
    return (uint8_t)((signbit(x) ? 8 : 0) | m);
}

/* ---------- tensor operations ---------- */

static int block_of(int fmt) { return fmt == ORC_FMT_MXFP4 ? 32 : 16; }

/* Largest finite |x| over a rows x cols bfloat16 matrix (row stride ldx). */
double orc_tensor_amax(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx)
{
    double m = 0.0;
    int64_t r, c;
    for (r = 0; r < rows; r++)
        for (c = 0; c < cols; c++) {
            double v = fabs(orc_bf16_value(x[r * ldx + c]));
            if (!isnan(v) && !isinf(v) && v > m) m = v;
        }
    return m;
}

/* Quantize a rows x cols bfloat16 matrix along its rows.
 *   codes : rows x cols/2 bytes, element 2i in bits 3:0 of byte i
 *   scales: rows x cols/B bytes (E8M0 for MXFP4, E4M3 for NVFP4)
 *   g     : NVFP4 global scale (ignored for MXFP4); the caller computes it
 *           with orc_nv_global_scale or chooses it.
 * Returns 0, or -1 when cols is not a multiple of the block size. */
int orc_quantize(int fmt, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                 uint8_t *codes, uint8_t *scales, double g)
{
    int B = block_of(fmt);
    int64_t r, b, j, nb;
    if (cols % B) return -1;
    nb = cols / B;
    for (r = 0; r < rows; r++) {
        for (b = 0; b < nb; b++) {
            const uint16_t *xb = x + r * ldx + b * B;
            double amax = 0.0, S;
            int bad = 0;
            uint8_t sb;
            for (j = 0; j < B; j++) {
                double v = orc_bf16_value(xb[j]);
                if (isnan(v) || isinf(v)) bad = 1;
                else if (fabs(v) > amax) amax = fabs(v);
            }
            if (bad) sb = (fmt == ORC_FMT_MXFP4) ? 0xFF : 0x7F;
            else sb = (fmt == ORC_FMT_MXFP4) ? orc_mx_scale_byte(amax) : orc_nv_scale_byte(amax, g);
            scales[r * nb + b] = sb;
            S = (fmt == ORC_FMT_MXFP4) ? orc_e8m0_value(sb) : orc_e4m3_value(sb) * g;
            for (j = 0; j < B; j++) {
                uint8_t c = bad ? 0 : orc_e2m1_encode(orc_bf16_value(xb[j]), S);
                int64_t k = b * B + j;
                uint8_t *p = &codes[r * (cols / 2) + k / 2];
                if (k % 2 == 0) *p = (uint8_t)((*p & 0xF0) | c);
                else *p = (uint8_t)((*p & 0x0F) | (c << 4));
            }
        }
    }
    return 0;
}

/* Dequantized value of element (r, k) from codes/scales/g. */
static double deq(int fmt, const uint8_t *codes, const uint8_t *scales, double g,
                  int64_t cols, int64_t r, int64_t k)
{
    int B = block_of(fmt);
    uint8_t byte = codes[r * (cols / 2) + k / 2];
    uint8_t c = (k % 2 == 0) ? (byte & 0xF) : (byte >> 4);
    uint8_t sb = scales[r * (cols / B) + k / B];
    double S = (fmt == ORC_FMT_MXFP4) ? orc_e8m0_value(sb) : orc_e4m3_value(sb) * g;
    return orc_e2m1_value(c) * S;
}

/* Dequantize to doubles (rows x cols, dense). */
void orc_dequantize(int fmt, const uint8_t *codes, const uint8_t *scales, double g,
                    int64_t rows, int64_t cols, double *out)
{
    int64_t r, k;
    for (r = 0; r < rows; r++)
        for (k = 0; k < cols; k++)
            out[r * cols + k] = deq(fmt, codes, scales, g, cols, r, k);
}

/* Fake-quant (the QAT forward's quantize-dequantize): quantize, then round
 * each dequantized value once to bfloat16.  y has row stride ldy. */
int orc_fakequant(int fmt, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                  uint16_t *y, int64_t ldy, double g, uint8_t *codes_tmp, uint8_t *scales_tmp)
{
    int64_t r, k;
    if (orc_quantize(fmt, x, rows, cols, ldx, codes_tmp, scales_tmp, g)) return -1;
    for (r = 0; r < rows; r++)
        for (k = 0; k < cols; k++)
            y[r * ldy + k] = orc_bf16_from_double(deq(fmt, codes_tmp, scales_tmp, g, cols, r, k));
    return 0;
}

/* Block-scaled FP4 x FP4 product, Y[m][n] = sum_k A^[m][k] * B^[n][k], with
 * A^, B^ the exact dequantized operands (global scales included), summed in
 * FP64 in k order.  rows [m0, m1) of Y only, so that a slice of a large
 * problem can be evaluated; y is (m1 - m0) x N, dense. */
void orc_gemm_rows(int fmt, int64_t M, int64_t N, int64_t K,
                   const uint8_t *a_codes, const uint8_t *a_scales, double ga,
                   const uint8_t *b_codes, const uint8_t *b_scales, double gb,
                   int64_t m0, int64_t m1, double *y)
{
    int64_t m, n, k;
    (void)M;
    for (m = m0; m < m1; m++)
        for (n = 0; n < N; n++) {
            double acc = 0.0;
            for (k = 0; k < K; k++)
                acc += deq(fmt, a_codes, a_scales, ga, K, m, k) *
                       deq(fmt, b_codes, b_scales, gb, K, n, k);
            y[(m - m0) * N + n] = acc;
        }
}

/* Same product for a list of (m, n) pairs (sampled checks at large sizes),
 * plus the sum of |products| for each pair (the scale of FP32 rounding). */
void orc_gemm_points(int fmt, int64_t K,
                     const uint8_t *a_codes, const uint8_t *a_scales, double ga,
                     const uint8_t *b_codes, const uint8_t *b_scales, double gb,
                     const int64_t *ms, const int64_t *ns, int64_t npts,
                     double *y, double *absy)
{
    int64_t p, k;
    for (p = 0; p < npts; p++) {
        double acc = 0.0, aacc = 0.0;
        for (k = 0; k < K; k++) {
            double t = deq(fmt, a_codes, a_scales, ga, K, ms[p], k) *
                       deq(fmt, b_codes, b_scales, gb, K, ns[p], k);
            acc += t;
            aacc += fabs(t);
        }
        y[p] = acc;
        absy[p] = aacc;
    }
}

/* ---------- array forms of the scalar rules (for exhaustive sweeps) ---------- */

void orc_e2m1_encode_array(const double *x, int64_t n, double S, uint8_t *out)
{
    int64_t i;
    for (i = 0; i < n; i++) out[i] = orc_e2m1_encode(x[i], S);
}

void orc_bf16_from_double_array(const double *v, int64_t n, uint16_t *out)
{
    int64_t i;
    for (i = 0; i < n; i++) out[i] = orc_bf16_from_double(v[i]);
}

/* ---------- block rotation before MXFP4 quantization ---------- */

/* MXFP4 activations in ReQAT are rotated block by block before quantization
 * (Sec. 4.3, "Additional implementation details"; App. C.2, "Challenges in
 * MXFP4 activation quantization"): a randomized Hadamard transform over each
 * 32-element block.  The paper fixes neither the normalization nor the sign
 * vector; the readings used here:
 *   - y = (1/sqrt(32)) * H_32 * D * x per block, H_32 the Sylvester Hadamard
 *     matrix (H[i][j] = (-1)^popcount(i & j)), D = diag(d) with d_j = -1 where
 *     bit j of the 32-bit `signs` word is set (the random draw is an input);
 *     the map is orthonormal, so rotating both operands of a product leaves
 *     the product unchanged;
 *   - y is the exact real value, and it is quantized exactly as a block of
 *     MXFP4 values: e the smallest integer in [-127, 127] with
 *     max_i |y_i| <= 6 * 2^e (127 if none; byte 0x00 for an all-zero y),
 *     then each code the nearest E2M1 value to |y_i| / 2^e (saturating at 6)
 *     with the sign of y_i (y_i == 0 gives code 0);
 *   - a block with a NaN or Inf input gets scale 0xFF and zero codes.
 * No rounding tie can occur: with s_i = sqrt(32) * y_i a dyadic rational,
 * |y_i| = t * 2^e would make sqrt(32) = |s_i| / (t * 2^e) rational.
 *
 * Every decision is made in exact integer arithmetic.  A bfloat16 value is
 * m * 2^u with an integer m < 256 and u >= -133, so S_i = s_i * 2^133 is an
 * integer below 2^266, accumulated here as a multi-word unsigned integer
 * (separate sums of the positive and the negative terms).  Then
 *     |y_i| <= 6 * 2^e          <=>  S_i^2 <= 1152 * 2^(2e + 266)
 *     |y_i| >  (k/4) * 2^e      <=>  S_i^2 >  2 k^2 * 2^(2e + 266)
 * (y_i = S_i * 2^-133 / sqrt(32), sqrt(32) = 4 sqrt(2)), and the E2M1
 * midpoints 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5 are k/4 for
 * k = 1, 3, 5, 7, 10, 14, 20. */

#define BIG_WORDS 20            /* 640 bits: S < 2^266, S^2 and the bounds < 2^532 */

typedef struct { uint32_t w[BIG_WORDS]; } big_t;

static void big_zero(big_t *a) { memset(a->w, 0, sizeof(a->w)); }

/* a += m * 2^sh (m < 2^32) */
static void big_add_shifted(big_t *a, uint32_t m, int sh)
{
    uint64_t carry = 0, add;
    int i, q = sh / 32, r = sh % 32;
    uint64_t t = (uint64_t)m << r;                     /* < 2^63 */
    for (i = q; i < BIG_WORDS; i++) {
        add = (i == q) ? (t & 0xFFFFFFFFu) : (i == q + 1) ? (t >> 32) : 0;
        carry += (uint64_t)a->w[i] + add;
        a->w[i] = (uint32_t)carry;
        carry >>= 32;
    }
}

static int big_cmp(const big_t *a, const big_t *b)
{
    int i;
    for (i = BIG_WORDS - 1; i >= 0; i--)
        if (a->w[i] != b->w[i]) return a->w[i] < b->w[i] ? -1 : 1;
    return 0;
}

/* out = a - b, a >= b */
static void big_sub(const big_t *a, const big_t *b, big_t *out)
{
    int64_t borrow = 0, d;
    int i;
    for (i = 0; i < BIG_WORDS; i++) {
        d = (int64_t)a->w[i] - (int64_t)b->w[i] - borrow;
        borrow = d < 0;
        out->w[i] = (uint32_t)(d + (borrow ? ((int64_t)1 << 32) : 0));
    }
}

/* out = a * a (a < 2^320) */
static void big_square(const big_t *a, big_t *out)
{
    int i, j;
    big_zero(out);
    for (i = 0; i < BIG_WORDS / 2; i++) {
        uint64_t carry = 0;
        for (j = 0; j < BIG_WORDS / 2; j++) {
            uint64_t cur = (uint64_t)a->w[i] * a->w[j] + out->w[i + j] + carry;
            out->w[i + j] = (uint32_t)cur;
            carry = cur >> 32;
        }
        for (j = i + BIG_WORDS / 2; carry && j < BIG_WORDS; j++) {
            uint64_t cur = (uint64_t)out->w[j] + carry;
            out->w[j] = (uint32_t)cur;
            carry = cur >> 32;
        }
    }
}

/* c * 2^sh for a small constant c */
static big_t big_const(uint32_t c, int sh)
{
    big_t b;
    big_zero(&b);
    big_add_shifted(&b, c, sh);
    return b;
}

/* bfloat16 h (finite) as sign and m * 2^(u + 133): returns the shift u + 133. */
static int bf16_int_parts(uint16_t h, int *neg, uint32_t *m)
{
    int e = (h >> 7) & 0xFF;
    *neg = (h >> 15) & 1;
    if (e == 0) {                                     /* subnormal: frac * 2^-133 */
        *m = h & 0x7F;
        return 0;
    }
    *m = 0x80 | (h & 0x7F);                           /* (128 + frac) * 2^(e - 134) */
    return e - 1;
}

/* E8M0 byte and the 32 codes of the rotated block of x (exact).  Returns 0, or
 * 1 for a block with a NaN or Inf input (byte 0xFF, codes 0). */
static int rht_block_exact(const uint16_t *x, uint32_t signs, uint8_t *sbyte, uint8_t *codes)
{
    static const uint32_t mid_k[7] = {1, 3, 5, 7, 10, 14, 20};
    big_t pos[32], neg[32], mag[32], sq, amax2, bound, zero;
    int negative[32];
    int i, j, e;
    for (j = 0; j < 32; j++)
        if (((x[j] >> 7) & 0xFF) == 0xFF) {
            *sbyte = 0xFF;
            memset(codes, 0, 32);
            return 1;
        }
    for (i = 0; i < 32; i++) {
        big_zero(&pos[i]);
        big_zero(&neg[i]);
    }
    for (j = 0; j < 32; j++) {
        int xneg, sh;
        uint32_t m;
        sh = bf16_int_parts(x[j], &xneg, &m);
        if (m == 0) continue;
        if ((signs >> j) & 1u) xneg = !xneg;             /* d_j = -1 */
        for (i = 0; i < 32; i++) {
            int hneg = __builtin_popcount((unsigned)(i & j)) & 1;   /* H[i][j] = -1 */
            if (hneg ^ xneg) big_add_shifted(&neg[i], m, sh);
            else big_add_shifted(&pos[i], m, sh);
        }
    }
    big_zero(&amax2);
    big_zero(&zero);
    for (i = 0; i < 32; i++) {
        int c = big_cmp(&pos[i], &neg[i]);
        negative[i] = c < 0;
        if (c >= 0) big_sub(&pos[i], &neg[i], &mag[i]);
        else big_sub(&neg[i], &pos[i], &mag[i]);
        big_square(&mag[i], &sq);
        if (big_cmp(&sq, &amax2) > 0) amax2 = sq;
    }
    memset(codes, 0, 32);
    if (big_cmp(&amax2, &zero) == 0) {                 /* y == 0 */
        *sbyte = 0;
        return 0;
    }
    for (e = -127; e < 127; e++) {                      /* smallest e with max|y| <= 6 * 2^e */
        bound = big_const(1152, 2 * e + 266);
        if (big_cmp(&amax2, &bound) <= 0) break;
    }
    *sbyte = (uint8_t)(e + 127);
    for (i = 0; i < 32; i++) {
        int k, m3 = 0;
        big_square(&mag[i], &sq);
        for (k = 0; k < 7; k++) {
            bound = big_const(2 * mid_k[k] * mid_k[k], 2 * e + 266);
            if (big_cmp(&sq, &bound) > 0) m3 = k + 1;
        }
        codes[i] = (uint8_t)(m3 | (negative[i] ? 8 : 0));     /* negative: S_i < 0, so y_i != 0 */
    }
    return 0;
}

/* MXFP4 quantization of the rotated blocks of a rows x cols bfloat16 matrix
 * (cols % 32 == 0): codes rows x cols/2, scales rows x cols/32.  With fake != 0
 * it writes instead y_out (row stride ldy): each dequantized rotated value
 * code * 2^e in bfloat16, exact (NaN for a non-finite block). */
static int quantize_mx_rht(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                           uint32_t signs, uint8_t *codes, uint8_t *scales,
                           uint16_t *y_out, int64_t ldy, int fake)
{
    int64_t r, b, nb;
    int j;
    if (cols % 32) return -1;
    nb = cols / 32;
    for (r = 0; r < rows; r++) {
        for (b = 0; b < nb; b++) {
            uint8_t sb, cs[32];
            int bad = rht_block_exact(x + r * ldx + b * 32, signs, &sb, cs);
            double S = orc_e8m0_value(sb);
            if (!fake) scales[r * nb + b] = sb;
            for (j = 0; j < 32; j++) {
                int64_t k = b * 32 + j;
                if (fake) {
                    y_out[r * ldy + k] = bad ? 0x7FC0 : orc_bf16_from_double(orc_e2m1_value(cs[j]) * S);
                } else {
                    uint8_t *p = &codes[r * (cols / 2) + k / 2];
                    if (k % 2 == 0) *p = (uint8_t)((*p & 0xF0) | cs[j]);
                    else *p = (uint8_t)((*p & 0x0F) | (cs[j] << 4));
                }
            }
        }
    }
    return 0;
}

int orc_quantize_mx_rht(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, uint32_t signs,
                        uint8_t *codes, uint8_t *scales)
{
    return quantize_mx_rht(x, rows, cols, ldx, signs, codes, scales, 0, 0, 0);
}

int orc_fakequant_mx_rht(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, uint32_t signs,
                         uint16_t *y, int64_t ldy)
{
    return quantize_mx_rht(x, rows, cols, ldx, signs, 0, 0, y, ldy, 1);
}

/* ---------- W4A16: MXFP4 weights, bfloat16 activations ---------- */

/* The MXFP4 W4A16 deployment setting (Sec. 2, "Microscaled FP4 formats";
 * Sec. 5.1; App. D.1): weights stored as MXFP4, activations bfloat16.
 * Readings: the weight is dequantized to the activation type,
 *     w^[n][k] = RN_bf16(E2M1(c) * 2^e)
 * (exact for E8M0 bytes 2..252; the bfloat16 rounding, overflow to Inf
 * included, otherwise; NaN for byte 0xFF), and
 *     Y[m][n] = sum_k x[m][k] * w^[n][k]
 * is evaluated here in FP64 in k order (every product is exact in FP64).
 * For each requested (m, n) pair it also returns sum_k |x w^|, the scale of
 * FP32 accumulation error. */
static double w4a16_weight(const uint8_t *w_codes, const uint8_t *w_scales, int64_t K, int64_t n, int64_t k)
{
    uint8_t byte = w_codes[n * (K / 2) + k / 2];
    uint8_t c = (k % 2 == 0) ? (byte & 0xF) : (byte >> 4);
    double v = orc_e2m1_value(c) * orc_e8m0_value(w_scales[n * (K / 32) + k / 32]);
    return orc_bf16_value(orc_bf16_from_double(v));
}

void orc_gemm_w4a16_points(int64_t K, const uint16_t *x, int64_t ldx, const uint8_t *w_codes,
                           const uint8_t *w_scales, const int64_t *ms, const int64_t *ns, int64_t npts,
                           double *y, double *absy)
{
    int64_t p, k;
    for (p = 0; p < npts; p++) {
        double acc = 0.0, aacc = 0.0;
        for (k = 0; k < K; k++) {
            double t = orc_bf16_value(x[ms[p] * ldx + k]) * w4a16_weight(w_codes, w_scales, K, ns[p], k);
            acc += t;
            aacc += fabs(t);
        }
        y[p] = acc;
        absy[p] = aacc;
    }
}

/* ---------- KV4: E1M2 elements with NVFP4-style scaling and the post-RoPE shift ---------- */

/* The KV cache of the NVFP4 W4A4KV4 setting is stored in 4 bits with the E1M2
 * element format (Sec. 4.3, "Additional implementation details"), and the
 * keys are shifted channel-wise after RoPE before quantization (Q-FIT,
 * Sec. 4.3, Eq. for K~: K~ = R(K_pre / s) - m; the pre-RoPE scale s is folded
 * into the projection weights, so the cache quantizer sees R(...) and m).
 * Readings:
 *   - E1M2: sign, 1 exponent bit (bias 0), 2 mantissa bits: magnitudes
 *     0, 0.5, 1, ..., 3.5 (code magnitude i is i / 2);
 *   - scaling as NVFP4: blocks of 16 along the channel dimension, an E4M3
 *     block scale (the smallest positive E4M3 value s with
 *     block_amax <= 3.5 * s * g) and an FP32 global scale g, computed as the
 *     smallest power of two 2^k (k >= -126) with tensor_amax <= 3.5 * 448 * 2^k
 *     (g = 1 for a tensor without non-zero finite values) or given;
 *   - the shifted value d = x - m[c] is rounded once to FP32 (m is FP32; no
 *     shift = all zeros), and d is what is quantized; a block with a
 *     non-finite d gets scale 0x7F and zero codes;
 *   - elements round to nearest, ties to the even magnitude code, saturating
 *     at 3.5; the sign is copied.
 * All comparisons are exact in FP64 (d has 24 significant bits, 3.5 * s * g
 * and the midpoints times s * g at most 3 + 4 + 24). */

double orc_e1m2_value(uint8_t code)
{
    double v = 0.5 * (double)(code & 7);
    return (code & 8) ? -v : v;
}

/* E1M2 code of v / S (S > 0): nearest of i / 2, ties to even i, saturating. */
uint8_t orc_e1m2_encode(double v, double S)
{
    double a = fabs(v);
    int i, m = 7;
    for (i = 0; i < 7; i++) {
        double t = (0.5 * i + 0.25) * S;       /* midpoint between i/2 and (i+1)/2 */
        if (a < t) { m = i; break; }
        if (a == t) { m = (i % 2 == 0) ? i : i + 1; break; }
    }
    return (uint8_t)((signbit(v) ? 8 : 0) | m);
}

/* Global scale: smallest 2^k, k >= -126, with amax <= 1568 * 2^k
 * (1568 = 3.5 * 448 = 1.53125 * 2^10), by exact search. */
float orc_kv4_global_scale(double amax)
{
    int k;
    if (!(amax > 0.0) || isinf(amax)) return 1.0f;
    for (k = -126; k < 128; k++)
        if (amax <= 1568.0 * ldexp(1.0, k)) break;
    return (float)ldexp(1.0, k);
}

/* Block scale: the smallest positive finite E4M3 value s with amax <= 3.5 s g
 * (exact product comparison); 448 when none is large enough; 0 for amax 0. */
uint8_t orc_kv4_scale_byte(double amax, double g)
{
    int i;
    if (isnan(amax) || isinf(amax)) return 0x7F;
    if (amax == 0.0) return 0x00;
    e4m3_init();
    for (i = 0; i < 126; i++)
        if (amax <= 3.5 * e4m3_pos_val[i] * g) return e4m3_pos_byte[i];
    return 0x7E;
}

/* d[r][c] = RN_fp32(x - m[c]) for a rows x cols bfloat16 matrix. */
static float kv4_shifted(const uint16_t *x, int64_t ldx, const float *shift, int64_t r, int64_t c)
{
    float v = (float)orc_bf16_value(x[r * ldx + c]);
    return shift ? v - shift[c] : v;
}

double orc_kv4_amax(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift)
{
    double m = 0.0;
    int64_t r, c;
    for (r = 0; r < rows; r++)
        for (c = 0; c < cols; c++) {
            double v = fabs((double)kv4_shifted(x, ldx, shift, r, c));
            if (!isnan(v) && !isinf(v) && v > m) m = v;
        }
    return m;
}

/* Quantize (codes rows x cols/2, scales rows x cols/16) or, with y != 0,
 * fake-quantize (y[r][c] = RN_bf16(E1M2(code) * s * g), in the shifted
 * domain; NaN for a non-finite block) the shifted rows.  g as given. */
int orc_kv4_quantize(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                     double g, uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy)
{
    int64_t r, b, nb;
    int j;
    if (cols % 16) return -1;
    nb = cols / 16;
    for (r = 0; r < rows; r++) {
        for (b = 0; b < nb; b++) {
            float d[16];
            double amax = 0.0, S;
            int bad = 0;
            uint8_t sb;
            for (j = 0; j < 16; j++) {
                d[j] = kv4_shifted(x, ldx, shift, r, b * 16 + j);
                if (isnan(d[j]) || isinf(d[j])) bad = 1;
                else if (fabs((double)d[j]) > amax) amax = fabs((double)d[j]);
            }
            sb = bad ? 0x7F : orc_kv4_scale_byte(amax, g);
            S = orc_e4m3_value(sb) * g;
            if (scales) scales[r * nb + b] = sb;
            for (j = 0; j < 16; j++) {
                uint8_t c = (bad || sb == 0) ? (uint8_t)(bad ? 0 : (signbit(d[j]) ? 8 : 0))
                                            : orc_e1m2_encode((double)d[j], S);
                int64_t k = b * 16 + j;
                if (y) {
                    y[r * ldy + k] = bad ? 0x7FC0 : orc_bf16_from_double(orc_e1m2_value(c) * (sb ? S : 0.0));
                } else {
                    uint8_t *p = &codes[r * (cols / 2) + k / 2];
                    if (k % 2 == 0) *p = (uint8_t)((*p & 0xF0) | c);
                    else *p = (uint8_t)((*p & 0x0F) | (c << 4));
                }
            }
        }
    }
    return 0;
}
