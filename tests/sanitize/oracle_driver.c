/* Sanitizer driver for the CPU oracle (test infrastructure): calls every
 * oracle entry point on small seeded inputs, specials included (zeros, -0,
 * subnormals, bfloat16 maxima, NaN, Inf, strided rows), so that an
 * AddressSanitizer / UndefinedBehaviorSanitizer build reports any
 * out-of-bounds access, overflow or undefined shift in them.  Built and run
 * by tests/test_sanitizers.py together with reqat_oracle.c. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double orc_e2m1_value(uint8_t);
double orc_e4m3_value(uint8_t);
double orc_e8m0_value(uint8_t);
double orc_bf16_value(uint16_t);
uint16_t orc_bf16_from_double(double);
uint8_t orc_mx_scale_byte(double);
float orc_nv_global_scale(double);
uint8_t orc_nv_scale_byte(double, double);
uint8_t orc_e2m1_encode(double, double);
double orc_tensor_amax(const uint16_t *, int64_t, int64_t, int64_t);
int orc_quantize(int, const uint16_t *, int64_t, int64_t, int64_t, uint8_t *, uint8_t *, double);
void orc_dequantize(int, const uint8_t *, const uint8_t *, double, int64_t, int64_t, double *);
int orc_fakequant(int, const uint16_t *, int64_t, int64_t, int64_t, uint16_t *, int64_t, double, uint8_t *,
                  uint8_t *);
void orc_gemm_rows(int, int64_t, int64_t, int64_t, const uint8_t *, const uint8_t *, double, const uint8_t *,
                   const uint8_t *, double, int64_t, int64_t, double *);
void orc_gemm_points(int, int64_t, const uint8_t *, const uint8_t *, double, const uint8_t *, const uint8_t *,
                     double, const int64_t *, const int64_t *, int64_t, double *, double *);
int orc_quantize_mx_rht(const uint16_t *, int64_t, int64_t, int64_t, uint32_t, uint8_t *, uint8_t *);
int orc_fakequant_mx_rht(const uint16_t *, int64_t, int64_t, int64_t, uint32_t, uint16_t *, int64_t);
void orc_gemm_w4a16_points(int64_t, const uint16_t *, int64_t, const uint8_t *, const uint8_t *, const int64_t *,
                           const int64_t *, int64_t, double *, double *);
double orc_e1m2_value(uint8_t);
uint8_t orc_e1m2_encode(double, double);
float orc_kv4_global_scale(double);
uint8_t orc_kv4_scale_byte(double, double);
double orc_kv4_amax(const uint16_t *, int64_t, int64_t, int64_t, const float *);
int orc_kv4_quantize(const uint16_t *, int64_t, int64_t, int64_t, const float *, double, uint8_t *, uint8_t *,
                     uint16_t *, int64_t);

static uint32_t state = 2463534242u;
static uint32_t rnd(void)
{
    state ^= state << 13;
    state ^= state >> 17;
    state ^= state << 5;
    return state;
}

int main(void)
{
    enum { R = 9, C = 128, LD = 136, M = 5, N = 7 };
    uint16_t *x = malloc(sizeof(uint16_t) * R * LD), *w = malloc(sizeof(uint16_t) * N * C);
    uint16_t *y = malloc(sizeof(uint16_t) * R * LD);
    uint8_t *codes = malloc(R * C / 2), *scales = malloc(R * C / 16);
    uint8_t *wc = malloc(N * C / 2), *ws = malloc(N * C / 16);
    double *deq = malloc(sizeof(double) * R * C), *yg = malloc(sizeof(double) * M * N);
    double *pts = malloc(sizeof(double) * 64), *apts = malloc(sizeof(double) * 64);
    int64_t ms[16], ns[16];
    float shift[C];
    int i, fmt, r, c;
    double acc = 0.0;
    for (i = 0; i < 256; i++) acc += orc_e2m1_value((uint8_t)(i & 15)) + orc_e1m2_value((uint8_t)(i & 15)) +
                                     (orc_e4m3_value((uint8_t)i) == orc_e4m3_value((uint8_t)i)) +
                                     (orc_e8m0_value((uint8_t)i) > 0);
    for (i = 0; i < 65536; i += 7) {
        double v = orc_bf16_value((uint16_t)i);
        acc += orc_bf16_from_double(v) + orc_mx_scale_byte(v < 0 ? -v : v) + orc_nv_global_scale(v < 0 ? -v : v) +
               orc_nv_scale_byte(v < 0 ? -v : v, 0.5) + orc_e2m1_encode(v, 1.0) + orc_e1m2_encode(v, 0.25) +
               orc_kv4_global_scale(v < 0 ? -v : v) + orc_kv4_scale_byte(v < 0 ? -v : v, 2.0);
    }
    for (i = 0; i < R * LD; i++) x[i] = (uint16_t)rnd();
    for (c = 0; c < C; c++) {                 /* finite rows 0..4, specials in rows 5..8 */
        for (r = 0; r < 5; r++) x[r * LD + c] = (uint16_t)((rnd() & 0x807F) | ((100 + rnd() % 50) << 7));
        x[5 * LD + c] = (uint16_t)(c % 3 ? 0x8000 : 0x0001);
        x[6 * LD + c] = (uint16_t)(c % 2 ? 0x7F7F : 0x0080);
        shift[c] = (float)(c % 5) - 2.0f;
    }
    x[7 * LD + 3] = 0x7FC0;
    x[8 * LD + 40] = 0xFF80;
    for (i = 0; i < N * C; i++) w[i] = (uint16_t)((rnd() & 0x807F) | ((110 + rnd() % 20) << 7));
    for (fmt = 0; fmt < 2; fmt++) {
        int B = fmt ? 32 : 16;
        double g = fmt ? 1.0 : orc_nv_global_scale(orc_tensor_amax(x, R, C, LD));
        if (orc_quantize(fmt, x, R, C, LD, codes, scales, g)) return 1;
        orc_dequantize(fmt, codes, scales, g, R, C, deq);
        if (orc_fakequant(fmt, x, R, C, LD, y, LD, g, codes, scales)) return 1;
        if (orc_quantize(fmt, w, N, C, C, wc, ws, 0.0123)) return 1;
        orc_gemm_rows(fmt, M, N, C, codes, scales, g, wc, ws, 0.0123, 0, M, yg);
        for (i = 0; i < 16; i++) {
            ms[i] = i % R;
            ns[i] = (i * 5) % N;
        }
        orc_gemm_points(fmt, C, codes, scales, g, wc, ws, 0.0123, ms, ns, 16, pts, apts);
        (void)B;
    }
    if (orc_quantize_mx_rht(x, R, C, LD, 0x9E3779B9u, codes, scales)) return 1;
    if (orc_fakequant_mx_rht(x, R, C, LD, 0x9E3779B9u, y, LD)) return 1;
    if (orc_quantize(1, w, N, C, C, wc, ws, 1.0)) return 1;
    orc_gemm_w4a16_points(C, x, LD, wc, ws, ms, ns, 16, pts, apts);
    acc += orc_kv4_amax(x, R, C, LD, shift);
    if (orc_kv4_quantize(x, R, C, LD, shift, 0.75, codes, scales, 0, 0)) return 1;
    if (orc_kv4_quantize(x, R, C, LD, 0, 2.0, codes, scales, y, LD)) return 1;
    printf("oracle driver ok %d\n", (int)(acc != 12345.678));
    free(x); free(w); free(y); free(codes); free(scales); free(wc); free(ws);
    free(deq); free(yg); free(pts); free(apts);
    return 0;
}
