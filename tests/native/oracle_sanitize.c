/*
 * Driver for a sanitizer build (AddressSanitizer + UndefinedBehaviorSanitizer)
 * of the CPU oracle: every exported function on small inputs that cover the
 * special cases (all-zero, constant, one-signed, subnormal-range and
 * largest-magnitude groups, W3 and W4, several rows and groups), with the
 * round trips checked.  Any sanitizer report aborts the run; a failed check
 * returns 1.  Prints "ok" on success.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

float laqo_f16_to_f32(uint16_t h);
uint16_t laqo_f32_to_f16(float v);
void laqo_quantize(const uint16_t *w, int64_t N, int64_t K, int bits, uint8_t *codes, uint16_t *scales,
                   uint8_t *zeros);
void laqo_codes_from_params(const uint16_t *w, int64_t N, int64_t K, int bits, const uint16_t *scales,
                            const uint8_t *zeros, uint8_t *codes);
int laqo_pack(const uint8_t *codes, int64_t N, int64_t K, int bits, uint32_t *qweight);
void laqo_unpack(const uint32_t *qweight, int64_t N, int64_t K, int bits, uint8_t *codes);
void laqo_dequant(const uint8_t *codes, const uint16_t *scales, const uint8_t *zeros, int64_t N, int64_t K,
                  double *w_hat);
void laqo_linear(const uint16_t *x, int64_t M, const uint8_t *codes, const uint16_t *scales,
                 const uint8_t *zeros, int64_t N, int64_t K, double *y);
void laqo_f16_to_f32_array(const uint16_t *h, int64_t n, float *out);
void laqo_f32_to_f16_array(const float *v, int64_t n, uint16_t *out);
int laqo_num_threads(void);

static uint32_t lcg_state = 12345u;
static uint32_t lcg(void)
{
    lcg_state = lcg_state * 1664525u + 1013904223u;
    return lcg_state >> 8;
}

/* a finite fp16 bit pattern of magnitude below 2^e (e <= 16) */
static uint16_t rand_half(int e)
{
    uint16_t h;
    do {
        h = (uint16_t)(lcg() & 0xffff);
    } while (((h >> 10) & 0x1f) == 0x1f || ((h >> 10) & 0x1f) >= 15 + e);
    return h;
}

static int check_case(int bits, int64_t N, int64_t K, const uint16_t *w)
{
    const int64_t G = K / 128;
    const int qmax = (1 << bits) - 1;
    uint8_t *codes = malloc((size_t)(N * K));
    uint8_t *codes2 = malloc((size_t)(N * K));
    uint16_t *scales = malloc((size_t)(N * G) * 2);
    uint8_t *zeros = malloc((size_t)(N * G));
    uint32_t *qw = malloc((size_t)(N * bits * (K / 32)) * 4);
    double *w_hat = malloc((size_t)(N * K) * 8);
    uint16_t *x = malloc((size_t)(3 * K) * 2);
    double *y = malloc((size_t)(3 * N) * 8);
    int bad = 0;
    laqo_quantize(w, N, K, bits, codes, scales, zeros);
    for (int64_t i = 0; i < N * K; ++i)
        bad |= codes[i] > qmax;
    for (int64_t i = 0; i < N * G; ++i)
        bad |= zeros[i] > qmax || scales[i] == 0 || (scales[i] & 0x8000);
    bad |= laqo_pack(codes, N, K, bits, qw) != 0;
    laqo_unpack(qw, N, K, bits, codes2);
    bad |= memcmp(codes, codes2, (size_t)(N * K)) != 0;
    laqo_codes_from_params(w, N, K, bits, scales, zeros, codes2);
    bad |= memcmp(codes, codes2, (size_t)(N * K)) != 0;
    laqo_dequant(codes, scales, zeros, N, K, w_hat);
    for (int64_t i = 0; i < 3 * K; ++i)
        x[i] = rand_half(2);
    laqo_linear(x, 3, codes, scales, zeros, N, K, y);
    for (int64_t n = 0; n < N; ++n) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k)
            acc += (double)laqo_f16_to_f32(x[2 * K + k]) * w_hat[n * K + k];
        double d = acc - y[2 * N + n];
        bad |= !(d < 1e-6 && d > -1e-6);
    }
    free(codes); free(codes2); free(scales); free(zeros); free(qw); free(w_hat); free(x); free(y);
    return bad;
}

int main(void)
{
    int bad = 0;
    /* every binary16 pattern: to float and back (NaNs map to the canonical NaN) */
    static uint16_t all[65536];
    static float f[65536];
    static uint16_t back[65536];
    for (int i = 0; i < 65536; ++i)
        all[i] = (uint16_t)i;
    laqo_f16_to_f32_array(all, 65536, f);
    laqo_f32_to_f16_array(f, 65536, back);
    for (int i = 0; i < 65536; ++i) {
        int nan = ((i >> 10) & 0x1f) == 0x1f && (i & 0x3ff);
        bad |= nan ? back[i] != 0x7e00 : back[i] != all[i];
    }
    bad |= laqo_f32_to_f16(1e9f) != 0x7c00 || laqo_f32_to_f16(-1e-30f) != 0x8000;

    const int64_t N = 7, K = 384;
    uint16_t *w = malloc((size_t)(N * K) * 2);
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k) {
            uint16_t h;
            switch (n) {
            case 0: h = 0; break;                                   /* all zero */
            case 1: h = 0x3c00; break;                              /* constant 1.0 */
            case 2: h = (uint16_t)(rand_half(0) | 0x8000); break;   /* one-signed, negative */
            case 3: h = (uint16_t)(lcg() & 0x83ff); break;          /* subnormals */
            case 4: h = (k % 2) ? 0x7bff : 0xfbff; break;           /* +-65504 */
            default: h = rand_half(-5 + (int)(k % 4)); break;
            }
            w[n * K + k] = h;
        }
    for (int bits = 3; bits <= 4; ++bits)
        bad |= check_case(bits, N, K, w);
    free(w);
    bad |= laqo_num_threads() < 1;
    if (bad) {
        printf("mismatch\n");
        return 1;
    }
    printf("ok\n");
    return 0;
}
