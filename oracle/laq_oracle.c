/*
 * laq_oracle.c -- plain CPU oracle for the W3G128 / W4G128 weight-only
 * quantized linear of LAQuant (arXiv 2605.08755).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the independent correctness
 * reference that the HIP library is checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark may load it.  It
 * shares no code, header, table or helper with the HIP library: every
 * formula below is written out again from the paper and from the packed
 * format definition, deliberately slowly and in the most literal order.
 *
 * What it computes
 * ----------------
 *  - Quantization, Eq. 1 of the paper (Sec. 2, "LLM Weight Quantization"):
 *        q = clip(round(w / s) + z, 0, 2^b - 1),   w_hat = s * (q - z),
 *    with scales and zeros shared by each run of g = 128 consecutive
 *    elements of a weight row (notation WbGg, here W3G128 and W4G128).
 *    The paper learns s and z by QAT; this library computes them by
 *    round-to-nearest min-max over the group, with the range widened to
 *    contain 0 (lo <= 0 <= hi).  Arithmetic: IEEE fp32, round-half-to-even,
 *    true division, the scale rounded to fp16 before it is used.  The codes
 *    of Eq. 1 for caller-supplied (e.g. trained) s and z are computed too.
 *  - Packing: 32 three-bit codes in three 32-bit words (App. H keeps this
 *    density of the GPTQ INT3 kernel), in this library's bit order; 4-bit
 *    codes eight per word.  The bit positions are computed here from the
 *    written definition, one code at a time.
 *  - The linear: y[m][n] = sum_k x[m][k] * w_hat[n][k], accumulated in fp64.
 *    Each term s*(q-z)*x is exact in fp64, so the result is the exact real
 *    value up to fp64 summation rounding (relative error ~1e-16).
 *
 * Build: gcc -O2 -std=c11 -fno-fast-math -ffp-contract=off -fopenmp -shared
 *        -fPIC -o liblaq_oracle.so laq_oracle.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define GROUP 128

/* ---------------------------------------------------------------------
 * IEEE 754 binary16 <-> binary32, written from the format definition:
 * 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits; exponent field
 * 0 encodes zero/subnormals (value = frac * 2^-24), field 31 inf/NaN.
 * ------------------------------------------------------------------- */
float laqo_f16_to_f32(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    float v;
    if (e == 0)
        v = ldexpf((float)f, -24);
    else if (e == 31)
        v = (f == 0) ? INFINITY : NAN;
    else
        v = ldexpf((float)(1024 + f), e - 25);
    return sign ? -v : v;
}

/* Round-to-nearest-even conversion of a float to binary16. */
uint16_t laqo_f32_to_f16(float v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    float a = fabsf(v);
    if (isnan(v))
        return 0x7e00;
    /* 65504 is the largest finite half; halfway to the next power of two
     * (65520) rounds to even, i.e. up to infinity. */
    if (a >= 65520.0f)
        return sign | 0x7c00;
    if (a == 0.0f)
        return sign;
    int ex;
    frexpf(a, &ex);            /* a = m * 2^ex, 0.5 <= m < 1 */
    int e = ex - 1;            /* a in [2^e, 2^(e+1)) */
    if (e < -14)
        e = -14;               /* subnormal range shares the quantum 2^-24 */
    /* quantum = 2^(e-10); n = a / quantum is exact (power-of-two scale) */
    float n = ldexpf(a, 10 - e);
    float r = rintf(n);        /* default rounding mode: ties to even */
    uint32_t ri = (uint32_t)r; /* 0 .. 2048 */
    if (ri >= 2048) {          /* rounded up into the next binade */
        ri = 1024;
        e += 1;
    }
    if (ri < 1024)             /* subnormal (only possible when e == -14) */
        return sign | (uint16_t)ri;
    return sign | (uint16_t)(((e + 15) << 10) | (ri - 1024));
}

/* ---------------------------------------------------------------------
 * Quantization (Eq. 1 with round-to-nearest min-max scales and zeros).
 *
 * For row n, group g (elements k = 128g .. 128g+127 of the row):
 *   1. lo = min(0, min_k w_k), hi = max(0, max_k w_k)       (exact)
 *   2. s32 = fl32( fl32(hi - lo) / (2^b - 1) )
 *   3. s16 = fp16_rne(s32); if s16 == +0 then s16 = 2^-24; s = float(s16)
 *   4. z = clamp(rint(fl32(-lo / s)), 0, 2^b - 1)
 *   5. q_k = clamp(rint(fl32(w_k / s)) + z, 0, 2^b - 1)
 * codes: uint8 [N][K] (one code per byte, unpacked)
 * scales: fp16 bits [N][K/128]; zeros: uint8 [N][K/128]
 * ------------------------------------------------------------------- */
void laqo_quantize(const uint16_t *w, int64_t N, int64_t K, int bits,
                   uint8_t *codes, uint16_t *scales, uint8_t *zeros)
{
    const int64_t G = K / GROUP;
    const int qmax = (1 << bits) - 1;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t g = 0; g < G; ++g) {
            const uint16_t *wg = w + n * K + g * GROUP;
            float lo = 0.0f, hi = 0.0f;
            for (int i = 0; i < GROUP; ++i) {
                float v = laqo_f16_to_f32(wg[i]);
                if (v < lo) lo = v;
                if (v > hi) hi = v;
            }
            float range = hi - lo;
            float s32 = range / (float)qmax;
            uint16_t s16 = laqo_f32_to_f16(s32);
            if (s16 == 0)
                s16 = 0x0001;  /* smallest subnormal, 2^-24 */
            float s = laqo_f16_to_f32(s16);
            float zf = rintf(-lo / s);
            int z = (int)zf;
            if (z < 0) z = 0;
            if (z > qmax) z = qmax;
            scales[n * G + g] = s16;
            zeros[n * G + g] = (uint8_t)z;
            for (int i = 0; i < GROUP; ++i) {
                float v = laqo_f16_to_f32(wg[i]);
                float t = rintf(v / s);
                int q = (int)t + z;
                if (q < 0) q = 0;
                if (q > qmax) q = qmax;
                codes[n * K + g * GROUP + i] = (uint8_t)q;
            }
        }
    }
}

/* ---------------------------------------------------------------------
 * Eq. 1 with given parameters: q = clip(round(w / s) + z, 0, 2^b - 1) for
 * every weight, with s = scales[n][g] (binary16, finite and > 0) and
 * z = zeros[n][g] (0 .. 2^b - 1) supplied by the caller, e.g. the scale and
 * zero point that LAQuant's QAT learned.  Same arithmetic as above: fp32
 * true division, round-half-to-even; the clip is taken on the real value,
 * so quotients far outside the code range never reach an integer
 * conversion.  A quotient that is not a number gives code 0.
 * ------------------------------------------------------------------- */
void laqo_codes_from_params(const uint16_t *w, int64_t N, int64_t K, int bits,
                            const uint16_t *scales, const uint8_t *zeros,
                            uint8_t *codes)
{
    const int64_t G = K / GROUP;
    const float qmax = (float)((1 << bits) - 1);
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t k = 0; k < K; ++k) {
            const int64_t g = k / GROUP;
            float s = laqo_f16_to_f32(scales[n * G + g]);
            float z = (float)zeros[n * G + g];
            float v = laqo_f16_to_f32(w[n * K + k]);
            float u = rintf(v / s) + z;
            if (!(u >= 0.0f))
                u = 0.0f;
            if (u > qmax)
                u = qmax;
            codes[n * K + k] = (uint8_t)u;
        }
    }
}

/* ---------------------------------------------------------------------
 * Packed layouts.
 *
 * W3: qweight is uint32 [N][3][K/32].  Chunk c of row n holds the codes of
 * k = 32c .. 32c+31 in the three words P_p = qweight[(n*3 + p)*(K/32) + c],
 * p = 0,1,2 ("planes").  Code i of the chunk:
 *   i < 30:  plane p = i / 10, r = i % 10, field f = r / 2, half h = r % 2,
 *            bits [16h + OFF[f], 16h + OFF[f] + 3) of P_p, OFF = {0,3,6,10,13}
 *   i = 30:  bit j of the code is bit 9 of P_j   (j = 0,1,2)
 *   i = 31:  bit j of the code is bit 25 of P_j
 * W4: qweight is uint32 [N][4][K/32].  Code i of chunk c is in plane
 *   p = i / 8, at bits [16*(i%2) + 4*((i%8)/2), +4).
 * The helpers below map (bits, i, code-bit j) -> (plane, bit position).
 * ------------------------------------------------------------------- */
static const int W3_OFF[5] = {0, 3, 6, 10, 13};

static void w3_bit_position(int i, int j, int *plane, int *bit)
{
    if (i < 30) {
        int r = i % 10;
        *plane = i / 10;
        *bit = 16 * (r % 2) + W3_OFF[r / 2] + j;
    } else {
        *plane = j;
        *bit = (i == 30) ? 9 : 25;
    }
}

static void w4_bit_position(int i, int j, int *plane, int *bit)
{
    *plane = i / 8;
    *bit = 16 * (i % 2) + 4 * ((i % 8) / 2) + j;
}

static void bit_position(int bits, int i, int j, int *plane, int *bit)
{
    if (bits == 3)
        w3_bit_position(i, j, plane, bit);
    else
        w4_bit_position(i, j, plane, bit);
}

/* codes uint8 [N][K] -> qweight uint32 [N][bits][K/32]; returns 0 on success,
 * -1 if a code does not fit in `bits` bits. */
int laqo_pack(const uint8_t *codes, int64_t N, int64_t K, int bits, uint32_t *qweight)
{
    const int64_t C = K / 32;
    int bad = 0;
    for (int64_t t = 0; t < N * bits * C; ++t)
        qweight[t] = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t c = 0; c < C; ++c) {
            for (int i = 0; i < 32; ++i) {
                unsigned q = codes[n * K + 32 * c + i];
                if (q >> bits)
                    bad = 1;
                for (int j = 0; j < bits; ++j) {
                    int plane, bit;
                    bit_position(bits, i, j, &plane, &bit);
                    uint32_t b = (q >> j) & 1u;
                    qweight[(n * bits + plane) * C + c] |= b << bit;
                }
            }
        }
    }
    return bad ? -1 : 0;
}

/* qweight uint32 [N][bits][K/32] -> codes uint8 [N][K] */
void laqo_unpack(const uint32_t *qweight, int64_t N, int64_t K, int bits, uint8_t *codes)
{
    const int64_t C = K / 32;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t c = 0; c < C; ++c) {
            for (int i = 0; i < 32; ++i) {
                unsigned q = 0;
                for (int j = 0; j < bits; ++j) {
                    int plane, bit;
                    bit_position(bits, i, j, &plane, &bit);
                    q |= ((qweight[(n * bits + plane) * C + c] >> bit) & 1u) << j;
                }
                codes[n * K + 32 * c + i] = (uint8_t)q;
            }
        }
    }
}

/* ---------------------------------------------------------------------
 * Dequantization and the linear.
 *   w_hat[n][k] = s16[n][g] * (q[n][k] - z[n][g])          (Eq. 1, exact)
 *   y[m][n]     = sum_g sum_{k in g} x[m][k] * w_hat[n][k]  (fp64)
 * x: fp16 bits [M][K]; y: double [M][N].
 * ------------------------------------------------------------------- */
void laqo_dequant(const uint8_t *codes, const uint16_t *scales, const uint8_t *zeros,
                  int64_t N, int64_t K, double *w_hat)
{
    const int64_t G = K / GROUP;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k) {
            int64_t g = k / GROUP;
            double s = (double)laqo_f16_to_f32(scales[n * G + g]);
            w_hat[n * K + k] = s * (double)((int)codes[n * K + k] - (int)zeros[n * G + g]);
        }
}

void laqo_linear(const uint16_t *x, int64_t M, const uint8_t *codes,
                 const uint16_t *scales, const uint8_t *zeros,
                 int64_t N, int64_t K, double *y)
{
    const int64_t G = K / GROUP;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t m = 0; m < M; ++m) {
            double acc = 0.0;
            for (int64_t g = 0; g < G; ++g) {
                double s = (double)laqo_f16_to_f32(scales[n * G + g]);
                int z = zeros[n * G + g];
                for (int64_t k = g * GROUP; k < (g + 1) * GROUP; ++k) {
                    double xv = (double)laqo_f16_to_f32(x[m * K + k]);
                    acc += xv * (s * (double)((int)codes[n * K + k] - z));
                }
            }
            y[m * N + n] = acc;
        }
    }
}

/* Bulk conversions, used by tests to check the two helpers above. */
void laqo_f16_to_f32_array(const uint16_t *h, int64_t n, float *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = laqo_f16_to_f32(h[i]);
}

void laqo_f32_to_f16_array(const float *v, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = laqo_f32_to_f16(v[i]);
}

int laqo_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
