/*
 * CPU oracle for carry-through checksum CNN inference: TEST INFRASTRUCTURE.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * use this file.  It is the plain, slow, obviously correct definition that
 * the GPU library is checked against; it shares no code with that library.
 *
 * Layer arithmetic for one image in NCHW fp32:
 *   - direct nested-loop convolution (Sec. II-A builds the carry-through
 *     filter out of an ordinary convolution, so the convolution itself is
 *     the textbook definition): zero padding is taken literally, i.e. the
 *     padded input is the image extended by zeros and every tap multiplies
 *     (0 * Inf gives NaN, as in any GEMM-based convolution);
 *   - accumulation in fp32 in the fixed order (c, r, s), one rounding per
 *     product and per sum (built with -ffp-contract=off);
 *   - then + bias, batch normalisation exactly as Eq. (1) is written,
 *     + residual, ReLU (NaN propagates: only x < 0 maps to 0);
 *   - fp16 networks: every stored tensor is rounded once to binary16 with
 *     round-to-nearest-even (overflow to +-Inf, subnormals kept), the
 *     conversion written from the IEEE 754 format definition below.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ---- IEEE 754 binary32 <-> binary16 ------------------------------------ */

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* binary32 -> binary16, round to nearest, ties to even. */
uint16_t or_f32_to_f16(float f)
{
    uint32_t b = f2u(f);
    uint32_t sign = (b >> 16) & 0x8000u;
    uint32_t e = (b >> 23) & 0xffu;
    uint32_t m = b & 0x7fffffu;
    if (e == 0xffu)                      /* Inf or NaN (NaN stays NaN) */
        return (uint16_t)(sign | 0x7c00u | (m ? (0x200u | (m >> 13)) : 0u));
    int E = (int)e - 127;                /* unbiased exponent */
    if (E > 15)                          /* beyond the largest finite */
        return (uint16_t)(sign | 0x7c00u);
    if (E >= -14) {                      /* normal binary16 range */
        uint32_t hm = m >> 13, rem = m & 0x1fffu;
        uint32_t h = ((uint32_t)(E + 15) << 10) | hm;
        if (rem > 0x1000u || (rem == 0x1000u && (hm & 1u)))
            h += 1u;                     /* a carry may reach Inf: correct */
        return (uint16_t)(sign | h);
    }
    if (e == 0)                          /* binary32 zero or subnormal */
        return (uint16_t)sign;
    /* binary16 subnormal: count units of 2^-24 */
    uint32_t sig = (1u << 23) | m;       /* value = sig * 2^(E-23) */
    int s = -(E + 1);                    /* value / 2^-24 = sig >> s */
    if (s > 24)
        return (uint16_t)sign;
    uint32_t q = sig >> s, rem = sig & ((1u << s) - 1u), half = 1u << (s - 1);
    if (rem > half || (rem == half && (q & 1u)))
        q += 1u;                         /* may become the smallest normal */
    return (uint16_t)(sign | q);
}

/* The binary32 bit pattern of the value a binary16 pattern stands for.
 * Exact for all 65536 patterns; a NaN keeps its payload (the quiet bit is
 * not forced), so the widening is one-to-one. */
uint32_t or_f16_widen_bits(uint16_t h)
{
    uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
    uint32_t e = ((uint32_t)h >> 10) & 0x1fu;
    uint32_t m = (uint32_t)h & 0x3ffu;
    if (e == 0) {
        if (m == 0)
            return sign;
        int k = 0;                       /* normalise the subnormal */
        while (!(m & 0x400u)) { m <<= 1; k++; }
        return sign | ((uint32_t)(113 - k) << 23) | ((m & 0x3ffu) << 13);
    }
    if (e == 31)
        return sign | 0x7f800000u | (m << 13);
    return sign | ((e - 15u + 127u) << 23) | (m << 13);
}

float or_f16_to_f32(uint16_t h) { return u2f(or_f16_widen_bits(h)); }

/* Inverse of the widening on its image: the binary16 pattern whose
 * widening is the binary32 pattern b, or -1 if there is none (b is not a
 * value of the binary16 format).  No rounding: a stored fp16 element is
 * recovered bit for bit, NaN payloads included. */
int32_t or_f16_narrow_exact_bits(uint32_t b)
{
    uint32_t sign = (b >> 16) & 0x8000u;
    uint32_t e = (b >> 23) & 0xffu;
    uint32_t m = b & 0x7fffffu;
    if (e == 0xffu)                      /* Inf / NaN: payload in the top 10 */
        return (m & 0x1fffu) ? -1 : (int32_t)(sign | 0x7c00u | (m >> 13));
    if (e == 0)                          /* zero (binary32 subnormals: none) */
        return m ? -1 : (int32_t)sign;
    int E = (int)e - 127;
    if (E > 15 || E < -24)
        return -1;
    if (E >= -14)                        /* binary16 normal */
        return (m & 0x1fffu) ? -1
                             : (int32_t)(sign | ((uint32_t)(E + 15) << 10) | (m >> 13));
    uint32_t sig = (1u << 23) | m;       /* binary16 subnormal: sig >> s units */
    int s = -(E + 1);                    /* of 2^-24 */
    if (sig & ((1u << s) - 1u))
        return -1;
    return (int32_t)(sign | (sig >> s));
}

/* Single-bit faults on fp16-stored elements held as binary32 patterns
 * (Sec. III-A): element idx[i] of v gets bit bit[i] of its binary16
 * pattern XOR-ed, working on the integer patterns only, so a second call
 * with the same arguments restores every element bit for bit.  Returns the
 * number of elements that hold no binary16 value (left unchanged). */
int64_t or_f16_flip_stored(uint32_t *v, const int64_t *idx, const int32_t *bit,
                           int64_t n)
{
    int64_t bad = 0;
    for (int64_t i = 0; i < n; i++) {
        int32_t h = or_f16_narrow_exact_bits(v[idx[i]]);
        if (h < 0 || bit[i] < 0 || bit[i] > 15) {
            bad++;
            continue;
        }
        v[idx[i]] = or_f16_widen_bits((uint16_t)((uint32_t)h ^ (1u << bit[i])));
    }
    return bad;
}

void or_f16_narrow_exact_array(const uint32_t *x, int32_t *y, int64_t n)
{
    for (int64_t i = 0; i < n; i++) y[i] = or_f16_narrow_exact_bits(x[i]);
}

void or_f16_widen_bits_array(const uint16_t *x, uint32_t *y, int64_t n)
{
    for (int64_t i = 0; i < n; i++) y[i] = or_f16_widen_bits(x[i]);
}

static float rnd16(float v) { return or_f16_to_f32(or_f32_to_f16(v)); }

void or_f32_to_f16_array(const float *x, uint16_t *y, int64_t n)
{
    for (int64_t i = 0; i < n; i++) y[i] = or_f32_to_f16(x[i]);
}

void or_f16_to_f32_array(const uint16_t *x, float *y, int64_t n)
{
    for (int64_t i = 0; i < n; i++) y[i] = or_f16_to_f32(x[i]);
}

void or_round_f16_array(float *x, int64_t n)
{
    for (int64_t i = 0; i < n; i++) x[i] = rnd16(x[i]);
}

/* ---- layers (one image) ------------------------------------------------- */

static float relu(float v) { return (v < 0.0f) ? 0.0f : v; }

/*
 * y[k][p][q] = act( BN( sum_{c,r,s} xpad[g*Cg+c][p*st-pad+r][q*st-pad+s]
 *                                   * w[k][c][r][s] + bias[k] ) + res[k][p][q] )
 * with g = k / (K/groups), Cg = C/groups.  Any of bias / BN (all four of
 * mean, var, gamma, beta) / residual may be NULL.
 */
void or_conv(const float *x, int C, int H, int W,
             const float *w, int K, int R, int S, int stride, int pad,
             int groups, const float *bias, const float *mean,
             const float *var, const float *gamma, const float *beta,
             float eps, const float *residual, int do_relu, int round16,
             float *y)
{
    int Cg = C / groups, Kg = K / groups;
    int P = (H + 2 * pad - R) / stride + 1;
    int Q = (W + 2 * pad - S) / stride + 1;
    for (int k = 0; k < K; k++) {
        int g = k / Kg;
        for (int p = 0; p < P; p++) {
            for (int q = 0; q < Q; q++) {
                float acc = 0.0f;
                for (int c = 0; c < Cg; c++) {
                    int ci = g * Cg + c;
                    for (int r = 0; r < R; r++) {
                        int h = p * stride - pad + r;
                        for (int s = 0; s < S; s++) {
                            int ww = q * stride - pad + s;
                            float xv = 0.0f;
                            if (h >= 0 && h < H && ww >= 0 && ww < W)
                                xv = x[((int64_t)ci * H + h) * W + ww];
                            float prod = xv * w[(((int64_t)k * Cg + c) * R + r) * S + s];
                            acc = acc + prod;
                        }
                    }
                }
                float v = acc;
                if (bias)
                    v = v + bias[k];
                if (mean) {                                    /* Eq. (1) */
                    float num = v - mean[k];
                    float den = sqrtf(var[k] + eps);
                    v = (num / den) * gamma[k] + beta[k];
                }
                int64_t o = ((int64_t)k * P + p) * Q + q;
                if (residual)
                    v = v + residual[o];
                if (do_relu)
                    v = relu(v);
                if (round16)
                    v = rnd16(v);
                y[o] = v;
            }
        }
    }
}

/* Max pooling; padding positions hold -Inf; a NaN in the window gives NaN. */
void or_maxpool(const float *x, int C, int H, int W, int k, int stride,
                int pad, int round16, float *y)
{
    int P = (H + 2 * pad - k) / stride + 1;
    int Q = (W + 2 * pad - k) / stride + 1;
    for (int c = 0; c < C; c++)
        for (int p = 0; p < P; p++)
            for (int q = 0; q < Q; q++) {
                float m = -INFINITY;
                int seen_nan = 0;
                float nanv = 0.0f;
                for (int r = 0; r < k; r++)
                    for (int s = 0; s < k; s++) {
                        int h = p * stride - pad + r, ww = q * stride - pad + s;
                        float v = -INFINITY;
                        if (h >= 0 && h < H && ww >= 0 && ww < W)
                            v = x[((int64_t)c * H + h) * W + ww];
                        if (v != v) {
                            if (!seen_nan) nanv = v;
                            seen_nan = 1;
                        } else if (v > m) {
                            m = v;
                        }
                    }
                float v = seen_nan ? nanv : m;
                if (round16)
                    v = rnd16(v);
                y[((int64_t)c * P + p) * Q + q] = v;
            }
}

/* Global average pooling: fp32 sum in (h, w) order, then one division. */
void or_gap(const float *x, int C, int H, int W, int round16, float *y)
{
    for (int c = 0; c < C; c++) {
        float acc = 0.0f;
        for (int i = 0; i < H * W; i++)
            acc = acc + x[(int64_t)c * H * W + i];
        float v = acc / (float)(H * W);
        if (round16)
            v = rnd16(v);
        y[c] = v;
    }
}

/* y[o] = act( sum_i x[i] * w[o][i] + b[o] ), fp32 sum in order i. */
void or_fc(const float *x, int IN, const float *w, int OUT, const float *b,
           int do_relu, int round16, float *y)
{
    for (int o = 0; o < OUT; o++) {
        float acc = 0.0f;
        for (int i = 0; i < IN; i++) {
            float prod = x[i] * w[(int64_t)o * IN + i];
            acc = acc + prod;
        }
        float v = acc;
        if (b)
            v = v + b[o];
        if (do_relu)
            v = relu(v);
        if (round16)
            v = rnd16(v);
        y[o] = v;
    }
}
