/*
 * FP8 KV oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * Paper: "Execution-State Capsules", §3 "Definition" (the KV region may be
 * held in FP8, which roughly halves the capsule, with a BF16 working stage
 * whose valid end is part of the boundary descriptor) and the §3 cost model
 * (restore copies bytes and rebinds; the BF16 stage is rebuilt lazily on the
 * next read).  The paper does not fix the FP8 format; the readings taken
 * here: OCP 8-bit floating point E4M3 ("E4M3FN": 1 sign, 4 exponent bits with
 * bias 7, 3 mantissa bits, no infinities, NaN = S.1111.111, largest finite
 * magnitude 448), one fp32 scale per buffer, values stored as x / scale.
 *
 * Quantize (bf16 -> e4m3): x = float(bf16) * inv_scale in fp32, inv_scale =
 *   1.0f / scale in fp32; the code is the representable value NEAREST to x,
 *   ties to the code with an even mantissa (round to nearest even);
 *   |x| >= 448 and +-inf saturate to +-448; NaN keeps its sign as S.1111.111.
 *   The nearest value is found by a plain search over the 127 non-negative
 *   finite codes -- no bit tricks -- so it can be checked by eye.
 * Dequantize (e4m3 -> bf16): y = decode(code) * scale in fp32, rounded to the
 *   nearest bf16 (ties to even); NaN codes give the canonical bf16 NaN with
 *   the code's sign.
 *
 * Parity status: pinned (the format's own values, round trips of every code,
 * rounding ties, saturation; see tests/oracle_pins.py).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* value of a non-negative E4M3 code with exponent field e and mantissa m */
static double e4m3_magnitude(unsigned e, unsigned m) {
    if (e == 0) return ldexp((double)m / 8.0, -6);         /* subnormal: m/8 * 2^(1-7) */
    return ldexp(1.0 + (double)m / 8.0, (int)e - 7);        /* normal: 1.m * 2^(e-7)    */
}

float orc_e4m3_decode(uint8_t code) {
    const unsigned s = code >> 7, e = (code >> 3) & 15u, m = code & 7u;
    if (e == 15u && m == 7u) return s ? -NAN : NAN;
    const double v = e4m3_magnitude(e, m);
    return (float)(s ? -v : v);
}

uint8_t orc_e4m3_encode(float x) {
    uint32_t bits;
    memcpy(&bits, &x, 4);
    const uint8_t sign = (uint8_t)((bits >> 31) << 7);
    if (isnan(x)) return (uint8_t)(sign | 0x7Fu);
    const double a = fabs((double)x);
    if (a >= 448.0) return (uint8_t)(sign | 0x7Eu);         /* saturate (inf included) */
    /* nearest of the finite non-negative codes 0x00 .. 0x7E (ascending values) */
    unsigned best = 0;
    double best_d = INFINITY;
    for (unsigned c = 0; c <= 0x7Eu; ++c) {
        const double v = e4m3_magnitude(c >> 3, c & 7u);
        const double d = fabs(v - a);
        if (d < best_d || (d == best_d && (c & 1u) == 0u)) {
            best = c;
            best_d = d;
        }
    }
    return (uint8_t)(sign | best);
}

/* nearest bf16 to an fp32 value, ties to even (NaN -> canonical quiet NaN) */
uint16_t orc_bf16_round(float y) {
    uint32_t u;
    memcpy(&u, &y, 4);
    if (isnan(y)) return (uint16_t)(((u >> 16) & 0x8000u) | 0x7FC0u);
    if (isinf(y)) return (uint16_t)(u >> 16);
    const uint32_t lo = u & 0xFFFF0000u;     /* truncation toward zero (in magnitude) */
    const uint32_t hi = lo + 0x10000u;       /* next bf16 away from zero               */
    float flo;
    memcpy(&flo, &lo, 4);
    /* the step above the largest finite bf16 is infinity; for rounding it
     * stands at 2^128, one unit in the last place beyond the largest value */
    double vhi;
    if ((hi & 0x7F800000u) == 0x7F800000u) {
        vhi = ldexp(1.0, 128);
        if (hi & 0x80000000u) vhi = -vhi;
    } else {
        float fhi;
        memcpy(&fhi, &hi, 4);
        vhi = (double)fhi;
    }
    const double dlo = fabs((double)y - (double)flo), dhi = fabs(vhi - (double)y);
    if (dlo < dhi) return (uint16_t)(lo >> 16);
    if (dhi < dlo) return (uint16_t)(hi >> 16);
    return (uint16_t)(((lo >> 16) & 1u) ? (hi >> 16) : (lo >> 16));
}

static float bf16_value(uint16_t h) {
    const uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

void orc_fp8_quantize(const uint16_t* src_bf16, uint8_t* dst, uint64_t n, float scale) {
    const float inv = 1.0f / scale;
    for (uint64_t i = 0; i < n; ++i) {
        const float x = bf16_value(src_bf16[i]) * inv;
        dst[i] = orc_e4m3_encode(x);
    }
}

void orc_fp8_dequantize(const uint8_t* src, uint16_t* dst_bf16, uint64_t n, float scale) {
    for (uint64_t i = 0; i < n; ++i) {
        const uint8_t c = src[i];
        if (((c >> 3) & 15u) == 15u && (c & 7u) == 7u) {
            dst_bf16[i] = (uint16_t)((c & 0x80u) ? 0xFFC0u : 0x7FC0u);
            continue;
        }
        const float y = orc_e4m3_decode(c) * scale;
        dst_bf16[i] = orc_bf16_round(y);
    }
}
