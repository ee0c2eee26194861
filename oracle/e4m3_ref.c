/*
 * OCP E4M3 encoder in plain C (oracle; test infrastructure only).
 *
 * Same definition as oracle/e4m3.py: round |v| to the nearest representable
 * e4m3 magnitude with ties to the even mantissa field, saturate to 448,
 * keep the sign (a negative value that rounds to zero encodes 0x80).
 * Every step is exact in binary64: a float32 |v| is exact, the quantum
 * q = 2^(e-3) is a power of two, |v|/q is exact, and nearbyint() in the
 * default rounding mode rounds half to even.
 *
 * It exists so that a test can compare the device codec against the
 * definition over all 2^32 float32 bit patterns in a few seconds.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <stddef.h>

static uint8_t encode_one(float v)
{
    uint32_t bits;
    memcpy(&bits, &v, 4);
    uint8_t sign = (uint8_t)((bits >> 31) << 7);
    double a = fabs((double)v);
    if (a == 0.0)
        return sign;
    int e = ilogb(a);            /* floor(log2 a); float32 subnormals are normal here */
    if (e < -6)
        e = -6;
    double q = ldexp(1.0, e - 3);
    double mag = nearbyint(a / q) * q;
    if (mag > 448.0)
        mag = 448.0;
    if (mag == 0.0)
        return sign;
    int e2 = ilogb(mag);
    uint8_t code;
    if (e2 < -6) {                                   /* subnormal: m * 2^-9 */
        code = (uint8_t)nearbyint(mag / ldexp(1.0, -9));
    } else {
        double frac = mag / ldexp(1.0, e2);          /* in [1, 2) */
        uint8_t man = (uint8_t)nearbyint((frac - 1.0) * 8.0);
        code = (uint8_t)(((e2 + 7) << 3) | man);
    }
    return (uint8_t)(sign | code);
}

/* codes of n float32 values */
void oracle_e4m3_encode(const float *v, uint8_t *out, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        out[i] = encode_one(v[i]);
}

/* codes of the n consecutive float32 bit patterns start, start+1, ... */
void oracle_e4m3_sweep(uint32_t start, size_t n, uint8_t *out)
{
    for (size_t i = 0; i < n; ++i) {
        uint32_t b = start + (uint32_t)i;
        float v;
        memcpy(&v, &b, 4);
        out[i] = encode_one(v);
    }
}

/* codes of x / 2^e for the n consecutive float32 bit patterns start,
 * start+1, ... (the cast under a power-of-two block scale s = 2^e): the
 * quotient x 2^-e is exact in binary64 for every finite x and e in
 * [-126, 127], the conversion to float is the single binary32 rounding
 * fl32(x / 2^e), and a quotient beyond the binary32 range (infinite after
 * that rounding) saturates to 448 like every magnitude above it. */
void oracle_e4m3_sweep_pow2(uint32_t start, size_t n, int e, uint8_t *out)
{
    for (size_t i = 0; i < n; ++i) {
        uint32_t b = start + (uint32_t)i;
        float v;
        memcpy(&v, &b, 4);
        float q = (float)ldexp((double)v, -e);
        if (isinf(q))
            out[i] = (uint8_t)(((b >> 31) << 7) | 0x7E);
        else
            out[i] = encode_one(q);
    }
}
