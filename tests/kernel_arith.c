/* Exhaustive checks of two fp32 identities the int8 epilogues rely on (IEEE binary32,
 * round to nearest even, denormals kept):
 *   div127:  x * RN(1/127) corrected once by fma from its exact remainder equals the
 *            correctly rounded x / 127, for every non-negative finite x;
 *   code:    for every y in [-127, 127], RN(y + 1.5 * 2^23) has the two's-complement low
 *            byte of the nearest-even integer to y.
 * Prints the number of mismatches of each; exit status 0 when both are zero. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float as_float(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t as_bits(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

int main(void)
{
    const float R = 1.0f / 127.0f;
    long long bad_div = 0, bad_code = 0;
#pragma omp parallel for reduction(+ : bad_div) schedule(static)
    for (long long u = 0; u < 0x7F800000LL; ++u) {
        const float x = as_float((uint32_t)u);
        const volatile float q = x * R;
        const float s = fmaf(fmaf(-q, 127.0f, x), R, q);
        const volatile float t = x / 127.0f;
        if (as_bits(s) != as_bits(t)) ++bad_div;
    }
    const uint32_t top = as_bits(127.0f);
#pragma omp parallel for reduction(+ : bad_code) schedule(static)
    for (long long u = 0; u <= (long long)top; ++u) {
        for (int sign = 0; sign < 2; ++sign) {
            const float y = as_float((uint32_t)u | (sign ? 0x80000000u : 0u));
            const volatile float t = y + 12582912.0f;
            const uint8_t got = (uint8_t)(as_bits(t) & 0xFFu);
            const uint8_t want = (uint8_t)(int8_t)(int)rintf(y);
            if (got != want) ++bad_code;
        }
    }
    printf("div127 %lld code %lld\n", bad_div, bad_code);
    return bad_div || bad_code;
}
