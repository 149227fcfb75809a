/*
 * Exhaustive check of the construct kernel's division by 3: for every
 * non-negative finite binary32 d, q = fl(d * fl(1/3)), rem = fma(-3, q, d),
 * s = fma(rem, fl(1/3), q) must equal the IEEE quotient fl(d / 3). Built with
 * -ffp-contract=off and hardware FMA (correctly rounded), so each step is one
 * IEEE binary32 operation, as in the kernel. Prints the mismatch count and
 * exits nonzero if there is any.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float from_bits(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t to_bits(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

int main(void)
{
    const float third = 0x1.555556p-2f;   /* fl(1/3) */
    unsigned long long bad = 0;
#pragma omp parallel for reduction(+ : bad) schedule(static)
    for (long long i = 0; i < 0x7F800000LL; ++i) {
        const float d = from_bits((uint32_t)i);
        const volatile float ref = d / 3.0f;
        const float q = d * third;
        const float rem = fmaf(-3.0f, q, d);
        const float s = fmaf(rem, third, q);
        if (to_bits(s) != to_bits(ref)) ++bad;
    }
    printf("%llu\n", bad);
    return bad != 0;
}
