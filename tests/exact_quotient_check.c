/*
 * Exhaustive / randomized check of the quotient recipe the quantization kernels use for
 * y = RN32(x / S) and u = RN32(y / M):
 *     u = v * r;  e = fma(u, d, -v);  q = fma(-e, r, u)       with r = RN32(1 / d)
 * (Markstein's correction of a reciprocal product).  Each q is compared with the IEEE binary32
 * quotient v / d that the oracle computes.  Built and run by tests/test_exact_arith.py with
 * -ffp-contract=off, so every operation below is the one written.
 *
 * Modes (argv[1]):
 *   norm  every bfloat16 bit pattern x (both signs) against `nscales` scales S spread
 *         log-uniformly over [2^-26, 2^26] with random significands, plus the powers of two
 *         at the ends; the kernels take this path only for |x| >= 2^-74 and S in that range.
 *   norm32 `count` random binary32 x (random sign and significand, |x| >= 2^-74) against
 *         random S in [2^-26, 2^26]: the same path for binary32 input.
 *   sig   `count` random binary32 y (random sign, exponent field 1..254) against the eight
 *         E4M3 significands M = 1 + b/8 with r = RN32(1/M), the emit step's quotient.  The
 *         emit takes this path for every y.  Where the quotient is below 2^-120 the remainder
 *         can underflow and the corrected quotient may differ from v / d in its last bits;
 *         such quotients (and the true ones) lie far below 2^-11, the smallest FP4 midpoint
 *         at the smallest positive E4M3 scale (0.25 * 2^-9), so both round to the E2M1 code 0
 *         at every scale; they are counted apart ("tiny_ok") when the sign also agrees.
 * Output: one line "checked <n> mismatch <m> nonfinite_ok <k> tiny_ok <t>" (and the first
 * mismatches).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float from_bits(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t bits(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

static float corrected_quotient(float v, float d, float r)
{
    float u = v * r;
    float e = fmaf(u, d, -v);
    return fmaf(-e, r, u);
}

/* splitmix64: a small deterministic generator for the test inputs */
static uint64_t sm_state;
static uint64_t sm_next(void)
{
    uint64_t z = (sm_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static int same(float a, float b)
{
    return bits(a) == bits(b);   /* also the sign of a zero */
}

int main(int argc, char** argv)
{
    if (argc < 3) return 2;
    sm_state = 12345;
    uint64_t checked = 0, mismatch = 0, nonfinite_ok = 0, tiny_ok = 0;
    if (strcmp(argv[1], "norm") == 0) {
        int nscales = atoi(argv[2]);
        for (int k = 0; k < nscales + 2; ++k) {
            float S;
            if (k == nscales) S = 0x1p-26f;
            else if (k == nscales + 1) S = 0x1p26f;
            else {
                double e = -26.0 + 52.0 * (double)(sm_next() >> 11) / 9007199254740992.0;
                S = (float)exp2(e);
            }
            float rS = 1.0f / S;
            for (uint32_t h = 0; h < 65536; ++h) {
                float x = from_bits(h << 16);
                if (!isfinite(x) || fabsf(x) < 0x1p-74f) continue;
                float want = x / S;
                float got = corrected_quotient(x, S, rS);
                checked++;
                if (!isfinite(want)) {
                    /* x / S overflows: the oracle rejects the input as non-finite; the
                     * recipe must not produce a finite value either */
                    if (!isfinite(got)) nonfinite_ok++;
                    else mismatch++;
                    continue;
                }
                if (!same(got, want)) {
                    if (mismatch < 5) printf("x=%a S=%a want=%a got=%a\n", x, S, want, got);
                    mismatch++;
                }
            }
        }
    } else if (strcmp(argv[1], "norm32") == 0) {
        long long count = atoll(argv[2]);
        for (long long t = 0; t < count; ++t) {
            uint64_t z = sm_next(), z2 = sm_next();
            /* exponent field 53..254: |x| from 2^-74 up to the largest finite values */
            uint32_t e = 53 + (uint32_t)((z >> 32) % 202u);
            float x = from_bits(((uint32_t)(z >> 63) << 31) | (e << 23) | (uint32_t)(z & 0x7FFFFFu));
            double ex = -26.0 + 52.0 * (double)(z2 >> 11) / 9007199254740992.0;
            float S = (float)exp2(ex);
            float rS = 1.0f / S;
            float want = x / S;
            float got = corrected_quotient(x, S, rS);
            checked++;
            if (!isfinite(want)) {
                if (!isfinite(got)) nonfinite_ok++;
                else mismatch++;
                continue;
            }
            if (!same(got, want)) {
                if (mismatch < 5) printf("x=%a S=%a want=%a got=%a\n", x, S, want, got);
                mismatch++;
            }
        }
    } else if (strcmp(argv[1], "sig") == 0) {
        long long count = atoll(argv[2]);
        for (int b = 0; b < 8; ++b) {
            float M = 1.0f + (float)b / 8.0f;
            float rM = 1.0f / M;
            for (long long t = 0; t < count; ++t) {
                uint64_t z = sm_next();
                uint32_t e = 1 + (uint32_t)((z >> 32) % 254u);
                uint32_t yb = ((uint32_t)(z >> 63) << 31) | (e << 23) | (uint32_t)(z & 0x7FFFFFu);
                float y = from_bits(yb);
                float want = y / M;
                float got = corrected_quotient(y, M, rM);
                checked++;
                if (!same(got, want)) {
                    if (fabsf(want) < 0x1p-120f && fabsf(got) < 0x1p-11f &&
                        signbit(got) == signbit(want)) {
                        tiny_ok++;
                        continue;
                    }
                    if (mismatch < 5) printf("y=%a M=%a want=%a got=%a\n", y, M, want, got);
                    mismatch++;
                }
            }
            /* signed zeros keep their sign (volatile: evaluated at run time, not folded) */
            volatile float pz = 0.0f, nz = -0.0f;
            float zp = corrected_quotient(pz, M, rM), zn = corrected_quotient(nz, M, rM);
            checked += 2;
            if (!same(zp, 0.0f)) mismatch++;
            if (!same(zn, -0.0f)) mismatch++;
        }
    } else {
        return 2;
    }
    printf("checked %llu mismatch %llu nonfinite_ok %llu tiny_ok %llu\n",
           (unsigned long long)checked, (unsigned long long)mismatch,
           (unsigned long long)nonfinite_ok, (unsigned long long)tiny_ok);
    return 0;
}
