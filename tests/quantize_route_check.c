/*
 * CPU check of the lemma behind the quantize kernel's reciprocal route
 * (fixed-grid round-to-nearest codes, Sec. 2.1 and Sec. 4): for bf16 weight
 * w, bf16 scale s with 2^-60 <= |s| <= 2^60 and zero-point |z| <= 64, the
 * binary32 steps
 *     q  = clamp(w * r, -2^30, 2^30)          r any value within 2 ulp of 1/s
 *     q' = fma(fma(-q, s, w), r, q)
 *     code = NaN(q') ? z : clamp(rint(q') + z, 0, 15)
 * give the code of the correctly rounded quotient w / s for every w.
 *
 * Usage: quantize_route_check STRIDE PART  -- scales with (bits % STRIDE) ==
 * PART of the 65536 bf16 patterns, every weight pattern, r at RN(1/s) and
 * 1 and 2 ulp either side, ten zero-points.  STRIDE 1 PART 0 is exhaustive.
 * Prints the number of checks and mismatches; exit status 1 on a mismatch.
 * Build with -ffp-contract=off so that only the fmas written here fuse.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float from_bf16(uint32_t bits) {
    uint32_t u = bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static unsigned code_of(float qf, float z) {
    float c = rintf(qf) + z;
    c = qf != qf ? z : fminf(fmaxf(c, 0.0f), 15.0f);
    return c != c || c < 0.0f ? 0u : (unsigned)c;
}

int main(int argc, char **argv) {
    if (argc != 3) return 2;
    const unsigned stride = (unsigned)atoi(argv[1]), part = (unsigned)atoi(argv[2]);
    const float zs[10] = {-64.0f, -63.5f, -20.0f, -7.0f, 0.0f, 3.5f, 8.0f, 15.0f, 40.0f, 64.0f};
    long long checks = 0, bad = 0;
    for (uint32_t sb = part; sb < 65536; sb += stride) {
        const float s = from_bf16(sb);
        if (!(fabsf(s) >= 0x1p-60f && fabsf(s) <= 0x1p60f)) continue;
        const float r0 = 1.0f / s;
        for (int dr = -2; dr <= 2; ++dr) {
            float r = r0;
            for (int t = 0; t < abs(dr); ++t) r = nextafterf(r, dr > 0 ? INFINITY : -INFINITY);
            for (uint32_t wb = 0; wb < 65536; ++wb) {
                const float w = from_bf16(wb);
                const float exact = w / s;
                const float q = fminf(fmaxf(w * r, -0x1p30f), 0x1p30f);
                const float qr = fmaf(fmaf(-q, s, w), r, q);
                for (int zi = 0; zi < 10; ++zi) {
                    ++checks;
                    if (code_of(exact, zs[zi]) != code_of(qr, zs[zi])) {
                        if (bad < 8) printf("mismatch s=%a w=%a r=%a z=%g\n", s, w, r, zs[zi]);
                        ++bad;
                    }
                }
            }
        }
    }
    printf("%lld checks, %lld mismatches\n", checks, bad);
    return bad != 0;
}
