/* Exhaustive check of the division-free quotient sequences of the GPU
 * quantizer for binary32 operands: for every binary32 value a in the binades
 * [2^lo, 2^hi) and M in {15, 255} (the asymmetric code ranges) and 127 (the
 * INT8 residual of the cold-tier upgrade),
 *   scale: c = RN(1/M), s0 = RN(a c), e = RN(a - s0 M), q = RN(s0 + e c)
 *          must equal RN(a / M);
 *   recip: for every r0 within 2 ulp of RN(1/a): q0 = RN(M r0),
 *          e = RN(M - q0 a), r = RN(q0 + e r0) must equal RN(M / a).
 *   clamp: RN(a RN(M / a)) < M + 1/2, so for |x| <= a the code of x never
 *          needs the clamp to [-M, M] (RN is monotone).
 * Every RN of an expression with one product is a fused multiply-add
 * (fmaf, correctly rounded), the reference quotients are IEEE binary32
 * divisions.  Prints the number of failures (0 expected) and exits 1 if any.
 * Usage: quotient_sweep LO HI */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <stdint.h>

static float bits_f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  const int lo = atoi(argv[1]), hi = atoi(argv[2]);
  const float Ms[3] = {15.0f, 127.0f, 255.0f};
  unsigned long long fails = 0, checked = 0;
  for (int mi = 0; mi < 3; ++mi) {
    const float M = Ms[mi];
    volatile float one = 1.0f;
    const float c = one / M;
    for (int e2 = lo; e2 < hi; ++e2) {
      const uint32_t base = (uint32_t)(e2 + 127) << 23;
      for (uint32_t m = 0; m < (1u << 23); ++m) {
        const float a = bits_f(base | m);
        volatile float av = a;
        const float want_s = av / M;
        const float s0 = a * c;
        const float e = fmaf(-s0, M, a);
        const float s = fmaf(e, c, s0);
        if (s != want_s) { ++fails; if (getenv("SHOW")) printf("scale M=%g a=%a got %a want %a\n", M, a, s, want_s); }
        const float want_r = M / av;
        volatile float prod = a * want_r;
        if (!(prod < M + 0.5f)) { ++fails; if (getenv("SHOW")) printf("clamp M=%g a=%a\n", M, a); }
        const float ra = one / av;
        float r0s[5];
        r0s[2] = ra;
        r0s[1] = nextafterf(ra, 0.0f);
        r0s[0] = nextafterf(r0s[1], 0.0f);
        r0s[3] = nextafterf(ra, INFINITY);
        r0s[4] = nextafterf(r0s[3], INFINITY);
        for (int k = 0; k < 5; ++k) {
          const float r0 = r0s[k];
          const float ey = fmaf(-a, r0, 1.0f);
          const float y = fmaf(ey, r0, r0);  /* reciprocal refined once */
          const float q0 = M * y;
          const float er = fmaf(-q0, a, M);
          const float r = fmaf(er, y, q0);
          if (r != want_r) { ++fails; if (getenv("SHOW")) printf("recip M=%g a=%a k=%d got %a want %a\n", M, a, k - 2, r, want_r); }
        }
        checked += 6;
      }
    }
  }
  printf("%llu checked, %llu failures\n", checked, fails);
  return fails ? 1 : 0;
}
