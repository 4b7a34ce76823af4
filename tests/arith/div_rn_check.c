/* Exhaustive check of the division scheme the quantization kernels use in
 * place of a per-element IEEE division: with r = RN(1/s),
 *     q0 = RN(a * r),  rem = RN(a - q0 * s) (one fma),  q = RN(q0 + rem * r) (one fma),
 * q must equal RN(a / s) for every operand pair the kernels can see.
 *
 * mode "fp16": s over every positive finite binary16 value, a over every
 *   non-negative finite binary16 value up to 128 * s (the activation and
 *   weight quantizers: |x| <= amax <= 127 * s * (1 + 2^-10)).
 * mode "kv": s over every positive finite binary16 value, a = RN(x - mn) for
 *   seeded random binary16 pairs x >= mn with (x - mn) <= 16 * s, plus every
 *   binary32 value within 64 ulps of each midpoint (k + 1/2) * s, k = 0..15
 *   (the KV4 quantizer: a = x - mn <= 15 * s * (1 + 2^-10)).
 * mode "qmax": s in {7, 127} (the block quantizers' scale s = RN(amax / qmax)),
 *   a over every non-negative finite binary16 value, r = RN(1/s).
 * With a second argument "nbr" (modes fp16 and kv), r also takes the two
 *   binary32 neighbours of RN(1/s): every result within one ulp of 1/s (what a
 *   hardware reciprocal guarantees) is covered.
 * Prints the number of pairs checked and of mismatches; exit status 1 on any
 * mismatch.  Built with -ffp-contract=off so a * r is a plain multiply. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float f16(uint16_t h) {
  uint32_t s = (uint32_t)(h >> 15) << 31, e = (h >> 10) & 31, f = h & 1023, u;
  if (e == 0) {
    float v = (float)f * 0x1p-24f;
    return (h >> 15) ? -v : v;
  }
  u = s | ((e + 112) << 23) | (f << 13);
  float v;
  memcpy(&v, &u, 4);
  return v;
}

static uint32_t bits(float v) {
  uint32_t u;
  memcpy(&u, &v, 4);
  return u;
}

static float from_bits(uint32_t u) {
  float v;
  memcpy(&v, &u, 4);
  return v;
}

static volatile float sink;

static int check1(float a, float s, float r) {
  float q0 = a * r;
  float rem = fmaf(-q0, s, a);
  float q = fmaf(rem, r, q0);
  float want = a / s;
  return bits(q) != bits(want);
}

static int nbr = 0;

static int check(float a, float s, float r) {
  int bad = check1(a, s, r);
  if (nbr) bad |= check1(a, s, nextafterf(r, 0.0f)) | check1(a, s, nextafterf(r, INFINITY));
  return bad;
}

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next64(void) {
  uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int main(int argc, char** argv) {
  const char* mode = argc > 1 ? argv[1] : "fp16";
  nbr = argc > 2 && !strcmp(argv[2], "nbr");
  unsigned long long n = 0, bad = 0;
  if (!strcmp(mode, "qmax")) {
    const float qs[2] = {7.0f, 127.0f};
    for (int i = 0; i < 2; ++i) {
      const float s = qs[i], r = 1.0f / s;
      for (uint32_t xh = 0; xh < 0x7C00; ++xh) {
        ++n;
        bad += check1(f16((uint16_t)xh), s, r);
      }
    }
    printf("%s: %llu pairs, %llu mismatches\n", mode, n, bad);
    return bad ? 1 : 0;
  }
  for (uint32_t sh = 1; sh < 0x7C00; ++sh) {
    float s = f16((uint16_t)sh);
    float r = 1.0f / s;
    if (!strcmp(mode, "fp16")) {
      for (uint32_t xh = 0; xh < 0x7C00; ++xh) {
        float a = f16((uint16_t)xh);
        if (a > 128.0f * s) break;
        ++n;
        bad += check(a, s, r);
      }
    } else {
      for (int i = 0; i < 256; ++i) {
        uint64_t w = next64();
        float x = f16((uint16_t)(w & 0xFFFF)), mn = f16((uint16_t)((w >> 16) & 0xFFFF));
        if (!(x == x) || !(mn == mn) || isinf(x) || isinf(mn)) continue;
        if (x < mn) {
          float t = x;
          x = mn;
          mn = t;
        }
        float a = x - mn;
        if (a > 16.0f * s) a = (float)ldexp((double)(w >> 40) / 16777216.0, 4) * s;
        ++n;
        bad += check(a, s, r);
      }
      for (int k = 0; k < 16; ++k) {
        float mid = ((float)k + 0.5f) * s; /* exact: 5 x 11 significant bits */
        uint32_t mb = bits(mid);
        for (int d = -64; d <= 64; ++d) {
          float a = from_bits(mb + (uint32_t)d);
          if (!(a >= 0.0f)) continue;
          ++n;
          bad += check(a, s, r);
        }
      }
    }
  }
  printf("%s: %llu pairs, %llu mismatches\n", mode, n, bad);
  sink = (float)bad;
  return bad ? 1 : 0;
}
