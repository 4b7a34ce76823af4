/*
 * oracle.c -- plain CPU definition of the COMET W4Ax path.
 *
 * TEST INFRASTRUCTURE ONLY (see oracle.h).  Written for clarity, not speed:
 * every function follows the definition in the paper's order, with no
 * blocking, fusion or reordering beyond what the definition states.  Built
 * with -ffp-contract=off and without fast-math so that every fp32 operation
 * below is one IEEE operation.
 */
#include "oracle.h"

#include <math.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------- */
/* IEEE 754 binary16, from the format's definition:                           */
/*   exponent field e (5 bits, bias 15), fraction f (10 bits);                */
/*   e = 0      -> value f * 2^-24 (subnormal);                               */
/*   1..30      -> value (1024 + f) * 2^(e - 25);                             */
/*   31         -> infinity (f = 0) or NaN.                                   */
/* Rounding to binary16 is to the nearest representable value, ties to the   */
/* one whose fraction is even.  The arithmetic below is done in double,       */
/* where every step is exact: a float has 24 significant bits and the         */
/* quantum is a power of two.                                                */
/* ------------------------------------------------------------------------- */

float orc_f32_from_f16(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 31;
  int f = h & 1023;
  double v;
  if (e == 0) {
    v = ldexp((double)f, -24);
  } else if (e == 31) {
    v = f ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + f), e - 25);
  }
  return (float)(sign ? -v : v);
}

uint16_t orc_f16_from_f32(float x) {
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs((double)x);
  if (isnan(x)) return (uint16_t)(sign | 0x7E00);
  if (isinf(x)) return (uint16_t)(sign | 0x7C00);
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: quantum 2^-24; a count of 1024 is the smallest normal */
    double n = rint(a / ldexp(1.0, -24)); /* exact division, rint = ties-to-even */
    return (uint16_t)(sign | (uint16_t)n);
  }
  int ex;
  frexp(a, &ex);  /* a = fr * 2^ex, fr in [0.5, 1) */
  int e = ex - 1; /* a in [2^e, 2^(e+1)) */
  if (e > 15) return (uint16_t)(sign | 0x7C00);
  double n = rint(a / ldexp(1.0, e - 10)); /* significand count in [1024, 2048] */
  long bits = ((long)(e + 15) << 10) + ((long)n - 1024); /* n = 2048 carries into e+1 */
  if (bits >= 0x7C00) return (uint16_t)(sign | 0x7C00);
  return (uint16_t)(sign | (uint16_t)bits);
}

void orc_f16_from_f32_array(const float* x, uint16_t* h, size_t n) {
  for (size_t i = 0; i < n; ++i) h[i] = orc_f16_from_f32(x[i]);
}

void orc_f32_from_f16_array(const uint16_t* h, float* x, size_t n) {
  for (size_t i = 0; i < n; ++i) x[i] = orc_f32_from_f16(h[i]);
}

/* ------------------------------------------------------------------------- */
/* Block quantizer Q (Sec. 3.2: one scale per block of k = 128 channels;      */
/* 4-bit for normal blocks, 8-bit for outlier blocks).                        */
/* ------------------------------------------------------------------------- */

static int qmax_of(int bits) { return bits == 4 ? 7 : (bits == 8 ? 127 : -1); }

int orc_quantize_group(const float* v, int G, int bits, uint16_t* s16, int8_t* q) {
  int qmax = qmax_of(bits);
  if (qmax < 0 || G <= 0) return -1;
  float amax = 0.0f;
  for (int c = 0; c < G; ++c) {
    if (!isfinite(v[c])) return -1;
    float a = fabsf(v[c]);
    if (a > amax) amax = a;
  }
  float s32 = amax / (float)qmax; /* one IEEE fp32 division */
  uint16_t h = orc_f16_from_f32(s32);
  float s = orc_f32_from_f16(h); /* quantize with the stored scale */
  *s16 = h;
  for (int c = 0; c < G; ++c) {
    if (s == 0.0f) {
      q[c] = 0;
      continue;
    }
    float t = v[c] / s;  /* one IEEE fp32 division */
    float r = rintf(t);  /* nearest integer, ties to even */
    if (r > (float)qmax) r = (float)qmax;
    if (r < (float)-qmax) r = (float)-qmax;
    q[c] = (int8_t)r;
  }
  return 0;
}

static int set_threads(int nthreads) {
#ifdef _OPENMP
  return nthreads > 0 ? nthreads : omp_get_max_threads();
#else
  (void)nthreads;
  return 1;
#endif
}

int orc_quantize_act(const uint16_t* X, const uint8_t* prec, int M, int K, int G, int8_t* qa,
                     uint16_t* sa16, int nthreads) {
  if (M < 0 || K <= 0 || G <= 0 || K % G || G > 1024) return -1;
  int NG = K / G;
  for (int g = 0; g < NG; ++g)
    if (prec[g] != 4 && prec[g] != 8) return -1;
  int err = 0;
  int nt = set_threads(nthreads);
#pragma omp parallel for num_threads(nt) reduction(| : err) schedule(static)
  for (int m = 0; m < M; ++m) {
    float v[1024];
    for (int g = 0; g < NG; ++g) {
      for (int c = 0; c < G; ++c) v[c] = orc_f32_from_f16(X[(size_t)m * K + (size_t)g * G + c]);
      uint16_t s;
      if (orc_quantize_group(v, G, prec[g], &s, qa + (size_t)m * K + (size_t)g * G)) err |= 1;
      sa16[(size_t)g * M + m] = s;
    }
  }
  return err ? -1 : 0;
}

int orc_quantize_weight(const uint16_t* W, int N, int K, int G, int8_t* qw, uint16_t* sw16,
                        int nthreads) {
  if (N < 0 || K <= 0 || G <= 0 || K % G || G > 1024) return -1;
  int NG = K / G;
  int err = 0;
  int nt = set_threads(nthreads);
#pragma omp parallel for num_threads(nt) reduction(| : err) schedule(static)
  for (int n = 0; n < N; ++n) {
    float v[1024];
    for (int g = 0; g < NG; ++g) {
      for (int c = 0; c < G; ++c) v[c] = orc_f32_from_f16(W[(size_t)n * K + (size_t)g * G + c]);
      uint16_t s;
      if (orc_quantize_group(v, G, 4, &s, qw + (size_t)n * K + (size_t)g * G)) err |= 1;
      sw16[(size_t)g * N + n] = s;
    }
  }
  return err ? -1 : 0;
}

/* ------------------------------------------------------------------------- */
/* Byte encodings.  Sign-magnitude codes; in a 4-bit chunk the sign bits of   */
/* the upper four codes of each 8-code dword are rotated one byte down (see   */
/* oracle.h), which is the storage contract of the packed operands.           */
/* ------------------------------------------------------------------------- */

static unsigned sgn(int8_t q) { return q < 0 ? 1u : 0u; }
static unsigned mag(int8_t q) { return (unsigned)(q < 0 ? -q : q); }

void orc_encode4(const int8_t* q, int G, uint8_t* out) {
  for (int j = 0; j < G / 8; ++j) {
    const int8_t* c = q + 8 * j;
    for (int k = 0; k < 4; ++k) {
      unsigned b = (sgn(c[k]) << 7) | (mag(c[4 + k]) << 4) | (sgn(c[4 + ((k + 3) & 3)]) << 3) |
                   mag(c[k]);
      out[4 * j + k] = (uint8_t)b;
    }
  }
}

void orc_encode8(const int8_t* q, int G, uint8_t* out) {
  for (int c = 0; c < G; ++c) out[c] = (uint8_t)((sgn(q[c]) << 7) | mag(q[c]));
}

size_t orc_act_packed_bytes(const uint8_t* prec, int M, int K, int G) {
  size_t total = 0;
  for (int g = 0; g < K / G; ++g) total += (size_t)M * (size_t)(prec[g] == 8 ? G : G / 2);
  return total;
}

int orc_pack_act(const int8_t* qa, const uint8_t* prec, int M, int K, int G, uint8_t* A_packed) {
  if (M < 0 || K <= 0 || G <= 0 || K % G || G % 8) return -1;
  size_t base = 0;
  for (int g = 0; g < K / G; ++g) {
    size_t bytes = prec[g] == 8 ? (size_t)G : (size_t)G / 2;
    if (prec[g] != 4 && prec[g] != 8) return -1;
    for (int m = 0; m < M; ++m) {
      const int8_t* src = qa + (size_t)m * K + (size_t)g * G;
      uint8_t* dst = A_packed + base + (size_t)m * bytes;
      if (prec[g] == 8)
        orc_encode8(src, G, dst);
      else
        orc_encode4(src, G, dst);
    }
    base += (size_t)M * bytes;
  }
  return 0;
}

int orc_pack_weight(const int8_t* qw, int N, int K, int G, uint8_t* W_packed) {
  if (N < 0 || K <= 0 || G <= 0 || K % G || G % 8) return -1;
  for (int n = 0; n < N; ++n)
    for (int g = 0; g < K / G; ++g)
      orc_encode4(qw + (size_t)n * K + (size_t)g * G, G,
                  W_packed + (size_t)n * (K / 2) + (size_t)g * (G / 2));
  return 0;
}

/* ------------------------------------------------------------------------- */
/* W4Ax contraction (Sec. 4.1 and Sec. 5, O = WX in the paper's notation;    */
/* here out = X W^T with X [M][K] tokens x channels and W [N][K]).            */
/* ------------------------------------------------------------------------- */

static int32_t block_dot(const int8_t* a, const int8_t* w, int G) {
  int32_t s = 0;
  for (int c = 0; c < G; ++c) s += (int32_t)a[c] * (int32_t)w[c];
  return s;
}

void orc_group_acc(const int8_t* qa, const int8_t* qw, int M, int N, int K, int G, int32_t* acc) {
  int NG = K / G;
  for (int m = 0; m < M; ++m)
    for (int n = 0; n < N; ++n)
      for (int g = 0; g < NG; ++g)
        acc[((size_t)m * N + n) * NG + g] =
            block_dot(qa + (size_t)m * K + (size_t)g * G, qw + (size_t)n * K + (size_t)g * G, G);
}

void orc_dequant_gemm(const int8_t* qa, const uint16_t* sa16, const int8_t* qw,
                      const uint16_t* sw16, int M, int N, int K, int G, const int* rows,
                      int nrows, double* ref, int nthreads) {
  int NG = K / G;
  if (!rows) nrows = M;
  int nt = set_threads(nthreads);
#pragma omp parallel for num_threads(nt) schedule(dynamic, 1)
  for (int i = 0; i < nrows; ++i) {
    int m = rows ? rows[i] : i;
    for (int n = 0; n < N; ++n) {
      double sum = 0.0;
      for (int g = 0; g < NG; ++g) {
        int32_t acc =
            block_dot(qa + (size_t)m * K + (size_t)g * G, qw + (size_t)n * K + (size_t)g * G, G);
        double sa = (double)orc_f32_from_f16(sa16[(size_t)g * M + m]);
        double sw = (double)orc_f32_from_f16(sw16[(size_t)g * N + n]);
        sum += (double)acc * sa * sw;
      }
      ref[(size_t)i * N + n] = sum;
    }
  }
}

void orc_exact_gemm(const uint16_t* X, const uint16_t* W, int M, int N, int K, double* exact,
                    int nthreads) {
  int nt = set_threads(nthreads);
#pragma omp parallel for num_threads(nt) schedule(static)
  for (int m = 0; m < M; ++m)
    for (int n = 0; n < N; ++n) {
      double s = 0.0;
      for (int k = 0; k < K; ++k)
        s += (double)orc_f32_from_f16(X[(size_t)m * K + k]) *
             (double)orc_f32_from_f16(W[(size_t)n * K + k]);
      exact[(size_t)m * N + n] = s;
    }
}
