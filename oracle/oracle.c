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
#include <stdlib.h>
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
  if (N < 0 || N % 16 || K <= 0 || G <= 0 || K % G || G % 8) return -1;
  const int NG = K / G;
  for (int n = 0; n < N; ++n)
    for (int g = 0; g < NG; ++g) {
      /* 16-row panel n / 16, block g, row n % 16 */
      const size_t chunk = ((size_t)(n / 16) * NG + g) * 16 + (size_t)(n % 16);
      orc_encode4(qw + (size_t)n * K + (size_t)g * G, G, W_packed + chunk * (G / 2));
    }
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

/* ------------------------------------------------------------------------- */
/* Channel permutation and the calibration map (Sec. 3.2).  Outlier channels  */
/* are found from sampled activations and gathered into a few blocks, which   */
/* are the ones quantized to 8 bits; the weight columns take the same         */
/* permutation, so X W^T is unchanged.                                        */
/* ------------------------------------------------------------------------- */

int orc_permute_columns(const uint16_t* X, const int32_t* perm, int R, int K, uint16_t* out) {
  if (R < 0 || K <= 0) return -1;
  for (int c = 0; c < K; ++c)
    if (perm[c] < 0 || perm[c] >= K) return -1;
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < K; ++c) out[(size_t)r * K + c] = X[(size_t)r * K + perm[c]];
  return 0;
}

void orc_channel_absmax(const uint16_t* X, int M, int K, float* absmax) {
  for (int m = 0; m < M; ++m)
    for (int c = 0; c < K; ++c) {
      float a = fabsf(orc_f32_from_f16(X[(size_t)m * K + c]));
      if (a > absmax[c]) absmax[c] = a;
    }
}

static int cmp_float_asc(const void* a, const void* b) {
  float x = *(const float*)a, y = *(const float*)b;
  return (x > y) - (x < y);
}

/* Ranking order: larger absmax first, equal values by smaller channel index. */
static const float* g_rank_key;
static int cmp_rank(const void* a, const void* b) {
  int i = *(const int32_t*)a, j = *(const int32_t*)b;
  float x = g_rank_key[i], y = g_rank_key[j];
  if (x != y) return x > y ? -1 : 1;
  return (i > j) - (i < j);
}

int orc_plan_channel_perm(const float* absmax, int K, int G, float outlier_ratio,
                          float max_frac8, int32_t* perm, uint8_t* prec, int* n_outliers) {
  if (K <= 0 || G <= 0 || K % G) return -1;
  if (!(max_frac8 >= 0.0f && max_frac8 <= 1.0f) || isnan(outlier_ratio)) return -1;
  for (int c = 0; c < K; ++c)
    if (!(absmax[c] >= 0.0f) || isinf(absmax[c])) return -1;
  const int NG = K / G;

  /* Lower median of the per-channel maxima. */
  float* sorted = (float*)malloc(sizeof(float) * (size_t)K);
  int32_t* rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
  unsigned char* taken = (unsigned char*)calloc((size_t)K, 1);
  if (!sorted || !rank || !taken) {
    free(sorted);
    free(rank);
    free(taken);
    return -1;
  }
  memcpy(sorted, absmax, sizeof(float) * (size_t)K);
  qsort(sorted, (size_t)K, sizeof(float), cmp_float_asc);
  double median = (double)sorted[(K - 1) / 2];

  /* Outlier channels: maxima above ratio x median (every channel if ratio <= 0). */
  int nout = 0;
  if (outlier_ratio <= 0.0f) {
    nout = K;
  } else {
    double thr = (double)outlier_ratio * median;
    for (int c = 0; c < K; ++c)
      if ((double)absmax[c] > thr) ++nout;
  }

  /* 8-bit blocks: enough to hold every outlier, at most a fraction of all blocks. */
  int need = (nout + G - 1) / G;
  int cap = (int)floor((double)max_frac8 * (double)NG);
  int n8 = need < cap ? need : cap;

  /* The n8*G highest-ranked channels fill the 8-bit blocks in rank order.
   * Every other position keeps its own channel, except the positions those
   * channels left: they take the channels displaced from the 8-bit blocks,
   * in ascending order on both sides. */
  for (int c = 0; c < K; ++c) rank[c] = c;
  g_rank_key = absmax;
  qsort(rank, (size_t)K, sizeof(int32_t), cmp_rank);
  const int head = n8 * G;
  for (int i = 0; i < head; ++i) {
    perm[i] = rank[i];
    taken[rank[i]] = 1;
  }
  int next_displaced = 0;
  for (int p = head; p < K; ++p) {
    if (!taken[p]) {
      perm[p] = p;
      continue;
    }
    while (taken[next_displaced]) ++next_displaced; /* a head channel not in the head set */
    perm[p] = next_displaced++;
  }
  for (int g = 0; g < NG; ++g) prec[g] = g < n8 ? 8 : 4;
  if (n_outliers) *n_outliers = nout;
  free(sorted);
  free(rank);
  free(taken);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* KV4: asymmetric 4-bit group quantization of the KV cache (Sec. 3.2, and    */
/* the setup of Sec. 6).  A group is G consecutive channels of one token's K  */
/* or V vector.  Per group: mn = min x, s = fp16(fp32(max x - mn) / 15),      */
/* q = clamp(rint(fp32(fp32(x - mn) / s)), 0, 15) (q = 0 when s == 0);        */
/* reconstruction x' = fp16(fp32(fp32(q * s) + mn)).                          */
/* codes: [T][C/2] bytes, channel 2j in the low nibble of byte j, 2j+1 in the */
/* high nibble; params: fp16 [T][C/G][2] = {s, mn}.                           */
/* ------------------------------------------------------------------------- */

int orc_kv4_quantize(const uint16_t* X, int T, int C, int G, uint8_t* codes, uint16_t* params) {
  if (T < 0 || C <= 0 || G <= 0 || G % 2 || C % G) return -1;
  const int NG = C / G;
  for (int t = 0; t < T; ++t)
    for (int g = 0; g < NG; ++g) {
      const uint16_t* x16 = X + (size_t)t * C + (size_t)g * G;
      float mn = orc_f32_from_f16(x16[0]), mx = mn;
      for (int c = 0; c < G; ++c) {
        float v = orc_f32_from_f16(x16[c]);
        if (!isfinite(v)) return -1;
        if (v < mn) mn = v;
        if (v > mx) mx = v;
      }
      /* zero extremes as +0, whatever the signs of the zeros (min and max of
       * +0 and -0 are value ties) */
      if (mn == 0.0f) mn = 0.0f;
      if (mx == 0.0f) mx = 0.0f;
      float range = mx - mn;
      uint16_t s16 = orc_f16_from_f32(range / 15.0f);
      float s = orc_f32_from_f16(s16);
      uint8_t* out = codes + (size_t)t * (C / 2) + (size_t)g * (G / 2);
      for (int c = 0; c < G; c += 2) {
        unsigned q2[2];
        for (int i = 0; i < 2; ++i) {
          float r = 0.0f;
          if (s != 0.0f) {
            float d = orc_f32_from_f16(x16[c + i]) - mn;
            r = rintf(d / s);
            if (r > 15.0f) r = 15.0f;
            if (r < 0.0f) r = 0.0f;
          }
          q2[i] = (unsigned)r;
        }
        out[c / 2] = (uint8_t)(q2[0] | (q2[1] << 4));
      }
      uint16_t* p = params + ((size_t)t * NG + g) * 2;
      p[0] = s16;
      p[1] = orc_f16_from_f32(mn); /* mn is an input value: exact in fp16 */
    }
  return 0;
}

int orc_kv4_dequantize(const uint8_t* codes, const uint16_t* params, int T, int C, int G,
                       uint16_t* out) {
  if (T < 0 || C <= 0 || G <= 0 || G % 2 || C % G) return -1;
  const int NG = C / G;
  for (int t = 0; t < T; ++t)
    for (int c = 0; c < C; ++c) {
      const uint16_t* p = params + ((size_t)t * NG + c / G) * 2;
      float s = orc_f32_from_f16(p[0]);
      float mn = orc_f32_from_f16(p[1]);
      uint8_t b = codes[(size_t)t * (C / 2) + c / 2];
      unsigned q = (c & 1) ? (unsigned)(b >> 4) : (unsigned)(b & 15);
      float prod = (float)q * s;
      out[(size_t)t * C + c] = orc_f16_from_f32(prod + mn);
    }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* SwiGLU and the next layer's quantization (the step after the path: the    */
/* gate/up GEMM's output becomes the down projection's input, h = SiLU(gate) */
/* * up, quantized by FMPQ in 128-channel blocks, Sec. 3.2).                 */
/*                                                                           */
/* exp is written out so that a GPU kernel can follow the same fp32 steps:   */
/* Cody-Waite reduction x = k ln2 + r with k = rint(x log2 e) and ln2 split  */
/* into a 24-bit-exact high part and a low part, exp(r) by its Taylor series */
/* to degree 7 in Horner form, then the exact scaling by 2^k.  The input is  */
/* clamped to [-87, 88], which keeps k within the normal exponent range.     */
/* ------------------------------------------------------------------------- */

float orc_exp_f32(float x) {
  if (x > 88.0f) x = 88.0f;
  if (x < -87.0f) x = -87.0f;
  const float log2e = 1.44269504088896341f;
  const float ln2_hi = 0.693145751953125f;     /* 0x3F317200: 16 significant bits */
  const float ln2_lo = 1.42860682030941723e-6f; /* ln 2 - ln2_hi */
  const float k = rintf(x * log2e);
  float r = fmaf(-k, ln2_hi, x);
  r = fmaf(-k, ln2_lo, r);
  /* 1/n! for n = 7 .. 0 */
  const float c[8] = {1.98412698412698413e-4f, 1.38888888888888889e-3f,
                      8.33333333333333333e-3f, 4.16666666666666667e-2f,
                      1.66666666666666667e-1f, 0.5f, 1.0f, 1.0f};
  float p = c[0];
  for (int i = 1; i < 8; ++i) p = fmaf(p, r, c[i]);
  return ldexpf(p, (int)k);
}

float orc_silu_f32(float x) { return x * (1.0f / (1.0f + orc_exp_f32(-x))); }

/* h = fp16(SiLU(g) * u) for fp16 g, u. */
uint16_t orc_swiglu_f16(uint16_t g, uint16_t u) {
  return orc_f16_from_f32(orc_silu_f32(orc_f32_from_f16(g)) * orc_f32_from_f16(u));
}

int orc_swiglu_quantize(const uint16_t* gu, int M, int I, int G, const uint8_t* prec,
                        uint8_t* A_packed, uint16_t* sa16, int nthreads) {
  if (M < 0 || I <= 0 || G <= 0 || I % G || G > 1024) return -1;
  uint16_t* h = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)M * (size_t)I);
  int8_t* q = (int8_t*)malloc((size_t)M * (size_t)I);
  if (!h || !q) {
    free(h);
    free(q);
    return -1;
  }
  /* gate/up columns come in 2G-wide groups: gate of channels jG..jG+G-1, then
   * up of the same channels */
  for (int m = 0; m < M; ++m)
    for (int c = 0; c < I; ++c) {
      const int j = c / G, i = c % G;
      const uint16_t g = gu[(size_t)m * 2 * I + (size_t)j * 2 * G + i];
      const uint16_t u = gu[(size_t)m * 2 * I + (size_t)j * 2 * G + G + i];
      h[(size_t)m * I + c] = orc_swiglu_f16(g, u);
    }
  int rc = orc_quantize_act(h, prec, M, I, G, q, sa16, nthreads);
  if (!rc) rc = orc_pack_act(q, prec, M, I, G, A_packed);
  free(h);
  free(q);
  return rc;
}
