/*
 * oracle.h -- CPU oracle for the COMET W4Ax path (FMPQ quantization + W4Ax GEMM).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, obviously correct
 * definition that the GPU path is checked against.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it.  It shares
 * no code, header, table or helper with the GPU library, and the GPU library
 * never calls it.
 *
 * Paper: "COMET: Towards Practical W4A4KV4 LLMs Serving" (arXiv 2410.12168).
 *   - Activations are split along the channel dimension only, into blocks of
 *     k = 128 channels; each block is quantized to 4 or 8 bits (Sec. 3.2).
 *   - The kernel computes O = WX with W4A4 and W4A8 tiles, integer products
 *     and dequantization by the scale factors (Sec. 4.1, 4.3, Sec. 5).
 *
 * Readings where the paper is silent (all listed with reasons in the design
 * notes of the repository):
 *   - symmetric quantization, restricted range [-qmax, qmax], qmax = 7 / 127;
 *   - one fp16 scale per (token, block) for activations and per
 *     (output channel, block) for weights; s = fp16(amax / qmax) computed by an
 *     IEEE fp32 division and rounded to nearest-even into binary16;
 *   - codes q = clamp(rint_half_even(fp32(x / s)), -qmax, qmax); s == 0 gives
 *     all-zero codes;
 *   - int32 products per block, fp64 dequantized sum over blocks.
 *
 * Byte encodings (the storage contract shared with the GPU library's header):
 *   4-bit code of q: sign bit s = (q < 0), magnitude m = |q| (0..7).
 *   A 4-bit chunk holds the G codes of one row and one block in G/2 bytes.
 *   For dword j (bytes 4j..4j+3) and byte k (0..3) of that dword:
 *       bit 7    : s[8j+k]
 *       bits 6..4: m[8j+4+k]
 *       bit 3    : s[8j+4+((k+3) mod 4)]
 *       bits 2..0: m[8j+k]
 *   An 8-bit chunk holds G bytes, byte c = (s[c] << 7) | m[c], m = 0..127.
 *   A_packed: block-major.  Block g starts at byte M * sum_{g'<g} B(p[g']),
 *             B(4) = G/2, B(8) = G; row m of block g follows at + m * B(p[g]).
 *   W_packed: 16-row panels, N a multiple of 16: row n, block g at byte
 *             ((n/16 * K/G + g) * 16 + n % 16) * G/2, so the 16 rows of a panel
 *             hold each block in 16*G/2 contiguous bytes.
 *   a_scales: fp16 [K/G][M]; w_scales: fp16 [K/G][N].
 */
#ifndef COMET_ORACLE_H
#define COMET_ORACLE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* IEEE 754 binary16 <-> binary32, round to nearest even, subnormals kept. */
uint16_t orc_f16_from_f32(float x);
float orc_f32_from_f16(uint16_t h);
void orc_f16_from_f32_array(const float* x, uint16_t* h, size_t n);
void orc_f32_from_f16_array(const uint16_t* h, float* x, size_t n);

/* Quantize one block of G fp32 values to b-bit codes (b = 4 or 8).
 * Returns 0, or -1 for a non-finite input or a bad argument. */
int orc_quantize_group(const float* v, int G, int bits, uint16_t* s16, int8_t* q);

/* FMPQ activation quantization.  X fp16 [M][K]; prec[K/G] in {4, 8}.
 * Outputs qa int8 [M][K] and sa16 fp16 [K/G][M].  Returns 0 or -1. */
int orc_quantize_act(const uint16_t* X, const uint8_t* prec, int M, int K, int G,
                     int8_t* qa, uint16_t* sa16, int nthreads);

/* 4-bit weight quantization.  W fp16 [N][K] -> qw int8 [N][K], sw16 fp16 [K/G][N]. */
int orc_quantize_weight(const uint16_t* W, int N, int K, int G, int8_t* qw, uint16_t* sw16,
                        int nthreads);

/* Byte encodings (see above). */
size_t orc_act_packed_bytes(const uint8_t* prec, int M, int K, int G);
void orc_encode4(const int8_t* q, int G, uint8_t* out); /* one 4-bit chunk, G/2 bytes */
void orc_encode8(const int8_t* q, int G, uint8_t* out); /* one 8-bit chunk, G bytes  */
int orc_pack_act(const int8_t* qa, const uint8_t* prec, int M, int K, int G, uint8_t* A_packed);
int orc_pack_weight(const int8_t* qw, int N, int K, int G, uint8_t* W_packed);

/* Per-block integer contraction acc[m][n][g] = sum_{c<G} qa[m][gG+c] * qw[n][gG+c]. */
void orc_group_acc(const int8_t* qa, const int8_t* qw, int M, int N, int K, int G, int32_t* acc);

/* ref[m][n] = sum_g acc[m][n][g] * sa[g][m] * sw[g][n], accumulated in fp64.
 * Rows rows[0..nrows) of the output are computed (rows == NULL: all M rows, nrows = M);
 * ref is [nrows][N]. */
void orc_dequant_gemm(const int8_t* qa, const uint16_t* sa16, const int8_t* qw,
                      const uint16_t* sw16, int M, int N, int K, int G, const int* rows,
                      int nrows, double* ref, int nthreads);

/* Unquantized reference exact[m][n] = sum_k X[m][k] * W[n][k] in fp64 (diagnostic). */
void orc_exact_gemm(const uint16_t* X, const uint16_t* W, int M, int N, int K, double* exact,
                    int nthreads);

/* Channel permutation and calibration map (Sec. 3.2).
 * orc_permute_columns: out[r][c] = X[r][perm[c]] for R rows of K fp16 values;
 *   -1 if an index is outside [0, K).
 * orc_channel_absmax: absmax[c] = max(absmax[c], max_m |X[m][c]|) (fp32,
 *   accumulating over calls; start from zeros).
 * orc_plan_channel_perm: from per-channel maxima, the lower median med (rank
 *   (K-1)/2 ascending) gives the outlier channels, absmax > ratio * med
 *   (compared in fp64; every channel if ratio <= 0).  The number of 8-bit
 *   blocks is n8 = min(ceil(n_out / G), floor(max_frac8 * K/G)).  Channels are
 *   ranked by absmax descending, ties by index; perm[0 .. n8*G) holds the first
 *   n8*G ranked channels in rank order.  For p >= n8*G, perm[p] = p unless
 *   channel p moved into the 8-bit blocks; those positions take the channels
 *   displaced from positions [0, n8*G) (the ones not ranked in), ascending
 *   channel to ascending position.  prec[g] = 8 for g < n8, else 4.  Returns
 *   0, or -1 for bad arguments (max_frac8 outside [0, 1], a negative or
 *   non-finite maximum). */
int orc_permute_columns(const uint16_t* X, const int32_t* perm, int R, int K, uint16_t* out);
void orc_channel_absmax(const uint16_t* X, int M, int K, float* absmax);
int orc_plan_channel_perm(const float* absmax, int K, int G, float outlier_ratio,
                          float max_frac8, int32_t* perm, uint8_t* prec, int* n_outliers);

/* KV4: asymmetric 4-bit group quantization of K/V rows (Sec. 3.2; Sec. 6 setup).
 * X fp16 [T][C], groups of G consecutive channels (G even, C % G == 0).
 *   mn = min, mx = max (zero extremes as +0), s = fp16(fp32(mx - mn) / 15),
 *   q = clamp(rint(fp32(fp32(x - mn) / s)), 0, 15)
 *   (all zero when s == 0).  codes [T][C/2]: channel 2j low nibble of byte j,
 *   2j+1 high nibble.  params fp16 [T][C/G][2] = {s, mn}.
 * Dequantization: x' = fp16(fp32(q * s) + mn).  Return 0, or -1 for bad
 * arguments or a non-finite input. */
int orc_kv4_quantize(const uint16_t* X, int T, int C, int G, uint8_t* codes, uint16_t* params);
int orc_kv4_dequantize(const uint8_t* codes, const uint16_t* params, int T, int C, int G,
                       uint16_t* out);

/* SwiGLU and next-layer quantization (the step after the W4Ax GEMM).
 * orc_exp_f32: exp by Cody-Waite reduction (k = rint(x log2e), r = x - k ln2
 *   with ln2 split in two, fmas), Taylor series to degree 7 in Horner form
 *   (fmas), ldexp by k; input clamped to [-87, 88].
 * orc_silu_f32(x) = x * (1 / (1 + orc_exp_f32(-x))), each an fp32 operation.
 * orc_swiglu_f16(g, u) = fp16(orc_silu_f32(g) * u).
 * orc_swiglu_quantize: gu fp16 [M][2I] whose columns come in 2G-wide groups
 *   (gate of channels jG .. jG+G-1, then up of the same channels); h [M][I] =
 *   swiglu(gate, up), then FMPQ quantization and packing of h with map prec
 *   [I/G] into A_packed / sa16 [I/G][M] (as orc_quantize_act + orc_pack_act). */
float orc_exp_f32(float x);
float orc_silu_f32(float x);
uint16_t orc_swiglu_f16(uint16_t g, uint16_t u);
int orc_swiglu_quantize(const uint16_t* gu, int M, int I, int G, const uint8_t* prec,
                        uint8_t* A_packed, uint16_t* sa16, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
