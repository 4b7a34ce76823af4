/*
 * comet.h -- C ABI of libcomet, an MI355X (gfx950) implementation of the hot
 * path of COMET (arXiv 2410.12168): FMPQ activation quantization and the W4Ax
 * mixed-precision GEMM.
 *
 * The method (paper, Sec. 3.2 and Sec. 4):
 *   - activations are split along the channel dimension only, into blocks of
 *     G = 128 channels; each block is stored as 4-bit or 8-bit codes with one
 *     scale per (token, block); weights are 4-bit with one scale per
 *     (output channel, block);
 *   - the GEMM contracts the codes block by block with exact integer products,
 *     dequantizes each block's result by its two scales and sums the blocks
 *     (Sec. 4.1; the product O = WX of Sec. 5 is out = X W^T here).
 *
 * Numbers and encodings (identical, byte for byte, to the CPU oracle):
 *   - fp16 buffers hold IEEE binary16 bit patterns (uint16_t).
 *   - Block quantizer: s = fp16_rne(fp32(amax / qmax)), qmax = 7 (4-bit) or
 *     127 (8-bit); code q = clamp(rint_even(fp32(x / s)), -qmax, qmax);
 *     s == 0 gives all-zero codes.  Codes -8 / -128 are never produced.
 *   - A code is stored sign-magnitude.  4-bit chunk (one row, one block,
 *     G/2 = 64 bytes): for dword j and byte k (0..3) of that dword
 *         bit 7 = sign of code 8j+k,        bits 6..4 = |code 8j+4+k|,
 *         bit 3 = sign of code 8j+4+((k+3)%4), bits 2..0 = |code 8j+k|.
 *     With this layout (dword & 0x87878787) and (rotr(dword, 4) & 0x87878787)
 *     are the OCP FP8-E4M3 encodings of codes 8j..8j+3 and 8j+4..8j+7 times
 *     2^-9 (the paper's "location switch" of Sec. 4.3, re-derived so that the
 *     int4 -> MFMA-operand conversion is two masks and one rotate).
 *     8-bit chunk (G = 128 bytes): byte c = (sign << 7) | |code c|.
 *   - A_packed: block-major.  Block g starts at byte M * sum_{g'<g} B(p[g']),
 *     B(4) = 64, B(8) = 128; row m of block g follows at + m * B(p[g]).
 *   - a_scales: fp16 [K/G][M];  w_scales: fp16 [K/G][N];  out: fp16 [M][N]
 *     row-major.
 *   - W_packed: N*K/2 bytes in 16-row panels (N a multiple of 16): row n's
 *     block g at byte ((n/16 * K/G + g) * 16 + n % 16) * 64, so the 16 rows of
 *     a panel hold each block in one contiguous kilobyte (Sec. 4.3: a weight
 *     layout made for the kernel's loads).
 *
 * Conventions for every call:
 *   - Device pointers are caller-owned HIP device allocations on the current
 *     device; the library never frees or retains them.  Work is enqueued on
 *     `stream` (0 = null stream) and returns immediately; the caller keeps the
 *     buffers alive until the stream has finished.
 *   - group_prec_map is a HOST array of K/G bytes, each 4 or 8 (the block
 *     precisions chosen offline by data sampling, Sec. 3.2).  It is read
 *     during the call and not retained.
 *   - Every argument is checked before anything is enqueued; on an error
 *     nothing is launched and comet_last_error() says why.
 *       COMET_ERR_INVALID_ARG : null pointer, M/N/K < 1, K % G != 0,
 *                               N % 16 != 0 (GEMM), device pointer not 16-byte
 *                               aligned, map entry not in {4, 8}, bad window.
 *       COMET_ERR_UNSUPPORTED : G != 128 (the paper's k = 128), K > 65536,
 *                               or a current device that is not gfx950.
 *       COMET_ERR_HIP         : a HIP runtime or launch error.
 *       COMET_ERR_OOM         : the library could not allocate its workspace.
 *   - Faults inside kernels surface at the caller's next synchronisation.
 *   - Calls on different streams may run concurrently.  The GEMM's split-tile
 *     workspace is owned by the library, one per device and stream.
 *   - The 128- and 256-row tile kernels run from a schedule (plan) that the
 *     library builds on the host and uploads on the first call for each
 *     (device, M, N, K, map, mode): that call allocates a few KB of device
 *     memory and enqueues the upload on its stream, ahead of the kernel (the
 *     host does not wait for it).  Plans stay cached until
 *     comet_release_caches(), so the cache grows with every distinct shape;
 *     the few-token kernels (small M) need no plan.
 *   - The environment variable COMET_SCHED selects the schedule mode (Sec.
 *     4.4, read at every call): "cost" (default: precision-batched K order,
 *     data-parallel full waves of tiles, the last wave split by cost),
 *     "dp" (precision-batched order, whole tiles only) or "natural" (the
 *     map's own K order, whole tiles only: no tile remapping and no tile
 *     decomposition; the fused SwiGLU entry point takes "dp" instead).
 *     Results do not depend on the mode beyond the fp32 summation order.
 */
#ifndef COMET_H
#define COMET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define COMET_API __attribute__((visibility("default")))
#else
#define COMET_API
#endif

typedef struct ihipStream_t* hipStream_t;

/* GEMM kernels (comet_gemm_kernel). */
typedef enum {
  COMET_KERNEL_FEW_TOKEN = 0,         /* one wave per 16 columns and split-K slot */
  COMET_KERNEL_FEW_TOKEN_SHARED = 1,  /* the same, activations shared through LDS */
  COMET_KERNEL_MID = 2,               /* 128-row tiles */
  COMET_KERNEL_TILE = 3,              /* 256-row tiles */
  COMET_KERNEL_STREAM = 4             /* up to 64 rows, weight panels divided evenly over the CUs */
} comet_kernel_t;

typedef enum {
  COMET_OK = 0,
  COMET_ERR_INVALID_ARG = 1,
  COMET_ERR_UNSUPPORTED = 2,
  COMET_ERR_HIP = 3,
  COMET_ERR_OOM = 4
} comet_status_t;

/* Bytes of A_packed for M tokens, K channels, block size G and the given map
 * (M * sum_g B(p[g])).  Returns 0 for invalid arguments. */
COMET_API size_t comet_act_packed_bytes(const uint8_t* group_prec_map, int M, int K, int G);

/* Online FMPQ activation quantization (Sec. 3.2): for every token m and block
 * g, quantize X[m, gG:(g+1)G] to p[g] bits and write the codes to A_packed and
 * the scale to a_scales[g][m].
 *   X        device, fp16 [M][K] row-major, 16-byte aligned.
 *   A_packed device, comet_act_packed_bytes(...) bytes, 16-byte aligned.
 *   a_scales device, fp16 [K/G][M].
 * M may be at most 2,097,120 (COMET_ERR_UNSUPPORTED beyond).
 * Non-finite inputs are not supported (the codes they produce are unspecified). */
COMET_API comet_status_t comet_fmpq_quantize_act(const uint16_t* X, const uint8_t* group_prec_map,
                                       uint8_t* A_packed, uint16_t* a_scales, int M, int K,
                                       int G, hipStream_t stream);

/* Offline 4-bit weight quantization and packing (weights are 4-bit, Sec. 3.2;
 * stored in the operand layout the GEMM reads, Sec. 4.3).
 *   W        device, fp16 [N][K] row-major (nn.Linear layout); N a multiple of 16.
 *   W_packed device, N*K/2 bytes in 16-row panels (see above).
 *   w_scales device, fp16 [K/G][N]. */
COMET_API comet_status_t comet_pack_w4(const uint16_t* W, uint8_t* W_packed, uint16_t* w_scales, int N,
                             int K, int G, hipStream_t stream);

/* Channel permutation (Sec. 3.2): outlier channels are gathered into a few
 * blocks so that only those need 8 bits; the weight columns take the same
 * permutation, so out = X W^T is unchanged up to quantization.
 *
 * Same as comet_fmpq_quantize_act, on the permuted activations: block g of
 * row m quantizes X[m][perm[gG + c]], c < G.  perm is a DEVICE int32 [K]
 * array, 16-byte aligned, normally a permutation of 0..K-1 (repeated entries
 * are gathered as written; an entry outside [0, K), negative ones included,
 * reads channel K-1, so no read leaves the row).  perm == NULL: no
 * permutation (identical to comet_fmpq_quantize_act).  Other arguments and
 * errors as there. */
COMET_API comet_status_t comet_fmpq_quantize_act_perm(const uint16_t* X, const int32_t* perm,
                                                      const uint8_t* group_prec_map,
                                                      uint8_t* A_packed, uint16_t* a_scales,
                                                      int M, int K, int G, hipStream_t stream);

/* comet_pack_w4 on the column-permuted weights W[n][perm[k]] (Sec. 3.2, the
 * matching permutation of the weight matrix).  perm as above; NULL = none. */
COMET_API comet_status_t comet_pack_w4_perm(const uint16_t* W, const int32_t* perm,
                                            uint8_t* W_packed, uint16_t* w_scales, int N, int K,
                                            int G, hipStream_t stream);

/* Data sampling for the calibration (Sec. 3.2): absmax[c] = max(absmax[c],
 * max_m |X[m][c]|) over the M rows of X (device, fp16 [M][K], 16-byte
 * aligned, K a multiple of 8).  absmax is a device fp32 [K] array, 4-byte
 * aligned, that the call ACCUMULATES into: start it at zeros and call once
 * per calibration batch.  It must hold non-negative values (the merge is an
 * unsigned compare of the bit patterns).  Bit-exact: max is order-free.
 * Non-finite inputs are not supported. */
COMET_API comet_status_t comet_channel_absmax(const uint16_t* X, float* absmax, int M, int K,
                                              hipStream_t stream);

/* Host-only calibration map (Sec. 3.2; nothing is launched).  From the
 * per-channel maxima absmax[K] (host), with med the lower median (rank
 * (K-1)/2 ascending):
 *   outlier channels: absmax > outlier_ratio * med, compared in fp64
 *                     (every channel when outlier_ratio <= 0);
 *   n8 = min(ceil(n_out / G), floor(max_frac_8bit * K/G)) 8-bit blocks;
 *   perm (host int32 [K]): positions [0, n8*G) hold the n8*G channels with
 *        the largest maxima (ties by index) in that order; a later position p
 *        holds channel p unless channel p moved up, and those positions hold
 *        the channels displaced from [0, n8*G), ascending to ascending (few
 *        channels move, which keeps the fused gather cheap);
 *   group_prec_map (host uint8 [K/G]): 8 for g < n8, else 4;
 *   *n_outliers (may be NULL): n_out.
 * G is any positive divisor of K here (the GEMM needs 128).  Errors:
 * COMET_ERR_INVALID_ARG for null pointers, K % G != 0, max_frac_8bit outside
 * [0, 1], a NaN ratio or a negative / non-finite maximum. */
COMET_API comet_status_t comet_plan_channel_perm(const float* absmax, int K, int G,
                                                 float outlier_ratio, float max_frac_8bit,
                                                 int32_t* perm, uint8_t* group_prec_map,
                                                 int* n_outliers);

/* KV4: 4-bit asymmetric group quantization of K/V cache rows (Sec. 3.2: the
 * KV cache is quantized to 4 bits channel-wise; Sec. 6 setup: asymmetric
 * INT4 groups).  X: device fp16 [T][C] (C = KV heads x head_dim), 16-byte
 * aligned; groups of G in {32, 64, 128} consecutive channels, C % G == 0.
 * Per group: mn = min x, mx = max x (zero extremes as +0), s = fp16(fp32(mx - mn) / 15),
 * q = clamp(rint(fp32(fp32(x - mn) / s)), 0, 15) (all 0 when s == 0).
 *   codes  device [T][C/2] bytes, 4-byte aligned: channel 2j in the low
 *          nibble of byte j, 2j+1 in the high nibble;
 *   params device fp16 [T][C/G][2] = {s, mn}, 4-byte aligned.
 * Bit-exact with the definition above.  Non-finite inputs are not supported. */
COMET_API comet_status_t comet_kv4_quantize(const uint16_t* X, uint8_t* codes, uint16_t* params,
                                            int T, int C, int G, hipStream_t stream);

/* Inverse of comet_kv4_quantize: out[t][c] = fp16(fp32(q * s) + mn) (device
 * fp16 [T][C], 16-byte aligned); the other arguments as there. */
COMET_API comet_status_t comet_kv4_dequantize(const uint8_t* codes, const uint16_t* params,
                                              uint16_t* out, int T, int C, int G,
                                              hipStream_t stream);

/* W4Ax GEMM (Sec. 4, O = WX): out[m][n] = fp16( sum_g a_scales[g][m] *
 * w_scales[g][n] * sum_{c<G} qa[m][gG+c] * qw[n][gG+c] ).  The per-block sums
 * are exact; the sum over blocks is fp32 in an unspecified order, rounded once
 * to fp16 (nearest even).  Output is deterministic for a given build, device,
 * shape and map.  N must be a multiple of 16; M at most 2,097,120 (larger M:
 * COMET_ERR_UNSUPPORTED). */
COMET_API comet_status_t comet_w4ax_gemm(const uint8_t* A_packed, const uint8_t* group_prec_map,
                               const uint16_t* a_scales, const uint8_t* W_packed,
                               const uint16_t* w_scales, uint16_t* out, int M, int N, int K,
                               int G, hipStream_t stream);

/* comet_w4ax_gemm for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results and errors; in addition:
 *   - the library's device memory for this call (the tile kernels' schedule,
 *     split-tile fp32 partials and arrival counters) is one static array per
 *     device of 66 MiB + 64 KiB, held until the process ends; the call makes
 *     no hipMalloc, hipFree or other allocating call;
 *   - every call on a device shares that array: calls that overlap on one
 *     device (e.g. on two streams) race and must not be issued;
 *   - a schedule that would split tiles into more partials than the array
 *     holds (64 MiB) runs with whole tiles instead (same results within the
 *     fp32 summation order); a schedule larger than 2 MiB (about 87,000
 *     output tiles) is refused with COMET_ERR_UNSUPPORTED;
 *   - the first call after the schedule changes (a new shape, map or mode)
 *     copies the schedule from host memory and waits for the copy; calls that
 *     repeat the previous shape only enqueue kernels. */
COMET_API comet_status_t comet_w4ax_gemm_noalloc(const uint8_t* A_packed,
                                                 const uint8_t* group_prec_map,
                                                 const uint16_t* a_scales,
                                                 const uint8_t* W_packed,
                                                 const uint16_t* w_scales, uint16_t* out, int M,
                                                 int N, int K, int G, hipStream_t stream);

/* SwiGLU and the next layer's quantization, fused into the W4Ax GEMM (the step
 * after the path: in a LLaMA MLP the gate/up GEMM's output feeds the down
 * projection through h = SiLU(gate) * up, whose activations FMPQ quantizes in
 * 128-channel blocks, Sec. 3.2).  The GEMM is comet_w4ax_gemm's, but instead
 * of storing its fp16 output the call writes the down projection's quantized
 * input:
 *   - the weight rows (output columns) come in 2G = 256-wide groups: rows
 *     256 j .. 256 j + 127 are the gate rows and 256 j + 128 .. 256 j + 255
 *     the up rows of channels 128 j .. 128 j + 127 (a caller interleaves W_gate
 *     and W_up this way before comet_pack_w4); N = 2 I, a multiple of 256;
 *   - with g, u the fp16-rounded GEMM outputs, h = fp16(SiLU(g) * u) where
 *     SiLU(x) = x * (1 / (1 + exp(-x))) and exp follows fixed fp32 steps
 *     (x clamped to [-87, 88]; k = rint(x log2 e); r = x - k ln2 by two fmas
 *     with ln2 = 0.693145751953125 + 1.42860682030941723e-6; the Taylor series
 *     of e^r to degree 7 in Horner form by fmas; ldexp(., k));
 *   - h [M][I] is quantized with out_prec (host, I/G entries of 4 or 8) into
 *     out_A_packed (device, comet_act_packed_bytes(out_prec, M, I, G) bytes)
 *     and out_a_scales (device, fp16 [I/G][M]), exactly as
 *     comet_fmpq_quantize_act would quantize h.
 * A channel permutation for the down projection needs no runtime step here:
 * permute the gate and up rows (and the down projection's weight columns,
 * comet_pack_w4_perm) offline.  Other arguments and errors as comet_w4ax_gemm;
 * M at most 2,097,120.  The epilogue fusion runs with the 128-row tile kernel
 * (comet_gemm_kernel() == COMET_KERNEL_MID); with the other kernels the GEMM
 * writes its fp16 output to a library-owned workspace (M * N * 2 bytes, per
 * device and stream, kept until comet_release_caches) that the SwiGLU
 * quantizer of comet_swiglu_quantize then reads, because that pair is faster
 * there. */
COMET_API comet_status_t comet_w4ax_gemm_swiglu_quant(
    const uint8_t* A_packed, const uint8_t* group_prec_map, const uint16_t* a_scales,
    const uint8_t* W_packed, const uint16_t* w_scales, int M, int N, int K, int G,
    const uint8_t* out_prec_map, uint8_t* out_A_packed, uint16_t* out_a_scales,
    hipStream_t stream);

/* The same SwiGLU and quantization on an fp16 gate/up output gu (device,
 * [M][2I] with the 256-wide gate/up column groups above, 16-byte aligned),
 * written to out_A_packed / out_a_scales as above.  I a multiple of G = 128;
 * M at most 2,097,120. */
COMET_API comet_status_t comet_swiglu_quantize(const uint16_t* gu, const uint8_t* out_prec_map,
                                               uint8_t* out_A_packed, uint16_t* out_a_scales,
                                               int M, int I, int G, hipStream_t stream);

/* Diagnostic form of the same contraction: writes the exact per-block integer
 * sums acc[m - m0][n - n0][g] = sum_{c<G} qa[m][gG+c] * qw[n][gG+c] (int32)
 * for the window m0 <= m < m1, n0 <= n < n1, computed by the GEMM's own
 * operand path (Sec. 4.1, the integer tile results before dequantization).
 *   acc device, int32 [m1-m0][n1-n0][K/G]. */
COMET_API comet_status_t comet_w4ax_gemm_acc(const uint8_t* A_packed, const uint8_t* group_prec_map,
                                   const uint16_t* a_scales, const uint8_t* W_packed,
                                   const uint16_t* w_scales, int32_t* acc, int M, int N, int K,
                                   int G, int m0, int m1, int n0, int n1, hipStream_t stream);

/* Host-only view of the per-block-precision tile schedule (Sec. 4.4: tile
 * remapping and tile decomposition) that comet_w4ax_gemm would use for this
 * shape and map on `num_cus` compute units.  Nothing is launched and no device
 * is touched.  Each work unit is five ints {tile, g_begin, g_end, slot, nslots}:
 * output tile `tile` (row-major over the tile grid), blocks [g_begin, g_end)
 * in the schedule's block order, written as partial `slot` of `nslots`
 * (nslots == 1: the unit owns the whole tile).  Units are listed per
 * persistent workgroup: wg_begin[w] .. wg_begin[w+1].  Returns the number of
 * units and workgroups through *n_units / *n_wgs; arrays may be NULL to query
 * sizes.  order (may be NULL) receives the K/G block order. */
COMET_API comet_status_t comet_schedule_query(int M, int N, int K, int G, const uint8_t* group_prec_map,
                                    int num_cus, int* units, int max_units, int* n_units,
                                    int* wg_begin, int max_wgs, int* n_wgs, int* order,
                                    int* tile_m, int* tile_n);

/* Host-only: which GEMM kernel (comet_kernel_t) comet_w4ax_gemm runs for this
 * shape on a device with `num_cus` compute units, or -1 for invalid
 * arguments (comet_last_error() says why).  Nothing is launched. */
COMET_API int comet_gemm_kernel(int M, int N, int K, int G, int num_cus);

/* SHA-256 (64 hex digits) of the sources and build flags the library was
 * built from; the same string follows "COMET_SOURCE_STAMP=" in the library
 * file, so a loader can compare it with its source tree before loading. */
COMET_API const char* comet_build_stamp(void);

COMET_API const char* comet_status_str(comet_status_t status);

/* Message for the last error on the calling thread ("" if none). */
COMET_API const char* comet_last_error(void);

/* Free the library's cached plans and workspaces on every device.  Not to be
 * called while work the library enqueued is still running. */
COMET_API void comet_release_caches(void);

#ifdef __cplusplus
}
#endif
#endif
