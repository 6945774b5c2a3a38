/*
 * mxfp4.h -- C ABI of libmxfp4.so, the MXFP4 backward-pass hot path of
 * "Training LLMs with MXFP4" (Tseng, Yu, Park, AISTATS 2025) on AMD MI355X
 * (gfx950).
 *
 * What the library computes
 * -------------------------
 * For a linear layer y = x W^T (Sec. 2.2) the backward GEMMs are dX = dY W and
 * dW = dY^T x. Algorithm 3 transforms each GEMM operand with a blockwise
 * random Hadamard transform (RHT, Sec. 3.2) along its reduction dimension,
 * quantises it to MXFP4 with the unbiased quantiser of Algorithm 2 (3/4
 * pre-scale, stochastic rounding), multiplies the MXFP4 operands with FP32
 * accumulation and rescales the product by 16/9.
 *
 * Conventions for every call
 * --------------------------
 * - Pointers to tensors are DEVICE pointers owned by the caller. bf16 tensors
 *   are passed as their 16-bit patterns. Every matrix is row-major and dense
 *   (row pitch = number of columns).
 * - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued on
 *   it; the library never synchronises it.
 * - Arguments are validated before anything is enqueued. On error a negative
 *   MX_ERR_* status is returned and nothing is enqueued. Faults inside kernels
 *   surface at the caller's next synchronisation of the stream.
 * - A call with an empty problem (a zero dimension) enqueues nothing and
 *   returns MX_OK; its pointers may then be NULL.
 * - Outputs are fully overwritten (except what mx_linear_backward_ex is asked
 *   to accumulate into). Calls are thread-safe.
 * - Graph capture: every call that enqueues work first asks whether `stream`
 *   is being captured into a HIP graph and, if so, returns MX_ERR_CAPTURE and
 *   enqueues nothing (these calls may allocate or free their workspace in
 *   stream order, which a graph cannot replay; a graph would also keep a
 *   workspace address that a later call may free).
 * - Only gfx950 devices are supported (MX_ERR_DEVICE otherwise).
 *
 * The quantised format (MXFP4)
 * ----------------------------
 * A logical [rows, cols] matrix, cols a multiple of 32, is stored as
 * - codes  [rows, cols/2] bytes: two 4-bit E2M1 codes per byte, the element
 *   with the even column index in the low nibble. Code bits: bit 3 = sign,
 *   bits 0..2 index the magnitudes {0, 0.5, 1, 1.5, 2, 3, 4, 6} (Table 1,
 *   Sec. 2.1). A zero magnitude is always the code 0.
 * - scales [rows, cols/32] bytes: one E8M0 byte E per 32-element block,
 *   meaning 2^(E-127); 0xFF means NaN.
 * Element (r, c) is value(code) * 2^(scales[r][c/32] - 127).
 *
 * Quantisation rule (RHT, then Algorithm 2), per logical row
 * ----------------------------------------------------------
 * 1. Sign flip and Hadamard, per g-block of g consecutive elements
 *    (g in {32, 64, 128, 256}, cols % g == 0): y = H_g (S o x) with H_g the
 *    +-1 Sylvester matrix (the Hadamard recursion of Sec. 3.2 without its
 *    scale factor; H H^T = g I) and S in {+-1}^g shared by every block.
 *    In FP32, evaluated by the
 *    Sylvester recursion: the two half-size transforms first, then their sum
 *    and difference; IEEE round-to-nearest-even, no FMA, subnormals kept.
 * 2. Per 32-element block of y: E = floor(log2 max|y|) - 2 + 127 (shared_exp
 *    of Algorithm 2 with emax_elem = 2), clamped to >= 0; an all-zero block
 *    gets E = 0. A block holding an infinity or NaN gets E = 0xFF and all
 *    codes 0 (outside the method's contract).
 * 3. w = fl32((3/4) * y * 2^(127-E)): one round-to-nearest multiply; |w| < 6.
 * 4. Stochastic rounding (Eq. 1 with 16-bit noise): if f <= |w| < c are the
 *    neighbouring E2M1 magnitudes and t = (|w| - f)/(c - f), |w| rounds up to
 *    c iff floor(t * 2^16) + r >= 2^16, r the element's 16-bit noise.
 * Randomness (Philox4x32-10, Salmon et al. SC'11; seed split lo32/hi32):
 * - S_j = -1 iff bit (j & 31) of word ((j >> 5) & 3) of
 *   Philox(counter = (j >> 7, 0, 0, 1), key = (0, hi32(seed))) is 1.
 *   So S depends on hi32(seed) only.
 * - Noise of logical element (r, c): L = r * cols + c;
 *   Philox(counter = (lo32(L >> 3), hi32(L >> 3), 0, 0),
 *          key = (lo32(seed), hi32(seed))), word (L >> 1) & 3, low 16 bits if
 *   L is even, high 16 bits if odd.
 * Operands that are multiplied together must share S (same hi32 of the seed)
 * and use independent noise (different lo32).
 */
#ifndef MXFP4_H
#define MXFP4_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum mx_status {
  MX_OK = 0,
  MX_ERR_NULL = -1,    /* a required pointer is NULL */
  MX_ERR_G = -2,       /* g is not 32, 64, 128 or 256 */
  MX_ERR_SHAPE = -3,   /* negative size, or a divisibility rule is broken */
  MX_ERR_ALIGN = -4,   /* a pointer is not aligned as documented */
  MX_ERR_HIP = -5,     /* a HIP runtime call or kernel launch failed */
  MX_ERR_NOMEM = -6,   /* workspace allocation failed */
  MX_ERR_DEVICE = -7,  /* the current device is not a gfx950 GPU */
  MX_ERR_MODE = -8,    /* mode is not one of MX_MODE_* */
  MX_ERR_FLAGS = -9,   /* flags holds a bit that is not one of MX_BWD_* */
  MX_ERR_CAPTURE = -10, /* the stream is being captured into a graph */
  MX_ERR_TOO_LARGE = -11 /* more scratch than mx_linear_backward_noalloc holds */
};

/*
 * Quantiser modes: the method, the ablation rows of Table 2, and a
 * cheaper-noise variant.
 *   MX_MODE_RHT_SR  blockwise RHT, then Algorithm 2 (3/4 pre-scale, stochastic
 *                   rounding): the method, and what the entry points without a
 *                   mode argument use.
 *   MX_MODE_SR      Algorithm 2 without the RHT.
 *   MX_MODE_RHT_NR  blockwise RHT, then Algorithm 1: no 3/4, w = y / 2^E
 *                   (exact), rounded to the nearest E2M1 value (ties to the even
 *                   code), saturating at 6.
 *   MX_MODE_NR      Algorithm 1 alone: the plain OCP MX conversion.
 *   MX_MODE_RHT_SR8 MX_MODE_RHT_SR with a cheaper dither, a deliberate change
 *                   of the rounding rule above (never a default): 8 noise
 *                   bits, |w| rounds up iff floor(t * 2^8) + r >= 2^8 (bias at
 *                   most 2^-8 of the grid step instead of 2^-16). Element
 *                   (r, c) of the logical matrix, c = 64 a + 32 h + 8 b + e
 *                   (h < 2, b < 4, e < 8), takes byte (8 h + e) & 3 of word
 *                   (8 h + e) >> 2 of Philox(counter = (lo32(P), hi32(P), 0, 0),
 *                   key = (lo32(seed), hi32(seed))), P = (r * cols + 64 a + 8 b)
 *                   >> 3: one generator call per 16 elements instead of 8.
 *                   Needs g in {64, 128, 256} (MX_ERR_G otherwise).
 * The E8M0 scale rule, code layout, canonical zero and non-finite handling are
 * the same in every mode. Modes without the RHT ignore g (their blocks are the
 * 32-element MX blocks) and hi32(seed); modes with round to nearest ignore
 * lo32(seed).
 */
enum mx_mode { MX_MODE_RHT_SR = 0, MX_MODE_SR = 1, MX_MODE_RHT_NR = 2, MX_MODE_NR = 3, MX_MODE_RHT_SR8 = 4 };

/* Human-readable name of a status code (static string, never NULL). */
const char* mx_status_string(int status);

/*
 * RHT + stochastic-rounding MXFP4 quantisation of a row-major bf16 matrix.
 * Blocks run along the rows of `in` (the reduction dimension is cols).
 *   in     [rows, cols] bf16 bits, 16-byte aligned.
 *   codes  [rows, cols/2] bytes out, 4-byte aligned.
 *   scales [rows, cols/32] bytes out.
 *   rows >= 0; cols >= 0 with cols % g == 0; g in {32, 64, 128, 256}.
 * Paper: Sec. 3.2 (blockwise RHT), Algorithm 2, Eq. 1.
 */
int mx_rht_sr_quantize(const uint16_t* in, uint8_t* codes, uint8_t* scales, int64_t rows,
                       int64_t cols, int g, uint64_t seed, void* stream);

/*
 * Same output as mx_rht_sr_quantize applied to the transpose of `in_t`:
 * in_t is stored [cols, rows] row-major (so logical element (r, c) is
 * in_t[c * rows + r]) and blocks run down its columns. This is the layout the
 * dW GEMM needs for dY^T and x^T (Algorithm 3; proof of Lemma 3.1).
 *   in_t 16-byte aligned when rows % 8 == 0, 2-byte aligned otherwise.
 *   Other arguments as for mx_rht_sr_quantize.
 */
int mx_rht_sr_quantize_t(const uint16_t* in_t, uint8_t* codes, uint8_t* scales, int64_t rows,
                         int64_t cols, int g, uint64_t seed, void* stream);

/*
 * Quantisation in any mode (see enum mx_mode), of `in` read row-major
 * (transposed == 0, as mx_rht_sr_quantize) or transposed (transposed != 0, as
 * mx_rht_sr_quantize_t). Modes with the RHT need g in {32, 64, 128, 256} and
 * cols % g == 0; the others cols % 32 == 0. MX_ERR_MODE for an unknown mode.
 * mx_quantize(..., MX_MODE_RHT_SR, t, s) is mx_rht_sr_quantize(_t).
 * Paper: Algorithms 1 and 2, Sec. 3.2, Table 2.
 */
int mx_quantize(const uint16_t* in, uint8_t* codes, uint8_t* scales, int64_t rows, int64_t cols, int g,
                uint64_t seed, int mode, int transposed, void* stream);

/*
 * Both quantisations of one matrix in one pass over it: Algorithm 3 quantises
 * dY twice, along out (dY for dX) and along the tokens (dY^T for dW).
 *   in       [rows, cols] bf16 bits, row-major, 16-byte aligned.
 *   codes    [rows, cols/2], scales [rows, cols/32]: in quantised along its
 *            rows with `seed` -- mx_quantize(in, codes, scales, rows, cols, g,
 *            seed, mode, 0, stream), byte for byte.
 *   codes_t  [cols, rows/2], scales_t [cols, rows/32]: in^T quantised along its
 *            rows (blocks run down the columns of `in`) with `seed_t` --
 *            mx_quantize(in, codes_t, scales_t, cols, rows, g, seed_t, mode, 1,
 *            stream), byte for byte.
 *   codes and codes_t 4-byte aligned. Both rows and cols must be multiples of
 *   the mode's block (g with the RHT, 32 without); g and mode as for
 *   mx_quantize. The four outputs must not overlap.
 * When the block is at most 64 and cols % 8 == 0, each workgroup quantises the
 * tile it has read in both directions, so the input is read from memory once;
 * otherwise both run in one launch as separate passes. Results are the same
 * either way.
 * Paper: Algorithm 3 (the two quantisations of dY), Algorithm 2, Sec. 3.2.
 */
int mx_quantize_pair(const uint16_t* in, uint8_t* codes, uint8_t* scales, uint8_t* codes_t, uint8_t* scales_t,
                     int64_t rows, int64_t cols, int g, uint64_t seed, uint64_t seed_t, int mode, void* stream);

/*
 * MXFP4 GEMM with FP32 accumulation: C[M, N] = sum_k deq(A)[m, k] * deq(B)[n, k]
 * (the MXFP4_GEMM of Algorithm 3 with groups along K; no 16/9 factor here).
 *   A_codes [M, K/2], A_scales [M, K/32]; B_codes [N, K/2], B_scales [N, K/32],
 *   in the MXFP4 layout above; code pointers 16-byte aligned.
 *   C [M, N] float32 out, 4-byte aligned.
 *   M >= 0; 0 <= N < 2^24; K >= 0 with K % 32 == 0 (MX_ERR_SHAPE otherwise).
 * The summation order is the kernel's own and fixed (results are reproducible
 * run to run); they agree with an exact sum to FP32 accumulation accuracy.
 * When K % 128 == 0 the operands are first copied, in the library's
 * per-stream workspace (as for mx_linear_backward), into the K-tiled layout
 * the GEMM kernels load fastest: about 0.53 byte of scratch per element of A
 * and of B. When few output tiles meet a long K, K is split and FP32 partial
 * sums go through the same workspace. mx_gemm_f4_workspace_bytes gives the
 * total.
 */
int mx_gemm_f4(const uint8_t* A_codes, const uint8_t* A_scales, const uint8_t* B_codes,
               const uint8_t* B_scales, float* C, int64_t M, int64_t N, int64_t K, void* stream);

/* Bytes of workspace mx_gemm_f4 needs for these sizes (0 for invalid or empty
 * sizes, or when it needs none). */
int64_t mx_gemm_f4_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * Frees the workspace the library keeps for the current device and `stream`
 * (see mx_linear_backward), in stream order: the block is released after the
 * work already enqueued on `stream`, so calls enqueued before stay valid, and
 * its memory goes back to the device at the next synchronisation (of the
 * stream, an event on it or the device). The next call on that stream
 * allocates a new one. MX_OK also when the stream has none; MX_ERR_HIP if the
 * free fails. Not for a stream that is being captured (MX_ERR_CAPTURE).
 */
int mx_release_workspace(void* stream);

/*
 * Algorithm 3: MXFP4 backward pass of a linear layer y = x W^T (no bias).
 *   dY [T, out_features] bf16 bits, X [T, in_features] bf16 bits,
 *   W [out_features, in_features] bf16 bits; all 16-byte aligned.
 *   dX [T, in_features] float32 out; dW [out_features, in_features] float32 out.
 *   T % g == 0 and out_features % g == 0 (the two reduction dimensions);
 *   0 <= in_features < 2^24 (the N of both GEMMs); MX_ERR_SHAPE otherwise.
 * Computes, with Q_i the quantisation above using seed ^ i:
 *   Q0 = Q(dY)    [T, out],  Q1 = Q(W^T) [in, out]     (dX reduces over out)
 *   Q2 = Q(dY^T)  [out, T],  Q3 = Q(X^T) [in, T]       (dW reduces over T)
 *   dX = alpha * Q0 Q1^T,   dW = alpha * Q2 Q3^T,   alpha = fl32(16/9) / g.
 * The 16/9 undoes the (3/4)^2 of the two operands (Lemma 3.1) and 1/g undoes
 * H H^T = g I of the +-1 Hadamard. Each Q_i equals what mx_rht_sr_quantize(_t)
 * returns for the same operand and seed ^ i.
 * Scratch -- the quantised operands (about 0.53 byte per element of
 * 2 dY + W + X) and, when a GEMM is split along K, its FP32 partial sums
 * (mx_linear_backward_workspace_bytes gives the total) -- lives in a workspace
 * the library keeps per (device, stream) and reuses for every call on that
 * stream. A call that needs more than the workspace holds grows it in stream
 * order (the old block is freed after the work already enqueued on `stream`,
 * the new one allocated from a pool the library owns); the workspace is held
 * until mx_release_workspace or the end of the process. Because a call may
 * allocate, it refuses a stream that is being captured into a graph
 * (MX_ERR_CAPTURE).
 */
int mx_linear_backward(const uint16_t* dY, const uint16_t* X, const uint16_t* W, float* dX,
                       float* dW, int64_t T, int64_t in_features, int64_t out_features, int g,
                       uint64_t seed, void* stream);

/*
 * mx_linear_backward with the operands quantised in any mode (see enum
 * mx_mode): the ablations of Table 2 through the same GEMMs. The rescale is
 * alpha = (16/9 for modes with stochastic rounding, else 1) / (g for modes
 * with the RHT, else 1). Modes with the RHT need T % g == 0 and
 * out_features % g == 0; the others T % 32 == 0 and out_features % 32 == 0.
 * MX_ERR_MODE for an unknown mode. With MX_MODE_RHT_SR this is
 * mx_linear_backward.
 */
int mx_linear_backward_mode(const uint16_t* dY, const uint16_t* X, const uint16_t* W, float* dX, float* dW,
                            int64_t T, int64_t in_features, int64_t out_features, int g, uint64_t seed,
                            int mode, void* stream);

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * result as mx_linear_backward, bit for bit, with no allocation at all.
 *   Arguments, layouts and alignment as for mx_linear_backward; the caller
 *   still provides dY, X, W, dX and dW.
 *   Scratch (the quantised operands and any split-K partial sums, the bytes
 *   mx_linear_backward_workspace_bytes reports) comes from a fixed array of
 *   MX_NOALLOC_SCRATCH_BYTES (64 MiB) in device memory that the library holds
 *   on every GPU it runs this call on, from the first such call until the
 *   process ends. A problem that needs more returns MX_ERR_TOO_LARGE and
 *   enqueues nothing: 64 MiB holds any linear of a GPT-345M-shaped block
 *   (4096 tokens, hidden 1024), not GPT-1.3B's MLP linears.
 *   All calls on one GPU share that array: calls that overlap in time on one
 *   GPU (other streams, other threads) race and give wrong results; calls
 *   ordered on one stream are safe. Nothing in it needs to start at zero.
 *   This call calls no hipMalloc/hipFree or allocating routine, and does not
 *   refuse a stream that is being captured (its launches are then not traced).
 */
#define MX_NOALLOC_SCRATCH_BYTES (64ll << 20)
int mx_linear_backward_noalloc(const uint16_t* dY, const uint16_t* X, const uint16_t* W, float* dX,
                               float* dW, int64_t T, int64_t in_features, int64_t out_features, int g,
                               uint64_t seed, void* stream);

/* Bytes of stream-ordered scratch mx_linear_backward allocates for a shape. */
int64_t mx_linear_backward_workspace_bytes(int64_t T, int64_t in_features, int64_t out_features);

/*
 * Options of mx_linear_backward_ex, for use inside a training framework.
 *   MX_BWD_DX_BF16     dX is written as bf16 bits, each the FP32 result rounded
 *                      to nearest (ties to even; NaN stays NaN): the gradient
 *                      that flows on to the previous layer in the activations'
 *                      precision, at half the output bytes.
 *   MX_BWD_ACCUMULATE  dW and db are added to, in FP32: dW[i] = dW[i] + r[i]
 *                      with r the FP32 result (one rounding for the add), for
 *                      gradient accumulation into a high-precision main
 *                      gradient (mixed precision keeps parameters, and so
 *                      their gradients, in high precision: Sec. 2.3).
 */
enum mx_backward_flags { MX_BWD_DX_BF16 = 1, MX_BWD_ACCUMULATE = 2 };

/*
 * The full backward pass of a linear layer y = x W^T + b (Sec. 2.2): dX and dW
 * by Algorithm 3 exactly as mx_linear_backward_mode computes them (same
 * quantisations, seeds seed ^ i, GEMMs and alpha), and the bias gradient
 * db = 1^T dY, the column sums of dY, which is not quantised.
 *   dY, X, W, T, in_features, out_features, g, seed, mode: as for
 *     mx_linear_backward_mode.
 *   dX  [T, in_features]: float32 (4-byte aligned) or, with MX_BWD_DX_BF16,
 *       bf16 bits (2-byte aligned); always overwritten.
 *   dW  [out_features, in_features] float32, overwritten or, with
 *       MX_BWD_ACCUMULATE, added to.
 *   db  [out_features] float32, 4-byte aligned, or NULL for a layer without
 *       bias. db[j] = sum over t of dY[t, j] from the bf16 values in FP32, in a
 *       fixed order (per block of the reduction: g tokens with the RHT, 32
 *       without, summed as the quantiser of dY^T reads them; then the block
 *       sums in sixteen runs), so results repeat bit for bit; overwritten or, with
 *       MX_BWD_ACCUMULATE, added to. It is formed in the same pass that
 *       quantises dY^T (Q2), so it costs no extra read of dY.
 *   flags  a combination of MX_BWD_*; other bits give MX_ERR_FLAGS.
 * With T == 0 or out_features == 0 the GEMM products are zero: dX is cleared,
 * dW and db are cleared or, accumulating, left as they are. in_features == 0
 * with db given computes db alone.
 * Scratch: mx_linear_backward_ex_workspace_bytes gives the bytes; with db it
 * adds (T / block) * out_features * 4 bytes of block sums to what
 * mx_linear_backward needs. Errors, streams and workspace otherwise as for
 * mx_linear_backward.
 */
int mx_linear_backward_ex(const uint16_t* dY, const uint16_t* X, const uint16_t* W, void* dX, float* dW,
                          float* db, int64_t T, int64_t in_features, int64_t out_features, int g,
                          uint64_t seed, int mode, unsigned flags, void* stream);

/* Bytes of scratch mx_linear_backward_ex needs (with_db != 0: db is given);
 * 0 for invalid arguments. */
int64_t mx_linear_backward_ex_workspace_bytes(int64_t T, int64_t in_features, int64_t out_features, int g,
                                              int mode, int with_db);

/*
 * Kernel tracing. Between mx_profile_start() and mx_profile_stop() every kernel
 * the library launches carries two HIP events that the runtime records at the
 * kernel's start and end (hipExtLaunchKernel), so the time between them is the
 * kernel's own execution. mx_profile_stop() waits for those events and fills `stats`
 * (up to `capacity` entries, one per kernel name; *count gets the number of
 * kernel names seen) with the number of launches, their summed GPU time and
 * their summed algorithmic work: bytes for the quantiser (2 bytes read per
 * input element, once also when one pass writes two quantisations of it, and
 * 0.53125 bytes written per quantised element), FLOPs (2 M N K) for the GEMM,
 * bytes for the split-K reduction. Tracing is process-wide; calls that overlap with
 * mx_profile_stop() from another thread are not traced. mx_profile_stop()
 * consumes the session's records (a second call reports nothing). Returns MX_OK
 * or MX_ERR_HIP.
 */
typedef struct mx_kernel_stat {
  char name[48];        /* kernel name, e.g. "quant_g64", "gemm_128x128" */
  int64_t launches;
  double total_ms;      /* summed event-to-event time of its launches */
  double work;          /* summed algorithmic work */
  int work_is_flops;    /* 1: work is FLOPs, 0: work is bytes */
} mx_kernel_stat;

int mx_profile_start(void);
int mx_profile_stop(mx_kernel_stat* stats, int capacity, int* count);

/*
 * The attainable MFMA rate, for the GEMM's roofline: every CU runs one
 * workgroup whose four waves issue `rounds` rounds of 16 independent FP4
 * V_MFMA_SCALE_F32_32X32X64_F8F6F4 from registers (no memory traffic), timed
 * over 50 launches after about 0.3 s of warm-up launches, on a stream of the
 * library's own; the call synchronises and is not for use during other work.
 * *tflops gets the dense FP4 rate achieved and *clock_ghz the shader clock it
 * ran at (s_memtime cycles of one wave over the launch time): under full MFMA
 * load the chip holds a clock below the nominal 2.4 GHz, so this is what a
 * GEMM can reach at best. rounds in [1, 2^20] (MX_ERR_SHAPE otherwise; 2000
 * gives launches of about half a millisecond).
 */
int mx_measure_mfma_peak(int rounds, double* tflops, double* clock_ghz);

#ifdef __cplusplus
}
#endif

#endif /* MXFP4_H */
