// Internal launch entry points of libmxfp4 (not part of the C ABI).
// Arguments are assumed validated by the ABI layer. Each returns 0 on success,
// -1 if the launch failed.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mx {

// One RHT + SR quantisation: logical [rows, cols] matrix, blocks along cols.
// transposed == false: `in` is the logical matrix, row-major.
// transposed == true:  `in` is stored [cols, rows] (the logical matrix's transpose).
// Output layouts of a quantised [rows, cols] operand:
// * row-major (the C ABI's): codes [rows][cols/2], scales [rows][cols/32];
// * K-tiled (internal, cols % 128 == 0): for each 128-column stage s, a
//   row-major [rows][64] block of codes and a [rows][4] block of scales, so
//   the stage of a run of rows is one contiguous range:
//   code byte of (r, c) at (c / 128) * rows * 64 + r * 64 + (c % 128) / 2,
//   scale of (r, c) at (c / 128) * rows * 4 + r * 4 + (c % 128) / 32.
// colsum (transposed jobs only, optional): per g-block sums of the logical
// rows' input values, FP32, laid out [cols / g][rows] (the g-blocks of a mode
// without the RHT are its 32-element MX blocks). colsum_reduce() adds them up
// per row.
struct QuantSpec {
  const uint16_t* in;
  uint8_t* codes;
  uint8_t* scales;
  int64_t rows, cols;
  uint64_t seed;
  bool transposed;
  bool ktiled;
  float* colsum = nullptr;
  // transposed only, optional (g <= 64, rows % 8 == 0, `in` 16-byte aligned):
  // also quantise the stored matrix itself -- [cols, rows], blocks along rows
  // -- with twin_seed into twin_codes / twin_scales (same layout kind), in the
  // same pass over the input.
  uint8_t* twin_codes = nullptr;
  uint8_t* twin_scales = nullptr;
  uint64_t twin_seed = 0;
};

// The paper's quantiser, its ablations (Table 2 rows) and the cheaper-noise
// variant (8-bit dither); values match the C ABI's MX_MODE_* constants.
enum class QuantMode : int { kRhtSr = 0, kSr = 1, kRhtNr = 2, kNr = 3, kRhtSr8 = 4 };

// Up to 4 quantisations with the same g and mode in one launch. Modes without
// the RHT ignore g (their blocks are the 32-element MX blocks).
int launch_quant(const QuantSpec* specs, int count, int g, QuantMode mode, hipStream_t stream);

// out[r] = (accumulate ? out[r] : 0) + sum over b < nblk of partial[b * rows + r],
// in a fixed order (sixteen contiguous runs of b, each summed in order, then
// the sixteen run sums in order), so results are reproducible.
int colsum_reduce(const float* partial, float* out, int64_t rows, int64_t nblk, bool accumulate,
                  hipStream_t stream);

// Sets `bytes` bytes (a multiple of 2, 2-byte aligned) at p to zero.
int zero_fill(void* p, int64_t bytes, hipStream_t stream);

// How a GEMM writes C: FP32 (overwrite), bf16 (round to nearest even of the
// FP32 result, overwrite), or FP32 added to what C holds.
enum class Store : int { kF32 = 0, kBf16 = 1, kAccF32 = 2 };

// Largest N + 1 the GEMM kernels take: their FP32 and bf16 epilogues address
// a 32-row block of C (32 * N * 4 bytes) with 32-bit buffer offsets.
constexpr int64_t kGemmMaxN = int64_t(1) << 24;

struct GemmArgs {
  const uint8_t* a_codes;
  const uint8_t* a_scales;
  const uint8_t* b_codes;
  const uint8_t* b_scales;
  void* c;       // [M, N], float32 or bf16 bits as `store` says
  int64_t M, N, K;
  float alpha;
  bool ktiled;   // both operands K-tiled (only where gemm_takes_ktiled() says so)
  Store store = Store::kF32;
};

// Whether launch_gemm() runs this group of problems on a kernel that accepts
// K-tiled operands (and so whose operands may be quantised K-tiled).
bool gemm_takes_ktiled(const GemmArgs* probs, int count);

// Copies a row-major MXFP4 operand [rows, K] (codes 16-byte aligned,
// K % 128 == 0) into the K-tiled layout above (kcodes rows * K / 2 bytes,
// 16-byte aligned; kscales rows * K / 32 bytes, 4-byte aligned).
int launch_ktile_repack(const uint8_t* codes, const uint8_t* scales, uint8_t* kcodes, uint8_t* kscales,
                        int64_t rows, int64_t K, hipStream_t stream);

// One or two independent GEMMs in one launch. Problems with few output tiles
// and a long K are split along K into partial sums (in `partial_ws`, of
// gemm_workspace_bytes() bytes) that a second kernel adds up in a fixed order;
// with partial_ws == NULL nothing is split.
int64_t gemm_workspace_bytes(const GemmArgs* probs, int count);
int launch_gemm(const GemmArgs* probs, int count, float* partial_ws, hipStream_t stream);

// The attainable MFMA rate (mx_measure_mfma_peak): FP4 MFMAs from registers
// on every CU, timed over 50 launches after a 0.3 s warm-up on a stream of its
// own; synchronises. Returns 0, or -1 if a HIP call failed.
int measure_mfma_peak(int rounds, double* tflops, double* clock_ghz);

// Tracing (mx_profile_start / mx_profile_stop): while tracing is on, a
// TraceScope holds a pair of HIP events for one launch; the launch passes them
// to hipExtLaunchKernel, which records them at the kernel's start and end
// (null events, and a plain launch, while tracing is off).
bool profiling();
// While a NoTraceScope lives, launches from this thread are not traced (used
// for work enqueued on a stream that is being captured into a graph).
class NoTraceScope {
 public:
  explicit NoTraceScope(bool active);
  ~NoTraceScope();
  NoTraceScope(const NoTraceScope&) = delete;
  NoTraceScope& operator=(const NoTraceScope&) = delete;

 private:
  bool active_;
};
class TraceScope {
 public:
  TraceScope(const char* name, double work, bool flops);
  TraceScope(const TraceScope&) = delete;
  TraceScope& operator=(const TraceScope&) = delete;
  hipEvent_t start() const { return start_; }
  hipEvent_t stop() const { return stop_; }

 private:
  hipEvent_t start_ = nullptr;
  hipEvent_t stop_ = nullptr;
};

}  // namespace mx
