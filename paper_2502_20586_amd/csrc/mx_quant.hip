// Entry point of the fused RHT + stochastic-rounding quantiser (the kernels
// are in mx_quant_impl.h, instantiated per group of modes in mx_quant_*.hip),
// and the small kernels that serve the backward pass beside it (column-sum
// reduction for the bias gradient, zero fill).

#include "mx_quant_impl.h"

namespace mx {

int launch_quant(const QuantSpec* specs, int count, int g, QuantMode mode, hipStream_t stream) {
  if (count < 1 || count > 4) return -1;
  quant::QuantJobs jobs{};
  jobs.count = 0;
  const bool kt = specs[0].ktiled;
  for (int i = 0; i < count; ++i)
    if (specs[i].ktiled != kt) return -1;   // one output layout per launch
  // Transposed jobs first: their workgroups run longer, and the short
  // row-major ones then fill the launch's tail (about 2% of a GPT-345M step).
  int order[4], n = 0;
  for (int pass = 0; pass < 2; ++pass)
    for (int i = 0; i < count; ++i)
      if (specs[i].transposed == (pass == 0)) order[n++] = i;
  for (int o = 0; o < count; ++o) {
    const int i = order[o];
    if (specs[i].rows == 0 || specs[i].cols == 0) continue;
    quant::QuantJob& j = jobs.j[jobs.count++];
    j.in = specs[i].in;
    j.codes = specs[i].codes;
    j.scales = specs[i].scales;
    j.rows = specs[i].rows;
    j.cols = specs[i].cols;
    j.seed = specs[i].seed;
    j.transposed = specs[i].transposed ? 1 : 0;
    j.colsum = specs[i].colsum;
    if (j.colsum && !j.transposed) return -1;
    j.tcodes = specs[i].twin_codes;
    j.tscales = specs[i].twin_scales;
    j.tseed = specs[i].twin_seed;
    if ((j.tcodes == nullptr) != (j.tscales == nullptr)) return -1;
    // The twin's K-tiled offsets are 32-bit too; its blocks run along `rows`.
    if (j.tcodes && kt && (j.rows % 128 != 0 || j.rows * j.cols / 2 >= (int64_t(1) << 31))) return -1;
    const uintptr_t addr = reinterpret_cast<uintptr_t>(j.in);
    j.load_rows = (j.rows % 4 == 0 && addr % 8 == 0) ? 4 : (j.rows % 2 == 0 && addr % 4 == 0) ? 2 : 1;
    j.codes16 = reinterpret_cast<uintptr_t>(j.codes) % 16 == 0 ? 1 : 0;
    // K-tiled offsets are 32-bit (see store_chunk).
    if (kt && (j.cols % 128 != 0 || j.rows * j.cols / 2 >= (int64_t(1) << 31))) return -1;
  }
  if (jobs.count == 0) return 0;
  switch (mode) {
    case QuantMode::kRhtSr: return quant::launch_rht_sr(jobs, g, kt, stream);
    case QuantMode::kRhtSr8: return quant::launch_rht_sr8(jobs, g, kt, stream);
    default: return quant::launch_ablation(jobs, g, kt, mode, stream);
  }
}

namespace {

// A workgroup owns 64 rows (one per lane); wave w of 16 sums the blocks of
// the w-th sixteenth of [0, nblk) in order, then wave 0 adds the sixteen run
// sums in order. Loads of one wave read 64 consecutive floats; sixteen waves
// keep few dependent loads per thread (the kernel is latency-bound).
constexpr int kColsumWaves = 16;
__global__ __launch_bounds__(64 * kColsumWaves) void colsum_reduce_kernel(const float* partial, float* out,
                                                                          int64_t rows, int64_t nblk,
                                                                          int accumulate) {
  __shared__ float run[kColsumWaves][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * 64 + lane;
  const int64_t b0 = nblk * w / kColsumWaves, b1 = nblk * (w + 1) / kColsumWaves;
  float s = 0.0f;
  if (row < rows) {
    const float* p = partial + row;
#pragma unroll 4
    for (int64_t b = b0; b < b1; ++b) s += p[b * rows];
  }
  run[w][lane] = s;
  __syncthreads();
  if (w == 0 && row < rows) {
    float t = run[0][lane];
#pragma unroll
    for (int i = 1; i < kColsumWaves; ++i) t += run[i][lane];
    out[row] = accumulate ? out[row] + t : t;
  }
}

// Clears n 16-bit words: every output the library clears is made of bf16 or
// FP32 elements, so a 2-byte granularity covers all of them. A kernel rather
// than a memset node keeps the clear well-defined inside a captured graph.
__global__ __launch_bounds__(256) void zero_fill_kernel(uint16_t* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0;
}

}  // namespace

int zero_fill(void* p, int64_t bytes, hipStream_t stream) {
  if (bytes <= 0) return 0;
  const int64_t n = bytes / 2;
  const int64_t wgs = (n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096;
  TraceScope trace("zero_fill", (double)bytes, false);
  hipExtLaunchKernelGGL(zero_fill_kernel, dim3((unsigned)wgs), dim3(256), 0, stream, trace.start(), trace.stop(), 0,
                        static_cast<uint16_t*>(p), n);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int colsum_reduce(const float* partial, float* out, int64_t rows, int64_t nblk, bool accumulate,
                  hipStream_t stream) {
  if (rows <= 0) return 0;
  const int64_t wgs = (rows + 63) / 64;
  TraceScope trace("colsum_reduce", (double)rows * (nblk + (accumulate ? 2 : 1)) * 4.0, false);
  hipExtLaunchKernelGGL(colsum_reduce_kernel, dim3((unsigned)wgs), dim3(64 * kColsumWaves), 0, stream, trace.start(),
                        trace.stop(), 0, partial, out, rows, nblk, accumulate ? 1 : 0);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mx
