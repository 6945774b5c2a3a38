// Kernel tracing for libmxfp4: HIP events recorded at the start and end of
// every kernel the library launches while tracing is on (see mx_profile_start / mx_profile_stop in mxfp4.h).

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "mx_internal.h"
#include "mxfp4.h"

namespace mx {
namespace {

struct Record {
  std::string name;
  hipEvent_t start, stop;
  double work;
  bool flops;
};

std::atomic<bool> g_on{false};
std::mutex g_mutex;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_spare;

hipEvent_t take_event() {
  if (!g_spare.empty()) {
    hipEvent_t e = g_spare.back();
    g_spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

thread_local int g_no_trace = 0;

}  // namespace

bool profiling() { return g_no_trace == 0 && g_on.load(std::memory_order_acquire); }

NoTraceScope::NoTraceScope(bool active) : active_(active) {
  if (active_) ++g_no_trace;
}
NoTraceScope::~NoTraceScope() {
  if (active_) --g_no_trace;
}

TraceScope::TraceScope(const char* name, double work, bool flops) {
  if (!profiling()) return;
  std::lock_guard<std::mutex> lock(g_mutex);
  Record r{name, take_event(), take_event(), work, flops};
  if (!r.start || !r.stop) return;
  g_records.push_back(r);
  start_ = r.start;
  stop_ = r.stop;
}

// ---------------------------------------------------------------------------
// Attainable MFMA rate. Each wave issues `rounds` rounds of 16 independent
// V_MFMA_SCALE_F32_32X32X64_F8F6F4 (FP4 x FP4; the 16 accumulator tiles of
// one 256 x 256 GEMM wave) from registers, with no memory traffic, so the
// launch runs at the rate the matrix cores sustain under full load -- at the
// clock the chip holds under that load, which is below the nominal one.
constexpr int kPeakTiles = 16;
// External linkage, so the device compiler keeps the stores (and with them the
// MFMAs) although no device code reads these back.
__device__ float g_peak_sink[kPeakTiles * 16];       // one sum per lane of block 0
__device__ uint64_t g_peak_cycles[2];                 // s_memtime span of block 0, wave 0

namespace {
typedef float v16f_p __attribute__((ext_vector_type(16)));
typedef int v8i_p __attribute__((ext_vector_type(8)));

__global__ __launch_bounds__(256, 1) void mfma_peak_kernel(int rounds, int salt) {
  v16f_p acc[kPeakTiles];
#pragma unroll
  for (int t = 0; t < kPeakTiles; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;
  // Four A and four B fragments of pseudo-random FP4 codes (a multiplicative
  // hash of lane, salt and word), combined as a GEMM wave combines its
  // fragments: every MFMA sees other operand bits than the one before, as in
  // a real K loop (constant operands would draw less power and let the clock
  // run higher than any GEMM could).
  const uint32_t lane = threadIdx.x & 63;
  v8i_p a[4], b[4];
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const uint32_t h = (lane * 8u + w + 0x9E3779B9u * (uint32_t)(salt + 16 * f + 1)) * 0x85EBCA6Bu;
      a[f][w] = w < 4 ? (int)(h ^ (h >> 13)) : 0;
      const uint32_t k = (lane * 8u + w + 0xC2B2AE35u * (uint32_t)(salt + 16 * f + 7)) * 0x27D4EB2Fu;
      b[f][w] = w < 4 ? (int)(k ^ (k >> 15)) : 0;
    }
  const uint64_t t0 = __builtin_amdgcn_s_memtime();
  for (int r = 0; r < rounds; ++r) {
#pragma unroll
    for (int t = 0; t < kPeakTiles; ++t)
      acc[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[t >> 2], b[t & 3], acc[t], 4, 4, 0, 120, 0, 121);
  }
  const uint64_t t1 = __builtin_amdgcn_s_memtime();
  float sum = 0.0f;                                    // element 0 of every tile keeps its MFMA chain
#pragma unroll
  for (int t = 0; t < kPeakTiles; ++t) sum += acc[t][0];
  // Block 0 writes its sums (plain vector stores).
  if (blockIdx.x == 0 && threadIdx.x < kPeakTiles * 16) g_peak_sink[threadIdx.x] = sum;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    g_peak_cycles[0] = t0;
    g_peak_cycles[1] = t1;
  }
}
}  // namespace

int measure_mfma_peak(int rounds, double* tflops, double* clock_ghz) {
  int dev = 0;
  hipDeviceProp_t prop;
  if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) return -1;
  const int blocks = prop.multiProcessorCount;          // one 4-wave workgroup per CU (512 registers a lane)
  hipStream_t s = nullptr;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) return -1;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int status = -1;
  if (hipEventCreate(&e0) == hipSuccess && hipEventCreate(&e1) == hipSuccess) {
    // Warm-up of about 0.3 s: the clocks settle under sustained load.
    bool ok = true;
    for (int i = 0; ok && i < 600; ++i) {
      hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(256), 0, s, rounds, i);
      ok = hipGetLastError() == hipSuccess;
    }
    const int reps = 50;
    ok = ok && hipEventRecord(e0, s) == hipSuccess;
    for (int i = 0; ok && i < reps; ++i) {
      hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(256), 0, s, rounds, i);
      ok = hipGetLastError() == hipSuccess;
    }
    ok = ok && hipEventRecord(e1, s) == hipSuccess && hipEventSynchronize(e1) == hipSuccess;
    float ms = 0.0f;
    uint64_t cyc[2] = {0, 0};
    ok = ok && hipEventElapsedTime(&ms, e0, e1) == hipSuccess &&
         hipMemcpyFromSymbol(cyc, HIP_SYMBOL(g_peak_cycles), sizeof(cyc), 0, hipMemcpyDeviceToHost) == hipSuccess;
    if (ok && ms > 0.0f) {
      const double per_launch_s = ms * 1e-3 / reps;
      const double flops = (double)blocks * 4 * rounds * kPeakTiles * (32.0 * 32 * 64 * 2);
      *tflops = flops / per_launch_s / 1e12;
      *clock_ghz = (double)(cyc[1] - cyc[0]) / per_launch_s / 1e9;
      status = 0;
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipStreamDestroy(s);
  return status;
}

}  // namespace mx

extern "C" {

int mx_profile_start(void) {
  std::lock_guard<std::mutex> lock(mx::g_mutex);
  for (auto& r : mx::g_records) {
    mx::g_spare.push_back(r.start);
    mx::g_spare.push_back(r.stop);
  }
  mx::g_records.clear();
  mx::g_on.store(true, std::memory_order_release);
  return MX_OK;
}

int mx_profile_stop(mx_kernel_stat* stats, int capacity, int* count) {
  mx::g_on.store(false, std::memory_order_release);
  std::lock_guard<std::mutex> lock(mx::g_mutex);
  std::vector<mx_kernel_stat> agg;
  int status = MX_OK;
  for (auto& r : mx::g_records) {
    float ms = 0.0f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      status = MX_ERR_HIP;
      continue;
    }
    mx_kernel_stat* s = nullptr;
    for (auto& a : agg)
      if (r.name == a.name) s = &a;
    if (!s) {
      agg.push_back(mx_kernel_stat{});
      s = &agg.back();
      std::strncpy(s->name, r.name.c_str(), sizeof(s->name) - 1);
      s->work_is_flops = r.flops ? 1 : 0;
    }
    s->launches += 1;
    s->total_ms += ms;
    s->work += r.work;
  }
  for (auto& r : mx::g_records) {  // the session's records are consumed
    mx::g_spare.push_back(r.start);
    mx::g_spare.push_back(r.stop);
  }
  mx::g_records.clear();
  if (count) *count = (int)agg.size();
  for (int i = 0; stats && i < capacity && i < (int)agg.size(); ++i) stats[i] = agg[i];
  return status;
}

}  // extern "C"
