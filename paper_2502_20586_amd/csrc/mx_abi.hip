// C ABI of libmxfp4: argument validation, device check and the Algorithm 3
// orchestration (four quantisations and two GEMMs on the caller's stream).
// The contract of every entry point is documented in include/mxfp4.h.

#include <atomic>
#include <map>
#include <memory>
#include <mutex>
#include <utility>

#include "mx_internal.h"
#include "mxfp4.h"

namespace {

constexpr int kMaxDevices = 64;
std::atomic<int> g_device_state[kMaxDevices];  // 0 unknown, 1 gfx950, 2 other

int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MX_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MX_ERR_DEVICE;
  int st = g_device_state[dev].load(std::memory_order_acquire);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return MX_ERR_HIP;
    const char* a = prop.gcnArchName;
    const bool ok = a[0] == 'g' && a[1] == 'f' && a[2] == 'x' && a[3] == '9' && a[4] == '5' && a[5] == '0' &&
                    (a[6] == '\0' || a[6] == ':');
    st = ok ? 1 : 2;
    g_device_state[dev].store(st, std::memory_order_release);
  }
  return st == 1 ? MX_OK : MX_ERR_DEVICE;
}

// Scratch: one workspace per (device, stream), kept by the library and reused
// by every call on that stream. Work on one stream runs in order, so a call
// can reuse the memory of the previous one. A call that needs more grows the
// workspace: the old block is freed in stream order (after the work already
// enqueued that uses it) and a larger one allocated in stream order from a
// pool the library owns. A lease holds the workspace's lock from the moment
// its address is handed out until the work that uses it has been enqueued,
// so a concurrent call on the same stream cannot free it in between.
// A workspace is held until mx_release_workspace frees it (in stream order)
// or the process ends.
std::mutex g_pool_mutex;
hipMemPool_t g_pools[kMaxDevices];
bool g_pool_tried[kMaxDevices];

hipMemPool_t pool_for(int dev) {
  std::lock_guard<std::mutex> lock(g_pool_mutex);
  if (!g_pool_tried[dev]) {
    g_pool_tried[dev] = true;
    hipMemPoolProps props = {};
    props.allocType = hipMemAllocationTypePinned;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipMemPool_t pool = nullptr;
    if (hipMemPoolCreate(&pool, &props) == hipSuccess) {
      // Release threshold 0: a block freed in stream order (a workspace that
      // grew, or mx_release_workspace) goes back to the device at the next
      // synchronisation instead of staying reserved by the pool. Workspaces in
      // use are not affected; they are kept, not freed, between calls.
      uint64_t keep = 0;
      (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
      g_pools[dev] = pool;
    }
  }
  return g_pools[dev];
}

struct Workspace {
  std::mutex mu;
  void* ptr = nullptr;
  int64_t bytes = 0;
};

std::mutex g_ws_mutex;
std::map<std::pair<int, hipStream_t>, std::unique_ptr<Workspace>> g_workspaces;

class WorkspaceLease {
 public:
  WorkspaceLease() = default;
  WorkspaceLease(const WorkspaceLease&) = delete;
  WorkspaceLease& operator=(const WorkspaceLease&) = delete;
  ~WorkspaceLease() {
    if (ws_) ws_->mu.unlock();
  }

  // At least `bytes` bytes of scratch usable by work enqueued on `s` while the
  // lease is held.
  int acquire(int64_t bytes, hipStream_t s, void** out) {
    *out = nullptr;
    if (bytes <= 0) return MX_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return MX_ERR_HIP;
    {
      std::lock_guard<std::mutex> lock(g_ws_mutex);
      std::unique_ptr<Workspace>& slot = g_workspaces[{dev, s}];
      if (!slot) slot.reset(new Workspace);
      ws_ = slot.get();
    }
    ws_->mu.lock();
    if (ws_->bytes < bytes) {
      if (ws_->ptr && hipFreeAsync(ws_->ptr, s) != hipSuccess) return MX_ERR_HIP;
      ws_->ptr = nullptr;
      ws_->bytes = 0;
      const int64_t grown = (bytes + (int64_t(1) << 21) - 1) & ~((int64_t(1) << 21) - 1);   // 2 MiB steps
      hipMemPool_t pool = pool_for(dev);
      void* p = nullptr;
      const hipError_t e = pool ? hipMallocFromPoolAsync(&p, (size_t)grown, pool, s)
                                : hipMallocAsync(&p, (size_t)grown, s);
      if (e != hipSuccess || !p) return MX_ERR_NOMEM;
      ws_->ptr = p;
      ws_->bytes = grown;
    }
    *out = ws_->ptr;
    return MX_OK;
  }

 private:
  Workspace* ws_ = nullptr;
};

// Entry points that enqueue work refuse a stream that is being captured into
// a graph: a call may allocate or free workspace in stream order, and a graph
// would also keep the workspace address it saw, which a later call that grows
// the workspace frees. (An implicit capture of the legacy default stream, when
// another stream captures in global mode, counts as capturing.)
int check_not_capturing(hipStream_t s) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  const hipError_t e = hipStreamIsCapturing(s, &cs);
  if (e == hipErrorStreamCaptureImplicit) return MX_ERR_CAPTURE;
  if (e != hipSuccess) return MX_ERR_HIP;
  return cs == hipStreamCaptureStatusNone ? MX_OK : MX_ERR_CAPTURE;
}

// Scratch of mx_linear_backward_noalloc: a fixed array in device memory, one
// copy per GPU that the library runs on, held until the process ends. In host
// code `scratch` only names the variable; its device address on a GPU is what
// hipGetSymbolAddress returns with that GPU current, looked up once per device
// and kept. Every call on a GPU shares that GPU's copy and leaves in it what
// it wrote (the quantised operands and split-K partial sums, all of which the
// next call writes before it reads them, so nothing has to start at zero);
// calls that overlap on one GPU race.
constexpr int64_t kNoallocScratchBytes = MX_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];

int scratch_for_device(void** out) {
  *out = nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MX_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MX_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MX_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MX_OK;
}

bool valid_g(int g) { return g == 32 || g == 64 || g == 128 || g == 256; }
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool valid_mode(int mode) { return mode >= MX_MODE_RHT_SR && mode <= MX_MODE_RHT_SR8; }
bool mode_has_rht(int mode) { return mode == MX_MODE_RHT_SR || mode == MX_MODE_RHT_NR || mode == MX_MODE_RHT_SR8; }
bool mode_has_sr(int mode) { return mode == MX_MODE_RHT_SR || mode == MX_MODE_SR || mode == MX_MODE_RHT_SR8; }
// g accepted by a mode with the RHT: 8-bit noise serves two 32-element chunks
// of a lane per generator call, so it needs g >= 64.
bool valid_g_for(int mode, int g) { return valid_g(g) && (mode != MX_MODE_RHT_SR8 || g >= 64); }
// Block along the reduction dimension that a mode needs whole: g with the
// RHT, the 32-element MX block without it (g is then ignored).
int mode_block(int mode, int g) { return mode_has_rht(mode) ? g : 32; }

int validate_quant(const uint16_t* in, const uint8_t* codes, const uint8_t* scales, int64_t rows,
                   int64_t cols, int g, bool transposed, int mode) {
  if (!valid_mode(mode)) return MX_ERR_MODE;
  if (mode_has_rht(mode) && !valid_g_for(mode, g)) return MX_ERR_G;
  if (rows < 0 || cols < 0 || cols % mode_block(mode, g) != 0) return MX_ERR_SHAPE;
  if (rows == 0 || cols == 0) return MX_OK;
  if (!in || !codes || !scales) return MX_ERR_NULL;
  const uintptr_t in_align = (!transposed || rows % 8 == 0) ? 16 : 2;
  if (!aligned(in, in_align) || !aligned(codes, 4)) return MX_ERR_ALIGN;
  return MX_OK;
}

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

struct MxBuf {
  uint8_t* codes;
  uint8_t* scales;
};

// Carve the four quantised operands, the GEMM partial sums and then
// `colsum_bytes` for the bias gradient's block sums out of one workspace
// (256-byte aligned parts).
int64_t layout_workspace(int64_t T, int64_t in_f, int64_t out_f, uint8_t* base, MxBuf q[4], float** partial,
                         int64_t colsum_bytes = 0, float** colsum = nullptr) {
  const int64_t elems[4] = {T * out_f, in_f * out_f, out_f * T, in_f * T};
  int64_t off = 0;
  for (int i = 0; i < 4; ++i) {
    if (q) q[i].codes = base ? base + off : nullptr;
    off = round_up(off + elems[i] / 2, 256);
    if (q) q[i].scales = base ? base + off : nullptr;
    off = round_up(off + elems[i] / 32, 256);
  }
  // The GEMMs' tile configuration, hence their K splits, can depend on the
  // output kinds (accumulating outputs run on 128 x 128 tiles): the partial
  // sums get the larger of the two requirements, so one size fits every flag.
  mx::GemmArgs g[2] = {{nullptr, nullptr, nullptr, nullptr, nullptr, T, in_f, out_f, 0.f, false},
                       {nullptr, nullptr, nullptr, nullptr, nullptr, out_f, in_f, T, 0.f, false}};
  int64_t partial_bytes = mx::gemm_workspace_bytes(g, 2);
  g[1].store = mx::Store::kAccF32;
  const int64_t acc_bytes = mx::gemm_workspace_bytes(g, 2);
  if (acc_bytes > partial_bytes) partial_bytes = acc_bytes;
  if (partial) *partial = base ? reinterpret_cast<float*>(base + off) : nullptr;
  off = round_up(off + partial_bytes, 256);
  if (colsum) *colsum = base && colsum_bytes > 0 ? reinterpret_cast<float*>(base + off) : nullptr;
  off = round_up(off + colsum_bytes, 256);
  return off;
}

constexpr unsigned kKnownFlags = MX_BWD_DX_BF16 | MX_BWD_ACCUMULATE;

// Algorithm 3 with the options of mx_linear_backward_ex (the contract is in
// include/mxfp4.h).
// noalloc: scratch comes from the fixed per-GPU array instead of the
// stream's workspace, nothing is allocated, and a capturing stream is allowed
// (its launches are then not traced).
int linear_backward(const uint16_t* dY, const uint16_t* X, const uint16_t* W, void* dX, float* dW, float* db,
                    int64_t T, int64_t in_features, int64_t out_features, int g, uint64_t seed, int mode,
                    unsigned flags, hipStream_t s, bool noalloc = false) {
  if (!valid_mode(mode)) return MX_ERR_MODE;
  if (flags & ~kKnownFlags) return MX_ERR_FLAGS;
  if (mode_has_rht(mode) && !valid_g_for(mode, g)) return MX_ERR_G;
  const int blk = mode_block(mode, g);
  if (T < 0 || in_features < 0 || out_features < 0 || T % blk != 0 || out_features % blk != 0 ||
      in_features >= mx::kGemmMaxN)
    return MX_ERR_SHAPE;
  const bool dx_bf16 = (flags & MX_BWD_DX_BF16) != 0;
  const bool accumulate = (flags & MX_BWD_ACCUMULATE) != 0;
  const bool need_dx = T > 0 && in_features > 0;
  const bool need_dw = out_features > 0 && in_features > 0;
  const bool need_db = db != nullptr && out_features > 0;
  if (!need_dx && !need_dw && !need_db) return MX_OK;
  if ((need_dx && !dX) || (need_dw && !dW)) return MX_ERR_NULL;
  if ((T > 0 && out_features > 0 && !dY) || (T > 0 && in_features > 0 && !X) ||
      (out_features > 0 && in_features > 0 && !W))
    return MX_ERR_NULL;
  if (!aligned(dY, 16) || !aligned(X, 16) || !aligned(W, 16) || !aligned(dX, dx_bf16 ? 2 : 4) ||
      !aligned(dW, 4) || !aligned(db, 4))
    return MX_ERR_ALIGN;
  int st = check_device();
  if (st != MX_OK) return st;
  bool capturing = false;
  if ((st = check_not_capturing(s)) == MX_ERR_CAPTURE && noalloc)
    capturing = true;
  else if (st != MX_OK)
    return st;
  const mx::NoTraceScope no_trace(capturing);
  // 16/9 undoes the 3/4 pre-scale of both operands (stochastic rounding only);
  // 1/g undoes H H^T = g I of the +-1 Hadamard (RHT modes only).
  const float alpha = (mode_has_sr(mode) ? 16.0f / 9.0f : 1.0f) / (float)(mode_has_rht(mode) ? g : 1);

  // K = 0 for a GEMM (T == 0 or out == 0): its product is all zeros, so an
  // overwritten output is cleared and an accumulated one is left as it is.
  if (T == 0 || out_features == 0) {
    if (need_dx && mx::zero_fill(dX, T * in_features * (dx_bf16 ? 2 : 4), s)) return MX_ERR_HIP;
    if (need_dw && !accumulate && mx::zero_fill(dW, out_features * in_features * 4, s)) return MX_ERR_HIP;
    if (need_db && !accumulate && mx::zero_fill(db, out_features * 4, s)) return MX_ERR_HIP;
    return MX_OK;
  }

  MxBuf q[4];
  float* partial = nullptr;
  float* colsum = nullptr;
  const int64_t nblk = T / blk;   // blocks of Q2's reduction dimension
  const int64_t colsum_bytes = need_db ? nblk * out_features * 4 : 0;
  const int64_t bytes = layout_workspace(T, in_features, out_features, nullptr, nullptr, nullptr, colsum_bytes);
  void* ws = nullptr;
  WorkspaceLease lease;
  if (noalloc) {
    if (bytes > kNoallocScratchBytes) return MX_ERR_TOO_LARGE;
    if ((st = scratch_for_device(&ws)) != MX_OK) return st;
  } else if ((st = lease.acquire(bytes, s, &ws)) != MX_OK) {
    return st;
  }
  layout_workspace(T, in_features, out_features, static_cast<uint8_t*>(ws), q, &partial, colsum_bytes, &colsum);

  int fail = 0;
  // dX = dY W reduces over out: Q0 = Q(dY) [T, out], Q1 = Q(W^T) [in, out].
  // dW = dY^T x reduces over T: Q2 = Q(dY^T) [out, T], Q3 = Q(x^T) [in, T].
  // When the GEMMs run on the LDS-ring kernels, the quantised operands are
  // written K-tiled (the layout those kernels load fastest); the values are
  // the same either way. The bias gradient 1^T dY is summed by the Q2
  // quantisation, which reads dY along T, into per-block partial sums.
  mx::GemmArgs gp[2] = {
      {q[0].codes, q[0].scales, q[1].codes, q[1].scales, dX, T, in_features, out_features, alpha, false,
       dx_bf16 ? mx::Store::kBf16 : mx::Store::kF32},
      {q[2].codes, q[2].scales, q[3].codes, q[3].scales, dW, out_features, in_features, T, alpha, false,
       accumulate ? mx::Store::kAccF32 : mx::Store::kF32}};
  const bool kt = in_features > 0 && mx::gemm_takes_ktiled(gp, 2);
  gp[0].ktiled = gp[1].ktiled = kt;
  mx::QuantSpec specs[4] = {
      {dY, q[0].codes, q[0].scales, T, out_features, seed ^ 0u, false, kt},
      {W, q[1].codes, q[1].scales, in_features, out_features, seed ^ 1u, true, kt},
      {dY, q[2].codes, q[2].scales, out_features, T, seed ^ 2u, true, kt},
      {X, q[3].codes, q[3].scales, in_features, T, seed ^ 3u, true, kt},
  };
  specs[2].colsum = colsum;
  // For blocks of at most 64 the dY^T pass also writes Q0 (its twin: the
  // stored dY quantised along out), so dY is read from memory once.
  const bool twin = blk <= 64 && out_features % 8 == 0 && aligned(dY, 16);
  if (in_features > 0 && twin) {
    specs[2].twin_codes = q[0].codes;
    specs[2].twin_scales = q[0].scales;
    specs[2].twin_seed = specs[0].seed;
    fail |= mx::launch_quant(specs + 1, 3, g, static_cast<mx::QuantMode>(mode), s);
  } else if (in_features > 0) {
    fail |= mx::launch_quant(specs, 4, g, static_cast<mx::QuantMode>(mode), s);
  } else if (need_db) {   // no GEMM to feed: only the pass that sums dY
    fail |= mx::launch_quant(&specs[2], 1, g, static_cast<mx::QuantMode>(mode), s);
  }
  if (in_features > 0) fail |= mx::launch_gemm(gp, 2, partial, s);
  if (need_db) fail |= mx::colsum_reduce(colsum, db, out_features, nblk, accumulate, s);
  return fail ? MX_ERR_HIP : MX_OK;
}

}  // namespace

extern "C" {

const char* mx_status_string(int status) {
  switch (status) {
    case MX_OK: return "MX_OK";
    case MX_ERR_NULL: return "MX_ERR_NULL: a required pointer is NULL";
    case MX_ERR_G: return "MX_ERR_G: g must be 32, 64, 128 or 256";
    case MX_ERR_SHAPE: return "MX_ERR_SHAPE: negative size or broken divisibility rule";
    case MX_ERR_ALIGN: return "MX_ERR_ALIGN: pointer not aligned as required";
    case MX_ERR_HIP: return "MX_ERR_HIP: HIP runtime call or kernel launch failed";
    case MX_ERR_NOMEM: return "MX_ERR_NOMEM: workspace allocation failed";
    case MX_ERR_DEVICE: return "MX_ERR_DEVICE: current device is not gfx950";
    case MX_ERR_MODE: return "MX_ERR_MODE: mode is not one of MX_MODE_*";
    case MX_ERR_FLAGS: return "MX_ERR_FLAGS: flags holds bits that are not MX_BWD_*";
    case MX_ERR_CAPTURE: return "MX_ERR_CAPTURE: the stream is being captured into a graph";
    case MX_ERR_TOO_LARGE:
      return "MX_ERR_TOO_LARGE: the problem needs more scratch than mx_linear_backward_noalloc holds";
    default: return "MX_ERR_UNKNOWN";
  }
}

int mx_quantize(const uint16_t* in, uint8_t* codes, uint8_t* scales, int64_t rows, int64_t cols, int g,
                uint64_t seed, int mode, int transposed, void* stream) {
  int st = validate_quant(in, codes, scales, rows, cols, g, transposed != 0, mode);
  if (st != MX_OK || rows == 0 || cols == 0) return st;
  if ((st = check_device()) != MX_OK) return st;
  if ((st = check_not_capturing((hipStream_t)stream)) != MX_OK) return st;
  const mx::QuantSpec spec{in, codes, scales, rows, cols, seed, transposed != 0, false};
  return mx::launch_quant(&spec, 1, g, static_cast<mx::QuantMode>(mode), (hipStream_t)stream) ? MX_ERR_HIP
                                                                                                 : MX_OK;
}

int mx_rht_sr_quantize(const uint16_t* in, uint8_t* codes, uint8_t* scales, int64_t rows, int64_t cols,
                       int g, uint64_t seed, void* stream) {
  return mx_quantize(in, codes, scales, rows, cols, g, seed, MX_MODE_RHT_SR, 0, stream);
}

int mx_rht_sr_quantize_t(const uint16_t* in_t, uint8_t* codes, uint8_t* scales, int64_t rows,
                         int64_t cols, int g, uint64_t seed, void* stream) {
  return mx_quantize(in_t, codes, scales, rows, cols, g, seed, MX_MODE_RHT_SR, 1, stream);
}

int mx_quantize_pair(const uint16_t* in, uint8_t* codes, uint8_t* scales, uint8_t* codes_t, uint8_t* scales_t,
                     int64_t rows, int64_t cols, int g, uint64_t seed, uint64_t seed_t, int mode, void* stream) {
  int st = validate_quant(in, codes, scales, rows, cols, g, false, mode);
  if (st != MX_OK) return st;
  if ((st = validate_quant(in, codes_t, scales_t, cols, rows, g, true, mode)) != MX_OK) return st;
  if (rows == 0 || cols == 0) return MX_OK;
  if (!aligned(in, 16)) return MX_ERR_ALIGN;
  if ((st = check_device()) != MX_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_not_capturing(s)) != MX_OK) return st;
  const mx::QuantMode m = static_cast<mx::QuantMode>(mode);
  mx::QuantSpec spec_t{in, codes_t, scales_t, cols, rows, seed_t, true, false};
  if (mode_block(mode, g) <= 64 && cols % 8 == 0) {
    spec_t.twin_codes = codes;
    spec_t.twin_scales = scales;
    spec_t.twin_seed = seed;
    return mx::launch_quant(&spec_t, 1, g, m, s) ? MX_ERR_HIP : MX_OK;
  }
  const mx::QuantSpec specs[2] = {spec_t, {in, codes, scales, rows, cols, seed, false, false}};
  return mx::launch_quant(specs, 2, g, m, s) ? MX_ERR_HIP : MX_OK;
}

}  // extern "C"

namespace {

// Workspace of mx_gemm_f4: split-K partial sums first, then (K-tiled
// kernels) the K-tiled copies of A's codes and scales and B's codes and
// scales at off[0..3]. Returns the total bytes.
int64_t gemm_f4_layout(const mx::GemmArgs& g, bool* kt, int64_t* partial_bytes, int64_t off[4]) {
  *kt = g.K > 0 && mx::gemm_takes_ktiled(&g, 1);
  *partial_bytes = round_up(mx::gemm_workspace_bytes(&g, 1), 256);
  int64_t bytes = *partial_bytes;
  for (int i = 0; i < 4; ++i) off[i] = 0;
  if (*kt) {
    const int64_t parts[4] = {g.M * g.K / 2, g.M * g.K / 32, g.N * g.K / 2, g.N * g.K / 32};
    for (int i = 0; i < 4; ++i) {
      off[i] = bytes;
      bytes = round_up(bytes + parts[i], 256);
    }
  }
  return bytes;
}

}  // namespace

extern "C" {

int mx_measure_mfma_peak(int rounds, double* tflops, double* clock_ghz) {
  if (!tflops || !clock_ghz) return MX_ERR_NULL;
  if (rounds < 1 || rounds > (1 << 20)) return MX_ERR_SHAPE;
  int st = check_device();
  if (st != MX_OK) return st;
  return mx::measure_mfma_peak(rounds, tflops, clock_ghz) ? MX_ERR_HIP : MX_OK;
}

int64_t mx_gemm_f4_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K < 0 || K % 32 != 0 || N >= mx::kGemmMaxN) return 0;
  const mx::GemmArgs g{nullptr, nullptr, nullptr, nullptr, nullptr, M, N, K, 1.0f, false};
  bool kt;
  int64_t partial_bytes, off[4];
  return gemm_f4_layout(g, &kt, &partial_bytes, off);
}

int mx_release_workspace(void* stream) {
  hipStream_t s = (hipStream_t)stream;
  int st = check_not_capturing(s);
  if (st != MX_OK) return st;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MX_ERR_HIP;
  Workspace* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    auto it = g_workspaces.find({dev, s});
    if (it == g_workspaces.end()) return MX_OK;
    ws = it->second.get();
  }
  std::lock_guard<std::mutex> lock(ws->mu);
  if (ws->ptr && hipFreeAsync(ws->ptr, s) != hipSuccess) return MX_ERR_HIP;
  ws->ptr = nullptr;
  ws->bytes = 0;
  return MX_OK;
}

int mx_gemm_f4(const uint8_t* A_codes, const uint8_t* A_scales, const uint8_t* B_codes,
               const uint8_t* B_scales, float* C, int64_t M, int64_t N, int64_t K, void* stream) {
  if (M < 0 || N < 0 || K < 0 || K % 32 != 0 || N >= mx::kGemmMaxN) return MX_ERR_SHAPE;
  if (M == 0 || N == 0) return MX_OK;
  if (!C) return MX_ERR_NULL;
  if (K > 0 && (!A_codes || !A_scales || !B_codes || !B_scales)) return MX_ERR_NULL;
  if (!aligned(A_codes, 16) || !aligned(B_codes, 16) || !aligned(C, 4)) return MX_ERR_ALIGN;
  int st = check_device();
  if (st != MX_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if ((st = check_not_capturing(s)) != MX_OK) return st;
  mx::GemmArgs g{A_codes, A_scales, B_codes, B_scales, C, M, N, K, 1.0f, false};
  // On the LDS-ring kernels the operands are first copied into the K-tiled
  // layout those kernels load fastest (one stage of a run of rows is one
  // contiguous range; row-major scale loads touch one cache line per row):
  // a memory-bound pass of about 1.06 bytes per operand element, small next
  // to the GEMM it speeds up.
  bool kt;
  int64_t partial_bytes, off[4];
  const int64_t bytes = gemm_f4_layout(g, &kt, &partial_bytes, off);
  void* ws = nullptr;
  WorkspaceLease lease;
  if ((st = lease.acquire(bytes, s, &ws)) != MX_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  if (kt) {
    if (mx::launch_ktile_repack(A_codes, A_scales, base + off[0], base + off[1], M, K, s) ||
        mx::launch_ktile_repack(B_codes, B_scales, base + off[2], base + off[3], N, K, s))
      return MX_ERR_HIP;
    g.a_codes = base + off[0];
    g.a_scales = base + off[1];
    g.b_codes = base + off[2];
    g.b_scales = base + off[3];
    g.ktiled = true;
  }
  return mx::launch_gemm(&g, 1, partial_bytes > 0 ? reinterpret_cast<float*>(base) : nullptr, s) ? MX_ERR_HIP
                                                                                                   : MX_OK;
}

int64_t mx_linear_backward_workspace_bytes(int64_t T, int64_t in_features, int64_t out_features) {
  if (T < 0 || in_features < 0 || out_features < 0) return 0;
  return layout_workspace(T, in_features, out_features, nullptr, nullptr, nullptr);
}

int mx_linear_backward_mode(const uint16_t* dY, const uint16_t* X, const uint16_t* W, float* dX, float* dW,
                            int64_t T, int64_t in_features, int64_t out_features, int g, uint64_t seed,
                            int mode, void* stream) {
  return linear_backward(dY, X, W, dX, dW, nullptr, T, in_features, out_features, g, seed, mode, 0u,
                         (hipStream_t)stream);
}

int mx_linear_backward_ex(const uint16_t* dY, const uint16_t* X, const uint16_t* W, void* dX, float* dW,
                          float* db, int64_t T, int64_t in_features, int64_t out_features, int g, uint64_t seed,
                          int mode, unsigned flags, void* stream) {
  return linear_backward(dY, X, W, dX, dW, db, T, in_features, out_features, g, seed, mode, flags,
                         (hipStream_t)stream);
}

int64_t mx_linear_backward_ex_workspace_bytes(int64_t T, int64_t in_features, int64_t out_features, int g,
                                              int mode, int with_db) {
  if (T < 0 || in_features < 0 || out_features < 0 || !valid_mode(mode)) return 0;
  if (mode_has_rht(mode) && !valid_g_for(mode, g)) return 0;
  const int64_t colsum_bytes = with_db ? T / mode_block(mode, g) * out_features * 4 : 0;
  return layout_workspace(T, in_features, out_features, nullptr, nullptr, nullptr, colsum_bytes);
}

int mx_linear_backward(const uint16_t* dY, const uint16_t* X, const uint16_t* W, float* dX, float* dW,
                       int64_t T, int64_t in_features, int64_t out_features, int g, uint64_t seed,
                       void* stream) {
  return mx_linear_backward_mode(dY, X, W, dX, dW, T, in_features, out_features, g, seed, MX_MODE_RHT_SR,
                                 stream);
}

int mx_linear_backward_noalloc(const uint16_t* dY, const uint16_t* X, const uint16_t* W, float* dX, float* dW,
                               int64_t T, int64_t in_features, int64_t out_features, int g, uint64_t seed,
                               void* stream) {
  return linear_backward(dY, X, W, dX, dW, nullptr, T, in_features, out_features, g, seed, MX_MODE_RHT_SR, 0u,
                         (hipStream_t)stream, true);
}

}  // extern "C"
