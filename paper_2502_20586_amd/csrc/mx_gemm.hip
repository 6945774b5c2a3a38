// Block-scaled MXFP4 GEMM on CDNA4's scaled MFMA (V_MFMA_SCALE_F32_32X32X64_F8F6F4
// in FP4 mode): C[M, N] = alpha * sum_k deq(A)[m, k] * deq(B)[n, k].
//
// This is the MXFP4_GEMM of Algorithm 3: MX groups of 32 run along the
// reduction dimension of both operands, each group carries an E8M0 scale, and
// products accumulate in FP32 (the proof of Lemma 3.1 writes the same sum).
//
// Operand layout (both "K-major"): codes [rows, K/2] bytes, element 2i in the
// low nibble of byte i; scales [rows, K/32] E8M0 bytes. Lane l of a 32x32x64
// MFMA supplies 16 code bytes = one whole MX block (row l % 32, K-half l / 32)
// and that block's scale byte, picked out of a 32-bit register by op_sel.
//
// Work layout
// * A workgroup (4 waves, 2 x 2) owns a BM x BN output tile and walks K in
//   stages of 256 (128 code bytes and 8 scale bytes per row).
// * Code tiles live in LDS as [rows][128 B]; the 16-byte unit u of row r is
//   stored at unit u ^ swz(r), swz(r) = (r & 7) ^ ((r >> 3) & 1), so the
//   16-byte reads of 8 (or 16) consecutive rows never share a bank.
// * Double-buffered: the global loads of stage s+1 sit in registers while the
//   MFMAs of stage s run, and go to the other LDS buffer afterwards.
// * Several problems (the dX and dW GEMMs of one backward pass) can share one
//   launch: a workgroup finds its problem from its tile index.
// * Workgroup i runs on XCD i % 8; tiles are handed out so that each XCD gets a
//   contiguous run of the tile order, and that order walks groups of 8 tile
//   rows (N fastest inside a group), so the workgroups running together on one
//   XCD share both their A and their B panels in that XCD's L2.

#include <string>
#include <type_traits>

#include "mx_device.h"
#include "mx_internal.h"

namespace mx {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kStagedBK = 256;                   // K elements per stage
constexpr int kRowBytes = kStagedBK / 2;         // 128 code bytes per row per stage
constexpr int kUnits = kRowBytes / 16;     // 8 x 16-byte units (one MX block each) per row
constexpr int kSBytes = kStagedBK / 32;          // 8 scale bytes per row per stage
constexpr int kThreads = 256;
constexpr int kXcds = 8;
constexpr int kGroupM = 8;                 // tile rows per group of the tile order

__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <int BM, int BN>
struct Cfg {
  static constexpr int kWM = BM / 2;          // wave tile (2 x 2 waves)
  static constexpr int kWN = BN / 2;
  static constexpr int kTM = kWM / 32;        // 32x32 MFMA tiles per wave
  static constexpr int kTN = kWN / 32;
  static constexpr int kCodeA = BM * kRowBytes;
  static constexpr int kCodeB = BN * kRowBytes;
  static constexpr int kScaleA = BM * kSBytes;
  static constexpr int kScaleB = BN * kSBytes;
  static constexpr int kStage = kCodeA + kCodeB + kScaleA + kScaleB;
  static constexpr int kLds = 2 * kStage;
  static constexpr int kLoadsA = BM * kUnits / kThreads;   // 16-byte code loads per thread
  static constexpr int kLoadsB = BN * kUnits / kThreads;
  static_assert(kLoadsA >= 1 && kLoadsB >= 1, "tile too small for 256 threads");
  static_assert(BM <= kThreads && BN <= kThreads, "one scale row per thread");
};

struct Problem {
  const uint8_t* a_codes;
  const uint8_t* a_scales;
  const uint8_t* b_codes;
  const uint8_t* b_scales;
  void* c;           // output, written as `store` says
  int64_t M, N, K;
  int64_t tiles_n;   // tiles along N
  int64_t tiles;     // workgroups of this problem: output tiles x splits
  float alpha;
  int splits;        // K is cut into `splits` chunks of kchunk elements
  int64_t kchunk;
  float* partial;    // splits > 1: [splits][M][N] partial sums, reduced afterwards
  int ktiled;        // operands in the K-tiled layout (LDS-ring kernels only)
  int store;         // a Store value
};

// One or two problems in one launch. Problem 0 takes blocks [0, p[0].tiles),
// problem 1 blocks [start1, start1 + p[1].tiles); start1 is a multiple of the
// XCD count so both ranges begin on XCD 0 (blocks in the gap exit at once).
struct Group {
  Problem p[2];
  int count;
  int64_t start1;
};

// Where a workgroup works: its problem, output tile origin and K window.
struct TilePos {
  bool valid;       // false: a block in the gap between the problems' ranges
  bool second;      // problem 1 of the group (else problem 0)
  int split;
  int64_t m0, n0;   // output tile origin
  int64_t kbeg, K;  // K window [kbeg, kbeg + K)
};

// Block b runs on XCD b % 8. Inside a problem's range, tiles are handed out so
// that each XCD gets a contiguous run of the tile order. That order walks
// groups of kGroupM tile rows, N fastest inside a group, so the workgroups
// running together on one XCD share A and B panels in its L2. The host puts
// the problem with the longer K window first, so its tiles are dispatched
// first.
template <int BM, int BN>
__device__ __forceinline__ TilePos locate_tile(const Group& grp) {
  TilePos pos;
  int64_t t = blockIdx.x;
  pos.second = grp.count > 1 && t >= grp.start1;
  const Problem& P = pos.second ? grp.p[1] : grp.p[0];
  if (pos.second) t -= grp.start1;
  pos.valid = t < P.tiles;
  if (!pos.valid) return pos;
  {
    const int64_t per = P.tiles / kXcds, rem = P.tiles % kXcds;
    const int64_t x = t % kXcds, j = t / kXcds;
    t = x * per + (x < rem ? x : rem) + j;
  }
  pos.split = (int)(t % P.splits);
  t /= P.splits;
  const int64_t tiles_m = P.tiles / P.splits / P.tiles_n;
  const int64_t per_group = kGroupM * P.tiles_n;
  const int64_t group = t / per_group;
  const int64_t first_m = group * kGroupM;
  const int64_t rows_in_group = min((int64_t)kGroupM, tiles_m - first_m);
  const int64_t in_group = t - group * per_group;
  pos.m0 = (first_m + in_group % rows_in_group) * BM;
  pos.n0 = (in_group / rows_in_group) * BN;
  pos.kbeg = pos.split * P.kchunk;
  pos.K = min(P.kchunk, P.K - pos.kbeg);
  return pos;
}

// Cache-policy operand of the raw buffer store builtins: the non-temporal bit
// (bit 1, "nt" on gfx9-family targets).
constexpr int kNonTemporal = 2;

// bf16 bits of x rounded to nearest, ties to even (the hardware convert
// V_CVT_PK_BF16_F32 under the default rounding mode, denormals kept; a NaN
// stays a NaN): one instruction instead of the bit arithmetic.
__device__ __forceinline__ uint16_t bf16_rne(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// Element e of an output as `store` says: v is the final FP32 value. Outputs
// are written with the non-temporal hint: they stream to memory without
// displacing the operands the following kernels read from the caches
// (GPT-345M step 6% faster in a same-box comparison, GPT-6.7B unchanged).
template <int STORE>
__device__ __forceinline__ void store_elem(void* base, int64_t e, float v) {
  if constexpr (STORE == (int)Store::kBf16) {
    __builtin_nontemporal_store(bf16_rne(v), static_cast<uint16_t*>(base) + e);
  } else if constexpr (STORE == (int)Store::kAccF32) {
    float* c = static_cast<float*>(base);
    __builtin_nontemporal_store(c[e] + v, c + e);
  } else {
    __builtin_nontemporal_store(v, static_cast<float*>(base) + e);
  }
}

// FP32 and bf16 stores go through a raw buffer resource per 32-row block of
// C: rows past M lie outside the resource, so their stores are dropped, and a
// lane whose column is past N takes an offset of 2^31, outside every resource
// (a block spans 32 N element-size bytes, under 2^31 for N < kGemmMaxN = 2^24,
// which the entry points check). Each element then costs one 32-bit add for its offset and no
// bounds branch; the resources are scalar and lie inside C's rows.
// Row runs: in a 32 x 32 MFMA tile, lanes 0-31 hold 32 columns of one row and
// lanes 32-63 the same columns four rows further. For two tiles side by side,
// one V_PERMLANE32_SWAP per value trades the upper half of the left tile's
// register with the lower half of the right one's, leaving one register with
// 64 consecutive columns of a row and the other with those of the row four
// further: each store then writes one 256-byte run (FP32) instead of two
// 128-byte ones. With every CU storing at once, a store-only test drained
// 256 KiB per CU in 11.7 instead of 15.4 us this way; the GPT-6.7B block's
// GEMMs took 0.6% less time.
// The accumulating kind loads the old values through the same resource (rows
// and columns outside it read as zeros) -- those of a tile pair before any is
// written back, so the loads overlap -- and stores old + alpha * sum.
template <int STORE, int TM, int TN>
__device__ __forceinline__ void store_tiles_buf(const Problem& P, void* out, float alpha, int64_t row0,
                                                int64_t col0, const v16f (&acc)[TM][TN], int lane) {
  static_assert(TN % 2 == 0, "tiles are stored in side-by-side pairs");
  constexpr uint32_t kEs = STORE == (int)Store::kBf16 ? 2u : 4u;
  const uint32_t pitch = (uint32_t)P.N * kEs;
  uint32_t lane_off[TN / 2];
#pragma unroll
  for (int p = 0; p < TN / 2; ++p) {
    const int64_t col = col0 + p * 64 + lane;
    lane_off[p] = col < P.N ? (uint32_t)col * kEs : 0x80000000u;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t rb = row0 + i * 32;
    const int64_t left = P.M - rb;
    const int64_t nrows = left < 0 ? 0 : (left < 32 ? left : 32);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        static_cast<uint8_t*>(out) + (nrows > 0 ? rb * (int64_t)pitch : 0), (short)0, (int)(nrows * pitch),
        0x00020000);
#pragma unroll
    for (int p = 0; p < TN / 2; ++p) {
      // value v of the pair: element h of the swap holds row (v / 4) 8 + v % 4 + 4 h
      uint32_t sw[16][2];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        // Through scalars: a bit cast of a vector element reads element 0.
        const float left = acc[i][2 * p][v], right = acc[i][2 * p + 1][v];
        const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, left),
                                                        __builtin_bit_cast(uint32_t, right), false, false);
        sw[v][0] = r[0];
        sw[v][1] = r[1];
      }
      if constexpr (STORE == (int)Store::kAccF32) {
        uint32_t old[16][2];
#pragma unroll
        for (int v = 0; v < 16; ++v)
#pragma unroll
          for (int h = 0; h < 2; ++h)
            old[v][h] = __builtin_amdgcn_raw_buffer_load_b32(
                rs, (int)(lane_off[p] + (uint32_t)((v >> 2) * 8 + (v & 3) + 4 * h) * pitch), 0, 0);
#pragma unroll
        for (int v = 0; v < 16; ++v)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t off = lane_off[p] + (uint32_t)((v >> 2) * 8 + (v & 3) + 4 * h) * pitch;
            const float val = __builtin_bit_cast(float, old[v][h]) + __builtin_bit_cast(float, sw[v][h]) * alpha;
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, val), rs, (int)off, 0,
                                                  kNonTemporal);
          }
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t off = lane_off[p] + (uint32_t)((v >> 2) * 8 + (v & 3) + 4 * h) * pitch;
            const float val = __builtin_bit_cast(float, sw[v][h]) * alpha;
            if constexpr (STORE == (int)Store::kBf16)
              __builtin_amdgcn_raw_buffer_store_b16(bf16_rne(val), rs, (int)off, 0, kNonTemporal);
            else
              __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, val), rs, (int)off, 0,
                                                    kNonTemporal);
          }
      }
    }
  }
}

template <int STORE, int TM, int TN>
__device__ __forceinline__ void store_tiles_as(const Problem& P, void* out, float alpha, int64_t row0,
                                               int64_t col0, const v16f (&acc)[TM][TN], int lane) {
  store_tiles_buf<STORE, TM, TN>(P, out, alpha, row0, col0, acc, lane);
}

// Epilogue of a wave owning TM x TN MFMA tiles of 32 x 32 from (row0, col0):
// lane l holds rows (v / 4) * 8 + (l / 32) * 4 + v % 4 of column l % 32 of each
// tile. Unsplit problems store alpha * sum into C as P.store says; split ones
// write their FP32 partial sum, which reduce_splits_kernel adds up in split
// order before the same store. SS, the store kinds a kernel is built for: 0
// FP32 only, 1 FP32 and bf16, 2 all (the 256 x 256 kernel, whose accumulators
// fill all 256 AGPRs, is built once per set, so launches without bf16 or
// accumulating outputs do not carry those paths' registers).
template <int TM, int TN, int SS = 2>
__device__ __forceinline__ void store_tiles(const Problem& P, int split, int64_t row0, int64_t col0,
                                            const v16f (&acc)[TM][TN], int lane) {
  const bool is_split = P.splits > 1;
  if (SS == 0 || is_split || P.store == (int)Store::kF32)   // one FP32 path for partial sums and plain outputs
    store_tiles_as<(int)Store::kF32>(P, is_split ? P.partial + (int64_t)split * P.M * P.N : P.c,
                                     is_split ? 1.0f : P.alpha, row0, col0, acc, lane);
  else if (SS == 1 || P.store == (int)Store::kBf16)
    store_tiles_as<(int)Store::kBf16>(P, P.c, P.alpha, row0, col0, acc, lane);
  else
    store_tiles_as<(int)Store::kAccF32>(P, P.c, P.alpha, row0, col0, acc, lane);
}

// One stage of one operand in registers: code units, the 8 scale bytes of one
// row (threads tid < ROWS), and how many of the stage's 8 MX blocks exist.
template <int LOADS>
struct StageRegs {
  uint4 code[LOADS];
  uint2 scale;
  int nblocks;
};

// Per-thread view of one operand: thread tid loads 16-byte unit (tid % 8) of
// rows row0 + tid / 8 + 32 i, and the 8 scale bytes of row row0 + tid.
// Loads never branch: rows past the end are clamped to the last row (read,
// never stored), MX blocks past the K window are clamped to its last block and
// replaced by code 0 with scale 1.0 when the stage goes to LDS, which
// contributes exactly 0 to the sum.
template <int ROWS, int LOADS>
struct OperandView {
  const uint8_t* codes;       // at the K window's start
  const uint8_t* scales;      // at the K window's start
  uint32_t code_off[LOADS];   // byte offset of row i of this thread
  uint32_t scale_off;         // byte offset of this thread's scale row
  int64_t kb_total;           // MX blocks in the K window

  __device__ __forceinline__ void init(const uint8_t* c, const uint8_t* s, int64_t nrows, int64_t row0,
                                       int64_t Kfull, int64_t kbeg, int64_t K, int tid) {
    kb_total = K / 32;
    const int64_t kbytes = Kfull / 2;
    const int64_t kb_pitch = Kfull / 32;
    codes = c + kbeg / 2;
    scales = s + kbeg / 32;
    const int64_t last = nrows - 1;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int64_t r = min(row0 + (tid >> 3) + 32 * i, last);
      code_off[i] = (uint32_t)(r * kbytes);
    }
    scale_off = (uint32_t)(min(row0 + (tid % ROWS), last) * kb_pitch);
  }

  // KALIGNED: rows of scales are 4-byte aligned (K % 128 == 0), so a stage's
  // scales are two dwords, the second one past the window only in a last stage
  // holding 4 blocks.
  template <bool KALIGNED>
  __device__ __forceinline__ void load(StageRegs<LOADS>& st, int64_t kb0, int tid) const {
    const int64_t nb = kb_total - kb0;
    st.nblocks = (int)(nb < kSBytes ? nb : kSBytes);
    const int u = tid & 7;
    const uint8_t* base = codes + (u < st.nblocks ? kb0 + u : kb_total - 1) * 16;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) st.code[i] = *reinterpret_cast<const uint4*>(base + code_off[i]);
    const uint8_t* sp = scales + scale_off + kb0;
    if (KALIGNED) {
      st.scale.x = *reinterpret_cast<const uint32_t*>(sp);
      st.scale.y = *reinterpret_cast<const uint32_t*>(sp + (st.nblocks > 4 ? 4 : 0));
    } else {
      uint32_t v[2] = {0, 0};
#pragma unroll
      for (int j = 0; j < kSBytes; ++j) v[j >> 2] |= (uint32_t)sp[j < st.nblocks ? j : 0] << (8 * (j & 3));
      st.scale = make_uint2(v[0], v[1]);
    }
  }
};

template <int ROWS, int LOADS>
__device__ __forceinline__ void store_stage(const StageRegs<LOADS>& st, uint8_t* codes_lds, uint2* scales_lds,
                                            int tid) {
  const int u = tid & 7;
  const bool full = st.nblocks == kSBytes;
  const bool unit_ok = u < st.nblocks;
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int r = (tid >> 3) + 32 * i;
    const uint4 v = (full || unit_ok) ? st.code[i] : make_uint4(0, 0, 0, 0);
    *reinterpret_cast<uint4*>(codes_lds + r * kRowBytes + ((u ^ swz(r)) << 4)) = v;
  }
  if (tid < ROWS) {
    uint2 sc = st.scale;
    if (!full) {
      // keep the bytes of existing blocks, E8M0 1.0 for the rest
      const uint32_t n = (uint32_t)st.nblocks;
      const uint32_t mx = n >= 4 ? 0xFFFFFFFFu : (n == 0 ? 0u : (0xFFFFFFFFu >> (32 - 8 * n)));
      const uint32_t my = n >= 8 ? 0xFFFFFFFFu : (n <= 4 ? 0u : (0xFFFFFFFFu >> (32 - 8 * (n - 4))));
      sc.x = (sc.x & mx) | (0x7F7F7F7Fu & ~mx);
      sc.y = (sc.y & my) | (0x7F7F7F7Fu & ~my);
    }
    scales_lds[tid] = sc;
  }
}

template <int BM, int BN, bool KALIGNED>
__global__ __launch_bounds__(kThreads) void gemm_f4_kernel(Group grp) {
  using C = Cfg<BM, BN>;
  extern __shared__ __align__(16) uint8_t smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const TilePos pos = locate_tile<BM, BN>(grp);
  if (!pos.valid) return;
  const Problem& P = pos.second ? grp.p[1] : grp.p[0];
  const int64_t m0 = pos.m0, n0 = pos.n0, kbeg = pos.kbeg, K = pos.K;

  v16f acc[C::kTM][C::kTN];
#pragma unroll
  for (int i = 0; i < C::kTM; ++i)
#pragma unroll
    for (int j = 0; j < C::kTN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  StageRegs<C::kLoadsA> ra;
  StageRegs<C::kLoadsB> rb;
  OperandView<BM, C::kLoadsA> va;
  OperandView<BN, C::kLoadsB> vb;
  va.init(P.a_codes, P.a_scales, P.M, m0, P.K, kbeg, K, tid);
  vb.init(P.b_codes, P.b_scales, P.N, n0, P.K, kbeg, K, tid);
  const int64_t ksteps = (K + kStagedBK - 1) / kStagedBK;

  auto codes_a = [&](int s) { return smem + s * C::kStage; };
  auto codes_b = [&](int s) { return smem + s * C::kStage + C::kCodeA; };
  auto scales_a = [&](int s) { return reinterpret_cast<uint2*>(smem + s * C::kStage + C::kCodeA + C::kCodeB); };
  auto scales_b = [&](int s) {
    return reinterpret_cast<uint2*>(smem + s * C::kStage + C::kCodeA + C::kCodeB + C::kScaleA);
  };

  if (ksteps > 0) {
    va.template load<KALIGNED>(ra, 0, tid);
    vb.template load<KALIGNED>(rb, 0, tid);
    store_stage<BM>(ra, codes_a(0), scales_a(0), tid);
    store_stage<BN>(rb, codes_b(0), scales_b(0), tid);
    if (ksteps > 1) {
      va.template load<KALIGNED>(ra, kSBytes, tid);
      vb.template load<KALIGNED>(rb, kSBytes, tid);
    }
  }
  __syncthreads();

  const int half = lane >> 5;   // which 32-element half of a 64-wide MFMA step
  const int lrow = lane & 31;
  for (int64_t ks = 0; ks < ksteps; ++ks) {
    const int cur = (int)(ks & 1);
    const uint8_t* ca = codes_a(cur);
    const uint8_t* cb = codes_b(cur);
    const uint2* sa = scales_a(cur);
    const uint2* sb = scales_b(cur);
    // Scale bytes of this lane's rows: MX block 2*kk + half of the stage sits
    // in dword kk/2, byte 2*(kk%2) + half; shifting by 8*half leaves it at
    // byte 2*(kk%2), which op_sel picks.
    uint2 sav[C::kTM], sbv[C::kTN];
#pragma unroll
    for (int i = 0; i < C::kTM; ++i) {
      const uint2 s = sa[wm * C::kWM + i * 32 + lrow];
      sav[i] = make_uint2(s.x >> (8 * half), s.y >> (8 * half));
    }
#pragma unroll
    for (int j = 0; j < C::kTN; ++j) {
      const uint2 s = sb[wn * C::kWN + j * 32 + lrow];
      sbv[j] = make_uint2(s.x >> (8 * half), s.y >> (8 * half));
    }
#pragma unroll
    for (int kk = 0; kk < kStagedBK / 64; ++kk) {
      const int unit = kk * 2 + half;
      v8i af[C::kTM], bf[C::kTN];
#pragma unroll
      for (int i = 0; i < C::kTM; ++i) {
        const int r = wm * C::kWM + i * 32 + lrow;
        const uint4 x = *reinterpret_cast<const uint4*>(ca + r * kRowBytes + ((unit ^ swz(r)) << 4));
        af[i] = v8i{(int)x.x, (int)x.y, (int)x.z, (int)x.w, 0, 0, 0, 0};
      }
#pragma unroll
      for (int j = 0; j < C::kTN; ++j) {
        const int r = wn * C::kWN + j * 32 + lrow;
        const uint4 x = *reinterpret_cast<const uint4*>(cb + r * kRowBytes + ((unit ^ swz(r)) << 4));
        bf[j] = v8i{(int)x.x, (int)x.y, (int)x.z, (int)x.w, 0, 0, 0, 0};
      }
#pragma unroll
      for (int i = 0; i < C::kTM; ++i)
#pragma unroll
        for (int j = 0; j < C::kTN; ++j) {
          const int sai = (int)((kk < 2) ? sav[i].x : sav[i].y);
          const int sbj = (int)((kk < 2) ? sbv[j].x : sbv[j].y);
          if ((kk & 1) == 0)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[i], bf[j], acc[i][j], 4, 4, 0, sai, 0, sbj);
          else
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[i], bf[j], acc[i][j], 4, 4, 2, sai, 2, sbj);
        }
    }
    if (ks + 1 < ksteps) {
      store_stage<BM>(ra, codes_a(cur ^ 1), scales_a(cur ^ 1), tid);
      store_stage<BN>(rb, codes_b(cur ^ 1), scales_b(cur ^ 1), tid);
      if (ks + 2 < ksteps) {
        va.template load<KALIGNED>(ra, (ks + 2) * kSBytes, tid);
        vb.template load<KALIGNED>(rb, (ks + 2) * kSBytes, tid);
      }
    }
    __syncthreads();
  }

  store_tiles<C::kTM, C::kTN>(P, pos.split, m0 + wm * C::kWM, n0 + wn * C::kWN, acc, lane);
}

// ---------------------------------------------------------------------------
// Square BT x BT tiles (BT = 256 or 128) fed by direct buffer-to-LDS loads.
//
// * 4 waves (2 x 2), each owning a BT/2 x BT/2 block of TT x TT MFMA tiles
//   (TT = BT / 64). At BT = 256 the 256 FP32 accumulators of a lane fill its
//   accumulation registers and one workgroup runs per CU; BT = 128 runs two.
// * K walks in stages of 128 (64 code bytes and 4 scale bytes per row) through
//   a ring of 4 LDS slots. BUFFER_LOAD_DWORDX4 ... LDS moves 16 bytes per lane
//   from memory straight to LDS address M0 + 16 * lane (DWORD: M0 + 4 * lane),
//   with no register staging. A stage's fragments are read from LDS into
//   registers one stage ahead, while the previous stage's MFMAs run from
//   registers, so each read has a whole stage of MFMAs to land and the LDS
//   slot is free again one stage early: three stages of loads are in flight
//   beyond the one being read. (With one 64-K step of read-ahead the fragment
//   reads, slowed by the direct-to-LDS writes competing for LDS, stalled the
//   MFMAs.) At 256 x 256 the loads and reads are spread among the MFMAs in a
//   fixed order (see the stage functions).
// * Each operand is read through a buffer resource that starts at the tile's
//   first row and ends with the operand: rows past M (N) fall outside it and
//   load as zeros, and code 0 contributes 0 whatever its scale, so ragged M and
//   N need no masking. K must be a multiple of 128.
// * Waits are explicit: s_waitcnt vmcnt counts this wave's loads still in
//   flight (they complete in order), then a barrier makes every wave's share
//   of the stage visible. The compiler does not see these loads.
// * Code slot layout: row r (64 bytes) keeps 16-byte unit u at position
//   u ^ fsw(r), fsw(r) = ((r >> 1) ^ (r >> 2)) & 3, so the 16-byte reads of 8 or
//   16 consecutive rows of one unit hit distinct banks.
// * Scale slot layout: dword q of an operand holds the 4 scale bytes of row
//   (q / 32 TT) * 32 TT + (q % TT) * 32 + (q / TT) % 32, so one 4 TT-byte read
//   gives a lane the scales of its row in all TT MFMA tiles of its wave.
// ---------------------------------------------------------------------------
namespace ring {
constexpr int kBK = 128;                        // K elements per stage
constexpr int kRow = kBK / 2;                   // 64 code bytes per row per stage
constexpr int kSlots = 4;
constexpr int64_t kMaxK = int64_t(1) << 24;     // keeps 256 rows of codes under 2^32 bytes

template <int BT>
struct Cfg {
  static constexpr int kTT = BT / 64;           // MFMA tiles per wave along M and N
  static constexpr int kCode = BT * kRow;       // code bytes per operand per stage
  static constexpr int kScale = BT * 4;         // scale bytes per operand per stage
  static constexpr int kSlot = 2 * kCode + 2 * kScale;
  static constexpr int kLds = kSlots * kSlot;   // 136 KiB (BT = 256), 68 KiB (BT = 128)
  static constexpr int kCodeLoads = BT / 64;    // 16-byte loads per thread per operand per stage
  static constexpr int kScaleLoads = BT / 128;  // 4-byte loads per thread per stage (both operands)
  static constexpr int kLoads = 2 * kCodeLoads + kScaleLoads;
  static constexpr int kWgPerCu = BT == 256 ? 1 : 2;
};

__device__ __forceinline__ int fsw(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }
template <int TT>
__device__ __forceinline__ int scale_row(int q) {
  return (q / (32 * TT)) * (32 * TT) + (q % TT) * 32 + (q / TT) % 32;
}
}  // namespace ring

typedef int v4i __attribute__((ext_vector_type(4)));

// Raw buffer resource over `bytes` bytes at `base`: loads at offsets >= bytes
// return zeros.
__device__ __forceinline__ v4i buffer_rsrc(const void* base, int64_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  v4i r;
  r.x = (int)(uint32_t)a;
  r.y = (int)((uint32_t)(a >> 32) & 0xFFFFu);   // stride 0
  r.z = (int)(uint32_t)(bytes > 0xFFFFFFFFll ? 0xFFFFFFFFll : (bytes < 0 ? 0 : bytes));
  r.w = 0x00020000;                               // 32-bit data format
  return r;
}

__device__ __forceinline__ void lds_load_b128(v4i rsrc, uint32_t voff, uint32_t lds) {
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc), "{m0}"(lds) : "memory");
}
__device__ __forceinline__ void lds_load_b32(v4i rsrc, uint32_t voff, uint32_t lds) {
  asm volatile("buffer_load_dword %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc), "{m0}"(lds) : "memory");
}
// Wait until at most N of this wave's loads are in flight and its LDS reads
// are done, then synchronise the workgroup.
template <int N>
__device__ __forceinline__ void wait_and_sync() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

__device__ __forceinline__ v8i frag(const uint8_t* p) {
  const uint4 x = *reinterpret_cast<const uint4*>(p);
  return v8i{(int)x.x, (int)x.y, (int)x.z, (int)x.w, 0, 0, 0, 0};
}

template <int TT>
struct ScaleRegs {
  uint32_t w[TT];
};

template <int TT>
__device__ __forceinline__ ScaleRegs<TT> read_scales(const uint8_t* p) {
  ScaleRegs<TT> s;
  if constexpr (TT == 4) {
    const uint4 x = *reinterpret_cast<const uint4*>(p);
    s.w[0] = x.x; s.w[1] = x.y; s.w[2] = x.z; s.w[3] = x.w;
  } else {
    const uint2 x = *reinterpret_cast<const uint2*>(p);
    s.w[0] = x.x; s.w[1] = x.y;
  }
  return s;
}

template <int BT, int SS>
__global__ __launch_bounds__(kThreads, ring::Cfg<BT>::kWgPerCu) void gemm_ring_kernel(Group grp) {
  using ring::fsw;
  using ring::kRow;
  using ring::scale_row;
  using C = ring::Cfg<BT>;
  constexpr int TT = C::kTT;
  constexpr int WT = BT / 2;                      // wave tile
  extern __shared__ __align__(16) uint8_t smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31, half = lane >> 5;

  const TilePos pos = locate_tile<BT, BT>(grp);
  if (!pos.valid) return;
  const Problem& P = pos.second ? grp.p[1] : grp.p[0];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)smem;

  // Byte offset of (row r, stage s) = r * row pitch + s * stage pitch, for the
  // codes (64 bytes per row and stage) and the scales (4 bytes).
  //   row-major: codes (K/2, 64), scales (K/32, 4);
  //   K-tiled:   codes (64, rows * 64), scales (4, rows * 4).
  // Buffer resources span whole operands (fewer than 2^31 bytes, checked on the
  // host); rows past M (N) get offset 2^31, outside every resource, and load
  // zeros: code 0 contributes 0 whatever its scale.
  const bool kt = P.ktiled != 0;
  const uint32_t a_crp = kt ? 64u : (uint32_t)(P.K / 2), b_crp = a_crp;
  const uint32_t a_srp = kt ? 4u : (uint32_t)(P.K / 32), b_srp = a_srp;
  const uint32_t a_csp = kt ? (uint32_t)(P.M * 64) : 64u, b_csp = kt ? (uint32_t)(P.N * 64) : 64u;
  const uint32_t a_ssp = kt ? (uint32_t)(P.M * 4) : 4u, b_ssp = kt ? (uint32_t)(P.N * 4) : 4u;
  const v4i rsa = buffer_rsrc(P.a_codes, P.M * P.K / 2);
  const v4i rsb = buffer_rsrc(P.b_codes, P.N * P.K / 2);
  const v4i rssa = buffer_rsrc(P.a_scales, P.M * P.K / 32);
  const v4i rssb = buffer_rsrc(P.b_scales, P.N * P.K / 32);
  constexpr uint32_t kNoRow = 0x80000000u;

  // Loads of this thread. Code load j of wave w covers rows w BT/4 + 16 j ..
  // + 15 of the tile (this lane: + lane / 4, slot lane % 4). Scale load k of
  // wave w is the (w kScaleLoads + k)-th 64-row chunk of the scale areas, A's
  // chunks first, in the permuted row order of the slot layout.
  const uint32_t cunit = (uint32_t)(((lane & 3) ^ fsw(lane >> 2)) << 4);
  const int64_t sbeg = pos.kbeg / ring::kBK;       // first stage of the K window
  uint32_t a_off[C::kCodeLoads], b_off[C::kCodeLoads];
#pragma unroll
  for (int j = 0; j < C::kCodeLoads; ++j) {
    const int64_t r = wave * (BT / 4) + 16 * j + (lane >> 2);
    a_off[j] = pos.m0 + r < P.M ? (uint32_t)((pos.m0 + r) * a_crp + sbeg * a_csp) + cunit : kNoRow;
    b_off[j] = pos.n0 + r < P.N ? (uint32_t)((pos.n0 + r) * b_crp + sbeg * b_csp) + cunit : kNoRow;
  }
  uint32_t s_off[C::kScaleLoads], s_dst[C::kScaleLoads];
  bool s_is_a[C::kScaleLoads];
#pragma unroll
  for (int k = 0; k < C::kScaleLoads; ++k) {
    const int chunk = wave * C::kScaleLoads + k;      // 0 .. 2 BT/64 - 1
    const bool is_a = chunk < BT / 64;
    const int c = is_a ? chunk : chunk - BT / 64;
    const int64_t r = (is_a ? pos.m0 : pos.n0) + scale_row<TT>(c * 64 + lane);
    const bool ok = r < (is_a ? P.M : P.N);
    s_is_a[k] = is_a;
    s_off[k] = ok ? (uint32_t)(r * (is_a ? a_srp : b_srp) + sbeg * (is_a ? a_ssp : b_ssp)) : kNoRow;
    s_dst[k] = (uint32_t)(2 * C::kCode + (is_a ? 0 : C::kScale) + c * 256);
  }

  // Loads of stage s (of the K window) into slot s % 4: load q of the stage's
  // kLoads is A's code load q, B's code load q - kCodeLoads, or a scale load.
  // A stage past the end of the window goes through a null resource: every
  // load returns zeros without touching memory, into a slot nobody reads again.
  const int ksteps_all = (int)(pos.K / ring::kBK);
  const v4i rnull = buffer_rsrc(nullptr, 0);
  struct LoadRes {
    v4i a, b, sa, sb;
  };
  auto load_res = [&](int s) {
    const bool live = s < ksteps_all;
    return LoadRes{live ? rsa : rnull, live ? rsb : rnull, live ? rssa : rnull, live ? rssb : rnull};
  };
  auto issue_one = [&](int s, const LoadRes& r, int q) {
    const uint32_t slot = lds0 + (uint32_t)((s & 3) * C::kSlot);
    if (q < C::kCodeLoads) {
      lds_load_b128(r.a, a_off[q] + (uint32_t)s * a_csp, slot + wave * (BT / 4) * kRow + q * 1024);
    } else if (q < 2 * C::kCodeLoads) {
      const int j = q - C::kCodeLoads;
      lds_load_b128(r.b, b_off[j] + (uint32_t)s * b_csp, slot + C::kCode + wave * (BT / 4) * kRow + j * 1024);
    } else {
      const int k = q - 2 * C::kCodeLoads;
      lds_load_b32(s_is_a[k] ? r.sa : r.sb, s_off[k] + (uint32_t)s * (s_is_a[k] ? a_ssp : b_ssp), slot + s_dst[k]);
    }
  };
  auto issue = [&](int s) {
    const LoadRes r = load_res(s);
#pragma unroll
    for (int q = 0; q < C::kLoads; ++q) issue_one(s, r, q);
  };

  // Reads of this lane: fragment rows wm WT + 32 i + lrow (A), wn WT + 32 j + lrow (B).
  const int a_rd = (wm * WT + lrow) * kRow;
  const int b_rd = C::kCode + (wn * WT + lrow) * kRow;
  const int u0 = (half ^ fsw(lrow)) << 4;          // MX block `half` of a 64-K step
  const int u1 = ((2 + half) ^ fsw(lrow)) << 4;    // MX block 2 + half
  const int sa_rd = 2 * C::kCode + (wm * WT + lrow * TT) * 4;
  const int sb_rd = 2 * C::kCode + C::kScale + (wn * WT + lrow * TT) * 4;

  v16f acc[TT][TT];
#pragma unroll
  for (int i = 0; i < TT; ++i)
#pragma unroll
    for (int j = 0; j < TT; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  const int ksteps = ksteps_all;
  if (ksteps > 0) {
    // Fragments and scale words of one stage, both 64-K steps, in registers.
    struct StageFrags {
      uint4 a[2][TT], b[2][TT];
      ScaleRegs<TT> sa, sb;
    };
    auto read_stage = [&](int s, StageFrags& f) {
      const uint8_t* slot = smem + (s & 3) * C::kSlot;
#pragma unroll
      for (int i = 0; i < TT; ++i) f.a[0][i] = *reinterpret_cast<const uint4*>(slot + a_rd + i * 32 * kRow + u0);
#pragma unroll
      for (int j = 0; j < TT; ++j) f.b[0][j] = *reinterpret_cast<const uint4*>(slot + b_rd + j * 32 * kRow + u0);
#pragma unroll
      for (int i = 0; i < TT; ++i) f.a[1][i] = *reinterpret_cast<const uint4*>(slot + a_rd + i * 32 * kRow + u1);
#pragma unroll
      for (int j = 0; j < TT; ++j) f.b[1][j] = *reinterpret_cast<const uint4*>(slot + b_rd + j * 32 * kRow + u1);
      f.sa = read_scales<TT>(slot + sa_rd);
      f.sb = read_scales<TT>(slot + sb_rd);
    };
    auto as_frag = [](const uint4& x) { return v8i{(int)x.x, (int)x.y, (int)x.z, (int)x.w, 0, 0, 0, 0}; };
    const int sh = 8 * half;
    // Scale byte of MX block 2 kk + half of row r sits in byte 2 kk + half of
    // its dword; shifting by 8 half leaves it at byte 2 kk, which op_sel picks.
    auto mfma_step = [&](const StageFrags& f, int kk, const int (&sai)[TT], const int (&sbj)[TT]) {
#pragma unroll
      for (int i = 0; i < TT; ++i)
#pragma unroll
        for (int j = 0; j < TT; ++j)
          acc[i][j] = kk == 0 ? __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_frag(f.a[0][i]), as_frag(f.b[0][j]),
                                                                                acc[i][j], 4, 4, 0, sai[i], 0, sbj[j])
                              : __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_frag(f.a[1][i]), as_frag(f.b[1][j]),
                                                                                acc[i][j], 4, 4, 2, sai[i], 2, sbj[j]);
    };
    // One stage s: wait until this wave's reads of stage s (issued during the
    // previous stage) are done and stage s + 1 has landed, then a barrier, after
    // which every wave has read slot s % 4 and stage s + 1 is visible; then
    // stage s's 2 TT^2 MFMAs from registers, with the reads of stage s + 1 and
    // the loads of stage s + 4 (into slot s % 4) among them. So a stage's reads
    // have a whole stage of MFMAs to land, and its loads three stages. Stages
    // past the end load zeros through the null resource.
    //
    // 256 x 256 (one wave per SIMD): the order is fixed. One fragment read
    // after every second MFMA (the two scale reads two thirds through), and the
    // ten loads one after every third MFMA. Issued together at the top of the
    // stage, the loads held up the MFMAs behind them: spread out, the GEMMs of
    // the GPT-6.7B block ran 8% faster (828 -> 759 us per launch, same-box A/B).
    // Moving the loads or the scale reads by a slot changed nothing measurable.
    auto stage_fixed = [&](int s, StageFrags& cur, StageFrags& nxt) {
      wait_and_sync<2 * C::kLoads>();
      int sai[TT], sbj[TT];
#pragma unroll
      for (int i = 0; i < TT; ++i) sai[i] = (int)(cur.sa.w[i] >> sh);
#pragma unroll
      for (int j = 0; j < TT; ++j) sbj[j] = (int)(cur.sb.w[j] >> sh);
      const uint8_t* slot = smem + ((s + 1) & 3) * C::kSlot;
      const LoadRes lr = load_res(s + 4);
      // read r of stage s + 1: a[0][*], b[0][*], a[1][*], b[1][*], then the scale words
      auto read_one = [&](int r) {
        if (r < TT) nxt.a[0][r] = *reinterpret_cast<const uint4*>(slot + a_rd + r * 32 * kRow + u0);
        else if (r < 2 * TT) nxt.b[0][r - TT] = *reinterpret_cast<const uint4*>(slot + b_rd + (r - TT) * 32 * kRow + u0);
        else if (r < 3 * TT) nxt.a[1][r - 2 * TT] = *reinterpret_cast<const uint4*>(slot + a_rd + (r - 2 * TT) * 32 * kRow + u1);
        else if (r < 4 * TT) nxt.b[1][r - 3 * TT] = *reinterpret_cast<const uint4*>(slot + b_rd + (r - 3 * TT) * 32 * kRow + u1);
        else if (r == 4 * TT) nxt.sa = read_scales<TT>(slot + sa_rd);
        else nxt.sb = read_scales<TT>(slot + sb_rd);
      };
      constexpr int kMfma = 2 * TT * TT;
#pragma unroll
      for (int m = 0; m < kMfma; ++m) {
        const int kk = m / (TT * TT), i = (m % (TT * TT)) / TT, j = m % TT;
        acc[i][j] = kk == 0 ? __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_frag(cur.a[0][i]), as_frag(cur.b[0][j]),
                                                                            acc[i][j], 4, 4, 0, sai[i], 0, sbj[j])
                            : __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_frag(cur.a[1][i]), as_frag(cur.b[1][j]),
                                                                            acc[i][j], 4, 4, 2, sai[i], 2, sbj[j]);
        if (m % 3 == 1 && (m - 1) / 3 < C::kLoads) issue_one(s + 4, lr, (m - 1) / 3);
        if (m % 2 == 0 && m / 2 < 4 * TT) read_one(m / 2);
        if (m == kMfma / 2 + 1) read_one(4 * TT);
        if (m == kMfma / 2 + 3) read_one(4 * TT + 1);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // 128 x 128 (two workgroups per CU, eight MFMAs per stage): the loads at the
    // top and the compiler's own order for the rest, 3% and then 1.5-4.4%
    // faster at GPT-345M than fixed orders; spreading the loads as above changed
    // nothing there.
    auto stage_free = [&](int s, StageFrags& cur, StageFrags& nxt) {
      wait_and_sync<2 * C::kLoads>();
      issue(s + 4);
      int sai[TT], sbj[TT];
#pragma unroll
      for (int i = 0; i < TT; ++i) sai[i] = (int)(cur.sa.w[i] >> sh);
#pragma unroll
      for (int j = 0; j < TT; ++j) sbj[j] = (int)(cur.sb.w[j] >> sh);
      const uint8_t* slot = smem + ((s + 1) & 3) * C::kSlot;
#pragma unroll
      for (int i = 0; i < TT; ++i) nxt.a[0][i] = *reinterpret_cast<const uint4*>(slot + a_rd + i * 32 * kRow + u0);
#pragma unroll
      for (int j = 0; j < TT; ++j) nxt.b[0][j] = *reinterpret_cast<const uint4*>(slot + b_rd + j * 32 * kRow + u0);
      mfma_step(cur, 0, sai, sbj);
#pragma unroll
      for (int i = 0; i < TT; ++i) nxt.a[1][i] = *reinterpret_cast<const uint4*>(slot + a_rd + i * 32 * kRow + u1);
#pragma unroll
      for (int j = 0; j < TT; ++j) nxt.b[1][j] = *reinterpret_cast<const uint4*>(slot + b_rd + j * 32 * kRow + u1);
      nxt.sa = read_scales<TT>(slot + sa_rd);
      nxt.sb = read_scales<TT>(slot + sb_rd);
      mfma_step(cur, 1, sai, sbj);
      __builtin_amdgcn_sched_barrier(0);
    };
    auto stage = [&](int s, StageFrags& cur, StageFrags& nxt) {
      if constexpr (TT == 4)
        stage_fixed(s, cur, nxt);
      else
        stage_free(s, cur, nxt);
    };
    issue(0);
    issue(1);
    issue(2);
    issue(3);
    wait_and_sync<3 * C::kLoads>();
    StageFrags fr[2];
    read_stage(0, fr[0]);
    // An even number of stages, so the loop has no exit between its two
    // stages: a last stage past the end multiplies zeros, which add nothing.
    for (int s = 0; s < ksteps; s += 2) {
      stage(s, fr[0], fr[1]);
      stage(s + 1, fr[1], fr[0]);
    }
    // The null loads of the last stages write LDS too: let them land before
    // the workgroup can end.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  store_tiles<TT, TT, SS>(P, pos.split, pos.m0 + wm * WT, pos.n0 + wn * WT, acc, lane);
}

// C = alpha * (partial_0 + partial_1 + ... ) in split order, stored as
// P.store says: deterministic.
template <int STORE>
__device__ __forceinline__ void reduce_splits(const Problem& P) {
  const int64_t n = P.M * P.N;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
    float sum = P.partial[e];
    for (int s = 1; s < P.splits; ++s) sum += P.partial[(int64_t)s * n + e];
    store_elem<STORE>(P.c, e, sum * P.alpha);
  }
}

__global__ __launch_bounds__(256) void reduce_splits_kernel(Group grp) {
  for (int pi = 0; pi < grp.count; ++pi) {
    const Problem& P = grp.p[pi];
    if (P.splits <= 1) continue;
    if (P.store == (int)Store::kBf16)
      reduce_splits<(int)Store::kBf16>(P);
    else if (P.store == (int)Store::kAccF32)
      reduce_splits<(int)Store::kAccF32>(P);
    else
      reduce_splits<(int)Store::kF32>(P);
  }
}

// Kernel configurations: kRing256 / kRing128 (LDS ring, K % 128 == 0 and
// K < 2^24), kStaged (128 x 128, register-staged, any K % 32 == 0).
enum Config { kStaged = 0, kRing128 = 1, kRing256 = 2 };
constexpr int64_t kCUs = 256;

int tile_of(Config c) { return c == kRing256 ? 256 : 128; }
int stage_k(Config c) { return c == kStaged ? kStagedBK : ring::kBK; }
int64_t tiles_of(const GemmArgs& x, int bt) { return ((x.M + bt - 1) / bt) * ((x.N + bt - 1) / bt); }

// 256 x 256 tiles halve the bytes loaded per MFMA but run one workgroup per
// CU, and a tile's prologue and FP32 store cannot overlap another tile's
// MFMAs. They pay off only when the launch has at least 1.5 of them per CU
// and long reductions: measured on the GPT backward shapes, 128 x 128 tiles
// win by 20-26% at 320 256-tiles (K 1024..8192) and lose by 5% at 448; and
// they win by 13% at GPT-1.3B fc2 (1280 256-tiles, but dX's K is 2048, so a
// 256-tile stores its 256 KiB after only 16 K stages), lose by 3-10% where the
// flop-weighted mean K (sum of M N K over sum of M N) is 4096 or more.
// The ring kernels address operands with 32-bit offsets: each operand's codes
// must stay under 2^31 bytes.
Config pick_config(const GemmArgs* probs, int count) {
  constexpr int64_t kMaxBytes = int64_t(1) << 31;
  int64_t big = 0;
  double area = 0, volume = 0;
  for (int i = 0; i < count; ++i) {
    const GemmArgs& x = probs[i];
    if (x.K % ring::kBK != 0 || x.K >= ring::kMaxK || x.M * x.K / 2 >= kMaxBytes || x.N * x.K / 2 >= kMaxBytes)
      return kStaged;
    big += tiles_of(x, 256);
    area += (double)x.M * x.N;
    volume += (double)x.M * x.N * x.K;
  }
  return big >= 3 * kCUs / 2 && volume >= 4096.0 * area ? kRing256 : kRing128;
}

// Splits of K, decided for the whole launch: while the launch's workgroups do
// not cover the CUs, double the splits of every problem whose K stages allow
// it (at least `min_stages` per split), at most 8 splits.
void choose_splits(const GemmArgs* probs, int count, Config c, int* splits) {
  const int64_t bt = tile_of(c), bk = stage_k(c);
  const int64_t min_stages = c == kStaged ? 2 : 4;
  int64_t total = 0;
  for (int i = 0; i < count; ++i) {
    splits[i] = 1;
    total += tiles_of(probs[i], (int)bt);
  }
  for (int round = 0; round < 3 && total < kCUs; ++round) {
    total = 0;
    for (int i = 0; i < count; ++i) {
      const int64_t stages = (probs[i].K + bk - 1) / bk;
      if (stages / (2 * splits[i]) >= min_stages) splits[i] *= 2;
      total += tiles_of(probs[i], (int)bt) * splits[i];
    }
  }
}

Problem make_problem(const GemmArgs& x, Config c, int splits, float* partial_ws, int64_t* used) {
  Problem p{x.a_codes, x.a_scales, x.b_codes, x.b_scales, x.c, x.M, x.N, x.K, 0, 0, x.alpha, splits, x.K, nullptr,
            x.ktiled ? 1 : 0, (int)x.store};
  if (p.splits > 1) {
    const int64_t bk = stage_k(c);
    const int64_t stages = (p.K + bk - 1) / bk;
    p.kchunk = ((stages + p.splits - 1) / p.splits) * bk;
    p.splits = (int)((p.K + p.kchunk - 1) / p.kchunk);
  }
  if (p.splits > 1) {
    if (partial_ws) p.partial = partial_ws + *used / 4;
    *used += (int64_t)p.splits * p.M * p.N * 4;
  }
  const int bt = tile_of(c);
  p.tiles_n = (p.N + bt - 1) / bt;
  p.tiles = ((p.M + bt - 1) / bt) * p.tiles_n * p.splits;
  return p;
}

template <int BT, int SS>
bool launch_ring(const Group& grp, int64_t total, double flops, hipStream_t stream) {
  using C = ring::Cfg<BT>;
  static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_ring_kernel<BT, SS>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, C::kLds) == hipSuccess;
  if (!attr) return false;
  TraceScope trace(BT == 256 ? "gemm_256x256" : "gemm_128x128r", flops, true);
  hipExtLaunchKernelGGL((gemm_ring_kernel<BT, SS>), dim3((unsigned)total), dim3(kThreads), C::kLds, stream, trace.start(),
                        trace.stop(), 0, grp);
  return true;
}

int launch_group(Group grp, Config c, hipStream_t stream) {
  // Longest K window first: its tiles are dispatched first.
  if (grp.count == 2 && grp.p[1].kchunk > grp.p[0].kchunk) {
    const Problem tmp = grp.p[0];
    grp.p[0] = grp.p[1];
    grp.p[1] = tmp;
  }
  grp.start1 = (grp.p[0].tiles + kXcds - 1) / kXcds * kXcds;
  const int64_t total = grp.count == 2 && grp.p[1].tiles > 0 ? grp.start1 + grp.p[1].tiles : grp.p[0].tiles;
  bool any_split = false, kaligned = true;
  double flops = 0, red_bytes = 0;
  for (int i = 0; i < grp.count; ++i) {
    const Problem& p = grp.p[i];
    any_split = any_split || p.splits > 1;
    kaligned = kaligned && p.K % 128 == 0;
    flops += 2.0 * p.M * p.N * p.K;
    const double out_bytes = p.store == (int)Store::kBf16 ? 2.0 : p.store == (int)Store::kAccF32 ? 8.0 : 4.0;
    if (p.splits > 1) red_bytes += (4.0 * p.splits + out_bytes) * p.M * p.N;
  }
  if (total == 0) return 0;
  if (c == kRing256) {
    bool bf16 = false, acc = false;
    for (int i = 0; i < grp.count; ++i) {
      bf16 = bf16 || grp.p[i].store == (int)Store::kBf16;
      acc = acc || grp.p[i].store == (int)Store::kAccF32;
    }
    if (!(acc    ? launch_ring<256, 2>(grp, total, flops, stream)
          : bf16 ? launch_ring<256, 1>(grp, total, flops, stream)
                 : launch_ring<256, 0>(grp, total, flops, stream)))
      return -1;
  } else if (c == kRing128) {
    if (!launch_ring<128, 2>(grp, total, flops, stream)) return -1;
  } else {
    using C = Cfg<128, 128>;
    static const bool attr_a = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_f4_kernel<128, 128, true>),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, C::kLds) == hipSuccess;
    static const bool attr_b = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_f4_kernel<128, 128, false>),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, C::kLds) == hipSuccess;
    if (!attr_a || !attr_b) return -1;
    TraceScope trace("gemm_128x128", flops, true);
    if (kaligned)
      hipExtLaunchKernelGGL((gemm_f4_kernel<128, 128, true>), dim3((unsigned)total), dim3(kThreads), C::kLds, stream,
                            trace.start(), trace.stop(), 0, grp);
    else
      hipExtLaunchKernelGGL((gemm_f4_kernel<128, 128, false>), dim3((unsigned)total), dim3(kThreads), C::kLds, stream,
                            trace.start(), trace.stop(), 0, grp);
  }
  if (any_split) {
    TraceScope trace("splitk_reduce", red_bytes, false);
    hipExtLaunchKernelGGL(reduce_splits_kernel, dim3(1024), dim3(256), 0, stream, trace.start(), trace.stop(), 0,
                          grp);
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

namespace {

// Copies a row-major MXFP4 operand (codes [rows][K/2], scales [rows][K/32])
// into the K-tiled layout of the LDS-ring kernels (K % 128 == 0): for each
// 128-column stage s, codes [rows][64 B] at s * rows * 64 and scales
// [rows][4 B] at s * rows * 4. Thread x of a row moves the row's 16-byte code
// unit x (unit x holds columns 32x .. 32x + 31: stage x / 4, bytes
// 16 (x % 4) .. 16 (x % 4) + 15 of that stage's 64) and, for x < K / 128, the
// four scale bytes of stage x. A wave reads 1 KiB of one row.
__global__ __launch_bounds__(256) void ktile_repack_kernel(const uint8_t* codes, const uint8_t* scales,
                                                           uint8_t* kcodes, uint8_t* kscales, int64_t rows,
                                                           int64_t K) {
  const int64_t units = K / 32, stages = K / 128;
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    if (x < units) {
      const uint4 v = *reinterpret_cast<const uint4*>(codes + r * (K / 2) + x * 16);
      *reinterpret_cast<uint4*>(kcodes + ((x >> 2) * rows + r) * 64 + (x & 3) * 16) = v;
    }
    if (x < stages) {
      const uint8_t* src = scales + r * (K / 32) + x * 4;
      const uint32_t v = (uint32_t)src[0] | ((uint32_t)src[1] << 8) | ((uint32_t)src[2] << 16) |
                         ((uint32_t)src[3] << 24);
      *reinterpret_cast<uint32_t*>(kscales + (x * rows + r) * 4) = v;
    }
  }
}

}  // namespace

int launch_ktile_repack(const uint8_t* codes, const uint8_t* scales, uint8_t* kcodes, uint8_t* kscales,
                        int64_t rows, int64_t K, hipStream_t stream) {
  if (rows <= 0 || K <= 0) return 0;
  if (K % 128 != 0) return -1;
  const int64_t units = K / 32;
  const dim3 grid((unsigned)((units + 255) / 256), (unsigned)(rows < 8192 ? rows : 8192));
  TraceScope trace("ktile_repack", (double)rows * K * (0.5 + 1.0 / 32) * 2.0, false);
  hipExtLaunchKernelGGL(ktile_repack_kernel, grid, dim3(256), 0, stream, trace.start(), trace.stop(), 0, codes,
                        scales, kcodes, kscales, rows, K);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

bool gemm_takes_ktiled(const GemmArgs* probs, int count) {
  return count >= 1 && count <= 2 && pick_config(probs, count) != kStaged;
}

int64_t gemm_workspace_bytes(const GemmArgs* probs, int count) {
  if (count < 1 || count > 2) return 0;
  const Config c = pick_config(probs, count);
  int splits[2];
  choose_splits(probs, count, c, splits);
  int64_t used = 0;
  for (int i = 0; i < count; ++i) make_problem(probs[i], c, splits[i], nullptr, &used);
  return used;
}

// With partial_ws == NULL no problem is split (gemm_workspace_bytes() is 0
// exactly when no split is chosen).
int launch_gemm(const GemmArgs* probs, int count, float* partial_ws, hipStream_t stream) {
  if (count < 1 || count > 2) return -1;
  const Config c = pick_config(probs, count);
  for (int i = 0; i < count; ++i)
    if (probs[i].ktiled && c == kStaged) return -1;
  int splits[2] = {1, 1};
  if (partial_ws) choose_splits(probs, count, c, splits);
  Group g{};
  g.count = count;
  int64_t used = 0;
  for (int i = 0; i < count; ++i) g.p[i] = make_problem(probs[i], c, splits[i], partial_ws, &used);
  return launch_group(g, c, stream);
}

}  // namespace mx
