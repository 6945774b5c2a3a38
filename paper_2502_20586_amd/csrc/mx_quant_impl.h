// Kernel templates of the fused RHT + stochastic-rounding quantiser, shared by
// the translation units that instantiate them (one per group of quantiser
// modes, so the build compiles them in parallel). See mx_quant.hip for the
// entry point.
//
// Fused blockwise random Hadamard transform + stochastic rounding to MXFP4.
//
// Computes, for every 32-element MX block of a logical [rows, cols] bf16 matrix
// (blocks along cols), the E8M0 scale byte and 32 packed E2M1 codes, following
// the paper's unbiased quantiser (Algorithm 2) applied after the blockwise RHT
// (Sec. 3.2). The exact rules (FP32 butterfly order, E8M0 clamp, 16-bit
// dithering, Philox counter layout) are documented in include/mxfp4.h.
//
// Work layout: four lanes of a wave -- a quad -- own the g-blocks of one or two
// logical rows. Quad lane q (0..3) holds g/4 elements of each of its rows as
// g/32 chunks of 8 consecutive elements: chunk r covers block positions
// r*32 + q*8 + [0, 8). So a chunk is one Philox call's worth of noise, the four
// lanes' chunk r form exactly one MX block, and the Hadamard butterfly needs
// only two cross-lane stages (quad_perm DPP); every other stage is in registers.
//
//   stage h = 1, 2, 4        : inside a chunk (element bits)
//   stage h = 8, 16          : across the quad (lane bits 0, 1)
//   stage h = 32 .. g/2      : across chunks of one lane (chunk bits)
//
// The cross-lane stages compute own + k * partner with k = +-1 in one FMA, which
// is exact in the product and rounds the sum once, like the add or subtract
// the butterfly asks for. The sign bookkeeping this needs is folded into the
// input sign flip: quad lanes 1 and 2 start negated and end with true values.
//
// Reads. Row-major input: a quad owns one g-block of one row; each lane loads
// its chunks with 16-byte loads (8 consecutive bf16 of its row). Transposed
// input (stored [cols, rows]): a quad owns the same g-block column range of
// four adjacent logical rows, which are adjacent stored columns, so one 8-byte
// load brings one logical column of all four. A wave covers 64 logical rows:
// each of its loads reads 128 contiguous bytes of 4 stored rows. No LDS and no
// barriers are needed on either path.


#pragma once

#include "mx_device.h"
#include "mx_internal.h"

namespace mx {
namespace quant {

// ---------------------------------------------------------------------------
// A quantisation job: one operand, row-major (the logical matrix is the stored
// one) or transposed (in_t stored [cols, rows], the logical matrix is its
// transpose). Several jobs can share one launch; workgroups [wg_begin, wg_end)
// serve job j.
struct QuantJob {
  const uint16_t* in;
  uint8_t* codes;
  uint8_t* scales;
  int64_t rows, cols;
  uint64_t seed;
  int transposed;
  int load_rows; // transposed: logical rows per load (4: 8-byte loads, 2: 4-byte, 1: 2-byte)
  int codes16;   // codes 16-byte aligned (16-byte stores of staged transposed output)
  int wg_begin, wg_end;
  float* colsum; // transposed, optional: [cols / g][rows] sums of the input per g-block
  // transposed, optional: the twin, the stored matrix itself ([cols, rows],
  // blocks along rows) quantised in the same pass with its own seed, into
  // tcodes / tscales in the same output layout.
  uint8_t* tcodes;
  uint8_t* tscales;
  uint64_t tseed;
};

struct QuantJobs {
  QuantJob j[4];
  int count;
};

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

// Launch of up to four jobs in one quantiser mode (mx_quant_*.hip); 0 on
// success, -1 if the jobs do not fit the mode or the launch failed.
int launch_rht_sr(const QuantJobs& jobs, int g, bool kt, hipStream_t stream);    // QuantMode::kRhtSr
int launch_rht_sr8(const QuantJobs& jobs, int g, bool kt, hipStream_t stream);   // QuantMode::kRhtSr8
int launch_ablation(const QuantJobs& jobs, int g, bool kt, QuantMode mode, hipStream_t stream);  // the others

}  // namespace quant

namespace {

using quant::QuantJob;
using quant::QuantJobs;
using quant::kThreads;
using quant::kWaves;


// Sign bits of the g-block positions of quad lane q: byte q of word (r & 3) of
// Philox(key = (0, hi32(seed)), ctr = (r >> 2, 0, 0, 1)) holds positions
// r*32 + q*8 + 0..7 (bit e for position + e). S_j = -1 iff its bit is set.
template <int G>
__device__ __forceinline__ void sign_bytes(uint32_t seed_hi, int q, uint32_t (&byte)[G / 32]) {
  constexpr int NC = G / 32;
  const Rand4 s0 = philox4x32_10(0, 0, 0, 1, 0, seed_hi);
  Rand4 s1 = s0;
  if (NC > 4) s1 = philox4x32_10(1, 0, 0, 1, 0, seed_hi);
#pragma unroll
  for (int r = 0; r < NC; ++r) byte[r] = ((r < 4 ? s0 : s1).w[r & 3] >> (8 * q)) & 0xFFu;
}

// Quad lanes 1 and 2 start negated (see the butterfly).
__device__ __forceinline__ uint32_t lane_flip(int q) { return (q == 1 || q == 2) ? 0x80008000u : 0u; }

// Row-major reads: dword d of chunk r holds positions 2d (low half) and 2d+1
// (high half); m[r][d] flips them (bit 15 / bit 31).
template <int G, bool RHT>
__device__ __forceinline__ void sign_masks_pairs(uint32_t seed_hi, int q, uint32_t (&m)[G / 32][4]) {
  constexpr int NC = G / 32;
  if (!RHT) {
#pragma unroll
    for (int r = 0; r < NC; ++r)
#pragma unroll
      for (int d = 0; d < 4; ++d) m[r][d] = 0u;
    return;
  }
  uint32_t byte[NC];
  sign_bytes<G>(seed_hi, q, byte);
  const uint32_t flip = lane_flip(q);
#pragma unroll
  for (int r = 0; r < NC; ++r)
#pragma unroll
    for (int d = 0; d < 4; ++d)
      m[r][d] = ((((byte[r] >> (2 * d)) & 1u) << 15) | (((byte[r] >> (2 * d + 1)) & 1u) << 31)) ^ flip;
}

// Transposed reads: dword e of chunk r holds position r*32 + q*8 + e of two
// rows (low and high half); its mask flips both halves alike. Kept in registers
// for g <= 128, rebuilt from the packed bits per tile for g = 256.
template <int G, bool RHT>
__device__ __forceinline__ uint32_t sign_mask_col(const uint32_t (&byte)[G / 32], uint32_t flip, int r, int e) {
  if (!RHT) return 0u;
  return ((0u - ((byte[r] >> e) & 1u)) & 0x80008000u) ^ flip;
}

// Hadamard butterfly over the quad's g-block, stages in increasing stride.
template <int G>
__device__ __forceinline__ void butterfly(float (&v)[G / 32][8], int q) {
  constexpr int NC = G / 32;
#pragma unroll
  for (int r = 0; r < NC; ++r) {
#pragma unroll
    for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (e & h) continue;
        const float a = v[r][e], b = v[r][e + h];
        v[r][e] = a + b;
        v[r][e + h] = a - b;
      }
    }
  }
  // Cross-lane stages h = 8 and 16: v = fma(partner's v, k, v) with the partner
  // read through DPP inside the FMA (V_FMAC_F32 with quad_perm). A DPP read of a
  // register needs two wait states after the VALU write of it; the s_nop covers
  // the writes before the block, and inside it each register is read again
  // eight instructions after it was written.
  const float k1 = (q & 1) ? 1.0f : -1.0f;
  const float k2 = (q & 2) ? 1.0f : -1.0f;
#pragma unroll
  for (int r = 0; r < NC; ++r) {
#define MX_DPP1(i) "v_fmac_f32_dpp %" #i ", %" #i ", %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
#define MX_DPP2(i) "v_fmac_f32_dpp %" #i ", %" #i ", %9 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
    asm("s_nop 1\n\t" MX_DPP1(0) MX_DPP1(1) MX_DPP1(2) MX_DPP1(3) MX_DPP1(4) MX_DPP1(5) MX_DPP1(6) MX_DPP1(7)
        MX_DPP2(0) MX_DPP2(1) MX_DPP2(2) MX_DPP2(3) MX_DPP2(4) MX_DPP2(5) MX_DPP2(6) MX_DPP2(7)
        : "+v"(v[r][0]), "+v"(v[r][1]), "+v"(v[r][2]), "+v"(v[r][3]), "+v"(v[r][4]), "+v"(v[r][5]),
          "+v"(v[r][6]), "+v"(v[r][7])
        : "v"(k1), "v"(k2));
#undef MX_DPP1
#undef MX_DPP2
  }
#pragma unroll
  for (int hc = 1; hc < NC; hc <<= 1) {
#pragma unroll
    for (int r = 0; r < NC; ++r) {
      if (r & hc) continue;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float a = v[r][e], b = v[r + hc][e];
        v[r][e] = a + b;
        v[r + hc][e] = a - b;
      }
    }
  }
}

// Stochastic rounding to E2M1 with CDNA4's converter V_CVT_SCALEF32_SR_PK_FP4_F32
// (scale 1) on a register pair (w_2i, w_2i+1). It rounds |w| up iff
// floor(t * 2^22) + R >= 2^22, where t is |w|'s position between its two
// neighbouring E2M1 values and R is a 22-bit field of the seed operand: bits
// 31..10 for the value in the first slot, bits 30..9 for the second. A 16-bit
// noise value r placed so that R = r << 6 (seed r << 16 for the first slot,
// r << 15 for the second) gives a carry that depends only on
// floor(t * 2^16) + r: exactly the rounding rule of include/mxfp4.h. Each pair
// is converted twice, once with the even element's seed (its code lands in the
// low nibble) and once with the odd element's (high nibble); the other nibble
// of each result is discarded. The converter writes one byte of its
// destination, chosen by op_sel, and keeps the other three: the accumulator is
// read and written, which the compiler builtin does not model, hence inline
// assembly. A register written by the converter is read again no sooner than
// two instructions later (the even and odd conversions alternate), and the
// closing s_nop covers the first read after the block.
typedef float v2f __attribute__((ext_vector_type(2)));
typedef uint32_t v2u32 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void sr_convert(const v2f (&w)[4], const uint32_t (&se)[4], const uint32_t (&so)[4],
                                           uint32_t* even, uint32_t* odd) {
  uint32_t e, o;
  asm volatile(
      "v_cvt_scalef32_sr_pk_fp4_f32 %0, %2, %6, 1.0\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %1, %2, %7, 1.0\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %0, %3, %8, 1.0 op_sel:[0,0,1,0]\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %1, %3, %9, 1.0 op_sel:[0,0,1,0]\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %0, %4, %10, 1.0 op_sel:[0,0,0,1]\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %1, %4, %11, 1.0 op_sel:[0,0,0,1]\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %0, %5, %12, 1.0 op_sel:[0,0,1,1]\n\t"
      "v_cvt_scalef32_sr_pk_fp4_f32 %1, %5, %13, 1.0 op_sel:[0,0,1,1]\n\t"
      "s_nop 0"
      : "=&v"(e), "=&v"(o)
      : "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(se[0]), "v"(so[0]), "v"(se[1]), "v"(so[1]), "v"(se[2]),
        "v"(so[2]), "v"(se[3]), "v"(so[3]));
  *even = e;
  *odd = o;
}

// One MX block (chunk r of the quad): E8M0 scale, then 8 codes of this lane.
// Returns the packed codes (element e in bits 4e..4e+3); *scale gets the byte.
// NB, the dither's noise bits: 16, Algorithm 2 (3/4 pre-scale, stochastic
// rounding) with the 16-bit noise of the chunk's own Philox call; 8, the same
// with the cheaper 8-bit noise, bytes 8 h .. 8 h + 7 of the call `rnd8` that
// serves this chunk (h = 0) and the one 32 columns further (h = 1); 0,
// Algorithm 1 (no 3/4, round to nearest with ties to the even code,
// saturation at 6).
template <int NB>
__device__ __forceinline__ uint32_t quantise_chunk(const float (&y)[8], uint64_t chunk_index,
                                                   uint32_t seed_lo, uint32_t seed_hi, uint32_t* scale,
                                                   const Rand4& rnd8 = Rand4{}, int h = 0) {
  // Block maximum of |y| on the bit patterns. As unsigned integers, patterns
  // with the sign bit set sort above all others and among themselves by
  // magnitude; as signed integers, non-negative patterns sort by magnitude
  // above all negative ones. So the unsigned maximum (sign cleared) is the
  // largest magnitude of a negative value if there is one, the signed maximum
  // the largest non-negative pattern, and the larger of the two is max |y|.
  // NaN patterns sort above infinity either way.
  uint32_t b[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(y[e]);
  const uint32_t um = max(max(max(b[0], b[1]), max(b[2], b[3])), max(max(b[4], b[5]), max(b[6], b[7])));
  const int32_t sm = max(max(max((int32_t)b[0], (int32_t)b[1]), max((int32_t)b[2], (int32_t)b[3])),
                         max(max((int32_t)b[4], (int32_t)b[5]), max((int32_t)b[6], (int32_t)b[7])));
  uint32_t m = (uint32_t)max((int32_t)(um & 0x7FFFFFFFu), sm);
  // Maximum over the quad: unsigned max with the partner's value read through
  // DPP (two wait states after each write of m before its DPP read).
  asm("s_nop 1\n\t"
      "v_max_u32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\t"
      "v_max_u32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf"
      : "+v"(m));
  const uint32_t efield = m >> 23;
  // shared_exp = floor(log2 amax) - 2, as a biased E8M0 byte, clamped at 0.
  const uint32_t ebyte = max(efield, 2u) - 2u;
  uint32_t packed;
  if constexpr (NB == 0) {
    // v = y / 2^shared_exp, an exact power-of-two scaling (finite blocks have
    // ebyte <= 252, so the factor is a normal float); the converter rounds to
    // nearest even and saturates.
    const float c = __uint_as_float((254u - ebyte) << 23);
    packed = 0u;
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, y[0] * c, y[1] * c, 1.0f, 0);
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, y[2] * c, y[3] * c, 1.0f, 1);
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, y[4] * c, y[5] * c, 1.0f, 2);
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, y[6] * c, y[7] * c, 1.0f, 3);
  } else {
    // c = (3/4) 2^-shared_exp = 1.5 * 2^(126 - ebyte): always a normal float.
    const float c = __uint_as_float(((253u - ebyte) << 23) | 0x400000u);
    v2f w[4];
    uint32_t se[4], so[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = v2f{y[2 * i] * c, y[2 * i + 1] * c};  // (3/4) y / X, one rounding each
    if constexpr (NB == 16) {
      // Noise: word i of the chunk's Philox block serves elements 2i (low
      // half) and 2i + 1 (high half).
      const Rand4 rnd = philox4x32_10((uint32_t)chunk_index, (uint32_t)(chunk_index >> 32), 0, 0,
                                      seed_lo, seed_hi);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        se[i] = rnd.w[i] << 16;
        so[i] = (rnd.w[i] >> 16) << 15;
      }
    } else {
      // 8-bit noise: element e takes byte e & 3 of word 2 h + (e >> 2). With
      // R = r << 14 the converter's rule floor(t 2^22) + R >= 2^22 is exactly
      // floor(t 2^8) + r >= 2^8: seed r << 24 (first slot), r << 23 (second).
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t wd = h ? rnd8.w[2 + (i >> 1)] : rnd8.w[i >> 1];
        se[i] = (i & 1) ? (wd << 8) & 0xFF000000u : wd << 24;
        so[i] = (i & 1) ? (wd >> 1) & 0x7F800000u : (wd << 15) & 0x7F800000u;
      }
    }
    // Byte i of `even` holds element 2i's code in its low nibble, byte i of
    // `odd` element 2i + 1's code in its high nibble.
    uint32_t even, odd;
    sr_convert(w, se, so, &even, &odd);
    packed = (even & 0x0F0F0F0Fu) | (odd & 0xF0F0F0F0u);
  }
  // A zero magnitude always gets code 0: clear the sign bit of nibbles whose
  // magnitude bits are all zero (the add carries into bit 3 of every nibble
  // with a nonzero magnitude).
  packed &= ((packed & 0x77777777u) + 0x77777777u) | 0x77777777u;
  // Inf or NaN in the block: flagged, codes cleared.
  const bool nonfinite = efield == 255u;
  *scale = nonfinite ? 0xFFu : ebyte;
  return nonfinite ? 0u : packed;
}


// Store the 8 codes (one dword) of the chunk whose first element is logical
// (row, col), and, from one lane of the quad, the block's scale byte.
// Row-major output (the C ABI's): codes [rows][cols/2], scales [rows][cols/32].
// K-tiled output (KT, written only for the GEMM's LDS-ring kernels, which take
// operands whose codes are under 2^31 bytes and whose K is a multiple of 128):
// the codes of stage s (logical columns 128s .. 128s + 127) of all rows form a
// [rows][64 B] block at s * rows * 64, the scales a [rows][4 B] block at
// s * rows * 4. Every K-tiled offset fits in 32 bits.
template <bool KT>
__device__ __forceinline__ void store_chunk(const QuantJob& job, int64_t row, int64_t col, uint32_t packed,
                                            uint32_t sbyte, bool scale_lane) {
  if constexpr (KT) {
    const uint32_t rows = (uint32_t)job.rows, c = (uint32_t)col, r = (uint32_t)row;
    const uint32_t st = c >> 7, cc = c & 127u;
    *reinterpret_cast<uint32_t*>(job.codes + (st * rows * 64u + r * 64u + (cc >> 1))) = packed;
    if (scale_lane) job.scales[st * rows * 4u + r * 4u + (cc >> 5)] = (uint8_t)sbyte;
  } else {
    const int64_t flat = row * job.cols + col;
    *reinterpret_cast<uint32_t*>(job.codes + (flat >> 1)) = packed;
    if (scale_lane) job.scales[flat >> 5] = (uint8_t)sbyte;
  }
}

// Row-major input: g | cols, so g-blocks never straddle rows and every address
// is a flat element index. A quad walks g-blocks b = first, first + stride, ...;
// its (row, block-in-row) pair advances by the grid stride's quotient and
// remainder, so no division runs inside the loop. For g <= 64 the next block's
// loads are issued before the current block is quantised.
template <int G, bool RHT, int NB, bool KT>
__device__ __forceinline__ void rows_body(const QuantJob& job, int64_t wg, int64_t nwg) {
  constexpr int NC = G / 32;
  static_assert(NB != 8 || NC % 2 == 0, "8-bit noise pairs chunk r with chunk r + 1 (g >= 64)");
  constexpr bool kPrefetch = NC <= 2;
  const int q = threadIdx.x & 3;
  const uint32_t seed_lo = (uint32_t)job.seed, seed_hi = (uint32_t)(job.seed >> 32);
  uint32_t smask[NC][4];
  sign_masks_pairs<G, RHT>(seed_hi, q, smask);
  const int64_t bpr = job.cols / G;      // g-blocks per row
  const int64_t total = job.rows * bpr;
  const int64_t qpw = kThreads / 4;      // quads per workgroup
  const int64_t stride = nwg * qpw;
  const int64_t drow = stride / bpr, dcb = stride - drow * bpr;
  int64_t b = wg * qpw + (threadIdx.x >> 2);
  int64_t row = b / bpr, cb = b - row * bpr;
  auto load = [&](int64_t blk, uint4 (&raw)[NC]) {
    const uint16_t* src = job.in + blk * G + q * 8;
#pragma unroll
    for (int r = 0; r < NC; ++r) raw[r] = *reinterpret_cast<const uint4*>(src + r * 32);
  };
  // Quantise the g-block b whose input is in raw, then step to the next block.
  auto block = [&](const uint4 (&raw)[NC]) {
    float v[NC][8];
#pragma unroll
    for (int r = 0; r < NC; ++r) {
      const uint32_t w[4] = {raw[r].x ^ smask[r][0], raw[r].y ^ smask[r][1], raw[r].z ^ smask[r][2],
                             raw[r].w ^ smask[r][3]};
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        v[r][2 * d] = __uint_as_float(w[d] << 16);
        v[r][2 * d + 1] = __uint_as_float(w[d] & 0xFFFF0000u);
      }
    }
    if (RHT) butterfly<G>(v, q);
    const int64_t col0 = cb * G + q * 8;
    const uint64_t chunk0 = (uint64_t)(b * G + q * 8) >> 3;
    Rand4 rnd8{};
#pragma unroll
    for (int r = 0; r < NC; ++r) {
      // 8-bit noise: one Philox call for chunks r and r + 1 (r even), the
      // counter of chunk r's 16-bit draw.
      if (NB == 8 && (r & 1) == 0)
        rnd8 = philox4x32_10((uint32_t)(chunk0 + 4 * r), (uint32_t)((chunk0 + 4 * r) >> 32), 0, 0, seed_lo, seed_hi);
      uint32_t sbyte;
      const uint32_t packed = quantise_chunk<NB>(v[r], chunk0 + 4 * r, seed_lo, seed_hi, &sbyte, rnd8, r & 1);
      store_chunk<KT>(job, row, col0 + r * 32, packed, sbyte, q == (r & 3));
    }
    b += stride;
    row += drow;
    cb += dcb;
    if (cb >= bpr) {
      cb -= bpr;
      ++row;
    }
  };
  if constexpr (kPrefetch) {
    // Two buffers in turn (the loop body is unrolled twice), so the prefetched
    // block is never copied between registers.
    uint4 ra[NC], rb[NC];
    if (b < total) load(b, ra);
    while (b < total) {
      if (b + stride < total) load(b + stride, rb);
      block(ra);
      if (b >= total) break;
      if (b + stride < total) load(b + stride, ra);
      block(rb);
    }
  } else {
    while (b < total) {
      uint4 raw[NC];
      load(b, raw);
      block(raw);
    }
  }
}

// Transposed input, stored [cols, rows]. Quad k of a wave owns RPQ adjacent
// logical rows (adjacent stored columns), so a wave tile is TR = 16 RPQ logical
// rows by g logical columns (g stored rows), and lane q loads, for each of its
// g/4 logical columns, the RPQ bf16 values of its rows in one load: 8 bytes
// (RPQ = 4: every load instruction of the wave reads 128 contiguous bytes of
// each of 4 stored rows) or 4 bytes (RPQ = 2). LW2 false: rows is odd or the
// input is not 4-byte aligned, so the two values of a pair are loaded
// separately. The rows are then processed a pair at a time (the low and high
// halves of each loaded 32-bit word).
//
// Output goes through LDS. The four waves of a workgroup take the four
// consecutive g-blocks of one row tile (a workgroup tile: TR rows by 4 g
// columns) and put their codes and scale bytes into a staging buffer laid out
// [row][4 g/2 code bytes] and [row][4 g/32 scale bytes]; after a barrier the
// workgroup writes the buffer out as whole 16-byte code units (one contiguous
// run of 2 g bytes per row, or of 64 bytes per row and 128-column stage,
// contiguous over the rows, when K-tiled) and scale bytes (dwords when
// K-tiled). Written directly, each store instruction would touch 16 rows with
// 16 bytes (or one byte) each. 16-byte code units of a staged row are
// XOR-swizzled by the quad index so that the quads' writes spread over the
// banks. Two buffers alternate, so one barrier per tile suffices: a wave
// refills a buffer only after every wave has passed the following tile's
// barrier, i.e. has written that buffer out. Workgroup tiles are walked with
// the row tile fastest, so neighbouring workgroups read adjacent pieces of the
// same stored rows.
template <int G>
struct ColsCfg {
  static constexpr int kRpqMax = G <= 64 ? 4 : 2;       // rows per quad with 8-byte loads
  static constexpr int kCodeRow = 4 * G / 2;           // staged code bytes per row
  static constexpr int kScaleRow = 4 * G / 32;         // staged scale bytes per row
  static constexpr int kUnits = kCodeRow / 16;         // 16-byte code units per row
  static constexpr int kSwz = kUnits < 8 ? kUnits - 1 : 7;
  static constexpr int kBuf = 16 * kRpqMax * (kCodeRow + kScaleRow);
  static constexpr int kLds = 2 * kBuf;
};

// CS: the job also wants colsum, the sum of each logical row's input values
// (bf16, before the sign flip) over each g-block, in FP32: every lane sums its
// g/4 values of a row in chunk-then-element order, the quad adds the four lane
// sums as (q0 + q1) + (q2 + q3), and lane q stores row RPQ k + q's sum.
//
// TW: the job also quantises its twin (see QuantJob) -- the same input, stored
// [cols, rows], along its stored rows. After writing a tile out, the workgroup
// quantises the twin's blocks that lie in the tile it has just read (its
// g-block group's stored rows and its TR stored columns), from the cache: the
// input is read from memory once for both outputs. Each quad takes blocks
// b = quad, quad + 64, ... of the tile's (stored row, column block) pairs and
// runs the row-major path's arithmetic on them, so the twin's codes and scales
// are exactly those of a row-major job on the stored matrix. Needs TR % G == 0
// (RPQ = 4, g <= 64) and stored rows whose length is a multiple of 8.
template <int G, bool RHT, int NB, bool KT, int RPQ, bool LW2, bool CS = false, bool TW = false>
__device__ __forceinline__ void cols_body(const QuantJob& job, int64_t wg, int64_t nwg, uint8_t* smem) {
  using CC = ColsCfg<G>;
  constexpr int NC = G / 32;
  static_assert(NB != 8 || NC % 2 == 0, "8-bit noise pairs chunk r with chunk r + 1 (g >= 64)");
  constexpr int NP = RPQ / 2;                  // row pairs per quad
  constexpr int TR = 16 * RPQ;                 // logical rows per tile
  constexpr bool kMaskRegs = G <= 128;
  constexpr bool kPrefetch = NC * NP <= 2;
  const int tid = threadIdx.x, lane = tid & 63, q = lane & 3, k = lane >> 2;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t seed_lo = (uint32_t)job.seed, seed_hi = (uint32_t)(job.seed >> 32);
  uint32_t sbits[NC];
  if (RHT) {
    sign_bytes<G>(seed_hi, q, sbits);
  } else {
#pragma unroll
    for (int r = 0; r < NC; ++r) sbits[r] = 0u;
  }
  const uint32_t flip = RHT ? lane_flip(q) : 0u;
  uint32_t smask[kMaskRegs ? NC : 1][8];
  if (kMaskRegs) {
#pragma unroll
    for (int r = 0; r < NC; ++r)
#pragma unroll
      for (int e = 0; e < 8; ++e) smask[r][e] = sign_mask_col<G, RHT>(sbits, flip, r, e);
  }
  // The twin: its row-major sign masks and seed, and a job view of its output
  // (the stored matrix, [cols, rows]).
  const uint32_t tseed_lo = (uint32_t)job.tseed, tseed_hi = (uint32_t)(job.tseed >> 32);
  uint32_t tmask[TW ? NC : 1][4];
  QuantJob twin{};
  if constexpr (TW) {
    sign_masks_pairs<G, RHT>(tseed_hi, q, tmask);
    twin.codes = job.tcodes;
    twin.scales = job.tscales;
    twin.rows = job.cols;
    twin.cols = job.rows;
  }
  const int64_t rows = job.rows, cols = job.cols;
  const int64_t rtiles = (rows + TR - 1) / TR;
  const int64_t ktiles = cols / G;
  const int64_t ntiles = rtiles * ((ktiles + kWaves - 1) / kWaves);   // workgroup tiles
  const int64_t dkg = nwg / rtiles, drt = nwg - dkg * rtiles;
  int64_t t = wg;
  int64_t kg = t / rtiles, rt = t - kg * rtiles;   // this wave's g-block: kg * kWaves + wave
  // Element offset of this lane's first load inside a tile: logical column
  // q * 8 (a stored row), logical row RPQ k (a stored column).
  const int64_t lane_off = (int64_t)q * 8 * rows + RPQ * k;
  // Loads of 8 (RPQ = 4) or 4 bytes (RPQ = 2, LW2) go through a raw buffer
  // resource that starts at the g-block's first stored row: the lane's part of
  // the offset is a 32-bit VGPR, the stored row's an SGPR, so a load costs no
  // address arithmetic, and lanes whose logical rows are past `rows` take
  // offset 2^31, outside the resource, and read zeros without a branch. This
  // needs the block's (g + 1) stored rows under 2^31 bytes; larger inputs take
  // the pointer loads below.
  constexpr bool kBufLoads = RPQ == 4 || LW2;
  const bool buf_ok = kBufLoads && (int64_t)(G + 1) * rows * 2 < (int64_t(1) << 31);
  const int64_t total_bytes = rows * cols * 2;
  auto load = [&](int64_t rt_, int64_t kt_, uint32_t (&raw)[NC][8][NP]) {
    const int64_t ra = rt_ * TR + RPQ * k;
    if (kBufLoads && buf_ok) {
      const int64_t blk = (kt_ * G) * rows * 2;            // byte offset of the block's first stored row
      const int64_t left = total_bytes - blk;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint8_t*>(reinterpret_cast<const uint8_t*>(job.in)) + blk, (short)0,
          (int)(left < 0x7FFFFFFF ? left : 0x7FFFFFFF), 0x00020000);
      const uint32_t voff = ra < rows ? (uint32_t)((rt_ * TR + lane_off) * 2) : 0x80000000u;
#pragma unroll
      for (int r = 0; r < NC; ++r)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int soff = (int)((int64_t)(r * 32 + e) * rows * 2);
          if constexpr (RPQ == 4) {
            const v2u32 v = __builtin_amdgcn_raw_buffer_load_b64(rs, (int)voff, soff, 0);
            raw[r][e][0] = v.x;
            raw[r][e][NP - 1] = v.y;
          } else {
            raw[r][e][0] = __builtin_amdgcn_raw_buffer_load_b32(rs, (int)voff, soff, 0);
          }
        }
      return;
    }
    const uint16_t* src = job.in + (kt_ * G) * rows + rt_ * TR + lane_off;
#pragma unroll
    for (int r = 0; r < NC; ++r)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint16_t* p = src + (int64_t)(r * 32 + e) * rows;
        if constexpr (RPQ == 4) {
          const uint2 v = ra < rows ? *reinterpret_cast<const uint2*>(p) : make_uint2(0u, 0u);
          raw[r][e][0] = v.x;
          raw[r][e][NP - 1] = v.y;
        } else if constexpr (LW2) {
          raw[r][e][0] = ra < rows ? *reinterpret_cast<const uint32_t*>(p) : 0u;
        } else {
          const uint32_t lo = ra < rows ? (uint32_t)p[0] : 0u;
          const uint32_t hi = ra + 1 < rows ? (uint32_t)p[1] : 0u;
          raw[r][e][0] = lo | (hi << 16);
        }
      }
  };
  uint32_t nxt[NC][8][NP];
  if (kPrefetch && t < ntiles && kg * kWaves + wave < ktiles) load(rt, kg * kWaves + wave, nxt);
  for (int it = 0; t < ntiles; t += nwg, ++it) {
    uint8_t* codes_lds = smem + (it & 1) * CC::kBuf;
    uint8_t* scales_lds = codes_lds + TR * CC::kCodeRow;
    const int64_t kt = kg * kWaves + wave;
    int64_t rt2 = rt + drt, kg2 = kg + dkg;
    if (rt2 >= rtiles) {
      rt2 -= rtiles;
      ++kg2;
    }
    // A row tile's last group may hold fewer than 4 g-blocks: waves past the
    // last one only take part in the barrier and the write-out.
    const bool active = kt < ktiles;
    uint32_t raw[NC][8][NP];
    if (active) {
      if (kPrefetch) {
#pragma unroll
        for (int r = 0; r < NC; ++r)
#pragma unroll
          for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int p = 0; p < NP; ++p) raw[r][e][p] = nxt[r][e][p];
      } else {
        load(rt, kt, raw);
      }
    }
    if (kPrefetch && t + nwg < ntiles && kg2 * kWaves + wave < ktiles) load(rt2, kg2 * kWaves + wave, nxt);
    if (active) {
      const int64_t col0 = kt * G + q * 8;
      if constexpr (CS) {
        float sum[RPQ];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
          for (int r = 0; r < NC; ++r)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              s0 += __uint_as_float(raw[r][e][p] << 16);
              s1 += __uint_as_float(raw[r][e][p] & 0xFFFF0000u);
            }
          s0 += quad_swap<kQuadXor1>(s0);
          s1 += quad_swap<kQuadXor1>(s1);
          sum[2 * p] = s0 + quad_swap<kQuadXor2>(s0);
          sum[2 * p + 1] = s1 + quad_swap<kQuadXor2>(s1);
        }
        float mine = sum[0];
#pragma unroll
        for (int i = 1; i < RPQ; ++i) mine = q == i ? sum[i] : mine;
        const int64_t row = rt * TR + RPQ * k + q;
        if (q < RPQ && row < rows) job.colsum[kt * rows + row] = mine;
      }
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        float v[2][NC][8];
#pragma unroll
        for (int r = 0; r < NC; ++r)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const uint32_t w = raw[r][e][p] ^
                               (kMaskRegs ? smask[kMaskRegs ? r : 0][e] : sign_mask_col<G, RHT>(sbits, flip, r, e));
            v[0][r][e] = __uint_as_float(w << 16);
            v[1][r][e] = __uint_as_float(w & 0xFFFF0000u);
          }
        if (RHT) {
          butterfly<G>(v[0], q);
          butterfly<G>(v[1], q);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int lr = RPQ * k + 2 * p + i;          // row inside the tile
          const int64_t row = rt * TR + lr;
          const uint64_t chunk0 = (uint64_t)(row * cols + col0) >> 3;
          Rand4 rnd8{};
#pragma unroll
          for (int r = 0; r < NC; ++r) {
            if (NB == 8 && (r & 1) == 0)
              rnd8 = philox4x32_10((uint32_t)(chunk0 + 4 * r), (uint32_t)((chunk0 + 4 * r) >> 32), 0, 0, seed_lo,
                                   seed_hi);
            uint32_t sbyte;
            const uint32_t packed =
                quantise_chunk<NB>(v[i][r], chunk0 + 4 * r, seed_lo, seed_hi, &sbyte, rnd8, r & 1);
            const int unit = wave * NC + r;            // 16-byte code unit of this chunk in the staged row
            *reinterpret_cast<uint32_t*>(codes_lds + lr * CC::kCodeRow + ((unit ^ (k & CC::kSwz)) << 4) + 4 * q) =
                packed;
            if (q == (r & 3)) scales_lds[lr * CC::kScaleRow + wave * NC + r] = (uint8_t)sbyte;
          }
        }
      }
    }
    __syncthreads();
    // Write the tile out. nk g-blocks exist in this group, rows past `rows`
    // are skipped.
    const int64_t nk = min((int64_t)kWaves, ktiles - kg * kWaves);
    const int64_t row0 = rt * TR;
    const int64_t kcol0 = kg * kWaves * G;             // first logical column of the group
    const int units = (int)nk * NC;                    // code units per row that exist
    for (int idx = tid; idx < TR * CC::kUnits; idx += kThreads) {
      const int lr = idx / CC::kUnits, u = idx - lr * CC::kUnits;
      const int64_t row = row0 + lr;
      if (u >= units || row >= rows) continue;
      const uint4 val = *reinterpret_cast<const uint4*>(codes_lds + lr * CC::kCodeRow +
                                                         ((u ^ ((lr / RPQ) & CC::kSwz)) << 4));
      const int64_t col = kcol0 + (int64_t)u * 32;
      if constexpr (KT) {
        const uint32_t c = (uint32_t)col;
        uint8_t* dst = job.codes + ((c >> 7) * (uint32_t)rows * 64u + (uint32_t)row * 64u + ((c & 127u) >> 1));
        *reinterpret_cast<uint4*>(dst) = val;
      } else {
        uint8_t* dst = job.codes + ((row * cols + col) >> 1);
        if (job.codes16) {
          *reinterpret_cast<uint4*>(dst) = val;
        } else {
          uint32_t* d = reinterpret_cast<uint32_t*>(dst);
          d[0] = val.x;
          d[1] = val.y;
          d[2] = val.z;
          d[3] = val.w;
        }
      }
    }
    if constexpr (KT) {
      // 4 scale bytes per row and 128-column stage: one dword.
      constexpr int kWords = CC::kScaleRow / 4;
      for (int idx = tid; idx < TR * kWords; idx += kThreads) {
        const int st = idx / TR, lr = idx - st * TR;
        const int64_t row = row0 + lr;
        if (st * 4 >= units || row >= rows) continue;
        const uint32_t c = (uint32_t)(kcol0 + (int64_t)st * 128);
        const uint32_t val = *reinterpret_cast<const uint32_t*>(scales_lds + lr * CC::kScaleRow + 4 * st);
        *reinterpret_cast<uint32_t*>(job.scales + ((c >> 7) * (uint32_t)rows * 4u + (uint32_t)row * 4u)) = val;
      }
    } else {
      for (int idx = tid; idx < TR * CC::kScaleRow; idx += kThreads) {
        const int lr = idx / CC::kScaleRow, bi = idx - lr * CC::kScaleRow;
        const int64_t row = row0 + lr;
        if (bi >= units || row >= rows) continue;
        job.scales[(row * cols + kcol0) / 32 + bi] = scales_lds[lr * CC::kScaleRow + bi];
      }
    }
    if constexpr (TW) {
      static_assert(TR % G == 0, "twin blocks must not straddle row tiles");
      constexpr int kBpt = TR / G;                      // twin blocks per stored row of the tile
      const int64_t srow0 = kcol0;                      // first stored row of the tile
      const int64_t nblk = min(nk * G, cols - srow0) * kBpt;
      for (int64_t b = tid >> 2; b < nblk; b += kThreads / 4) {
        const int64_t srow = srow0 + b / kBpt;
        const int64_t scol = row0 + (b % kBpt) * G;     // first stored column of the block
        if (scol >= rows) continue;                     // rows % G == 0: a block is whole or absent
        const uint16_t* src = job.in + srow * rows + scol + q * 8;
        uint4 raw2[NC];
#pragma unroll
        for (int r = 0; r < NC; ++r) raw2[r] = *reinterpret_cast<const uint4*>(src + r * 32);
        float v2[NC][8];
#pragma unroll
        for (int r = 0; r < NC; ++r) {
          const uint32_t w[4] = {raw2[r].x ^ tmask[r][0], raw2[r].y ^ tmask[r][1], raw2[r].z ^ tmask[r][2],
                                 raw2[r].w ^ tmask[r][3]};
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            v2[r][2 * d] = __uint_as_float(w[d] << 16);
            v2[r][2 * d + 1] = __uint_as_float(w[d] & 0xFFFF0000u);
          }
        }
        if (RHT) butterfly<G>(v2, q);
        const uint64_t chunk0 = (uint64_t)(srow * rows + scol + q * 8) >> 3;
        Rand4 rnd8{};
#pragma unroll
        for (int r = 0; r < NC; ++r) {
          if (NB == 8 && (r & 1) == 0)
            rnd8 = philox4x32_10((uint32_t)(chunk0 + 4 * r), (uint32_t)((chunk0 + 4 * r) >> 32), 0, 0, tseed_lo,
                                 tseed_hi);
          uint32_t sbyte;
          const uint32_t packed = quantise_chunk<NB>(v2[r], chunk0 + 4 * r, tseed_lo, tseed_hi, &sbyte, rnd8, r & 1);
          store_chunk<KT>(twin, srow, scol + q * 8 + r * 32, packed, sbyte, q == (r & 3));
        }
      }
    }
    rt = rt2;
    kg = kg2;
  }
}

// CS: the launch holds a job that wants column sums (its own instantiation,
// so that the extra registers of that path do not cost the others occupancy).
// g <= 64 fits 128 VGPRs: four waves per SIMD to hide the loads' latency
// behind the VALU work of the others.
// TW likewise for a launch that holds a job with a twin (g <= 64, at
// load_rows == 4; at most one such job per launch in practice, the dY^T of a
// backward pass, which may also sum its input).
template <int G, bool RHT, int NB, bool KT, bool CS, bool TW>
__global__ __launch_bounds__(kThreads, G <= 64 ? 4 : 1) void quant_kernel(QuantJobs jobs) {
  extern __shared__ __align__(16) uint8_t smem[];
  int j = 0;
#pragma unroll
  for (int i = 1; i < 4; ++i)
    if (i < jobs.count && (int)blockIdx.x >= jobs.j[i].wg_begin) j = i;
  const QuantJob& job = jobs.j[j];
  const int64_t wg = (int64_t)blockIdx.x - job.wg_begin;
  const int64_t nwg = job.wg_end - job.wg_begin;
  if (!job.transposed)
    rows_body<G, RHT, NB, KT>(job, wg, nwg);
  else if (TW && job.tcodes && job.colsum)
    cols_body<G, RHT, NB, KT, 4, true, true, TW>(job, wg, nwg, smem);
  else if (TW && job.tcodes)
    cols_body<G, RHT, NB, KT, 4, true, false, TW>(job, wg, nwg, smem);
  else if (CS && job.colsum)   // launch_jobs_g admits colsum jobs only at load_rows == kRpqMax
    cols_body<G, RHT, NB, KT, ColsCfg<G>::kRpqMax, true, CS>(job, wg, nwg, smem);
  else if (job.load_rows == 4)
    cols_body<G, RHT, NB, KT, ColsCfg<G>::kRpqMax, true>(job, wg, nwg, smem);
  else if (job.load_rows == 2)
    cols_body<G, RHT, NB, KT, 2, true>(job, wg, nwg, smem);
  else
    cols_body<G, RHT, NB, KT, 2, false>(job, wg, nwg, smem);
}

// Kernel names for tracing: g-block size, "_nr" for round to nearest, "_sr8"
// for 8-bit noise; "sr" / "nr" alone without the RHT.
template <int G, bool RHT, int NB>
const char* quant_name() {
  if (!RHT) return NB ? "quant_sr" : "quant_nr";
  if (NB == 16) return G == 32 ? "quant_g32" : G == 64 ? "quant_g64" : G == 128 ? "quant_g128" : "quant_g256";
  if (NB == 8) return G == 64 ? "quant_g64_sr8" : G == 128 ? "quant_g128_sr8" : "quant_g256_sr8";
  return G == 32 ? "quant_g32_nr" : G == 64 ? "quant_g64_nr" : G == 128 ? "quant_g128_nr" : "quant_g256_nr";
}

template <int G, bool RHT, int NB, bool KT>
int launch_jobs_g(QuantJobs jobs, hipStream_t stream) {
  constexpr int64_t kMaxWgPerJob = 256 * 8;
  int wg = 0;
  for (int i = 0; i < jobs.count; ++i) {
    QuantJob& jb = jobs.j[i];
    // Four rows per quad only where the registers allow it (g <= 64).
    if (G > 64 && jb.load_rows == 4) jb.load_rows = 2;
    if (jb.colsum && jb.load_rows != ColsCfg<G>::kRpqMax) return -1;
    // A twin needs four rows per quad (g <= 64) and 16-byte loads along the
    // stored rows (rows % 8 == 0, 16-byte aligned input).
    if (jb.tcodes && (G > 64 || !jb.transposed || jb.load_rows != 4 || jb.rows % 8 != 0 || jb.rows % G != 0 ||
                      reinterpret_cast<uintptr_t>(jb.in) % 16 != 0))
      return -1;
    int64_t need;
    if (!jb.transposed) {
      const int64_t nblocks = jb.rows * (jb.cols / G);
      need = (nblocks + kThreads / 4 - 1) / (kThreads / 4);
    } else {
      const int64_t tr = jb.load_rows == 4 ? 64 : 32;   // logical rows per wave tile
      need = ((jb.rows + tr - 1) / tr) * ((jb.cols / G + kWaves - 1) / kWaves);   // workgroup tiles
    }
    if (need > kMaxWgPerJob) need = kMaxWgPerJob;
    jb.wg_begin = wg;
    wg += (int)need;
    jb.wg_end = wg;
  }
  if (wg == 0) return 0;
  // Algorithmic bytes: a twin adds its codes and scales, not another read.
  double bytes = 0;
  for (int i = 0; i < jobs.count; ++i)
    bytes += (double)jobs.j[i].rows * jobs.j[i].cols * (2.0 + (jobs.j[i].tcodes ? 2.0 : 1.0) * (0.5 + 1.0 / 32));
  TraceScope trace(quant_name<G, RHT, NB>(), bytes, false);
  bool any_t = false;
  for (int i = 0; i < jobs.count; ++i) any_t = any_t || jobs.j[i].transposed;
  bool any_cs = false, any_tw = false;
  for (int i = 0; i < jobs.count; ++i) any_cs = any_cs || jobs.j[i].colsum != nullptr;
  for (int i = 0; i < jobs.count; ++i) any_tw = any_tw || jobs.j[i].tcodes != nullptr;
  const int lds = any_t ? ColsCfg<G>::kLds : 0;
  if constexpr (G <= 64) {
    if (any_tw) {
      if (any_cs)
        hipExtLaunchKernelGGL((quant_kernel<G, RHT, NB, KT, true, true>), dim3((unsigned)wg), dim3(kThreads), lds,
                              stream, trace.start(), trace.stop(), 0, jobs);
      else
        hipExtLaunchKernelGGL((quant_kernel<G, RHT, NB, KT, false, true>), dim3((unsigned)wg), dim3(kThreads), lds,
                              stream, trace.start(), trace.stop(), 0, jobs);
      return hipGetLastError() == hipSuccess ? 0 : -1;
    }
  }
  if (any_cs)
    hipExtLaunchKernelGGL((quant_kernel<G, RHT, NB, KT, true, false>), dim3((unsigned)wg), dim3(kThreads), lds,
                          stream, trace.start(), trace.stop(), 0, jobs);
  else
    hipExtLaunchKernelGGL((quant_kernel<G, RHT, NB, KT, false, false>), dim3((unsigned)wg), dim3(kThreads), lds,
                          stream, trace.start(), trace.stop(), 0, jobs);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <bool RHT, int NB, bool KT>
int launch_jobs_mode(const QuantJobs& jobs, int g, hipStream_t stream) {
  if constexpr (!RHT) {
    return launch_jobs_g<32, false, NB, KT>(jobs, stream);   // MX blocks of 32, no g-blocks
  } else if constexpr (NB == 8) {
    switch (g) {   // pairs of 32-element chunks: g >= 64
      case 64: return launch_jobs_g<64, true, 8, KT>(jobs, stream);
      case 128: return launch_jobs_g<128, true, 8, KT>(jobs, stream);
      case 256: return launch_jobs_g<256, true, 8, KT>(jobs, stream);
      default: return -1;
    }
  } else {
    switch (g) {
      case 32: return launch_jobs_g<32, true, NB, KT>(jobs, stream);
      case 64: return launch_jobs_g<64, true, NB, KT>(jobs, stream);
      case 128: return launch_jobs_g<128, true, NB, KT>(jobs, stream);
      case 256: return launch_jobs_g<256, true, NB, KT>(jobs, stream);
      default: return -1;
    }
  }
}

}  // namespace
}  // namespace mx
