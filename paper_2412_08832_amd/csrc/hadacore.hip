// hadacore.hip -- batched normalized Walsh-Hadamard transform for gfx950.
//
// Computes out[i][j] = scale * sum_k (-1)^popcount(j & k) * in[i][k] for
// 16-bit rows of length n = 2^L, 0 <= L <= 16 in one pass (HadaCore, arXiv
// 2412.08832: the transform of Sec. 2.1-2.2, sizes of Sec. 3.2 -- 2^7 to 2^15
// -- plus the smaller ones and 2^16, in place per Appendix B, fp16 and bf16
// per Appendix C), and up to 2^20 in two passes through a workspace.
// Rows of n <= 8 are one per thread (fwht_row_kernel), or, when n <= 4 and the
// rows are dense, 8/n rows per thread (fwht_dense_kernel); the tile structure
// below applies from n = 16.
//
// Structure of one launch.  The radix-2 stages of the fast transform (Sec.
// 2.2) act on the bits of the element index, one stage per bit, and stages on
// different bits commute.  Each lane holds C chunks of 8 consecutive 16-bit
// elements (one 16-byte global access each), widened to fp32 registers.  For
// a tile of 512*C*NW elements the tile index of register (chunk k, element j)
// of lane l in wave w is
//     t = ((w*C + k)*64 + l)*8 + j,
// so bits 0-2 of t live inside a lane, bits 3-8 across the 64 lanes of a
// wave, the next log2(C) bits across a lane's chunks and the top log2(NW)
// bits across the waves of a workgroup.  Stages are executed where their bit
// lives:
//   * chunk and in-chunk bits: register butterflies (a, b) -> (a+b, a-b);
//   * lane bits: the partner lane's value arrives by DPP (xor 1, xor 2 by
//     quad_perm; xor 8 by row_ror:8, fused into one v_fmac_f32_dpp), by
//     ds_swizzle (xor 4, xor 16) or by ds_bpermute (xor 32).  After the
//     matrix-core front a change of basis replaces xor 4 with xor 7
//     (row_half_mirror), so all its lane stages are DPP, and moves where each
//     lane stores (lane_stages, lane_frequency);
//   * wave bits (n > 512*C): an LDS exchange swaps the wave bits with the low
//     chunk bits, after which they are register butterflies too.  The store
//     uses the exchanged layout, so there is no exchange back.
// Global loads and stores are 16-byte per lane and 1 KiB contiguous per wave
// instruction in every layout.
//
// Lane-bit butterflies are computed in "twisted" form: every lane forms
// self + sign * partner with sign = -1 on the lane whose bit is set, which is
// one fused instruction and leaves that lane holding the negated difference.
// The negation is tracked per lane (it depends only on which lane bits were
// processed) and undone by flipping sign bits of the packed 16-bit results.
//
// Two front ends do the first stages on the raw 16-bit data (see "front
// ends" below): fp32 VALU butterflies, or one radix-32 step as a pair of
// MFMA 16x16x32 products -- the paper's Tensor-Core idea (Sec. 3) on CDNA4
// matrix cores, applied to the exact 16-bit inputs only.  Per size the
// dispatcher uses whichever measured faster.
//
// Numerics: inputs are scaled before any addition (the VALU front multiplies
// while widening; the MFMA front puts the power-of-two part of the scale into
// its H_32 operand and applies the rest at the end), so large bf16 rows do
// not overflow fp32 partial sums.  Every intermediate is fp32 and the result
// is rounded once, round-to-nearest-even.
//
// Where this differs from the paper's kernel: the paper chains 16x16
// Tensor-Core products with fp16/bf16 intermediates and transposes between
// them (Sec. 3.1-3.2); here only the first step may use the matrix cores,
// everything after it is fp32 VALU butterflies with wave64 DPP and LDS
// exchanges, which keeps one rounding, and the kernel is HBM-bound.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <mutex>

#include "hadacore.h"

namespace hadacore {
namespace {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

// ---- global memory --------------------------------------------------------------

// 16-byte loads and stores; NT selects the nontemporal (streaming) cache policy.
template <bool NT>
__device__ __forceinline__ u4 gload(const uint16_t *p) {
  const u4 *q = reinterpret_cast<const u4 *>(p);
  if constexpr (NT) {
    return __builtin_nontemporal_load(q);
  } else {
    return *q;
  }
}

template <bool NT>
__device__ __forceinline__ void gstore(uint16_t *p, u4 v) {
  u4 *q = reinterpret_cast<u4 *>(p);
  if constexpr (NT) {
    __builtin_nontemporal_store(v, q);
  } else {
    *q = v;
  }
}

// The same at base + byte offset.  With a wave-uniform base and a 32-bit
// offset this is one global access with the base in scalar registers and no
// per-lane 64-bit address arithmetic.
template <bool NT>
__device__ __forceinline__ u4 gload_at(const void *base, uint32_t off) {
  return gload<NT>(reinterpret_cast<const uint16_t *>(static_cast<const char *>(base) + off));
}

template <bool NT>
__device__ __forceinline__ void gstore_at(void *base, uint32_t off, u4 v) {
  gstore<NT>(reinterpret_cast<uint16_t *>(static_cast<char *>(base) + off), v);
}

// Output stores from a wave-uniform base.  With SC1, a nontemporal store also
// sets the SC1 cache-policy bit, which plain C++ cannot ask for, so it goes
// out as a raw buffer store (a buffer resource over the 4 GiB from the base,
// so no range check applies) with the policy NT | SC1.  Measured on MI355X
// against plain nontemporal stores (interleaved, same box, bit-identical
// outputs): +1.5% to +3.3% for the wave kernel (n <= 512) and the n <= 8
// kernels, +1% to +2.2% in place at n = 2048-8192, 0 to +2.7% for the
// quantized outputs, +1.8% for the device copy; but -0.2% to -4% for 16-bit
// rows of 16384 elements and more, which keep plain nontemporal stores.  A
// store instruction that leaves part of a 128-byte line unwritten is costly
// with SC1 (-9% to -18% for unaligned strided rows), so the dispatcher asks
// for it only where every store writes whole lines (whole_lines).  The cache
// bits of the loads made no difference.  `base` must be the same in every
// lane of the wave: it is read from the first active lane.
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer resource word 3 on gfx9: 32-bit data format
constexpr int kPolicyNtSc1 = 2 | 16;    // buffer cache-policy operand: NT (bit 1) | SC1 (bit 4)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void *base) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void *>((hi << 32) | lo), (short)0,
                                           -1, kRsrcWord3);
}

// 16-byte nontemporal load from a wave-uniform base as a raw buffer load (same
// cache policy as gload_at).  Used by the row loops, where it measured +0.7% to
// +1.3% at n = 65536 against the global load (the uniform part of the address
// stays in scalar registers).
constexpr int kPolicyNt = 2;  // buffer cache-policy operand: NT (bit 1)

__device__ __forceinline__ u4 gload_u(const void *base, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(uniform_rsrc(base), (int)off, 0, kPolicyNt);
}

template <bool NT, bool SC1>
__device__ __forceinline__ void gstore_u(void *base, uint32_t off, u4 v) {
  if constexpr (NT && SC1) {
    __builtin_amdgcn_raw_buffer_store_b128(v, uniform_rsrc(base), (int)off, 0, kPolicyNtSc1);
  } else {
    gstore_at<NT>(base, off, v);
  }
}

// ---- 16-bit <-> fp32 ------------------------------------------------------

// Widens the packed pair in `u` (element 2i in the low half), multiplies by
// the scale and applies the radix-2 stage on element bit 0 (the pair itself):
// returns (s*lo + s*hi, s*lo - s*hi).
template <int DT>
__device__ __forceinline__ f2 widen_stage0(uint32_t u, float s) {
  float lo, hi;
  if constexpr (DT == HADACORE_FP16) {
    const f2 p = __builtin_convertvector(__builtin_bit_cast(h2, u), f2) * s;
    lo = p.x;
    hi = p.y;
    return f2{lo + hi, lo - hi};
  } else {
    lo = __builtin_bit_cast(float, u << 16);
    hi = __builtin_bit_cast(float, u & 0xffff0000u);
    const float t = hi * s;
    return f2{__builtin_fmaf(lo, s, t), __builtin_fmaf(lo, s, -t)};
  }
}

// Rounds a pair to the 16-bit dtype (round-to-nearest-even), packs it and
// flips both sign bits when `flip` is 0x80008000.
template <int DT>
__device__ __forceinline__ uint32_t narrow(float lo, float hi, uint32_t flip) {
  const f2 v = {lo, hi};
  uint32_t r;
  if constexpr (DT == HADACORE_FP16) {
    r = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
  } else {
    r = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf2));
  }
  return r ^ flip;
}

// ---- butterflies ------------------------------------------------------------

// Radix-2 stage on bit B of the register index (register r = chunk*8 + element).
template <int B, int N>
__device__ __forceinline__ void reg_stage(float (&v)[N]) {
  constexpr int h = 1 << B;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if ((i & h) == 0) {
      const float a = v[i];
      const float b = v[i + h];
      v[i] = a + b;
      v[i + h] = a - b;
    }
  }
}

// Twisted lane stage through DPP, 8 registers per asm block:
//   v = dpp(v) * sgn + v   (v_fmac_f32_dpp).
// The leading s_nop 1 provides the two wait states that a DPP read needs after
// a VALU write of the same VGPR; inside the block each instruction reads a
// register that no earlier instruction of the block wrote.
#define HC_FMAC_DPP8(CTRL)                                                                     \
  asm("s_nop 1\n\t"                                                                            \
      "v_fmac_f32_dpp %0, %0, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %1, %1, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %2, %2, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %3, %3, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %4, %4, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %5, %5, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %6, %6, %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"                       \
      "v_fmac_f32_dpp %7, %7, %8 " CTRL " row_mask:0xf bank_mask:0xf"                           \
      : "+v"(v[i]), "+v"(v[i + 1]), "+v"(v[i + 2]), "+v"(v[i + 3]), "+v"(v[i + 4]),             \
        "+v"(v[i + 5]), "+v"(v[i + 6]), "+v"(v[i + 7])                                          \
      : "v"(sgn))

// Radix-2 stage on lane bit LB in twisted form: each lane keeps
// self + sgn * partner with sgn = -1 where the lane bit is set.
template <int LB, int N>
__device__ __forceinline__ void lane_stage(float (&v)[N], int lane) {
  static_assert(N % 8 == 0, "registers come in chunks of 8");
  const float sgn = __builtin_bit_cast(
      float, 0x3F800000u | (((uint32_t)lane << (31 - LB)) & 0x80000000u));  // -1 iff bit LB
  if constexpr (LB == 0) {
#pragma unroll
    for (int i = 0; i < N; i += 8) HC_FMAC_DPP8("quad_perm:[1,0,3,2]");
  } else if constexpr (LB == 1) {
#pragma unroll
    for (int i = 0; i < N; i += 8) HC_FMAC_DPP8("quad_perm:[2,3,0,1]");
  } else if constexpr (LB == 3) {
#pragma unroll
    for (int i = 0; i < N; i += 8) HC_FMAC_DPP8("row_ror:8");
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      // 128 registers per lane (n = 65536): issue the LDS-path permutes in
      // groups of 16 so that their results do not pile up in registers
      if constexpr (N >= 128) {
        if (i % 16 == 0 && i > 0) __builtin_amdgcn_sched_barrier(0);
      }
      const int x = __builtin_bit_cast(int, v[i]);
      int p;
      if constexpr (LB == 2) {
        p = __builtin_amdgcn_ds_swizzle(x, 0x101F);             // bitmask mode, xor 4
      } else if constexpr (LB == 4) {
        p = __builtin_amdgcn_ds_swizzle(x, 0x401F);             // bitmask mode, xor 16
      } else {
        p = __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, x);  // xor 32
      }
      v[i] = __builtin_fmaf(__builtin_bit_cast(float, p), sgn, v[i]);
    }
  }
}

// Lane stages over the lane bits in MASK.  With DUAL (the matrix-core front)
// lane bits 0-2 are all done by DPP.  There is no DPP pattern for
// partner l ^ 4, but row_half_mirror gives l ^ 7, and the butterflies of a
// Walsh-Hadamard transform may run along any basis of the index space: with
// partners l ^ b for b = 1, 2, 7 and lane l "high" in the stage along b_i
// where <psi_i, l> is odd, psi_i being the dual basis (masks 5, 6, 4), lane p
// ends up holding (-1)^popcount(p & 7) * y[j(p)] with
// j(p) = (p0^p2, p1^p2, p0^p1^p2) on bits 0-2 (lane_frequency).  The sign is
// the usual twist; j only moves where a lane's result is stored.  Higher lane
// bits keep their own stages (xor 8 by DPP, xor 16 and 32 through the LDS
// unit).  The VALU front keeps the swizzle for xor 4: there it runs beside
// the VALU in the LDS unit, and the extra DPP stage measured 1% slower.
template <int PHI>
__device__ __forceinline__ float dual_sign(int lane) {
  const uint32_t odd = (uint32_t)__builtin_popcount(lane & PHI) & 1u;
  return __builtin_bit_cast(float, 0x3F800000u | (odd << 31));
}

template <int MASK, bool DUAL, int N>
__device__ __forceinline__ void lane_stages(float (&v)[N], int lane) {
  static_assert(N % 8 == 0, "registers come in chunks of 8");
  if constexpr (DUAL && (MASK & 7) == 7) {
    {
      const float sgn = dual_sign<5>(lane);
#pragma unroll
      for (int i = 0; i < N; i += 8) HC_FMAC_DPP8("quad_perm:[1,0,3,2]");
    }
    {
      const float sgn = dual_sign<6>(lane);
#pragma unroll
      for (int i = 0; i < N; i += 8) HC_FMAC_DPP8("quad_perm:[2,3,0,1]");
    }
    {
      const float sgn = dual_sign<4>(lane);
#pragma unroll
      for (int i = 0; i < N; i += 8) HC_FMAC_DPP8("row_half_mirror");
    }
  } else {
    if constexpr (MASK & 1) lane_stage<0>(v, lane);
    if constexpr (MASK & 2) lane_stage<1>(v, lane);
    if constexpr (MASK & 4) lane_stage<2>(v, lane);
  }
  if constexpr (MASK & 8) lane_stage<3>(v, lane);
  if constexpr (MASK & 16) lane_stage<4>(v, lane);
  if constexpr (MASK & 32) lane_stage<5>(v, lane);
}

// Lane position p (bits 0-5) -> the index of the transform output it holds
// after lane_stages<MASK, DUAL>.
template <int MASK, bool DUAL>
__device__ __forceinline__ int lane_frequency(int p) {
  if constexpr (DUAL && (MASK & 7) == 7) {
    const int p2 = (p >> 2) & 1;
    const int b0 = (p & 1) ^ p2;
    const int b1 = ((p >> 1) & 1) ^ p2;
    return b0 | (b1 << 1) | ((b0 ^ b1 ^ p2) << 2) | (p & ~7);
  } else {
    return p;
  }
}

// ---- front ends: the stages applied to the raw 16-bit data ----------------------
//
// kValu: each lane widens its 16-byte chunk (8 consecutive elements) to fp32,
//   multiplies by the scale and runs the butterflies on element bits 0-2 in
//   registers; lane l holds tile bits 3-8 equal to l.
// kMfma: the radix-32 step on tile bits 0-4 is one pair of 16x16x32 MFMAs on
//   the raw 16-bit data (the Tensor-Core idea of the paper's Sec. 3, as a
//   32-point product on CDNA4 matrix cores).  Lane l loads chunk (l >> 4) of
//   the 32-element vector pi(l & 15) -- exactly the MFMA B-operand layout --
//   and the A operands are the top and bottom 16 rows of H_32 times 2^e, which
//   are exact in 16 bits.  The fp32 products come back as element 4(l>>4)+i
//   and 16+4(l>>4)+i of the lane's vector; one v_permlane16_swap per register
//   pair turns that into 8 consecutive elements, 8*hsel(l >> 4) onwards, so
//   stores stay 16 bytes per lane.  What remains are the vector bits (tile
//   bits 5-8, on lane bits 0-3) and the chunk and wave bits; the result is
//   multiplied by scale / 2^e at the end.
constexpr int kValu = 0;
constexpr int kMfma = 1;

// Vector index (tile bits 5-8) held by lane l in the MFMA layout.  For n = 256
// the vector's third bit sits on lane bit 3 so that all three element-carrying
// lane bits are DPP lanes (xor 1, 2, 8); otherwise the identity.
template <int L>
__device__ __forceinline__ int mfma_vector(int l) {
  l &= 15;
  if constexpr (L == 8) l = (l & 3) | ((l & 4) << 1) | ((l & 8) >> 1);
  return l;
}

// Tile bits 3-8 of the chunk lane l loads / holds after the front end.
template <int FRONT, int L>
__device__ __forceinline__ int lane_field_load(int l) {
  if constexpr (FRONT == kValu) {
    return l;
  } else {
    return 4 * mfma_vector<L>(l) + (l >> 4);
  }
}

// Lane bits that carry element bits still to be processed after the front end
// (a mask over lane bits 0-5).
template <int FRONT, int L>
constexpr int lane_stage_mask() {
  if constexpr (FRONT == kValu) {
    return (1 << (L - 3 >= 6 ? 6 : L - 3)) - 1;
  } else {
    return L == 7 ? 0x3 : (L == 8 ? 0xB : 0xF);
  }
}

// Tile bits 3-8 whose transform outputs lane l holds after all lane stages
// (the store layout; lane_frequency moves bits 0-2 after the basis change).
// DUAL must match the wave_stages call of the same kernel.
template <int FRONT, int L, bool DUAL = FRONT == kMfma>
__device__ __forceinline__ int lane_field(int l) {
  constexpr int mask = lane_stage_mask<FRONT, L>();
  if constexpr (FRONT == kValu) {
    return lane_frequency<mask, DUAL>(l);
  } else {
    const int g = l >> 4;
    return 4 * lane_frequency<mask, DUAL>(mfma_vector<L>(l)) +
           (((g & 1) << 1) | (g >> 1));  // hsel = {0, 2, 1, 3}
  }
}

// A lane holds negated values iff an odd number of its processed lane bits are set.
template <int FRONT, int L>
__device__ __forceinline__ bool twisted(int lane) {
  return (__builtin_popcount(lane & lane_stage_mask<FRONT, L>()) & 1) != 0;
}

// Widen + scale + stage on bit 0 for all registers (kValu front).
template <int DT, int C>
__device__ __forceinline__ void widen_chunks(const u4 (&raw)[C], float (&v)[C * 8], float s) {
#pragma unroll
  for (int k = 0; k < C; ++k) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f2 p = widen_stage0<DT>(raw[k][q], s);
      v[k * 8 + 2 * q] = p.x;
      v[k * 8 + 2 * q + 1] = p.y;
    }
  }
}

// MFMA A operands: lane l holds 8 consecutive 16-bit entries, columns
// 8*(l >> 4) .. +7, of row (l & 15) (top) and of row 16 + (l & 15) (bottom) of
// H_32 * 2^e, where H_32[r][c] = (-1)^popcount(r & c).  The sign bits depend
// on the lane only and come from a 2 KiB table (words 0-3 top, 4-7 bottom);
// the magnitude 2^e (fp16: 1) is OR-ed in per call.
struct H32Signs {
  uint32_t w[kWave][8];
};

constexpr int parity_of(int x) {
  int p = 0;
  for (; x != 0; x &= x - 1) p ^= 1;
  return p;
}

constexpr H32Signs make_h32_signs() {
  H32Signs t{};
  for (int l = 0; l < kWave; ++l) {
    for (int half = 0; half < 2; ++half) {
      const int r = 16 * half + (l & 15);
      for (int q = 0; q < 4; ++q) {
        const int c = 8 * (l >> 4) + 2 * q;
        t.w[l][4 * half + q] = (parity_of(r & c) ? 0x8000u : 0u) |
                               (parity_of(r & (c + 1)) ? 0x80000000u : 0u);
      }
    }
  }
  return t;
}

__device__ const H32Signs kH32Signs = make_h32_signs();

template <int DT>
__device__ __forceinline__ void h32_operands(int lane, int e2, u4 &top, u4 &bot) {
  const uint32_t one = DT == HADACORE_FP16 ? 0x3C00u : (uint32_t)(0x3F80 + e2 * 128);
  const uint32_t mag = one | (one << 16);
  const u4 *p = reinterpret_cast<const u4 *>(kH32Signs.w[lane]);
  top = p[0] | mag;
  bot = p[1] | mag;
}

// Radix-32 step of one chunk on the matrix cores (kMfma front).
template <int DT>
__device__ __forceinline__ void mfma_front(u4 raw, u4 a_top, u4 a_bot, float *v) {
  const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  f4 top, bot;
  if constexpr (DT == HADACORE_FP16) {
    top = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a_top),
                                                 __builtin_bit_cast(h8, raw), zero, 0, 0, 0);
    bot = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a_bot),
                                                 __builtin_bit_cast(h8, raw), zero, 0, 0, 0);
  } else {
    top = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a_top),
                                                  __builtin_bit_cast(bf8, raw), zero, 0, 0, 0);
    bot = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a_bot),
                                                  __builtin_bit_cast(bf8, raw), zero, 0, 0, 0);
  }
  // Bit-cast whole vectors: __builtin_bit_cast of a single ext-vector element
  // reads element 0 in this compiler.
  const u4 tu = __builtin_bit_cast(u4, top);
  const u4 bu = __builtin_bit_cast(u4, bot);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const auto s = __builtin_amdgcn_permlane16_swap(tu[i], bu[i], false, false);
    v[i] = __builtin_bit_cast(float, (uint32_t)s[0]);
    v[4 + i] = __builtin_bit_cast(float, (uint32_t)s[1]);
  }
}

// The front end for all chunks of a lane.
template <int DT, int FRONT, int C>
__device__ __forceinline__ void front(const u4 (&raw)[C], float (&v)[C * 8], int lane, float scale,
                                      int e2) {
  if constexpr (FRONT == kValu) {
    widen_chunks<DT, C>(raw, v, scale);
    reg_stage<1>(v);
    reg_stage<2>(v);
  } else {
    u4 a_top, a_bot;
    h32_operands<DT>(lane, e2, a_top, a_bot);
#pragma unroll
    for (int k = 0; k < C; ++k) mfma_front<DT>(raw[k], a_top, a_bot, &v[k * 8]);
  }
}

// The remaining stages inside one wave: the chunk bits that are element bits
// (tile bits 9.. below L) and the lane bits that still carry element bits.
// DUAL selects the all-DPP lane stages (lane_stages); by default the
// matrix-core front uses them and the VALU front does not.
template <int FRONT, int L, int C, bool DUAL = FRONT == kMfma, int N>
__device__ __forceinline__ void wave_stages(float (&v)[N], int lane) {
  static_assert(C == 1 || C == 2 || C == 4 || C == 8 || C == 16, "1 to 16 chunks per lane");
  if constexpr (C >= 2 && L > 9) reg_stage<3>(v);
  if constexpr (C >= 4 && L > 10) reg_stage<4>(v);
  if constexpr (C >= 8 && L > 11) reg_stage<5>(v);
  if constexpr (C >= 16 && L > 12) reg_stage<6>(v);
  lane_stages<lane_stage_mask<FRONT, L>(), DUAL>(v, lane);
}

// Undo the twist (and, for kMfma, apply the part of the scale the front end
// left out), round once and pack 8 elements.
template <int DT, int FRONT>
struct Finisher {
  uint32_t flip;
  float post;
  __device__ __forceinline__ Finisher(bool tw, float post_scale) {
    if constexpr (FRONT == kValu) {
      flip = tw ? 0x80008000u : 0u;
      post = 1.0f;
    } else {
      flip = 0u;
      post = tw ? -post_scale : post_scale;
    }
  }
  __device__ __forceinline__ u4 operator()(const float *v) const {
    float w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = FRONT == kValu ? v[i] : v[i] * post;
    u4 r;
    r.x = narrow<DT>(w[0], w[1], flip);
    r.y = narrow<DT>(w[2], w[3], flip);
    r.z = narrow<DT>(w[4], w[5], flip);
    r.w = narrow<DT>(w[6], w[7], flip);
    return r;
  }
};

// Scale arguments: kValu multiplies by `scale` while widening; kMfma puts 2^e2
// into the H_32 operand and multiplies by `post` = scale / 2^e2 at the end.
struct ScaleArgs {
  float scale;
  float post;
  int e2;
};

// ---- fused FP8 epilogue ------------------------------------------------------------
//
// The transform followed by per-row quantization (the fused transform +
// quantization the paper names as future work, Sec. 5), with
// amax = max_j |y_j| (NaN ignored unless the row is all NaN) and Q = 448 (OCP
// FP8 e4m3) or 127 (symmetric INT8):
//   s = amax / Q,  code_j = round(y_j * inv),  inv = Q / amax,
// the divisions and the product correctly rounded in fp32.  FP8 rounds to
// e4m3 (to nearest even) and takes inv = 0 where Q / amax is not finite (a
// zero or NaN row, or amax < Q * 2^-128); INT8 rounds half to even to an
// integer in [-127, 127] and gives those rows, and rows whose amax is Inf,
// all-zero codes.  y ~ code * s.

constexpr int kStore16 = 0;  // 16-bit output in the input dtype
constexpr int kFp8 = 1;      // e4m3 codes + one fp32 scale per row
constexpr int kInt8 = 2;     // int8 codes + one fp32 scale per row

struct QuantOut {
  uint8_t *codes;
  int64_t stride;  // bytes between rows of codes
  float *scales;   // one per row
};

typedef uint32_t u2 __attribute__((ext_vector_type(2)));

// Maximum of x over the lanes that differ from this one only in the lane
// bits of MASK.  Every operand is a result of arithmetic, so NaNs are quiet
// and a plain v_max_f32 -- which returns the number when the other operand is
// a quiet NaN -- is the maxNum of the definition.  It is written in asm so
// that the compiler adds no canonicalizing v_max per step; the DPP forms fold
// the exchange into the max.  The leading s_nop 1 gives the two wait states a
// DPP read needs after a VALU write of its register.  Requires all lanes active.
#define HC_MAX_DPP(CTRL) \
  asm("s_nop 1\n\tv_max_f32_dpp %0, %0, %0 " CTRL " row_mask:0xf bank_mask:0xf" : "+v"(x))

__device__ __forceinline__ float max_with(float x, int partner_bits) {
  asm("v_max_f32 %0, %0, %1" : "+v"(x) : "v"(partner_bits));
  return x;
}

template <int MASK>
__device__ __forceinline__ float lane_max(float x, int lane) {
  if constexpr ((MASK & 1) != 0) HC_MAX_DPP("quad_perm:[1,0,3,2]");
  if constexpr ((MASK & 2) != 0) HC_MAX_DPP("quad_perm:[2,3,0,1]");
  if constexpr ((MASK & 4) != 0)
    x = max_with(x, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x101F));  // xor 4
  if constexpr ((MASK & 8) != 0) HC_MAX_DPP("row_ror:8");                                 // xor 8
  if constexpr ((MASK & 16) != 0)
    x = max_with(x, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));  // xor 16
  if constexpr ((MASK & 32) != 0)
    x = max_with(x, __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, __builtin_bit_cast(int, x)));
  return x;
}
#undef HC_MAX_DPP

// Lane bits along which one row's elements are spread after the stages.
template <int FRONT, int L>
constexpr int row_lane_mask() {
  return FRONT == kValu ? lane_stage_mask<kValu, L>() : (lane_stage_mask<kMfma, L>() | 0x30);
}

// max |v[j]| over 8 registers (maxNum: quiet NaNs lose), 4 instructions.
__device__ __forceinline__ float abs_max8(const float *v) {
  float a;
  asm("v_max3_f32 %0, |%1|, |%2|, |%3|" : "=v"(a) : "v"(v[0]), "v"(v[1]), "v"(v[2]));
  asm("v_max3_f32 %0, %0, |%1|, |%2|" : "+v"(a) : "v"(v[3]), "v"(v[4]));
  asm("v_max3_f32 %0, %0, |%1|, |%2|" : "+v"(a) : "v"(v[5]), "v"(v[6]));
  asm("v_max_f32_e64 %0, %0, |%1|" : "+v"(a) : "v"(v[7]));
  return a;
}

// 8 values times `mul` to 8 e4m3 codes, round-to-nearest-even (v_cvt_pk_fp8_f32).
__device__ __forceinline__ u2 to_e4m3x8(const float *v, float mul) {
  int lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[0] * mul, v[1] * mul, 0, false);
  lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[2] * mul, v[3] * mul, lo, true);
  int hi = __builtin_amdgcn_cvt_pk_fp8_f32(v[4] * mul, v[5] * mul, 0, false);
  hi = __builtin_amdgcn_cvt_pk_fp8_f32(v[6] * mul, v[7] * mul, hi, true);
  return u2{(uint32_t)lo, (uint32_t)hi};
}

// 8 values times `mul` to 8 int8 codes, round half to even, AND-ed with `keep`
// (0 clears the codes of a row without a usable scale).  q + 1.5 * 2^23 rounds
// q (|q| <= 127) to an integer in the low mantissa bits, whose low byte is the
// two's-complement code.  The product is rounded before the addition, as in
// the definition, so contraction into an fma is switched off.
__device__ __forceinline__ u2 to_int8x8(const float *v, float mul, uint32_t keep) {
#pragma clang fp contract(off)
  uint32_t b[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) b[j] = __builtin_bit_cast(uint32_t, v[j] * mul + 12582912.0f);
  // byte j of the result is the low byte of b[j]
  const uint32_t p01 = __builtin_amdgcn_perm(b[1], b[0], 0x0C0C0400u);
  const uint32_t p23 = __builtin_amdgcn_perm(b[3], b[2], 0x0C0C0400u);
  const uint32_t p45 = __builtin_amdgcn_perm(b[5], b[4], 0x0C0C0400u);
  const uint32_t p67 = __builtin_amdgcn_perm(b[7], b[6], 0x0C0C0400u);
  return u2{__builtin_amdgcn_perm(p23, p01, 0x05040100u) & keep,
            __builtin_amdgcn_perm(p67, p45, 0x05040100u) & keep};
}

template <bool NT>
__device__ __forceinline__ void gstore8_at(void *base, uint32_t off, u2 v) {
  u2 *q = reinterpret_cast<u2 *>(static_cast<char *>(base) + off);
  if constexpr (NT) {
    __builtin_nontemporal_store(v, q);
  } else {
    *q = v;
  }
}

// 8-byte output store from a wave-uniform base (see gstore_u).
template <bool NT, bool SC1>
__device__ __forceinline__ void gstore8_u(void *base, uint32_t off, u2 v) {
  if constexpr (NT && SC1) {
    __builtin_amdgcn_raw_buffer_store_b64(v, uniform_rsrc(base), (int)off, 0, kPolicyNtSc1);
  } else {
    gstore8_at<NT>(base, off, v);
  }
}

// Row scale and quantization multiplier of a lane, given the largest |register|
// of its row.  The multiplier includes the twist sign (and, for kMfma, the part
// of the scale the front end left out).  Both correctly rounded quotients come
// from one division: even lanes form Q / amax, odd lanes amax / Q, and the
// pair swaps them (lanes 2i and 2i+1 always hold the same row).  Requires all
// lanes active.
template <int FRONT, int EPI>
struct RowQuant {
  float scale;    // amax / Q
  float mul;      // (twist sign) * (kMfma: post) * Q / amax, 0 where Q / amax is not finite
  uint32_t keep;  // kInt8: all ones, or 0 to clear the codes of a row without a usable scale
  __device__ __forceinline__ RowQuant(float reg_amax, bool tw, float post, int lane) {
    constexpr float Q = EPI == kFp8 ? 448.0f : 127.0f;
    const float mag = FRONT == kMfma ? fabsf(post) : 1.0f;
    const float amax = reg_amax * mag;
    const bool odd = (lane & 1) != 0;
    const float q = (odd ? amax : Q) / (odd ? Q : amax);
    const float qp = __builtin_bit_cast(
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, q), 0xB1, 0xF, 0xF, true));
    scale = odd ? q : qp;
    finish(amax, odd ? qp : q, FRONT == kMfma ? (tw ? -post : post) : (tw ? -1.0f : 1.0f));
  }
  // One thread holds the whole row (no twist, no residual scale): both
  // quotients computed directly, amax / Q by div_by_q.
  __device__ __forceinline__ explicit RowQuant(float amax) {
    constexpr float Q = EPI == kFp8 ? 448.0f : 127.0f;
    scale = div_by_q(amax);
    finish(amax, Q / amax, 1.0f);
  }
  // amax / Q correctly rounded.  With R = RN(1/Q), q0 = RN(amax * R) and one
  // fma correction q = RN(q0 + RN(amax - q0 * Q) * R) give the correctly
  // rounded quotient for every finite amax >= 0 when Q = 127, and for every
  // amax whose quotient is normal when Q = 448 (an exhaustive check over all
  // fp32 inputs; a sampled version runs in the CPU tests).  Other inputs take
  // the division.  This saves one of the two divisions per row where a
  // thread quantizes whole rows.
  __device__ __forceinline__ static float div_by_q(float amax) {
    constexpr float Q = EPI == kFp8 ? 448.0f : 127.0f;
    constexpr float R = 1.0f / Q;
    constexpr float kMin = EPI == kFp8 ? 448.0f * 0x1p-126f : 0.0f;
    if (__builtin_expect(amax >= kMin && amax < __builtin_inff(), 1)) {
      const float q0 = amax * R;
      return __builtin_fmaf(__builtin_fmaf(-q0, Q, amax), R, q0);
    }
    return amax / Q;
  }
  __device__ __forceinline__ void finish(float amax, float inv_raw, float to_true) {
    const bool finite_inv = inv_raw < __builtin_inff();  // false for Inf and NaN
    const bool usable = EPI == kFp8 ? finite_inv : (finite_inv && amax < __builtin_inff());
    mul = to_true * (usable ? inv_raw : 0.0f);
    keep = usable ? 0xFFFFFFFFu : 0u;
  }
  __device__ __forceinline__ u2 codes(const float *v) const {
    if constexpr (EPI == kFp8) {
      return to_e4m3x8(v, mul);
    } else {
      return to_int8x8(v, mul, keep);
    }
  }
};

// ---- kernels ------------------------------------------------------------------

// n <= 512*C: a tile of 512*C elements is 512*C/n whole rows and every stage
// of a tile runs inside one wave.  Each wave processes T consecutive tiles,
// loading tile t+1 while it computes tile t, so that per-wave setup (operand
// constants, signs, addressing) is paid once per T tiles while only one or two
// tiles per wave are in flight.  WPB independent waves per workgroup.  Only
// the last tile can end past row m; it masks those rows.  Addresses are a
// wave-uniform tile base plus per-lane byte offsets inside the tile, which the
// row stride limit (2^26 elements) keeps below 2^32.
template <int DT, int L, int C, int T, int WPB, bool NT, int FRONT, int EPI, bool SC1 = false>
__global__ __launch_bounds__(kWave *WPB) void fwht_wave_kernel(
    const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride, int64_t m,
    ScaleArgs sc, QuantOut qo) {
  constexpr int kTile = 512 * C;
  static_assert((1 << L) <= kTile, "row does not fit a wave tile");
  constexpr int kRows = kTile >> L;
  static_assert(kRows <= 32, "in-tile offsets must stay below 2^32 bytes");
  constexpr int kMask = (1 << L) - 1;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  int64_t row0 = ((int64_t)blockIdx.x * WPB + wave) * (int64_t)(T * kRows);
  if (row0 >= m) return;

  const int lf_load = lane_field_load<FRONT, L>(lane);
  const int lf = lane_field<FRONT, L>(lane);
  const int64_t out_pitch = EPI == kStore16 ? out_stride * 2 : qo.stride;  // bytes per row
  int ld_row[C], st_row[C];
  uint32_t ld_off[C], st_off[C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int tl = (k * kWave + lf_load) * 8;
    ld_row[k] = tl >> L;
    ld_off[k] = (uint32_t)ld_row[k] * (uint32_t)(in_stride * 2) + (uint32_t)(tl & kMask) * 2u;
    const int ts = (k * kWave + lf) * 8;
    st_row[k] = ts >> L;
    st_off[k] = (uint32_t)st_row[k] * (uint32_t)out_pitch +
                (uint32_t)(ts & kMask) * (EPI == kStore16 ? 2u : 1u);
  }
  const Finisher<DT, FRONT> fin(twisted<FRONT, L>(lane), sc.post);
  u4 a_top = {0, 0, 0, 0}, a_bot = {0, 0, 0, 0};
  if constexpr (FRONT == kMfma) h32_operands<DT>(lane, sc.e2, a_top, a_bot);

  const char *src = reinterpret_cast<const char *>(in) + row0 * in_stride * 2;
  char *dst = EPI == kStore16 ? reinterpret_cast<char *>(out) + row0 * out_pitch
                              : reinterpret_cast<char *>(qo.codes) + row0 * out_pitch;
  float *scales = EPI == kStore16 ? nullptr : qo.scales + row0;
  auto rows_in_tile = [&](int64_t r0) { return (int)(m - r0 < kRows ? m - r0 : kRows); };
  auto load_tile = [&](const char *base, int valid, u4(&raw)[C]) {
#pragma unroll
    for (int k = 0; k < C; ++k) {
      if (kRows == 1 || ld_row[k] < valid) {
        raw[k] = gload_at<NT>(base, ld_off[k]);
      } else {
        raw[k] = u4{0, 0, 0, 0};
      }
    }
  };

  int valid = rows_in_tile(row0);
  u4 next[C];
  load_tile(src, valid, next);
#pragma unroll 1
  for (int it = 0; it < T; ++it) {
    u4 raw[C];
#pragma unroll
    for (int k = 0; k < C; ++k) raw[k] = next[k];
    const int cur_valid = valid;
    const bool more = it + 1 < T && row0 + kRows < m;
    if (more) {
      src += (int64_t)kRows * in_stride * 2;
      valid = rows_in_tile(row0 + kRows);
      load_tile(src, valid, next);
    }
    float v[C * 8];
    if constexpr (FRONT == kValu) {
      widen_chunks<DT, C>(raw, v, sc.scale);
      reg_stage<1>(v);
      reg_stage<2>(v);
    } else {
#pragma unroll
      for (int k = 0; k < C; ++k) mfma_front<DT>(raw[k], a_top, a_bot, &v[k * 8]);
    }
    wave_stages<FRONT, L, C>(v, lane);
    if constexpr (EPI == kStore16) {
#pragma unroll
      for (int k = 0; k < C; ++k) {
        if (kRows == 1 || st_row[k] < cur_valid) gstore_u<NT, SC1>(dst, st_off[k], fin(&v[k * 8]));
      }
    } else {
      // row maxima: within each chunk, across the chunks of one row (chunk
      // bits that are element bits), then across the row's lanes
      constexpr int kChunkRow = (C >= 2 && L > 9 ? 1 : 0) | (C >= 4 && L > 10 ? 2 : 0) |
                                (C >= 8 && L > 11 ? 4 : 0);
      float a[C];
#pragma unroll
      for (int k = 0; k < C; ++k) a[k] = abs_max8(&v[k * 8]);
#pragma unroll
      for (int k = 0; k < C; ++k) {
        if ((k & kChunkRow) == 0) {
#pragma unroll
          for (int j = 1; j < C; ++j) {
            if ((j & ~kChunkRow) == 0) a[k] = max_with(a[k], __builtin_bit_cast(int, a[k | j]));
          }
        }
      }
      const bool tw = twisted<FRONT, L>(lane);
#pragma unroll
      for (int k = 0; k < C; ++k) {
        if ((k & kChunkRow) != 0) continue;  // same row as chunk k & ~kChunkRow
        const RowQuant<FRONT, EPI> qz(lane_max<row_lane_mask<FRONT, L>()>(a[k], lane), tw,
                                      sc.post, lane);
#pragma unroll
        for (int j = 0; j < C; ++j) {
          if ((j & ~kChunkRow) != k) continue;
          if (kRows == 1 || st_row[j] < cur_valid) {
            gstore8_u<NT, SC1>(dst, st_off[j], qz.codes(&v[j * 8]));
          }
        }
        if ((lane & row_lane_mask<FRONT, L>()) == 0 && (kRows == 1 || st_row[k] < cur_valid)) {
          scales[st_row[k]] = qz.scale;
        }
      }
    }
    if (!more) break;
    row0 += kRows;
    dst += (int64_t)kRows * out_pitch;
    if constexpr (EPI != kStore16) scales += kRows;
  }
}

// Exchange of the NW wave bits with the low log2(NW) chunk bits through LDS
// (fp32, in HALVES passes over the 4-element halves of each chunk), then the
// register stages on the exchanged bits.  After the call, chunk k of wave w
// holds tile chunk W = (k % NW)*C + (k / NW)*NW + w; the wave that held it
// before is W / C, as its chunk W % C.
//
// LDS slot s (16 bytes per lane, 1 KiB per wave access, so no access has a
// bank conflict) holds, in pass p = h / (2 / HALVES), the half h % (2 /
// HALVES) of one chunk at float4 index ((s*(2/HALVES) + h % (2/HALVES))*64 +
// lane).  Two maps from chunks to slots alternate:
//   direct:     wave w writes its chunk k to slot w*C + k, and reads its
//               chunk k from slot (k % NW)*C + (k / NW)*NW + w;
//   transposed: wave w writes its chunk k to slot (k % NW)*C + (k / NW)*NW + w,
//               and reads its chunk k from slot w*C + k.
// In both, the writer of a slot is the wave that holds the chunk and the reader
// the wave that takes it.  Each pass takes the other map from the pass before
// it (pass 0 the map TR0, pass 1 the other), so the slots a wave writes are
// exactly those it read itself in the previous pass: a wave can start writing
// as soon as its own reads of that pass are issued (LDS accesses of one wave
// run in order), and the only barrier is the one between the writes and the
// reads of a pass.  A caller that runs several exchanges on the same LDS (the
// row loops) alternates TR0 accordingly.
template <int C, int NW, int HALVES, bool TR0, int N>
__device__ __forceinline__ void exchange_wave_bits(float (&v)[N], float4 *lds) {
  static_assert(NW >= 2 && NW <= C && NW <= 8, "wave bits must fit the chunk bits");
  static_assert(HALVES == 1 || HALVES == 2, "one or two exchange passes");
  constexpr int kParts = 2 / HALVES;
  // per-lane bases built from threadIdx.x (= w*64 + lane) plus immediate
  // offsets, rather than a register per distinct uniform part:
  //   own  = ((w*C)*kParts)*64 + lane, slot w*C + k at + (k*kParts)*64
  //   gath = (w*kParts)*64 + lane,     slot Wk + w at + (Wk*kParts)*64
  const int t = (int)threadIdx.x, tw = t & ~(kWave - 1);
  float4 *own = lds + (t + (C * kParts - 1) * tw);
  float4 *gath = lds + (t + (kParts - 1) * tw);
#pragma unroll
  for (int pass = 0; pass < HALVES; ++pass) {
    const bool tr = TR0 != (pass == 1);
    // keep the passes apart in the schedule (the barrier between them used to):
    // mixing them keeps more values live and spills at n = 65536
    if (pass > 0) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int Wk = (k % NW) * C + (k / NW) * NW;
#pragma unroll
      for (int hh = 0; hh < kParts; ++hh) {
        const int h = pass * kParts + hh;
        const float4 f = make_float4(v[k * 8 + 4 * h], v[k * 8 + 4 * h + 1],
                                     v[k * 8 + 4 * h + 2], v[k * 8 + 4 * h + 3]);
        if (tr)
          gath[(Wk * kParts + hh) * kWave] = f;
        else
          own[(k * kParts + hh) * kWave] = f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int Wk = (k % NW) * C + (k / NW) * NW;
#pragma unroll
      for (int hh = 0; hh < kParts; ++hh) {
        const int h = pass * kParts + hh;
        const float4 f = tr ? own[(k * kParts + hh) * kWave] : gath[(Wk * kParts + hh) * kWave];
        v[k * 8 + 4 * h] = f.x;
        v[k * 8 + 4 * h + 1] = f.y;
        v[k * 8 + 4 * h + 2] = f.z;
        v[k * 8 + 4 * h + 3] = f.w;
      }
    }
  }
  reg_stage<3>(v);
  if constexpr (NW >= 4) reg_stage<4>(v);
  if constexpr (NW >= 8) reg_stage<5>(v);
}

// n = 512*C*NW with NW >= 2 waves per row: one row per workgroup.  After the
// in-wave stages the wave bits are exchanged with the low log2(NW) chunk bits
// through LDS (fp32), then finished as register stages.  HALVES = 2 runs the
// exchange in two passes over the two 4-element halves of each chunk, which
// halves the LDS footprint (more workgroups per CU) at the cost of one more
// barrier.  The exchange keeps every value in its lane, so the lane layout
// of the front end carries through to the store.  At n = 65536 (C = 16,
// NW = 8) a lane holds 128 fp32 values, so the 512 lanes of the workgroup
// keep the whole row in registers (256 KiB, half the CU's register file) and
// each exchange pass takes 128 KiB of LDS: one workgroup per CU.
//
// IN32 (second pass of n > 2^16): the input rows are fp32, already scaled, and
// row r of the input is block r & (2^sub - 1) of output row r >> sub.
template <int DT, int L, int C, int HALVES, bool NT, int FRONT, int EPI, bool IN32 = false,
          bool SC1 = false>
__global__ __launch_bounds__((1 << L) / (8 * C)) void fwht_block_kernel(
    const void *in, int64_t in_stride, uint16_t *out, int64_t out_stride, ScaleArgs sc,
    QuantOut qo, int sub) {
  static_assert(!IN32 || (FRONT == kValu && EPI == kStore16), "fp32 input: VALU, 16-bit output");
  constexpr int n = 1 << L;
  constexpr int NW = n / (512 * C);
  __shared__ float4 lds[n / 4 / HALVES];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int64_t row = blockIdx.x;
  // The waves run at raised priority until their front end is done, so a
  // workgroup that has just started (its loads, then the first stages on
  // them) goes ahead of the in-wave stages of the workgroup already resident
  // on the CU.  Measured against the same kernel without it, n = 8192-32768:
  // bf16 input +0.4-3.7%, FP8/INT8 output +0-4.1%; fp16 input with 16-bit
  // output -0.4-3.5%, so that case keeps the default priority.  Raising it for
  // the exchange or the stores instead, or dropping it before the front end,
  // was neutral or slower.
  constexpr bool kRaise = !IN32 && !(EPI == kStore16 && DT == HADACORE_FP16);
  if constexpr (kRaise) __builtin_amdgcn_s_setprio(3);
  // output stores with the SC1 bit (see gstore_u) if asked, except 16-bit rows of 2^14 and more
  constexpr bool kSc1 = SC1 && (EPI != kStore16 || L <= 13);

  float v[C * 8];
  if constexpr (IN32) {
    // the workspace keeps each 512-element tile G as two 1 KiB halves:
    // elements G*512 + l*8 + j sit at G*512 + (j/4)*256 + l*4 + j%4 (see
    // fwht_column_kernel), so both loads of a wave are contiguous
    const float *src = static_cast<const float *>(in) + row * in_stride;
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const uint32_t off = (uint32_t)(((w * C + k) * 512 + lane * 4) * 4);
      // whole-vector bit casts: a bit cast of one ext-vector element reads element 0
      const f4 lo = __builtin_bit_cast(f4, gload_at<NT>(src, off));
      const f4 hi = __builtin_bit_cast(f4, gload_at<NT>(src, off + 1024));
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[k * 8 + q] = lo[q];
        v[k * 8 + 4 + q] = hi[q];
      }
    }
    reg_stage<0>(v);
    reg_stage<1>(v);
    reg_stage<2>(v);
  } else {
    const uint16_t *src = static_cast<const uint16_t *>(in) + row * in_stride;
    u4 raw[C];
    const int lf_load = lane_field_load<FRONT, L>(lane);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      raw[k] = gload_at<NT>(src, (uint32_t)(((w * C + k) * kWave + lf_load) * 16));
    }
    front<DT, FRONT, C>(raw, v, lane, sc.scale, sc.e2);
    if constexpr (kRaise) __builtin_amdgcn_s_setprio(0);
  }
  wave_stages<FRONT, L, C>(v, lane);
  exchange_wave_bits<C, NW, HALVES, false>(v, lds);
  const int lf = lane_field<FRONT, L>(lane);
  if constexpr (EPI == kStore16) {
    const Finisher<DT, FRONT> fin(twisted<FRONT, L>(lane), sc.post);
    uint16_t *dst = out + (row >> sub) * out_stride + ((row & ((int64_t(1) << sub) - 1)) << L);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int W = (k % NW) * C + (k / NW) * NW + w;
      gstore_u<NT, kSc1>(dst, (uint32_t)((W * kWave + lf) * 16), fin(&v[k * 8]));
    }
  } else {
    // the row spans the workgroup: registers, then lanes, then waves (through LDS)
    __shared__ float wave_max[NW];
    float a = abs_max8(&v[0]);
#pragma unroll
    for (int k = 1; k < C; ++k) a = max_with(a, __builtin_bit_cast(int, abs_max8(&v[k * 8])));
    a = lane_max<0x3F>(a, lane);
    if (lane == 0) wave_max[w] = a;
    __syncthreads();
    a = wave_max[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) a = fmaxf(a, wave_max[i]);
    const RowQuant<FRONT, EPI> qz(a, twisted<FRONT, L>(lane), sc.post, lane);
    uint8_t *codes = qo.codes + row * qo.stride;
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int W = (k % NW) * C + (k / NW) * NW + w;
      gstore8_u<NT, kSc1>(codes, (uint32_t)((W * kWave + lf) * 8), qz.codes(&v[k * 8]));
    }
    if (threadIdx.x == 0) qo.scales[row] = qz.scale;
  }
}

// n = 65536 (and 16-bit n = 32768 from 4096 rows), matrix-core front: the
// block kernel's row as a persistent loop.  At n = 65536 a row fills half the
// register file and 128 KiB of LDS, so a CU holds one workgroup and, without a
// loop, its HBM traffic would pause while the row is transformed.  Here the
// grid is one workgroup per CU; each takes rows blockIdx.x, + gridDim.x, ...
// and issues the loads of PRE chunks of its next row right after the front end
// of the current one, so they are in flight during the in-wave stages, the
// exchange and the epilogue.  16-bit output prefetches the whole row (n =
// 65536: 16 chunks, 64 VGPRs beside the 128 fp32 values; n = 32768: 8 chunks,
// 32 VGPRs beside 64, with the exchange in one 128 KiB pass); the FP8/INT8
// epilogues at n = 65536 need more registers and prefetch 14, and issue the
// last C - PRE chunks between their first code stores, as those free
// registers.  They fit because every address is a wave-uniform base plus one
// per-lane offset.  Same arithmetic as the block kernel, so the results are
// bit-identical.

// The loops' 16-byte loads: buffer loads for 16-bit output (gload_u); global
// ones for the quantized epilogues, whose n = 65536 loop spills two VGPRs with
// buffer loads and measured the same either way.
template <bool NT, int EPI>
__device__ __forceinline__ u4 loop_load(const uint16_t *base, uint32_t off) {
  if constexpr (NT && EPI == kStore16) {
    return gload_u(base, off);
  } else {
    return gload_at<NT>(base, off);
  }
}

// One row of the loop: transform `raw` (row `row`), prefetch row `row` +
// gridDim.x into `raw` when it exists, store; returns whether it did.
template <int DT, int L, int C, int HALVES, bool NT, int EPI, int PRE, bool TR0>
__device__ __forceinline__ bool loop_row(u4 (&raw)[C], int64_t row, const uint16_t *in,
                                         int64_t in_stride, uint16_t *out, int64_t out_stride,
                                         const ScaleArgs &sc, const QuantOut &qo, int64_t m,
                                         float4 *lds, float *wave_max, int w, int lane) {
  constexpr int NW = (1 << L) / (512 * C);
  float v[C * 8];
  front<DT, kMfma, C>(raw, v, lane, sc.scale, sc.e2);
  // keep the next row's loads after the front end: both sets of raw
  // registers live at once would not fit
  __builtin_amdgcn_sched_barrier(0);
  const int64_t next = row + gridDim.x;
  const bool more = next < m;
  // The quantized epilogues load without a branch (with the loads under
  // `if (more)` the register allocator spills beside the row): a workgroup
  // past its last row reads row m - 1, the same row for every such
  // workgroup, so those reads come from cache.
  if (EPI == kStore16 && more) {
    const uint16_t *src = in + next * in_stride;
    const uint32_t ld_off = (uint32_t)(lane_field_load<kMfma, L>(lane) * 16);
#pragma unroll
    for (int k = 0; k < PRE; ++k) raw[k] = loop_load<NT, EPI>(src + (w * C + k) * 512, ld_off);
  } else if (EPI != kStore16) {
    const uint16_t *src = in + (more ? next : m - 1) * in_stride;
    const uint32_t ld_off = (uint32_t)(lane_field_load<kMfma, L>(lane) * 16);
#pragma unroll
    for (int k = 0; k < PRE; ++k) raw[k] = loop_load<NT, EPI>(src + (w * C + k) * 512, ld_off);
  }
  wave_stages<kMfma, L, C>(v, lane);
  exchange_wave_bits<C, NW, HALVES, TR0>(v, lds);
  const int lf = lane_field<kMfma, L>(lane);
  if constexpr (EPI == kStore16) {
    const Finisher<DT, kMfma> fin(twisted<kMfma, L>(lane), sc.post);
    uint16_t *dst = out + row * out_stride;
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int W = (k % NW) * C + (k / NW) * NW + w;
      gstore_u<NT, false>(dst + W * 512, (uint32_t)(lf * 16), fin(&v[k * 8]));
    }
  } else {
    // row amax: registers, lanes, then waves through LDS (the exchange's
    // barriers order this row's writes of wave_max after the last row's reads)
    float a = abs_max8(&v[0]);
#pragma unroll
    for (int k = 1; k < C; ++k) a = max_with(a, __builtin_bit_cast(int, abs_max8(&v[k * 8])));
    a = lane_max<0x3F>(a, lane);
    if (lane == 0) wave_max[w] = a;
    __syncthreads();
    a = wave_max[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) a = fmaxf(a, wave_max[i]);
    const RowQuant<kMfma, EPI> qz(a, twisted<kMfma, L>(lane), sc.post, lane);
    uint8_t *codes = qo.codes + row * qo.stride;
    const uint16_t *src = in + (more ? next : m - 1) * in_stride;
    const uint32_t ld_off = (uint32_t)(lane_field_load<kMfma, L>(lane) * 16);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int W = (k % NW) * C + (k / NW) * NW + w;
      gstore8_u<NT, false>(codes + W * 512, (uint32_t)(lf * 8), qz.codes(&v[k * 8]));
      // the chunks not prefetched yet go out as stored chunks free registers
      if (k < C - PRE) raw[PRE + k] = loop_load<NT, EPI>(src + (w * C + PRE + k) * 512, ld_off);
    }
    if (threadIdx.x == 0) qo.scales[row] = qz.scale;
  }
  return more;
}

template <int DT, int L, int C, int HALVES, bool NT, int EPI>
__global__ __launch_bounds__((1 << L) / (8 * C)) void fwht_block_loop_kernel(
    const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride, ScaleArgs sc,
    QuantOut qo, int64_t m) {
  constexpr int PRE = EPI == kStore16 ? C : (C < 14 ? C : 14);
  static_assert(PRE <= C, "prefetch at most the row's chunks");
  __shared__ float4 lds[(1 << L) / 4 / HALVES];
  __shared__ float wave_max[(1 << L) / (512 * C)];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  int64_t row = blockIdx.x;
  u4 raw[C];
  const uint16_t *src = in + row * in_stride;
  const uint32_t ld_off = (uint32_t)(lane_field_load<kMfma, L>(lane) * 16);
#pragma unroll
  for (int k = 0; k < C; ++k) raw[k] = loop_load<NT, EPI>(src + (w * C + k) * 512, ld_off);
  // The first row is peeled so that the loop is entered, like it is
  // re-entered, with the next row's loads older than this row's stores: the
  // compiler's wait before the front end then covers the loads only, not the
  // stores that follow them.
  //
  // With two exchange passes every row takes both slot maps; with one,
  // consecutive rows take them in turn (the loop is unrolled by two).  Either
  // way the LDS needs no barrier before a row's exchange writes.
  if (!loop_row<DT, L, C, HALVES, NT, EPI, PRE, false>(raw, row, in, in_stride, out, out_stride,
                                                         sc, qo, m, lds, wave_max, w, lane))
    return;
  if constexpr (HALVES == 2) {
    do {
      row += gridDim.x;
    } while (loop_row<DT, L, C, HALVES, NT, EPI, PRE, false>(raw, row, in, in_stride, out,
                                                               out_stride, sc, qo, m, lds,
                                                               wave_max, w, lane));
  } else {
    for (;;) {
      row += gridDim.x;
      if (!loop_row<DT, L, C, HALVES, NT, EPI, PRE, true>(raw, row, in, in_stride, out,
                                                            out_stride, sc, qo, m, lds, wave_max,
                                                            w, lane))
        return;
      row += gridDim.x;
      if (!loop_row<DT, L, C, HALVES, NT, EPI, PRE, false>(raw, row, in, in_stride, out,
                                                             out_stride, sc, qo, m, lds, wave_max,
                                                             w, lane))
        return;
    }
  }
}

// n <= 8: one row per thread.  A row is n consecutive 16-bit values, 2n bytes
// aligned to 2n by the stride rules, loaded and stored as one access; its
// L stages are register butterflies after scaling, and quantized outputs
// reduce, divide and convert inside the thread.  Consecutive threads take
// consecutive rows, so dense rows are read and written contiguously.
template <int N>
struct RowBits;
template <>
struct RowBits<1> {
  typedef uint16_t T;
};
template <>
struct RowBits<2> {
  typedef uint32_t T;
};
template <>
struct RowBits<4> {
  typedef u2 T;
};
template <>
struct RowBits<8> {
  typedef u4 T;
};

template <int N>
__device__ __forceinline__ void unpack16(typename RowBits<N>::T r, uint32_t (&h)[N]) {
  if constexpr (N == 1) {
    h[0] = r;
  } else if constexpr (N == 2) {
    h[0] = r & 0xFFFFu;
    h[1] = r >> 16;
  } else {
#pragma unroll
    for (int q = 0; q < N / 2; ++q) {
      h[2 * q] = r[q] & 0xFFFFu;
      h[2 * q + 1] = r[q] >> 16;
    }
  }
}

template <int DT>
__device__ __forceinline__ float widen1(uint32_t h) {
  if constexpr (DT == HADACORE_FP16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
  } else {
    return __builtin_bit_cast(float, h << 16);
  }
}

// DENSE_SC1 (n = 8 only): the rows and codes are contiguous and 128-byte
// aligned, so a wave's stores cover whole lines and take the SC1 bit (gstore_u).
template <int DT, int L, bool NT, int EPI, bool DENSE_SC1 = false>
__global__ __launch_bounds__(256) void fwht_row_kernel(const uint16_t *in, int64_t in_stride,
                                                       uint16_t *out, int64_t out_stride,
                                                       int64_t m, ScaleArgs sc, QuantOut qo) {
  constexpr int N = 1 << L;
  typedef typename RowBits<N>::T T;
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (row >= m) return;
  const T *src = reinterpret_cast<const T *>(in + row * in_stride);
  const T raw = NT ? __builtin_nontemporal_load(src) : *src;
  uint32_t h[N];
  unpack16<N>(raw, h);
  float v[N > 8 ? N : 8];
#pragma unroll
  for (int j = 0; j < N; ++j) v[j] = widen1<DT>(h[j]) * sc.scale;
#pragma unroll
  for (int b = 0; b < L; ++b) {
#pragma unroll
    for (int j = 0; j < N; ++j) {
      if ((j & (1 << b)) == 0) {
        const float a = v[j], c = v[j + (1 << b)];
        v[j] = a + c;
        v[j + (1 << b)] = a - c;
      }
    }
  }
  if constexpr (EPI == kStore16) {
    T r;
    if constexpr (N == 1) {
      r = (T)(narrow<DT>(v[0], 0.0f, 0u) & 0xFFFFu);
    } else if constexpr (N == 2) {
      r = narrow<DT>(v[0], v[1], 0u);
    } else {
#pragma unroll
      for (int q = 0; q < N / 2; ++q) r[q] = narrow<DT>(v[2 * q], v[2 * q + 1], 0u);
    }
    T *dst = reinterpret_cast<T *>(out + row * out_stride);
    if constexpr (DENSE_SC1 && N == 8) {
      gstore_u<NT, true>(out + (int64_t)blockIdx.x * 256 * 8, threadIdx.x * 16u, r);
    } else if constexpr (NT) {
      __builtin_nontemporal_store(r, dst);
    } else {
      *dst = r;
    }
  } else {
    float amax = fabsf(v[0]);
#pragma unroll
    for (int j = 1; j < N; ++j) amax = fmaxf(amax, fabsf(v[j]));
#pragma unroll
    for (int j = N; j < 8; ++j) v[j] = 0.0f;
    const RowQuant<kValu, EPI> qz(amax);
    const u2 c = qz.codes(v);
    uint8_t *dst = qo.codes + row * qo.stride;
    if constexpr (DENSE_SC1 && N == 8) {
      gstore8_u<NT, true>(qo.codes + (int64_t)blockIdx.x * 256 * 8, threadIdx.x * 8u, c);
    } else if constexpr (N == 8) {
      gstore8_at<NT>(dst, 0, c);
    } else if constexpr (N == 4) {
      *reinterpret_cast<uint32_t *>(dst) = c.x;
    } else if constexpr (N == 2) {
      *reinterpret_cast<uint16_t *>(dst) = (uint16_t)c.x;
    } else {
      *dst = (uint8_t)c.x;
    }
    qo.scales[row] = qz.scale;
  }
}

// n = A * 2^15 with A = 4..32 (sizes beyond the paper's range), first of two
// passes: for every row and every group of CW consecutive columns c of the
// 2^15-element blocks, the A values x[t * 2^15 + c] (t < A) are scaled and
// run through the stages on index bits 15 and up (butterflies across t), then
// written as fp32 to the workspace, which holds n floats per row.  The second
// pass is the n = 2^15 block kernel on those fp32 rows, so every intermediate
// stays fp32 and the result is rounded once.
// Workspace layout: within each block, the 512-element tile G (the elements
// a wave of the second pass loads, 8 per lane) is stored as two 1 KiB halves,
// element G*512 + l*8 + j at G*512 + (j/4)*256 + l*4 + j%4.  A wave of either
// pass then covers 1 KiB contiguously per fp32 access.  CW = 8: a thread takes
// the 8 columns of one lane l of one tile (16-byte load, two 16-byte stores);
// CW = 4 (A >= 16, to keep A*CW <= 128 values): the 4 columns of one half
// (8-byte load, one 16-byte store), waves ordered by (tile, half).
template <int DT, int A, int CW, bool NT, bool SC1 = false>
__global__ __launch_bounds__(256) void fwht_column_kernel(const uint16_t *in, int64_t in_stride,
                                                          float *ws, int64_t m, float scale) {
  static_assert(CW == 8 || CW == 4, "8 or 4 columns per thread");
  constexpr int kBlock = 1 << 15;
  constexpr int kGroups = kBlock / CW;
  typedef typename RowBits<CW>::T T16;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (g >= m * kGroups) return;
  const int64_t i = g / kGroups;
  const int q = (int)(g % kGroups);
  const int l = q & 63;
  const int half = CW == 8 ? 0 : (q >> 6) & 1;
  const int tile = CW == 8 ? q >> 6 : q >> 7;
  const int c = tile * 512 + l * 8 + half * 4;           // first column
  const int p = tile * 512 + half * 256 + l * 4;          // its workspace position
  const uint16_t *src = in + i * in_stride + c;
  float v[A][CW];
#pragma unroll
  for (int t = 0; t < A; ++t) {
    const T16 *ptr = reinterpret_cast<const T16 *>(src + (int64_t)t * kBlock);
    const T16 r = NT ? __builtin_nontemporal_load(ptr) : *ptr;
    uint32_t h[CW];
    unpack16<CW>(r, h);
#pragma unroll
    for (int j = 0; j < CW; ++j) v[t][j] = widen1<DT>(h[j]) * scale;
  }
#pragma unroll
  for (int b = 1; b < A; b <<= 1) {
#pragma unroll
    for (int t = 0; t < A; ++t) {
      if ((t & b) == 0) {
#pragma unroll
        for (int j = 0; j < CW; ++j) {
          const float a = v[t][j], d = v[t + b][j];
          v[t][j] = a + d;
          v[t + b][j] = a - d;
        }
      }
    }
  }
  float *dst = ws + i * (int64_t)(A * kBlock) + p;
  // a wave's 64 threads are lanes l = 0..63 of one (row, tile, half): their
  // stores start at the wave-uniform dst - 4l (see gstore_u)
  float *wdst = dst - l * 4;
#pragma unroll
  for (int t = 0; t < A; ++t) {
#pragma unroll
    for (int hh = 0; hh < CW / 4; ++hh) {
      const f4 x = {v[t][4 * hh], v[t][4 * hh + 1], v[t][4 * hh + 2], v[t][4 * hh + 3]};
      gstore_u<NT, SC1>(wdst + (int64_t)t * kBlock, (uint32_t)(l * 16 + hh * 1024),
                        __builtin_bit_cast(u4, x));
    }
  }
}

// n <= 4 with dense rows (both strides equal to n): the rows form one
// contiguous array of m*n elements, so each thread takes 8 consecutive
// elements -- 8/n whole rows -- with one 16-byte load and store, like the wider
// kernels.  A final partial chunk (m*n not a multiple of 8, still whole rows)
// is read and written element by element.  Quantized outputs (codes dense as
// well) store the 8 codes as one 8-byte access and one scale per row; each row
// has its own amax and both correctly rounded quotients, as in the row kernel.
template <int DT, int L, bool NT, int EPI, bool SC1 = false>
__global__ __launch_bounds__(256) void fwht_dense_kernel(const uint16_t *in, uint16_t *out,
                                                         int64_t total, ScaleArgs sc,
                                                         QuantOut qo) {
  constexpr int N = 1 << L;
  const int64_t base = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (base >= total) return;
  const int count = total - base >= 8 ? 8 : (int)(total - base);  // a multiple of 2^L
  uint32_t h[8];
  if (count == 8) {
    unpack16<8>(gload<NT>(in + base), h);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = j < count ? in[base + j] : 0u;
  }
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = widen1<DT>(h[j]) * sc.scale;
#pragma unroll
  for (int b = 0; b < L; ++b) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if ((j & (1 << b)) == 0) {
        const float a = v[j], c = v[j + (1 << b)];
        v[j] = a + c;
        v[j + (1 << b)] = a - c;
      }
    }
  }
  if constexpr (EPI == kStore16) {
    u4 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = narrow<DT>(v[2 * q], v[2 * q + 1], 0u);
    if (count == 8) {
      // the workgroup's 4 KiB start at a uniform base; this thread's 16 bytes follow
      gstore_u<NT, SC1>(out + (int64_t)blockIdx.x * 256 * 8, threadIdx.x * 16u, r);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (j < count) out[base + j] = (uint16_t)(r[j / 2] >> (16 * (j % 2)));
      }
    }
  } else {
#pragma clang fp contract(off)
    // rows i0 .. i0 + 8/N - 1; products rounded to fp32 before the conversion
    const int64_t i0 = base >> L;
    float w[8];
    uint32_t keep[2] = {0u, 0u};
    float sc8[8 / N];
#pragma unroll
    for (int r = 0; r < 8 / N; ++r) {
      float amax = fabsf(v[r * N]);
#pragma unroll
      for (int j = 1; j < N; ++j) amax = fmaxf(amax, fabsf(v[r * N + j]));
      if constexpr (N == 1) {
        // A one-element row: wherever Q / amax is finite, RN(Q / amax) * v lies
        // within 2^-23 of +-Q, which both conversions map to the largest code
        // of v's sign, so that code is written without the quotient.  Codes,
        // scale and mask are those of the general path below.
        if (amax >= 0x1p-100f && amax < __builtin_inff()) {
          w[r] = __builtin_copysignf(EPI == kFp8 ? 448.0f : 127.0f, v[r]);
          keep[r / 4] |= 0xFFu << (8 * (r % 4));
          sc8[r] = RowQuant<kValu, EPI>::div_by_q(amax);
          continue;
        }
      }
      const RowQuant<kValu, EPI> qz(amax);
#pragma unroll
      for (int j = 0; j < N; ++j) w[r * N + j] = v[r * N + j] * qz.mul;
      // byte mask of this row's codes (INT8 clears rows without a usable scale)
#pragma unroll
      for (int j = 0; j < N; ++j) {
        const int b = r * N + j;
        keep[b / 4] |= (qz.keep & 0xFFu) << (8 * (b % 4));
      }
      sc8[r] = qz.scale;
    }
    // 8 / N consecutive row scales, at a multiple of 8 / N (i0 is one): 16-byte
    // stores for n <= 2, one 8-byte store for n = 4, when the scales array is
    // aligned for them; a scales array that is only 4-byte aligned takes the loop
    constexpr uintptr_t kAlign = N <= 2 ? 15 : 7;
    if (count == 8 && N <= 4 && (reinterpret_cast<uintptr_t>(qo.scales) & kAlign) == 0) {
      // the workgroup's scales start at a uniform base (see gstore_u)
      float *sbase = qo.scales + (int64_t)blockIdx.x * 256 * (8 / N);
      const uint32_t soff = threadIdx.x * (uint32_t)(8 / N) * 4u;
      // first row of this wave (its 64 threads hold 512 consecutive rows)
      const int64_t wave_row = ((int64_t)blockIdx.x * 256 + (threadIdx.x & ~63u)) * 8;
      if constexpr (N == 1 && SC1) {
        if (wave_row + 512 <= total) {
          // A lane holds the scales of 8 consecutive rows; written as they are,
          // each 16-byte store instruction would leave gaps.  Two lane
          // shuffles give each instruction a contiguous 1 KiB instead: lane l
          // stores rows 4l..4l+3 and then 256+4l..256+4l+3 of the wave, held
          // by lanes l/2 and 32+l/2 (their first or second four, by l's parity).
          const int lane = threadIdx.x & 63;
          const bool odd = (lane & 1) != 0;
          f4 a, b;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float a0 = __shfl(sc8[q], lane >> 1), a1 = __shfl(sc8[4 + q], lane >> 1);
            const float b0 = __shfl(sc8[q], 32 + (lane >> 1)), b1 = __shfl(sc8[4 + q], 32 + (lane >> 1));
            a[q] = odd ? a1 : a0;
            b[q] = odd ? b1 : b0;
          }
          float *wbase = qo.scales + wave_row;
          gstore_u<NT, true>(wbase, (uint32_t)lane * 16u, __builtin_bit_cast(u4, a));
          gstore_u<NT, true>(wbase + 256, (uint32_t)lane * 16u, __builtin_bit_cast(u4, b));
        } else {
#pragma unroll
          for (int q = 0; q < 8; q += 4)
            *reinterpret_cast<f4 *>(qo.scales + i0 + q) = f4{sc8[q], sc8[q + 1], sc8[q + 2], sc8[q + 3]};
        }
      } else if constexpr (N == 1) {
        // two 16-byte stores 32 bytes apart per lane: each instruction leaves
        // gaps that the other fills, so these stay ordinary stores, which the
        // L2 merges into whole lines (with NT | SC1 they ran 3.3x slower)
#pragma unroll
        for (int q = 0; q < 8; q += 4)
          *reinterpret_cast<f4 *>(qo.scales + i0 + q) = f4{sc8[q], sc8[q + 1], sc8[q + 2], sc8[q + 3]};
      } else if constexpr (N == 2) {
        gstore_u<NT, SC1>(sbase, soff,
                          __builtin_bit_cast(u4, f4{sc8[0], sc8[1], sc8[2], sc8[3]}));
      } else {
        gstore8_u<NT, SC1>(sbase, soff, __builtin_bit_cast(u2, f2{sc8[0], sc8[1]}));
      }
    } else {
#pragma unroll
      for (int r = 0; r < 8 / N; ++r)
        if (r * N < count) qo.scales[i0 + r] = sc8[r];
    }
    const u2 raw = EPI == kFp8 ? to_e4m3x8(w, 1.0f) : to_int8x8(w, 1.0f, 0xFFFFFFFFu);
    const u2 c = EPI == kFp8 ? raw : u2{raw.x & keep[0], raw.y & keep[1]};
    if (count == 8) {
      gstore8_u<NT, SC1>(qo.codes + (int64_t)blockIdx.x * 256 * 8, threadIdx.x * 8u, c);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (j < count) qo.codes[base + j] = (uint8_t)((j < 4 ? c.x : c.y) >> (8 * (j % 4)));
      }
    }
  }
}

// 16-byte streaming copy, one access per thread, the bandwidth reference for
// the transform (same load and store cache policies as the transform's).
template <bool SC1>
__global__ __launch_bounds__(256) void stream_copy_kernel(const uint16_t *src, uint16_t *dst,
                                                          int64_t count) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x, i = i0 + threadIdx.x;
  if (i < count) gstore_u<true, SC1>(dst + i0 * 8, threadIdx.x * 16u, gload<true>(src + i * 8));
}

// ---- host dispatch ------------------------------------------------------------

// Splits the scale for the kMfma front: 2^e2 goes into the 16-bit H_32 operand
// (a normal number in that dtype), the rest is applied at the end.  fp16 rows
// cannot overflow fp32 (|x| <= 65504, n <= 2^16), so their operand is +-1.
ScaleArgs split_scale(float scale, int dtype) {
  ScaleArgs a{scale, scale, 0};
  if (dtype == HADACORE_BF16 && scale != 0.0f) {
    int e = 0;
    frexpf(fabsf(scale), &e);  // |scale| = f * 2^e, f in [0.5, 1)
    e -= 1;                    // 2^e <= |scale| < 2^(e+1)
    if (e < -126) e = -126;
    if (e > 127) e = 127;
    a.e2 = e;
    a.post = scale / ldexpf(1.0f, e);
  }
  return a;
}

int device_cus();

// Whether rows of `row_bytes` at `pitch_bytes` from `p` lie in whole 128-byte
// lines: p is aligned to 128 and either the rows are contiguous or both the
// row and the pitch are multiples of 128 bytes.  Row bytes 0 checks p only.
bool whole_lines(const void *p, int64_t pitch_bytes, int64_t row_bytes) {
  if ((reinterpret_cast<uintptr_t>(p) & 127) != 0) return false;
  return pitch_bytes == row_bytes || (pitch_bytes % 128 == 0 && row_bytes % 128 == 0);
}

// C: chunks per lane; T: tiles per wave (wave kernel) ; WPB: waves per workgroup
// (wave kernel); HALVES: LDS exchange passes (block kernel); FRONT: kValu / kMfma.
template <int DT, int L, int C, int T, int WPB, int HALVES, int FRONT, int EPI = kStore16>
hipError_t launch_cfg(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                      int64_t m, const ScaleArgs &sc, hipStream_t stream, QuantOut qo = {}) {
  // output stores with the SC1 bit (see gstore_u) only where every store
  // instruction writes whole 128-byte lines
  const bool sc1 = EPI == kStore16 ? whole_lines(out, out_stride * 2, 2 << L)
                                   : whole_lines(qo.codes, qo.stride, 1 << L);
  if constexpr (L <= 2) {
    const int64_t out_pitch = EPI == kStore16 ? out_stride : qo.stride;
    if (in_stride == (1 << L) && out_pitch == (1 << L)) {
      const int64_t total = m << L;
      const dim3 grid((uint32_t)((total + 8 * 256 - 1) / (8 * 256)));
      if (sc1 && (EPI == kStore16 || whole_lines(qo.scales, 0, 0)))
        hipLaunchKernelGGL((fwht_dense_kernel<DT, L, true, EPI, true>), grid, dim3(256), 0, stream,
                           in, out, total, sc, qo);
      else
        hipLaunchKernelGGL((fwht_dense_kernel<DT, L, true, EPI, false>), grid, dim3(256), 0,
                           stream, in, out, total, sc, qo);
    } else {
      hipLaunchKernelGGL((fwht_row_kernel<DT, L, true, EPI>), dim3((uint32_t)((m + 255) / 256)),
                         dim3(256), 0, stream, in, in_stride, out, out_stride, m, sc, qo);
    }
  } else if constexpr (L <= 3) {
    const int64_t out_pitch = EPI == kStore16 ? out_stride : qo.stride;
    if (sc1 && out_pitch == 8)
      hipLaunchKernelGGL((fwht_row_kernel<DT, L, true, EPI, true>), dim3((uint32_t)((m + 255) / 256)),
                         dim3(256), 0, stream, in, in_stride, out, out_stride, m, sc, qo);
    else
      hipLaunchKernelGGL((fwht_row_kernel<DT, L, true, EPI>), dim3((uint32_t)((m + 255) / 256)),
                         dim3(256), 0, stream, in, in_stride, out, out_stride, m, sc, qo);
  } else if constexpr ((1 << L) <= 512 * C) {
    constexpr int64_t rows_per_wave = (int64_t)T * ((512 * C) >> L);
    const int64_t waves = (m + rows_per_wave - 1) / rows_per_wave;
    const dim3 grid((uint32_t)((waves + WPB - 1) / WPB));
    if (sc1)
      hipLaunchKernelGGL((fwht_wave_kernel<DT, L, C, T, WPB, true, FRONT, EPI, true>), grid,
                         dim3(kWave * WPB), 0, stream, in, in_stride, out, out_stride, m, sc, qo);
    else
      hipLaunchKernelGGL((fwht_wave_kernel<DT, L, C, T, WPB, true, FRONT, EPI, false>), grid,
                         dim3(kWave * WPB), 0, stream, in, in_stride, out, out_stride, m, sc, qo);
  } else if constexpr (L == 16 && FRONT == kMfma) {
    // one resident workgroup per CU, each looping over rows
    const int64_t cus = device_cus();
    const int64_t blocks = m < cus ? m : cus;
    hipLaunchKernelGGL((fwht_block_loop_kernel<DT, L, C, HALVES, true, EPI>),
                       dim3((uint32_t)blocks), dim3((1 << L) / (8 * C)), 0, stream, in, in_stride,
                       out, out_stride, sc, qo, m);
  } else {
    // 16-bit rows of 2^14 and more store without SC1 (see gstore_u)
    constexpr bool kMaySc1 = EPI != kStore16 || L <= 13;
    if (kMaySc1 && sc1)
      hipLaunchKernelGGL((fwht_block_kernel<DT, L, C, HALVES, true, FRONT, EPI, false, kMaySc1>),
                         dim3((uint32_t)m), dim3((1 << L) / (8 * C)), 0, stream, in, in_stride, out,
                         out_stride, sc, qo, 0);
    else
      hipLaunchKernelGGL((fwht_block_kernel<DT, L, C, HALVES, true, FRONT, EPI, false, false>),
                         dim3((uint32_t)m), dim3((1 << L) / (8 * C)), 0, stream, in, in_stride, out,
                         out_stride, sc, qo, 0);
  }
  return hipGetLastError();
}

// Launch configuration of one (size, epilogue, front end).
// Rows from which 16-bit n = 32768 runs as the persistent loop (one workgroup
// per CU, next row prefetched into registers, one 128 KiB exchange pass).
constexpr int64_t kLoopRows32768 = 4096;

struct Cfg {
  int C;       // chunks of 8 elements per lane
  int T;       // tiles per wave (wave kernel)
  int WPB;     // waves per workgroup (wave kernel)
  int HALVES;  // LDS exchange passes (block kernel)
};

// Per-size configurations, chosen from sustained HBM throughput measured on
// MI355X (2^28-element sweeps over chunks per lane, tiles per wave, waves per
// workgroup, exchange passes and front end, interleaved so that every
// candidate sees the same clock state).  16-bit output: the smallest per-wave
// footprint that holds a row wins up to n = 1024, and from n = 2048 a row
// spreads over the waves of a workgroup with one LDS exchange.  Quantized
// output (FP8, INT8) has more arithmetic per byte, so small rows amortize the
// per-wave setup and the row reduction over two tiles or chunks per wave, and
// n = 4096 stays in one wave.  n = 65536 takes 16 chunks per lane in every
// case, the only shape whose 512 lanes hold the row.
template <int L, int EPI, int FRONT>
constexpr Cfg config() {
  if constexpr (L <= 6) {
    // n <= 8: one row per thread (C, T unused); n = 16..64: one tile per wave for
    // 16-bit output, while quantized output spreads the per-wave setup and row
    // reduction over four tiles (n = 16) or two chunks per lane (n = 32, 64)
    if constexpr (EPI == kStore16 || L <= 3) return {1, 1, 1, 1};
    if constexpr (L == 4) return {1, 4, 1, 1};
    return {2, 1, 1, 1};
  } else if constexpr (EPI == kStore16) {
    if constexpr (L <= 9) return {1, 1, 1, 1};
    if constexpr (L == 10) return {2, 1, 1, 1};
    if constexpr (L == 11) return {2, 1, 1, 1};  // two waves per row, one exchange
    if constexpr (L == 12) return {4, 1, 1, 1};
    if constexpr (L == 13) return {4, 1, 1, FRONT == kMfma ? 1 : 2};
    if constexpr (L == 14) return {8, 1, 1, FRONT == kMfma ? 1 : 2};
    if constexpr (L == 15) return {8, 1, 1, 2};
    return {16, 1, 1, 2};  // n = 65536: the row in registers, exchanged in two 128 KiB halves
  } else if constexpr (FRONT == kMfma) {
    if constexpr (L <= 8) return {2, 1, 1, 1};
    if constexpr (L == 9 || L == 10) return {4, 1, 1, 1};
    if constexpr (L == 11 || L == 12) return {8, 1, 1, 1};
    if constexpr (L <= 15) return {8, 1, 1, 2};
    return {16, 1, 1, 2};
  } else {
    if constexpr (L <= 9) return {2, 1, 1, 1};
    if constexpr (L == 10 || L == 11) return {4, 1, 1, 1};
    if constexpr (L == 12) return {8, 1, 1, 1};
    if constexpr (L == 13) return {4, 1, 1, 2};
    if constexpr (L <= 15) return {8, 1, 1, 2};
    return {16, 1, 1, 2};
  }
}

// Front end used unless HADACORE_VARIANT forces one: the matrix cores from
// n = 4096 for 16-bit output, everywhere from n = 128 for quantized output.
// Below n = 128 there is only the VALU front (the radix-32 step needs 16 vectors
// of 32 elements per wave with four lanes per vector row group).
template <int L, int EPI>
constexpr int default_front() {
  return L >= 7 && (EPI != kStore16 || L >= 12) ? kMfma : kValu;
}

template <int DT, int L, int EPI, int FRONT>
hipError_t launch_front(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                        int64_t m, const ScaleArgs &sc, hipStream_t stream, QuantOut qo) {
  constexpr Cfg c = config<L, EPI, FRONT>();
  if constexpr (L == 15 && EPI == kStore16 && FRONT == kMfma) {
    // n = 32768 with 16-bit output, from 4096 rows: the persistent loop.  With
    // one workgroup per CU a lane has 256 VGPRs, enough to hold the next row's
    // 16-bit chunks beside this row's fp32 values, and all 128 KiB of the row's
    // exchange fit the LDS in one pass.  Measured against the block kernels
    // (both dtypes, both modes, bit-identical output): +0.5-5% at 4096 rows,
    // +3-8% at 8192 and 16384; mixed (-1.4 to +2.9%) at 2048, so fewer rows
    // keep the block kernel.  FP8/INT8 output lost 8-12% in the loop.
    if (m >= kLoopRows32768) {
      const int64_t cus = device_cus();
      const int64_t blocks = m < cus ? m : cus;
      hipLaunchKernelGGL((fwht_block_loop_kernel<DT, L, 8, 1, true, EPI>), dim3((uint32_t)blocks),
                         dim3((1 << L) / (8 * 8)), 0, stream, in, in_stride, out, out_stride, sc,
                         qo, m);
      return hipGetLastError();
    }
  }
  return launch_cfg<DT, L, c.C, c.T, c.WPB, c.HALVES, FRONT, EPI>(in, in_stride, out, out_stride,
                                                                  m, sc, stream, qo);
}

// `front` < 0 takes the default; kValu / kMfma force one front end.
template <int DT, int L, int EPI>
hipError_t launch(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                  int64_t m, const ScaleArgs &sc, int front, hipStream_t stream, QuantOut qo) {
  if constexpr (L < 7) {
    (void)front;
    return launch_front<DT, L, EPI, kValu>(in, in_stride, out, out_stride, m, sc, stream, qo);
  } else {
    const int f = front < 0 ? default_front<L, EPI>() : front;
    return f == kMfma
               ? launch_front<DT, L, EPI, kMfma>(in, in_stride, out, out_stride, m, sc, stream, qo)
               : launch_front<DT, L, EPI, kValu>(in, in_stride, out, out_stride, m, sc, stream, qo);
  }
}

template <int DT, int EPI>
hipError_t launch_dt_one(int L, const uint16_t *in, int64_t in_stride, uint16_t *out,
                         int64_t out_stride, int64_t m, const ScaleArgs &sc, int front,
                         hipStream_t stream, QuantOut qo) {
  switch (L) {
    case 0: return launch<DT, 0, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 1: return launch<DT, 1, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 2: return launch<DT, 2, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 3: return launch<DT, 3, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 4: return launch<DT, 4, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 5: return launch<DT, 5, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 6: return launch<DT, 6, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 7: return launch<DT, 7, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 8: return launch<DT, 8, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 9: return launch<DT, 9, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 10: return launch<DT, 10, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 11: return launch<DT, 11, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 12: return launch<DT, 12, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 13: return launch<DT, 13, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 14: return launch<DT, 14, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 15: return launch<DT, 15, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    case 16: return launch<DT, 16, EPI>(in, in_stride, out, out_stride, m, sc, front, stream, qo);
    default: return hipErrorInvalidValue;
  }
}

// n = A * 2^15, A = 4..32: the column pass into the fp32 workspace, then the
// n = 2^15 block kernel on the workspace rows (fp32 input, VALU front), each
// writing block t of its output row.
template <int DT, int A>
hipError_t launch_large(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                        int64_t m, float scale, float *ws, hipStream_t stream) {
  constexpr int CW = A <= 8 ? 8 : 4;
  constexpr int kBlock = 1 << 15;
  const int64_t threads = m * (kBlock / CW);
  const dim3 grid((uint32_t)((threads + 255) / 256));
  if (whole_lines(ws, 0, 0))
    hipLaunchKernelGGL((fwht_column_kernel<DT, A, CW, true, true>), grid, dim3(256), 0, stream, in,
                       in_stride, ws, m, scale);
  else
    hipLaunchKernelGGL((fwht_column_kernel<DT, A, CW, true, false>), grid, dim3(256), 0, stream, in,
                       in_stride, ws, m, scale);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  constexpr Cfg c = config<15, kStore16, kValu>();
  constexpr int sub = A == 4 ? 2 : A == 8 ? 3 : A == 16 ? 4 : 5;
  const ScaleArgs unit{1.0f, 1.0f, 0};
  hipLaunchKernelGGL((fwht_block_kernel<DT, 15, c.C, c.HALVES, true, kValu, kStore16, true>),
                     dim3((uint32_t)(m * A)), dim3(kBlock / (8 * c.C)), 0, stream,
                     static_cast<const void *>(ws), (int64_t)kBlock, out, out_stride, unit,
                     QuantOut{}, sub);
  return hipGetLastError();
}

template <int DT>
hipError_t launch_large_one(int L, const uint16_t *in, int64_t in_stride, uint16_t *out,
                            int64_t out_stride, int64_t m, float scale, float *ws,
                            hipStream_t stream) {
  switch (L) {
    case 17: return launch_large<DT, 4>(in, in_stride, out, out_stride, m, scale, ws, stream);
    case 18: return launch_large<DT, 8>(in, in_stride, out, out_stride, m, scale, ws, stream);
    case 19: return launch_large<DT, 16>(in, in_stride, out, out_stride, m, scale, ws, stream);
    case 20: return launch_large<DT, 32>(in, in_stride, out, out_stride, m, scale, ws, stream);
    default: return hipErrorInvalidValue;
  }
}

// Rows per launch.  Every kernel uses at most max(1, n/4) work-items per row
// (the column pass of n > 2^16: 2^15/4 per row; the others n/(8*C*T) or one
// per row or per 8/n rows), so launches of at most 2^31 / max(1, n/4) rows keep
// the grid's work-item count below 2^31.  Larger m is split into several
// launches on the same stream, each starting at its own first row (a multiple
// of 1024, so every row start keeps its alignment); they run in stream order,
// and rows are independent, so the result is that of one launch.
constexpr int64_t kMaxItemsPerLaunch = int64_t(1) << 31;

int64_t rows_per_launch(int L) {
  const int64_t per_row = L >= 2 ? (int64_t(1) << (L - 2)) : 1;
  return (kMaxItemsPerLaunch / per_row) & ~int64_t(1023);
}

template <int DT, int EPI = kStore16>
hipError_t launch_dt(int L, const uint16_t *in, int64_t in_stride, uint16_t *out,
                     int64_t out_stride, int64_t m, const ScaleArgs &sc, int front,
                     hipStream_t stream, QuantOut qo = {}) {
  const int64_t chunk = rows_per_launch(L);
  for (int64_t r0 = 0; r0 < m; r0 += chunk) {
    const int64_t mc = m - r0 < chunk ? m - r0 : chunk;
    QuantOut q = qo;
    if constexpr (EPI != kStore16) {
      q.codes = qo.codes + r0 * qo.stride;
      q.scales = qo.scales + r0;
    }
    uint16_t *o = EPI == kStore16 ? out + r0 * out_stride : nullptr;
    const hipError_t e =
        launch_dt_one<DT, EPI>(L, in + r0 * in_stride, in_stride, o, out_stride, mc, sc, front,
                               stream, q);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// n > 2^16 through the workspace: row r0 of a launch uses workspace row r0 too.
template <int DT>
hipError_t launch_large_dt(int L, const uint16_t *in, int64_t in_stride, uint16_t *out,
                           int64_t out_stride, int64_t m, float scale, float *ws,
                           hipStream_t stream) {
  const int64_t chunk = rows_per_launch(L);
  for (int64_t r0 = 0; r0 < m; r0 += chunk) {
    const int64_t mc = m - r0 < chunk ? m - r0 : chunk;
    const hipError_t e = launch_large_one<DT>(L, in + r0 * in_stride, in_stride,
                                              out + r0 * out_stride, out_stride, mc, scale,
                                              ws + r0 * (int64_t(1) << L), stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// HADACORE_VARIANT=valu|mfma forces a front end (testing and tuning); unset,
// empty or anything else keeps the per-size table.  Read on every call.
int front_override() {
  const char *v = getenv("HADACORE_VARIANT");
  if (v == nullptr) return -1;
  if (strcmp(v, "valu") == 0) return kValu;
  if (strcmp(v, "mfma") == 0) return kMfma;
  return -1;
}

// Architecture check, cached per device: 0 unknown, 1 gfx950, 2 other.
constexpr int kMaxDevices = 64;
std::atomic<int> g_arch_state[kMaxDevices];
std::atomic<int> g_cus[kMaxDevices];

hadacore_status check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return HADACORE_ERROR_UNSUPPORTED_DEVICE;
  if (dev < kMaxDevices) {
    const int st = g_arch_state[dev].load(std::memory_order_relaxed);
    if (st == 1) return HADACORE_SUCCESS;
    if (st == 2) return HADACORE_ERROR_UNSUPPORTED_DEVICE;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return HADACORE_ERROR_UNSUPPORTED_DEVICE;
  const bool ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev < kMaxDevices) {
    g_cus[dev].store(prop.multiProcessorCount, std::memory_order_relaxed);
    g_arch_state[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
  }
  return ok ? HADACORE_SUCCESS : HADACORE_ERROR_UNSUPPORTED_DEVICE;
}

// Compute units of the current device (the grid of the persistent kernel);
// check_device() has run before any launch and cached it.
int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < kMaxDevices) {
    const int c = g_cus[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int c = 0;
  if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && c > 0)
    return c;
  return 256;
}

// Largest row stride (elements, or bytes for FP8 codes): keeps every offset
// inside a wave tile (at most 32 rows) below 2^32 bytes.
constexpr int64_t kMaxStride = int64_t(1) << 26;

// Largest log2 n of one pass (a row of n = 65536 fills the registers of a
// 512-thread workgroup in fp32) and of hadamard_transform_ws (two passes
// through the workspace above that).
constexpr int kMaxOnePassL = 16;
constexpr int kMaxLargeL = 20;

int log2_exact(int64_t n) {
  if (n <= 0 || (n & (n - 1)) != 0) return -1;
  int l = 0;
  while ((int64_t(1) << l) < n) ++l;
  return l;
}

// Byte range [lo, hi) touched by m rows of n 16-bit elements at the given stride.
void row_span(const void *p, int64_t stride, int64_t m, int64_t n, uintptr_t *lo, uintptr_t *hi) {
  *lo = reinterpret_cast<uintptr_t>(p);
  *hi = *lo + (uintptr_t)(((m - 1) * stride + n) * 2);
}

// Synchronous argument validation shared by the entry points (no HIP calls).
hadacore_status validate(const void *in, int64_t in_row_stride, const void *out,
                         int64_t out_row_stride, int64_t m, int64_t n, hadacore_dtype dtype,
                         float scale, int *L_out, int max_L = kMaxOnePassL) {
  if (m < 0) return HADACORE_ERROR_INVALID_VALUE;
  const int L = log2_exact(n);
  if (L < 0 || L > max_L) return HADACORE_ERROR_INVALID_SIZE;
  if (dtype != HADACORE_FP16 && dtype != HADACORE_BF16) return HADACORE_ERROR_INVALID_DTYPE;
  if (!isfinite(scale)) return HADACORE_ERROR_INVALID_VALUE;
  const int64_t align = n < 8 ? n : 8;  // rows start on 2*min(n, 8)-byte boundaries
  if (in_row_stride < n || out_row_stride < n || (in_row_stride % align) != 0 ||
      (out_row_stride % align) != 0 || in_row_stride > kMaxStride || out_row_stride > kMaxStride)
    return HADACORE_ERROR_INVALID_STRIDE;
  *L_out = L;
  if (m == 0) return HADACORE_SUCCESS;
  if (in == nullptr || out == nullptr) return HADACORE_ERROR_INVALID_VALUE;
  if ((reinterpret_cast<uintptr_t>(in) & 15) != 0 || (reinterpret_cast<uintptr_t>(out) & 15) != 0)
    return HADACORE_ERROR_MISALIGNED;
  if (m >= (int64_t(1) << 31)) return HADACORE_ERROR_TOO_LARGE;
  if (in_row_stride > (int64_t(1) << 40) / m || out_row_stride > (int64_t(1) << 40) / m)
    return HADACORE_ERROR_TOO_LARGE;
  uintptr_t ilo, ihi, olo, ohi;
  row_span(in, in_row_stride, m, n, &ilo, &ihi);
  row_span(out, out_row_stride, m, n, &olo, &ohi);
  const bool same = in == out && in_row_stride == out_row_stride;
  if (!same && ilo < ohi && olo < ihi) return HADACORE_ERROR_OVERLAP;
  return HADACORE_SUCCESS;
}

// Fixed device workspace of hadamard_transform_ws_noalloc: one array per GPU
// (each device holds its own copy of this module's globals), kScratchBytes
// long, alive until the process ends.  Host code never uses the symbol's name
// as an address: on its first call on a device the entry point asks the
// runtime for that device's address of the array (hipGetSymbolAddress, with
// the device current) and keeps it here.  The two-pass kernels write every
// workspace element in pass 1 before pass 2 reads it, so nothing needs
// clearing between calls; calls that overlap on one GPU share the array and
// race.
constexpr int64_t kScratchBytes = HADACORE_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

std::atomic<float *> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

// This device's address of `scratch`, or nullptr if the runtime cannot give it.
float *scratch_address() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  float *p = g_scratch[dev].load(std::memory_order_acquire);
  if (p != nullptr) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (p == nullptr) {
    void *addr = nullptr;
    if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || addr == nullptr)
      return nullptr;
    p = static_cast<float *>(addr);
    g_scratch[dev].store(p, std::memory_order_release);
  }
  return p;
}

}  // namespace
}  // namespace hadacore

using namespace hadacore;

extern "C" hadacore_status hadamard_transform_strided(const void *in, int64_t in_row_stride,
                                                      void *out, int64_t out_row_stride,
                                                      int64_t m, int64_t n, hadacore_dtype dtype,
                                                      float scale, void *stream) {
  int L = 0;
  const hadacore_status st =
      validate(in, in_row_stride, out, out_row_stride, m, n, dtype, scale, &L);
  if (st != HADACORE_SUCCESS || m == 0) return st;
  const hadacore_status dev = check_device();
  if (dev != HADACORE_SUCCESS) return dev;

  const uint16_t *src = static_cast<const uint16_t *>(in);
  uint16_t *dst = static_cast<uint16_t *>(out);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const ScaleArgs sc = split_scale(scale, dtype);
  const int front = front_override();
  const hipError_t err =
      dtype == HADACORE_FP16
          ? launch_dt<HADACORE_FP16>(L, src, in_row_stride, dst, out_row_stride, m, sc, front, s)
          : launch_dt<HADACORE_BF16>(L, src, in_row_stride, dst, out_row_stride, m, sc, front, s);
  return err == hipSuccess ? HADACORE_SUCCESS : HADACORE_ERROR_LAUNCH;
}

extern "C" int64_t hadamard_transform_workspace_size(int64_t m, int64_t n) {
  const int L = log2_exact(n);
  if (m <= 0 || L <= kMaxOnePassL || L > kMaxLargeL || m >= (int64_t(1) << 31)) return 0;
  if (m > (int64_t(1) << 40) / n) return 0;  // the call itself reports TOO_LARGE
  return 4 * m * n;
}

namespace hadacore {
namespace {

// hadamard_transform_ws after its workspace has been chosen: `workspace` of
// `workspace_bytes`, or with `fixed` the scratch array (whose size is the
// limit, reported as HADACORE_ERROR_SCRATCH).
hadacore_status transform_two_pass(const void *in, int64_t in_row_stride, void *out,
                                   int64_t out_row_stride, int64_t m, int64_t n,
                                   hadacore_dtype dtype, float scale, void *workspace,
                                   int64_t workspace_bytes, bool fixed, void *stream) {
  int L = 0;
  const hadacore_status st =
      validate(in, in_row_stride, out, out_row_stride, m, n, dtype, scale, &L, kMaxLargeL);
  if (st != HADACORE_SUCCESS || m == 0) return st;
  if (L <= kMaxOnePassL) {
    return hadamard_transform_strided(in, in_row_stride, out, out_row_stride, m, n, dtype, scale,
                                      stream);
  }
  const int64_t need = hadamard_transform_workspace_size(m, n);
  if (need == 0) return HADACORE_ERROR_TOO_LARGE;
  if (fixed) {
    if (need > kScratchBytes) return HADACORE_ERROR_SCRATCH;
  } else {
    if (workspace == nullptr || workspace_bytes < need) return HADACORE_ERROR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15) != 0) return HADACORE_ERROR_MISALIGNED;
  }
  if ((m * (n >> 15)) >= (int64_t(1) << 31)) return HADACORE_ERROR_TOO_LARGE;
  auto overlaps = [&](const void *w) {
    uintptr_t ilo, ihi, olo, ohi;
    row_span(in, in_row_stride, m, n, &ilo, &ihi);
    row_span(out, out_row_stride, m, n, &olo, &ohi);
    const uintptr_t wlo = reinterpret_cast<uintptr_t>(w);
    const uintptr_t whi = wlo + (uintptr_t)need;
    return (wlo < ihi && ilo < whi) || (wlo < ohi && olo < whi);
  };
  if (!fixed && overlaps(workspace)) return HADACORE_ERROR_OVERLAP;
  const hadacore_status dev = check_device();
  if (dev != HADACORE_SUCCESS) return dev;
  if (fixed) {
    workspace = scratch_address();
    if (workspace == nullptr) return HADACORE_ERROR_LAUNCH;
    if (overlaps(workspace)) return HADACORE_ERROR_OVERLAP;
  }
  const uint16_t *src = static_cast<const uint16_t *>(in);
  uint16_t *dst = static_cast<uint16_t *>(out);
  float *ws = static_cast<float *>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t err =
      dtype == HADACORE_FP16
          ? launch_large_dt<HADACORE_FP16>(L, src, in_row_stride, dst, out_row_stride, m, scale, ws, s)
          : launch_large_dt<HADACORE_BF16>(L, src, in_row_stride, dst, out_row_stride, m, scale, ws, s);
  return err == hipSuccess ? HADACORE_SUCCESS : HADACORE_ERROR_LAUNCH;
}

}  // namespace
}  // namespace hadacore

extern "C" hadacore_status hadamard_transform_ws(const void *in, int64_t in_row_stride, void *out,
                                                 int64_t out_row_stride, int64_t m, int64_t n,
                                                 hadacore_dtype dtype, float scale,
                                                 void *workspace, int64_t workspace_bytes,
                                                 void *stream) {
  return transform_two_pass(in, in_row_stride, out, out_row_stride, m, n, dtype, scale, workspace,
                            workspace_bytes, false, stream);
}

extern "C" hadacore_status hadamard_transform_ws_noalloc(const void *in, int64_t in_row_stride,
                                                         void *out, int64_t out_row_stride,
                                                         int64_t m, int64_t n,
                                                         hadacore_dtype dtype, float scale,
                                                         void *stream) {
  return transform_two_pass(in, in_row_stride, out, out_row_stride, m, n, dtype, scale, nullptr, 0,
                            true, stream);
}

extern "C" hadacore_status hadamard_transform(const void *in, void *out, int64_t m, int64_t n,
                                              hadacore_dtype dtype, float scale, void *stream) {
  return hadamard_transform_strided(in, n, out, n, m, n, dtype, scale, stream);
}

namespace hadacore {
namespace {

// Validation and launch shared by the quantizing entry points.
template <int EPI>
hadacore_status transform_quantized(const void *in, int64_t in_row_stride, void *out_codes,
                                    int64_t out_row_stride, float *out_scales, int64_t m,
                                    int64_t n, hadacore_dtype dtype, float scale, void *stream) {
  if (m < 0) return HADACORE_ERROR_INVALID_VALUE;
  const int L = log2_exact(n);
  if (L < 0 || L > kMaxOnePassL) return HADACORE_ERROR_INVALID_SIZE;
  if (dtype != HADACORE_FP16 && dtype != HADACORE_BF16) return HADACORE_ERROR_INVALID_DTYPE;
  if (!isfinite(scale)) return HADACORE_ERROR_INVALID_VALUE;
  // input rows start on 2*min(n, 8)-byte boundaries, code rows on min(n, 16)
  if (in_row_stride < n || (in_row_stride % (n < 8 ? n : 8)) != 0 || out_row_stride < n ||
      (out_row_stride % (n < 16 ? n : 16)) != 0 || in_row_stride > kMaxStride ||
      out_row_stride > kMaxStride)
    return HADACORE_ERROR_INVALID_STRIDE;
  if (m == 0) return HADACORE_SUCCESS;
  if (in == nullptr || out_codes == nullptr || out_scales == nullptr)
    return HADACORE_ERROR_INVALID_VALUE;
  if ((reinterpret_cast<uintptr_t>(in) & 15) != 0 ||
      (reinterpret_cast<uintptr_t>(out_codes) & 15) != 0 ||
      (reinterpret_cast<uintptr_t>(out_scales) & 3) != 0)
    return HADACORE_ERROR_MISALIGNED;
  if (m >= (int64_t(1) << 31)) return HADACORE_ERROR_TOO_LARGE;
  if (in_row_stride > (int64_t(1) << 40) / m || out_row_stride > (int64_t(1) << 40) / m)
    return HADACORE_ERROR_TOO_LARGE;
  // byte ranges of the input rows, the code rows and the scales must be disjoint
  uintptr_t ilo, ihi;
  row_span(in, in_row_stride, m, n, &ilo, &ihi);
  const uintptr_t clo = reinterpret_cast<uintptr_t>(out_codes);
  const uintptr_t chi = clo + (uintptr_t)((m - 1) * out_row_stride + n);
  const uintptr_t slo = reinterpret_cast<uintptr_t>(out_scales);
  const uintptr_t shi = slo + (uintptr_t)(4 * m);
  if ((ilo < chi && clo < ihi) || (ilo < shi && slo < ihi) || (clo < shi && slo < chi))
    return HADACORE_ERROR_OVERLAP;

  const hadacore_status dev = check_device();
  if (dev != HADACORE_SUCCESS) return dev;
  const uint16_t *src = static_cast<const uint16_t *>(in);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const ScaleArgs sc = split_scale(scale, dtype);
  const QuantOut qo{static_cast<uint8_t *>(out_codes), out_row_stride, out_scales};
  const int front = front_override();
  const hipError_t err =
      dtype == HADACORE_FP16
          ? launch_dt<HADACORE_FP16, EPI>(L, src, in_row_stride, nullptr, 0, m, sc, front, s, qo)
          : launch_dt<HADACORE_BF16, EPI>(L, src, in_row_stride, nullptr, 0, m, sc, front, s, qo);
  return err == hipSuccess ? HADACORE_SUCCESS : HADACORE_ERROR_LAUNCH;
}

}  // namespace
}  // namespace hadacore

extern "C" hadacore_status hadamard_transform_fp8(const void *in, int64_t in_row_stride,
                                                  void *out_codes, int64_t out_row_stride,
                                                  float *out_scales, int64_t m, int64_t n,
                                                  hadacore_dtype dtype, float scale, void *stream) {
  return transform_quantized<kFp8>(in, in_row_stride, out_codes, out_row_stride, out_scales, m, n,
                                   dtype, scale, stream);
}

extern "C" hadacore_status hadamard_transform_int8(const void *in, int64_t in_row_stride,
                                                   void *out_codes, int64_t out_row_stride,
                                                   float *out_scales, int64_t m, int64_t n,
                                                   hadacore_dtype dtype, float scale, void *stream) {
  return transform_quantized<kInt8>(in, in_row_stride, out_codes, out_row_stride, out_scales, m,
                                    n, dtype, scale, stream);
}

extern "C" hadacore_status hadacore_stream_copy(const void *src, void *dst, int64_t bytes,
                                                void *stream) {
  if (bytes < 0 || (bytes % 16) != 0) return HADACORE_ERROR_INVALID_VALUE;
  if (bytes == 0) return HADACORE_SUCCESS;
  if (src == nullptr || dst == nullptr) return HADACORE_ERROR_INVALID_VALUE;
  if ((reinterpret_cast<uintptr_t>(src) & 15) != 0 || (reinterpret_cast<uintptr_t>(dst) & 15) != 0)
    return HADACORE_ERROR_MISALIGNED;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + (uintptr_t)bytes && d0 < s0 + (uintptr_t)bytes) return HADACORE_ERROR_OVERLAP;
  const int64_t count = bytes / 16;
  if ((count + 255) / 256 >= (int64_t(1) << 31)) return HADACORE_ERROR_TOO_LARGE;
  const hadacore_status dev = check_device();
  if (dev != HADACORE_SUCCESS) return dev;
  const dim3 grid((uint32_t)((count + 255) / 256));
  if (whole_lines(dst, 0, 0))
    hipLaunchKernelGGL(stream_copy_kernel<true>, grid, dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<const uint16_t *>(src),
                       static_cast<uint16_t *>(dst), count);
  else
    hipLaunchKernelGGL(stream_copy_kernel<false>, grid, dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<const uint16_t *>(src),
                       static_cast<uint16_t *>(dst), count);
  return hipGetLastError() == hipSuccess ? HADACORE_SUCCESS : HADACORE_ERROR_LAUNCH;
}

extern "C" const char *hadacore_status_string(hadacore_status status) {
  switch (status) {
    case HADACORE_SUCCESS: return "success";
    case HADACORE_ERROR_INVALID_VALUE: return "invalid value (m < 0, null pointer or non-finite scale)";
    case HADACORE_ERROR_INVALID_SIZE: return "invalid size (n must be a power of two in [1, 65536], or up to 2^20 with a workspace)";
    case HADACORE_ERROR_INVALID_DTYPE: return "invalid dtype (expected HADACORE_FP16 or HADACORE_BF16)";
    case HADACORE_ERROR_INVALID_STRIDE:
      return "invalid row stride (>= n, <= 2^26, a multiple of min(n, 8) (codes: min(n, 16)))";
    case HADACORE_ERROR_MISALIGNED: return "misaligned pointer (16-byte alignment required)";
    case HADACORE_ERROR_OVERLAP: return "input and output overlap without being the same layout";
    case HADACORE_ERROR_LAUNCH: return "kernel launch failed";
    case HADACORE_ERROR_UNSUPPORTED_DEVICE: return "current device is not gfx950";
    case HADACORE_ERROR_TOO_LARGE: return "problem too large for one launch";
    case HADACORE_ERROR_WORKSPACE:
      return "workspace missing or smaller than hadamard_transform_workspace_size(m, n)";
    case HADACORE_ERROR_SCRATCH:
      return "workspace needed exceeds the fixed scratch array of hadamard_transform_ws_noalloc "
             "(HADACORE_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

extern "C" int32_t hadacore_version(void) { return HADACORE_VERSION; }
