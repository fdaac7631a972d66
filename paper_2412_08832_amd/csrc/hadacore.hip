// hadacore.hip -- batched normalized Walsh-Hadamard transform for gfx950.
//
// Computes out[i][j] = scale * sum_k (-1)^popcount(j & k) * in[i][k] for
// 16-bit rows of length n = 2^L, 7 <= L <= 15 (HadaCore, arXiv 2412.08832:
// the transform of Sec. 2.1-2.2, sizes of Sec. 3.2, in place per Appendix B,
// fp16 and bf16 per Appendix C).
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
//     ds_swizzle (xor 4, xor 16) or by ds_bpermute (xor 32);
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
// Numerics: inputs are widened exactly and multiplied by the scale before
// any addition (folded into the first butterfly), so large bf16 rows do not
// overflow fp32 partial sums; every intermediate is fp32 and the result is
// rounded once, round-to-nearest-even.
//
// Where this differs from the paper's kernel: the paper maps 16-point
// transforms onto 16x16 Tensor-Core matmuls (Sec. 3) and keeps fp16/bf16
// intermediates; here the stages are fp32 VALU butterflies with wave64 DPP
// and LDS exchanges, which keeps one rounding and is bound by HBM bandwidth.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#include "hadacore.h"

namespace hadacore {
namespace {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

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
  const float sgn = (lane & (1 << LB)) ? -1.0f : 1.0f;
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

// Lane bits of a wave that carry element bits for rows of 2^L elements.
template <int L>
constexpr int lane_bits() {
  return L - 3 >= 6 ? 6 : L - 3;
}

// Sign-flip mask for the packed results of this lane: a lane holds negated
// values iff an odd number of its processed lane bits are set.
template <int L>
__device__ __forceinline__ uint32_t twist_flip(int lane) {
  const int processed = lane & ((1 << lane_bits<L>()) - 1);
  return (__builtin_popcount(processed) & 1) ? 0x80008000u : 0u;
}

// Widen + scale + stage on bit 0 for all registers.
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

// Every stage whose bit lies inside one wave except element bit 0 (done while
// widening): in-chunk bits 1-2, the chunk bits that are element bits (tile
// bits 9.. below L), and the lane bits (tile bits 3-8) below L.
template <int L, int C, int N>
__device__ __forceinline__ void wave_stages(float (&v)[N], int lane) {
  reg_stage<1>(v);
  reg_stage<2>(v);
  static_assert(C == 1 || C == 2 || C == 4 || C == 8, "1, 2, 4 or 8 chunks per lane");
  if constexpr (C >= 2 && L > 9) reg_stage<3>(v);
  if constexpr (C >= 4 && L > 10) reg_stage<4>(v);
  if constexpr (C >= 8 && L > 11) reg_stage<5>(v);
  if constexpr (L > 3) lane_stage<0>(v, lane);
  if constexpr (L > 4) lane_stage<1>(v, lane);
  if constexpr (L > 5) lane_stage<2>(v, lane);
  if constexpr (L > 6) lane_stage<3>(v, lane);
  if constexpr (L > 7) lane_stage<4>(v, lane);
  if constexpr (L > 8) lane_stage<5>(v, lane);
}

template <int DT>
__device__ __forceinline__ u4 narrow_chunk(const float *v, uint32_t flip) {
  u4 r;
  r.x = narrow<DT>(v[0], v[1], flip);
  r.y = narrow<DT>(v[2], v[3], flip);
  r.z = narrow<DT>(v[4], v[5], flip);
  r.w = narrow<DT>(v[6], v[7], flip);
  return r;
}

// ---- kernels ------------------------------------------------------------------

// n <= 512*C: each wave owns a tile of 512*C elements = 512*C/n whole rows and
// runs every stage inside the wave.  WPB independent waves per workgroup.
// Tiles that end past row m (only the last one) mask their rows.
template <int DT, int L, int C, int WPB, bool NT>
__global__ __launch_bounds__(kWave *WPB) void fwht_wave_kernel(
    const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride, int64_t m,
    float scale) {
  constexpr int kTile = 512 * C;
  static_assert((1 << L) <= kTile, "row does not fit a wave tile");
  constexpr int kRows = kTile >> L;
  constexpr int kMask = (1 << L) - 1;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int64_t row0 = ((int64_t)blockIdx.x * WPB + wave) * kRows;
  if (row0 >= m) return;
  const bool full = row0 + kRows <= m;
  const uint16_t *src = in + row0 * in_stride;
  uint16_t *dst = out + row0 * out_stride;

  u4 raw[C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int t = (k * kWave + lane) * 8;
    if (full || row0 + (t >> L) < m) {
      raw[k] = gload<NT>(src + (int64_t)(t >> L) * in_stride + (t & kMask));
    } else {
      raw[k] = u4{0, 0, 0, 0};
    }
  }
  float v[C * 8];
  widen_chunks<DT, C>(raw, v, scale);
  wave_stages<L, C>(v, lane);
  const uint32_t flip = twist_flip<L>(lane);
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int t = (k * kWave + lane) * 8;
    if (full || row0 + (t >> L) < m) {
      gstore<NT>(dst + (int64_t)(t >> L) * out_stride + (t & kMask),
                 narrow_chunk<DT>(&v[k * 8], flip));
    }
  }
}

// n = 512*C*NW with NW >= 2 waves per row: one row per workgroup.  After the
// in-wave stages the wave bits are exchanged with the low log2(NW) chunk bits
// through LDS (fp32), then finished as register stages.  HALVES = 2 runs the
// exchange in two passes over the two 4-element halves of each chunk, which
// halves the LDS footprint (more workgroups per CU) at the cost of two extra
// barriers.
template <int DT, int L, int C, int HALVES, bool NT>
__global__ __launch_bounds__((1 << L) / (8 * C)) void fwht_block_kernel(
    const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride, float scale) {
  constexpr int n = 1 << L;
  constexpr int NW = n / (512 * C);
  static_assert(NW >= 2 && NW <= C, "wave bits must fit the chunk bits");
  static_assert(HALVES == 1 || HALVES == 2, "one or two exchange passes");
  // LDS word address of tile element ((W*64 + l)*8 + 4h + q) in pass p = h / (2 / HALVES):
  // ((W*(2/HALVES) + h % (2/HALVES))*64 + l)*4 + q, so each 16-byte access of a wave is
  // 1 KiB contiguous and free of bank conflicts.
  constexpr int kParts = 2 / HALVES;
  __shared__ float4 lds[n / 4 / HALVES];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int64_t row = blockIdx.x;
  const uint16_t *src = in + row * in_stride;
  uint16_t *dst = out + row * out_stride;

  u4 raw[C];
#pragma unroll
  for (int k = 0; k < C; ++k) raw[k] = gload<NT>(src + ((w * C + k) * kWave + lane) * 8);
  float v[C * 8];
  widen_chunks<DT, C>(raw, v, scale);
  wave_stages<L, C>(v, lane);

#pragma unroll
  for (int pass = 0; pass < HALVES; ++pass) {
    if (pass > 0) __syncthreads();  // the previous pass's reads are done
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int W = w * C + k;
#pragma unroll
      for (int hh = 0; hh < kParts; ++hh) {
        const int h = pass * kParts + hh;
        lds[(W * kParts + hh) * kWave + lane] =
            make_float4(v[k * 8 + 4 * h], v[k * 8 + 4 * h + 1], v[k * 8 + 4 * h + 2],
                        v[k * 8 + 4 * h + 3]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int W = (k % NW) * C + (k / NW) * NW + w;
#pragma unroll
      for (int hh = 0; hh < kParts; ++hh) {
        const int h = pass * kParts + hh;
        const float4 f = lds[(W * kParts + hh) * kWave + lane];
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
  const uint32_t flip = twist_flip<L>(lane);
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int W = (k % NW) * C + (k / NW) * NW + w;
    gstore<NT>(dst + (W * kWave + lane) * 8, narrow_chunk<DT>(&v[k * 8], flip));
  }
}

// 16-byte streaming copy, one access per thread, the bandwidth reference for
// the transform.
__global__ __launch_bounds__(256) void stream_copy_kernel(const uint16_t *src, uint16_t *dst,
                                                          int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) gstore<true>(dst + i * 8, gload<true>(src + i * 8));
}

// ---- host dispatch ------------------------------------------------------------

// Launch configuration of one (dtype, n).
struct Config {
  int chunks;     // C: 16-byte chunks per lane
  int waves;      // WPB for the wave kernel (NW is implied by n and C)
  int halves;     // block kernel: LDS exchange passes
};

template <int DT, int L, int C, int WPB, int HALVES>
hipError_t launch_cfg(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                      int64_t m, float scale, hipStream_t stream) {
  if constexpr ((1 << L) <= 512 * C) {
    constexpr int64_t rows_per_wave = (512 * C) >> L;
    const int64_t waves = (m + rows_per_wave - 1) / rows_per_wave;
    const int64_t blocks = (waves + WPB - 1) / WPB;
    hipLaunchKernelGGL((fwht_wave_kernel<DT, L, C, WPB, true>), dim3((uint32_t)blocks),
                       dim3(kWave * WPB), 0, stream, in, in_stride, out, out_stride, m, scale);
  } else {
    hipLaunchKernelGGL((fwht_block_kernel<DT, L, C, HALVES, true>), dim3((uint32_t)m),
                       dim3((1 << L) / (8 * C)), 0, stream, in, in_stride, out, out_stride,
                       scale);
  }
  return hipGetLastError();
}

// Per-size configuration, chosen from measured HBM throughput on MI355X
// (2^28-element in-place sweeps over chunks per lane, waves per workgroup,
// exchange passes and cache policy): the smallest per-wave footprint that
// holds a row wins for n <= 2048; from n = 4096 on, a row is spread over
// several waves with one LDS exchange, run in two passes where that lets two
// or more workgroups share a CU.
template <int DT, int L>
hipError_t launch(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                  int64_t m, float scale, hipStream_t stream) {
  //                                      C  WPB HALVES
  if constexpr (L <= 9) {
    return launch_cfg<DT, L, 1, 1, 1>(in, in_stride, out, out_stride, m, scale, stream);
  } else if constexpr (L == 10) {
    return launch_cfg<DT, L, 2, 1, 1>(in, in_stride, out, out_stride, m, scale, stream);
  } else if constexpr (L == 11) {
    return launch_cfg<DT, L, 4, 1, 1>(in, in_stride, out, out_stride, m, scale, stream);
  } else if constexpr (L == 12) {
    return launch_cfg<DT, L, 4, 1, 1>(in, in_stride, out, out_stride, m, scale, stream);
  } else if constexpr (L == 13) {
    return launch_cfg<DT, L, 4, 1, 2>(in, in_stride, out, out_stride, m, scale, stream);
  } else {
    return launch_cfg<DT, L, 8, 1, 2>(in, in_stride, out, out_stride, m, scale, stream);
  }
}

template <int DT>
hipError_t launch_dt(int L, const uint16_t *in, int64_t in_stride, uint16_t *out,
                     int64_t out_stride, int64_t m, float scale, hipStream_t stream) {
  switch (L) {
    case 7: return launch<DT, 7>(in, in_stride, out, out_stride, m, scale, stream);
    case 8: return launch<DT, 8>(in, in_stride, out, out_stride, m, scale, stream);
    case 9: return launch<DT, 9>(in, in_stride, out, out_stride, m, scale, stream);
    case 10: return launch<DT, 10>(in, in_stride, out, out_stride, m, scale, stream);
    case 11: return launch<DT, 11>(in, in_stride, out, out_stride, m, scale, stream);
    case 12: return launch<DT, 12>(in, in_stride, out, out_stride, m, scale, stream);
    case 13: return launch<DT, 13>(in, in_stride, out, out_stride, m, scale, stream);
    case 14: return launch<DT, 14>(in, in_stride, out, out_stride, m, scale, stream);
    case 15: return launch<DT, 15>(in, in_stride, out, out_stride, m, scale, stream);
    default: return hipErrorInvalidValue;
  }
}

// Architecture check, cached per device: 0 unknown, 1 gfx950, 2 other.
constexpr int kMaxDevices = 64;
std::atomic<int> g_arch_state[kMaxDevices];

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
  if (dev < kMaxDevices) g_arch_state[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
  return ok ? HADACORE_SUCCESS : HADACORE_ERROR_UNSUPPORTED_DEVICE;
}

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
                         float scale, int *L_out) {
  if (m < 0) return HADACORE_ERROR_INVALID_VALUE;
  const int L = log2_exact(n);
  if (L < 7 || L > 15) return HADACORE_ERROR_INVALID_SIZE;
  if (dtype != HADACORE_FP16 && dtype != HADACORE_BF16) return HADACORE_ERROR_INVALID_DTYPE;
  if (!isfinite(scale)) return HADACORE_ERROR_INVALID_VALUE;
  if (in_row_stride < n || out_row_stride < n || (in_row_stride % 8) != 0 ||
      (out_row_stride % 8) != 0)
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
  const hipError_t err =
      dtype == HADACORE_FP16
          ? launch_dt<HADACORE_FP16>(L, src, in_row_stride, dst, out_row_stride, m, scale, s)
          : launch_dt<HADACORE_BF16>(L, src, in_row_stride, dst, out_row_stride, m, scale, s);
  return err == hipSuccess ? HADACORE_SUCCESS : HADACORE_ERROR_LAUNCH;
}

extern "C" hadacore_status hadamard_transform(const void *in, void *out, int64_t m, int64_t n,
                                              hadacore_dtype dtype, float scale, void *stream) {
  return hadamard_transform_strided(in, n, out, n, m, n, dtype, scale, stream);
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
  hipLaunchKernelGGL(stream_copy_kernel, dim3((uint32_t)((count + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint16_t *>(src),
                     static_cast<uint16_t *>(dst), count);
  return hipGetLastError() == hipSuccess ? HADACORE_SUCCESS : HADACORE_ERROR_LAUNCH;
}

extern "C" const char *hadacore_status_string(hadacore_status status) {
  switch (status) {
    case HADACORE_SUCCESS: return "success";
    case HADACORE_ERROR_INVALID_VALUE: return "invalid value (m < 0, null pointer or non-finite scale)";
    case HADACORE_ERROR_INVALID_SIZE: return "invalid size (n must be a power of two in [128, 32768])";
    case HADACORE_ERROR_INVALID_DTYPE: return "invalid dtype (expected HADACORE_FP16 or HADACORE_BF16)";
    case HADACORE_ERROR_INVALID_STRIDE: return "invalid row stride (must be >= n and a multiple of 8)";
    case HADACORE_ERROR_MISALIGNED: return "misaligned pointer (16-byte alignment required)";
    case HADACORE_ERROR_OVERLAP: return "input and output overlap without being the same layout";
    case HADACORE_ERROR_LAUNCH: return "kernel launch failed";
    case HADACORE_ERROR_UNSUPPORTED_DEVICE: return "current device is not gfx950";
    case HADACORE_ERROR_TOO_LARGE: return "problem too large for one launch";
    default: return "unknown status";
  }
}

extern "C" int32_t hadacore_version(void) { return HADACORE_VERSION; }
