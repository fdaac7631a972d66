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
//     quad_perm; xor 8 by row_ror:8), ds_swizzle (xor 4, xor 16) or
//     ds_bpermute (xor 32), and each lane forms partner + sign*self;
//   * wave bits (n > 512*C): one LDS exchange swaps the wave bits with low
//     chunk bits, after which they are register butterflies too.  The store
//     uses the exchanged layout, so there is no exchange back.
// Global loads and stores are 16-byte per lane and 1 KiB contiguous per wave
// instruction in every layout.  Inputs are widened exactly and multiplied by
// the scale first (no fp32 overflow for large bf16 rows), every intermediate
// is fp32 and the result is rounded once, round-to-nearest-even.
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

constexpr int kWave = 64;

// ---- 16-bit <-> fp32 ------------------------------------------------------

// Widens the packed pair in `u` (element 2i in the low half) and scales it.
template <int DT>
__device__ __forceinline__ f2 widen(uint32_t u, float s) {
  if constexpr (DT == HADACORE_FP16) {
    return __builtin_convertvector(__builtin_bit_cast(h2, u), f2) * s;
  } else {
    f2 r = {__builtin_bit_cast(float, u << 16), __builtin_bit_cast(float, u & 0xffff0000u)};
    return r * s;
  }
}

// Rounds a pair to the 16-bit dtype (round-to-nearest-even) and packs it.
template <int DT>
__device__ __forceinline__ uint32_t narrow(float lo, float hi) {
  f2 v = {lo, hi};
  if constexpr (DT == HADACORE_FP16) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
  } else {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf2));
  }
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

// Value of `x` held by lane (lane ^ (1 << LB)).
template <int LB>
__device__ __forceinline__ float partner(float x, int lane) {
  const int xi = __builtin_bit_cast(int, x);
  int r;
  if constexpr (LB == 0) {
    r = __builtin_amdgcn_mov_dpp(xi, 0xB1, 0xF, 0xF, true);   // quad_perm:[1,0,3,2]
  } else if constexpr (LB == 1) {
    r = __builtin_amdgcn_mov_dpp(xi, 0x4E, 0xF, 0xF, true);   // quad_perm:[2,3,0,1]
  } else if constexpr (LB == 2) {
    r = __builtin_amdgcn_ds_swizzle(xi, 0x101F);              // bitmask mode, xor 4
  } else if constexpr (LB == 3) {
    r = __builtin_amdgcn_mov_dpp(xi, 0x128, 0xF, 0xF, true);  // row_ror:8 == xor 8
  } else if constexpr (LB == 4) {
    r = __builtin_amdgcn_ds_swizzle(xi, 0x401F);              // bitmask mode, xor 16
  } else {
    r = __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, xi);   // xor 32
  }
  return __builtin_bit_cast(float, r);
}

// Radix-2 stage on lane bit LB: the lane with the bit clear keeps a + b, the
// lane with the bit set keeps a - b, where a is the lower lane's value.
template <int LB, int N>
__device__ __forceinline__ void lane_stage(float (&v)[N], int lane) {
  const float sgn = (lane & (1 << LB)) ? -1.0f : 1.0f;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const float p = partner<LB>(v[i], lane);
    v[i] = __builtin_fmaf(v[i], sgn, p);
  }
}

// All stages whose bits lie inside one wave: in-chunk bits 0-2, the chunk bits
// that are element bits (tile bits 9.. below L), and the lane bits (tile bits
// 3-8) below L.
template <int L, int C, int N>
__device__ __forceinline__ void wave_stages(float (&v)[N], int lane) {
  reg_stage<0>(v);
  reg_stage<1>(v);
  reg_stage<2>(v);
  if constexpr (C >= 2 && L > 9) reg_stage<3>(v);
  if constexpr (C >= 4 && L > 10) reg_stage<4>(v);
  if constexpr (C >= 8 && L > 11) reg_stage<5>(v);
  static_assert(C <= 8, "at most 8 chunks per lane");
  if constexpr (L > 3) lane_stage<0>(v, lane);
  if constexpr (L > 4) lane_stage<1>(v, lane);
  if constexpr (L > 5) lane_stage<2>(v, lane);
  if constexpr (L > 6) lane_stage<3>(v, lane);
  if constexpr (L > 7) lane_stage<4>(v, lane);
  if constexpr (L > 8) lane_stage<5>(v, lane);
}

template <int DT, int C>
__device__ __forceinline__ void widen_chunks(const uint4 (&raw)[C], float (&v)[C * 8], float s) {
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const uint32_t w[4] = {raw[k].x, raw[k].y, raw[k].z, raw[k].w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f2 p = widen<DT>(w[q], s);
      v[k * 8 + 2 * q] = p.x;
      v[k * 8 + 2 * q + 1] = p.y;
    }
  }
}

template <int DT>
__device__ __forceinline__ uint4 narrow_chunk(const float *v) {
  uint4 r;
  r.x = narrow<DT>(v[0], v[1]);
  r.y = narrow<DT>(v[2], v[3]);
  r.z = narrow<DT>(v[4], v[5]);
  r.w = narrow<DT>(v[6], v[7]);
  return r;
}

// ---- kernels ------------------------------------------------------------------

// n <= 512*C: each wave owns a tile of 512*C elements = 512*C/n whole rows and
// runs every stage inside the wave.  WPB independent waves per workgroup.
template <int DT, int L, int C, int WPB>
__global__ __launch_bounds__(kWave *WPB) void fwht_wave_kernel(
    const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride, int64_t m,
    float scale) {
  constexpr int kTile = 512 * C;
  static_assert((1 << L) <= kTile, "row does not fit a wave tile");
  constexpr int kRows = kTile >> L;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int64_t row0 = ((int64_t)blockIdx.x * WPB + wave) * kRows;
  if (row0 >= m) return;

  uint4 raw[C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int t = (k * kWave + lane) * 8;
    const int64_t row = row0 + (t >> L);
    const int col = t & ((1 << L) - 1);
    if (row < m) {
      raw[k] = *reinterpret_cast<const uint4 *>(in + row * in_stride + col);
    } else {
      raw[k] = make_uint4(0, 0, 0, 0);
    }
  }
  float v[C * 8];
  widen_chunks<DT, C>(raw, v, scale);
  wave_stages<L, C>(v, lane);
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int t = (k * kWave + lane) * 8;
    const int64_t row = row0 + (t >> L);
    const int col = t & ((1 << L) - 1);
    if (row < m) {
      *reinterpret_cast<uint4 *>(out + row * out_stride + col) = narrow_chunk<DT>(&v[k * 8]);
    }
  }
}

// n = 512*C*NW with NW >= 2 waves per row: one row per workgroup.  After the
// in-wave stages the wave bits are exchanged with the low log2(NW) chunk bits
// through LDS (fp32), then finished as register stages.
template <int DT, int L, int C>
__global__ __launch_bounds__((1 << L) / (8 * C)) void fwht_block_kernel(
    const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride, float scale) {
  constexpr int n = 1 << L;
  constexpr int NW = n / (512 * C);
  static_assert(NW >= 2 && NW <= C, "wave bits must fit the chunk bits");
  // LDS word address of tile element ((W*64 + l)*8 + 4h + q): ((W*2 + h)*64 + l)*4 + q,
  // so each 16-byte access of a wave is 1 KiB contiguous (no bank conflicts).
  __shared__ float4 lds[n / 4];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int64_t row = blockIdx.x;
  const uint16_t *src = in + row * in_stride;
  uint16_t *dst = out + row * out_stride;

  uint4 raw[C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    raw[k] = *reinterpret_cast<const uint4 *>(src + ((w * C + k) * kWave + lane) * 8);
  }
  float v[C * 8];
  widen_chunks<DT, C>(raw, v, scale);
  wave_stages<L, C>(v, lane);

#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int W = w * C + k;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      lds[(W * 2 + h) * kWave + lane] =
          make_float4(v[k * 8 + 4 * h], v[k * 8 + 4 * h + 1], v[k * 8 + 4 * h + 2],
                      v[k * 8 + 4 * h + 3]);
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int W = (k % NW) * C + (k / NW) * NW + w;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float4 f = lds[(W * 2 + h) * kWave + lane];
      v[k * 8 + 4 * h] = f.x;
      v[k * 8 + 4 * h + 1] = f.y;
      v[k * 8 + 4 * h + 2] = f.z;
      v[k * 8 + 4 * h + 3] = f.w;
    }
  }
  reg_stage<3>(v);
  if constexpr (NW >= 4) reg_stage<4>(v);
  if constexpr (NW >= 8) reg_stage<5>(v);
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int W = (k % NW) * C + (k / NW) * NW + w;
    *reinterpret_cast<uint4 *>(dst + (W * kWave + lane) * 8) = narrow_chunk<DT>(&v[k * 8]);
  }
}

// 16-byte streaming copy (grid-stride), the bandwidth reference for the transform.
__global__ __launch_bounds__(256) void stream_copy_kernel(const uint4 *src, uint4 *dst,
                                                          int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) {
    dst[i] = src[i];
  }
}

// ---- host dispatch ------------------------------------------------------------

constexpr int kChunks = 8;     // fp32 registers per lane = 8 * kChunks
constexpr int kWavesPerBlock = 4;

template <int DT, int L>
hipError_t launch(const uint16_t *in, int64_t in_stride, uint16_t *out, int64_t out_stride,
                  int64_t m, float scale, hipStream_t stream) {
  if constexpr ((1 << L) <= 512 * kChunks) {
    constexpr int64_t rows_per_wave = (512 * kChunks) >> L;
    const int64_t waves = (m + rows_per_wave - 1) / rows_per_wave;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((fwht_wave_kernel<DT, L, kChunks, kWavesPerBlock>), dim3((uint32_t)blocks),
                       dim3(kWave * kWavesPerBlock), 0, stream, in, in_stride, out, out_stride, m,
                       scale);
  } else {
    hipLaunchKernelGGL((fwht_block_kernel<DT, L, kChunks>), dim3((uint32_t)m),
                       dim3((1 << L) / (8 * kChunks)), 0, stream, in, in_stride, out, out_stride,
                       scale);
  }
  return hipGetLastError();
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

}  // namespace
}  // namespace hadacore

using namespace hadacore;

extern "C" hadacore_status hadamard_transform_strided(const void *in, int64_t in_row_stride,
                                                      void *out, int64_t out_row_stride,
                                                      int64_t m, int64_t n, hadacore_dtype dtype,
                                                      float scale, void *stream) {
  if (m < 0) return HADACORE_ERROR_INVALID_VALUE;
  const int L = log2_exact(n);
  if (L < 7 || L > 15) return HADACORE_ERROR_INVALID_SIZE;
  if (dtype != HADACORE_FP16 && dtype != HADACORE_BF16) return HADACORE_ERROR_INVALID_DTYPE;
  if (!isfinite(scale)) return HADACORE_ERROR_INVALID_VALUE;
  if (in_row_stride < n || out_row_stride < n || (in_row_stride % 8) != 0 ||
      (out_row_stride % 8) != 0)
    return HADACORE_ERROR_INVALID_STRIDE;
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
  const hadacore_status dev = check_device();
  if (dev != HADACORE_SUCCESS) return dev;
  const int64_t count = bytes / 16;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 256 * 64) blocks = 256 * 64;  // grid-stride beyond 64 blocks per CU
  hipLaunchKernelGGL(stream_copy_kernel, dim3((uint32_t)blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint4 *>(src),
                     static_cast<uint4 *>(dst), count);
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
