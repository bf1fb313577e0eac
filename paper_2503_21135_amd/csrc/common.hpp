// common.hpp -- helpers shared by the gfx950 kernels of the MoE expert-FFN
// library.  Everything here is device arithmetic on bit patterns or HIP
// plumbing; no file of the CPU reference is included or mirrored.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>

#include "moe_quant.h"

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- host side
inline bool debug_sync() {
  static int v = -1;
  if (v < 0) {
    const char* e = std::getenv("MOE_DEBUG");
    v = (e && e[0] == '1') ? 1 : 0;
  }
  return v == 1;
}

inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

// Status of the launches just enqueued on `s`.
inline int launch_status(hipStream_t s) {
  if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
  if (debug_sync()) {
    if (hipStreamSynchronize(s) != hipSuccess) return MOE_ERR_HIP;
    if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
  }
  return MOE_OK;
}

// Quantized bit-widths (codes, copies, requantization).
inline bool valid_bits(int b) { return b == 2 || b == 3 || b == 4 || b == 6 || b == 8; }
// Widths an expert of the FFN may have: the quantized ones, or 16 for the
// unquantized bf16 reference weights.
inline bool valid_expert_bits(int b) { return valid_bits(b) || b == 16; }

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Row stride (32-bit words) of packed code matrices: K*bits/32 plus 64 bytes
// (128 bytes at 8 and 16 bits), so that rows never start a power of two of bytes
// apart -- a wavefront reads 16 rows at once, and rows 2^n bytes apart fall on
// few HBM channels (measured on MI355X: 4-bit rows of 2048 bytes stream at
// 6.1 TB/s unpadded, 6.8 TB/s padded).
__host__ __device__ constexpr int64_t code_row_words(int64_t K, int bits) {
  return K * bits / 32 + (bits >= 8 ? 32 : 16);
}

// ---------------------------------------------------------------- device side
__device__ __forceinline__ float bf16_lo(uint32_t w) {
  return __uint_as_float(w << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t w) {
  return __uint_as_float(w & 0xFFFF0000u);
}

// fp32 -> bf16 bit pattern, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// true when f converts to a finite binary16 value (|f| <= 65504; NaN and
// larger magnitudes do not)
__device__ __forceinline__ bool fp16_finite(float f) { return __builtin_fabsf(f) <= 65504.0f; }

__device__ __forceinline__ float fp16_bits_to_f32(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}

__device__ __forceinline__ f32x4 mfma16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

}  // namespace moe
