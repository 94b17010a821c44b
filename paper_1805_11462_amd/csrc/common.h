// Device-side building blocks shared by the gfx950 kernels of libonmt.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace onmt {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;
constexpr int kMaxBeam = 16;        // largest beam the register top-K lists support
constexpr int kUnitGroup = 16;      // LSTM units per gate block in packed weights (one MFMA tile width)

// Round-to-nearest-even float -> bfloat16 bits (finite inputs).
__device__ __host__ inline uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float bf16_bits_to_f32(uint16_t h) {
  return __builtin_bit_cast(float, (uint32_t)h << 16);
}

__device__ inline float sigmoidf_(float x) { return 1.0f / (1.0f + __expf(-x)); }

// Order used by every top-K: larger value first, then smaller id (ids are unique, so this is total).
template <class V, class I>
__device__ inline bool before(V v, I id, V w, I jd) {
  return v > w || (v == w && id < jd);
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

}  // namespace onmt
