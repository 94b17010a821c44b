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

// Candidate order used everywhere a top-K is taken: larger value first, then smaller id.
__device__ inline bool better(float v, int id, float w, int jd) {
  return v > w || (v == w && id < jd);
}
__device__ inline bool better_d(double v, long long id, double w, long long jd) {
  return v > w || (v == w && id < jd);
}

// Stable insertion of (v, id) into a descending list of KMAX entries held in registers.
template <int KMAX>
__device__ inline void topk_insert(float (&val)[KMAX], int (&ids)[KMAX], float v, int id) {
  if (!better(v, id, val[KMAX - 1], ids[KMAX - 1])) return;
  bool moving = false;
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    bool take = moving || better(v, id, val[i], ids[i]);
    if (take) {
      float tv = val[i];
      int ti = ids[i];
      val[i] = v;
      ids[i] = id;
      v = tv;
      id = ti;
      moving = true;
    }
  }
}

template <int KMAX>
__device__ inline void topk_clear(float (&val)[KMAX], int (&ids)[KMAX]) {
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    val[i] = -__builtin_inff();
    ids[i] = 0x7fffffff;
  }
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
