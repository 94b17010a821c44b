// Global "general" attention over the source memory (Section 2 attention pooling; Section 4.2 attention
// types; Figure 1(a) caption) for all beam rows of one sentence per workgroup.
//
// score e[k, s] = q_k . keys[s] with keys = W_a m_s precomputed once per batch; pads (s >= n_b) are
// excluded, so their weight is exactly zero; a[k, :] = softmax over the real positions;
// ctx_k = sum_s a[k, s] m_s. The sentence's keys and memory are read from memory once per step and
// shared by its K beam rows.

#include "common.h"
#include "kernels.h"

namespace onmt {

constexpr int kAttnThreads = 256;
constexpr int kLanesPerPos = 16;     // lanes cooperating on one source position's dot products

template <int KMAX>
__global__ __launch_bounds__(kAttnThreads) void k_attention(const float* __restrict__ q, int ld_q,
                                                            const float* __restrict__ keys,
                                                            const float* __restrict__ mem,
                                                            const int32_t* __restrict__ lens, int S_max, int H,
                                                            int Hm, int K, float* __restrict__ ctx,
                                                            float* __restrict__ attn) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  float* qs = lds;                       // [K][H]
  float* es = lds + K * H;               // [K][S_max]
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int n = lens[b];
  const int r0 = b * K;

  for (int e = tid; e < K * (H / 4); e += kAttnThreads) {
    const int k = e / (H / 4), c = e % (H / 4);
    *(float4*)(qs + k * H + 4 * c) = *(const float4*)(q + (size_t)(r0 + k) * ld_q + 4 * c);
  }
  __syncthreads();

  // scores: groups of 16 lanes per source position
  const int grp = tid / kLanesPerPos, sub = tid % kLanesPerPos;
  constexpr int kGroups = kAttnThreads / kLanesPerPos;
  const float* kb = keys + (size_t)b * S_max * H;
  for (int s0 = 0; s0 < n; s0 += kGroups) {
    const int s = s0 + grp;
    float acc[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) acc[k] = 0.f;
    if (s < n) {
      for (int c = sub; c < H / 4; c += kLanesPerPos) {
        const float4 kv = *(const float4*)(kb + (size_t)s * H + 4 * c);
#pragma unroll
        for (int k = 0; k < KMAX; ++k) {
          if (k < K) {
            const float4 qv = *(const float4*)(qs + k * H + 4 * c);
            acc[k] += kv.x * qv.x + kv.y * qv.y + kv.z * qv.z + kv.w * qv.w;
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
#pragma unroll
      for (int o = kLanesPerPos / 2; o > 0; o >>= 1) acc[k] += __shfl_xor(acc[k], o, kWave);
    }
    if (s < n && sub == 0) {
#pragma unroll
      for (int k = 0; k < KMAX; ++k)
        if (k < K) es[k * S_max + s] = acc[k];
    }
  }
  __syncthreads();

  // softmax over real positions, one wave per row
  const int wave = tid / kWave, lane = tid % kWave;
  for (int k = wave; k < K; k += kAttnThreads / kWave) {
    float mx = -__builtin_inff();
    for (int s = lane; s < n; s += kWave) mx = fmaxf(mx, es[k * S_max + s]);
    mx = wave_max(mx);
    float sm = 0.f;
    for (int s = lane; s < n; s += kWave) {
      const float p = __expf(es[k * S_max + s] - mx);
      es[k * S_max + s] = p;
      sm += p;
    }
    sm = wave_sum(sm);
    const float inv = 1.0f / sm;
    for (int s = lane; s < S_max; s += kWave) {
      const float a = s < n ? es[k * S_max + s] * inv : 0.f;
      if (s < n) es[k * S_max + s] = a;
      if (attn) attn[(size_t)(r0 + k) * S_max + s] = a;
    }
  }
  __syncthreads();

  // context: each thread owns 4 memory columns
  const float* mb = mem + (size_t)b * S_max * Hm;
  for (int c = tid; c < Hm / 4; c += kAttnThreads) {
    float4 acc[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < n; ++s) {
      const float4 mv = *(const float4*)(mb + (size_t)s * Hm + 4 * c);
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        if (k < K) {
          const float a = es[k * S_max + s];
          acc[k].x += a * mv.x;
          acc[k].y += a * mv.y;
          acc[k].z += a * mv.z;
          acc[k].w += a * mv.w;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (k < K) *(float4*)(ctx + (size_t)(r0 + k) * Hm + 4 * c) = acc[k];
  }
}

size_t attention_lds_bytes(int S_max, int H, int K) { return (size_t)K * (H + S_max) * sizeof(float); }

hipError_t attention(const float* q, int ld_q, const float* keys, const float* mem, const int32_t* lens, int B,
                     int S_max, int H, int Hm, int K, float* ctx, float* attn, hipStream_t st) {
  const size_t lds = attention_lds_bytes(S_max, H, K);
  dim3 grid(B), block(kAttnThreads);
  if (K <= 1)
    hipLaunchKernelGGL(k_attention<1>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, ctx, attn);
  else if (K <= 2)
    hipLaunchKernelGGL(k_attention<2>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, ctx, attn);
  else if (K <= 4)
    hipLaunchKernelGGL(k_attention<4>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, ctx, attn);
  else if (K <= 8)
    hipLaunchKernelGGL(k_attention<8>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, ctx, attn);
  else
    hipLaunchKernelGGL(k_attention<16>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, ctx, attn);
  return hipGetLastError();
}

}  // namespace onmt
