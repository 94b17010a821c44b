// Global "general" attention over the source memory (Section 2 attention pooling; Section 4.2 attention
// types; Figure 1(a) caption) for all beam rows of one sentence per workgroup.
//
// score e[k, s] = q_k . keys[s] with keys = W_a m_s precomputed once per batch; pads (s >= n_b) are
// excluded, so their weight is exactly zero; a[k, :] = softmax over the real positions;
// ctx_k = sum_s a[k, s] m_s. The sentence's keys and memory are read once per step and shared by its
// K beam rows. The step is latency-bound (a few hundred KB per sentence), so every phase issues its
// loads in unrolled batches to keep many of them in flight.

#include "common.h"
#include "kernels.h"

namespace onmt {

constexpr int kAttnThreads = 512;
constexpr int kLanesPerPos = 16;     // lanes cooperating on one source position's dot products
constexpr int kKeyChunks = 16;       // float4 chunks of one key row held per lane (H <= 1024)
constexpr int kCtxUnroll = 4;

template <int KMAX>
__global__ __launch_bounds__(kAttnThreads) void k_attention(const float* __restrict__ q, int ld_q,
                                                            const float* __restrict__ keys,
                                                            const float* __restrict__ mem,
                                                            const int32_t* __restrict__ lens, int S_max, int H,
                                                            int Hm, int K, int G, float* __restrict__ ctx,
                                                            float* __restrict__ attn) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  float* qs = lds;                       // [K][H]
  float* es = lds + K * H;               // [K][S_max]
  float* red = es + K * S_max;           // [groups - 1][K][Hm] partial contexts
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int n = lens[b];
  const int r0 = b * K;
  const int H4 = H / 4, Hm4 = Hm / 4;

  for (int e = tid; e < K * H4; e += kAttnThreads) {
    const int k = e / H4, c = e % H4;
    *(float4*)(qs + k * H + 4 * c) = *(const float4*)(q + (size_t)(r0 + k) * ld_q + 4 * c);
  }
  __syncthreads();

  // scores: 16 lanes per source position, the position's key row loaded in one batch
  const int grp = tid / kLanesPerPos, sub = tid % kLanesPerPos;
  constexpr int kGroups = kAttnThreads / kLanesPerPos;
  const float* kb = keys + (size_t)b * S_max * H;
  for (int s0 = 0; s0 < n; s0 += kGroups) {
    const int s = s0 + grp;
    float4 kv[kKeyChunks];
#pragma unroll
    for (int j = 0; j < kKeyChunks; ++j) {
      const int c = sub + j * kLanesPerPos;
      kv[j] = (s < n && c < H4) ? *(const float4*)(kb + (size_t)s * H + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float acc[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      acc[k] = 0.f;
      if (k < K) {
#pragma unroll
        for (int j = 0; j < kKeyChunks; ++j) {
          const int c = sub + j * kLanesPerPos;
          if (c < H4) {
            const float4 qv = *(const float4*)(qs + k * H + 4 * c);
            acc[k] += kv[j].x * qv.x + kv[j].y * qv.y + kv[j].z * qv.z + kv[j].w * qv.w;
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

  // context: thread (group gi, column chunk c) sums positions gi, gi + G, ...; groups are then
  // combined in a fixed order through LDS (deterministic).
  const float* mb = mem + (size_t)b * S_max * Hm;
  for (int c0 = 0; c0 < Hm4; c0 += kAttnThreads / G) {
    const int c = c0 + tid % (kAttnThreads / G);
    const int gi = tid / (kAttnThreads / G);
    const bool act = c < Hm4 && gi < G;
    float4 acc[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (act) {
      for (int s = gi; s < n; s += G * kCtxUnroll) {
        float4 mv[kCtxUnroll];
#pragma unroll
        for (int u = 0; u < kCtxUnroll; ++u) {
          const int ss = s + u * G;
          mv[u] = ss < n ? *(const float4*)(mb + (size_t)ss * Hm + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < kCtxUnroll; ++u) {
          const int ss = s + u * G;
          if (ss < n) {
#pragma unroll
            for (int k = 0; k < KMAX; ++k) {
              if (k < K) {
                const float a = es[k * S_max + ss];
                acc[k].x += a * mv[u].x;
                acc[k].y += a * mv[u].y;
                acc[k].z += a * mv[u].z;
                acc[k].w += a * mv[u].w;
              }
            }
          }
        }
      }
    }
    if (G > 1) {
      if (act && gi > 0) {
#pragma unroll
        for (int k = 0; k < KMAX; ++k)
          if (k < K) *(float4*)(red + ((size_t)(gi - 1) * K + k) * Hm + 4 * c) = acc[k];
      }
      __syncthreads();
      if (act && gi == 0) {
        for (int j = 1; j < G; ++j) {
#pragma unroll
          for (int k = 0; k < KMAX; ++k) {
            if (k < K) {
              const float4 o = *(const float4*)(red + ((size_t)(j - 1) * K + k) * Hm + 4 * c);
              acc[k].x += o.x;
              acc[k].y += o.y;
              acc[k].z += o.z;
              acc[k].w += o.w;
            }
          }
        }
      }
      __syncthreads();
    }
    if (act && gi == 0) {
#pragma unroll
      for (int k = 0; k < KMAX; ++k)
        if (k < K) *(float4*)(ctx + (size_t)(r0 + k) * Hm + 4 * c) = acc[k];
    }
  }
}

constexpr size_t kAttnLdsLimit = 64 * 1024;

static size_t lds_for(int S_max, int H, int K, int G) {
  return (size_t)K * (H + S_max) * sizeof(float) + (size_t)(G - 1) * K * H * sizeof(float);
}

// Position groups for the context phase: as many as the threads allow (at most 4) within the LDS limit.
static int ctx_groups(int S_max, int H, int K) {
  int g = kAttnThreads / (H / 4);
  g = g < 1 ? 1 : (g > 4 ? 4 : g);
  while (g > 1 && lds_for(S_max, H, K, g) > kAttnLdsLimit) --g;
  return g;
}

size_t attention_lds_bytes(int S_max, int H, int K) { return lds_for(S_max, H, K, 1); }

hipError_t attention(const float* q, int ld_q, const float* keys, const float* mem, const int32_t* lens, int B,
                     int S_max, int H, int Hm, int K, float* ctx, float* attn, hipStream_t st) {
  if (H / 4 > kLanesPerPos * kKeyChunks || Hm != H) return hipErrorInvalidValue;
  const int G = ctx_groups(S_max, H, K);
  const size_t lds = lds_for(S_max, H, K, G);
  if (lds > kAttnLdsLimit) return hipErrorInvalidValue;
  dim3 grid(B), block(kAttnThreads);
  if (K <= 1)
    hipLaunchKernelGGL(k_attention<1>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, G, ctx, attn);
  else if (K <= 2)
    hipLaunchKernelGGL(k_attention<2>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, G, ctx, attn);
  else if (K <= 4)
    hipLaunchKernelGGL(k_attention<4>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, G, ctx, attn);
  else if (K <= 8)
    hipLaunchKernelGGL(k_attention<8>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, G, ctx, attn);
  else
    hipLaunchKernelGGL(k_attention<16>, grid, block, lds, st, q, ld_q, keys, mem, lens, S_max, H, Hm, K, G, ctx, attn);
  return hipGetLastError();
}

}  // namespace onmt
