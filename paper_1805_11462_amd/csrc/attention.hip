// Global attention over the source memory (Section 2 attention pooling; Section 4.2 attention types;
// Figure 1(a) caption).
//
// Scores, with keys precomputed once per batch:
//   general  e[k, s] = q_k . keys[s], keys = W_a m_s;
//   dot      e[k, s] = q_k . m_s (the keys are the memory);
//   concat   e[k, s] = v_a . tanh(q'_k + keys[s]), q'_k = W_q q_k (one GEMM per step), keys = W_m m_s,
//            where W_a = [W_q | W_m] splits the score's weight into its query and memory columns.
// Pads (s >= n_b) are excluded, so their weight is exactly zero; a[k, :] = softmax over the real
// positions; ctx_k = sum_s a[k, s] m_s.
//
// The step moves a few hundred KB per sentence, so it is bound by how many loads are in flight, not by
// arithmetic. It runs as two launches that each issue all of their loads up front:
//   k_attn_scores  one workgroup per (sentence, 8 source positions): the positions' key rows are read
//                  once and dotted with the sentence's K query rows;
//   k_attn_context one workgroup per (sentence, group of memory columns): every group repeats the
//                  (cheap) softmax over the sentence's K x n scores, then reduces its columns of the
//                  memory rows, which it started loading before the softmax.
// Keys and memory are each read once per step, and all reductions run in a fixed order.

#include "common.h"
#include "kernels.h"

namespace onmt {

constexpr int kScoreThreads = 256;
constexpr int kScoreLanes = 32;                             // lanes per source position
constexpr int kScorePos = kScoreThreads / kScoreLanes;      // source positions per workgroup
constexpr int kScoreChunks = 8;                             // float4 chunks of a key row per lane (H <= 1024)
constexpr int kCtxThreads = 512;
constexpr int kCtxBatch = 4;                                // memory rows in flight per thread
constexpr int kCtxTargetBlocks = 256;                       // at least one workgroup per CU when B allows
constexpr size_t kAttnLdsLimit = 64 * 1024;

// tanh(x) = 1 - 2 / (exp(2x) + 1) with the hardware exponential and reciprocal; it saturates to +-1 for
// large |x| (the exponential overflows to inf or underflows to 0). Absolute error about 1e-7.
__device__ inline float tanh_fast(float x) { return 1.f - 2.f * __builtin_amdgcn_rcpf(__expf(2.f * x) + 1.f); }

template <bool CONCAT>
__device__ inline float score_term(float4 k, float4 q, float4 v) {
  if (CONCAT)
    return v.x * tanh_fast(k.x + q.x) + v.y * tanh_fast(k.y + q.y) + v.z * tanh_fast(k.z + q.z) +
           v.w * tanh_fast(k.w + q.w);
  return k.x * q.x + k.y * q.y + k.z * q.z + k.w * q.w;
}

// e [B*K, S_max]: raw scores of the real positions (pads are never written). v: concat's v_a [H], unused
// otherwise.
template <int KMAX, bool CONCAT>
__global__ __launch_bounds__(kScoreThreads) void k_attn_scores(const float* __restrict__ q, int ld_q,
                                                               const float* __restrict__ keys,
                                                               const float* __restrict__ v,
                                                               const int32_t* __restrict__ lens, int S_max, int H,
                                                               int K, int nchunk, float* __restrict__ e) {
  extern __shared__ __attribute__((aligned(16))) float qs[];      // [K][H]
  const int b = blockIdx.x / nchunk, p = blockIdx.x % nchunk;
  const int n = lens[b];
  const int s0 = p * kScorePos;
  if (s0 >= n) return;
  const int tid = threadIdx.x;
  const int sub = tid % kScoreLanes;
  const int s = s0 + tid / kScoreLanes;
  const int H4 = H / 4;
  // the key row first: its loads depend on nothing (rows past n re-read row s0, results unused)
  const float* kr = keys + ((size_t)b * S_max + (s < n ? s : s0)) * H;
  float4 kv[kScoreChunks];
#pragma unroll
  for (int j = 0; j < kScoreChunks; ++j) {
    const int c = sub + j * kScoreLanes;
    kv[j] = c < H4 ? *(const float4*)(kr + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float4 vv[kScoreChunks];
#pragma unroll
  for (int j = 0; j < kScoreChunks; ++j) {
    const int c = sub + j * kScoreLanes;
    vv[j] = CONCAT && c < H4 ? *(const float4*)(v + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  // the sentence's K query rows to LDS, all loads issued before the first store
  const int r0 = b * K;
  constexpr int QPT = KMAX * kScoreChunks * kScoreLanes / kScoreThreads;   // >= K * H4 / threads
  float4 qv[QPT];
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int i = tid + u * kScoreThreads;
    qv[u] = i < K * H4 ? *(const float4*)(q + (size_t)(r0 + i / H4) * ld_q + 4 * (i % H4))
                       : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int i = tid + u * kScoreThreads;
    if (i < K * H4) *(float4*)(qs + (i / H4) * H + 4 * (i % H4)) = qv[u];
  }
  __syncthreads();
  float acc[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    acc[k] = 0.f;
    if (k < K) {
#pragma unroll
      for (int j = 0; j < kScoreChunks; ++j) {
        const int c = sub + j * kScoreLanes;
        if (c < H4) {
          acc[k] += score_term<CONCAT>(kv[j], *(const float4*)(qs + k * H + 4 * c), vv[j]);
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
#pragma unroll
    for (int o = kScoreLanes / 2; o > 0; o >>= 1) acc[k] += __shfl_xor(acc[k], o, kWave);
  }
  if (sub == 0 && s < n) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (k < K) e[(size_t)(r0 + k) * S_max + s] = acc[k];
  }
}

// Thread (pl, c): pl = one of PL position lanes (adjacent lanes of a wave), c = one float4 column of the
// group's CW = kCtxThreads / PL columns. Positions pl, pl + PL, ... are summed per thread, then across
// the PL lanes by butterfly shuffles.
template <int KMAX, int PL>
__global__ __launch_bounds__(kCtxThreads) void k_attn_context(const float* __restrict__ e,
                                                              const float* __restrict__ mem,
                                                              const int32_t* __restrict__ lens, int S_max, int Hm,
                                                              int K, int G, float* __restrict__ ctx,
                                                              float* __restrict__ attn, Coverage cov,
                                                              int32_t* __restrict__ align) {
  extern __shared__ __attribute__((aligned(16))) float as[];      // [K][S_max] attention weights
  constexpr int CW = kCtxThreads / PL;
  const int b = blockIdx.x / G, g = blockIdx.x % G;
  const int n = lens[b];
  const int tid = threadIdx.x;
  const int pl = tid % PL;
  const int c = g * CW + tid / PL;
  const int Hm4 = Hm / 4;
  const bool col_ok = c < Hm4;
  const float* mb = mem + (size_t)b * S_max * Hm + 4 * (col_ok ? c : 0);
  // first batch of memory rows, issued before the softmax, which it does not depend on
  float4 mv[kCtxBatch];
#pragma unroll
  for (int u = 0; u < kCtxBatch; ++u) {
    const int s = pl + u * PL;
    mv[u] = (col_ok && s < n) ? *(const float4*)(mb + (size_t)s * Hm) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  // the sentence's K x n scores to LDS, kCtxBatch loads in flight per thread
  const int r0 = b * K;
  for (int i0 = 0; i0 < K * n; i0 += kCtxBatch * kCtxThreads) {
    float ev[kCtxBatch];
#pragma unroll
    for (int u = 0; u < kCtxBatch; ++u) {
      const int i = i0 + tid + u * kCtxThreads;
      ev[u] = i < K * n ? e[(size_t)(r0 + i / n) * S_max + i % n] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kCtxBatch; ++u) {
      const int i = i0 + tid + u * kCtxThreads;
      if (i < K * n) as[(i / n) * S_max + i % n] = ev[u];
    }
  }
  __syncthreads();

  // softmax over the real positions, one wave per row
  const int wave = tid / kWave, lane = tid % kWave;
  for (int k = wave; k < K; k += kCtxThreads / kWave) {
    float* row = as + k * S_max;
    float mx = -__builtin_inff();
    for (int s = lane; s < n; s += kWave) mx = fmaxf(mx, row[s]);
    mx = wave_max(mx);
    float sm = 0.f;
    for (int s = lane; s < n; s += kWave) {
      const float pv = __expf(row[s] - mx);
      row[s] = pv;
      sm += pv;
    }
    sm = wave_sum(sm);
    const float inv = 1.0f / sm;
    for (int s = lane; s < n; s += kWave) row[s] *= inv;
    if (attn && g == 0) {
      for (int s = lane; s < S_max; s += kWave) attn[(size_t)(r0 + k) * S_max + s] = s < n ? row[s] : 0.f;
    }
    if (align && g == 0) {
      // largest weight, smaller position on ties
      float bv = -1.f;
      int bs = 0x7fffffff;
      for (int s = lane; s < n; s += kWave) {
        if (row[s] > bv) {                    // s increases per lane, so strict keeps the smaller s
          bv = row[s];
          bs = s;
        }
      }
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) {
        const float ov = __shfl_xor(bv, o, kWave);
        const int os = __shfl_xor(bs, o, kWave);
        if (ov > bv || (ov == bv && os < bs)) {
          bv = ov;
          bs = os;
        }
      }
      if (lane == 0) align[r0 + k] = bs;
    }
    if (cov.out && g == 0) {
      // coverage of this row's hypothesis: its parent's coverage plus this step's weights
      const int r = r0 + k;
      const float* ci = cov.in + (size_t)cov.parent[r] * S_max;
      float* co = cov.out + (size_t)r * S_max;
      double lsum = 0.0;
      for (int s = lane; s < S_max; s += kWave) {
        const float c = s < n ? ci[s] + row[s] : 0.f;
        co[s] = c;
        if (s < n) lsum += (double)logf(fminf(c, 1.f));
      }
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) lsum += __shfl_xor(lsum, o, kWave);
      if (lane == 0) cov.cp[r] = cov.beta * lsum;
    }
  }
  __syncthreads();

  float4 acc[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
  // batches of kCtxBatch rows per thread; the next batch is loaded while the current one is reduced
  for (int sb = 0; sb < n; sb += PL * kCtxBatch) {
    float4 nv[kCtxBatch];
    const int sn = sb + PL * kCtxBatch;
#pragma unroll
    for (int u = 0; u < kCtxBatch; ++u) {
      const int s = sn + pl + u * PL;
      nv[u] = (col_ok && s < n) ? *(const float4*)(mb + (size_t)s * Hm) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < kCtxBatch; ++u) {
      const int s = sb + pl + u * PL;
      if (s < n) {
#pragma unroll
        for (int k = 0; k < KMAX; ++k) {
          if (k < K) {
            const float a = as[k * S_max + s];
            acc[k].x += a * mv[u].x;
            acc[k].y += a * mv[u].y;
            acc[k].z += a * mv[u].z;
            acc[k].w += a * mv[u].w;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kCtxBatch; ++u) mv[u] = nv[u];
  }
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    if (k < K) {                                      // uniform: no shuffles for the rows past K
#pragma unroll
      for (int o = PL / 2; o > 0; o >>= 1) {
        acc[k].x += __shfl_xor(acc[k].x, o, kWave);
        acc[k].y += __shfl_xor(acc[k].y, o, kWave);
        acc[k].z += __shfl_xor(acc[k].z, o, kWave);
        acc[k].w += __shfl_xor(acc[k].w, o, kWave);
      }
    }
  }
  if (pl == 0 && col_ok) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (k < K) *(float4*)(ctx + (size_t)(r0 + k) * Hm + 4 * c) = acc[k];
  }
}

size_t attention_lds_bytes(int S_max, int H, int K) {
  const size_t a = (size_t)K * H * sizeof(float), c = (size_t)K * S_max * sizeof(float);
  return a > c ? a : c;
}

// Position lanes for the context launch: the fewest (widest column groups) that still give every CU a
// workgroup, else 64.
static int ctx_lanes(int B, int Hm4) {
  for (int pl = 4; pl < 64; pl *= 2) {
    const int cw = kCtxThreads / pl;
    if ((long long)B * ((Hm4 + cw - 1) / cw) >= kCtxTargetBlocks) return pl;
  }
  return 64;
}

template <int KMAX>
static void launch_context(int pl, dim3 grid, size_t lds, hipStream_t st, const float* e, const float* mem,
                           const int32_t* lens, int S_max, int Hm, int K, int G, float* ctx, float* attn,
                           const Coverage& cov, int32_t* align) {
  const dim3 block(kCtxThreads);
  switch (pl) {
    case 4: hipLaunchKernelGGL((k_attn_context<KMAX, 4>), grid, block, lds, st, e, mem, lens, S_max, Hm, K, G, ctx, attn, cov, align); break;
    case 8: hipLaunchKernelGGL((k_attn_context<KMAX, 8>), grid, block, lds, st, e, mem, lens, S_max, Hm, K, G, ctx, attn, cov, align); break;
    case 16: hipLaunchKernelGGL((k_attn_context<KMAX, 16>), grid, block, lds, st, e, mem, lens, S_max, Hm, K, G, ctx, attn, cov, align); break;
    case 32: hipLaunchKernelGGL((k_attn_context<KMAX, 32>), grid, block, lds, st, e, mem, lens, S_max, Hm, K, G, ctx, attn, cov, align); break;
    default: hipLaunchKernelGGL((k_attn_context<KMAX, 64>), grid, block, lds, st, e, mem, lens, S_max, Hm, K, G, ctx, attn, cov, align); break;
  }
}

template <bool CONCAT>
static void launch_scores(int K, dim3 grid, size_t lds, hipStream_t st, const float* q, int ld_q,
                          const float* keys, const float* v, const int32_t* lens, int S_max, int H, int nchunk,
                          float* e) {
  const dim3 block(kScoreThreads);
  if (K <= 1)
    hipLaunchKernelGGL((k_attn_scores<1, CONCAT>), grid, block, lds, st, q, ld_q, keys, v, lens, S_max, H, K, nchunk, e);
  else if (K <= 2)
    hipLaunchKernelGGL((k_attn_scores<2, CONCAT>), grid, block, lds, st, q, ld_q, keys, v, lens, S_max, H, K, nchunk, e);
  else if (K <= 4)
    hipLaunchKernelGGL((k_attn_scores<4, CONCAT>), grid, block, lds, st, q, ld_q, keys, v, lens, S_max, H, K, nchunk, e);
  else if (K <= 8)
    hipLaunchKernelGGL((k_attn_scores<8, CONCAT>), grid, block, lds, st, q, ld_q, keys, v, lens, S_max, H, K, nchunk, e);
  else
    hipLaunchKernelGGL((k_attn_scores<16, CONCAT>), grid, block, lds, st, q, ld_q, keys, v, lens, S_max, H, K, nchunk, e);
}

hipError_t attention(const float* q, int ld_q, const float* keys, const float* v_a, const float* mem,
                     const int32_t* lens, int B, int S_max, int H, int Hm, int K, float* scores, float* ctx,
                     float* attn, const AttnExtra& ex, hipStream_t st) {
  const Coverage cv = ex.cov ? *ex.cov : Coverage{};
  if (H / 4 > kScoreLanes * kScoreChunks || H % 4 || Hm % 4 || K < 1 || K > kMaxBeam) return hipErrorInvalidValue;
  if (attention_lds_bytes(S_max, H, K) > kAttnLdsLimit) return hipErrorInvalidValue;
  const int nchunk = (S_max + kScorePos - 1) / kScorePos;
  const dim3 sgrid(B * nchunk);
  const size_t slds = (size_t)K * H * sizeof(float);
  if (v_a)
    launch_scores<true>(K, sgrid, slds, st, q, ld_q, keys, v_a, lens, S_max, H, nchunk, scores);
  else
    launch_scores<false>(K, sgrid, slds, st, q, ld_q, keys, v_a, lens, S_max, H, nchunk, scores);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;

  const int Hm4 = Hm / 4;
  const int pl = ctx_lanes(B, Hm4);
  const int cw = kCtxThreads / pl;
  const int G = (Hm4 + cw - 1) / cw;
  const dim3 cgrid(B * G);
  const size_t clds = (size_t)K * S_max * sizeof(float);
  if (K <= 1) launch_context<1>(pl, cgrid, clds, st, scores, mem, lens, S_max, Hm, K, G, ctx, attn, cv, ex.align);
  else if (K <= 2) launch_context<2>(pl, cgrid, clds, st, scores, mem, lens, S_max, Hm, K, G, ctx, attn, cv, ex.align);
  else if (K <= 4) launch_context<4>(pl, cgrid, clds, st, scores, mem, lens, S_max, Hm, K, G, ctx, attn, cv, ex.align);
  else if (K <= 8) launch_context<8>(pl, cgrid, clds, st, scores, mem, lens, S_max, Hm, K, G, ctx, attn, cv, ex.align);
  else launch_context<16>(pl, cgrid, clds, st, scores, mem, lens, S_max, Hm, K, G, ctx, attn, cv, ex.align);
  return hipGetLastError();
}

}  // namespace onmt
