// Softmax merge, beam step and backtrack kernels (Section 2: softmax layer and item (d) beam search;
// Section 4.2: length normalisation), plus small layout helpers.

#include "common.h"
#include "kernels.h"

namespace onmt {

// ------------------------------------------------------------------ softmax merge
// One workgroup per row: combine per-tile (max, sum exp) into the row's logsumexp, and select the row's
// top-K (larger logit first, smaller id on ties) from the per-tile top-K lists by K rounds of a
// workgroup-wide argmax. Candidates are processed in chunks of 256 * kMergeCap; the running top-K of
// earlier chunks takes part in every later chunk's rounds. Outputs log-probs z - lse.
constexpr int kMergeThreads = 256;
constexpr int kMergeCap = 8;

__device__ inline void block_best(float& v, int& id, float* sv, int* si) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(v, o, kWave);
    const int oi = __shfl_xor(id, o, kWave);
    if (better(ov, oi, v, id)) {
      v = ov;
      id = oi;
    }
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sv[wave] = v;
    si[wave] = id;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kMergeThreads / kWave; ++w)
    if (better(sv[w], si[w], v, id)) {
      v = sv[w];
      id = si[w];
    }
  __syncthreads();
}

__global__ __launch_bounds__(kMergeThreads) void k_lse_topk(const float* __restrict__ pmax,
                                                           const float* __restrict__ psum,
                                                           const float* __restrict__ pval,
                                                           const int32_t* __restrict__ pid, int M, int ntiles,
                                                           int K, float* __restrict__ out_val,
                                                           int32_t* __restrict__ out_id, float* __restrict__ out_lse) {
  __shared__ float sv[kMergeThreads / kWave];
  __shared__ int si[kMergeThreads / kWave];
  __shared__ float run_v[kMaxBeam];
  __shared__ int run_i[kMaxBeam];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const float ninf = -__builtin_inff();
  const size_t base = (size_t)row * ntiles;
  // logsumexp
  float mx = ninf;
  for (int t = tid; t < ntiles; t += kMergeThreads) mx = fmaxf(mx, pmax[base + t]);
  int dummy = 0;
  {
    float v = mx;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    if ((tid & 63) == 0) sv[tid >> 6] = v;
    __syncthreads();
    mx = sv[0];
#pragma unroll
    for (int w = 1; w < kMergeThreads / kWave; ++w) mx = fmaxf(mx, sv[w]);
    __syncthreads();
  }
  float sm = 0.f;
  for (int t = tid; t < ntiles; t += kMergeThreads) sm += psum[base + t] * __expf(pmax[base + t] - mx);
  {
    float v = wave_sum(sm);
    if ((tid & 63) == 0) sv[tid >> 6] = v;
    __syncthreads();
    sm = 0.f;
#pragma unroll
    for (int w = 0; w < kMergeThreads / kWave; ++w) sm += sv[w];
    __syncthreads();
  }
  const float lse = mx + __logf(sm);
  (void)dummy;
  // top-K
  if (tid < kMaxBeam) {
    run_v[tid] = ninf;
    run_i[tid] = 0x7fffffff;
  }
  __syncthreads();
  const int n = ntiles * K;
  for (int c0 = 0; c0 < n; c0 += kMergeThreads * kMergeCap) {
    float v[kMergeCap + 1];
    int id[kMergeCap + 1];
#pragma unroll
    for (int i = 0; i < kMergeCap; ++i) {
      const int c = c0 + tid + i * kMergeThreads;
      v[i] = c < n ? pval[base * K + c] : ninf;
      id[i] = c < n ? pid[base * K + c] : 0x7fffffff;
    }
    v[kMergeCap] = tid < K ? run_v[tid] : ninf;
    id[kMergeCap] = tid < K ? run_i[tid] : 0x7fffffff;
    __syncthreads();
    uint32_t taken = 0;
    for (int k = 0; k < K; ++k) {
      float bv = ninf;
      int bi = 0x7fffffff;
      int bj = -1;
#pragma unroll
      for (int i = 0; i <= kMergeCap; ++i) {
        if (!((taken >> i) & 1u) && better(v[i], id[i], bv, bi)) {
          bv = v[i];
          bi = id[i];
          bj = i;
        }
      }
      const int mine = bi;
      block_best(bv, bi, sv, si);
      if (bj >= 0 && mine == bi && bv > ninf) taken |= 1u << bj;
      if (tid == 0) {
        run_v[k] = bv;
        run_i[k] = bi;
      }
    }
    __syncthreads();
  }
  if (tid < K) {
    out_val[(size_t)row * K + tid] = run_v[tid] - lse;
    if (out_id) out_id[(size_t)row * K + tid] = run_i[tid];
  }
  if (tid == 0 && out_lse) out_lse[row] = lse;
}

hipError_t lse_topk_merge(const float* pmax, const float* psum, const float* pval, const int32_t* pid, int M,
                          int ntiles, int K, float* out_val, int32_t* out_id, float* out_lse, hipStream_t st) {
  hipLaunchKernelGGL(k_lse_topk, dim3(M), dim3(kMergeThreads), 0, st, pmax, psum, pval, pid, M, ntiles, K, out_val,
                     out_id, out_lse);
  return hipGetLastError();
}

__global__ void k_subtract_rows(float* x, int ld, const float* lse, int M, int ncols) {
  const int row = blockIdx.y;
  const float l = lse[row];
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < ncols; c += gridDim.x * blockDim.x)
    x[(size_t)row * ld + c] -= l;
}

hipError_t subtract_rows(float* x, int ld, const float* lse, int M, int ncols, hipStream_t st) {
  dim3 grid((ncols + 255) / 256 < 64 ? (ncols + 255) / 256 : 64, M), block(256);
  hipLaunchKernelGGL(k_subtract_rows, grid, block, 0, st, x, ld, lse, M, ncols);
  return hipGetLastError();
}

// ------------------------------------------------------------------ beam search
__global__ void k_beam_init(BeamParams p, int bos) {
  const int N = p.B * p.K;
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < N; r += gridDim.x * blockDim.x) {
    p.score[r] = (r % p.K == 0) ? 0.0 : -__builtin_inf();
    p.parent[r] = r;
    p.tok[r] = bos;
    if (r < p.B) {
      p.done[r] = 0;
      p.steps[r] = 0;
      p.best_norm[r] = -__builtin_inf();
      p.best_raw[r] = -__builtin_inf();
      p.best_t[r] = 0;
      p.best_slot[r] = 0;
      p.best_tok[r] = p.pad;
      p.best_logp[r] = 0.f;
    }
    if (r == 0) *p.done_count = 0;
  }
  if (p.tr_slot) {
    const size_t n = (size_t)p.T_max * N;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
      p.tr_slot[i] = -1;
      p.tr_tok[i] = -1;
      p.tr_cand[i] = -__builtin_inf();
    }
  }
}

hipError_t beam_init(const BeamParams& p, int bos, hipStream_t st) {
  const int N = p.B * p.K;
  hipLaunchKernelGGL(k_beam_init, dim3((N + 255) / 256), dim3(256), 0, st, p, bos);
  return hipGetLastError();
}

// One wave per sentence. Candidates are the K per-row top-K entries of every live slot; the sentence's
// top-K over them (larger score first, smaller flat index slot*V + token on ties) is taken with K rounds
// of a wave-wide argmax, then walked in rank order by lane 0: EOS (or any choice at the last step) goes
// to the finished pool, which only keeps its best entry by normalised score, the rest fill live slots.
__global__ __launch_bounds__(64) void k_beam_step(BeamParams p, int t) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  if (p.done[b]) return;
  const int K = p.K;
  const int r0 = b * K;
  constexpr int PER = (kMaxBeam * kMaxBeam) / kWave;   // candidates per lane
  double cv[PER];
  long long cf[PER];
  float cl[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int c = lane + i * kWave;
    cv[i] = -__builtin_inf();
    cf[i] = 0x7fffffffffffffffLL;
    cl[i] = 0.f;
    if (c < K * K) {
      const int k = c / K, j = c % K;
      const double s = p.score[r0 + k];
      if (s > -__builtin_inf()) {
        const float lp = p.tk_val[(size_t)(r0 + k) * K + j];
        cv[i] = s + (double)lp;
        cf[i] = (long long)k * p.V + p.tk_id[(size_t)(r0 + k) * K + j];
        cl[i] = lp;
      }
    }
  }
  __shared__ double sel_v[kMaxBeam];
  __shared__ long long sel_f[kMaxBeam];
  __shared__ float sel_l[kMaxBeam];
  for (int k = 0; k < K; ++k) {
    double bv = cv[0];
    long long bf = cf[0];
#pragma unroll
    for (int i = 1; i < PER; ++i)
      if (better_d(cv[i], cf[i], bv, bf)) {
        bv = cv[i];
        bf = cf[i];
      }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const double ov = __shfl_xor(bv, o, kWave);
      const long long of = __shfl_xor(bf, o, kWave);
      if (better_d(ov, of, bv, bf)) {
        bv = ov;
        bf = of;
      }
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (bv > -__builtin_inf() && cf[i] == bf && cv[i] == bv) {   // flat indices are unique: one owner
        sel_l[k] = cl[i];
        cv[i] = -__builtin_inf();
        cf[i] = 0x7fffffffffffffffLL;
      }
    }
    if (lane == 0) {
      sel_v[k] = bv;
      sel_f[k] = bf;
    }
  }
  __syncthreads();
  if (lane != 0) return;

  const double lp_t = pow((5.0 + t) / 6.0, p.alpha);
  const size_t N = (size_t)p.B * K;
  int live = 0;
  double live_max = -__builtin_inf();
  for (int k = 0; k < K; ++k) {
    const double v = sel_v[k];
    if (!(v > -__builtin_inf())) break;                    // fewer finite candidates than K
    const int slot = (int)(sel_f[k] / p.V);
    const int w = (int)(sel_f[k] % p.V);
    if (p.tr_slot) {
      const size_t o = ((size_t)(t - 1) * p.B + b) * K + k;
      p.tr_slot[o] = slot;
      p.tr_tok[o] = w;
      p.tr_cand[o] = v;
    }
    if (w == p.eos || t == p.T_max) {
      const double norm = v / lp_t;
      if (norm > p.best_norm[b]) {
        p.best_norm[b] = norm;
        p.best_raw[b] = v;
        p.best_t[b] = t;
        p.best_slot[b] = slot;
        p.best_tok[b] = w;
        p.best_logp[b] = sel_l[k];
      }
    } else {
      const int j = live++;
      p.score[r0 + j] = v;
      p.parent[r0 + j] = r0 + slot;
      p.tok[r0 + j] = w;
      p.bp_slot[(size_t)(t - 1) * N + r0 + j] = slot;
      p.bp_tok[(size_t)(t - 1) * N + r0 + j] = w;
      p.bp_logp[(size_t)(t - 1) * N + r0 + j] = sel_l[k];
      if (v > live_max) live_max = v;
    }
  }
  for (int j = live; j < K; ++j) {
    p.score[r0 + j] = -__builtin_inf();
    p.parent[r0 + j] = r0;
    p.tok[r0 + j] = p.pad;
  }
  if (p.tr_slot) {
    for (int k = 0; k < K; ++k) {
      if (!(sel_v[k] > -__builtin_inf())) {
        const size_t o = ((size_t)(t - 1) * p.B + b) * K + k;
        p.tr_slot[o] = -1;
        p.tr_tok[o] = -1;
        p.tr_cand[o] = -__builtin_inf();
      }
    }
  }
  const bool stop = (t == p.T_max) || (live == 0) || (p.best_t[b] > 0 && p.best_norm[b] >= live_max / p.lp_tmax);
  if (stop) {
    p.done[b] = 1;
    p.steps[b] = t;
    atomicAdd(p.done_count, 1);
  }
}

hipError_t beam_step(const BeamParams& p, int t, hipStream_t st) {
  hipLaunchKernelGGL(k_beam_step, dim3(p.B), dim3(64), 0, st, p, t);
  return hipGetLastError();
}

// One thread per sentence: follow back-pointers from the best finished hypothesis.
__global__ void k_backtrack(BeamParams p, int32_t* out_tok, int32_t* out_len, double* out_raw, double* out_norm,
                            float* out_tok_logp) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= p.B) return;
  const int K = p.K;
  const size_t N = (size_t)p.B * K;
  const int tb = p.best_t[b];
  int32_t* tok = out_tok + (size_t)b * p.T_max;
  float* lp = out_tok_logp ? out_tok_logp + (size_t)b * p.T_max : nullptr;
  for (int i = tb; i < p.T_max; ++i) {
    tok[i] = p.pad;
    if (lp) lp[i] = 0.f;
  }
  out_len[b] = tb;
  out_raw[b] = p.best_raw[b];
  out_norm[b] = p.best_norm[b];
  if (tb == 0) return;
  tok[tb - 1] = p.best_tok[b];
  if (lp) lp[tb - 1] = p.best_logp[b];
  int slot = p.best_slot[b];
  for (int tt = tb - 1; tt >= 1; --tt) {
    const size_t o = (size_t)(tt - 1) * N + (size_t)b * K + slot;
    tok[tt - 1] = p.bp_tok[o];
    if (lp) lp[tt - 1] = p.bp_logp[o];
    slot = p.bp_slot[o];
  }
}

hipError_t backtrack(const BeamParams& p, int32_t* out_tok, int32_t* out_len, double* out_raw, double* out_norm,
                     float* out_tok_logp, hipStream_t st) {
  hipLaunchKernelGGL(k_backtrack, dim3((p.B + 63) / 64), dim3(64), 0, st, p, out_tok, out_len, out_raw, out_norm,
                     out_tok_logp);
  return hipGetLastError();
}

// ------------------------------------------------------------------ layout helpers
__global__ void k_replicate_rows(const float* src, int ld_src, int rows, int K, float* dst, int ld_dst, int ncols) {
  const int r = blockIdx.y;                 // destination row
  const float* s = src + (size_t)(r / K) * ld_src;
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < ncols; c += gridDim.x * blockDim.x)
    dst[(size_t)r * ld_dst + c] = s[c];
}

hipError_t replicate_rows(const float* src, int ld_src, int rows, int K, float* dst, int ld_dst, int ncols,
                          hipStream_t st) {
  if (rows * K == 0) return hipSuccess;
  hipLaunchKernelGGL(k_replicate_rows, dim3((ncols + 255) / 256, rows * K), dim3(256), 0, st, src, ld_src, rows, K,
                     dst, ld_dst, ncols);
  return hipGetLastError();
}

__global__ void k_fill(float* dst, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = v;
}

hipError_t fill_f32(float* dst, size_t n, float v, hipStream_t st) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)blocks), dim3(256), 0, st, dst, n, v);
  return hipGetLastError();
}

__global__ void k_copy_cols(const float* src, int ld_src, float* dst, int ld_dst, int ncols) {
  const int r = blockIdx.y;
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < ncols; c += gridDim.x * blockDim.x)
    dst[(size_t)r * ld_dst + c] = src[(size_t)r * ld_src + c];
}

hipError_t copy_cols(const float* src, int ld_src, float* dst, int ld_dst, int rows, int ncols, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_cols, dim3((ncols + 255) / 256, rows), dim3(256), 0, st, src, ld_src, dst, ld_dst, ncols);
  return hipGetLastError();
}

}  // namespace onmt
