// Softmax merge, beam step and backtrack kernels (Section 2: softmax layer and item (d) beam search;
// Section 4.2: length normalisation), plus small layout helpers.

#include <cmath>

#include "common.h"
#include "kernels.h"

namespace onmt {

// ------------------------------------------------------------------ softmax merge
// One wave merges one row's generator partials (per column tile: max, sum of exp, top-K list) into the
// row's logsumexp and top-K (larger logit first, smaller id on ties).
//
// theta = the K-th largest of the 64 per-lane tile maxima is a lower bound on the row's K-th largest
// logit (those K values are maxima of K distinct tiles), so only tiles whose maximum reaches theta can
// contribute. Their lists are loaded in one batch (one qualifying tile per lane), the entries >= theta
// are appended to LDS, and each survivor's position in the result is the number of survivors that come
// before it, which every lane counts for its own entry independently. Rows with more qualifying tiles
// or survivors than fit (ties at theta) are merged by the same rank rule over all entries instead.
constexpr int kMaxTilesPerLane = 16;          // tiles per row <= 64 * 16 (vocabulary <= 131072)
constexpr int kSurvivorCap = 256;
constexpr int kQualCap = 256;                 // qualifying tiles listed per row

// Row partials start at pmax/psum + row * ntiles (loaded by row_tiles_load) and pval/pid + row * ntiles * K. Lane 0 writes
// out_val[k] = logit - lse (K entries), out_id[k] and *out_lse. sv/si/cnt/qt: this wave's LDS scratch
// (kSurvivorCap survivors, kQualCap qualifying tile ids).
// pfmax (optional, filters active): per-tile largest allowed logit, which then replaces the tile maximum
// in the bound (the lists hold allowed entries only; the logsumexp still covers every column).
// The row's tile maxima and sums (lane l holds tiles l + 64 j), every load issued before the first use.
__device__ __forceinline__ void row_tiles_load(const float* __restrict__ pmax, const float* __restrict__ psum,
                                               int ntiles, float (&tm)[kMaxTilesPerLane],
                                               float (&tq)[kMaxTilesPerLane]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) {
    const int t = lane + j * kWave;
    tm[j] = t < ntiles ? pmax[t] : -__builtin_inff();
    tq[j] = t < ntiles ? psum[t] : 0.f;
  }
}

// tm / tq: the row's tile maxima and sums from row_tiles_load (tm is overwritten).
__device__ __forceinline__ void row_merge_wave(float (&tm)[kMaxTilesPerLane], const float (&tq)[kMaxTilesPerLane],
                                               const float* __restrict__ pval, const int32_t* __restrict__ pid,
                                               const float* __restrict__ pfmax, int ntiles, int K, float* sv,
                                               int* si, int* cnt, int* qt, float* out_val, int32_t* out_id,
                                               float* out_lse) {
  const int lane = threadIdx.x & 63;
  const float ninf = -__builtin_inff();
  float mx = ninf;
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) mx = fmaxf(mx, tm[j]);
  const float gmx = wave_max(mx);
  float sm = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) {
    const int t = lane + j * kWave;
    if (t < ntiles) sm += tq[j] * __expf(tm[j] - gmx);
  }
  const float lse = gmx + __logf(wave_sum(sm));
  if (pfmax) {
    mx = ninf;
#pragma unroll
    for (int j = 0; j < kMaxTilesPerLane; ++j) {
      const int t = lane + j * kWave;
      tm[j] = t < ntiles ? pfmax[t] : ninf;
      mx = fmaxf(mx, tm[j]);
    }
  }

  // theta: K rounds of a wave maximum, each removing the (lowest) lane that holds it
  float cur = mx, theta = ninf;
  for (int k = 0; k < K; ++k) {
    const float m = wave_max(cur);
    theta = m;
    const unsigned long long owner = __ballot(cur == m);
    if (lane == __builtin_ctzll(owner)) cur = ninf;
  }

  // qualifying tiles (maximum >= theta), listed in LDS in (j, lane) order
  const unsigned long long below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  int nq = 0;
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) {
    const int t = lane + j * kWave;
    const bool q = t < ntiles && tm[j] >= theta;
    const unsigned long long m = __ballot(q);
    if (q) {
      const int pos = nq + __popcll(m & below);
      if (pos < kQualCap) qt[pos] = t;
    }
    nq += __popcll(m);
  }
  if (lane == 0) *cnt = 0;
  __builtin_amdgcn_wave_barrier();

  // survivors: the lists of the qualifying tiles, one tile per lane, loaded in one batch
  if (nq <= kQualCap) {
    for (int q0 = 0; q0 < nq; q0 += kWave) {
      const int qi = q0 + lane;
      if (qi < nq) {
        const size_t o = (size_t)qt[qi] * K;
        float v[kMaxBeam];
        int id[kMaxBeam];
#pragma unroll
        for (int i = 0; i < kMaxBeam; ++i) {
          v[i] = i < K ? pval[o + i] : ninf;
          id[i] = i < K ? pid[o + i] : 0;
        }
#pragma unroll
        for (int i = 0; i < kMaxBeam; ++i) {
          if (i < K && v[i] >= theta) {
            const int pos = atomicAdd(cnt, 1);
            if (pos < kSurvivorCap) {
              sv[pos] = v[i];
              si[pos] = id[i];
            }
          }
        }
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
  const int n = *cnt;
  if (nq <= kQualCap && n <= kWave) {
    // one survivor per lane, ranked against the others through the scalar unit
    const float v = lane < n ? sv[lane] : ninf;
    const int id = lane < n ? si[lane] : 0x7fffffff;
    int r = 0;
    for (int d = 0; d < n; ++d) r += before(readlane_f(v, d), readlane_i(id, d), v, id) ? 1 : 0;
    if (lane < n && r < K) {
      out_val[r] = v - lse;
      if (out_id) out_id[r] = id;
    }
  } else if (nq <= kQualCap && n <= kSurvivorCap) {
    for (int c = lane; c < n; c += kWave) {
      const float v = sv[c];
      const int id = si[c];
      int r = 0;
      for (int d = 0; d < n; ++d) r += before(sv[d], si[d], v, id) ? 1 : 0;
      if (r < K) {
        out_val[r] = v - lse;
        if (out_id) out_id[r] = id;
      }
    }
  } else {
    // many ties at theta: rank every list entry against every other (slow, but only for degenerate rows)
    for (int c = lane; c < ntiles * K; c += kWave) {
      const float v = pval[c];
      const int id = pid[c];
      if (v < theta) continue;
      int r = 0;
      for (int d = 0; d < ntiles * K && r < K; ++d) r += before(pval[d], pid[d], v, id) ? 1 : 0;
      if (r < K) {
        out_val[r] = v - lse;
        if (out_id) out_id[r] = id;
      }
    }
  }
  if (lane == 0 && out_lse) *out_lse = lse;
}

constexpr int kMergeWaves = 4;

__global__ __launch_bounds__(kMergeWaves * kWave) void k_lse_topk(const float* __restrict__ pmax,
                                                                  const float* __restrict__ psum,
                                                                  const float* __restrict__ pval,
                                                                  const int32_t* __restrict__ pid, int M, int ntiles,
                                                                  int K, float* __restrict__ out_val,
                                                                  int32_t* __restrict__ out_id,
                                                                  float* __restrict__ out_lse) {
  __shared__ float sv[kMergeWaves][kSurvivorCap];
  __shared__ int si[kMergeWaves][kSurvivorCap];
  __shared__ int qt[kMergeWaves][kQualCap];
  __shared__ int cnt[kMergeWaves];
  const int w = threadIdx.x >> 6;
  const int row = blockIdx.x * kMergeWaves + w;
  if (row >= M) return;
  const size_t base = (size_t)row * ntiles;
  float tm[kMaxTilesPerLane], tq[kMaxTilesPerLane];
  row_tiles_load(pmax + base, psum + base, ntiles, tm, tq);
  row_merge_wave(tm, tq, pval + base * K, pid + base * K, nullptr, ntiles, K, sv[w], si[w], &cnt[w], qt[w],
                 out_val + (size_t)row * K, out_id ? out_id + (size_t)row * K : nullptr,
                 out_lse ? out_lse + row : nullptr);
}

hipError_t lse_topk_merge(const float* pmax, const float* psum, const float* pval, const int32_t* pid, int M,
                          int ntiles, int K, float* out_val, int32_t* out_id, float* out_lse, hipStream_t st) {
  if (ntiles > kWave * kMaxTilesPerLane || K > kMaxBeam) return hipErrorInvalidValue;
  const dim3 grid((M + kMergeWaves - 1) / kMergeWaves), block(kMergeWaves * kWave);
  hipLaunchKernelGGL(k_lse_topk, grid, block, 0, st, pmax, psum, pval, pid, M, ntiles, K, out_val, out_id, out_lse);
  return hipGetLastError();
}

// Teacher-forced scores of all steps at once. Row r = t * B + b (step t of sentence b); one wave per row
// forms the logsumexp from the per-tile maxima and sums, as in row_merge_wave, and writes
// logp[b, t] = logit of the target - logsumexp (0 past the sentence's length).
__global__ __launch_bounds__(kMergeWaves * kWave) void k_score_rows(const float* __restrict__ pmax,
                                                                    const float* __restrict__ psum, int ntiles,
                                                                    const float* __restrict__ want_logit,
                                                                    const int32_t* __restrict__ len, int B, int M,
                                                                    float* __restrict__ logp, int ld) {
  const int row = blockIdx.x * kMergeWaves + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const int t = row / B, b = row % B;
  if (t >= len[b]) {
    if (lane == 0) logp[(size_t)b * ld + t] = 0.f;
    return;
  }
  const float* pm = pmax + (size_t)row * ntiles;
  const float* ps = psum + (size_t)row * ntiles;
  const float ninf = -__builtin_inff();
  float tm[kMaxTilesPerLane], tq[kMaxTilesPerLane];
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) {
    const int tt = lane + j * kWave;
    tm[j] = tt < ntiles ? pm[tt] : ninf;
    tq[j] = tt < ntiles ? ps[tt] : 0.f;
  }
  float mx = ninf;
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) mx = fmaxf(mx, tm[j]);
  const float gmx = wave_max(mx);
  float sm = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxTilesPerLane; ++j) {
    const int tt = lane + j * kWave;
    if (tt < ntiles) sm += tq[j] * __expf(tm[j] - gmx);
  }
  const float lse = gmx + __logf(wave_sum(sm));
  if (lane == 0) logp[(size_t)b * ld + t] = want_logit[row] - lse;
}

// nll[b] = -sum over t < len[b] of logp[b, t], summed in fp64 in step order.
__global__ void k_score_nll(const float* __restrict__ logp, int ld, const int32_t* __restrict__ len, int B,
                            double* __restrict__ nll) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  double s = 0.0;
  for (int t = 0; t < len[b]; ++t) s -= (double)logp[(size_t)b * ld + t];
  nll[b] = s;
}

hipError_t score_rows(const float* pmax, const float* psum, int ntiles, const float* want_logit, const int32_t* len,
                      int B, int steps, float* logp, int ld, double* nll, hipStream_t st) {
  if (ntiles > kWave * kMaxTilesPerLane) return hipErrorInvalidValue;
  const int M = B * steps;
  hipLaunchKernelGGL(k_score_rows, dim3((M + kMergeWaves - 1) / kMergeWaves), dim3(kMergeWaves * kWave), 0, st, pmax,
                     psum, ntiles, want_logit, len, B, M, logp, ld);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_score_nll, dim3((B + 255) / 256), dim3(256), 0, st, logp, ld, len, B, nll);
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
    if (p.unk_cnt) p.unk_cnt[r] = 0;
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

// One workgroup per sentence, one wave per beam slot. Each live slot's wave first merges its row's
// generator partials (logsumexp and per-row top-K, as in k_lse_topk). The sentence's top K of the K x K
// candidates cand = score_k + logp (fp64; larger first, smaller flat index k*V + w on ties) is then a
// K-way merge: every row list is in that order already (adding the slot's score keeps it, and equal sums
// come only from equal log-probs, listed by ascending id), so each round takes the largest list head,
// the smaller slot winning ties. Lane r of wave 0 ends up holding the rank-r choice, and the lanes write
// the outcome together: EOS (or any choice at the last step) goes to the finished pool, which keeps only
// its best entry by normalised score (earlier rank on ties), the others fill the live slots in rank order.
__global__ __launch_bounds__(kMaxBeam * kWave) void k_beam_step(BeamParams p, GenPartials gp, int t, double lp_t) {
  __shared__ float sv[kMaxBeam][kSurvivorCap];
  __shared__ int si[kMaxBeam][kSurvivorCap];
  __shared__ int qt[kMaxBeam][kQualCap];
  __shared__ int cnt[kMaxBeam];
  __shared__ float tkv[kMaxBeam][kMaxBeam];
  __shared__ int tki[kMaxBeam][kMaxBeam];
  const int b = blockIdx.x;
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int K = p.K;
  const int r0 = b * K;
  const double ninf = -__builtin_inf();
  // the finished flag, the slot's score and its row's tile partials are loaded together (one memory round
  // trip instead of three dependent ones; a finished sentence's loads are simply not used)
  const int done = p.done[b];
  const double my_score = p.score[r0 + w];
  const size_t base = (size_t)(r0 + w) * gp.ntiles;
  float tm[kMaxTilesPerLane], tq[kMaxTilesPerLane];
  row_tiles_load(gp.pmax + base, gp.psum + base, gp.ntiles, tm, tq);
  if (done) return;
  // sentence state, fetched up front so that the tail below does not wait on memory
  double best_norm0 = ninf;
  int best_t0 = 0;
  if (w == 0) {
    best_norm0 = p.best_norm[b];
    best_t0 = p.best_t[b];
  }
  if (my_score > ninf) {
    row_merge_wave(tm, tq, gp.pval + base * K, gp.pid + base * K,
                   gp.pfmax ? gp.pfmax + base : nullptr, gp.ntiles, K, sv[w], si[w], &cnt[w], qt[w], tkv[w], tki[w],
                   nullptr);
  }
  __syncthreads();
  if (w != 0) return;

  // K-way merge: lane k < K holds slot k's score and the head of its list
  const double sc = lane < K ? p.score[r0 + lane] : ninf;
  int h = 0;
  double my_v = ninf;
  int my_slot = 0, my_tok = 0;
  float my_l = 0.f;
  int nsel = 0;
  for (int r = 0; r < K; ++r) {
    const bool has = lane < K && sc > ninf && h < K;
    const float hv = has ? tkv[lane][h] : 0.f;
    const int hi = has ? tki[lane][h] : 0;
    const double cand = has ? sc + (double)hv : ninf;
    double best = ninf;
    int bk = -1;
    for (int k = 0; k < K; ++k) {
      const double v = readlane_d(cand, k);
      if (v > best) {            // strict: the smaller slot wins ties
        best = v;
        bk = k;
      }
    }
    if (bk < 0) break;           // fewer finite candidates than K
    const int wt = readlane_i(hi, bk);
    const float wl = readlane_f(hv, bk);
    if (lane == r) {
      my_v = best;
      my_slot = bk;
      my_tok = wt;
      my_l = wl;
    }
    if (lane == bk) ++h;
    nsel = r + 1;
  }

  const bool has = lane < nsel;
  const bool fin = has && (my_tok == p.eos || t == p.T_max);
  const bool liv = has && !fin;
  if (has && p.tr_slot) {
    const size_t o = ((size_t)(t - 1) * p.B + b) * K + lane;
    p.tr_slot[o] = my_slot;
    p.tr_tok[o] = my_tok;
    p.tr_cand[o] = my_v;
  }
  // live slots in rank order
  const unsigned long long below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  const unsigned long long lm = __ballot(liv);
  const int live = __popcll(lm);
  const size_t N = (size_t)p.B * K;
  // per-candidate facts of its slot (read by every lane before any slot is rewritten)
  const int my_align = (has && p.align) ? p.align[r0 + my_slot] : -1;
  const int my_unk = (has && p.unk_cnt) ? p.unk_cnt[r0 + my_slot] + (my_tok == p.unk_id ? 1 : 0) : 0;
  __threadfence_block();       // those loads complete before any slot below is rewritten
  if (liv) {
    const int j = __popcll(lm & below);
    p.score[r0 + j] = my_v;
    p.parent[r0 + j] = r0 + my_slot;
    p.tok[r0 + j] = my_tok;
    p.bp_slot[(size_t)(t - 1) * N + r0 + j] = my_slot;
    p.bp_tok[(size_t)(t - 1) * N + r0 + j] = my_tok;
    p.bp_logp[(size_t)(t - 1) * N + r0 + j] = my_l;
    if (p.align) p.bp_align[(size_t)(t - 1) * N + r0 + j] = my_align;
    if (p.unk_cnt) p.unk_cnt[r0 + j] = my_unk;
  }
  if (lane >= live && lane < K) {
    p.score[r0 + lane] = ninf;
    p.parent[r0 + lane] = r0;
    p.tok[r0 + lane] = p.pad;
    if (p.unk_cnt) p.unk_cnt[r0 + lane] = 0;
  }
  // finished pool: the best new entry by normalised score (earliest rank on ties) replaces the pool's
  // entry if strictly better
  const double norm = fin ? my_v / lp_t + (p.cp ? p.cp[r0 + my_slot] : 0.0) : ninf;
  double bn = ninf, live_max = ninf;
  int bl = -1;
  for (int k = 0; k < nsel; ++k) {
    const double nv = readlane_d(norm, k);
    if (nv > bn) {
      bn = nv;
      bl = k;
    }
    if ((lm >> k) & 1ull) live_max = fmax(live_max, readlane_d(my_v, k));
  }
  double best_norm = best_norm0;
  int best_t = best_t0;
  if (bl >= 0 && bn > best_norm0) {
    best_norm = bn;
    best_t = t;
    if (lane == bl) {
      p.best_norm[b] = bn;
      p.best_raw[b] = my_v;
      p.best_t[b] = t;
      p.best_slot[b] = my_slot;
      p.best_tok[b] = my_tok;
      p.best_logp[b] = my_l;
      if (p.align) p.best_align[b] = my_align;
    }
  }
  const bool stop = (t == p.T_max) || (live == 0) || (best_t > 0 && best_norm >= live_max / p.lp_tmax);
  if (stop && lane == 0) {
    p.done[b] = 1;
    p.steps[b] = t;
    atomicAdd(p.done_count, 1);
  }
}

hipError_t beam_step(const BeamParams& p, const GenPartials& gp, int t, hipStream_t st) {
  if (gp.ntiles > kWave * kMaxTilesPerLane || p.K > kMaxBeam) return hipErrorInvalidValue;
  const double lp_t = std::pow((5.0 + t) / 6.0, p.alpha);     // GNMT length penalty of this step
  hipLaunchKernelGGL(k_beam_step, dim3(p.B), dim3(p.K * kWave), 0, st, p, gp, t, lp_t);
  return hipGetLastError();
}

// One workgroup per sentence: the sentence's back-pointer slots are staged in LDS (coalesced loads,
// kBtChunk steps at a time, from the finish step backwards), then one lane follows them from the best
// finished hypothesis; tokens and log-probs are gathered by all lanes once the slot path is known.
constexpr int kBtThreads = 256;
constexpr int kBtChunk = 256;      // steps staged per round

__global__ __launch_bounds__(kBtThreads) void k_backtrack(BeamParams p, int32_t* out_tok, int32_t* out_len,
                                                          double* out_raw, double* out_norm, float* out_tok_logp,
                                                          int32_t* out_align) {
  __shared__ int8_t slots[kBtChunk * kMaxBeam];   // slot (< 16) of each (step, rank) in the current chunk
  __shared__ int8_t path[kBtChunk];               // rank of the path's entry at each step of the chunk
  __shared__ int s_slot;
  const int b = blockIdx.x;
  const int K = p.K;
  const size_t N = (size_t)p.B * K;
  const int tb = p.best_t[b];
  int32_t* tok = out_tok + (size_t)b * p.T_max;
  float* lp = out_tok_logp ? out_tok_logp + (size_t)b * p.T_max : nullptr;
  int32_t* al = out_align ? out_align + (size_t)b * p.T_max : nullptr;
  for (int i = tb + threadIdx.x; i < p.T_max; i += kBtThreads) {
    tok[i] = p.pad;
    if (lp) lp[i] = 0.f;
    if (al) al[i] = -1;
  }
  if (threadIdx.x == 0) {
    out_len[b] = tb;
    out_raw[b] = p.best_raw[b];
    out_norm[b] = p.best_norm[b];
    s_slot = p.best_slot[b];
  }
  if (tb == 0) return;
  if (threadIdx.x == 0) {
    tok[tb - 1] = p.best_tok[b];
    if (lp) lp[tb - 1] = p.best_logp[b];
    if (al) al[tb - 1] = p.best_align[b];
  }
  // entries at steps tt = tb-1 .. 1 (1-based step tt is stored at row tt - 1), walked downwards in chunks
  for (int hi = tb - 1; hi >= 1; hi -= kBtChunk) {
    const int lo = hi - kBtChunk + 1 > 1 ? hi - kBtChunk + 1 : 1;
    const int n = hi - lo + 1;
    __syncthreads();
    for (int e = threadIdx.x; e < n * K; e += kBtThreads) {
      const int i = e / K, k = e % K;
      slots[i * kMaxBeam + k] = (int8_t)p.bp_slot[(size_t)(lo + i - 1) * N + (size_t)b * K + k];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int slot = s_slot;
      for (int tt = hi; tt >= lo; --tt) {
        path[tt - lo] = (int8_t)slot;
        slot = slots[(tt - lo) * kMaxBeam + slot];
      }
      s_slot = slot;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += kBtThreads) {
      const int tt = lo + i;
      const size_t o = (size_t)(tt - 1) * N + (size_t)b * K + path[i];
      tok[tt - 1] = p.bp_tok[o];
      if (lp) lp[tt - 1] = p.bp_logp[o];
      if (al) al[tt - 1] = p.bp_align[o];
    }
  }
}

hipError_t backtrack(const BeamParams& p, int32_t* out_tok, int32_t* out_len, double* out_raw, double* out_norm,
                     float* out_tok_logp, int32_t* out_align, hipStream_t st) {
  if (p.K > kMaxBeam || (out_align && !p.align)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_backtrack, dim3(p.B), dim3(kBtThreads), 0, st, p, out_tok, out_len, out_raw, out_norm,
                     out_tok_logp, out_align);
  return hipGetLastError();
}

// ------------------------------------------------------------------ unknown-word replacement
// out[b, t] = src[b, align[b, t]] where the output token tok[b, t] (t < len[b]) is the UNK id and its
// alignment is a position of the source row, else -1.
__global__ void k_replace_unk(const int32_t* __restrict__ src, int B, int S, const int32_t* __restrict__ tok,
                              const int32_t* __restrict__ len, const int32_t* __restrict__ align, int T, int unk,
                              int32_t* __restrict__ out) {
  const size_t n = (size_t)B * T;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int b = (int)(i / T), t = (int)(i % T);
    int v = -1;
    if (t < len[b] && tok[i] == unk) {
      const int a = align[i];
      if (a >= 0 && a < S) v = src[(size_t)b * S + a];
    }
    out[i] = v;
  }
}

hipError_t replace_unk(const int32_t* src, int B, int S, const int32_t* tok, const int32_t* len, const int32_t* align,
                       int T, int unk, int32_t* out, hipStream_t st) {
  const size_t n = (size_t)B * T;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_replace_unk, dim3((unsigned)blocks), dim3(256), 0, st, src, B, S, tok, len, align, T, unk, out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ input validation on the device
// The checks the host otherwise makes after copying the inputs over (one stream sync per call), done by a
// kernel instead: invalid values are replaced by safe ones (length clamped to [1, S], ids by 0, a parent
// by the row itself), so every later kernel stays in bounds, and the first kind of violation seen is
// recorded in *err (a word of host-visible memory the host reads once the stream is synchronized). Several
// threads may store different codes; any nonzero code reports the failure.
__global__ void k_sanitize_src(const int32_t* __restrict__ src, const int32_t* __restrict__ len, int B, int S, int V,
                               int32_t* __restrict__ clean, int32_t* __restrict__ lens, int32_t* __restrict__ rowmap,
                               int32_t* err) {
  const size_t n = (size_t)B * S;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int b = (int)(i / S), s = (int)(i % S);
    const int l = len[b];
    const int lc = l < 1 ? 1 : (l > S ? S : l);
    if (s == 0) {
      lens[b] = lc;
      if (l != lc) *err = kErrLength;
    }
    int id = 0;
    if (s < lc) {
      id = src[i];
      if (id < 0 || id >= V) {
        *err = kErrSourceId;
        id = 0;
      }
    }
    clean[i] = id;
    rowmap[(size_t)s * B + b] = (int32_t)i;
  }
}

__global__ void k_sanitize_step(const int32_t* __restrict__ tok, const int32_t* __restrict__ parent, int N, int V,
                                int32_t* __restrict__ tok_out, int32_t* __restrict__ par_out, int32_t* err) {
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < N; r += gridDim.x * blockDim.x) {
    int t = tok[r];
    if (t < 0 || t >= V) {
      *err = kErrToken;
      t = 0;
    }
    tok_out[r] = t;
    if (par_out) {
      int p = parent[r];
      if (p < 0 || p >= N) {
        *err = kErrParent;
        p = r;
      }
      par_out[r] = p;
    }
  }
}

hipError_t sanitize_src(const int32_t* src, const int32_t* len, int B, int S, int V, int32_t* clean, int32_t* lens,
                        int32_t* rowmap, int32_t* err, hipStream_t st) {
  const size_t n = (size_t)B * S;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_sanitize_src, dim3((unsigned)blocks), dim3(256), 0, st, src, len, B, S, V, clean, lens, rowmap,
                     err);
  return hipGetLastError();
}

hipError_t sanitize_step(const int32_t* tok, const int32_t* parent, int N, int V, int32_t* tok_out, int32_t* par_out,
                         int32_t* err, hipStream_t st) {
  int blocks = (N + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_sanitize_step, dim3(blocks), dim3(256), 0, st, tok, parent, N, V, tok_out,
                     parent ? par_out : nullptr, err);
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
