// MFMA GEMM for gfx950 with fused epilogues.
//
// Computes acc[r, n] = sum_k A[r, k] * W[n, k] where A is gathered on the fly from up to three
// row-mapped segments (embedding rows by token id, state rows by beam parent, plain activations)
// and W is a packed weight matrix. The tile is staged through LDS (two buffers, one barrier per
// K stage) and multiplied with 16x16 MFMA tiles: v_mfma_f32_16x16x4_f32 for fp32 operands and
// v_mfma_f32_16x16x32_bf16 for bf16 operands, always accumulating in fp32. Waves may split K
// inside the workgroup (WK > 1); their partial tiles are summed in LDS before the epilogue.
//
// Epilogues: plain bias(+tanh) store; LSTM gate nonlinearities and cell update (Section 2 item
// (a) of the OpenNMT paper) over gate-blocked columns; and the generator's per-tile row max,
// sum of exponentials and top-K, so the vocabulary logits never need to reach memory.

#include "common.h"
#include "kernels.h"

namespace onmt {

template <class T, int WM_, int WN_, int WK_, int TM_, int TN_>
struct Tile {
  static constexpr int WM = WM_, WN = WN_, WK = WK_, TM = TM_, TN = TN_;
  static constexpr bool kBf16 = sizeof(T) == 2;
  static constexpr int CH = 16 / sizeof(T);          // elements per 16-byte chunk
  static constexpr int KW = kBf16 ? 32 : 16;         // K per wave per stage
  static constexpr int BM = WM * TM * 16;
  static constexpr int BN = WN * TN * 16;
  static constexpr int BK = WK * KW;
  static constexpr int NT = 64 * WM * WN * WK;
  static constexpr int ROW = BK + CH;                // LDS row stride in elements (16-byte pad)
  static constexpr int CPR = BK / CH;                // chunks per tile row
  static constexpr int A_CH = BM * CPR;
  static constexpr int B_CH = BN * CPR;
  static constexpr int A_PT = (A_CH + NT - 1) / NT;
  static constexpr int B_PT = (B_CH + NT - 1) / NT;
  static constexpr int STAGE = (BM + BN) * ROW * (int)sizeof(T);
  static constexpr int CROW = BN + 4;                // fp32 output tile row stride
  static constexpr int CT = WK * BM * CROW * 4;
  static constexpr int LDS = (2 * STAGE > CT) ? 2 * STAGE : CT;
};

// XCD-aware tile order: blocks are dealt round-robin to the 8 XCDs, so renumber them so that each
// XCD receives a contiguous range of logical tiles; M varies fastest, so the M tiles that share a
// weight tile run on the same XCD and share its L2.
__device__ inline int xcd_remap(int bid, int nblocks) {
  const int xcd = bid & 7, local = bid >> 3;
  const int full = nblocks >> 3, rem = nblocks & 7;
  return xcd * full + (xcd < rem ? xcd : rem) + local;
}

__device__ inline uint4 zero4() { return make_uint4(0u, 0u, 0u, 0u); }

// Load one 16-byte chunk of A (CH elements starting at padded column k) for GEMM row r.
template <class T>
__device__ inline uint4 load_a_chunk(const AOp& a, const char* const (&rowp)[3], int k) {
  int off = 0;
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    if (s < a.nseg) {
      const Seg& g = a.seg[s];
      if (k < off + g.kpad) {
        const int kk = k - off;
        if (rowp[s] == nullptr || kk >= g.width) return zero4();
        if constexpr (sizeof(T) == 4) {
          return *(const uint4*)(rowp[s] + (size_t)kk * 4);
        } else {
          if (g.bf16) return *(const uint4*)(rowp[s] + (size_t)kk * 2);
          // fp32 source feeding a bf16 product: round to nearest even
          const float4 lo = *(const float4*)(rowp[s] + (size_t)kk * 4);
          float4 hi = make_float4(0.f, 0.f, 0.f, 0.f);
          if (kk + 4 < g.width) hi = *(const float4*)(rowp[s] + (size_t)(kk + 4) * 4);
          uint4 r;
          r.x = f32_to_bf16_bits(lo.x) | ((uint32_t)f32_to_bf16_bits(lo.y) << 16);
          r.y = f32_to_bf16_bits(lo.z) | ((uint32_t)f32_to_bf16_bits(lo.w) << 16);
          r.z = f32_to_bf16_bits(hi.x) | ((uint32_t)f32_to_bf16_bits(hi.y) << 16);
          r.w = f32_to_bf16_bits(hi.z) | ((uint32_t)f32_to_bf16_bits(hi.w) << 16);
          return r;
        }
      }
      off += g.kpad;
    }
  }
  return zero4();
}

// Main loop: leaves the (WK-way partial) fp32 output tile in LDS at smem, layout [WK][BM][CROW].
template <class T, class C>
__device__ inline void gemm_tile(const AOp& a, const BOp& b, int m0, int n0, char* smem) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wk = wave % C::WK;
  const int wn = (wave / C::WK) % C::WN;
  const int wm = wave / (C::WK * C::WN);
  const int i16 = lane & 15, g = lane >> 4;

  // Per-thread A row pointers (rows fixed across K stages).
  const char* arow[C::A_PT][3];
  int acol[C::A_PT];
  bool aok[C::A_PT];
#pragma unroll
  for (int i = 0; i < C::A_PT; ++i) {
    const int c = tid + i * C::NT;
    const int row = c / C::CPR;
    acol[i] = (c % C::CPR) * C::CH;
    aok[i] = c < C::A_CH;
    const int r = m0 + row;
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      arow[i][s] = nullptr;
      if (aok[i] && s < a.nseg && r < a.M) {
        const Seg& sg = a.seg[s];
        const int rr = sg.idx ? sg.idx[r] : r;
        arow[i][s] = (const char*)sg.base + (size_t)rr * sg.ld * (sg.bf16 ? 2 : 4);
      }
    }
  }
  const char* brow[C::B_PT];
  int bcol[C::B_PT];
  bool bok[C::B_PT];
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) {
    const int c = tid + i * C::NT;
    const int row = c / C::CPR;
    bcol[i] = (c % C::CPR) * C::CH;
    bok[i] = c < C::B_CH;
    brow[i] = (const char*)b.W + (size_t)(n0 + row) * b.Kp * sizeof(T);
  }

  T* As[2] = {(T*)smem, (T*)(smem + C::STAGE)};
  T* Bs[2] = {As[0] + C::BM * C::ROW, As[1] + C::BM * C::ROW};

  uint4 ra[C::A_PT], rb[C::B_PT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::A_PT; ++i) {
      const int k = k0 + acol[i];
      ra[i] = (aok[i] && k < b.Kp) ? load_a_chunk<T>(a, arow[i], k) : zero4();
    }
#pragma unroll
    for (int i = 0; i < C::B_PT; ++i) {
      const int k = k0 + bcol[i];
      rb[i] = (bok[i] && k < b.Kp) ? *(const uint4*)(brow[i] + (size_t)k * sizeof(T)) : zero4();
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < C::A_PT; ++i) {
      const int c = tid + i * C::NT;
      if (aok[i]) *(uint4*)(As[buf] + (c / C::CPR) * C::ROW + acol[i]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < C::B_PT; ++i) {
      const int c = tid + i * C::NT;
      if (bok[i]) *(uint4*)(Bs[buf] + (c / C::CPR) * C::ROW + bcol[i]) = rb[i];
    }
  };

  f32x4 acc[C::TM][C::TN];
#pragma unroll
  for (int x = 0; x < C::TM; ++x)
#pragma unroll
    for (int y = 0; y < C::TN; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nst = (b.Kp + C::BK - 1) / C::BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    if (st + 1 < nst) gload((st + 1) * C::BK);
    const T* Ab = As[buf] + (wm * C::TM * 16 + i16) * C::ROW + wk * C::KW;
    const T* Bb = Bs[buf] + (wn * C::TN * 16 + i16) * C::ROW + wk * C::KW;
    if constexpr (!C::kBf16) {
      f32x4 av[C::TM], bv[C::TN];
#pragma unroll
      for (int x = 0; x < C::TM; ++x) av[x] = *(const f32x4*)(Ab + x * 16 * C::ROW + 4 * g);
#pragma unroll
      for (int y = 0; y < C::TN; ++y) bv[y] = *(const f32x4*)(Bb + y * 16 * C::ROW + 4 * g);
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int x = 0; x < C::TM; ++x)
#pragma unroll
          for (int y = 0; y < C::TN; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[x][m], bv[y][m], acc[x][y], 0, 0, 0);
    } else {
      bf16x8 av[C::TM], bv[C::TN];
#pragma unroll
      for (int x = 0; x < C::TM; ++x) av[x] = *(const bf16x8*)(Ab + x * 16 * C::ROW + 8 * g);
#pragma unroll
      for (int y = 0; y < C::TN; ++y) bv[y] = *(const bf16x8*)(Bb + y * 16 * C::ROW + 8 * g);
#pragma unroll
      for (int x = 0; x < C::TM; ++x)
#pragma unroll
        for (int y = 0; y < C::TN; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[x], bv[y], acc[x][y], 0, 0, 0);
    }
    if (st + 1 < nst) lstore(buf ^ 1);
    __syncthreads();
  }

  // Partial tiles to LDS: lane holds rows 4g..4g+3 of column i16 of each 16x16 block.
  float* Ct = (float*)smem + wk * C::BM * C::CROW;
#pragma unroll
  for (int x = 0; x < C::TM; ++x)
#pragma unroll
    for (int y = 0; y < C::TN; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Ct[(wm * C::TM * 16 + x * 16 + 4 * g + v) * C::CROW + wn * C::TN * 16 + y * 16 + i16] = acc[x][y][v];
  __syncthreads();
}

template <class C>
__device__ inline float ctile(const float* smem, int r, int c) {
  float s = smem[r * C::CROW + c];
#pragma unroll
  for (int w = 1; w < C::WK; ++w) s += smem[(w * C::BM + r) * C::CROW + c];
  return s;
}

// ---------------------------------------------------------------- kernels

template <class T, class C>
__global__ __launch_bounds__(C::NT) void k_gemm_store(AOp a, BOp b, StoreParams p, int nm, int nblocks) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const int L = xcd_remap(blockIdx.x, nblocks);
  const int m0 = (L % nm) * C::BM, n0 = (L / nm) * C::BN;
  gemm_tile<T, C>(a, b, m0, n0, smem);
  const float* Ct = (const float*)smem;
  for (int e = threadIdx.x; e < C::BM * (C::BN / 4); e += C::NT) {
    const int r = e / (C::BN / 4), c = (e % (C::BN / 4)) * 4;
    const int gr = m0 + r, gc = n0 + c;
    if (gr >= a.M || gc >= p.ncols) continue;
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = ctile<C>(Ct, r, c + j) + (p.bias ? p.bias[gc + j] : 0.f);
      if (p.act == 1) v[j] = tanhf(v[j]);
    }
    *(float4*)(p.out + (size_t)gr * p.ldo + gc) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <class T, class C>
__global__ __launch_bounds__(C::NT) void k_gemm_lstm(AOp a, BOp b, LstmParams p, int nm, int nblocks) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const int L = xcd_remap(blockIdx.x, nblocks);
  const int m0 = (L % nm) * C::BM, n0 = (L / nm) * C::BN;
  gemm_tile<T, C>(a, b, m0, n0, smem);
  const float* Ct = (const float*)smem;
  constexpr int UPT = C::BN / 4;                      // units per tile
  for (int e = threadIdx.x; e < C::BM * UPT; e += C::NT) {
    const int r = e / UPT, uu = e % UPT;
    const int row = m0 + r;
    const int unit = n0 / 4 + uu;
    if (row >= a.M || unit >= p.H) continue;
    const int cbase = (uu / kUnitGroup) * 64 + (uu % kUnitGroup);
    float z[4];
#pragma unroll
    for (int gt = 0; gt < 4; ++gt) {
      const int col = cbase + gt * kUnitGroup;
      z[gt] = ctile<C>(Ct, r, col) + (p.bias ? p.bias[n0 + col] : 0.f);
      if (p.gx) z[gt] += p.gx[(size_t)(row * p.gx_S + p.gx_s) * p.ld_gx + p.gx_col0 + n0 + col];
    }
    const int crow = p.c_idx ? p.c_idx[row] : row;
    const float c_prev = p.c_in ? p.c_in[(size_t)crow * p.ld_c + unit] : 0.f;
    float h_new, c_new, y;
    if (p.lens && p.y_s >= p.lens[row]) {
      c_new = c_prev;
      h_new = p.h_in ? p.h_in[(size_t)row * p.ld_h_in + unit] : 0.f;
      y = 0.f;
    } else {
      const float ig = sigmoidf_(z[0]), fg = sigmoidf_(z[1]), gg = tanhf(z[2]), og = sigmoidf_(z[3]);
      c_new = fg * c_prev + ig * gg;
      h_new = og * tanhf(c_new);
      y = h_new;
    }
    p.h_out[(size_t)row * p.ld_out + unit] = h_new;
    p.c_out[(size_t)row * p.ld_out + unit] = c_new;
    if (p.y_out) p.y_out[(size_t)(row * p.y_S + p.y_s) * p.ld_y + p.y_col0 + unit] = y;
  }
}

// Generator: 4 threads per row, 32 contiguous columns each, merged with lane shuffles.
template <class T, class C, int KMAX>
__global__ __launch_bounds__(C::NT) void k_gemm_gen(AOp a, BOp b, GenParams p, int nm, int nblocks) {
  static_assert(C::NT / C::BM == 4 && C::BN == 128, "generator tile is 64 x 128 with 256 threads");
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const int L = xcd_remap(blockIdx.x, nblocks);
  const int mt = L % nm, nt = L / nm;
  const int m0 = mt * C::BM, n0 = nt * C::BN;
  gemm_tile<T, C>(a, b, m0, n0, smem);
  const float* Ct = (const float*)smem;
  const int r = threadIdx.x >> 2, part = threadIdx.x & 3;
  const int row = m0 + r;
  const int c0 = part * 32;
  float z[32];
  float mx = -__builtin_inff();
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const int gc = n0 + c0 + j;
    z[j] = (gc < p.V) ? ctile<C>(Ct, r, c0 + j) + p.bias[gc] : -__builtin_inff();
    mx = fmaxf(mx, z[j]);
  }
  if (p.logits && row < a.M) {
#pragma unroll
    for (int j = 0; j < 32; j += 4) {
      const int gc = n0 + c0 + j;
      if (gc + 3 < p.V && (p.ld_logits & 3) == 0) {
        *(float4*)(p.logits + (size_t)row * p.ld_logits + gc) = make_float4(z[j], z[j + 1], z[j + 2], z[j + 3]);
      } else {
        for (int q = 0; q < 4; ++q)
          if (gc + q < p.V) p.logits[(size_t)row * p.ld_logits + gc + q] = z[j + q];
      }
    }
  }
  float val[KMAX];
  int ids[KMAX];
  topk_clear<KMAX>(val, ids);
  float sm = 0.f;
  if (mx > -__builtin_inff()) {
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      if (z[j] > -__builtin_inff()) {
        sm += __expf(z[j] - mx);
        topk_insert<KMAX>(val, ids, z[j], n0 + c0 + j);
      }
    }
  }
  // merge the 4 parts of the row (lanes 4q .. 4q+3 of one wave)
#pragma unroll
  for (int o = 1; o < 4; o <<= 1) {
    const float omx = __shfl_xor(mx, o, kWave);
    const float osm = __shfl_xor(sm, o, kWave);
    const float nmx = fmaxf(mx, omx);
    sm = (mx > -__builtin_inff() ? sm * __expf(mx - nmx) : 0.f) + (omx > -__builtin_inff() ? osm * __expf(omx - nmx) : 0.f);
    mx = nmx;
    float ov[KMAX];
    int oi[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      ov[i] = __shfl_xor(val[i], o, kWave);
      oi[i] = __shfl_xor(ids[i], o, kWave);
    }
#pragma unroll
    for (int i = 0; i < KMAX; ++i) topk_insert<KMAX>(val, ids, ov[i], oi[i]);
  }
  if (part == 0 && row < a.M) {
    const size_t o = (size_t)row * p.ntiles + nt;
    p.pmax[o] = mx;
    p.psum[o] = sm;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      if (i < p.K) {
        p.pval[o * p.K + i] = val[i];
        p.pid[o * p.K + i] = ids[i];
      }
    }
  }
}

// ---------------------------------------------------------------- launchers

using TileWide32 = Tile<float, 2, 2, 1, 2, 4>;
using TileSplit32 = Tile<float, 1, 1, 4, 2, 4>;
using TileThin32 = Tile<float, 1, 1, 4, 1, 4>;
using TileWide16 = Tile<__bf16, 2, 2, 1, 2, 4>;
using TileSplit16 = Tile<__bf16, 1, 1, 4, 2, 4>;
using TileThin16 = Tile<__bf16, 1, 1, 4, 1, 4>;

template <class C>
static inline void grid_of(const AOp& a, const BOp& b, int& nm, int& nblocks) {
  nm = (a.M + C::BM - 1) / C::BM;
  nblocks = nm * (b.Np / C::BN);
}

int gemm_tile_cols(int shape) { return shape == kShapeWide ? TileWide32::BN : TileSplit32::BN; }
int gen_tile_cols() { return TileWide32::BN; }

template <class T, class C>
static hipError_t launch_store(const AOp& a, const BOp& b, const StoreParams& p, hipStream_t st) {
  int nm, nb;
  grid_of<C>(a, b, nm, nb);
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_store<T, C>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  return hipGetLastError();
}

template <class T, class C>
static hipError_t launch_lstm(const AOp& a, const BOp& b, const LstmParams& p, hipStream_t st) {
  int nm, nb;
  grid_of<C>(a, b, nm, nb);
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_lstm<T, C>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  return hipGetLastError();
}

template <class T, class C, int KMAX>
static hipError_t launch_gen(const AOp& a, const BOp& b, const GenParams& p, hipStream_t st) {
  int nm, nb;
  grid_of<C>(a, b, nm, nb);
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_gen<T, C, KMAX>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  return hipGetLastError();
}

hipError_t gemm_store(int bf16, int shape, const AOp& a, const BOp& b, const StoreParams& p, hipStream_t st) {
  if (bf16) {
    if (shape == kShapeWide) return launch_store<__bf16, TileWide16>(a, b, p, st);
    if (shape == kShapeSplitK) return launch_store<__bf16, TileSplit16>(a, b, p, st);
    return launch_store<__bf16, TileThin16>(a, b, p, st);
  }
  if (shape == kShapeWide) return launch_store<float, TileWide32>(a, b, p, st);
  if (shape == kShapeSplitK) return launch_store<float, TileSplit32>(a, b, p, st);
  return launch_store<float, TileThin32>(a, b, p, st);
}

hipError_t gemm_lstm(int bf16, int shape, const AOp& a, const BOp& b, const LstmParams& p, hipStream_t st) {
  if (bf16) {
    if (shape == kShapeWide) return launch_lstm<__bf16, TileWide16>(a, b, p, st);
    if (shape == kShapeSplitK) return launch_lstm<__bf16, TileSplit16>(a, b, p, st);
    return launch_lstm<__bf16, TileThin16>(a, b, p, st);
  }
  if (shape == kShapeWide) return launch_lstm<float, TileWide32>(a, b, p, st);
  if (shape == kShapeSplitK) return launch_lstm<float, TileSplit32>(a, b, p, st);
  return launch_lstm<float, TileThin32>(a, b, p, st);
}

hipError_t gemm_gen(int bf16, const AOp& a, const BOp& b, const GenParams& p, hipStream_t st) {
  if (p.K <= 1) return bf16 ? launch_gen<__bf16, TileWide16, 1>(a, b, p, st) : launch_gen<float, TileWide32, 1>(a, b, p, st);
  if (p.K <= 2) return bf16 ? launch_gen<__bf16, TileWide16, 2>(a, b, p, st) : launch_gen<float, TileWide32, 2>(a, b, p, st);
  if (p.K <= 4) return bf16 ? launch_gen<__bf16, TileWide16, 4>(a, b, p, st) : launch_gen<float, TileWide32, 4>(a, b, p, st);
  if (p.K <= 8) return bf16 ? launch_gen<__bf16, TileWide16, 8>(a, b, p, st) : launch_gen<float, TileWide32, 8>(a, b, p, st);
  return bf16 ? launch_gen<__bf16, TileWide16, 16>(a, b, p, st) : launch_gen<float, TileWide32, 16>(a, b, p, st);
}

}  // namespace onmt
