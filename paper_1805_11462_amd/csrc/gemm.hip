// MFMA GEMM for gfx950 with fused epilogues.
//
// Computes acc[r, n] = sum_k A[r, k] * W[n, k] where A is gathered on the fly from up to three
// row-mapped segments (embedding rows by token id, state rows by beam parent, plain activations)
// and W is a packed weight matrix. Tiles are staged through two LDS buffers; global loads run two
// K stages ahead in registers so that a stage's loads have a full stage of MFMA work to hide behind.
// Where the bf16 operands are pre-split term planes (the bf16 generator and decoder layers), buffer
// loads with an LDS destination move them straight into the stage buffers instead.
// Products use 16x16 MFMA tiles: v_mfma_f32_16x16x4_f32 for fp32 operands and
// v_mfma_f32_16x16x32_bf16 for bf16 operands, always accumulating in fp32. Waves may split K
// inside the workgroup (WK > 1); their partial tiles are summed in LDS before the epilogue.
//
// Epilogues: plain bias(+tanh) store; LSTM gate nonlinearities and cell update (Section 2 item
// (a) of the OpenNMT paper) over gate-blocked columns; and the generator's per-tile row max,
// sum of exponentials and top-K, so the vocabulary logits never need to reach memory.

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace onmt {

template <class T, int WM_, int WN_, int WK_, int TM_, int TN_, int KW_>
struct Tile {
  static constexpr int WM = WM_, WN = WN_, WK = WK_, TM = TM_, TN = TN_;
  static constexpr bool kBf16 = sizeof(T) == 2;
  static constexpr int CH = 16 / sizeof(T);          // elements per 16-byte chunk
  static constexpr int KW = KW_;                     // K per wave per stage
  static constexpr int KSUB = kBf16 ? 32 : 16;       // K consumed per MFMA round (one 16-byte read per lane)
  static constexpr int BM = WM * TM * 16;
  static constexpr int BN = WN * TN * 16;
  static constexpr int BK = WK * KW;
  static constexpr int NT = 64 * WM * WN * WK;
  static constexpr int ROW = BK;                     // LDS row stride in elements (rows are swizzled)
  static constexpr int CPR = BK / CH;                // 16-byte chunks per tile row
  // Chunk c of tile row r is stored in slot c ^ swz(r). A 16-byte LDS read is served eight lanes at a
  // time from 128 bytes of banks; the eight lanes of a fragment read take eight consecutive rows at the
  // same logical chunk, so swz spreads those rows over distinct 16-byte bank slots: 64-byte rows (two per
  // bank window) XOR with (r >> 1) & 3, 128-byte rows with r & 7, longer rows with r & 15. (Measured on
  // gfx950: with (r >> 2) & 3 for 64-byte rows half the LDS cycles of such reads were bank conflicts, with
  // (r >> 1) & 3 none, and read throughput rose 1.65x.)
  static constexpr int RSH = CPR == 4 ? 1 : 0;
  static constexpr int SMASK = (CPR >= 16 ? 16 : CPR) - 1;
  static constexpr int A_CH = BM * CPR;
  static constexpr int B_CH = BN * CPR;
  static constexpr int A_PT = A_CH / NT;
  static constexpr int B_PT = B_CH / NT;
  // bf16 products carry each fp32 activation as kPlanes bf16 terms (p0 + p1 + p2, ~24 significant bits,
  // the precision of the fp32 value); the A tile holds one copy per term. Weights are bf16 already, so
  // W a = W p0 + W p1 + W p2 exactly up to the fp32 accumulation.
  static constexpr int AREP = kBf16 ? kPlanes : 1;
  static constexpr int STAGE = (AREP * BM + BN) * ROW * (int)sizeof(T);
  static constexpr int CROW = BN + 4;                // fp32 output tile row stride
  static constexpr int CT = WK * BM * CROW * 4;
  static constexpr int LDS = (2 * STAGE > CT) ? 2 * STAGE : CT;
  static_assert(KW % KSUB == 0 && kSegK % BK == 0, "stage must divide the segment padding");
  static_assert(CPR == 4 || CPR == 8 || CPR >= 16, "swizzle covers 64-, 128- and >=256-byte rows");
  __device__ static int swz(int row) { return (row >> RSH) & SMASK; }
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

// Split 8 fp32 values into three bf16 terms p0 = RNE(x), p1 = RNE(x - p0), p2 = RNE(x - p0 - p1). Each
// remainder is exact in fp32 (it drops leading bits of x), so p0 + p1 + p2 keeps about 24 significant
// bits of x: the fp32 value itself, as the bf16 products see it. (Two terms keep ~16 bits, which over the
// 120 steps of the 4 x 1000 decoder recurrence let a hypothesis's log-prob drift to the bf16 tolerance.)
// The conversions are gfx950's packed fp32 -> bf16 (round to nearest even), two values per instruction.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ inline void split_bf16x8(const float4& a, const float4& b, uint4& p0, uint4& p1, uint4& p2) {
  const f32x2_t x[4] = {{a.x, a.y}, {a.z, a.w}, {b.x, b.y}, {b.z, b.w}};
  uint32_t t0[4], t1[4], t2[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2_t v0 = __builtin_convertvector(x[i], bf16x2_t);
    const f32x2_t r1 = x[i] - __builtin_convertvector(v0, f32x2_t);
    const bf16x2_t v1 = __builtin_convertvector(r1, bf16x2_t);
    const f32x2_t r2 = r1 - __builtin_convertvector(v1, f32x2_t);
    const bf16x2_t v2 = __builtin_convertvector(r2, bf16x2_t);
    t0[i] = __builtin_bit_cast(uint32_t, v0);
    t1[i] = __builtin_bit_cast(uint32_t, v1);
    t2[i] = __builtin_bit_cast(uint32_t, v2);
  }
  p0 = make_uint4(t0[0], t0[1], t0[2], t0[3]);
  p1 = make_uint4(t1[0], t1[1], t1[2], t1[3]);
  p2 = make_uint4(t2[0], t2[1], t2[2], t2[3]);
}

__device__ inline void split_bf16(float x, uint16_t& p0, uint16_t& p1, uint16_t& p2) {
  uint4 a, b, c;
  split_bf16x8(make_float4(x, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f), a, b, c);
  p0 = (uint16_t)(a.x & 0xffffu);
  p1 = (uint16_t)(b.x & 0xffffu);
  p2 = (uint16_t)(c.x & 0xffffu);
}

// Buffer resource descriptor (gfx9 family word 3). Loads through it return zeros past num_records, so
// an invalid row is given an offset beyond every buffer instead of a branch.
constexpr int kBufWord3 = 0x00020000;
constexpr uint32_t kNoRow = 0x80000000u;      // byte offset past the end of any buffer (buffers < 2 GiB)

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufWord3);
}

// LDS address of a byte in a __shared__ array, as the LDS-destination buffer loads take it. (Declared at
// file scope: a local typedef of this pointer type inside a kernel template stops the host stub from
// being emitted.)
typedef __attribute__((address_space(3))) void* lds_ptr_t;
__device__ inline lds_ptr_t lds_at(char* p) { return (lds_ptr_t)p; }

__device__ inline uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

// Main loop: leaves the (WK-way partial) fp32 output tile in LDS at smem, layout [WK][BM][CROW].
// CBIAS (single-K-group tiles): cb[y] is added to the lane's column of output block y as the tile is
// written (the generator's bias, loaded before the main loop by gen_col_bias).
template <class T, class C, int NSEG, bool CBIAS = false>
__device__ inline void gemm_tile(const AOp& a, const BOp& b, int m0, int n0, char* smem, const float* cb = nullptr) {
  static_assert(!CBIAS || C::WK == 1, "a bias is added to whole sums only");
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wk = wave % C::WK;
  const int wn = (wave / C::WK) % C::WN;
  const int wm = wave / (C::WK * C::WN);
  const int i16 = lane & 15, g = lane >> 4;

  // Thread chunk c = tid + i * NT covers tile row c / CPR, columns (c % CPR) * CH ...; NT is a multiple
  // of CPR, so the column is the same for every i and the row advances by NT / CPR.
  constexpr int RSTEP = C::NT / C::CPR;
  static_assert(C::NT % C::CPR == 0, "threads must cover whole tile rows");
  static_assert(C::A_CH % C::NT == 0 && C::B_CH % C::NT == 0 && C::A_PT > 0, "chunks must divide evenly among threads");
  const int arow0 = tid / C::CPR;
  const int acol = (tid % C::CPR) * C::CH;

  // Every segment field is read with a constant index into a scalar, so the argument struct is never
  // indexed at run time (which would put it in private memory).
  constexpr int nseg = NSEG;             // segments in use (a.nseg, checked by the launcher)
  // Per-thread byte offsets of the thread's A rows inside each segment's buffer (kNoRow past M).
#define ONMT_SEG_SETUP(S)                                                                             \
  const int kp##S = a.seg[S].kpad, wd##S = a.seg[S].width, bf##S = a.seg[S].bf16;                     \
  const uint32_t es##S = bf##S ? 2u : 4u;                                                              \
  const __amdgpu_buffer_rsrc_t rs##S = make_rsrc(a.seg[S].base, (uint32_t)a.seg[S].rows * a.seg[S].ld * es##S); \
  const bool pre##S = C::kBf16 && a.seg[S].lo;                                                        \
  const __amdgpu_buffer_rsrc_t rl##S = make_rsrc(pre##S ? a.seg[S].lo : a.seg[S].base,                 \
                                                 (uint32_t)a.seg[S].rows * a.seg[S].ld * es##S);       \
  const __amdgpu_buffer_rsrc_t rm##S = make_rsrc(pre##S ? a.seg[S].lo2 : a.seg[S].base,                \
                                                 (uint32_t)a.seg[S].rows * a.seg[S].ld * es##S);       \
  uint32_t ao##S[C::A_PT];                                                                             \
  _Pragma("unroll") for (int i = 0; i < C::A_PT; ++i) {                                                \
    const int r = m0 + arow0 + i * RSTEP;                                                              \
    const bool ok = S < nseg && r < a.M;                                                               \
    const int rr = ok ? (a.seg[S].idx ? a.seg[S].idx[r] : r) : 0;                                      \
    ao##S[i] = ok ? ((uint32_t)rr * a.seg[S].ld + acol) * es##S : kNoRow;                              \
  }
  ONMT_SEG_SETUP(0)
  ONMT_SEG_SETUP(1)
  ONMT_SEG_SETUP(2)
#undef ONMT_SEG_SETUP

  const __amdgpu_buffer_rsrc_t rw = make_rsrc(b.W, (uint32_t)b.Np * b.Kp * sizeof(T));
  uint32_t bo[C::B_PT];
#pragma unroll
  for (int i = 0; i < C::B_PT; ++i) bo[i] = ((uint32_t)(n0 + arow0 + i * RSTEP) * b.Kp + acol) * sizeof(T);

  // LDS stage layout: [A (hi) rows | A lo rows (bf16 only) | B rows].
  T* As[2] = {(T*)smem, (T*)(smem + C::STAGE)};
  T* Bs[2] = {As[0] + C::AREP * C::BM * C::ROW, As[1] + C::AREP * C::BM * C::ROW};

  // One K stage of operands in flight: the raw global loads, held in registers until the stage is stored
  // to LDS. Everything that reads the loaded values (the zeroing of a segment's K padding, the split of an
  // fp32 source into its bf16 term planes) happens at that store, one stage after the loads were issued: done at
  // the load, it made every wave wait for its loads right after issuing them.
  struct Regs {
    uint4 a[C::A_PT];
    uint4 alo[C::AREP > 1 ? C::A_PT : 1];    // bf16 products: plane p1, or the second half of an fp32 row chunk
    uint4 alo2[C::AREP > 1 ? C::A_PT : 1];   // bf16 products from pre-split planes: plane p2
    uint4 b[C::B_PT];
    bool ok, ok1;                            // the A chunk (and its second fp32 half) lies inside the segment width
  };
  // RSTEP and BM are multiples of 16, so every row this thread stores has the swizzle of arow0.
  static_assert(RSTEP % 16 == 0 && C::BM % 16 == 0, "row steps must keep the swizzle");
  const int scol = ((acol / C::CH) ^ C::swz(arow0)) * C::CH;
  // pre: the segment gives the bf16 term planes; src_bf16: an exact bf16 operand; else (bf16 products) an
  // fp32 source split here into kPlanes terms
  auto lstore = [&](int buf, const Regs& r, bool pre, bool src_bf16) {
#pragma unroll
    for (int i = 0; i < C::A_PT; ++i) {
      uint4 p0, p1 = zero4(), p2 = zero4();
      if constexpr (!C::kBf16) {
        p0 = r.ok ? r.a[i] : zero4();
      } else if (pre || src_bf16) {
        p0 = r.ok ? r.a[i] : zero4();
        p1 = (r.ok && pre) ? r.alo[i] : zero4();
        p2 = (r.ok && pre) ? r.alo2[i] : zero4();
      } else {
        const float4 f0 = __builtin_bit_cast(float4, r.a[i]);
        const float4 f1 = r.ok1 ? __builtin_bit_cast(float4, r.alo[i]) : make_float4(0.f, 0.f, 0.f, 0.f);
        split_bf16x8(f0, f1, p0, p1, p2);
        p0 = r.ok ? p0 : zero4();
        p1 = r.ok ? p1 : zero4();
        p2 = r.ok ? p2 : zero4();
      }
      *(uint4*)(As[buf] + (arow0 + i * RSTEP) * C::ROW + scol) = p0;
      if constexpr (C::AREP > 1) {
        *(uint4*)(As[buf] + (C::BM + arow0 + i * RSTEP) * C::ROW + scol) = p1;
        *(uint4*)(As[buf] + (2 * C::BM + arow0 + i * RSTEP) * C::ROW + scol) = p2;
      }
    }
#pragma unroll
    for (int i = 0; i < C::B_PT; ++i) *(uint4*)(Bs[buf] + (arow0 + i * RSTEP) * C::ROW + scol) = r.b[i];
  };

  f32x4 acc[C::TM][C::TN];
#pragma unroll
  for (int x = 0; x < C::TM; ++x)
#pragma unroll
    for (int y = 0; y < C::TN; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  // MFMA operand reads: lane (i16, g) reads chunk (first chunk of the sub-step) + g of rows i16 + 16 x; the
  // swizzle depends only on i16.
  const int lsw = C::swz(i16);
  auto compute = [&](int buf, bool has_lo) {
    const T* Ab = As[buf] + (wm * C::TM * 16 + i16) * C::ROW;
    const T* Bb = Bs[buf] + (wn * C::TN * 16 + i16) * C::ROW;
#pragma unroll
    for (int sub = 0; sub < C::KW / C::KSUB; ++sub) {
      const int col = (((wk * C::KW + sub * C::KSUB) / C::CH + g) ^ lsw) * C::CH;
      if constexpr (!C::kBf16) {
        f32x4 av[C::TM], bv[C::TN];
#pragma unroll
        for (int x = 0; x < C::TM; ++x) av[x] = *(const f32x4*)(Ab + x * 16 * C::ROW + col);
#pragma unroll
        for (int y = 0; y < C::TN; ++y) bv[y] = *(const f32x4*)(Bb + y * 16 * C::ROW + col);
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
        for (int x = 0; x < C::TM; ++x) av[x] = *(const bf16x8*)(Ab + x * 16 * C::ROW + col);
#pragma unroll
        for (int y = 0; y < C::TN; ++y) bv[y] = *(const bf16x8*)(Bb + y * 16 * C::ROW + col);
#pragma unroll
        for (int x = 0; x < C::TM; ++x)
#pragma unroll
          for (int y = 0; y < C::TN; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[x], bv[y], acc[x][y], 0, 0, 0);
        if (has_lo) {               // uniform: the segment's source is fp32 (planes p1 and p2)
#pragma unroll
          for (int pl = 1; pl < C::AREP; ++pl) {
#pragma unroll
            for (int x = 0; x < C::TM; ++x)
              av[x] = *(const bf16x8*)(Ab + (pl * C::BM + x * 16) * C::ROW + col);
#pragma unroll
            for (int x = 0; x < C::TM; ++x)
#pragma unroll
              for (int y = 0; y < C::TN; ++y)
                acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[x], bv[y], acc[x][y], 0, 0, 0);
          }
        }
      }
    }
  };

  // K runs segment by segment, each with its own two-stage pipeline. Loads are unconditional: rows past
  // M read zeros through the descriptor bound, columns in a segment's padding are zeroed at the LDS store,
  // and past the last stage the loads re-read the last stage into a buffer that is never multiplied.
  uint32_t kbyte_w = 0;                 // byte offset of the segment inside a weight row
  auto run_segment = [&](__amdgpu_buffer_rsrc_t rs, __amdgpu_buffer_rsrc_t rl, __amdgpu_buffer_rsrc_t rm, bool pre,
                         const uint32_t (&ao)[C::A_PT], uint32_t es, int width, int kpad) {
    const bool src_bf16 = es == 2 && !pre;              // exact bf16 operand: no lo part
    auto gload = [&](int st) -> Regs {
      Regs r;
      const int kk = st * C::BK + acol;
      r.ok = kk < width;
      r.ok1 = kk + 4 < width;
#pragma unroll
      for (int i = 0; i < C::A_PT; ++i) {
        const uint32_t off = ao[i] + (uint32_t)(st * C::BK) * es;
        if constexpr (!C::kBf16) {
          r.a[i] = buf_load16(rs, off);
        } else {
          // bf16 source: 8 elements in one 16-byte load (exact, no lo part); pre-split source: 8 elements
          // of each plane; fp32 source: two 16-byte loads, split into bf16 terms at the LDS store (widths
          // are multiples of 4, so the second half may be past the end).
          r.a[i] = buf_load16(rs, off);
          r.alo[i] = pre ? buf_load16(rl, off) : buf_load16(rs, off + 16);
          if (pre) r.alo2[i] = buf_load16(rm, off);
        }
      }
      const uint32_t kb = kbyte_w + (uint32_t)(st * C::BK) * sizeof(T);
#pragma unroll
      for (int i = 0; i < C::B_PT; ++i) r.b[i] = buf_load16(rw, bo[i] + kb);
      return r;
    };
    const int nst = kpad / C::BK;       // segment widths are padded to multiples of kSegK, hence of BK
    const int last = nst - 1;
    Regs r0 = gload(0);
    Regs r1 = gload(min(1, last));
    lstore(0, r0, pre, src_bf16);
    __syncthreads();
    for (int st = 0; st < nst; st += 2) {
      // even stage: LDS buffer 0 holds stage st, r1 holds st + 1
      r0 = gload(min(st + 2, last));
      compute(0, !src_bf16);
      lstore(1, r1, pre, src_bf16);
      __syncthreads();
      // whole pairs of stages when the stage count is even by construction: a single loop exit keeps
      // the accumulators in place (no copies between the two exits' register assignments)
      if constexpr ((kSegK / C::BK) % 2 != 0) {
        if (st + 1 >= nst) break;
      }
      // odd stage: LDS buffer 1 holds stage st + 1, r0 holds st + 2
      r1 = gload(min(st + 3, last));
      compute(1, !src_bf16);
      lstore(0, r0, pre, src_bf16);
      __syncthreads();
    }
    kbyte_w += (uint32_t)kpad * sizeof(T);
  };
  run_segment(rs0, rl0, rm0, pre0, ao0, es0, wd0, kp0);
  if constexpr (nseg > 1) run_segment(rs1, rl1, rm1, pre1, ao1, es1, wd1, kp1);
  if constexpr (nseg > 2) run_segment(rs2, rl2, rm2, pre2, ao2, es2, wd2, kp2);
  (void)bf0;
  (void)bf1;
  (void)bf2;

  // Partial tiles to LDS: lane holds rows 4g..4g+3 of column i16 of each 16x16 block.
  float* Ct = (float*)smem + wk * C::BM * C::CROW;
#pragma unroll
  for (int x = 0; x < C::TM; ++x)
#pragma unroll
    for (int y = 0; y < C::TN; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float o = acc[x][y][v];
        if constexpr (CBIAS) o += cb[y];
        Ct[(wm * C::TM * 16 + x * 16 + 4 * g + v) * C::CROW + wn * C::TN * 16 + y * 16 + i16] = o;
      }
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

template <class T, class C, int NSEG>
__global__ __launch_bounds__(C::NT) void k_gemm_store(AOp a, BOp b, StoreParams p, int nm, int nblocks) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const int L = xcd_remap(blockIdx.x, nblocks);
  const int m0 = (L % nm) * C::BM, n0 = (L / nm) * C::BN;
  gemm_tile<T, C, NSEG>(a, b, m0, n0, smem);
  const float* Ct = (const float*)smem;
  for (int e = threadIdx.x; e < C::BM * (C::BN / 4); e += C::NT) {
    const int r = e / (C::BN / 4), c = (e % (C::BN / 4)) * 4;
    const int gr = m0 + r, gc = n0 + c;
    const bool out = gc < p.ncols;                      // ncols is a multiple of 4
    const bool split = p.hi && gc < p.ncols_hl;
    if (gr >= a.M || !(out || split)) continue;
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = ctile<C>(Ct, r, c + j) + (p.bias && out ? p.bias[gc + j] : 0.f);
      if (p.act == 1) v[j] = tanhf(v[j]);
    }
    if (out) *(float4*)(p.out + (size_t)gr * p.ldo + gc) = make_float4(v[0], v[1], v[2], v[3]);
    if (split) {
      uint4 t0, t1, t2;
      split_bf16x8(make_float4(v[0], v[1], v[2], v[3]), make_float4(0.f, 0.f, 0.f, 0.f), t0, t1, t2);
      *(uint2*)(p.hi + (size_t)gr * p.ld_hl + gc) = make_uint2(t0.x, t0.y);
      *(uint2*)(p.lo + (size_t)gr * p.ld_hl + gc) = make_uint2(t1.x, t1.y);
      *(uint2*)(p.lo2 + (size_t)gr * p.ld_hl + gc) = make_uint2(t2.x, t2.y);
    }
  }
}

// Main loop with LDS-destination loads for bf16 products whose A segments are all pre-split planes (defined
// with the other LDS-destination kernel below); same LDS result as gemm_tile.
template <class C, int NSEG>
__device__ inline void gemm_tile_dma(const AOp& a, const BOp& b, int m0, int n0, char* smem);
// LDS bytes of a tile with the LDS-destination main loop (kLstmStages stages, or the output tile).
constexpr int kLstmStages = 2;
template <class C>
constexpr int dma_lds() {
  constexpr int stg = ((C::kBf16 ? kPlanes : 1) * C::BM + C::BN) * C::BK * (C::kBf16 ? 2 : 4);
  return kLstmStages * stg > C::CT ? kLstmStages * stg : C::CT;
}

// The precomputed input-projection terms (gx) of this thread's (row, unit) elements of an LSTM output tile,
// loaded before the main loop so that their latency (table rows gathered by token id) hides behind it.
template <class C>
struct LstmGx {
  static constexpr int UPT = C::BN / 4;                          // units per tile
  static constexpr int EPT = (C::BM * UPT + C::NT - 1) / C::NT;  // (row, unit) elements per thread
  float v[EPT][4];
  __device__ void load(const LstmParams& p, int M, int m0, int n0) {
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const int e = threadIdx.x + i * C::NT;
      const int r = e / UPT, uu = e % UPT;
      const int row = m0 + r, unit = n0 / 4 + uu;
      const bool ok = p.gx && e < C::BM * UPT && row < M && unit < p.H;
      const int grow = !ok ? 0 : (p.gx_idx ? min((unsigned)p.gx_idx[row], (unsigned)p.gx_rows - 1u) : row * p.gx_S + p.gx_s);
      const int cbase = (uu / kUnitGroup) * (4 * kUnitGroup) + (uu % kUnitGroup);
#pragma unroll
      for (int gt = 0; gt < 4; ++gt)
        v[i][gt] = ok ? p.gx[(size_t)grow * p.ld_gx + p.gx_col0 + n0 + cbase + gt * kUnitGroup] : 0.f;
    }
  }
};

// Gate nonlinearities and cell update over an output tile: acc(r, col) gives the tile's product at tile row
// r and (gate-blocked) tile column col; bias, gx, the previous cell state (through c_idx) complete z.
template <class C, class Acc>
__device__ inline void lstm_epilogue(Acc acc, const LstmParams& p, int M, int m0, int n0, const LstmGx<C>& gx) {
  using G = LstmGx<C>;
#pragma unroll
  for (int i = 0; i < G::EPT; ++i) {
    const int e = threadIdx.x + i * C::NT;
    if (e >= C::BM * G::UPT) break;
    const int r = e / G::UPT, uu = e % G::UPT;
    const int row = m0 + r;
    const int unit = n0 / 4 + uu;
    if (row >= M || unit >= p.H) continue;
    const int cbase = (uu / kUnitGroup) * (4 * kUnitGroup) + (uu % kUnitGroup);
    float z[4];
#pragma unroll
    for (int gt = 0; gt < 4; ++gt) {
      const int col = cbase + gt * kUnitGroup;
      z[gt] = acc(r, col) + (p.bias ? p.bias[n0 + col] : 0.f) + gx.v[i][gt];
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
    if (p.h_hi) {
      uint16_t t0, t1, t2;
      split_bf16(h_new, t0, t1, t2);
      p.h_hi[(size_t)row * p.ld_hl + unit] = t0;
      p.h_lo[(size_t)row * p.ld_hl + unit] = t1;
      p.h_lo2[(size_t)row * p.ld_hl + unit] = t2;
    }
    if (p.y_out) p.y_out[(size_t)(row * p.y_S + p.y_s) * p.ld_y + p.y_col0 + unit] = y;
  }
}

// One output tile of an LSTM GEMM (block bid of nblocks) with the gate/cell epilogue.
template <class T, class C, int NSEG, bool DMA = false>
__device__ inline void lstm_tile(const AOp& a, const BOp& b, const LstmParams& p, int nm, int nblocks, int bid,
                                 char* smem) {
  const int L = xcd_remap(bid, nblocks);
  const int m0 = (L % nm) * C::BM, n0 = (L / nm) * C::BN;
  LstmGx<C> gx;
  gx.load(p, a.M, m0, n0);
  if constexpr (DMA)
    gemm_tile_dma<C, NSEG>(a, b, m0, n0, smem);
  else
    gemm_tile<T, C, NSEG>(a, b, m0, n0, smem);
  const float* Ct = (const float*)smem;
  lstm_epilogue<C>([&](int r, int col) { return ctile<C>(Ct, r, col); }, p, a.M, m0, n0, gx);
}

template <class T, class C, int NSEG, bool DMA = false>
__global__ __launch_bounds__(C::NT) void k_gemm_lstm(AOp a, BOp b, LstmParams p, int nm, int nblocks) {
  __shared__ __attribute__((aligned(16))) char smem[DMA ? dma_lds<C>() : C::LDS];
  lstm_tile<T, C, NSEG, DMA>(a, b, p, nm, nblocks, blockIdx.x, smem);
}

// Two independent LSTM GEMMs in one launch (the encoder's two directions at one step, or two stacked
// layers at consecutive timesteps): blocks [0, nb[0]) run problem 0, the next nb[1] blocks problem 1.
// nb[0] is a multiple of 8, so both problems see the same block-to-XCD dealing.
template <class T, class C, int NS0, int NS1>
__global__ __launch_bounds__(C::NT) void k_gemm_lstm2(LstmPair g) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const int bid = blockIdx.x;
  if (bid < g.nb[0]) {
    if (bid < g.nt[0]) lstm_tile<T, C, NS0>(g.a[0], g.b[0], g.p[0], g.nm[0], g.nt[0], bid, smem);
  } else {
    lstm_tile<T, C, NS1>(g.a[1], g.b[1], g.p[1], g.nm[1], g.nt[1], bid - g.nb[0], smem);
  }
}

// Exchange with lane l ^ X (X = 1 or 2) inside each group of four lanes: a DPP quad permutation, so the
// four threads of an epilogue row trade values without a round trip through LDS.
template <int X>
__device__ inline int quad_xor(int v) {
  static_assert(X == 1 || X == 2, "quad lanes");
  return __builtin_amdgcn_mov_dpp(v, X == 1 ? 0xB1 : 0x4E, 0xF, 0xF, false);   // quad_perm [1,0,3,2] / [2,3,0,1]
}
template <int X>
__device__ inline float quad_xor(float v) {
  return __builtin_bit_cast(float, quad_xor<X>(__builtin_bit_cast(int, v)));
}

// Generator epilogue over the 64 x 128 output tile in LDS: 4 threads per row, 32 interleaved columns
// each. Row max and sum of exponentials are combined across the row's four lanes (quad_xor); the tile's
// top-K is taken with K rounds of a 4-lane argmax (larger logit first, smaller id on ties), each thread
// skipping the columns it already gave away.
// BIASED: the output tile already holds product + bias (added as the tile was written, the same single
// fp32 addition), so the epilogue issues no bias loads of its own.
template <class C, bool BIASED = false>
__device__ inline void gen_epilogue(const char* smem, const GenParams& p, int M, int m0, int n0, int nt, int tid) {
  static_assert(C::NT / C::BM == 4 && C::BN == 128, "generator tile is 64 x 128 with 256 threads");
  const float* Ct = (const float*)smem;
  // thread tid = (row r, part p) owns columns 4 j + p, j < 32: the 64 lanes of a wave then read 64
  // different banks of the output tile for every j
  const int r = tid >> 2, part = tid & 3;
  const int row = m0 + r;
  const float ninf = -__builtin_inff();
  float z[32];
  float mx = ninf;
  if (n0 + C::BN <= p.V) {                 // uniform: every column of the tile is a vocabulary entry
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      if constexpr (BIASED)
        z[j] = ctile<C>(Ct, r, 4 * j + part);
      else
        z[j] = ctile<C>(Ct, r, 4 * j + part) + p.bias[n0 + 4 * j + part];
    }
  } else {
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const int gc = n0 + 4 * j + part;
      if constexpr (BIASED)
        z[j] = gc < p.V ? ctile<C>(Ct, r, 4 * j + part) : ninf;
      else
        z[j] = gc < p.V ? ctile<C>(Ct, r, 4 * j + part) + p.bias[gc] : ninf;
    }
  }
#pragma unroll
  for (int j = 0; j < 32; ++j) mx = fmaxf(mx, z[j]);
  if (p.want && row < M) {
    const int wc = p.want[row] - n0;      // this thread holds column 4 j + part of the tile
    if (wc >= 0 && wc < C::BN && (wc & 3) == part) {
#pragma unroll
      for (int j = 0; j < 32; ++j)
        if (4 * j + part == wc) p.want_logit[row] = z[j];
    }
  }
  if (p.logits && row < M) {
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const int gc = n0 + 4 * j + part;
      if (gc < p.V) p.logits[(size_t)row * p.ld_logits + gc] = z[j];
    }
  }
  float rmx = fmaxf(mx, quad_xor<1>(mx));
  rmx = fmaxf(rmx, quad_xor<2>(rmx));
  float sm = 0.f;
#pragma unroll
  for (int j = 0; j < 32; ++j) sm += __expf(z[j] - rmx);     // exp(-inf) = 0 for columns past V
  sm += quad_xor<1>(sm);
  sm += quad_xor<2>(sm);
  const size_t o = (size_t)row * p.ntiles + nt;
  if (part == 0 && row < M) {
    p.pmax[o] = rmx;
    p.psum[o] = sm;
  }
  // filtered columns start out taken, so the top-K never picks them
  uint32_t taken = 0;
  if (p.banned_bits) {
    uint32_t words[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c0 = n0 + 32 * i;
      words[i] = c0 < p.V ? p.banned_bits[c0 >> 5] : 0u;
    }
#pragma unroll
    for (int j = 0; j < 32; ++j) {            // column offset 4 j + part lies in word j / 8
      if ((words[j >> 3] >> (4 * (j & 7) + part)) & 1u) taken |= 1u << j;
    }
  }
  if (p.unk_cnt && row < M && p.max_unk >= 0 && p.unk_cnt[row] >= p.max_unk) {
    const int c = p.unk_id - n0;
    if (c >= 0 && c < C::BN && (c & 3) == part) taken |= 1u << (c >> 2);
  }
  // with no filter every column is free in the first round, whose best is then the thread's maximum at
  // its first (smallest-id) position
  const bool fast0 = !p.banned_bits && !p.unk_cnt;
  for (int k = 0; k < p.K; ++k) {
    float bv = ninf;
    int bj = 0;
    if (k == 0 && fast0) {
#pragma unroll
      for (int j = 31; j >= 0; --j) {
        if (z[j] == mx) {
          bv = z[j];
          bj = j;
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        const bool free = !((taken >> j) & 1u);
        if (free && z[j] > bv) {                  // strict: the earlier (smaller id) column wins ties
          bv = z[j];
          bj = j;
        }
      }
    }
    int bid = bv > ninf ? n0 + 4 * bj + part : 0x7fffffff;
    const int mine = bid;
    {
      const float ov = quad_xor<1>(bv);
      const int oi = quad_xor<1>(bid);
      if (before(ov, oi, bv, bid)) {
        bv = ov;
        bid = oi;
      }
    }
    {
      const float ov = quad_xor<2>(bv);
      const int oi = quad_xor<2>(bid);
      if (before(ov, oi, bv, bid)) {
        bv = ov;
        bid = oi;
      }
    }
    if (bid == mine && bv > ninf) taken |= 1u << bj;
    if (part == 0 && row < M) {
      p.pval[o * p.K + k] = bv;
      p.pid[o * p.K + k] = bid;
      if (k == 0 && p.pfmax) p.pfmax[o] = bv;
    }
  }
}


// The generator bias of the columns this lane writes in the output tile (column wn * TN * 16 + 16 y + i16
// of the tile at n0, for y < TN; 0 past V), loaded before the main loop so that its latency hides there.
template <class C>
__device__ inline void gen_col_bias(const GenParams& p, int n0, int wn, int i16, float (&cb)[C::TN]) {
#pragma unroll
  for (int y = 0; y < C::TN; ++y) {
    const int gc = n0 + wn * C::TN * 16 + y * 16 + i16;
    cb[y] = gc < p.V ? p.bias[gc] : 0.f;
  }
}

template <class T, class C, int NSEG>
__global__ __launch_bounds__(C::NT) void k_gemm_gen(AOp a, BOp b, GenParams p, int nm, int nblocks) {
  __shared__ __attribute__((aligned(16))) char smem[C::LDS];
  const int L = xcd_remap(blockIdx.x, nblocks);
  const int mt = L % nm, nt = L / nm;
  const int m0 = mt * C::BM, n0 = nt * C::BN;
  const int wave = threadIdx.x >> 6;
  float cb[C::TN];
  gen_col_bias<C>(p, n0, (wave / C::WK) % C::WN, threadIdx.x & 15, cb);
  gemm_tile<T, C, NSEG, true>(a, b, m0, n0, smem, cb);
  gen_epilogue<C, true>(smem, p, a.M, m0, n0, nt, threadIdx.x);
}

// ---------------------------------------------------------------- launchers

using TileWide32 = Tile<float, 2, 2, 1, 2, 4, 32>;
using TileSplit32 = Tile<float, 1, 1, 4, 2, 4, 16>;
// 16 x 32 tiles for GEMMs with few rows: twice the workgroups of a 16 x 64 tiling, which keeps more
// loads in flight per CU (the decoder GEMMs at a few hundred rows are bound by that, not by MFMA).
using TileThin32 = Tile<float, 1, 1, 4, 1, 2, 16>;
// fp32 plain stores with few rows (W_c, concat's query projection): 16 x 16 tiles, twice the workgroups
// of the 16 x 32 LSTM tile (W_c at 320 rows: 8.9 instead of 10.0 us)
using TileStore32 = Tile<float, 1, 1, 4, 1, 1, 16>;
// bf16 stores over many rows (encoder projections, keys, the embedding-gate table): 128 x 128 tiles of
// 8 waves, K stages of 32 (28% faster than 64 x 128 with K stages of 64 at 20480 x 4096 x 1024).
using TileWide16 = Tile<__bf16, 4, 2, 1, 2, 4, 32>;
using TileSplit16 = Tile<__bf16, 1, 1, 4, 2, 4, 32>;
using TileThin16 = Tile<__bf16, 1, 1, 4, 1, 4, 32>;
// bf16 LSTM GEMMs of a few hundred rows: 32 x 64 tiles, two waves per K half. Against the 16 x 64 tile
// the weights are re-read by half as many row tiles, which matters more than the halved workgroup count
// once the bf16 products are cheap (decoder layers at 320-512 rows: 16-32% faster).
using TileMid16 = Tile<__bf16, 1, 2, 2, 2, 2, 32>;
// fp32 generator (fp32 MFMA): the 64 x 128 tile of the wide shapes with a 16-element K stage, which
// halves the LDS stage buffers so that four workgroups fit on a CU.
using TileGen32 = Tile<float, 2, 2, 1, 2, 4, 16>;
// 32 x 128 fp32 generator tiles (two waves) where the last 64-row tile would be at most half full and the
// rows are few: at 160 rows 91 us instead of 108 us (64-row tiles compute 192 rows), at 96 rows 64 instead
// of 78 us; at multiples of 64 rows, and at 480, the 64-row tile is faster. Same partials, bitwise.
using TileGen32h = Tile<float, 1, 2, 1, 2, 4, 16>;
static inline bool gen_rows32(int M) {
  const int r = M % 64;
  return M <= 256 && r > 0 && r <= 32;
}
static_assert(TileGen32h::BN == TileGen32::BN && TileGen32::BN == 128,
              "all generator tiles give the same 128-column partial tiles");
// Pre-split bf16 generator: 64 x 256 tiles (8 waves of 32 x 64; the activations are re-read by half as
// many column tiles as with 64 x 128) and two LDS stages of 24 KB; at 320 and 512 rows this measured
// 10-15% faster than 64 x 128 tiles with three 16 KB stages, and three or four stages of 64 x 256 slower.
constexpr int kGenStages = 2;
constexpr int kGenWN = 4;
// The pre-split generator multiplies the first two of the operand's bf16 term planes (~17 significant bits
// of each activation, a relative error under 2^-16): its output leaves the recurrence, so the error stays
// per step, ~1e-5 on a logit over 1000-wide rows, instead of compounding over the steps the way an error
// of the decoder layers' operands does. The third plane serves those layers.
constexpr int kGenPlanes = 2;
// Three weight planes (fp32 weights): 64 x 128 tiles (four waves, two 36 KB stages, two workgroups per
// CU). At 320 rows the generator took 108 us against 121 us with 64 x 256 tiles (one workgroup per CU)
// and 140 us with the fp32 MFMA kernel. Where the last 64-row tile would be at most half full, the fp32
// kernel's 32-row tiles win instead (160 rows: 84 us against 88 us; 32-row tiles of the three-plane
// kernel, two waves per workgroup and one wave per SIMD, took 140 us), so those row counts stay on it.
constexpr int kGen3WN = 2;
bool gemm_gen_split_rows(int M) { return !gen_rows32(M); }

// One 16-byte-per-lane buffer load into LDS (lane l writes 16 bytes at lds + 16 l). (A function of its
// own: called directly under control flow inside a kernel template, the builtin stops the host-side
// launch stub from being emitted.)
__device__ inline void dma16(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds_at(lds), 16, off, 0, 0, 0);
}

// Vector-memory wait until at most n loads of this wave are outstanding (expcnt and lgkmcnt left alone).
constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | (((n >> 4) & 3) << 14); }

// bf16 generator on a pre-split operand with its operands moved straight into LDS: buffer loads with an
// LDS destination write one 1 KB slice per wave instruction (16 tile rows of 64 bytes, lane l at byte
// 16 l), so a stage needs no staging registers and NSTG stages can be in flight at once. Each wave's loads
// complete in issue order, so waiting until at most SPW (NSTG - 2) of its loads are outstanding (SPW per
// stage) means its share of the oldest stage has landed; a barrier then makes the whole stage visible.
// The barrier is the bare instruction: the fences of __syncthreads would also wait for the stages still
// in flight. Fragment reads, products and the epilogue are those of the register-staged kernel.
template <int WM, int WN, int NSTG, int NPA, int NPB>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_gen_lds(GenSplitA a, BOp b, GenParams p, int nm,
                                                              int nblocks) {
  using C = Tile<__bf16, WM, WN, 1, 2, 4, 32>;         // (32 WM) x (64 WN) tile, waves of 32 x 64
  using CE = Tile<__bf16, WM, 2, 1, 2, 4, 32>;          // the (32 WM) x 128 sub-tiles the epilogue works on
  static_assert(C::BM % 16 == 0 && C::BK == 32 && C::CPR == 4 && C::WK == 1 && CE::BN == 128 &&
                    C::BN % 128 == 0 && CE::BM == C::BM,
                "the slice layout below is written for bf16 generator tiles of 16-row slices with 64-byte rows");
  static_assert(C::BK == kGenKBlock, "a K stage is one block of the K-blocked weights");
  constexpr int NW = C::NT / 64;
  constexpr int ROWB = C::BK * 2;                       // bytes per tile row
  constexpr int RPS = 16;                               // tile rows per 1 KB slice
  constexpr int SA = C::BM / RPS, SB = C::BN / RPS;     // slices per plane of A, and of B
  constexpr int NSL = NPA * SA + NPB * SB;              // slices per stage
  constexpr int SPW = (NSL + NW - 1) / NW;              // slices (loads) per wave per stage, at most
  constexpr int STG = (NPA * C::BM + NPB * C::BN) * ROWB;   // one stage: the A planes' rows, then B's
  // term products kept: plane pair (pa, pb) with pa + pb < NPROD_MAX (two A planes against exact bf16
  // weights; the six leading pairs of three planes each)
  constexpr int NPROD_MAX = NPA > NPB ? NPA : NPB;
  constexpr int NSUB = C::BN / 128;
  constexpr int LDSB = NSTG * STG > NSUB * CE::CT ? NSTG * STG : NSUB * CE::CT;
  // waves may move different numbers of slices only when every wait is for all loads (two stages)
  static_assert((NSL % NW == 0 || NSTG == 2) && NSTG >= 2 && SPW * (NSTG - 2) < 64, "slice layout / wait count");
  __shared__ __attribute__((aligned(16))) char smem[LDSB];
  const int L = xcd_remap(blockIdx.x, nblocks);
  const int mt = L % nm, nt = L / nm;
  const int m0 = mt * C::BM, n0 = nt * C::BN;
  // the wave index read into a scalar register: slice kinds derived from it are then known to be uniform,
  // so the descriptor each load uses is picked by scalar branches rather than a per-lane loop
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i16 = lane & 15, g = lane >> 4;
  const int wn = wave % C::WN, wm = wave / C::WN;
  float cb[C::TN];
  gen_col_bias<C>(p, n0, wn, i16, cb);

  // slice q of a stage: rows 16 q.. of A plane q / SA (q < NPA SA), then of the B planes; wave w moves slices
  // w, w + NW, ... (below NSL); lane's place in a slice: tile row lane / 4, 16-byte slot lane % 4 (chunk
  // slot ^ swz)
  const int srow = lane >> 2, sslot = lane & 3;
  static_assert(NPA >= 1 && NPA <= kPlanes && (NPB == 1 || NPB == 3), "term planes of the operands");
  const __amdgpu_buffer_rsrc_t rpl[kPlanes] = {make_rsrc(a.hi, (uint32_t)a.M * a.ld * 2),
                                               make_rsrc(a.lo, (uint32_t)a.M * a.ld * 2),
                                               make_rsrc(a.lo2, (uint32_t)a.M * a.ld * 2)};
  const uint32_t wplane = (uint32_t)b.Np * b.Kp * 2;    // bytes per weight plane
  __amdgpu_buffer_rsrc_t rw[NPB];
#pragma unroll
  for (int pb = 0; pb < NPB; ++pb) rw[pb] = make_rsrc((const char*)b.W + (size_t)pb * wplane, wplane);
  int sl_kind[SPW], sl_lds[SPW];                        // A plane pa (pa), B plane pb (NPA + pb), -1 none
  uint32_t sl_off[SPW];                                 // lane's byte offset in its operand at K = 0
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int q = wave + NW * i;
    const int kind = q >= NSL ? -1 : (q < NPA * SA ? q / SA : NPA + (q - NPA * SA) / SB);
    const int trow = (kind >= NPA ? (q - NPA * SA) % SB : q % SA) * RPS + srow;   // row in its plane
    const int chunk = sslot ^ C::swz(trow);
    sl_kind[i] = kind;
    sl_lds[i] = ((kind >= NPA ? NPA * C::BM + (kind - NPA) * C::BN : kind * C::BM) + trow - srow) * ROWB;
    if (kind < 0) {
      sl_off[i] = 0;
    } else if (kind >= NPA) {                           // B rows past the packed matrix re-read its last row
      const int br = min(n0 + trow, b.Np - 1);
      sl_off[i] = ((uint32_t)br * C::BK + chunk * C::CH) * 2;   // in K block 0 (the stage adds its block)
    } else {                                            // A rows past M re-read row M - 1 (never stored)
      const int ar = min(m0 + trow, a.M - 1);
      sl_off[i] = ((uint32_t)ar * a.ld + chunk * C::CH) * 2;
    }
  }
  const int nst = a.kpad / C::BK;

  f32x4 acc[C::TM][C::TN];
#pragma unroll
  for (int x = 0; x < C::TM; ++x)
#pragma unroll
    for (int y = 0; y < C::TN; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int col = (g ^ C::swz(i16)) * C::CH;           // this lane's 16-byte chunk of a fragment row
  // stages past the last re-load the last one into a buffer that is never multiplied, which keeps every
  // wave's count of loads in flight the same on every iteration; stage st of A is ROWB bytes into each
  // row, of B the st-th K block of the weights
#define ONMT_GEN_ISSUE(ST)                                                                              \
  do {                                                                                                  \
    char* sb_ = smem + ((ST) % NSTG) * STG;                                                             \
    const uint32_t ks_ = (uint32_t)((ST) < nst ? (ST) : nst - 1);                                       \
    const uint32_t ko_ = ks_ * ROWB, kb_ = ks_ * (uint32_t)b.Np * ROWB;                                 \
    _Pragma("unroll") for (int i = 0; i < SPW; ++i) {                                                   \
      if (sl_kind[i] == NPA)                                                                            \
        dma16(rw[0], sb_ + sl_lds[i], sl_off[i] + kb_);                                                 \
      else if (NPB > 1 && sl_kind[i] == NPA + 1)                                                        \
        dma16(rw[NPB > 1 ? 1 : 0], sb_ + sl_lds[i], sl_off[i] + kb_);                                   \
      else if (NPB > 2 && sl_kind[i] == NPA + 2)                                                        \
        dma16(rw[NPB > 2 ? 2 : 0], sb_ + sl_lds[i], sl_off[i] + kb_);                                   \
      else if (sl_kind[i] == 0)                                                                         \
        dma16(rpl[0], sb_ + sl_lds[i], sl_off[i] + ko_);                                               \
      else if (sl_kind[i] == 1)                                                                         \
        dma16(rpl[1], sb_ + sl_lds[i], sl_off[i] + ko_);                                               \
      else if (NPA > 2 && sl_kind[i] == 2)                                                              \
        dma16(rpl[2], sb_ + sl_lds[i], sl_off[i] + ko_);                                               \
    }                                                                                                   \
  } while (0)
#pragma unroll
  for (int st = 0; st < NSTG - 1; ++st) ONMT_GEN_ISSUE(st);
  for (int st = 0; st < nst; ++st) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(SPW * (NSTG - 2)));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    ONMT_GEN_ISSUE(st + NSTG - 1);                      // refills the buffer multiplied at st - 1
    const char* base = smem + (st % NSTG) * STG;
    const __bf16* Ah = (const __bf16*)base + (wm * C::TM * 16 + i16) * C::ROW;
    const __bf16* Bb = (const __bf16*)base + (NPA * C::BM + wn * C::TN * 16 + i16) * C::ROW;
    bf16x8 av[C::TM], bv[NPB][C::TN];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
      for (int y = 0; y < C::TN; ++y) bv[pb][y] = *(const bf16x8*)(Bb + (pb * C::BN + y * 16) * C::ROW + col);
#pragma unroll
    for (int pa = 0; pa < NPA; ++pa) {
#pragma unroll
      for (int x = 0; x < C::TM; ++x) av[x] = *(const bf16x8*)(Ah + (pa * C::BM + x * 16) * C::ROW + col);
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb) {
        if (pa + pb >= NPROD_MAX) continue;
#pragma unroll
        for (int x = 0; x < C::TM; ++x)
#pragma unroll
          for (int y = 0; y < C::TN; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[x], bv[pb][y], acc[x][y], 0, 0, 0);
      }
    }
  }
#undef ONMT_GEN_ISSUE
  // every load (including the re-loads past the end) has landed before the output tiles reuse the buffers
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();
  // the BM x BN output as BN / 128 sub-tiles of BM x 128, each in the epilogue's layout, reduced at once
  // (threads CE::NT s .. take sub-tile s, one partials tile of 128 columns); staging the
  // sub-tiles one after the other through one buffer measured far slower
  {
    const int sub = (wn * C::TN * 16) / 128, c0 = (wn * C::TN * 16) % 128;
    float* Ct = (float*)(smem + sub * CE::CT);
#pragma unroll
    for (int x = 0; x < C::TM; ++x)
#pragma unroll
      for (int y = 0; y < C::TN; ++y)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          Ct[(wm * C::TM * 16 + x * 16 + 4 * g + v) * CE::CROW + c0 + y * 16 + i16] = acc[x][y][v] + cb[y];
  }
  __syncthreads();
  const int sub = tid / CE::NT, n0s = n0 + 128 * sub;
  if (n0s < b.Np) gen_epilogue<CE, true>(smem + sub * CE::CT, p, a.M, m0, n0s, n0s / 128, tid % CE::NT);
}


// Vector-memory "no wait", LDS wait until nothing is outstanding (for LDS stores before a bare barrier).
constexpr int kWaitLgkm0 = 15 | (7 << 4) | (0 << 8) | (3 << 14);

// gemm_tile for fp32 products, or bf16 products whose A segments (one or two) are all pre-split term
// planes, with the operands moved straight into LDS: a stage of the A rows of every plane (fp32: one) and
// the B rows is sliced into 1 KB pieces
// (RPS tile rows each; lane l writes row l / (ROWB / 16), 16-byte slot l % (ROWB / 16)), kLstmStages stages
// in flight, waits and bare barriers as in k_gemm_gen_lds. A rows come through the segment's row map
// (beam parents) and rows past M re-read row M - 1. The planes' columns past a segment's width are not
// assumed to be zero: on a segment's last stage they are cleared in LDS before the products. Products,
// their order and the output tile (WK partial planes) are those of gemm_tile, so the results are equal.
template <class C, int NSEG>
__device__ inline void gemm_tile_dma(const AOp& a, const BOp& b, int m0, int n0, char* smem) {
  static_assert(C::KW == C::KSUB && NSEG >= 1 && NSEG <= 2, "one MFMA K step per wave and stage");
  // bf16 products: kPlanes term planes of A; fp32 products: A itself
  constexpr int ES = C::kBf16 ? 2 : 4, NPA = C::kBf16 ? kPlanes : 1;
  constexpr int NW = C::NT / 64, ROWB = C::BK * ES, RPS = 1024 / ROWB, LPR = ROWB / 16;
  constexpr int SA = C::BM / RPS, SB = C::BN / RPS, SPW = (NPA * SA + SB) / NW;
  constexpr int STG = (NPA * C::BM + C::BN) * ROWB, NSTG = kLstmStages;
  static_assert(1024 % ROWB == 0 && C::BM % RPS == 0 && C::BN % RPS == 0 && (NPA * SA + SB) % NW == 0 &&
                    SPW * (NSTG - 2) < 64 && dma_lds<C>() >= NSTG * STG,
                "slice layout");
  // the wave index read into a scalar register: slice kinds derived from it are then known to be uniform,
  // so the descriptor each load uses is picked by scalar branches rather than a per-lane loop
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i16 = lane & 15, g = lane >> 4;
  const int wk = wave % C::WK, wn = (wave / C::WK) % C::WN, wm = wave / (C::WK * C::WN);
  const int srow = lane / LPR, sslot = lane % LPR;
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(b.W, (uint32_t)b.Np * b.Kp * ES);
  // per segment (constant indices only): plane descriptors, stage count, width
  __amdgpu_buffer_rsrc_t rp[2][kPlanes];
  int nst[2] = {0, 0}, wd[2] = {0, 0};
#pragma unroll
  for (int s = 0; s < NSEG; ++s) {
    const uint32_t bytes = (uint32_t)a.seg[s].rows * a.seg[s].ld * ES;
    rp[s][0] = make_rsrc(a.seg[s].base, bytes);
    rp[s][1] = NPA > 1 ? make_rsrc(a.seg[s].lo, bytes) : rp[s][0];
    rp[s][2] = NPA > 2 ? make_rsrc(a.seg[s].lo2, bytes) : rp[s][0];
    nst[s] = a.seg[s].kpad / C::BK;
    wd[s] = a.seg[s].width;
  }
  const int total = nst[0] + nst[1];
  const int kb1 = NSEG > 1 ? a.seg[0].kpad : 0;        // K offset of segment 1 in the weight rows
  int sl_kind[SPW], sl_lds[SPW];
  uint32_t aoff[2][SPW], boff[SPW];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int q = wave + NW * i;
    const int kind = q < NPA * SA ? q / SA : NPA;           // an A plane, or NPA for B
    const int trow = (kind == NPA ? q - NPA * SA : q % SA) * RPS + srow;
    const int chunk = sslot ^ C::swz(trow);
    sl_kind[i] = kind;
    sl_lds[i] = ((kind == NPA ? NPA * C::BM : kind * C::BM) + trow - srow) * ROWB;
    boff[i] = ((uint32_t)min(n0 + trow, b.Np - 1) * b.Kp + chunk * C::CH) * ES;
    const int r = min(m0 + trow, a.M - 1);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      aoff[s][i] = 0;
      if (s < NSEG) {
        const int rr = a.seg[s].idx ? a.seg[s].idx[r] : r;
        aoff[s][i] = ((uint32_t)rr * a.seg[s].ld + chunk * C::CH) * ES;
      }
    }
  }
  f32x4 acc[C::TM][C::TN];
#pragma unroll
  for (int x = 0; x < C::TM; ++x)
#pragma unroll
    for (int y = 0; y < C::TN; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
  // stages past the last re-load the last one into a buffer that is never multiplied. The segment is a
  // template constant of issue_seg, so every descriptor and offset array is indexed by constants and stays
  // in registers (a runtime segment index put them in scratch memory).
  auto issue_seg = [&](auto seg_c, int ls, char* sb) {
    constexpr int S = decltype(seg_c)::value;
    const uint32_t ka = (uint32_t)ls * ROWB, kb = (uint32_t)((S ? kb1 : 0) + ls * C::BK) * ES;
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      if (sl_kind[i] == NPA)
        dma16(rw, sb + sl_lds[i], boff[i] + kb);
      else if (NPA == 1 || sl_kind[i] == 0)
        dma16(rp[S][0], sb + sl_lds[i], aoff[S][i] + ka);
      else if (sl_kind[i] == 1)
        dma16(rp[S][1], sb + sl_lds[i], aoff[S][i] + ka);
      else
        dma16(rp[S][2], sb + sl_lds[i], aoff[S][i] + ka);
    }
  };
  auto issue = [&](int G) {
    const int gg = G < total ? G : total - 1;
    char* sb = smem + (G % NSTG) * STG;
    if constexpr (NSEG > 1) {
      if (gg >= nst[0]) {
        issue_seg(std::integral_constant<int, 1>{}, gg - nst[0], sb);
        return;
      }
    }
    issue_seg(std::integral_constant<int, 0>{}, gg, sb);
  };
#pragma unroll
  for (int G = 0; G < NSTG - 1; ++G) issue(G);
  const int col = ((wk * C::KW / C::CH + g) ^ C::swz(i16)) * C::CH;
  for (int G = 0; G < total; ++G) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(SPW * (NSTG - 2)));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    char* base = smem + (G % NSTG) * STG;
    {
      const int s = G >= nst[0] ? 1 : 0;
      const int ls = G - (s ? nst[0] : 0);
      const int w = s ? wd[1] : wd[0];
      if ((ls + 1) * C::BK > w) {                      // the segment's last stage reaches past its width
        for (int e = tid; e < NPA * C::BM * C::CPR; e += C::NT) {
          const int row = e / C::CPR, c = e % C::CPR;   // row of the A planes, one after the other; chunk
          if (ls * C::BK + c * C::CH >= w)
            *(uint4*)(base + row * ROWB + ((c ^ C::swz(row % C::BM)) * 16)) = zero4();
        }
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
      }
    }
    issue(G + NSTG - 1);                                // refills the buffer multiplied at G - 1
    if constexpr (C::kBf16) {
      const __bf16* Ah = (const __bf16*)base + (wm * C::TM * 16 + i16) * C::ROW;
      const __bf16* Bb = (const __bf16*)base + (NPA * C::BM + wn * C::TN * 16 + i16) * C::ROW;
      bf16x8 av[C::TM], bv[C::TN];
#pragma unroll
      for (int y = 0; y < C::TN; ++y) bv[y] = *(const bf16x8*)(Bb + y * 16 * C::ROW + col);
#pragma unroll
      for (int pl = 0; pl < NPA; ++pl) {
#pragma unroll
        for (int x = 0; x < C::TM; ++x) av[x] = *(const bf16x8*)(Ah + (pl * C::BM + x * 16) * C::ROW + col);
#pragma unroll
        for (int x = 0; x < C::TM; ++x)
#pragma unroll
          for (int y = 0; y < C::TN; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[x], bv[y], acc[x][y], 0, 0, 0);
      }
    } else {      // fp32: one 16-byte chunk (K = 4 g .. 4 g + 3) per lane and row, four K = 4 products
      const float* Af = (const float*)base + (wm * C::TM * 16 + i16) * C::ROW;
      const float* Bf = (const float*)base + (C::BM + wn * C::TN * 16 + i16) * C::ROW;
      f32x4 av[C::TM], bv[C::TN];
#pragma unroll
      for (int x = 0; x < C::TM; ++x) av[x] = *(const f32x4*)(Af + x * 16 * C::ROW + col);
#pragma unroll
      for (int y = 0; y < C::TN; ++y) bv[y] = *(const f32x4*)(Bf + y * 16 * C::ROW + col);
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int x = 0; x < C::TM; ++x)
#pragma unroll
          for (int y = 0; y < C::TN; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[x][m], bv[y][m], acc[x][y], 0, 0, 0);
    }
  }
  // every load (including the re-loads past the end) has landed before the output tile reuses the buffers
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();
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
static inline void grid_of(const AOp& a, const BOp& b, int& nm, int& nblocks) {
  nm = (a.M + C::BM - 1) / C::BM;
  nblocks = nm * (b.Np / C::BN);
}

// Buffer descriptors address at most 2 GiB: reject operands that do not fit (never the case for the
// supported model shapes, which the C ABI validates).
template <class T>
static inline bool operands_fit(const AOp& a, const BOp& b) {
  const uint64_t lim = 1ull << 31;
  if ((uint64_t)b.Np * b.Kp * sizeof(T) >= lim || b.Np % 128 || b.Kp % kSegK) return false;
  for (int s = 0; s < a.nseg; ++s)
    if ((uint64_t)a.seg[s].rows * a.seg[s].ld * (a.seg[s].bf16 ? 2 : 4) >= lim || a.seg[s].kpad % kSegK) return false;
  return true;
}

int gen_tile_cols() { return TileGen32::BN; }

// Kernels are specialised on the number of A segments, so that a stage's segment is known at compile
// time wherever there is only one.
template <class T, class C>
static hipError_t launch_store(const AOp& a, const BOp& b, const StoreParams& p, hipStream_t st) {
  int nm, nb;
  grid_of<C>(a, b, nm, nb);
  if (!operands_fit<T>(a, b) || a.nseg < 1 || a.nseg > 3) return hipErrorInvalidValue;
  if (nb == 0) return hipSuccess;
  if (a.nseg == 1) hipLaunchKernelGGL((k_gemm_store<T, C, 1>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  else if (a.nseg == 2) hipLaunchKernelGGL((k_gemm_store<T, C, 2>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  else hipLaunchKernelGGL((k_gemm_store<T, C, 3>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  return hipGetLastError();
}

// The LDS-destination main loop applies to bf16 products whose one or two A segments are all pre-split ...
static inline bool all_pre_split(const AOp& a) {
  if (a.nseg < 1 || a.nseg > 2) return false;
  for (int s = 0; s < a.nseg; ++s)
    if (!a.seg[s].bf16 || !a.seg[s].lo || !a.seg[s].lo2 || a.seg[s].ld < a.seg[s].kpad) return false;
  return true;
}

// ... and to fp32 products whose one or two A segments have 16-byte aligned rows (widths and strides are
// multiples of 4 elements): with the 16 x 32 fp32 LSTM tiles the decoder layers of the default workload
// took 19.2 instead of 20.3 us (a 32 x 64 tile with two waves per K half, LDS-destination too, 26.4 us).
static inline bool all_fp32_rows(const AOp& a) {
  if (a.nseg < 1 || a.nseg > 2) return false;
  for (int s = 0; s < a.nseg; ++s)
    if (a.seg[s].bf16 || a.seg[s].ld % 4 || a.seg[s].width % 4) return false;
  return true;
}

template <class T, class C>
static hipError_t launch_lstm(const AOp& a, const BOp& b, const LstmParams& p, hipStream_t st) {
  int nm, nb;
  grid_of<C>(a, b, nm, nb);
  if (!operands_fit<T>(a, b) || a.nseg < 1 || a.nseg > 3) return hipErrorInvalidValue;
  if (nb == 0) return hipSuccess;
  if constexpr (!C::kBf16 && C::KW == C::KSUB) {
    if (all_fp32_rows(a)) {
      if (a.nseg == 1)
        hipLaunchKernelGGL((k_gemm_lstm<T, C, 1, true>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
      else
        hipLaunchKernelGGL((k_gemm_lstm<T, C, 2, true>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
      return hipGetLastError();
    }
  }
  if constexpr (C::kBf16 && C::KW == C::KSUB && C::CPR == 8) {
    if (all_pre_split(a)) {
      if (a.nseg == 1)
        hipLaunchKernelGGL((k_gemm_lstm<T, C, 1, true>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
      else
        hipLaunchKernelGGL((k_gemm_lstm<T, C, 2, true>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
      return hipGetLastError();
    }
  }
  if (a.nseg == 1) hipLaunchKernelGGL((k_gemm_lstm<T, C, 1>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  else if (a.nseg == 2) hipLaunchKernelGGL((k_gemm_lstm<T, C, 2>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  else hipLaunchKernelGGL((k_gemm_lstm<T, C, 3>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
  return hipGetLastError();
}

template <class T, class C, int NS0, int NS1>
static hipError_t launch_lstm2(LstmPair g, hipStream_t st) {
  for (int i = 0; i < 2; ++i) {
    grid_of<C>(g.a[i], g.b[i], g.nm[i], g.nt[i]);
    if (!operands_fit<T>(g.a[i], g.b[i])) return hipErrorInvalidValue;
  }
  if (g.a[0].nseg != NS0 || g.a[1].nseg != NS1) return hipErrorInvalidValue;
  g.nb[0] = (g.nt[0] + 7) / 8 * 8;
  g.nb[1] = g.nt[1];
  const int nb = g.nb[0] + g.nb[1];
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_lstm2<T, C, NS0, NS1>), dim3(nb), dim3(C::NT), 0, st, g);
  return hipGetLastError();
}

// The generator's A operand is the attentional vector alone (one segment).
template <class T, class C>
static hipError_t launch_gen(const AOp& a, const BOp& b, const GenParams& p, hipStream_t st) {
  int nm, nb;
  grid_of<C>(a, b, nm, nb);
  if (!operands_fit<T>(a, b) || a.nseg != 1) return hipErrorInvalidValue;
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_gen<T, C, 1>), dim3(nb), dim3(C::NT), 0, st, a, b, p, nm, nb);
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
  return launch_store<float, TileStore32>(a, b, p, st);
}

hipError_t gemm_lstm(int bf16, int shape, const AOp& a, const BOp& b, const LstmParams& p, hipStream_t st) {
  if (bf16) {
    if (shape == kShapeWide) return launch_lstm<__bf16, TileWide16>(a, b, p, st);
    if (shape == kShapeSplitK) return launch_lstm<__bf16, TileSplit16>(a, b, p, st);
    if (shape == kShapeMid) return launch_lstm<__bf16, TileMid16>(a, b, p, st);
    return launch_lstm<__bf16, TileThin16>(a, b, p, st);
  }
  if (shape == kShapeWide) return launch_lstm<float, TileWide32>(a, b, p, st);
  if (shape == kShapeSplitK) return launch_lstm<float, TileSplit32>(a, b, p, st);
  return launch_lstm<float, TileThin32>(a, b, p, st);
}

template <class T, class C>
static hipError_t lstm2_dispatch(const LstmPair& g, hipStream_t st) {
  const int n0 = g.a[0].nseg, n1 = g.a[1].nseg;
  if (n0 == 1 && n1 == 1) return launch_lstm2<T, C, 1, 1>(g, st);
  if (n0 == 1 && n1 == 2) return launch_lstm2<T, C, 1, 2>(g, st);
  if (n0 == 2 && n1 == 2) return launch_lstm2<T, C, 2, 2>(g, st);
  return hipErrorInvalidValue;
}

hipError_t gemm_lstm2(int bf16, int shape, const LstmPair& g, hipStream_t st) {
  if (shape != kShapeSplitKThin && shape != kShapeMid) return hipErrorInvalidValue;
  if (!bf16) return lstm2_dispatch<float, TileThin32>(g, st);
  return shape == kShapeMid ? lstm2_dispatch<__bf16, TileMid16>(g, st) : lstm2_dispatch<__bf16, TileThin16>(g, st);
}

__global__ void k_split_rows(const float* __restrict__ src, int ld_src, int rows, int cols, uint16_t* __restrict__ hi,
                             uint16_t* __restrict__ lo, uint16_t* __restrict__ lo2, int ld_dst) {
  const size_t n = (size_t)rows * ld_dst;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / ld_dst), c = (int)(i % ld_dst);
    uint16_t t0 = 0, t1 = 0, t2 = 0;
    if (c < cols) split_bf16(src[(size_t)r * ld_src + c], t0, t1, t2);
    hi[i] = t0;
    lo[i] = t1;
    lo2[i] = t2;
  }
}

hipError_t split_rows(const float* src, int ld_src, int rows, int cols, uint16_t* hi, uint16_t* lo, uint16_t* lo2,
                      int ld_dst, hipStream_t st) {
  const size_t n = (size_t)rows * ld_dst;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_split_rows, dim3((unsigned)blocks), dim3(256), 0, st, src, ld_src, rows, cols, hi, lo, lo2,
                     ld_dst);
  return hipGetLastError();
}

hipError_t gemm_gen(const AOp& a, const BOp& b, const GenParams& p, hipStream_t st) {
  return gen_rows32(a.M) ? launch_gen<float, TileGen32h>(a, b, p, st) : launch_gen<float, TileGen32>(a, b, p, st);
}

hipError_t gemm_gen_split(const GenSplitA& a, const BOp& b, int b_planes, const GenParams& p, hipStream_t st) {
  if (b_planes != 1 && b_planes != 3) return hipErrorInvalidValue;
  const uint64_t lim = 1ull << 31;
  // the K-blocked weights are read up to the operand's padded width: a.kpad == b.Kp
  if (a.M < 1 || a.kpad % kSegK || a.kpad != b.Kp || a.ld < a.kpad || b.Np % 128 ||
      (uint64_t)a.M * a.ld * 2 >= lim || (uint64_t)b.Np * b.Kp * 2 >= lim)
    return hipErrorInvalidValue;
  auto launch = [&](auto kernel, int BM, int BN, int threads) {
    const int nm = (a.M + BM - 1) / BM;
    const int nblocks = nm * ((b.Np + BN - 1) / BN);
    hipLaunchKernelGGL(kernel, dim3(nblocks), dim3(threads), 0, st, a, b, p, nm, nblocks);
  };
  if (b_planes == 1)
    launch(k_gemm_gen_lds<2, kGenWN, kGenStages, kGenPlanes, 1>, 64, 64 * kGenWN, 128 * kGenWN);
  else
    launch(k_gemm_gen_lds<2, kGen3WN, kGenStages, kPlanes, 3>, 64, 64 * kGen3WN, 128 * kGen3WN);
  return hipGetLastError();
}

}  // namespace onmt
