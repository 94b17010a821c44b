// Host-visible launch interface of the libonmt kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace onmt {

// K segments of GEMM operands are padded to multiples of this many elements; every tile's K stage
// (32, 64 or 128 elements) divides it, so a stage never straddles two segments.
constexpr int kSegK = 128;

// bf16 products carry each fp32 activation as this many bf16 terms (RNE of the value, then of each
// remainder), ~24 significant bits: the products see the fp32 value itself.
constexpr int kPlanes = 3;

// One K-segment of a GEMM's A operand: A[r, off + k] = base[map(r) * ld + k] for k < width,
// 0 for width <= k < kpad. map(r) = idx ? idx[r] : r. The buffer must be smaller than 2 GiB.
struct Seg {
  const void* base;
  const int32_t* idx;
  int rows;      // rows in the source buffer (reads are bounded by rows * ld elements)
  int ld;
  int width;
  int kpad;
  int bf16;      // 1: base holds bf16 values (exact operands)
  const void* lo;   // bf16 products only: base, lo and lo2 are the kPlanes bf16 term planes of fp32 values
  const void* lo2;  // (bf16 = 1, width a multiple of 8); the operand is their sum, as if split on load
};

struct AOp {
  Seg seg[3];
  int nseg;
  int M;
};

// Packed weight matrix [Np, Kp], K contiguous. Np is a multiple of 128, Kp of kSegK.
struct BOp {
  const void* W;
  int Np;
  int Kp;
};

// Plain store epilogue: out[r, n] = act(acc + bias[n]) for n < ncols. act: 0 none, 1 tanh.
// Optionally (hi != nullptr) the same values split into the bf16 term planes hi, lo, lo2 [rows, ld_hl]
// for columns n < ncols_hl (columns past ncols hold act(0), zero for the tanh stores).
struct StoreParams {
  const float* bias;
  float* out;
  int ldo;
  int ncols;
  int act;
  uint16_t* hi;
  uint16_t* lo;
  int ld_hl;
  int ncols_hl;
  uint16_t* lo2;
};

// LSTM cell epilogue over gate-blocked columns (groups of 32 = 4 gates x kUnitGroup = 8 units).
struct LstmParams {
  const float* bias;            // packed [Np]
  const float* gx;              // optional precomputed input projection (packed columns)
  int ld_gx, gx_col0, gx_S, gx_s;   // gx row for GEMM row b is b * gx_S + gx_s ...
  const int32_t* gx_idx;        // ... or gx_idx[b] when given (a table row per GEMM row), clamped to
  int gx_rows;                  // [0, gx_rows)
  const float* c_in;            // previous cell state rows, through c_idx (nullable = identity)
  const int32_t* c_idx;
  int ld_c;
  const float* h_in;            // previous hidden (identity rows), used when a row is masked
  int ld_h_in;
  float* h_out;
  float* c_out;
  int ld_out;
  uint16_t* h_hi;               // optional bf16 term planes of h_out (row stride ld_hl)
  uint16_t* h_lo;
  int ld_hl;
  uint16_t* h_lo2;
  float* y_out;                 // optional layer output row b * y_S + y_s, column offset y_col0
  int ld_y, y_S, y_s, y_col0;
  const int32_t* lens;          // optional: GEMM row b is active iff y_s < lens[b]
  int H;                        // real units
};

// Two LSTM GEMM problems for one launch (nm/nt/nb are filled in by the launcher).
struct LstmPair {
  AOp a[2];
  BOp b[2];
  LstmParams p[2];
  int nm[2];     // row tiles
  int nt[2];     // tiles
  int nb[2];     // blocks (problem 0's rounded up to a multiple of 8)
};

// Generator epilogue: per (row, column tile) max, sum of exp and top-K; optional raw logits.
struct GenParams {
  const float* bias;
  int V;
  int K;
  int ntiles;
  float* pmax;                  // [M, ntiles]
  float* psum;                  // [M, ntiles]
  float* pval;                  // [M, ntiles, K]
  int32_t* pid;                 // [M, ntiles, K]
  float* logits;                // optional [M, ld_logits]
  int ld_logits;
  const int32_t* want;          // optional [M]: column whose logit is copied to want_logit[row]
  float* want_logit;
  // hypothesis filters (optional): columns never entered into the top-K lists (max and sum of exp
  // still cover every column): banned_bits[c >> 5] bit c & 31, and unk_id on rows whose UNK count has
  // reached max_unk (max_unk < 0: no limit). pfmax (set when filtering) = each tile's largest allowed logit.
  const uint32_t* banned_bits;
  const int32_t* unk_cnt;       // [M]
  int unk_id, max_unk;
  float* pfmax;                 // [M, ntiles]
};

// kShapeMid: 32 x 64 tiles with two waves splitting K, for bf16 LSTM GEMMs of a few hundred rows (fp32 maps
// it to the thin tile); when every A segment is a pre-split plane pair the operands go straight into LDS.
enum GemmShape { kShapeWide = 0, kShapeSplitK = 1, kShapeSplitKThin = 2, kShapeMid = 3 };

hipError_t gemm_store(int bf16, int shape, const AOp& a, const BOp& b, const StoreParams& p, hipStream_t st);
hipError_t gemm_lstm(int bf16, int shape, const AOp& a, const BOp& b, const LstmParams& p, hipStream_t st);
// Two independent thin-shape LSTM GEMMs in one launch (segment counts 1+1, 1+2 or 2+2).
hipError_t gemm_lstm2(int bf16, int shape, const LstmPair& g, hipStream_t st);
// The generator with fp32 operands and the fp32 MFMA (fp32 models at the row counts gemm_gen_split_rows
// leaves to it).
hipError_t gemm_gen(const AOp& a, const BOp& b, const GenParams& p, hipStream_t st);


// bf16 generator operand already split into its bf16 term planes (A = hi + lo + lo2), row-major [M, ld]
// each with zeros in the K padding (columns width .. kpad - 1).
struct GenSplitA {
  const uint16_t* hi;
  const uint16_t* lo;
  int M;
  int ld;      // elements per row, >= kpad
  int kpad;    // multiple of kSegK
  const uint16_t* lo2;
};
// The generator on a pre-split operand, operands moved straight into LDS, the weights given as b_planes
// bf16 term planes (plane p of the K-blocked [Np, Kp] matrix at element offset p * Np * Kp).
// b_planes = 1 (bf16 weights): the first two term planes of A are multiplied (A ~ hi + lo; lo2 is not
// read), since the logits do not feed back into the decoder. b_planes = 3 (fp32 weights as three bf16
// terms): the six term products whose order of magnitude is at least 2^-16 of the leading one
// (hi.hi, hi.lo, lo.hi, lo.lo, hi.lo2, lo2.hi), accumulated in fp32: the six-product bf16 scheme of
// Henry, Tang and Heinecke (ARITH 2019), whose dropped products lie below one fp32 rounding.
// Its weights are K-blocked: element (n, k) of the [Np, Kp] matrix sits at (k / kGenKBlock) * Np *
// kGenKBlock + n * kGenKBlock + k % kGenKBlock, so that one K stage of a column tile is one contiguous block
// (with row-major weights each load instruction touched 16 rows 2 KB apart for 64 bytes each).
constexpr int kGenKBlock = 32;
hipError_t gemm_gen_split(const GenSplitA& a, const BOp& b, int b_planes, const GenParams& p, hipStream_t st);
// fp32 models: whether M rows take the three-plane generator (else the fp32 MFMA kernel, gemm_gen).
bool gemm_gen_split_rows(int M);
int gen_tile_cols();

// Attention coverage of the hypotheses (optional): out[r, s] = in[parent[r], s] + a[r, s] for the real
// positions (0 at pads), cp[r] = beta * sum over the real positions of log(min(out[r, s], 1)).
struct Coverage {
  const float* in;              // [N, S_max]
  float* out;                   // [N, S_max]
  const int32_t* parent;        // [N]
  double beta;
  double* cp;                   // [N]
};

// Optional per-row outputs of the attention softmax (beyond the weights themselves).
struct AttnExtra {
  const Coverage* cov;          // coverage update and penalty
  int32_t* align;               // [N]: position of the largest weight (smaller position on ties)
};

// v_a != nullptr selects concat scores v_a . tanh(q_k + keys[s]) (q = the projected query); else q_k . keys[s].
hipError_t attention(const float* q, int ld_q, const float* keys, const float* v_a, const float* mem,
                     const int32_t* lens, int B, int S_max, int H, int Hm, int K, float* scores, float* ctx,
                     float* attn, const AttnExtra& ex, hipStream_t st);
size_t attention_lds_bytes(int S_max, int H, int K);

hipError_t lse_topk_merge(const float* pmax, const float* psum, const float* pval, const int32_t* pid, int M,
                          int ntiles, int K, float* out_val, int32_t* out_id, float* out_lse, hipStream_t st);
// Teacher-forced scoring of all steps: rows r = t * B + b of the generator partials; logp[b * ld + t] =
// want_logit[r] - logsumexp(r) for t < len[b] (0 otherwise, t < steps); nll[b] = -sum_t logp[b, t] in fp64.
hipError_t score_rows(const float* pmax, const float* psum, int ntiles, const float* want_logit, const int32_t* len,
                      int B, int steps, float* logp, int ld, double* nll, hipStream_t st);
hipError_t subtract_rows(float* x, int ld, const float* lse, int M, int ncols, hipStream_t st);

struct BeamParams {
  int B, K, V, T_max, eos, pad;
  double alpha, lp_tmax;
  double* score;
  int32_t* parent;
  int32_t* tok;
  int32_t* bp_slot;
  int32_t* bp_tok;
  float* bp_logp;
  int32_t* done;
  int32_t* steps;
  int32_t* done_count;
  double* best_norm;
  double* best_raw;
  int32_t* best_t;
  int32_t* best_slot;
  int32_t* best_tok;
  float* best_logp;
  const double* cp;             // optional coverage penalty of each row's hypothesis this step [N]
  const int32_t* align;         // optional [N]: attention argmax of each row at this step
  int32_t* bp_align;            // [T_max, N] (with align)
  int32_t* best_align;          // [B] (with align)
  int32_t* unk_cnt;             // [N] UNK tokens of each slot's hypothesis
  int unk_id;
  int32_t* tr_slot;             // optional trace [T_max, B, K]
  int32_t* tr_tok;
  double* tr_cand;
};

// Generator partials of one decoder step (per row and column tile), as written by gemm_gen.
struct GenPartials {
  const float* pmax;
  const float* psum;
  const float* pval;
  const int32_t* pid;
  int ntiles;
  const float* pfmax;           // optional: per-tile largest allowed logit (filters active)
};

hipError_t beam_init(const BeamParams& p, int bos, hipStream_t st);
hipError_t beam_step(const BeamParams& p, const GenPartials& gp, int t, hipStream_t st);
hipError_t backtrack(const BeamParams& p, int32_t* out_tok, int32_t* out_len, double* out_raw, double* out_norm,
                     float* out_tok_logp, int32_t* out_align, hipStream_t st);

// out [B, T] = the source id at the aligned position of every UNK output token (t < len[b]), -1 elsewhere.
hipError_t replace_unk(const int32_t* src, int B, int S, const int32_t* tok, const int32_t* len, const int32_t* align,
                       int T, int unk, int32_t* out, hipStream_t st);

// Device-side input validation (see beam.hip): error kinds recorded in the host-visible word.
enum { kErrLength = 1, kErrSourceId = 2, kErrToken = 3, kErrParent = 4 };
// clean [B, S] = src with ids past each length (and invalid ids) set to 0; lens [B] = len clamped to [1, S];
// rowmap [S, B] = b * S + s.
hipError_t sanitize_src(const int32_t* src, const int32_t* len, int B, int S, int V, int32_t* clean, int32_t* lens,
                        int32_t* rowmap, int32_t* err, hipStream_t st);
// tok_out [N] = tok with invalid ids set to 0; par_out [N] (when parent != NULL) = parent with rows outside
// [0, N) replaced by the row itself.
hipError_t sanitize_step(const int32_t* tok, const int32_t* parent, int N, int V, int32_t* tok_out, int32_t* par_out,
                         int32_t* err, hipStream_t st);

hipError_t replicate_rows(const float* src, int ld_src, int rows, int K, float* dst, int ld_dst, int ncols,
                          hipStream_t st);
// hi / lo / lo2 [rows, ld_dst] = the bf16 term planes of src [rows, ld_src] columns < cols, zeros in
// columns cols .. ld_dst.
hipError_t split_rows(const float* src, int ld_src, int rows, int cols, uint16_t* hi, uint16_t* lo, uint16_t* lo2,
                      int ld_dst, hipStream_t st);
hipError_t fill_f32(float* dst, size_t n, float v, hipStream_t st);
hipError_t copy_cols(const float* src, int ld_src, float* dst, int ld_dst, int rows, int ncols, hipStream_t st);

}  // namespace onmt
