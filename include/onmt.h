/*
 * onmt.h — C interface of libonmt, batched beam-search translation with an attention-based LSTM
 * encoder-decoder on one AMD Instinct MI355X (gfx950).
 *
 * The model is the one the OpenNMT paper (Klein et al., arXiv 1805.11462) describes in Section 2
 * ("Background") and Figure 1(a): a conditional language model p(w_1:T | x) = prod_t p(w_t | w_<t, x)
 * computed by a stacked (optionally bidirectional, Tables 3-4) LSTM encoder, an input-feeding LSTM
 * decoder (Section 2 item (c)) with global attention of the general, dot or concat type (Section 4.2),
 * a softmax generator and beam search with length normalisation (Section 2 item (d); Section 4.2). The
 * paper's deployment section (Section 4.1, "C/Mobile/GPU Translation") describes a batched GPU
 * translator and a C implementation; this library is that translator behind a C ABI.
 *
 * Where the paper is silent the library follows these readings: forget-gate LSTM without peepholes,
 * one bias per gate, gate order (i, f, g, o); zero initial encoder state; no source BOS/EOS; packed
 * padding (pads never update state, memory is 0 and attention weight exactly 0 at pads);
 * bidirectional final state [forward after last token ; backward after token 0]; scores without
 * biases (general q^T W_a m_s, dot q^T m_s, concat v_a^T tanh(W_a [q ; m_s])); attentional vector
 * tanh(W_c [ctx ; q]) without bias; input feed starts at 0 and the first decoder layer sees
 * [embedding ; feed]; generator with bias, nothing masked.
 *
 * Conventions for every function:
 *   - Return 0 (ONMT_OK) or a negative error code; never throw or abort. onmt_last_error() gives a
 *     thread-local message for the last failure.
 *   - All size and id checks happen before any compute is enqueued. On error no kernel has been
 *     launched and output buffers are unspecified. (With ONMT_VALIDATE_DEVICE, ids and lengths are
 *     instead checked by a kernel on the stream; see "Input validation".)
 *   - The caller owns all device memory: it allocates the buffers whose sizes the *_bytes queries
 *     return and passes device pointers. The library never allocates device memory (the allocation-free
 *     decoder step uses a scratch array built into the library).
 *   - `stream` is a hipStream_t (NULL = default stream). Work is ordered on that stream.
 *   - Matrices are row-major. Beam rows are numbered r = b * K + k (sentence b, slot k).
 *   - A model handle is not thread-safe; separate handles are independent.
 */
#ifndef ONMT_H
#define ONMT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ONMT_OK = 0,
  ONMT_EINVAL = -1,       /* bad argument: null pointer, out-of-range id/length/size */
  ONMT_ESIZE = -2,        /* a device buffer is smaller than the matching *_bytes query */
  ONMT_EDEVICE = -3,      /* a HIP runtime call failed */
  ONMT_EUNSUPPORTED = -4  /* valid but outside what the kernels support (e.g. beam > 16) */
};

/* Model shape. enc_layers must equal dec_layers (the decoder starts from the encoder's final states,
 * Figure 1(a)). When bidirectional, each encoder direction has hidden/2 units and their outputs are
 * concatenated, so the memory width is `hidden` either way. emb and hidden (and hidden/2 when
 * bidirectional) must be multiples of 4; with wdtype = 1 emb must be a multiple of 8. Kernel limits
 * (ONMT_EUNSUPPORTED beyond them): tgt_vocab <= 131072; the decoder calls need hidden <= 1024. */
typedef struct {
  int enc_layers, dec_layers, bidirectional;
  int emb, hidden;
  int src_vocab, tgt_vocab;
  int wdtype;                      /* 0 = fp32 weights and fp32-accurate products (the vocabulary
                                      projection runs them as six bf16 term products of three-term
                                      splits of both operands, accumulated in fp32); 1 = bf16 weights
                                      and MFMA operands (activations as bf16 terms), fp32 accumulation,
                                      cell state and softmax */
  int pad_id, unk_id, bos_id, eos_id;
  int attn_type;                   /* attention score (Section 4.2 names three types, none with biases):
                                      ONMT_ATTN_GENERAL e_s = q . W_a m_s;
                                      ONMT_ATTN_DOT     e_s = q . m_s;
                                      ONMT_ATTN_CONCAT  e_s = v_a . tanh(W_a [q ; m_s]) */
} onmt_config;

enum { ONMT_ATTN_GENERAL = 0, ONMT_ATTN_DOT = 1, ONMT_ATTN_CONCAT = 2 };

/* Beam search settings (Section 2 item (d); Section 4.2 length and attention coverage normalisation,
 * GNMT forms lp(n) = ((5 + n) / 6)^alpha and cp = beta * sum over the real source positions i of
 * log(min(c_i, 1)), c_i = attention on position i summed over the hypothesis's steps). max_len counts
 * generated tokens including EOS. beta >= 0 (0 = no coverage penalty). Every check_every steps (<= 0:
 * every step when max_len <= 32, else every 8) the "all sentences finished" counter is copied to the host
 * without waiting; the host then waits for the previous such copy and stops when it shows every sentence
 * finished, so a finished batch runs at most one check period of extra steps (which change no output). */
typedef struct {
  int beam;
  int max_len;
  double alpha;
  int check_every;
  double beta;
  /* Hypothesis filters (Section 4.2 names limits on unknown words and word-level constraints on the
   * search): a candidate whose token is one of banned[0 .. n_banned) (host array, ids in
   * [0, tgt_vocab)), or an unk_id beyond max_unk UNKs of its hypothesis (max_unk < 0: no limit), is not
   * a candidate; log-probs stay normalised over the whole vocabulary. */
  int max_unk;
  const int32_t* banned;
  int n_banned;
} onmt_search_params;

/* Optional per-step record of the search, device pointers, each [max_len, B, beam] by rank:
 * slot = parent slot of the chosen candidate (-1 = none), tok = chosen token, cand = its fp64
 * score (parent score + log-prob). steps[B] = step after which the sentence finished. */
typedef struct {
  int32_t* slot;
  int32_t* tok;
  double* cand;
  int32_t* steps;
} onmt_trace;

typedef struct onmt_model onmt_model;

const char* onmt_last_error(void);

/* Number of host weight arrays onmt_model_create expects, and the element count of array i, in this
 * order: E_src [src_vocab, emb]; for each encoder layer l and direction (forward, then backward when
 * bidirectional): W [4*Hd, in + Hd] (gate row blocks i, f, g, o; columns [input | recurrent]) and
 * b [4*Hd], with Hd = hidden (/2 if bidirectional) and in = emb for l = 0, hidden above; E_tgt
 * [tgt_vocab, emb]; for each decoder layer l: W [4*hidden, in + hidden] with in = emb + hidden for
 * l = 0 (columns [embedding | input feed | recurrent]) and hidden above, b [4*hidden];
 * attention score weights: general W_a [hidden, hidden], dot none, concat W_a [hidden, 2*hidden]
 * (columns [decoder state | memory]) then v_a [hidden]; W_c [hidden, 2*hidden] (columns
 * [context | decoder state]);
 * W_s [tgt_vocab, hidden]; b_s [tgt_vocab]. Returns < 0 for an invalid config. */
int onmt_num_weights(const onmt_config* cfg);
int64_t onmt_weight_numel(const onmt_config* cfg, int i);

/* Device bytes for the packed weights of `cfg` (0 for an invalid config). */
size_t onmt_model_bytes(const onmt_config* cfg);

/* Validate cfg, copy and pack the host fp32 weights (order above; the host arrays may be freed when the
 * call returns) into dev_buf, which must hold onmt_model_bytes(cfg) bytes, 256-byte aligned, and stay
 * allocated while the model lives. With wdtype = 1 weights are rounded to bf16 (nearest, ties to even).
 * Synchronizes `stream`. On success *out receives a handle that owns host metadata only. */
int onmt_model_create(const onmt_config* cfg, const float* const* host_weights, int n_weights, void* dev_buf,
                      size_t dev_bytes, void* stream, onmt_model** out);
int onmt_model_destroy(onmt_model* model);

/* ---- Encoder (Section 2: encoder RNN over word vectors; Figure 1(a)) -------------------------------
 * src [B, S_max] int32 token ids (device), len [B] int32 true lengths (device), 1 <= len[b] <= S_max,
 * ids in [0, src_vocab). Positions >= len[b] are ignored. Writes the memory bank, the attention keys
 * (general: W_a m_s; concat: the memory columns of W_a times m_s; dot: none, the scores read the
 * memory) and the final states into enc_ws (>= onmt_encode_ws_bytes(model, B, S_max)), which the
 * decoder calls then read. With host validation (the default) src and len are copied to the host and
 * checked (one stream sync), then the encoder is enqueued asynchronously; with device validation nothing
 * waits. The GEMMs read operands through 2 GiB buffer descriptors: a batch whose memory bank
 * (B * S_max rows of the memory width padded to 128 columns, fp32) or decoder state rows (B * beam rows)
 * would reach 2 GiB is refused with ONMT_EUNSUPPORTED, as is a model whose embedding table or packed
 * weight matrix would (onmt_num_weights / onmt_model_bytes report it), and scoring over B * T_max rows. */
size_t onmt_encode_ws_bytes(const onmt_model* model, int B, int S_max);
int onmt_encode(onmt_model* model, const int32_t* src, const int32_t* len, int B, int S_max, void* enc_ws,
                size_t enc_ws_bytes, void* stream);

/* ---- Decoder step: one evaluation of p(w_t | w_<t, x) for N = B*K rows (Section 2; Figure 1(a)) ----
 * A decoder state buffer holds, fp32: h [dec_layers, N, hidden], c [dec_layers, N, hidden],
 * feed [N, hidden] (the previous attentional vector), in that order, onmt_state_bytes(model, N) bytes.
 *
 * onmt_decode_init writes into state_out the decoder's initial state: every layer's (h, c) from the
 * encoder's final step of sentence b = r / K, and feed = 0.
 *
 * onmt_decode_step reads row parent[r] of state_in (parent NULL = row r) and prev_tok[r] (ids in
 * [0, tgt_vocab); parent in [0, N)), runs the decoder layers, attention over sentence r / K's memory,
 * the attentional vector and the generator, and writes row r of state_out (state_in != state_out).
 *   mode 0 (full):  logp [N, tgt_vocab] = log-softmax of the logits; ids unused (may be NULL).
 *   mode 1 (top-K): logp [N, K] and ids [N, K] = the K largest log-probs of each row, larger first,
 *                   smaller id on ties.
 *   lse [N] (optional) = logsumexp of each row's logits. attn [N, S_max] (optional) = attention weights,
 *   exactly 0 at pads.
 * step_ws holds onmt_step_ws_bytes(model, B, S_max, K) bytes of scratch. With host validation (the default)
 * prev_tok and parent are copied to the host and checked (one stream sync), then the compute is enqueued
 * asynchronously; with device validation (onmt_set_validation below) nothing waits. */
size_t onmt_state_bytes(const onmt_model* model, int N);
size_t onmt_step_ws_bytes(const onmt_model* model, int B, int S_max, int K);
int onmt_decode_init(onmt_model* model, const void* enc_ws, int B, int S_max, int K, void* state_out,
                     void* stream);
int onmt_decode_step(onmt_model* model, const void* enc_ws, int B, int S_max, int K, const void* state_in,
                     void* state_out, const int32_t* prev_tok, const int32_t* parent, int mode, float* logp,
                     int32_t* ids, float* lse, float* attn, void* step_ws, size_t step_ws_bytes, void* stream);

/* ---- Input validation ---------------------------------------------------------------------------------
 * ONMT_VALIDATE_HOST (the default): onmt_encode, onmt_decode_step and onmt_beam_search copy their device
 * id / length inputs to the host and check them before enqueuing anything, returning ONMT_EINVAL on a bad
 * value (one stream sync per call). ONMT_VALIDATE_DEVICE: a kernel enqueued on the stream checks them
 * instead, so the call does not wait for the device; a bad value is replaced by a safe one (a length
 * clamped to [1, S_max], an id by 0, a parent by the row itself), the computation goes on, and the model
 * records the failure. In this mode the encoder steps over all S_max positions (the host does not learn
 * the longest length), which gives the same results. onmt_device_status sets *code to ONMT_OK or
 * ONMT_EINVAL (onmt_last_error then says what was wrong) for the work enqueued since its last call and
 * clears the record; call it after synchronizing the stream(s) the work ran on. It does not synchronize. */
enum { ONMT_VALIDATE_HOST = 0, ONMT_VALIDATE_DEVICE = 1 };
int onmt_set_validation(onmt_model* model, int mode);
int onmt_device_status(onmt_model* model, int* code);

/* ---- Decoder step without allocation ------------------------------------------------------------------
 * For callers that cannot allocate memory or synchronize per call (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): onmt_decode_step without the step_ws argument. Its
 * scratch (what step_ws holds) is a device array of ONMT_NOALLOC_SCRATCH_BYTES built into the library,
 * one per GPU, located when a model is created on that device (or at the first call on it); the call
 * itself allocates nothing and never waits. Inputs are validated on the device as with
 * ONMT_VALIDATE_DEVICE (check onmt_device_status). A step whose onmt_step_ws_bytes(model, B, S_max, K)
 * exceeds ONMT_NOALLOC_SCRATCH_BYTES is refused with ONMT_EUNSUPPORTED (16 MiB holds every workload of
 * this library's benchmarks: 320 rows over a 50000-word vocabulary at beam 5 take 7.3 MB). All calls on
 * one GPU share its array, which keeps the last call's contents: calls that overlap on one GPU (on
 * different streams, or from different threads) race and must not be issued. Arguments, outputs and
 * error codes are those of onmt_decode_step. */
#define ONMT_NOALLOC_SCRATCH_BYTES (16u << 20)
int onmt_decode_step_noalloc(onmt_model* model, const void* enc_ws, int B, int S_max, int K, const void* state_in,
                             void* state_out, const int32_t* prev_tok, const int32_t* parent, int mode, float* logp,
                             int32_t* ids, float* lse, float* attn, void* stream);

/* ---- Beam search (Section 2 item (d); Section 4.2; Section 4.1 batched GPU translator) --------------
 * Translates B sentences with beam width K = params->beam (1 <= K <= 16, K <= tgt_vocab). Per sentence:
 * slot scores start [0, -inf, ...] with input BOS; each step scores cand = s_k + logp_k(w) in fp64 and
 * keeps the K best (larger first, smaller k*V + w on ties); a chosen EOS, or any choice at step
 * max_len, enters the finished pool with norm = cand / lp(t) + cp (cp over the attention of the
 * hypothesis's steps, this one included); the others become the next live slots in
 * rank order. A sentence stops at max_len, when no live slot remains, or when the pool's best norm is
 * >= best live score / lp(max_len) (no descendant can beat it). The result is the pool entry with the
 * largest norm (earlier step, then better rank, on ties).
 * Outputs (device pointers): out_tok [B, max_len] (BOS excluded, EOS included if chosen, pad_id after
 * the end), out_len [B], out_raw [B] (sum of log-probs), out_norm [B], out_tok_logp [B, max_len]
 * (optional; 0 after the end), out_align [B, max_len] (optional; for every output token the source
 * position with the largest attention weight of its step, smaller position on ties, -1 after the end:
 * the alignment for unknown-word replacement, Section 4.2 OOV handling), trace (optional). ws holds
 * onmt_search_ws_bytes(...) bytes. src/len as in onmt_encode. Returns when the outputs are written (the
 * stream is synchronized). */
size_t onmt_search_ws_bytes(const onmt_model* model, int B, int S_max, const onmt_search_params* params);
int onmt_beam_search(onmt_model* model, const int32_t* src, const int32_t* len, int B, int S_max,
                     const onmt_search_params* params, void* ws, size_t ws_bytes, int32_t* out_tok,
                     int32_t* out_len, double* out_raw, double* out_norm, float* out_tok_logp,
                     int32_t* out_align, const onmt_trace* trace, void* stream);

/* ---- Unknown-word replacement (Section 4.2 OOV handling, after Luong et al. 2015b) -------------------
 * For the outputs of onmt_beam_search run with out_align: out_src[b, t] = src[b, out_align[b, t]] for every
 * output token t < out_len[b] that is the model's unk_id (the source word at the position the UNK's step
 * attended to most), -1 for every other entry. A bilingual dictionary would map that source id to a target
 * word; without one the caller copies it. src [B, S_max] as given to the search; out_tok, out_align,
 * out_src [B, max_len]; all device pointers. Asynchronous on the stream; alignments outside [0, S_max) give
 * -1. */
int onmt_replace_unk(onmt_model* model, const int32_t* src, int B, int S_max, const int32_t* out_tok,
                     const int32_t* out_len, const int32_t* out_align, int max_len, int32_t* out_src, void* stream);

/* ---- Teacher-forced scoring: the training objective's per-token terms (Section 2: the model is trained
 * to minimise the negative log-likelihood of the corpus; the same conditional factorisation) ----------
 * For sentence b the decoder is fed BOS, tgt[b, 0], ..., tgt[b, tgt_len[b] - 2] and scores the next target
 * token at every step: out_logp[b, t] = log p(tgt[b, t] | tgt[b, <t], src_b) for t < tgt_len[b], 0 after;
 * out_nll[b] = -sum_t out_logp[b, t] (fp64). tgt [B, T_max] and tgt_len [B] are device int32 arrays
 * (1 <= tgt_len[b] <= T_max, ids in [0, tgt_vocab) below the length); they are copied to the host for
 * validation. src/len as in onmt_encode. ws holds onmt_score_ws_bytes(model, B, S_max, T_max) bytes.
 * out_logp [B, T_max] fp32 and out_nll [B] fp64 are device pointers. Returns when the outputs are
 * written (the stream is synchronized). */
size_t onmt_score_ws_bytes(const onmt_model* model, int B, int S_max, int T_max);
int onmt_score(onmt_model* model, const int32_t* src, const int32_t* len, int B, int S_max, const int32_t* tgt,
               const int32_t* tgt_len, int T_max, void* ws, size_t ws_bytes, float* out_logp, double* out_nll,
               void* stream);

/* ---- Kernel timing -----------------------------------------------------------------------------------
 * onmt_profile_enable(model, every, kinds): every >= 1 makes onmt_beam_search and onmt_score record HIP
 * events on `stream` around every `every`-th launch of each kind of kernel below whose bit
 * (1 << ONMT_KERNEL_*) is set in `kinds` (counting launches of each kind from this call); every = 0
 * switches timing off; every < 0, or kinds outside ONMT_KERNEL_ALL, is ONMT_EINVAL. Kinds: the generator (the vocabulary
 * projection with its fused log-softmax/top-K epilogue; the search launches it once per step, scoring
 * once over all steps), a decoder LSTM layer (GEMM with the gate/cell epilogue), the attention (scores
 * and context launches together), the attentional output tanh(W_c [ctx ; q]), and the beam step (search
 * only). onmt_profile_read_kernel returns how many launches of `kind` were timed and their summed
 * duration in milliseconds since its last reset; onmt_profile_read does so for the generator. Each timed
 * launch adds two event records to the stream. */
enum { ONMT_KERNEL_GENERATOR = 0, ONMT_KERNEL_LSTM = 1, ONMT_KERNEL_ATTENTION = 2, ONMT_KERNEL_OUTPUT = 3,
       ONMT_KERNEL_BEAM = 4, ONMT_KERNEL_KINDS = 5, ONMT_KERNEL_ALL = (1 << 5) - 1 };
int onmt_profile_enable(onmt_model* model, int every, unsigned kinds);
int onmt_profile_read(onmt_model* model, int* n_launches, double* total_ms, int reset);
int onmt_profile_read_kernel(onmt_model* model, int kind, int* n_launches, double* total_ms, int reset);

#ifdef __cplusplus
}
#endif

#endif /* ONMT_H */
