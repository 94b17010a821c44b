// C ABI of libonmt: validation, weight packing, workspace carving and the encode / decode-step /
// beam-search orchestration. All arithmetic runs in the kernels of gemm.hip, attention.hip and beam.hip.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/onmt.h"
#include "common.h"
#include "kernels.h"

using namespace onmt;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                              \
  do {                                                                                             \
    hipError_t e_ = (expr);                                                                        \
    if (e_ != hipSuccess) return fail(ONMT_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_));       \
  } while (0)

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }
inline int ceil_to(int x, int m) { return (x + m - 1) / m * m; }

// Byte-offset allocator over a caller-provided buffer (used for sizing with base == 0, then carving).
struct Carver {
  size_t off = 0;
  char* base = nullptr;
  template <class T>
  T* take(size_t count) {
    off = align_up(off);
    T* p = base ? (T*)(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

struct Packed {      // packed weight matrix inside the model buffer
  const void* W = nullptr;
  int Np = 0, Kp = 0;
  size_t off = 0;
};

Seg seg(const void* base, const int32_t* idx, int rows, int ld, int width, int kpad, int bf16) {
  Seg s;
  s.base = base;
  s.idx = idx;
  s.rows = rows;
  s.ld = ld;
  s.width = width;
  s.kpad = kpad;
  s.bf16 = bf16;
  s.lo = nullptr;
  s.lo2 = nullptr;
  return s;
}

BOp bop(const Packed& p) {
  BOp b;
  b.W = p.W;
  b.Np = p.Np;
  b.Kp = p.Kp;
  return b;
}

struct Dims {
  int L, ndir, Hd, Hm, H, E, Vs, Vt;
  int Hd_pad, H_pad;   // units padded to multiples of 32 (gate-blocked groups, 128-column tiles)
  bool bf16;
  int esz;             // operand element size
  int attn;            // ONMT_ATTN_GENERAL / _DOT / _CONCAT
  // The generator's weights packed K-blocked as gwp bf16 term planes (bf16 models: 1, their exact values;
  // fp32 models: 3, each fp32 value as the sum of three bf16 terms, multiplied in six term products),
  // read with the attentional vector's term planes (split by the W_c epilogue). fp32 models also keep
  // the fp32 matrix for the row counts where the fp32 MFMA kernel is faster (gemm_gen_split_rows).
  int gwp;
  // Every K segment of a GEMM operand is padded to a multiple of kSegK so that no K stage of any tile
  // shape straddles two segments.
  int pad(int w) const { return ceil_to(w, kSegK); }
};

bool dims_of(const onmt_config* c, Dims* d) {
  if (!c) return false;
  d->L = c->enc_layers;
  d->ndir = c->bidirectional ? 2 : 1;
  d->H = c->hidden;
  d->Hd = c->bidirectional ? c->hidden / 2 : c->hidden;
  d->Hm = d->ndir * d->Hd;
  d->E = c->emb;
  d->Vs = c->src_vocab;
  d->Vt = c->tgt_vocab;
  d->Hd_pad = ceil_to(d->Hd, 32);
  d->H_pad = ceil_to(d->H, 32);
  d->bf16 = c->wdtype == 1;
  d->esz = d->bf16 ? 2 : 4;
  d->attn = c->attn_type;
  d->gwp = d->bf16 ? 1 : 3;
  return true;
}

// The GEMMs address their operands through buffer descriptors, whose byte counts and row offsets are
// 32-bit and which treat offsets from 2 GiB on as "no row" (zeros): every operand read that way must be
// smaller than 2 GiB. These checks run before anything is enqueued.
constexpr uint64_t kDescLimit = 1ull << 31;
size_t model_layout(const onmt_config* c, onmt_model* m, std::vector<uint64_t>* mats = nullptr);

int check_model_limits(const onmt_config* c) {
  std::vector<uint64_t> mats;
  model_layout(c, nullptr, &mats);   // embeddings, packed LSTM / attention / generator matrices
  for (uint64_t b : mats)
    if (b >= kDescLimit)
      return fail(ONMT_EUNSUPPORTED, "a packed weight matrix or embedding table needs %llu bytes (limit 2 GiB)",
                  (unsigned long long)b);
  return ONMT_OK;
}

int check_config(const onmt_config* c) {
  if (!c) return fail(ONMT_EINVAL, "config is NULL");
  if (c->enc_layers < 1 || c->dec_layers < 1) return fail(ONMT_EINVAL, "layers must be >= 1");
  if (c->enc_layers != c->dec_layers)
    return fail(ONMT_EINVAL, "enc_layers (%d) must equal dec_layers (%d)", c->enc_layers, c->dec_layers);
  if (c->bidirectional != 0 && c->bidirectional != 1) return fail(ONMT_EINVAL, "bidirectional must be 0 or 1");
  if (c->wdtype != 0 && c->wdtype != 1) return fail(ONMT_EINVAL, "wdtype must be 0 (fp32) or 1 (bf16)");
  if (c->attn_type < ONMT_ATTN_GENERAL || c->attn_type > ONMT_ATTN_CONCAT)
    return fail(ONMT_EINVAL, "attn_type must be 0 (general), 1 (dot) or 2 (concat)");
  if (c->emb < 4 || c->hidden < 4 || c->src_vocab < 1 || c->tgt_vocab < 4)
    return fail(ONMT_EINVAL, "emb/hidden >= 4, src_vocab >= 1, tgt_vocab >= 4 required");
  if (c->emb > 8192 || c->hidden > 8192 || c->enc_layers > 64) return fail(ONMT_EUNSUPPORTED, "model too large");
  if (c->tgt_vocab > 131072) return fail(ONMT_EUNSUPPORTED, "target vocabulary larger than 131072");
  const int Hd = c->bidirectional ? c->hidden / 2 : c->hidden;
  if (c->bidirectional && c->hidden % 2) return fail(ONMT_EINVAL, "bidirectional needs an even hidden size");
  if (c->emb % 4 || c->hidden % 4 || Hd % 4)
    return fail(ONMT_EUNSUPPORTED, "emb, hidden and per-direction hidden must be multiples of 4");
  if (c->wdtype == 1 && c->emb % 8) return fail(ONMT_EUNSUPPORTED, "bf16 models need emb a multiple of 8");
  const int ids[4] = {c->pad_id, c->unk_id, c->bos_id, c->eos_id};
  for (int i = 0; i < 4; ++i)
    if (ids[i] < 0 || ids[i] >= c->tgt_vocab) return fail(ONMT_EINVAL, "special ids must be in [0, tgt_vocab)");
  return check_model_limits(c);
}

struct WeightSpec {
  int64_t rows, cols;   // cols = 1 for vectors
};

std::vector<WeightSpec> weight_specs(const onmt_config* c) {
  Dims d;
  dims_of(c, &d);
  std::vector<WeightSpec> v;
  v.push_back({d.Vs, d.E});
  for (int l = 0; l < d.L; ++l) {
    const int in = l == 0 ? d.E : d.Hm;
    for (int dir = 0; dir < d.ndir; ++dir) {
      v.push_back({4LL * d.Hd, in + d.Hd});
      v.push_back({4LL * d.Hd, 1});
    }
  }
  v.push_back({d.Vt, d.E});
  for (int l = 0; l < d.L; ++l) {
    const int in = l == 0 ? d.E + d.H : d.H;
    v.push_back({4LL * d.H, in + d.H});
    v.push_back({4LL * d.H, 1});
  }
  if (d.attn == ONMT_ATTN_GENERAL) v.push_back({d.H, d.Hm});
  if (d.attn == ONMT_ATTN_CONCAT) {
    v.push_back({d.H, d.H + d.Hm});
    v.push_back({d.H, 1});
  }
  v.push_back({d.H, d.Hm + d.H});
  v.push_back({d.Vt, d.H});
  v.push_back({d.Vt, 1});
  return v;
}

// Row of packed gate-blocked matrices for (gate, unit): groups of kUnitGroup units hold 4 gates x kUnitGroup rows.
inline int gate_row(int gate, int unit) {
  return (unit / kUnitGroup) * (4 * kUnitGroup) + gate * kUnitGroup + unit % kUnitGroup;
}

}  // namespace

struct onmt_model {
  onmt_config cfg;
  Dims d;
  char* dev = nullptr;
  const void* E_src = nullptr;
  const void* E_tgt = nullptr;
  // Encoder. Bidirectional: every layer has an input projection (both directions stacked) and a recurrent
  // matrix per direction. Unidirectional: layer 0 likewise; layers >= 1 keep [input | recurrent] in one
  // matrix, so that they can run one timestep behind the layer below in the same launch.
  std::vector<Packed> enc_x;               // per layer: both directions stacked [ndir * 4 Hd_pad, pad(in)]
  std::vector<const float*> enc_bias;      // per layer [ndir * 4 Hd_pad]
  std::vector<Packed> enc_h;               // per layer * ndir: [4 Hd_pad, pad(Hd)]
  std::vector<Packed> enc_xh;              // unidirectional layers >= 1: [4 Hd_pad, pad(in) + pad(Hd)]
  std::vector<Packed> dec_w;               // per layer [4 H_pad, sum of padded segment widths]
  std::vector<const float*> dec_bias;      // per layer [4 H_pad]
  Packed W_a;                              // memory side of the score: general W_a, concat's memory columns
  Packed W_q;                              // concat: the query columns of W_a
  const float* v_a = nullptr;              // concat [H]
  Packed W_c, W_s;
  Packed W_s32;        // fp32 models: the generator's fp32 weights, row-major
  const float* b_s = nullptr;
  // decoder layer 0's input-projection rows for every target token, E_tgt[v] W_e^T in the packed (gate-
  // blocked) column order, fp32 [Vt, 4 H_pad]; computed on the device when the model is created
  float* emb_gates = nullptr;
  size_t image_bytes = 0;    // the uploaded part of the model buffer (everything before emb_gates)
  // kernel timing
  int prof = 0;              // time every prof-th generator launch (0: off)
  unsigned prof_kinds = 0;                      // bit k: launches of kind k are timed
  long long prof_seq[ONMT_KERNEL_KINDS] = {};   // launches of each kind seen while timing is on
  bool prof_open[ONMT_KERNEL_KINDS] = {};       // the current launch of the kind has a start event
  size_t prof_pair[ONMT_KERNEL_KINDS] = {};     // ... recorded as event pair ev[prof_pair], ev[prof_pair + 1]
  int prof_n[ONMT_KERNEL_KINDS] = {};
  double prof_ms[ONMT_KERNEL_KINDS] = {};
  std::vector<hipEvent_t> ev;   // reusable start/stop pairs
  std::vector<int> ev_kind;     // kind of each recorded pair
  size_t ev_used = 0;
  // finish checks of the beam search: two pinned host words the done count is copied into, one event each
  int32_t* done_host = nullptr;
  hipEvent_t done_ev[2] = {nullptr, nullptr};
  // input validation: ONMT_VALIDATE_HOST or ONMT_VALIDATE_DEVICE; the device checks report into err_host
  // (pinned host memory, written by the validation kernels, read by onmt_device_status)
  int validation = ONMT_VALIDATE_HOST;
  int32_t* err_host = nullptr;
};

namespace {

// Model buffer layout (offsets only); fills m's offsets when m != nullptr, and the byte size of every
// matrix the GEMMs read through buffer descriptors into *mats when given.
size_t model_layout(const onmt_config* c, onmt_model* m, std::vector<uint64_t>* mats) {
  Dims d;
  dims_of(c, &d);
  Carver cv;
  auto mat = [&](int Np, int Kp) {
    Packed p;
    cv.off = align_up(cv.off);
    p.off = cv.off;
    p.Np = Np;
    p.Kp = Kp;
    cv.off += (size_t)Np * Kp * d.esz;
    if (mats) mats->push_back((uint64_t)Np * Kp * d.esz);
    return p;
  };
  auto vec = [&](size_t n) {
    cv.off = align_up(cv.off);
    size_t o = cv.off;
    cv.off += n * sizeof(float);
    return o;
  };
  Packed esrc = mat(d.Vs, d.E);
  std::vector<Packed> ex, eh, exh, dw;
  std::vector<size_t> eb, db;
  for (int l = 0; l < d.L; ++l) {
    const int in = l == 0 ? d.E : d.Hm;
    if (d.ndir == 1 && l > 0) {
      ex.push_back(Packed{});
      eh.push_back(Packed{});
      exh.push_back(mat(4 * d.Hd_pad, d.pad(in) + d.pad(d.Hd)));
    } else {
      ex.push_back(mat(d.ndir * 4 * d.Hd_pad, d.pad(in)));
      for (int dir = 0; dir < d.ndir; ++dir) eh.push_back(mat(4 * d.Hd_pad, d.pad(d.Hd)));
      exh.push_back(Packed{});
    }
    eb.push_back(vec((size_t)d.ndir * 4 * d.Hd_pad));
  }
  Packed etgt = mat(d.Vt, d.E);
  for (int l = 0; l < d.L; ++l) {
    const int kp = l == 0 ? d.pad(d.E) + 2 * d.pad(d.H) : 2 * d.pad(d.H);
    dw.push_back(mat(4 * d.H_pad, kp));
    db.push_back(vec((size_t)4 * d.H_pad));
  }
  Packed wa = d.attn != ONMT_ATTN_DOT ? mat(ceil_to(d.H, 128), d.pad(d.Hm)) : Packed{};
  Packed wq = d.attn == ONMT_ATTN_CONCAT ? mat(ceil_to(d.H, 128), d.pad(d.H)) : Packed{};
  const size_t va = d.attn == ONMT_ATTN_CONCAT ? vec(d.H) : 0;
  Packed wc = mat(ceil_to(d.H, 128), d.pad(d.Hm) + d.pad(d.H));
  Packed ws;         // K-blocked bf16 planes, each read through its own descriptor
  cv.off = align_up(cv.off);
  ws.off = cv.off;
  ws.Np = ceil_to(d.Vt, 128);
  ws.Kp = d.pad(d.H);
  const uint64_t plane = (uint64_t)ws.Np * ws.Kp * 2;
  cv.off += plane * d.gwp;
  if (mats) mats->push_back(plane);
  Packed ws32 = d.bf16 ? Packed{} : mat(ceil_to(d.Vt, 128), d.pad(d.H));
  size_t bs = vec(ceil_to(d.Vt, 128));
  const size_t image = align_up(cv.off);
  const size_t eg = vec((size_t)d.Vt * 4 * d.H_pad);
  const size_t total = align_up(cv.off);
  if (m) {
    char* base = m->dev;
    auto fix = [&](Packed p) {
      p.W = base + p.off;
      return p;
    };
    m->E_src = base + esrc.off;
    m->E_tgt = base + etgt.off;
    for (auto& p : ex) m->enc_x.push_back(fix(p));
    for (auto o : eb) m->enc_bias.push_back((const float*)(base + o));
    for (auto& p : eh) m->enc_h.push_back(fix(p));
    for (auto& p : exh) m->enc_xh.push_back(fix(p));
    for (auto& p : dw) m->dec_w.push_back(fix(p));
    for (auto o : db) m->dec_bias.push_back((const float*)(base + o));
    if (d.attn != ONMT_ATTN_DOT) m->W_a = fix(wa);
    if (d.attn == ONMT_ATTN_CONCAT) {
      m->W_q = fix(wq);
      m->v_a = (const float*)(base + va);
    }
    m->W_c = fix(wc);
    m->W_s = fix(ws);
    if (!d.bf16) m->W_s32 = fix(ws32);
    m->b_s = (const float*)(base + bs);
    m->emb_gates = (float*)(base + eg);
    m->image_bytes = image;
  }
  return total;
}

// Host-side packing into the image of the device buffer.
struct HostImage {
  std::vector<char> buf;
  bool bf16;
  void put(size_t off, size_t idx, float v) {
    if (bf16) {
      ((uint16_t*)(buf.data() + off))[idx] = f32_to_bf16_bits(v);
    } else {
      ((float*)(buf.data() + off))[idx] = v;
    }
  }
  void putf(size_t off, size_t idx, float v) { ((float*)(buf.data() + off))[idx] = v; }
};

// Copy columns [c0, c0 + w) of src rows into packed row `prow` at packed column pc0.
void pack_row(HostImage& img, const Packed& p, int prow, int pc0, const float* src_row, int c0, int w) {
  for (int j = 0; j < w; ++j) img.put(p.off, (size_t)prow * p.Kp + pc0 + j, src_row[c0 + j]);
}

}  // namespace

// ====================================================================== allocation-free step scratch

// Scratch of onmt_decode_step_noalloc: the step workspace of one decoder step (attention scores and
// context, generator partials, checked ids), a file-scope device array instead of a caller's buffer. Each
// GPU holds its own copy, at its own address, until the process ends. In host code `scratch` names a
// host-side stand-in, never the device memory: kernels get the address hipGetSymbolAddress returns for
// the current device, kept per device below.
static __device__ __align__(256) char scratch[ONMT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device (at onmt_model_create, the
// library's set-up call, or at the entry point's first call on a device no model was created on).
int noalloc_scratch(void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(ONMT_EUNSUPPORTED, "device index %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(ONMT_EDEVICE, "no device address for the step scratch");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ONMT_OK;
}

}  // namespace

// ====================================================================== ABI

extern "C" {

const char* onmt_last_error(void) { return g_err.c_str(); }

int onmt_num_weights(const onmt_config* cfg) {
  int rc = check_config(cfg);
  if (rc) return rc;
  return (int)weight_specs(cfg).size();
}

int64_t onmt_weight_numel(const onmt_config* cfg, int i) {
  int rc = check_config(cfg);
  if (rc) return rc;
  auto v = weight_specs(cfg);
  if (i < 0 || i >= (int)v.size()) return fail(ONMT_EINVAL, "weight index %d out of range", i);
  return v[i].rows * v[i].cols;
}

size_t onmt_model_bytes(const onmt_config* cfg) {
  if (check_config(cfg)) return 0;
  return model_layout(cfg, nullptr);
}

int onmt_model_create(const onmt_config* cfg, const float* const* host_weights, int n_weights, void* dev_buf,
                      size_t dev_bytes, void* stream, onmt_model** out) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!out) return fail(ONMT_EINVAL, "out is NULL");
  *out = nullptr;
  auto specs = weight_specs(cfg);
  if (n_weights != (int)specs.size()) return fail(ONMT_EINVAL, "expected %d weight arrays, got %d", (int)specs.size(), n_weights);
  if (!host_weights) return fail(ONMT_EINVAL, "host_weights is NULL");
  for (int i = 0; i < n_weights; ++i)
    if (!host_weights[i]) return fail(ONMT_EINVAL, "host weight %d is NULL", i);
  if (!dev_buf) return fail(ONMT_EINVAL, "dev_buf is NULL");
  if ((uintptr_t)dev_buf % kAlign) return fail(ONMT_EINVAL, "dev_buf must be 256-byte aligned");
  const size_t need = model_layout(cfg, nullptr);
  if (dev_bytes < need) return fail(ONMT_ESIZE, "model buffer %zu bytes < %zu", dev_bytes, need);

  onmt_model* m = new onmt_model();
  m->cfg = *cfg;
  dims_of(cfg, &m->d);
  m->dev = (char*)dev_buf;
  model_layout(cfg, m);
  const Dims& d = m->d;

  HostImage img;
  img.bf16 = d.bf16;
  img.buf.assign(m->image_bytes, 0);
  auto off_of = [&](const void* p) { return (size_t)((const char*)p - m->dev); };
  int wi = 0;
  // E_src
  {
    const float* s = host_weights[wi++];
    const size_t o = off_of(m->E_src);
    for (size_t i = 0; i < (size_t)d.Vs * d.E; ++i) img.put(o, i, s[i]);
  }
  for (int l = 0; l < d.L; ++l) {
    const int in = l == 0 ? d.E : d.Hm;
    const size_t bo = off_of(m->enc_bias[l]);
    const bool joint = d.ndir == 1 && l > 0;
    for (int dir = 0; dir < d.ndir; ++dir) {
      const float* W = host_weights[wi++];
      const float* bvec = host_weights[wi++];
      for (int g = 0; g < 4; ++g)
        for (int u = 0; u < d.Hd; ++u) {
          const float* row = W + (size_t)(g * d.Hd + u) * (in + d.Hd);
          const int xr = dir * 4 * d.Hd_pad + gate_row(g, u);
          if (joint) {   // segments [layer below | recurrent]
            pack_row(img, m->enc_xh[l], xr, 0, row, 0, in);
            pack_row(img, m->enc_xh[l], xr, d.pad(in), row, in, d.Hd);
          } else {
            pack_row(img, m->enc_x[l], xr, 0, row, 0, in);
            pack_row(img, m->enc_h[l * d.ndir + dir], gate_row(g, u), 0, row, in, d.Hd);
          }
          img.putf(bo, xr, bvec[g * d.Hd + u]);
        }
    }
  }
  {
    const float* s = host_weights[wi++];
    const size_t o = off_of(m->E_tgt);
    for (size_t i = 0; i < (size_t)d.Vt * d.E; ++i) img.put(o, i, s[i]);
  }
  for (int l = 0; l < d.L; ++l) {
    const float* W = host_weights[wi++];
    const float* bvec = host_weights[wi++];
    const Packed& P = m->dec_w[l];
    const size_t bo = off_of(m->dec_bias[l]);
    const int in = l == 0 ? d.E + d.H : d.H;
    for (int g = 0; g < 4; ++g)
      for (int u = 0; u < d.H; ++u) {
        const float* row = W + (size_t)(g * d.H + u) * (in + d.H);
        const int pr = gate_row(g, u);
        if (l == 0) {   // segments [embedding | feed | recurrent]
          pack_row(img, P, pr, 0, row, 0, d.E);
          pack_row(img, P, pr, d.pad(d.E), row, d.E, d.H);
          pack_row(img, P, pr, d.pad(d.E) + d.pad(d.H), row, d.E + d.H, d.H);
        } else {        // segments [layer below | recurrent]
          pack_row(img, P, pr, 0, row, 0, d.H);
          pack_row(img, P, pr, d.pad(d.H), row, d.H, d.H);
        }
        img.putf(bo, pr, bvec[g * d.H + u]);
      }
  }
  {
    if (d.attn == ONMT_ATTN_GENERAL) {
      const float* Wa = host_weights[wi++];
      for (int r = 0; r < d.H; ++r) pack_row(img, m->W_a, r, 0, Wa + (size_t)r * d.Hm, 0, d.Hm);
    } else if (d.attn == ONMT_ATTN_CONCAT) {   // columns [query | memory]
      const float* Wa = host_weights[wi++];
      for (int r = 0; r < d.H; ++r) {
        pack_row(img, m->W_q, r, 0, Wa + (size_t)r * (d.H + d.Hm), 0, d.H);
        pack_row(img, m->W_a, r, 0, Wa + (size_t)r * (d.H + d.Hm), d.H, d.Hm);
      }
      const float* va = host_weights[wi++];
      const size_t vo = off_of(m->v_a);
      for (int r = 0; r < d.H; ++r) img.putf(vo, r, va[r]);
    }
    const float* Wc = host_weights[wi++];
    for (int r = 0; r < d.H; ++r) {
      pack_row(img, m->W_c, r, 0, Wc + (size_t)r * (d.Hm + d.H), 0, d.Hm);
      pack_row(img, m->W_c, r, d.pad(d.Hm), Wc + (size_t)r * (d.Hm + d.H), d.Hm, d.H);
    }
    const float* Ws = host_weights[wi++];
    {   // K-blocked bf16 term planes for the pre-split generator (see gemm_gen_split)
      const size_t Np = (size_t)m->W_s.Np, plane = Np * m->W_s.Kp;
      uint16_t* o = (uint16_t*)(img.buf.data() + m->W_s.off);
      for (int r = 0; r < d.Vt; ++r)
        for (int k = 0; k < d.H; ++k) {
          const size_t at = (size_t)(k / kGenKBlock) * Np * kGenKBlock + (size_t)r * kGenKBlock + k % kGenKBlock;
          float x = Ws[(size_t)r * d.H + k];
          for (int p = 0; p < d.gwp; ++p) {   // RNE of the value, then of each remainder
            const uint16_t t = f32_to_bf16_bits(x);
            o[p * plane + at] = t;
            x -= host_bf16_to_f32(t);
          }
        }
    }
    if (!d.bf16)
      for (int r = 0; r < d.Vt; ++r) pack_row(img, m->W_s32, r, 0, Ws + (size_t)r * d.H, 0, d.H);
    const float* bs = host_weights[wi++];
    const size_t bo = off_of(m->b_s);
    for (int r = 0; r < d.Vt; ++r) img.putf(bo, r, bs[r]);
  }
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(dev_buf, img.buf.data(), m->image_bytes, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) {
    // decoder layer 0: the embedding columns of its packed matrix against every target embedding row
    AOp a{};
    a.M = d.Vt;
    a.nseg = 1;
    a.seg[0] = seg(m->E_tgt, nullptr, d.Vt, d.E, d.E, d.pad(d.E), d.bf16);
    StoreParams sp{nullptr, m->emb_gates, 4 * d.H_pad, 4 * d.H_pad, 0};
    e = gemm_store(d.bf16, kShapeWide, a, bop(m->dec_w[0]), sp, st);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e == hipSuccess) {
    e = hipHostMalloc((void**)&m->err_host, sizeof(int32_t), hipHostMallocDefault);
    if (e == hipSuccess) *m->err_host = 0;
  }
  if (e != hipSuccess) {
    if (m->err_host) hipHostFree(m->err_host);
    delete m;
    return fail(ONMT_EDEVICE, "weight upload failed: %s", hipGetErrorString(e));
  }
  void* sp = nullptr;
  rc = noalloc_scratch(&sp);    // this device's copy of the allocation-free entry point's scratch array
  if (rc) {
    hipHostFree(m->err_host);
    delete m;
    return rc;
  }
  *out = m;
  return ONMT_OK;
}

int onmt_model_destroy(onmt_model* m) {
  if (!m) return fail(ONMT_EINVAL, "model is NULL");
  for (auto e : m->ev) hipEventDestroy(e);
  for (auto e : m->done_ev)
    if (e) hipEventDestroy(e);
  if (m->done_host) hipHostFree(m->done_host);
  if (m->err_host) hipHostFree(m->err_host);
  delete m;
  return ONMT_OK;
}

}  // extern "C"

// ====================================================================== workspaces

namespace {

struct EncWs {
  int32_t* lens;
  int32_t* src;
  float* memory;     // [B*S, Hm]
  float* keys;       // [B*S, H]: W_a m_s (general), the memory-side term of concat, the memory itself (dot)
  float* final_h;    // [L, B, H]
  float* final_c;
  float* gx;         // [B*S, ndir * 4 Hd_pad]
  float* y[2];       // [B*S, Hm]
  float* hs[2];      // [max(ndir, L), B, Hd]: state after an even / odd timestep, one slot per direction or layer
  float* cs[2];
  int32_t* rowmap;   // [S, B]: rowmap[s * B + b] = b * S + s (row of position s of sentence b)
};

size_t enc_layout(const Dims& d, int B, int S, char* base, EncWs* w) {
  Carver c;
  c.base = base;
  EncWs t;
  const size_t BS = (size_t)B * S;
  t.lens = c.take<int32_t>(B);
  t.src = c.take<int32_t>(BS);
  t.memory = c.take<float>(BS * d.Hm);
  t.keys = d.attn == ONMT_ATTN_DOT ? t.memory : c.take<float>(BS * d.H);
  t.final_h = c.take<float>((size_t)d.L * B * d.H);
  t.final_c = c.take<float>((size_t)d.L * B * d.H);
  t.gx = c.take<float>(BS * d.ndir * 4 * d.Hd_pad);
  for (int i = 0; i < 2; ++i) t.y[i] = c.take<float>(BS * d.Hm);
  const size_t slots = (size_t)(d.ndir > d.L ? d.ndir : d.L);
  for (int i = 0; i < 2; ++i) t.hs[i] = c.take<float>(slots * B * d.Hd);
  for (int i = 0; i < 2; ++i) t.cs[i] = c.take<float>(slots * B * d.Hd);
  t.rowmap = c.take<int32_t>(BS);
  if (w) *w = t;
  return align_up(c.off);
}

struct State {
  float* h;      // [L, N, H]
  float* c;
  float* feed;   // [N, H]
  // bf16 models: h and feed as their kPlanes bf16 term planes, [L, N, pad(H)] and [N, pad(H)] each (the
  // operands of the decoder's products, split once by their producers)
  uint16_t* h_hi;
  uint16_t* h_lo;
  uint16_t* h_lo2;
  uint16_t* feed_hi;
  uint16_t* feed_lo;
  uint16_t* feed_lo2;
};

size_t state_layout(const Dims& d, int N, char* base, State* s) {
  Carver c;
  c.base = base;
  State t;
  t.h = c.take<float>((size_t)d.L * N * d.H);
  t.c = c.take<float>((size_t)d.L * N * d.H);
  t.feed = c.take<float>((size_t)N * d.H);
  const size_t pl = (size_t)N * d.pad(d.H);
  t.h_hi = d.bf16 ? c.take<uint16_t>(d.L * pl) : nullptr;
  t.h_lo = d.bf16 ? c.take<uint16_t>(d.L * pl) : nullptr;
  t.h_lo2 = d.bf16 ? c.take<uint16_t>(d.L * pl) : nullptr;
  t.feed_hi = c.take<uint16_t>(pl);
  t.feed_lo = c.take<uint16_t>(pl);
  t.feed_lo2 = c.take<uint16_t>(pl);
  if (s) *s = t;
  return align_up(c.off);
}

struct StepWs {
  float* ctx;      // [N, Hm]
  float* scores;   // [N, S_max] raw attention scores
  float* qproj;    // [N, H] concat: query columns of W_a times the decoder output
  float* pmax;     // [N, ntiles]
  float* psum;
  float* pval;     // [N, ntiles, K]
  int32_t* pid;
  float* tk_val;   // [N, K]
  int32_t* tk_id;
  float* lse;      // [N]
  int32_t* align;  // [N] attention argmax
  float* pfmax;    // [N, ntiles] largest allowed logit per tile (hypothesis filters)
  int32_t* tok_s;  // [N] previous tokens and parents checked on the device (device validation)
  int32_t* par_s;
  int ntiles;
};

size_t step_layout(const Dims& d, int B, int S, int K, char* base, StepWs* w) {
  Carver c;
  c.base = base;
  StepWs t;
  const size_t N = (size_t)B * K;
  t.ntiles = (d.Vt + gen_tile_cols() - 1) / gen_tile_cols();
  t.ctx = c.take<float>(N * d.Hm);
  t.scores = c.take<float>(N * S);
  t.qproj = d.attn == ONMT_ATTN_CONCAT ? c.take<float>(N * d.H) : nullptr;
  t.pmax = c.take<float>(N * t.ntiles);
  t.psum = c.take<float>(N * t.ntiles);
  t.pval = c.take<float>(N * t.ntiles * K);
  t.pid = c.take<int32_t>(N * t.ntiles * K);
  t.tk_val = c.take<float>(N * K);
  t.tk_id = c.take<int32_t>(N * K);
  t.lse = c.take<float>(N);
  t.align = c.take<int32_t>(N);
  t.pfmax = c.take<float>(N * t.ntiles);
  t.tok_s = c.take<int32_t>(N);
  t.par_s = c.take<int32_t>(N);
  if (w) *w = t;
  return align_up(c.off);
}

struct SearchWs {
  EncWs enc;
  State st[2];
  StepWs step;
  BeamParams bp;
  float* cov[2];     // [N, S] attention coverage of the hypotheses (ping-pong with the state)
  double* cp;        // [N] coverage penalty of each row's hypothesis at the current step
  uint32_t* banned_bits;   // [ceil(V / 32)]
};

size_t search_layout(const Dims& d, int B, int S, int K, int T, char* base, SearchWs* w) {
  Carver c;
  c.base = base;
  SearchWs t{};
  const size_t N = (size_t)B * K;
  const size_t eb = enc_layout(d, B, S, nullptr, nullptr);
  char* e = c.take<char>(eb);
  enc_layout(d, B, S, e, &t.enc);
  for (int i = 0; i < 2; ++i) {
    const size_t sb = state_layout(d, (int)N, nullptr, nullptr);
    char* s = c.take<char>(sb);
    state_layout(d, (int)N, s, &t.st[i]);
  }
  const size_t pb = step_layout(d, B, S, K, nullptr, nullptr);
  char* p = c.take<char>(pb);
  step_layout(d, B, S, K, p, &t.step);
  BeamParams& q = t.bp;
  q.score = c.take<double>(N);
  q.parent = c.take<int32_t>(N);
  q.tok = c.take<int32_t>(N);
  q.bp_slot = c.take<int32_t>((size_t)T * N);
  q.bp_tok = c.take<int32_t>((size_t)T * N);
  q.bp_logp = c.take<float>((size_t)T * N);
  q.done = c.take<int32_t>(B);
  q.steps = c.take<int32_t>(B);
  q.done_count = c.take<int32_t>(1);
  q.best_norm = c.take<double>(B);
  q.best_raw = c.take<double>(B);
  q.best_t = c.take<int32_t>(B);
  q.best_slot = c.take<int32_t>(B);
  q.best_tok = c.take<int32_t>(B);
  q.best_logp = c.take<float>(B);
  for (int i = 0; i < 2; ++i) t.cov[i] = c.take<float>(N * S);
  t.cp = c.take<double>(N);
  q.bp_align = c.take<int32_t>((size_t)T * N);
  q.best_align = c.take<int32_t>(B);
  q.unk_cnt = c.take<int32_t>(N);
  t.banned_bits = c.take<uint32_t>((size_t)(d.Vt + 31) / 32);
  if (w) *w = t;
  return align_up(c.off);
}

struct ScoreWs {
  EncWs enc;
  State st[2];
  StepWs step;
  int32_t* in_tok;     // [T, B] decoder input at step t
  int32_t* want;       // [T, B] target predicted at step t
  int32_t* tlen;       // [B]
  float* feeds;        // [T, B, H] attentional vector of every step (the generator's input)
  uint16_t* feeds_hi;  // bf16 models: [T, B, pad(H)] each, the same as bf16 term planes
  uint16_t* feeds_lo;
  uint16_t* feeds_lo2;
  float* gpmax;        // [T * B, ntiles] generator partials of all steps
  float* gpsum;
  float* want_logit;   // [T, B]
  double* nll;         // [B]
};

size_t score_layout(const Dims& d, int B, int S, int T, char* base, ScoreWs* w) {
  Carver c;
  c.base = base;
  ScoreWs t{};
  const size_t eb = enc_layout(d, B, S, nullptr, nullptr);
  char* e = c.take<char>(eb);
  enc_layout(d, B, S, e, &t.enc);
  for (int i = 0; i < 2; ++i) {
    const size_t sb = state_layout(d, B, nullptr, nullptr);
    char* p = c.take<char>(sb);
    state_layout(d, B, p, &t.st[i]);
  }
  const size_t pb = step_layout(d, B, S, 1, nullptr, nullptr);
  char* p = c.take<char>(pb);
  step_layout(d, B, S, 1, p, &t.step);
  t.in_tok = c.take<int32_t>((size_t)T * B);
  t.want = c.take<int32_t>((size_t)T * B);
  t.tlen = c.take<int32_t>(B);
  t.feeds = c.take<float>((size_t)T * B * d.H);
  t.feeds_hi = c.take<uint16_t>((size_t)T * B * d.pad(d.H));
  t.feeds_lo = c.take<uint16_t>((size_t)T * B * d.pad(d.H));
  t.feeds_lo2 = c.take<uint16_t>((size_t)T * B * d.pad(d.H));
  t.gpmax = c.take<float>((size_t)T * B * t.step.ntiles);
  t.gpsum = c.take<float>((size_t)T * B * t.step.ntiles);
  t.want_logit = c.take<float>((size_t)T * B);
  t.nll = c.take<double>(B);
  if (w) *w = t;
  return align_up(c.off);
}

// Workspace operands that the GEMMs read through buffer descriptors (see kDescLimit): the encoder's
// memory, layer outputs and keys [B * S, Hm or H], the decoder's state rows and attentional vectors
// [B * K, Hm or H] (and their bf16 planes), and scoring's attentional vectors of all steps [T * B, H].
int check_ws_limits(const Dims& d, long long B, long long S, long long K, long long T) {
  const long long w = d.Hm > d.H ? d.Hm : d.H;
  const uint64_t enc = (uint64_t)(B * S) * (uint64_t)ceil_to((int)w, kSegK) * 4;
  const uint64_t dec = (uint64_t)(B * K) * (uint64_t)ceil_to((int)w, kSegK) * 4;
  const uint64_t sco = (uint64_t)(B * T) * (uint64_t)ceil_to(d.H, kSegK) * 4;
  if (enc >= kDescLimit)
    return fail(ONMT_EUNSUPPORTED, "B * S_max = %lld source positions need a %llu-byte memory bank (limit 2 GiB)",
                B * S, (unsigned long long)enc);
  if (dec >= kDescLimit)
    return fail(ONMT_EUNSUPPORTED, "B * beam = %lld hypothesis rows need %llu-byte state operands (limit 2 GiB)",
                B * K, (unsigned long long)dec);
  if (sco >= kDescLimit)
    return fail(ONMT_EUNSUPPORTED, "B * T_max = %lld scored rows need %llu bytes of attentional vectors (limit 2 GiB)",
                B * T, (unsigned long long)sco);
  return ONMT_OK;
}

// Small-M GEMMs: the 16-row split-K tile unless the 32-row tile already gives this many workgroups
// (measured on the decoder layers: more, smaller workgroups win while M is a few hundred rows).
#ifndef ONMT_SMALL_M_TILES
#define ONMT_SMALL_M_TILES 4096
#endif
// Unidirectional encoders with fewer rows than this run their layers as a wavefront (see encode_compute).
constexpr int kWavefrontMaxRows = 256;

int small_shape(int M, int Np) {
  const long tiles32 = (long)((M + 31) / 32) * (Np / 64);
  return tiles32 >= ONMT_SMALL_M_TILES ? kShapeSplitK : kShapeSplitKThin;
}

// LSTM GEMMs: bf16 models with at least this many rows use the 32-row two-way split-K tile.
constexpr int kMidMinRows = 256;
int lstm_shape(const Dims& d, int M, int Np) {
  if (d.bf16 && M >= kMidMinRows) return kShapeMid;
  return small_shape(M, Np);
}

// Copies src/len to the host, validates them, and uploads the token ids with every position at or beyond
// its sentence's length replaced by 0 into clean_src (device, [B, S]), so no kernel gathers an embedding
// row through an unchecked id.
int check_len_src(const onmt_model* m, const int32_t* src, const int32_t* len, int B, int S, hipStream_t st,
                  int* max_len, int32_t* clean_src, int32_t* rowmap) {
  if (!src || !len) return fail(ONMT_EINVAL, "src/len is NULL");
  if (B < 1 || S < 1) return fail(ONMT_EINVAL, "B and S_max must be >= 1");
  if ((long long)B * S > (1LL << 28)) return fail(ONMT_EUNSUPPORTED, "B * S_max too large");
  std::vector<int32_t> hl(B), hs((size_t)B * S);
  HIP_TRY(hipMemcpyAsync(hl.data(), len, sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipMemcpyAsync(hs.data(), src, sizeof(int32_t) * hs.size(), hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  int mx = 0;
  for (int b = 0; b < B; ++b) {
    if (hl[b] < 1 || hl[b] > S) return fail(ONMT_EINVAL, "len[%d] = %d outside [1, %d]", b, hl[b], S);
    mx = hl[b] > mx ? hl[b] : mx;
    for (int s = 0; s < hl[b]; ++s) {
      const int v = hs[(size_t)b * S + s];
      if (v < 0 || v >= m->cfg.src_vocab) return fail(ONMT_EINVAL, "src[%d, %d] = %d outside [0, %d)", b, s, v, m->cfg.src_vocab);
    }
  }
  for (int b = 0; b < B; ++b)
    for (int s = hl[b]; s < S; ++s) hs[(size_t)b * S + s] = 0;
  HIP_TRY(hipMemcpyAsync(clean_src, hs.data(), sizeof(int32_t) * hs.size(), hipMemcpyHostToDevice, st));
  std::vector<int32_t> rm((size_t)B * S);
  for (int s = 0; s < S; ++s)
    for (int b = 0; b < B; ++b) rm[(size_t)s * B + b] = b * S + s;
  HIP_TRY(hipMemcpyAsync(rowmap, rm.data(), sizeof(int32_t) * rm.size(), hipMemcpyHostToDevice, st));
  HIP_TRY(hipStreamSynchronize(st));
  *max_len = mx;
  return ONMT_OK;
}

// Source ids and lengths, checked either on the host (ONMT_VALIDATE_HOST: copied over, one stream sync; the
// longest length bounds the encoder's steps) or on the device (ONMT_VALIDATE_DEVICE: a kernel writes the
// checked copies and records violations; the encoder then steps over all S_max positions, which the packed
// padding leaves unchanged past each sentence's length). On return w.src, w.rowmap and (device mode)
// w.lens hold the checked inputs; *lens_src is what encode_compute copies into w.lens (nullptr: in place).
int checked_source(onmt_model* m, const int32_t* src, const int32_t* len, int B, int S, const EncWs& w, hipStream_t st,
                   int* max_len, const int32_t** lens_src) {
  if (m->validation == ONMT_VALIDATE_DEVICE) {
    if (!src || !len) return fail(ONMT_EINVAL, "src/len is NULL");
    if ((long long)B * S > (1LL << 28)) return fail(ONMT_EUNSUPPORTED, "B * S_max too large");
    HIP_TRY(sanitize_src(src, len, B, S, m->cfg.src_vocab, w.src, w.lens, w.rowmap, m->err_host, st));
    *max_len = S;
    *lens_src = nullptr;
    return ONMT_OK;
  }
  *lens_src = len;
  return check_len_src(m, src, len, B, S, st, max_len, w.src, w.rowmap);
}

// Encoder compute on validated inputs (Section 2 encoder RNN; Tables 3-4 bidirectional; readings R2-R5).
// len == nullptr: the lengths are already in w.lens (checked on the device).
int encode_compute(onmt_model* m, const int32_t* src, const int32_t* len, int B, int S, int max_len, const EncWs& w,
                   hipStream_t st) {
  const Dims& d = m->d;
  const int BS = B * S;
  (void)src;   // the validated, pad-cleaned ids are already in w.src
  if (len) HIP_TRY(hipMemcpyAsync(w.lens, len, sizeof(int32_t) * B, hipMemcpyDeviceToDevice, st));
  HIP_TRY(fill_f32(w.memory, (size_t)BS * d.Hm, 0.f, st));
  const int gxw = d.ndir * 4 * d.Hd_pad;
  const size_t SB = (size_t)B * d.Hd;       // one state slot
  // Recurrent GEMM of (layer l, direction dir) at position s, its step-th step, state slot `slot`: the
  // state after step k goes to buffer k & 1 and step k reads the other buffer (buffer 1 holds the zero
  // state before step 0).
  // Unidirectional layers >= 1 keep [W_x | W_h] in one matrix: `joint` steps read [y_{l-1} at s | h]
  // against all of it; otherwise the step reads h against the W_h columns and adds the projection gx.
  const bool uni = d.ndir == 1;
  auto recurrent = [&](int l, int dir, int s, int step, int slot, bool joint, AOp& r, BOp& wb, LstmParams& lp) {
    const int pin = (step + 1) & 1;
    const float* hp = w.hs[pin] + slot * SB;
    const float* cp = w.cs[pin] + slot * SB;
    r = AOp{};
    r.M = B;
    if (joint) {   // [output of layer l-1 at position s | h]
      r.nseg = 2;
      r.seg[0] = seg(w.y[(l - 1) & 1], w.rowmap + (size_t)s * B, BS, d.Hm, d.Hm, d.pad(d.Hm), 0);
      r.seg[1] = seg(hp, nullptr, B, d.Hd, d.Hd, d.pad(d.Hd), 0);
      wb = bop(m->enc_xh[l]);
    } else {       // h, plus the precomputed input projection
      r.nseg = 1;
      r.seg[0] = seg(hp, nullptr, B, d.Hd, d.Hd, d.pad(d.Hd), 0);
      if (uni && l > 0) {   // the W_h columns of the joint matrix (row stride unchanged)
        wb = bop(m->enc_xh[l]);
        wb.W = (const char*)wb.W + (size_t)d.pad(d.Hm) * d.esz;
      } else {
        wb = bop(m->enc_h[l * d.ndir + dir]);
      }
    }
    lp = LstmParams{};
    lp.bias = joint ? m->enc_bias[l] : nullptr;
    lp.gx = joint ? nullptr : w.gx;
    lp.ld_gx = gxw;
    lp.gx_col0 = dir * 4 * d.Hd_pad;
    lp.gx_S = S;
    lp.gx_s = s;
    lp.c_in = cp;
    lp.c_idx = nullptr;
    lp.ld_c = d.Hd;
    lp.h_in = hp;
    lp.ld_h_in = d.Hd;
    lp.h_out = w.hs[pin ^ 1] + slot * SB;
    lp.c_out = w.cs[pin ^ 1] + slot * SB;
    lp.ld_out = d.Hd;
    lp.y_out = (l == d.L - 1) ? w.memory : w.y[l & 1];
    lp.ld_y = d.Hm;
    lp.y_S = S;
    lp.y_s = s;
    lp.y_col0 = dir * d.Hd;
    lp.lens = w.lens;
    lp.H = d.Hd;
  };
  auto run_one = [&](int l, int dir, int s, int step, int slot, bool joint) -> int {
    AOp r;
    BOp wb;
    LstmParams lp;
    recurrent(l, dir, s, step, slot, joint, r, wb, lp);
    HIP_TRY(gemm_lstm(d.bf16, lstm_shape(d, B, wb.Np), r, wb, lp, st));
    return ONMT_OK;
  };
  auto run_two = [&](int l0, int dir0, int s0, int step0, int slot0, bool joint0, int l1, int dir1, int s1,
                     int step1, int slot1, bool joint1) -> int {
    LstmPair g{};
    recurrent(l0, dir0, s0, step0, slot0, joint0, g.a[0], g.b[0], g.p[0]);
    recurrent(l1, dir1, s1, step1, slot1, joint1, g.a[1], g.b[1], g.p[1]);
    HIP_TRY(gemm_lstm2(d.bf16, d.bf16 && B >= kMidMinRows ? kShapeMid : kShapeSplitKThin, g, st));
    return ONMT_OK;
  };
  auto project = [&](int l) -> int {   // input projection of every position, both directions at once
    AOp a{};
    a.M = BS;
    a.nseg = 1;
    if (l == 0) a.seg[0] = seg(m->E_src, w.src, d.Vs, d.E, d.E, d.pad(d.E), d.bf16);
    else a.seg[0] = seg(w.y[(l - 1) & 1], nullptr, BS, d.Hm, d.Hm, d.pad(d.Hm), 0);
    StoreParams sp{m->enc_bias[l], w.gx, gxw, gxw, 0};
    // unidirectional layers >= 1: the W_x columns of the joint matrix (the product reads only pad(Hm))
    HIP_TRY(gemm_store(d.bf16, kShapeWide, a, bop(uni && l > 0 ? m->enc_xh[l] : m->enc_x[l]), sp, st));
    return ONMT_OK;
  };
  const int slots = d.ndir > d.L ? d.ndir : d.L;
  HIP_TRY(fill_f32(w.hs[1], (size_t)slots * SB, 0.f, st));
  HIP_TRY(fill_f32(w.cs[1], (size_t)slots * SB, 0.f, st));
  const int last = (max_len - 1) & 1;      // buffer holding the state after the last step
  int rc = ONMT_OK;
  if (uni && B < kWavefrontMaxRows) {
    // few rows per step (launch-bound): layer l processes position s = wave - l, one step behind the
    // layer below, and the layers of one wave go out two per launch
    if ((rc = project(0))) return rc;
    for (int wave = 0; wave < max_len + d.L - 1; ++wave) {
      const int lo = wave - max_len + 1 > 0 ? wave - max_len + 1 : 0;
      const int hi = wave < d.L - 1 ? wave : d.L - 1;
      for (int l = lo; l <= hi; l += 2) {
        const int t0 = wave - l, t1 = wave - l - 1;   // position = step for a forward layer
        rc = l + 1 <= hi ? run_two(l, 0, t0, t0, l, l > 0, l + 1, 0, t1, t1, l + 1, true)
                         : run_one(l, 0, t0, t0, l, l > 0);
        if (rc) return rc;
      }
    }
    for (int l = 0; l < d.L; ++l) {
      HIP_TRY(copy_cols(w.hs[last] + l * SB, d.Hd, w.final_h + (size_t)l * B * d.H, d.H, B, d.Hd, st));
      HIP_TRY(copy_cols(w.cs[last] + l * SB, d.Hd, w.final_c + (size_t)l * B * d.H, d.H, B, d.Hd, st));
    }
  } else if (uni) {
    // many rows per step (compute-bound): layer by layer, each with its input projection of every
    // position done as one large GEMM first
    for (int l = 0; l < d.L; ++l) {
      if ((rc = project(l))) return rc;
      for (int step = 0; step < max_len; ++step)
        if ((rc = run_one(l, 0, step, step, l, false))) return rc;
    }
    for (int l = 0; l < d.L; ++l) {
      HIP_TRY(copy_cols(w.hs[last] + l * SB, d.Hd, w.final_h + (size_t)l * B * d.H, d.H, B, d.Hd, st));
      HIP_TRY(copy_cols(w.cs[last] + l * SB, d.Hd, w.final_c + (size_t)l * B * d.H, d.H, B, d.Hd, st));
    }
  } else {
    // both directions of a layer step together, one launch per step
    for (int l = 0; l < d.L; ++l) {
      if ((rc = project(l))) return rc;
      if (l > 0) {
        HIP_TRY(fill_f32(w.hs[1], (size_t)slots * SB, 0.f, st));
        HIP_TRY(fill_f32(w.cs[1], (size_t)slots * SB, 0.f, st));
      }
      for (int step = 0; step < max_len; ++step)
        if ((rc = run_two(l, 0, step, step, 0, false, l, 1, max_len - 1 - step, step, 1, false))) return rc;
      for (int dir = 0; dir < d.ndir; ++dir) {
        HIP_TRY(copy_cols(w.hs[last] + dir * SB, d.Hd, w.final_h + (size_t)l * B * d.H + dir * d.Hd, d.H, B, d.Hd, st));
        HIP_TRY(copy_cols(w.cs[last] + dir * SB, d.Hd, w.final_c + (size_t)l * B * d.H + dir * d.Hd, d.H, B, d.Hd, st));
      }
    }
  }
  // attention keys W_a m_s (concat: its memory columns), once per batch; dot scores read the memory
  if (d.attn == ONMT_ATTN_DOT) return ONMT_OK;
  AOp a{};
  a.M = BS;
  a.nseg = 1;
  a.seg[0] = seg(w.memory, nullptr, BS, d.Hm, d.Hm, d.pad(d.Hm), 0);
  StoreParams kp{nullptr, w.keys, d.H, d.H, 0};
  HIP_TRY(gemm_store(d.bf16, kShapeWide, a, bop(m->W_a), kp, st));
  return ONMT_OK;
}

int decode_init_compute(onmt_model* m, const EncWs& w, int B, int K, const State& s, hipStream_t st) {
  const Dims& d = m->d;
  const int N = B * K;
  for (int l = 0; l < d.L; ++l) {
    HIP_TRY(replicate_rows(w.final_h + (size_t)l * B * d.H, d.H, B, K, s.h + (size_t)l * N * d.H, d.H, d.H, st));
    HIP_TRY(replicate_rows(w.final_c + (size_t)l * B * d.H, d.H, B, K, s.c + (size_t)l * N * d.H, d.H, d.H, st));
  }
  HIP_TRY(fill_f32(s.feed, (size_t)N * d.H, 0.f, st));
  if (d.bf16) {   // the operand planes of the first step
    HIP_TRY(split_rows(s.h, d.H, d.L * N, d.H, s.h_hi, s.h_lo, s.h_lo2, d.pad(d.H), st));
    HIP_TRY(split_rows(s.feed, d.H, N, d.H, s.feed_hi, s.feed_lo, s.feed_lo2, d.pad(d.H), st));
  }
  return ONMT_OK;
}

// Kernel timing: an event pair around every prof-th launch of each kind (ONMT_KERNEL_*), on the stream the
// kernel is launched on; the pairs are read back by time_collect once the stream has been synchronized.
void time_begin(onmt_model* m, hipStream_t st, int kind = ONMT_KERNEL_GENERATOR) {
  m->prof_open[kind] = false;
  if (!m->prof || !((m->prof_kinds >> kind) & 1u) || (m->prof_seq[kind]++ % m->prof) != 0) return;
  while (m->ev.size() < m->ev_used + 2) {
    hipEvent_t e;
    // timing-only events: no system-scope fence, so recording them does not stall the next kernel
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return;
    m->ev.push_back(e);
  }
  if (m->ev_kind.size() < m->ev.size()) m->ev_kind.resize(m->ev.size());
  hipEventRecord(m->ev[m->ev_used], st);
  m->ev_kind[m->ev_used] = kind;
  m->prof_pair[kind] = m->ev_used;
  m->ev_used += 2;
  m->prof_open[kind] = true;
}
void time_end(onmt_model* m, hipStream_t st, int kind = ONMT_KERNEL_GENERATOR) {
  if (!m->prof_open[kind]) return;
  m->prof_open[kind] = false;
  hipEventRecord(m->ev[m->prof_pair[kind] + 1], st);
}
void time_collect(onmt_model* m) {
  for (size_t i = 0; i + 1 < m->ev_used; i += 2) {
    float ms = 0.f;
    if (hipEventSynchronize(m->ev[i + 1]) == hipSuccess && hipEventElapsedTime(&ms, m->ev[i], m->ev[i + 1]) == hipSuccess) {
      m->prof_ms[m->ev_kind[i]] += ms;
      m->prof_n[m->ev_kind[i]] += 1;
    }
  }
  m->ev_used = 0;
}

// One decoder step on validated inputs (Section 2; Figure 1(a); items (a)-(c); Section 4.2 attention).
// mode 0: logp [N, V] full log-softmax; mode 1: top-K (logp [N, K], ids [N, K]); mode 2 (beam search):
// stop after the generator, leaving its per-tile partials in the step workspace for the beam step;
// mode 3 (teacher forcing): stop after the attentional vector (out.feed), the generator runs later over
// all steps at once.
// Optional work of a decoder step beyond the log-distribution.
struct StepExtras {
  // bf16 models: where the attentional vector's term planes go (default: the output state's)
  uint16_t* feed_hi = nullptr;
  uint16_t* feed_lo = nullptr;
  uint16_t* feed_lo2 = nullptr;
  const int32_t* want = nullptr;        // the logit of column want[r] of every row goes to want_logit[r]
  float* want_logit = nullptr;
  const Coverage* cov = nullptr;        // attention coverage and its penalty
  int32_t* align = nullptr;             // attention argmax per row
  const uint32_t* banned_bits = nullptr;   // hypothesis filters of the generator's top-K lists
  const int32_t* unk_cnt = nullptr;
  int unk_id = 0, max_unk = -1;
  float* pfmax = nullptr;
};

int decode_compute(onmt_model* m, const EncWs& w, int B, int S, int K, const State& in, const State& out,
                   const int32_t* prev_tok, const int32_t* parent, int mode, float* logp, int32_t* ids, float* lse,
                   float* attn, const StepWs& sw, hipStream_t st, const StepExtras& ex = StepExtras{},
                   bool timing = true) {
  const Dims& d = m->d;
  const int N = B * K;
  const size_t LH = (size_t)N * d.H;
  const int pH = d.pad(d.H);
  const size_t LP = (size_t)N * pH;
  // bf16 models read the pre-split planes of h and feed (widths that are multiples of 8)
  const bool pre = d.bf16 && d.H % 8 == 0;
  auto act = [&](const float* x, const uint16_t* hi, const uint16_t* lo, const uint16_t* lo2, const int32_t* idx) {
    if (!pre) return seg(x, idx, N, d.H, d.H, pH, 0);
    Seg s = seg(hi, idx, N, pH, d.H, pH, 1);
    s.lo = lo;
    s.lo2 = lo2;
    return s;
  };
  for (int l = 0; l < d.L; ++l) {
    AOp a{};
    a.M = N;
    BOp wb = bop(m->dec_w[l]);
    LstmParams lp{};
    a.nseg = 2;
    if (l == 0) {
      // [feed ; h] against the feed and recurrent columns; the embedding columns' product is the
      // precomputed row of the previous token (emb_gates), added in the epilogue
      a.seg[0] = act(in.feed, in.feed_hi, in.feed_lo, in.feed_lo2, parent);
      a.seg[1] = act(in.h, in.h_hi, in.h_lo, in.h_lo2, parent);
      wb.W = (const char*)wb.W + (size_t)d.pad(d.E) * d.esz;
      lp.gx = m->emb_gates;
      lp.gx_idx = prev_tok;
      lp.gx_rows = d.Vt;
      lp.ld_gx = 4 * d.H_pad;
    } else {
      a.seg[0] = act(out.h + (l - 1) * LH, pre ? out.h_hi + (l - 1) * LP : nullptr,
                     pre ? out.h_lo + (l - 1) * LP : nullptr, pre ? out.h_lo2 + (l - 1) * LP : nullptr, nullptr);
      a.seg[1] = act(in.h + l * LH, pre ? in.h_hi + l * LP : nullptr, pre ? in.h_lo + l * LP : nullptr,
                     pre ? in.h_lo2 + l * LP : nullptr, parent);
    }
    if (d.bf16) {
      lp.h_hi = out.h_hi + l * LP;
      lp.h_lo = out.h_lo + l * LP;
      lp.h_lo2 = out.h_lo2 + l * LP;
      lp.ld_hl = pH;
    }
    lp.bias = m->dec_bias[l];
    lp.c_in = in.c + l * LH;
    lp.c_idx = parent;
    lp.ld_c = d.H;
    lp.h_out = out.h + l * LH;
    lp.c_out = out.c + l * LH;
    lp.ld_out = d.H;
    lp.H = d.H;
    if (timing) time_begin(m, st, ONMT_KERNEL_LSTM);
    HIP_TRY(gemm_lstm(d.bf16, lstm_shape(d, N, m->dec_w[l].Np), a, wb, lp, st));
    if (timing) time_end(m, st, ONMT_KERNEL_LSTM);
  }
  const float* q = out.h + (d.L - 1) * LH;
  const float* sq = q;
  if (d.attn == ONMT_ATTN_CONCAT) {   // the query side of concat's tanh argument, W_q q
    AOp a{};
    a.M = N;
    a.nseg = 1;
    a.seg[0] = seg(q, nullptr, N, d.H, d.H, d.pad(d.H), 0);
    StoreParams sp{nullptr, sw.qproj, d.H, d.H, 0};
    HIP_TRY(gemm_store(d.bf16, small_shape(N, m->W_q.Np), a, bop(m->W_q), sp, st));
    sq = sw.qproj;
  }
  const AttnExtra ax{ex.cov, ex.align};
  if (timing) time_begin(m, st, ONMT_KERNEL_ATTENTION);
  HIP_TRY(attention(sq, d.H, w.keys, m->v_a, w.memory, w.lens, B, S, d.H, d.Hm, K, sw.scores, sw.ctx, attn, ax,
                    st));
  if (timing) time_end(m, st, ONMT_KERNEL_ATTENTION);
  {
    AOp a{};
    a.M = N;
    a.nseg = 2;
    a.seg[0] = seg(sw.ctx, nullptr, N, d.Hm, d.Hm, d.pad(d.Hm), 0);
    a.seg[1] = seg(q, nullptr, N, d.H, d.H, d.pad(d.H), 0);
    StoreParams sp{nullptr, out.feed, d.H, d.H, 1};
    {                        // the generator's operand, split once here instead of in every column tile
      sp.hi = ex.feed_hi ? ex.feed_hi : out.feed_hi;
      sp.lo = ex.feed_lo ? ex.feed_lo : out.feed_lo;
      sp.lo2 = ex.feed_lo2 ? ex.feed_lo2 : out.feed_lo2;
      sp.ld_hl = sp.ncols_hl = d.pad(d.H);
    }
    if (timing) time_begin(m, st, ONMT_KERNEL_OUTPUT);
    HIP_TRY(gemm_store(d.bf16, small_shape(N, m->W_c.Np), a, bop(m->W_c), sp, st));
    if (timing) time_end(m, st, ONMT_KERNEL_OUTPUT);
  }
  if (mode == 3) return ONMT_OK;
  {
    AOp a{};
    a.M = N;
    a.nseg = 1;
    a.seg[0] = seg(out.feed, nullptr, N, d.H, d.H, d.pad(d.H), 0);
    GenParams gp{};
    gp.bias = m->b_s;
    gp.V = d.Vt;
    gp.K = K;
    gp.ntiles = sw.ntiles;
    gp.pmax = sw.pmax;
    gp.psum = sw.psum;
    gp.pval = sw.pval;
    gp.pid = sw.pid;
    gp.logits = mode == 0 ? logp : nullptr;
    gp.ld_logits = d.Vt;
    gp.want = ex.want;
    gp.want_logit = ex.want_logit;
    gp.banned_bits = ex.banned_bits;
    gp.unk_cnt = ex.unk_cnt;
    gp.unk_id = ex.unk_id;
    gp.max_unk = ex.max_unk;
    gp.pfmax = ex.pfmax;
    if (timing) time_begin(m, st);
    if (d.bf16 || gemm_gen_split_rows(N))
      HIP_TRY(gemm_gen_split(GenSplitA{out.feed_hi, out.feed_lo, N, d.pad(d.H), d.pad(d.H), out.feed_lo2},
                             bop(m->W_s), d.gwp, gp, st));
    else
      HIP_TRY(gemm_gen(a, bop(m->W_s32), gp, st));
    if (timing) time_end(m, st);
  }
  if (mode == 2) return ONMT_OK;
  float* lse_out = lse ? lse : sw.lse;
  if (mode == 0) {
    HIP_TRY(lse_topk_merge(sw.pmax, sw.psum, sw.pval, sw.pid, N, sw.ntiles, K, sw.tk_val, sw.tk_id, lse_out, st));
    HIP_TRY(subtract_rows(logp, d.Vt, lse_out, N, d.Vt, st));
  } else {
    HIP_TRY(lse_topk_merge(sw.pmax, sw.psum, sw.pval, sw.pid, N, sw.ntiles, K, logp, ids, lse_out, st));
  }
  return ONMT_OK;
}

int check_beam(const onmt_model* m, int S, int K) {
  if (K < 1 || K > kMaxBeam) return fail(ONMT_EUNSUPPORTED, "beam %d outside [1, %d]", K, kMaxBeam);
  if (K > m->cfg.tgt_vocab) return fail(ONMT_EINVAL, "beam %d larger than the vocabulary", K);
  if (m->d.H > 1024) return fail(ONMT_EUNSUPPORTED, "attention supports hidden <= 1024");
  if (attention_lds_bytes(S, m->d.H, K) > 64 * 1024)
    return fail(ONMT_EUNSUPPORTED, "beam * max(hidden, S_max) too large for the attention workgroups");
  return ONMT_OK;
}

}  // namespace

extern "C" {

size_t onmt_encode_ws_bytes(const onmt_model* m, int B, int S) {
  if (!m || B < 1 || S < 1) return 0;
  return enc_layout(m->d, B, S, nullptr, nullptr);
}

int onmt_encode(onmt_model* m, const int32_t* src, const int32_t* len, int B, int S, void* ws, size_t ws_bytes,
                void* stream) {
  if (!m) return fail(ONMT_EINVAL, "model is NULL");
  if (!ws) return fail(ONMT_EINVAL, "enc_ws is NULL");
  hipStream_t st = (hipStream_t)stream;
  if (B < 1 || S < 1) return fail(ONMT_EINVAL, "B and S_max must be >= 1");
  int rc = check_ws_limits(m->d, B, S, 1, 0);
  if (rc) return rc;
  if (ws_bytes < enc_layout(m->d, B, S, nullptr, nullptr)) return fail(ONMT_ESIZE, "encoder workspace too small");
  EncWs w;
  enc_layout(m->d, B, S, (char*)ws, &w);
  int mx = 0;
  const int32_t* lsrc = nullptr;
  rc = checked_source(m, src, len, B, S, w, st, &mx, &lsrc);
  if (rc) return rc;
  return encode_compute(m, src, lsrc, B, S, mx, w, st);
}

size_t onmt_state_bytes(const onmt_model* m, int N) {
  if (!m || N < 1) return 0;
  return state_layout(m->d, N, nullptr, nullptr);
}

size_t onmt_step_ws_bytes(const onmt_model* m, int B, int S, int K) {
  if (!m || B < 1 || S < 1 || K < 1) return 0;
  return step_layout(m->d, B, S, K, nullptr, nullptr);
}

int onmt_decode_init(onmt_model* m, const void* enc_ws, int B, int S, int K, void* state_out, void* stream) {
  if (!m || !enc_ws || !state_out) return fail(ONMT_EINVAL, "NULL argument");
  if (B < 1 || S < 1 || K < 1) return fail(ONMT_EINVAL, "B, S_max, K must be >= 1");
  int rc = check_ws_limits(m->d, B, S, K, 0);
  if (rc) return rc;
  EncWs w;
  enc_layout(m->d, B, S, (char*)enc_ws, &w);
  State s;
  state_layout(m->d, B * K, (char*)state_out, &s);
  return decode_init_compute(m, w, B, K, s, (hipStream_t)stream);
}

int onmt_decode_step(onmt_model* m, const void* enc_ws, int B, int S, int K, const void* state_in, void* state_out,
                     const int32_t* prev_tok, const int32_t* parent, int mode, float* logp, int32_t* ids, float* lse,
                     float* attn, void* step_ws, size_t step_ws_bytes, void* stream) {
  if (!m || !enc_ws || !state_in || !state_out || !prev_tok || !logp || !step_ws) return fail(ONMT_EINVAL, "NULL argument");
  if (state_in == state_out) return fail(ONMT_EINVAL, "state_in and state_out must differ");
  if (B < 1 || S < 1) return fail(ONMT_EINVAL, "B and S_max must be >= 1");
  int rc = check_beam(m, S, K);
  if (rc) return rc;
  if ((rc = check_ws_limits(m->d, B, S, K, 0))) return rc;
  if (mode != 0 && mode != 1) return fail(ONMT_EINVAL, "mode must be 0 (full) or 1 (top-K)");
  if (mode == 1 && !ids) return fail(ONMT_EINVAL, "ids is NULL in top-K mode");
  if (step_ws_bytes < step_layout(m->d, B, S, K, nullptr, nullptr)) return fail(ONMT_ESIZE, "step workspace too small");
  hipStream_t st = (hipStream_t)stream;
  const int N = B * K;
  StepWs sw;
  step_layout(m->d, B, S, K, (char*)step_ws, &sw);
  if (m->validation == ONMT_VALIDATE_DEVICE) {
    HIP_TRY(sanitize_step(prev_tok, parent, N, m->cfg.tgt_vocab, sw.tok_s, sw.par_s, m->err_host, st));
    prev_tok = sw.tok_s;
    parent = parent ? sw.par_s : nullptr;
  } else {
    std::vector<int32_t> ht(N), hp(parent ? N : 0);
    HIP_TRY(hipMemcpyAsync(ht.data(), prev_tok, sizeof(int32_t) * N, hipMemcpyDeviceToHost, st));
    if (parent) HIP_TRY(hipMemcpyAsync(hp.data(), parent, sizeof(int32_t) * N, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    for (int r = 0; r < N; ++r) {
      if (ht[r] < 0 || ht[r] >= m->cfg.tgt_vocab) return fail(ONMT_EINVAL, "prev_tok[%d] = %d out of range", r, ht[r]);
      if (parent && (hp[r] < 0 || hp[r] >= N)) return fail(ONMT_EINVAL, "parent[%d] = %d out of range", r, hp[r]);
    }
  }
  EncWs w;
  enc_layout(m->d, B, S, (char*)enc_ws, &w);
  State si, so;
  state_layout(m->d, N, (char*)state_in, &si);
  state_layout(m->d, N, (char*)state_out, &so);
  rc = decode_compute(m, w, B, S, K, si, so, prev_tok, parent, mode, logp, ids, lse, attn, sw, st);
  if (m->prof) {
    HIP_TRY(hipStreamSynchronize(st));
    time_collect(m);
  }
  return rc;
}

int onmt_set_validation(onmt_model* m, int mode) {
  if (!m) return fail(ONMT_EINVAL, "model is NULL");
  if (mode != ONMT_VALIDATE_HOST && mode != ONMT_VALIDATE_DEVICE)
    return fail(ONMT_EINVAL, "validation mode must be ONMT_VALIDATE_HOST or ONMT_VALIDATE_DEVICE");
  m->validation = mode;
  return ONMT_OK;
}

int onmt_decode_step_noalloc(onmt_model* m, const void* enc_ws, int B, int S, int K, const void* state_in,
                             void* state_out, const int32_t* prev_tok, const int32_t* parent, int mode, float* logp,
                             int32_t* ids, float* lse, float* attn, void* stream) {
  if (!m || !enc_ws || !state_in || !state_out || !prev_tok || !logp) return fail(ONMT_EINVAL, "NULL argument");
  if (state_in == state_out) return fail(ONMT_EINVAL, "state_in and state_out must differ");
  if (B < 1 || S < 1) return fail(ONMT_EINVAL, "B and S_max must be >= 1");
  int rc = check_beam(m, S, K);
  if (rc) return rc;
  if ((rc = check_ws_limits(m->d, B, S, K, 0))) return rc;
  if (mode != 0 && mode != 1) return fail(ONMT_EINVAL, "mode must be 0 (full) or 1 (top-K)");
  if (mode == 1 && !ids) return fail(ONMT_EINVAL, "ids is NULL in top-K mode");
  const size_t need = step_layout(m->d, B, S, K, nullptr, nullptr);
  if (need > ONMT_NOALLOC_SCRATCH_BYTES)
    return fail(ONMT_EUNSUPPORTED, "this step needs %zu bytes of scratch, more than the %u of the allocation-free call",
                need, (unsigned)ONMT_NOALLOC_SCRATCH_BYTES);
  void* sp = nullptr;
  if ((rc = noalloc_scratch(&sp))) return rc;
  hipStream_t st = (hipStream_t)stream;
  const int N = B * K;
  StepWs sw;
  step_layout(m->d, B, S, K, (char*)sp, &sw);
  HIP_TRY(sanitize_step(prev_tok, parent, N, m->cfg.tgt_vocab, sw.tok_s, sw.par_s, m->err_host, st));
  EncWs w;
  enc_layout(m->d, B, S, (char*)enc_ws, &w);
  State si, so;
  state_layout(m->d, N, (char*)state_in, &si);
  state_layout(m->d, N, (char*)state_out, &so);
  return decode_compute(m, w, B, S, K, si, so, sw.tok_s, parent ? sw.par_s : nullptr, mode, logp, ids, lse, attn, sw,
                        st, StepExtras{}, false);
}

int onmt_device_status(onmt_model* m, int* code) {
  if (!m || !code) return fail(ONMT_EINVAL, "NULL argument");
  volatile int32_t* e = m->err_host;
  const int32_t kind = *e;
  *e = 0;
  *code = kind ? ONMT_EINVAL : ONMT_OK;
  if (kind) {
    static const char* what[] = {"", "a source length outside [1, S_max]", "a source id outside [0, src_vocab)",
                                 "a previous token outside [0, tgt_vocab)", "a parent row outside [0, B * beam)"};
    fail(ONMT_EINVAL, "device validation found %s (replaced by a safe value)", kind >= 1 && kind <= 4 ? what[kind] : "an invalid input");
  }
  return ONMT_OK;
}

size_t onmt_search_ws_bytes(const onmt_model* m, int B, int S, const onmt_search_params* p) {
  if (!m || !p || B < 1 || S < 1 || p->beam < 1 || p->max_len < 1) return 0;
  return search_layout(m->d, B, S, p->beam, p->max_len, nullptr, nullptr);
}

int onmt_beam_search(onmt_model* m, const int32_t* src, const int32_t* len, int B, int S,
                     const onmt_search_params* prm, void* ws, size_t ws_bytes, int32_t* out_tok, int32_t* out_len,
                     double* out_raw, double* out_norm, float* out_tok_logp, int32_t* out_align,
                     const onmt_trace* trace, void* stream) {
  if (!m || !prm || !ws) return fail(ONMT_EINVAL, "NULL argument");
  if (!out_tok || !out_len || !out_raw || !out_norm) return fail(ONMT_EINVAL, "NULL output pointer");
  const int K = prm->beam, T = prm->max_len;
  if (T < 1 || T > 100000) return fail(ONMT_EINVAL, "max_len %d outside [1, 100000]", T);
  if (!(prm->alpha >= 0.0) || !std::isfinite(prm->alpha)) return fail(ONMT_EINVAL, "alpha must be finite and >= 0");
  if (!(prm->beta >= 0.0) || !std::isfinite(prm->beta)) return fail(ONMT_EINVAL, "beta must be finite and >= 0");
  if (prm->n_banned < 0 || (prm->n_banned > 0 && !prm->banned)) return fail(ONMT_EINVAL, "banned list invalid");
  for (int i = 0; i < prm->n_banned; ++i)
    if (prm->banned[i] < 0 || prm->banned[i] >= m->cfg.tgt_vocab)
      return fail(ONMT_EINVAL, "banned[%d] = %d outside [0, %d)", i, prm->banned[i], m->cfg.tgt_vocab);
  if (trace && (!trace->slot || !trace->tok || !trace->cand || !trace->steps))
    return fail(ONMT_EINVAL, "trace given with a NULL array");
  if (B < 1 || S < 1) return fail(ONMT_EINVAL, "B and S_max must be >= 1");
  int rc = check_beam(m, S, K);
  if (rc) return rc;
  if ((rc = check_ws_limits(m->d, B, S, K, 0))) return rc;
  if (ws_bytes < search_layout(m->d, B, S, K, T, nullptr, nullptr)) return fail(ONMT_ESIZE, "search workspace too small");
  hipStream_t st = (hipStream_t)stream;
  SearchWs w;
  search_layout(m->d, B, S, K, T, (char*)ws, &w);
  int mx = 0;
  const int32_t* lsrc = nullptr;
  rc = checked_source(m, src, len, B, S, w.enc, st, &mx, &lsrc);
  if (rc) return rc;

  BeamParams bp = w.bp;
  bp.B = B;
  bp.K = K;
  bp.V = m->cfg.tgt_vocab;
  bp.T_max = T;
  bp.eos = m->cfg.eos_id;
  bp.pad = m->cfg.pad_id;
  bp.alpha = prm->alpha;
  bp.lp_tmax = std::pow((5.0 + T) / 6.0, prm->alpha);
  bp.tr_slot = trace ? trace->slot : nullptr;
  bp.tr_tok = trace ? trace->tok : nullptr;
  bp.tr_cand = trace ? trace->cand : nullptr;

  GenPartials gp{w.step.pmax, w.step.psum, w.step.pval, w.step.pid, w.step.ntiles};
  rc = encode_compute(m, src, lsrc, B, S, mx, w.enc, st);
  if (rc) return rc;
  rc = decode_init_compute(m, w.enc, B, K, w.st[0], st);
  if (rc) return rc;
  const bool coverage = prm->beta > 0.0;
  bp.cp = coverage ? w.cp : nullptr;
  const bool filtering = prm->n_banned > 0 || prm->max_unk >= 0;
  bp.unk_cnt = filtering ? bp.unk_cnt : nullptr;
  bp.unk_id = m->cfg.unk_id;
  bp.align = out_align ? w.step.align : nullptr;
  std::vector<uint32_t> bits;
  if (prm->n_banned > 0) {
    bits.assign((size_t)(m->cfg.tgt_vocab + 31) / 32, 0u);
    for (int i = 0; i < prm->n_banned; ++i) bits[prm->banned[i] >> 5] |= 1u << (prm->banned[i] & 31);
    HIP_TRY(hipMemcpyAsync(w.banned_bits, bits.data(), bits.size() * sizeof(uint32_t), hipMemcpyHostToDevice, st));
  }
  StepExtras ex;
  ex.align = bp.align ? w.step.align : nullptr;
  if (filtering) {
    ex.banned_bits = prm->n_banned > 0 ? w.banned_bits : nullptr;
    ex.unk_cnt = prm->max_unk >= 0 ? bp.unk_cnt : nullptr;
    ex.unk_id = m->cfg.unk_id;
    ex.max_unk = prm->max_unk;
    ex.pfmax = w.step.pfmax;
    gp.pfmax = w.step.pfmax;
  }
  HIP_TRY(beam_init(bp, m->cfg.bos_id, st));
  if (coverage) HIP_TRY(fill_f32(w.cov[0], (size_t)B * K * S, 0.f, st));
  const int every = prm->check_every > 0 ? prm->check_every : (T <= 32 ? 1 : 8);
  if (!m->done_host) {
    HIP_TRY(hipHostMalloc((void**)&m->done_host, 2 * sizeof(int32_t), hipHostMallocDefault));
    for (auto& e : m->done_ev) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  } else {
    // a search that returned early on an error may have left a count copy queued (possibly on another
    // stream): it must land before this search's copies reuse the two slots
    for (auto& e : m->done_ev) HIP_TRY(hipEventSynchronize(e));
  }
  int cur = 0, nchk = 0;
  for (int t = 1; t <= T; ++t) {
    // coverage of the rows' hypotheses: the parents' coverage (previous layout) plus this step's weights
    const Coverage cv{w.cov[cur], w.cov[cur ^ 1], bp.parent, prm->beta, w.cp};
    ex.cov = coverage ? &cv : nullptr;
    rc = decode_compute(m, w.enc, B, S, K, w.st[cur], w.st[cur ^ 1], bp.tok, bp.parent, 2, nullptr, nullptr,
                        nullptr, nullptr, w.step, st, ex);
    if (rc) return rc;
    time_begin(m, st, ONMT_KERNEL_BEAM);
    HIP_TRY(beam_step(bp, gp, t, st));
    time_end(m, st, ONMT_KERNEL_BEAM);
    cur ^= 1;
    if (t < T && t % every == 0) {
      // this step's done count goes to the host asynchronously and the host waits only for the previous
      // check's, so a check period of steps stays queued on the device; a finished batch runs at most one
      // extra period, in which the beam step leaves every finished sentence unchanged
      const int slot = nchk & 1;
      HIP_TRY(hipMemcpyAsync(m->done_host + slot, bp.done_count, sizeof(int32_t), hipMemcpyDeviceToHost, st));
      HIP_TRY(hipEventRecord(m->done_ev[slot], st));
      if (nchk++ > 0) {
        HIP_TRY(hipEventSynchronize(m->done_ev[slot ^ 1]));
        if (m->done_host[slot ^ 1] >= B) break;
      }
    }
  }
  HIP_TRY(backtrack(bp, out_tok, out_len, out_raw, out_norm, out_tok_logp, out_align, st));
  if (trace) HIP_TRY(hipMemcpyAsync(trace->steps, bp.steps, sizeof(int32_t) * B, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipStreamSynchronize(st));
  if (m->prof) time_collect(m);
  return ONMT_OK;
}

int onmt_replace_unk(onmt_model* m, const int32_t* src, int B, int S, const int32_t* out_tok, const int32_t* out_len,
                     const int32_t* out_align, int T, int32_t* out_src, void* stream) {
  if (!m || !src || !out_tok || !out_len || !out_align || !out_src) return fail(ONMT_EINVAL, "NULL argument");
  if (B < 1 || S < 1 || T < 1) return fail(ONMT_EINVAL, "B, S_max and max_len must be >= 1");
  if ((long long)B * T > (1LL << 30) || (long long)B * S > (1LL << 30)) return fail(ONMT_EUNSUPPORTED, "batch too large");
  HIP_TRY(replace_unk(src, B, S, out_tok, out_len, out_align, T, m->cfg.unk_id, out_src, (hipStream_t)stream));
  return ONMT_OK;
}

size_t onmt_score_ws_bytes(const onmt_model* m, int B, int S, int T) {
  if (!m || B < 1 || S < 1 || T < 1) return 0;
  return score_layout(m->d, B, S, T, nullptr, nullptr);
}

int onmt_score(onmt_model* m, const int32_t* src, const int32_t* len, int B, int S, const int32_t* tgt,
               const int32_t* tgt_len, int T, void* ws, size_t ws_bytes, float* out_logp, double* out_nll,
               void* stream) {
  if (!m || !ws || !tgt || !tgt_len) return fail(ONMT_EINVAL, "NULL argument");
  if (!out_logp || !out_nll) return fail(ONMT_EINVAL, "NULL output pointer");
  if (B < 1 || S < 1) return fail(ONMT_EINVAL, "B and S_max must be >= 1");
  if (T < 1 || T > 100000) return fail(ONMT_EINVAL, "T_max %d outside [1, 100000]", T);
  int rc = check_beam(m, S, 1);
  if (rc) return rc;
  if ((rc = check_ws_limits(m->d, B, S, 1, T))) return rc;
  if (ws_bytes < score_layout(m->d, B, S, T, nullptr, nullptr)) return fail(ONMT_ESIZE, "score workspace too small");
  hipStream_t st = (hipStream_t)stream;
  ScoreWs w;
  score_layout(m->d, B, S, T, (char*)ws, &w);
  int mx = 0;
  rc = check_len_src(m, src, len, B, S, st, &mx, w.enc.src, w.enc.rowmap);
  if (rc) return rc;
  // targets: validated on the host, then laid out per step (decoder input and predicted token)
  std::vector<int32_t> ht((size_t)B * T), hl(B);
  HIP_TRY(hipMemcpyAsync(hl.data(), tgt_len, sizeof(int32_t) * B, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipMemcpyAsync(ht.data(), tgt, sizeof(int32_t) * ht.size(), hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  int steps = 0;
  for (int b = 0; b < B; ++b) {
    if (hl[b] < 1 || hl[b] > T) return fail(ONMT_EINVAL, "tgt_len[%d] = %d outside [1, %d]", b, hl[b], T);
    steps = hl[b] > steps ? hl[b] : steps;
    for (int t = 0; t < hl[b]; ++t) {
      const int v = ht[(size_t)b * T + t];
      if (v < 0 || v >= m->cfg.tgt_vocab)
        return fail(ONMT_EINVAL, "tgt[%d, %d] = %d outside [0, %d)", b, t, v, m->cfg.tgt_vocab);
    }
  }
  std::vector<int32_t> in((size_t)T * B), want((size_t)T * B);
  for (int t = 0; t < T; ++t)
    for (int b = 0; b < B; ++b) {
      const bool on = t < hl[b];
      in[(size_t)t * B + b] = !on ? m->cfg.pad_id : (t == 0 ? m->cfg.bos_id : ht[(size_t)b * T + t - 1]);
      want[(size_t)t * B + b] = on ? ht[(size_t)b * T + t] : 0;
    }
  HIP_TRY(hipMemcpyAsync(w.in_tok, in.data(), sizeof(int32_t) * in.size(), hipMemcpyHostToDevice, st));
  HIP_TRY(hipMemcpyAsync(w.want, want.data(), sizeof(int32_t) * want.size(), hipMemcpyHostToDevice, st));
  HIP_TRY(hipMemcpyAsync(w.tlen, hl.data(), sizeof(int32_t) * B, hipMemcpyHostToDevice, st));

  rc = encode_compute(m, src, len, B, S, mx, w.enc, st);
  if (rc) return rc;
  rc = decode_init_compute(m, w.enc, B, 1, w.st[0], st);
  if (rc) return rc;
  HIP_TRY(fill_f32(out_logp, (size_t)B * T, 0.f, st));
  // the recurrence step by step (input feeding makes each step depend on the previous attentional
  // vector); every step's attentional vector is kept for the generator
  const Dims& d = m->d;
  int cur = 0;
  for (int t = 0; t < steps; ++t) {
    State in = w.st[cur], out = w.st[cur ^ 1];
    if (t > 0) {
      in.feed = w.feeds + (size_t)(t - 1) * B * d.H;
      if (d.bf16) {
        in.feed_hi = w.feeds_hi + (size_t)(t - 1) * B * d.pad(d.H);
        in.feed_lo = w.feeds_lo + (size_t)(t - 1) * B * d.pad(d.H);
        in.feed_lo2 = w.feeds_lo2 + (size_t)(t - 1) * B * d.pad(d.H);
      }
    }
    out.feed = w.feeds + (size_t)t * B * d.H;
    StepExtras ex;
    {
      ex.feed_hi = w.feeds_hi + (size_t)t * B * d.pad(d.H);
      ex.feed_lo = w.feeds_lo + (size_t)t * B * d.pad(d.H);
      ex.feed_lo2 = w.feeds_lo2 + (size_t)t * B * d.pad(d.H);
    }
    rc = decode_compute(m, w.enc, B, S, 1, in, out, w.in_tok + (size_t)t * B, nullptr, 3, nullptr, nullptr, nullptr,
                        nullptr, w.step, st, ex);
    if (rc) return rc;
    cur ^= 1;
  }
  // one generator pass over the steps * B rows: per-tile max and sum of exponentials, and the target's logit
  {
    const int M = steps * B;
    AOp a{};
    a.M = M;
    a.nseg = 1;
    a.seg[0] = seg(w.feeds, nullptr, M, d.H, d.H, d.pad(d.H), 0);
    GenParams gp{};
    gp.bias = m->b_s;
    gp.V = d.Vt;
    gp.K = 0;
    gp.ntiles = w.step.ntiles;
    gp.pmax = w.gpmax;
    gp.psum = w.gpsum;
    gp.want = w.want;
    gp.want_logit = w.want_logit;
    time_begin(m, st);
    if (d.bf16 || gemm_gen_split_rows(M))
      HIP_TRY(gemm_gen_split(GenSplitA{w.feeds_hi, w.feeds_lo, M, d.pad(d.H), d.pad(d.H), w.feeds_lo2}, bop(m->W_s),
                             d.gwp, gp, st));
    else
      HIP_TRY(gemm_gen(a, bop(m->W_s32), gp, st));
    time_end(m, st);
    HIP_TRY(score_rows(w.gpmax, w.gpsum, w.step.ntiles, w.want_logit, w.tlen, B, steps, out_logp, T, w.nll, st));
  }
  HIP_TRY(hipMemcpyAsync(out_nll, w.nll, sizeof(double) * B, hipMemcpyDeviceToDevice, st));
  HIP_TRY(hipStreamSynchronize(st));
  if (m->prof) time_collect(m);
  return ONMT_OK;
}

int onmt_profile_enable(onmt_model* m, int every, unsigned kinds) {
  if (!m) return fail(ONMT_EINVAL, "model is NULL");
  if (every < 0) return fail(ONMT_EINVAL, "timing period must be >= 0");
  if (kinds & ~(unsigned)ONMT_KERNEL_ALL) return fail(ONMT_EINVAL, "kernel kind mask 0x%x unknown", kinds);
  m->prof = every;
  m->prof_kinds = kinds;
  for (auto& q : m->prof_seq) q = 0;
  return ONMT_OK;
}

int onmt_profile_read_kernel(onmt_model* m, int kind, int* n, double* ms, int reset) {
  if (!m || !n || !ms) return fail(ONMT_EINVAL, "NULL argument");
  if (kind < 0 || kind >= ONMT_KERNEL_KINDS) return fail(ONMT_EINVAL, "kernel kind %d unknown", kind);
  *n = m->prof_n[kind];
  *ms = m->prof_ms[kind];
  if (reset) {
    m->prof_n[kind] = 0;
    m->prof_ms[kind] = 0.0;
  }
  return ONMT_OK;
}

int onmt_profile_read(onmt_model* m, int* n, double* ms, int reset) {
  return onmt_profile_read_kernel(m, ONMT_KERNEL_GENERATOR, n, ms, reset);
}

}  // extern "C"
