"""Plain CPU oracle for attention-based LSTM encoder-decoder beam-search translation.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run this module. The product
path (the HIP library and its Python binding) never calls it and shares no code
with it; the two meet only in the seeded inputs of the ``workloads`` package.

Everything is float64 NumPy (model_from(..., dtype=np.float32) gives an fp32 copy whose products run in
single precision, used only to time the CPU baseline; beam scores stay fp64), written for a reader
holding the OpenNMT paper
(Klein et al., arXiv 1805.11462). The paper names the pieces but prints no
equations, so the standard published forms of the cited works are written out
here; every place where the paper is silent carries its reading (R1..R20, the
same numbering as the design notes).

What the paper fixes, and where:

* Section 2 (Background): the conditional language model
  ``p(w_1:T | x) = prod_t p(w_t | w_1:t-1, x)``; a source encoder RNN maps word
  vectors to hidden vectors h_1..h_S; a target decoder RNN combines its hidden
  state with the source vectors through an attention pooling layer; a softmax
  layer gives the next-word distribution.
* Section 2, items (a)-(d): gated cell (LSTM), stacked layers, input feeding
  (previous attention vector fed back with the predicted word), beam search.
* Figure 1(a) caption: the encoder's final step initialises the target RNN;
  attention is combined with the current hidden state to make the prediction,
  which is fed back.
* Section 4.2 ("Extensible Data, Models, and Search"): attention types
  general / dot / concat; beam search with length normalisation.
* Tables 3 and 4 captions: bidirectional RNN encoders.

Readings where the paper is silent (R-numbers):

R1  LSTM: forget-gate LSTM without peepholes, one bias per gate, gate order
    (i, f, g, o), sigma(x) = 1 / (1 + exp(-x)).
R2  Encoder initial state is zero.
R3  No BOS/EOS is added to the source.
R4  Padding is packed: pad positions never update the state; memory rows at
    pads are 0; attention weight at pads is exactly 0.
R5  Bidirectional final state handed to the decoder, per layer:
    [forward state after the last real token ; backward state after token 0].
R6  "general" score e_s = q^T W_a m_s with no bias; attentional vector
    tanh(W_c [ctx ; q]) with no bias.
R7  Input feed starts at 0; decoder layer-1 input is [embedding ; feed].
R8  Generator has a bias; no token is masked.
R9  Beam: scores s_0 = 0, s_1.. = -inf; candidates cand = s_k + logp_k(w) in
    fp64; top-K finite candidates, ties to the smaller flat index k*V + w; a
    chosen EOS (or any choice at t = T_max) enters the finished pool; the rest
    fill live slots in rank order; stop when t = T_max, or no live slot, or the
    pool's best normalised score >= best live score / lp(T_max).
R10 GNMT length penalty lp(n) = ((5 + n) / 6) ** alpha, applied to finished
    hypotheses only; n counts EOS.
R11 max_len = most generated tokens, EOS included.
R12 bf16 workloads: the oracle runs in fp64 on the bf16-rounded weights. (The GPU path keeps bf16
    weights and fp32 accumulation; it carries each activation entering a product as two bf16 terms,
    which keeps the chaotic decoder recurrence within the bf16 tolerance over full-length outputs.)
R15 Throughput counts target tokens of the 1-best, EOS included.
R18 Hypothesis filters (Section 4.2 names a limit on unknown words and word-level constraints on the
    search): a candidate whose token is in the banned set, or which would be an UNK beyond
    max_unk UNKs, is not a candidate (log-probs stay normalised over the whole vocabulary).
R19 Unknown-word replacement (Section 4.2 OOV handling, citing Luong et al. 2015b): every output token
    is aligned to the source position with the largest attention weight of its step (smaller position
    on ties); an UNK output takes the source token there.
R20 Attention types (Section 4.2 names general, dot product and concatenation, citing Luong et al.
    2015 and Britz et al. 2017), all without biases: "dot" e_s = q^T m_s (the memory width equals H);
    "concat" e_s = v_a^T tanh(W_a [q ; m_s]) with W_a [H, H + Hm] (attention size H, query columns
    first) and v_a [H]. Softmax, context and the attentional vector are the same for every type.
R17 Coverage normalisation (named with length normalisation in Section 4.2, citing GNMT): a finished
    hypothesis is ranked by raw / lp(n) + beta * sum over the real source positions of
    log(min(c_i, 1)), c_i = the attention it put on position i summed over its steps (EOS included);
    live hypotheses are ranked by raw score only, as with the length penalty. Since the penalty is
    <= 0, the stop rule's bound stays exact.
R16 Near-ties: any choice within the tolerance is a correct result.

Pins (tests that tie this file to the mathematics rather than to itself) live
in ``tests/test_oracle_*.py``. The whole pipeline against the paper's printed
results is parity unpinned: the paper prints only BLEU and speed on data and
trained weights that are not available.
"""

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
import os

import numpy as np

from workloads.configs import PAD_ID, UNK_ID, BOS_ID, EOS_ID

F64 = np.float64


# --------------------------------------------------------------------------
# Model container
# --------------------------------------------------------------------------

@dataclass
class Model:
    """fp64 copy of the weights plus the shape fields the oracle needs."""
    enc_layers: int
    dec_layers: int
    bidirectional: bool
    emb: int
    hidden: int
    src_vocab: int
    tgt_vocab: int
    w: dict = field(repr=False)
    attn: str = "general"

    @property
    def enc_hidden(self):
        return self.hidden // 2 if self.bidirectional else self.hidden


def model_from(workload, weights, dtype=F64) -> Model:
    """The oracle's model; activations follow the weights' dtype (fp64 unless asked otherwise)."""
    return Model(workload.enc_layers, workload.dec_layers, workload.bidirectional,
                 workload.emb, workload.hidden, workload.src_vocab, workload.tgt_vocab,
                 {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}, workload.attn)


# --------------------------------------------------------------------------
# Cell (Section 2 item (a); R1)
# --------------------------------------------------------------------------

def sigmoid(x):
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


def lstm_cell(W, b, x, h, c):
    """One LSTM step on rows of x, h, c.

    z = W[:, :in] x + W[:, in:] h + b ; (z_i, z_f, z_g, z_o) blocks of z;
    c' = sigma(z_f) * c + sigma(z_i) * tanh(z_g) ; h' = sigma(z_o) * tanh(c').
    """
    n_in = x.shape[-1]
    Hl = h.shape[-1]
    z = x @ W[:, :n_in].T + h @ W[:, n_in:].T + b
    i = sigmoid(z[..., 0 * Hl:1 * Hl])
    f = sigmoid(z[..., 1 * Hl:2 * Hl])
    g = np.tanh(z[..., 2 * Hl:3 * Hl])
    o = sigmoid(z[..., 3 * Hl:4 * Hl])
    c_new = f * c + i * g
    h_new = o * np.tanh(c_new)
    return h_new, c_new


# --------------------------------------------------------------------------
# Encoder (Section 2; Figure 1(a); stacked layers item (b); bi-RNN Tables 3-4)
# --------------------------------------------------------------------------

@dataclass
class Encoded:
    memory: np.ndarray      # [B, S, Hm], zero at pads (R4)
    mask: np.ndarray        # [B, S] bool, True on real positions
    final_h: list           # per layer [B, H] (R5 for bi)
    final_c: list


def run_direction(W, b, x, real, reverse):
    """One LSTM direction over [B, S, in] with packed padding (R2, R4)."""
    B, S, _ = x.shape
    Hl = W.shape[0] // 4
    h = np.zeros((B, Hl), x.dtype)
    c = np.zeros((B, Hl), x.dtype)
    out = np.zeros((B, S, Hl), x.dtype)
    steps = range(S - 1, -1, -1) if reverse else range(S)
    for s in steps:
        h_new, c_new = lstm_cell(W, b, x[:, s], h, c)
        act = real[:, s][:, None]
        h = np.where(act, h_new, h)
        c = np.where(act, c_new, c)
        out[:, s] = np.where(act, h_new, 0.0)
    return out, h, c


def encode(m: Model, src, lens) -> Encoded:
    src = np.asarray(src)
    lens = np.asarray(lens)
    B, S = src.shape
    real = np.arange(S)[None, :] < lens[:, None]
    x = m.w["E_src"][src]                                   # word vectors (R3: no BOS/EOS)
    final_h, final_c = [], []
    for l in range(m.enc_layers):
        outs, hs, cs = [], [], []
        for d in (("fwd", "bwd") if m.bidirectional else ("fwd",)):
            o, h, c = run_direction(m.w[f"enc{l}_{d}_W"], m.w[f"enc{l}_{d}_b"], x, real,
                                    reverse=(d == "bwd"))
            outs.append(o)
            hs.append(h)
            cs.append(c)
        x = np.concatenate(outs, axis=-1)
        final_h.append(np.concatenate(hs, axis=-1))
        final_c.append(np.concatenate(cs, axis=-1))
    return Encoded(x, real, final_h, final_c)


# --------------------------------------------------------------------------
# Decoder step (Section 2; items (b), (c); Figure 1(a); Section 4.2 attention)
# --------------------------------------------------------------------------

@dataclass
class State:
    h: list      # per layer [N, H]
    c: list      # per layer [N, H]
    feed: np.ndarray   # [N, H], the previous attentional vector (R7)

    def take(self, rows):
        rows = np.asarray(rows)
        return State([a[rows] for a in self.h], [a[rows] for a in self.c], self.feed[rows])


def init_state(m: Model, enc: Encoded, K: int) -> State:
    """Decoder state from the encoder's final step (Figure 1(a)), copied to K beam rows."""
    rep = lambda a: np.repeat(a, K, axis=0)
    N = enc.memory.shape[0] * K
    return State([rep(h) for h in enc.final_h], [rep(c) for c in enc.final_c],
                 np.zeros((N, m.hidden), enc.memory.dtype))


def attention_scores(m: Model, q, memory):
    """Raw scores e [N, S] of rows q [N, H] against per-row memory [N, S, Hm] (R6, R20)."""
    if m.attn == "general":
        Wm = memory @ m.w["W_a"].T                           # W_a m_s, [N, S, H]
        return np.einsum("nh,nsh->ns", q, Wm)
    if m.attn == "dot":
        return np.einsum("nh,nsh->ns", q, memory)
    if m.attn == "concat":
        N, S, _ = memory.shape
        qm = np.concatenate([np.broadcast_to(q[:, None, :], (N, S, q.shape[-1])), memory], axis=-1)
        return np.tanh(qm @ m.w["W_a"].T) @ m.w["v_a"]       # v_a . tanh(W_a [q ; m_s])
    raise ValueError(f"unknown attention type {m.attn!r}")


def attention(m: Model, q, memory, mask):
    """Global attention for rows q [N, H] over their sentences' memory (type m.attn).

    memory [N, S, Hm] and mask [N, S] are already per row. Returns (a [N, S],
    ctx [N, Hm], h_tilde [N, H]). R4, R6, R20.
    """
    e = np.where(mask, attention_scores(m, q, memory), -np.inf)
    e_max = e.max(axis=1, keepdims=True)
    p = np.exp(e - e_max)                                    # exactly 0 on pads
    a = p / p.sum(axis=1, keepdims=True)
    ctx = np.einsum("ns,nsh->nh", a, memory)
    h_tilde = np.tanh(np.concatenate([ctx, q], axis=-1) @ m.w["W_c"].T)
    return a, ctx, h_tilde


def log_softmax(z):
    z_max = z.max(axis=-1, keepdims=True)
    return z - (z_max + np.log(np.exp(z - z_max).sum(axis=-1, keepdims=True)))


def rows_in_parallel(fn, x):
    """fn applied to blocks of rows of x in worker threads (NumPy releases the GIL inside its ufuncs).
    fn must treat rows independently; each row's arithmetic is then that of fn(x) and so is the result."""
    n = x.shape[0]
    workers = min(len(os.sched_getaffinity(0)), 16, n // 16)
    if workers <= 1:
        return fn(x)
    bounds = np.linspace(0, n, workers + 1).astype(int)
    with ThreadPoolExecutor(workers) as ex:
        parts = list(ex.map(lambda i: fn(x[bounds[i]:bounds[i + 1]]), range(workers)))
    return np.concatenate(parts)


def generator(m: Model, h_tilde):
    """Next-word log-distribution over the whole target vocabulary (Section 2; R8)."""
    return rows_in_parallel(log_softmax, h_tilde @ m.w["W_s"].T + m.w["b_s"])


def decode_step(m: Model, enc: Encoded, st: State, prev_tok, row_sentence):
    """p(w_t | w_<t, x) for every row: returns (new state, logp [N, V], attention [N, S])."""
    x = np.concatenate([m.w["E_tgt"][np.asarray(prev_tok)], st.feed], axis=-1)
    hs, cs = [], []
    for l in range(m.dec_layers):
        h, c = lstm_cell(m.w[f"dec{l}_W"], m.w[f"dec{l}_b"], x, st.h[l], st.c[l])
        hs.append(h)
        cs.append(c)
        x = h
    rows = np.asarray(row_sentence)
    a, _, h_tilde = attention(m, x, enc.memory[rows], enc.mask[rows])
    return State(hs, cs, h_tilde), generator(m, h_tilde), a


# --------------------------------------------------------------------------
# Search (Section 2 item (d); Section 4.2 length normalisation; R9-R11)
# --------------------------------------------------------------------------

def length_penalty(n, alpha):
    """GNMT length penalty ((5 + n) / 6) ** alpha (R10)."""
    return ((5.0 + n) / 6.0) ** alpha


@dataclass
class Hyp:
    tokens: list
    logps: list
    cov: np.ndarray = None   # attention summed over the hypothesis's steps, per source position (R17)
    align: list = None       # per token: source position of the largest attention weight (R19)
    n_unk: int = 0           # UNK tokens so far (R18)


def coverage_penalty(cov, n_src, beta):
    """GNMT coverage penalty beta * sum_{i < n_src} log(min(cov_i, 1)) (Section 4.2 names attention
    coverage normalisation beside length normalisation; R17). 0 when beta is 0."""
    if beta == 0.0:
        return 0.0
    c = np.minimum(np.asarray(cov, F64)[:n_src], 1.0)
    with np.errstate(divide="ignore"):
        return float(beta * np.log(c).sum())


@dataclass
class Result:
    tokens: list            # 1-best tokens per sentence (BOS excluded, EOS included if chosen)
    raw: np.ndarray         # [B] summed log-prob
    norm: np.ndarray        # [B] raw / lp(len)
    logps: list             # per-token log-probs of the 1-best
    steps: np.ndarray       # [B] step after which the sentence was done
    trace: dict = None      # per step: chosen (slot, token, cand) by rank, and each sentence's margin
    align: list = None      # per token of the 1-best: argmax source position of its step's attention
    margin: np.ndarray = None   # [B] smallest decision margin of the sentence's run (see beam_search)


def allowed(w, n_unk, banned, max_unk):
    """Hypothesis filter (Section 4.2 names a limit on unknown words and word-level constraints on the
    search; R18): a banned token, or an UNK beyond max_unk UNKs (max_unk < 0: no limit),
    cannot extend a hypothesis."""
    if w in banned:
        return False
    return not (max_unk >= 0 and w == UNK_ID and n_unk >= max_unk)


def attention_argmax(a, n_src):
    """Source position with the largest attention weight, the smaller position on ties (R19)."""
    return int(np.argmax(np.asarray(a)[:n_src]))


def replace_unk(tokens, align, src_row, unk_id=None):
    """Unknown-word replacement (Section 4.2 OOV handling): every UNK output token takes the source token at
    its aligned position. Source and target ids share no vocabulary here, so the result marks a copied
    source token as ('src', id) and keeps other tokens as ('tgt', id)."""
    unk = UNK_ID if unk_id is None else unk_id
    return [("src", int(src_row[a])) if t == unk else ("tgt", int(t)) for t, a in zip(tokens, align)]


def beam_search(m: Model, src, lens, K, max_len, alpha=0.0, stop_rule=True, record=False, beta=0.0,
                banned=(), max_unk=-1):
    """Beam search for every sentence, one set of K slots per sentence.

    Sentences are independent; the decoder runs all B*K rows at once only to
    share the matrix products. A finished hypothesis is ranked by
    raw / lp(n) + coverage_penalty (R10, R17).

    ``Result.margin[b]`` is the smallest gap between the two quantities compared by any decision of
    sentence b's run that can change its output: the K-th against the (K+1)-th finite candidate of every
    step (which hypotheses survive; the order inside the chosen K only renumbers slots), the stop rule's
    best finished score against the best live score / lp(max_len), and the best finished entry against the
    second best. Another implementation whose scores differ from these by less than half the margin makes
    every decision the same way, so its output tokens must be identical (R16). With ``record`` the trace
    also holds, per step, each sentence's margin of that step's selection and stop decisions (inf once
    the sentence is done): the other implementation's choices must be the same at every step before the
    first one whose margin is within its tolerance.
    """
    src = np.asarray(src)
    lens = np.asarray(lens)
    B, S = src.shape
    V = m.tgt_vocab
    enc = encode(m, src, lens)
    st = init_state(m, enc, K)
    row_sentence = np.repeat(np.arange(B), K)
    scores = np.full((B, K), -np.inf)
    scores[:, 0] = 0.0
    banned = set(int(x) for x in banned)
    filtering = bool(banned) or max_unk >= 0
    hyps = [[Hyp([], [], np.zeros(S, F64), []) for _ in range(K)] for _ in range(B)]
    tok = np.full(B * K, BOS_ID, np.int64)
    done = np.zeros(B, bool)
    steps = np.zeros(B, np.int64)
    best = [None] * B              # (norm, raw, Hyp)
    pool_norms = [[] for _ in range(B)]
    margin = np.full(B, np.inf)
    trace = {"slot": [], "tok": [], "cand": [], "margin": []} if record else None
    lp_max = length_penalty(max_len, alpha)
    for t in range(1, max_len + 1):
        st_new, logp, attn = decode_step(m, enc, st, tok, row_sentence)
        parent = np.arange(B * K)
        new_tok = np.full(B * K, PAD_ID, np.int64)
        if record:
            t_slot = np.full((B, K), -1, np.int64)
            t_tok = np.full((B, K), -1, np.int64)
            t_cand = np.full((B, K), -np.inf)
            t_margin = np.full(B, np.inf)
        for b in range(B):
            if done[b]:
                continue
            rows = slice(b * K, (b + 1) * K)
            cand = scores[b][:, None] + logp[rows]              # [K, V]; dead slots stay -inf
            if filtering:                                       # R18, the same rule as allowed()
                if banned:
                    cand[:, sorted(banned)] = -np.inf
                for k in range(K):
                    if max_unk >= 0 and hyps[b][k].n_unk >= max_unk:
                        cand[k, UNK_ID] = -np.inf
            flat = cand.ravel()
            order = np.argsort(-flat, kind="stable")            # ties: smaller flat index first
            chosen = [i for i in order[:K] if np.isfinite(flat[i])]
            step_margin = np.inf
            if order.size > K and np.isfinite(flat[order[K]]):      # the selection boundary
                step_margin = flat[order[K - 1]] - flat[order[K]]
            new_scores = np.full(K, -np.inf)
            new_hyps = [Hyp([], [], np.zeros(S, F64), []) for _ in range(K)]
            j = 0
            for rank, i in enumerate(chosen):
                k, w = divmod(int(i), V)
                hyp = Hyp(hyps[b][k].tokens + [w], hyps[b][k].logps + [logp[b * K + k, w]],
                          hyps[b][k].cov + attn[b * K + k],
                          hyps[b][k].align + [attention_argmax(attn[b * K + k], lens[b])],
                          hyps[b][k].n_unk + (1 if w == UNK_ID else 0))
                if record:
                    t_slot[b, rank], t_tok[b, rank], t_cand[b, rank] = k, w, flat[i]
                if w == EOS_ID or t == max_len:
                    norm = flat[i] / length_penalty(t, alpha) + coverage_penalty(hyp.cov, lens[b], beta)
                    pool_norms[b].append(norm)
                    if best[b] is None or norm > best[b][0]:
                        best[b] = (norm, flat[i], hyp)
                else:
                    new_hyps[j] = hyp
                    new_scores[j] = flat[i]
                    parent[b * K + j] = b * K + k
                    new_tok[b * K + j] = w
                    j += 1
            scores[b] = new_scores
            hyps[b] = new_hyps
            live = new_scores[np.isfinite(new_scores)]
            if stop_rule and best[b] is not None and live.size and t < max_len:
                step_margin = min(step_margin, abs(best[b][0] - live.max() / lp_max))
            margin[b] = min(margin[b], step_margin)
            if record:
                t_margin[b] = step_margin
            if (t == max_len or live.size == 0
                    or (stop_rule and best[b] is not None and best[b][0] >= live.max() / lp_max)):
                done[b] = True
                steps[b] = t
        if record:
            trace["slot"].append(t_slot)
            trace["tok"].append(t_tok)
            trace["cand"].append(t_cand)
            trace["margin"].append(t_margin)
        st = st_new.take(parent)
        tok = new_tok
        if done.all():
            break
    for b in range(B):                                      # the final argmax over the pool
        if len(pool_norms[b]) > 1:
            top = sorted(pool_norms[b], reverse=True)
            margin[b] = min(margin[b], top[0] - top[1])
    return Result([bst[2].tokens for bst in best],
                  np.array([bst[1] for bst in best]), np.array([bst[0] for bst in best]),
                  [bst[2].logps for bst in best], steps, trace, [bst[2].align for bst in best], margin)


def greedy(m: Model, src, lens, max_len):
    """Argmax decoding (smallest id on ties), stopping at EOS or max_len. Separate code from beam_search."""
    src = np.asarray(src)
    B = src.shape[0]
    enc = encode(m, src, lens)
    st = init_state(m, enc, 1)
    tok = np.full(B, BOS_ID, np.int64)
    out = [[] for _ in range(B)]
    lps = [[] for _ in range(B)]
    finished = np.zeros(B, bool)
    for _ in range(max_len):
        st, logp, _ = decode_step(m, enc, st, tok, np.arange(B))
        tok = logp.argmax(axis=1)
        for b in range(B):
            if not finished[b]:
                out[b].append(int(tok[b]))
                lps[b].append(logp[b, tok[b]])
                finished[b] = tok[b] == EOS_ID
        if finished.all():
            break
    return out, np.array([sum(x) for x in lps])


def score_forced(m: Model, src_row, n_src, target):
    """Teacher-forced per-token log-probs of ``target`` for one sentence, from scratch."""
    src_row = np.asarray(src_row)[None, :]
    enc = encode(m, src_row, np.array([n_src]))
    st = init_state(m, enc, 1)
    prev = BOS_ID
    out = []
    for w in target:
        st, logp, _ = decode_step(m, enc, st, np.array([prev]), np.array([0]))
        out.append(logp[0, w])
        prev = w
    return np.array(out)


def score_batch(m: Model, src, lens, tgt, tgt_len):
    """Teacher-forced scoring of a batch: the per-token terms of the training objective.

    Section 2: the model is trained to minimise the negative log-likelihood of the corpus under
    p(w_1:T | x) = prod_t p(w_t | w_<t, x). Sentence b's decoder is fed BOS, tgt[b, 0], ... and scores
    tgt[b, t] at step t. Returns (logp [B, T] with 0 from tgt_len[b] on, nll [B] = -sum of the row).
    """
    src = np.asarray(src)
    tgt = np.asarray(tgt)
    tgt_len = np.asarray(tgt_len)
    B, T = tgt.shape
    enc = encode(m, src, np.asarray(lens))
    st = init_state(m, enc, 1)
    logp = np.zeros((B, T), F64)
    prev = np.full(B, BOS_ID)
    rows = np.arange(B)
    for t in range(int(tgt_len.max())):
        st, lp, _ = decode_step(m, enc, st, prev, rows)
        on = t < tgt_len
        logp[on, t] = lp[rows[on], tgt[on, t]]
        prev = np.where(on, tgt[:, t], PAD_ID)
    return logp, -logp.sum(axis=1)


def coverage_forced(m: Model, src_row, n_src, target):
    """Attention summed over the teacher-forced steps of ``target`` for one sentence, per source position."""
    src_row = np.asarray(src_row)[None, :]
    enc = encode(m, src_row, np.array([n_src]))
    st = init_state(m, enc, 1)
    prev = BOS_ID
    cov = np.zeros(src_row.shape[1], F64)
    for w in target:
        st, _, a = decode_step(m, enc, st, np.array([prev]), np.array([0]))
        cov += a[0]
        prev = w
    return cov


def brute_force(m: Model, src_row, n_src, max_len, alpha=0.0, beta=0.0, banned=(), max_unk=-1):
    """Best normalised score over every output sequence (exhaustive; tiny vocabularies only).

    Sequences: those whose first EOS ends them at length n <= max_len, plus
    every EOS-free sequence of length max_len. Returns (tokens, raw, norm).
    """
    V = m.tgt_vocab
    best = None
    stack = [[]]
    while stack:
        prefix = stack.pop()
        for w in range(V):
            if not allowed(w, sum(1 for x in prefix if x == UNK_ID), set(banned), max_unk):
                continue
            seq = prefix + [w]
            if w == EOS_ID or len(seq) == max_len:
                raw = score_forced(m, src_row, n_src, seq).sum()
                norm = raw / length_penalty(len(seq), alpha)
                if beta:
                    norm += coverage_penalty(coverage_forced(m, src_row, n_src, seq), n_src, beta)
                if best is None or norm > best[2]:
                    best = (seq, raw, norm)
            else:
                stack.append(seq)
    return best


# --------------------------------------------------------------------------
# Replay of a recorded search (parity protocol for near-ties, R16)
# --------------------------------------------------------------------------

def chosen_hypotheses(trace, b, t_end, K):
    """The token sequences chosen at each step 1..t_end of sentence b in a record by rank (slot, tok):
    a list (per step) of sets of tuples. Slots are numbered as R9 fills them (live choices in rank order)."""
    live = {0: ()}
    out = []
    for t in range(1, t_end + 1):
        slot = np.asarray(trace["slot"][t - 1][b])
        tok = np.asarray(trace["tok"][t - 1][b])
        step, nxt = set(), {}
        for r in range(K):
            k = int(slot[r])
            if k < 0 or k not in live:
                continue
            seq = live[k] + (int(tok[r]),)
            step.add(seq)
            if int(tok[r]) != EOS_ID:
                nxt[len(nxt)] = seq
        out.append(step)
        live = nxt
    return out


def prefix_agreement(oracle_trace, other_trace, sentences, K, tol):
    """Per-step free-run parity (R16): for each sentence, the other implementation must choose the same
    hypotheses as the oracle at every step before the first step whose recorded oracle margin is within
    ``tol`` (ties and near-ties may go either way from there on). Returns (violations, number of steps
    compared per sentence)."""
    bad, n_cmp = [], {}
    T = len(oracle_trace["slot"])
    for b in sentences:
        t_stop = 0
        while t_stop < T and np.asarray(oracle_trace["slot"][t_stop][b])[0] >= 0 \
                and oracle_trace["margin"][t_stop][b] > tol:
            t_stop += 1
        n_cmp[b] = t_stop
        if t_stop == 0:
            continue
        want = chosen_hypotheses(oracle_trace, b, t_stop, K)
        got = chosen_hypotheses(other_trace, b, min(t_stop, len(other_trace["slot"])), K)
        for t, (a, g) in enumerate(zip(want, got), start=1):
            if a != g:
                bad.append(f"b{b} t{t}: chose {len(g - a)} hypotheses the oracle did not, although every "
                           f"oracle margin up to this step exceeds {tol:.3g}")
                break
        else:
            if len(got) < len(want):
                bad.append(f"b{b}: record ends at step {len(got)}, the oracle's agrees to step {t_stop}")
    return bad, n_cmp


def replay_verify(m: Model, src, lens, K, max_len, alpha, trace, tau, sentences=None, steps=None, result=None,
                  beta=0.0):
    """Check another implementation's beam decisions step by step (parity protocol for near-ties, R16).

    ``trace`` holds, per step t (list index t-1), arrays [B, K] by rank: ``slot`` (parent slot, -1 = nothing
    chosen), ``tok`` and ``cand`` (that implementation's fp64 score). The oracle follows the recorded
    decisions, teacher forcing its own fp64 decoder through them (all listed sentences in one batch, like
    beam_search), and keeps the finished pool of R9 on the recorded scores. It checks that
      * every chosen candidate's log-prob agrees with the oracle's within tau;
      * the chosen set is a valid top-K under the oracle's log-probs added to the recorded scores
        (chosen >= K-th - tau, rejected <= K-th + tau);
      * every recorded score stays within t * tau of the oracle's running sum;
      * a chosen EOS (or any choice at max_len) leaves the live slots: the next step's slots are the
        other choices in rank order, so a finished hypothesis kept live shows up there as wrong log-probs
        or scores;
      * the sentence stops exactly when rule (iii) fires on the recorded numbers (no choices recorded
        after that step, some at every step before it; ``steps[b]``, if given, is that step), and the
        same rule on the oracle's running sums agrees wherever its two sides differ by more than t * tau;
      * ``result`` (dict of [B] arrays ``len``, ``raw``, ``norm`` and [B, T] ``tokens``), if given, is the
        pool's best entry by normalised score on the recorded numbers (earlier step, then better rank, on
        ties), and on the oracle's numbers no pool entry beats it by more than t * tau.
    With beta > 0 the coverage penalty of an entry is the oracle's, from the attention along its
    replayed steps. Returns a list of violation strings (empty = pass).
    """
    src = np.asarray(src)
    lens = np.asarray(lens)
    B, S = src.shape
    V = m.tgt_vocab
    sel = list(range(B)) if sentences is None else [int(x) for x in sentences]
    nb = len(sel)
    bad = []
    if nb == 0:
        return bad
    ninf = -np.inf
    enc = encode(m, src[sel], lens[sel])
    st = init_state(m, enc, K)
    row_sentence = np.repeat(np.arange(nb), K)
    lp_max = length_penalty(max_len, alpha)
    s_rec = np.full((nb, K), ninf)        # recorded scores of the live slots
    s_orc = np.full((nb, K), ninf)        # oracle running sums along the same hypotheses
    s_rec[:, 0] = s_orc[:, 0] = 0.0
    toks = [[[] for _ in range(K)] for _ in range(nb)]
    cov = np.zeros((nb, K, S), F64)
    pool = [[] for _ in range(nb)]        # (norm_rec, norm_orc, raw_rec, t, rank, tokens)
    active = np.ones(nb, bool)
    tok = np.full(nb * K, BOS_ID, np.int64)
    T = len(trace["slot"])
    rel = lambda x: 1e-12 * max(1.0, abs(x))
    for t in range(1, T + 1):
        if not active.any():
            break
        st_new, logp, attn = decode_step(m, enc, st, tok, row_sentence)
        parent = np.arange(nb * K)
        new_tok = np.full(nb * K, PAD_ID, np.int64)
        lp_t = length_penalty(t, alpha)
        for i, b in enumerate(sel):
            if not active[i]:
                continue
            slot = np.asarray(trace["slot"][t - 1][b])
            wtok = np.asarray(trace["tok"][t - 1][b])
            cand_rec = np.asarray(trace["cand"][t - 1][b])
            rows = slice(i * K, (i + 1) * K)
            if (slot < 0).all():
                bad.append(f"b{b} t{t}: nothing chosen while the sentence is live")
                active[i] = False
                continue
            oc = s_rec[i][:, None] + logp[rows]               # oracle log-probs on recorded scores
            flat = oc.ravel()
            n_fin = int(np.isfinite(flat).sum())
            kk = min(K, n_fin)
            theta = -np.partition(-flat, kk - 1)[kk - 1]      # the oracle's K-th value
            chosen = set()
            ns_rec = np.full(K, ninf)
            ns_orc = np.full(K, ninf)
            n_toks = [[] for _ in range(K)]
            n_cov = np.zeros((K, S), F64)
            j = 0
            for r in range(K):
                k = int(slot[r])
                if k < 0:
                    continue
                w = int(wtok[r])
                if k >= K or not 0 <= w < V:
                    bad.append(f"b{b} t{t} r{r}: slot {k} / token {w} out of range")
                    continue
                chosen.add(k * V + w)
                if not np.isfinite(s_rec[i, k]):
                    bad.append(f"b{b} t{t} r{r}: chose dead slot {k}")
                    continue
                lpk = logp[i * K + k, w]
                lp_rec = cand_rec[r] - s_rec[i, k]
                if abs(lp_rec - lpk) > tau:
                    bad.append(f"b{b} t{t} r{r}: logp {lp_rec:.6g} vs oracle {lpk:.6g}")
                if oc[k, w] < theta - tau:
                    bad.append(f"b{b} t{t} r{r}: chosen {oc[k, w]:.8g} below K-th {theta:.8g} - tau")
                run = s_orc[i, k] + lpk
                if abs(cand_rec[r] - run) > t * tau:
                    bad.append(f"b{b} t{t} r{r}: score drift {cand_rec[r] - run:.3g}")
                hyp_toks = toks[i][k] + [w]
                hyp_cov = cov[i, k] + attn[i * K + k]
                if w == EOS_ID or t == max_len:
                    cp = coverage_penalty(hyp_cov, lens[b], beta)
                    pool[i].append((cand_rec[r] / lp_t + cp, run / lp_t + cp, cand_rec[r], t, r, hyp_toks))
                else:
                    parent[i * K + j] = i * K + k
                    new_tok[i * K + j] = w
                    ns_rec[j] = cand_rec[r]
                    ns_orc[j] = run
                    n_toks[j] = hyp_toks
                    n_cov[j] = hyp_cov
                    j += 1
            if len(chosen) != kk:
                bad.append(f"b{b} t{t}: {len(chosen)} chosen, expected {kk}")
            masked = oc.copy().ravel()
            if chosen:
                masked[np.fromiter(chosen, np.int64)] = ninf
            if masked.max() > theta + tau:
                bad.append(f"b{b} t{t}: rejected {masked.max():.8g} above K-th {theta:.8g} + tau")
            s_rec[i], s_orc[i], toks[i], cov[i] = ns_rec, ns_orc, n_toks, n_cov
            # rule (iii) on the recorded numbers decides; the oracle's numbers must agree outside t * tau
            stop = t == max_len or j == 0
            if not stop and pool[i]:
                best_rec = max(e[0] for e in pool[i])
                bound_rec = ns_rec[:j].max() / lp_max
                tol = rel(bound_rec) if beta == 0.0 else t * tau
                stop = best_rec >= bound_rec
                if abs(best_rec - bound_rec) <= tol:
                    stop = None                                # a tie within rounding: either is correct
                best_orc = max(e[1] for e in pool[i])
                bound_orc = ns_orc[:j].max() / lp_max
                if stop is not None and (best_orc >= bound_orc) != stop and abs(best_orc - bound_orc) > t * tau:
                    bad.append(f"b{b} t{t}: stop rule {stop} on the recorded scores, {not stop} on the oracle's "
                               f"({best_orc:.10g} vs {bound_orc:.10g})")
            if stop is None:                                   # follow what the implementation did
                stop = (t < T and (np.asarray(trace["slot"][t][b]) < 0).all())
            if stop:
                active[i] = False
                if steps is not None and int(steps[b]) != t:
                    bad.append(f"b{b}: finished at step {int(steps[b])}, rule (iii) fires at step {t}")
                if t < T and not all((np.asarray(trace["slot"][u][b]) < 0).all() for u in range(t, T)):
                    bad.append(f"b{b}: choices recorded after the sentence finished at step {t}")
        st = st_new.take(parent)
        tok = new_tok
    for i, b in enumerate(sel):
        if active[i]:
            bad.append(f"b{b}: the record ends at step {T} before the sentence finished")
        if result is None or not pool[i]:
            continue
        best = None                                            # first maximum in (step, rank) order
        for e in pool[i]:
            if best is None or e[0] > best[0]:
                best = e
        n = int(result["len"][b])
        got = [int(x) for x in np.asarray(result["tokens"][b])[:n]]
        if got != best[5]:
            # a tie within rounding on the recorded numbers leaves either entry correct
            alt = [e for e in pool[i] if e[5] == got]
            if not alt or abs(alt[0][0] - best[0]) > rel(best[0]):
                bad.append(f"b{b}: returned hypothesis is not the pool's best ({n} tokens vs {len(best[5])})")
                continue
            best = alt[0]
        if abs(float(result["raw"][b]) - best[2]) > rel(best[2]):
            bad.append(f"b{b}: returned raw {float(result['raw'][b]):.12g} vs pool entry {best[2]:.12g}")
        if abs(float(result["norm"][b]) - best[0]) > (rel(best[0]) if beta == 0.0 else best[3] * tau):
            bad.append(f"b{b}: returned norm {float(result['norm'][b]):.12g} vs pool entry {best[0]:.12g}")
        top_orc = max(e[1] for e in pool[i])
        if best[1] < top_orc - best[3] * tau:
            bad.append(f"b{b}: on the oracle's numbers the pool's best beats the returned entry by "
                       f"{top_orc - best[1]:.3g}")
    return bad
