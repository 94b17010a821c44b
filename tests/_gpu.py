"""Shared set-up for the GPU parity tests: seeded workloads -> (oracle model, GPU translator, batch)."""

import numpy as np
import torch

import workloads as W
from oracle import onmt_oracle as O

TAU = {"fp32": 1e-4, "bf16": 2e-2}          # per-step log-prob tolerance
ATTN_TOL = {"fp32": 1e-5, "bf16": 1e-2}


def translator_for(w, weights):
    from paper_1805_11462_amd.translator import Translator, make_config
    cfg = make_config(w.enc_layers, w.dec_layers, w.bidirectional, w.emb, w.hidden, w.src_vocab, w.tgt_vocab,
                      w.wdtype, attn=w.attn)
    return Translator(cfg, [weights[n] for n, _ in W.weight_specs(w)])


class Setup:
    def __init__(self, w, peaked=False, data_seed=None, batch=None):
        self.w = w
        self.weights = W.make_weights(w, peaked=peaked)
        self.model = O.model_from(w, self.weights)
        self.src, self.lens = W.make_batch(w, seed=data_seed, batch=batch)
        self.tr = translator_for(w, self.weights)
        self.src_d = torch.from_numpy(self.src).cuda()
        self.lens_d = torch.from_numpy(self.lens).cuda()
        self.tau = TAU[w.wdtype]


def with_workload(w, **kw):
    return W.Workload(**{**w.as_dict(), **kw})


def golden_search(name, seed):
    """Stored oracle results of a whole batch (written by tests/golden/make_search_golden.py)."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", f"search_{name}_seed{seed}.npz")
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def check_search(s, buf, sentences, K, T, alpha, golden=None, log=None):
    """Parity of one GPU search against the oracle, on the listed sentences (section P1-P3 protocol).

    * the GPU's result is internally consistent (log-probs sum to raw; norm = raw / lp; pad after the end);
    * P3: the oracle's own search of the same sentences (``golden``: its stored results for the whole
      batch) gives the same tokens wherever its decision margin exceeds 2 tau, and where tokens agree the
      raw scores agree within n tau; a sentence may differ only where the margin is within 2 tau;
    * every GPU 1-best is rescored by the oracle's teacher-forced decoder: per-token log-probs within tau;
    * P2: every listed sentence's recorded decisions are replayed through the oracle (log-probs, top-K
      validity, finished pool, stop step and the returned entry).
    Returns the sentences whose tokens differ from the oracle's (all replay-verified).
    """
    tau = s.tau
    sel = [int(b) for b in sentences]
    say = log or (lambda msg: None)
    g_tok = buf["tok"].cpu().numpy()
    g_len = buf["len"].cpu().numpy()
    g_raw = buf["raw"].cpu().numpy()
    g_norm = buf["norm"].cpu().numpy()
    g_lp = buf["tok_logp"].cpu().numpy()
    g_steps = buf["trace_steps"].cpu().numpy()
    trace = {k: [a for a in buf[f"trace_{k}"].cpu().numpy()] for k in ("slot", "tok", "cand")}
    for b in sel:
        n = int(g_len[b])
        assert 1 <= n <= T
        assert (g_tok[b, n:] == W.PAD_ID).all()
        assert abs(g_lp[b, :n].astype(np.float64).sum() - g_raw[b]) < 1e-6 * max(1, n)
        assert abs(g_norm[b] - g_raw[b] / O.length_penalty(n, alpha)) < 1e-9 * max(1.0, abs(g_raw[b]))
    # the oracle's own search: tokens, raw score, decision margins and per-step record per sentence
    if golden is None:
        res = O.beam_search(s.model, s.src[sel], s.lens[sel], K, T, alpha, record=True)
        o_tok = {b: res.tokens[i] for i, b in enumerate(sel)}
        o_raw = {b: res.raw[i] for i, b in enumerate(sel)}
        o_margin = {b: res.margin[i] for i, b in enumerate(sel)}
        o_trace = res.trace
    else:
        assert (golden["src"] == s.src).all() and (golden["lens"] == s.lens).all()
        o_tok = {b: [int(x) for x in golden["tokens"][b, :int(golden["len"][b])]] for b in sel}
        o_raw = {b: golden["raw"][b] for b in sel}
        o_margin = {b: golden["margin"][b] for b in sel}
        o_trace = {"slot": [a[sel] for a in golden["trace_slot"]], "tok": [a[sel] for a in golden["trace_tok"]],
                   "margin": [a[sel] for a in golden["trace_margin"]]}
    say(f"oracle search ready for {len(sel)} sentences")
    # P3 per step: the same hypotheses as the oracle at every step before its first margin within 2 tau
    g_trace = {k: [a[sel] for a in trace[k]] for k in ("slot", "tok")}
    bad, n_cmp = O.prefix_agreement(o_trace, g_trace, range(len(sel)), K, 2 * tau)
    assert bad == [], [f"sentence {sel[int(x.split()[0][1:].rstrip(':'))]}: {x}" for x in bad[:10]]
    say(f"P3 per step: choices identical over the oracle's first {int(np.median(list(n_cmp.values())))} steps "
        f"(median; {sum(n_cmp.values())} sentence-steps) before a decision margin within 2 tau")
    # teacher-forced rescoring of every GPU 1-best, all listed sentences in one batch
    forced, _ = O.score_batch(s.model, s.src[sel], s.lens[sel], g_tok[sel], g_len[sel])
    for i, b in enumerate(sel):
        n = int(g_len[b])
        err = np.abs(forced[i, :n] - g_lp[b, :n]).max()
        assert err <= tau, f"sentence {b}: per-token log-prob error {err:.3g} > {tau}"
        assert abs(forced[i, :n].sum() - g_raw[b]) <= n * tau
    say("teacher-forced rescoring passed")
    mismatched, unexplained = [], []
    for b in sel:
        n = int(g_len[b])
        toks = [int(x) for x in g_tok[b, :n]]
        if toks == o_tok[b]:
            assert abs(o_raw[b] - g_raw[b]) <= n * tau
        else:
            mismatched.append(b)
            if o_margin[b] > 2 * tau:
                unexplained.append((b, float(o_margin[b])))
    assert not unexplained, f"tokens differ although every oracle decision margin exceeds 2 tau: {unexplained[:10]}"
    say(f"P3: {len(sel) - len(mismatched)} of {len(sel)} sentences token-identical, "
        f"{sum(1 for b in sel if o_margin[b] > 2 * tau)} of them with every margin > 2 tau")
    # P2: replay every listed sentence's decisions, including its finish step and returned entry
    result = {"tokens": g_tok, "len": g_len, "raw": g_raw, "norm": g_norm}
    bad = O.replay_verify(s.model, s.src, s.lens, K, T, alpha, trace, tau, sentences=sel, steps=g_steps,
                          result=result)
    assert bad == [], bad[:10]
    say("replay passed")
    return mismatched
