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


def check_search(s, buf, sentences, K, T, alpha):
    tau = s.tau
    g_tok = buf["tok"].cpu().numpy()
    g_len = buf["len"].cpu().numpy()
    g_raw = buf["raw"].cpu().numpy()
    g_norm = buf["norm"].cpu().numpy()
    g_lp = buf["tok_logp"].cpu().numpy()
    trace = {k: [a for a in buf[f"trace_{k}"].cpu().numpy()] for k in ("slot", "tok", "cand")}
    mismatched = []
    for b in sentences:
        res = O.beam_search(s.model, s.src[b:b + 1], s.lens[b:b + 1], K, T, alpha)
        n = int(g_len[b])
        toks = list(g_tok[b, :n])
        assert (g_tok[b, n:] == W.PAD_ID).all()
        # the GPU's own result is internally consistent: per-token log-probs sum to raw, norm = raw / lp
        assert abs(g_lp[b, :n].astype(np.float64).sum() - g_raw[b]) < 1e-6 * max(1, n)
        assert abs(g_norm[b] - g_raw[b] / O.length_penalty(n, alpha)) < 1e-9 * max(1.0, abs(g_raw[b]))
        # teacher-forced oracle rescoring of the GPU's hypothesis
        forced = O.score_forced(s.model, s.src[b], s.lens[b], toks)
        assert np.abs(forced - g_lp[b, :n]).max() <= tau
        assert abs(forced.sum() - g_raw[b]) <= n * tau
        if toks == res.tokens[0]:
            assert abs(res.raw[0] - g_raw[b]) <= n * tau
        else:
            mismatched.append(b)
    # every sentence (matched or not) must pass the step-by-step replay of the GPU's decisions
    bad = O.replay_verify(s.model, s.src, s.lens, K, T, alpha, trace, tau, sentences=sentences)
    assert bad == [], bad[:10]
    return mismatched
