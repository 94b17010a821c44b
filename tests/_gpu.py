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
                      w.wdtype)
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
