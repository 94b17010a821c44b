"""Small model shapes for the CPU pins (built with the shared seeded generator)."""

import numpy as np

from workloads.configs import Workload
from workloads.gen import make_weights, make_batch
from oracle.onmt_oracle import model_from


def workload(**kw):
    base = dict(name="small", index=1, enc_layers=1, dec_layers=1, bidirectional=False, emb=4, hidden=8,
                src_vocab=6, tgt_vocab=6, batch=2, len_lo=2, len_hi=4, beam=2, max_len=3, alpha=0.0,
                wdtype="fp32", zipf_s=1.0)
    base.update(kw)
    return Workload(**base)


def model(seed=5, scale=None, **kw):
    w = workload(**kw)
    ws = make_weights(w, seed=seed)
    if scale:
        for k, f in scale.items():
            ws[k] = (ws[k] * np.float32(f)).astype(np.float32)
    return w, ws, model_from(w, ws)


def batch(w, seed=11):
    return make_batch(w, seed=seed)
