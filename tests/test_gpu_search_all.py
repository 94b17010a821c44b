"""GPU parity of whole beam searches: every sentence of the five workloads, three data seeds each.

Section 2 item (d) (beam search) and Section 4.2 (length normalisation) define the search; Table 2 gives
the paper-default shape (2x500, batch 64, beam 5). Each case runs one full-batch search through the C ABI
and checks every sentence against the oracle: the oracle's own search of the same batch (stored by
tests/golden/make_search_golden.py) must give identical tokens wherever its decision margins exceed
twice the tolerance (1e-4 fp32, 2e-2 bf16 per-step log-probs), every GPU 1-best is rescored by the
oracle's teacher-forced decoder, and every sentence's recorded decisions are replayed step by step
(top-K validity, finished pool, stop step, returned entry).
"""

import time

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import TAU, check_search, golden_search, translator_for

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

NAMES = ("tiny", "default", "larger", "greedy", "long")
OFFSETS = (0, 1, 2)
_models = {}


class _Batch:
    """One workload's model (oracle and GPU) on the seeded batch of one data seed."""

    def __init__(self, w, seed):
        if w.name not in _models:
            _models.clear()                      # one GPU model alive at a time
            weights = W.make_weights(w)
            _models[w.name] = (weights, O.model_from(w, weights), translator_for(w, weights))
        self.weights, self.model, self.tr = _models[w.name]
        self.w = w
        self.src, self.lens = W.make_batch(w, seed=seed)
        self.src_d = torch.from_numpy(self.src).cuda()
        self.lens_d = torch.from_numpy(self.lens).cuda()
        self.tau = TAU[w.wdtype]


@pytest.mark.parametrize("name,off", [(n, o) for n in NAMES for o in OFFSETS])
def test_search_every_sentence(name, off):
    w = W.get(name)
    seed = 1000 + w.index + off
    t0 = time.perf_counter()
    say = lambda msg: print(f"  [{time.perf_counter() - t0:6.1f} s] {msg}", flush=True)
    print(f"[case] search workload={name} seed={seed} B={w.batch} beam={w.beam} max_len={w.max_len}", flush=True)
    s = _Batch(w, seed)
    g = golden_search(name, seed)
    B, S = s.src.shape
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, w.alpha, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    say("GPU search done")
    mism = check_search(s, buf, range(B), w.beam, w.max_len, w.alpha, golden=g, log=say)
    print(f"  token-identical {B - len(mism)}/{B}; differing (all within 2 tau of a decision, replay-verified): "
          f"{len(mism)}", flush=True)
