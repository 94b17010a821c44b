"""GPU: a batch that finishes long before max_len (Section 2 beam search: a sentence stops once no live
hypothesis can still beat its best finished one). The host learns that every sentence has finished from a
counter that it reads without stalling the device, one check period late, so the device may run extra
steps; those steps must change no output. The same search with finish checks every step, every 3 steps
and never (a period longer than max_len) must give identical outputs and traces, which match the oracle.
The end-of-sentence token's bias is raised so that it wins at the first step (the oracle confirms it).
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import TAU, check_search, translator_for

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


class EarlyEos:
    def __init__(self, w, eos_bias):
        wt = dict(W.make_weights(w, peaked=True))
        bs = np.array(wt["b_s"], dtype=np.float32).copy()
        bs[W.EOS_ID] += eos_bias
        wt["b_s"] = bs
        self.w, self.weights = w, wt
        self.model = O.model_from(w, wt)
        self.src, self.lens = W.make_batch(w)
        self.tr = translator_for(w, wt)
        self.src_d = torch.from_numpy(self.src).cuda()
        self.lens_d = torch.from_numpy(self.lens).cuda()
        self.tau = TAU[w.wdtype]


@pytest.mark.parametrize("alpha", [0.0, 0.6])
def test_extra_steps_after_the_batch_finished_change_nothing(alpha):
    w = W.get("tiny")
    s = EarlyEos(w, 3.0)
    B, S = s.src.shape
    K, T = 3, 20
    print(f"[case] early_finish alpha={alpha} B={B} K={K} T={T}", flush=True)
    ref = O.beam_search(s.model, s.src[:1], s.lens[:1], K, T, alpha)
    assert len(ref.tokens[0]) < T // 2            # the batch really finishes early
    outs = {}
    for every in (1, 3, 100):
        buf = s.tr.search_buffers(B, S, K, T, alpha, check_every=every, trace=True)
        s.tr.beam_search(s.src_d, s.lens_d, buf)
        torch.cuda.synchronize()
        outs[every] = {k: buf[k].cpu().numpy() for k in ("tok", "len", "raw", "norm", "tok_logp", "trace_steps")}
        outs[every]["trace"] = {k: buf[f"trace_{k}"].cpu().numpy() for k in ("slot", "tok", "cand")}
        if every == 1:
            mism = check_search(s, buf, range(B), K, T, alpha)
            assert mism == []
    assert (outs[1]["len"] < T // 2).all()
    for every in (3, 100):
        for k in ("tok", "len", "raw", "norm", "tok_logp", "trace_steps"):
            np.testing.assert_array_equal(outs[every][k], outs[1][k], err_msg=f"{k} with checks every {every}")
        steps = outs[1]["trace_steps"]
        for k in ("slot", "tok", "cand"):            # the trace up to each sentence's last step
            for b in range(B):
                np.testing.assert_array_equal(outs[every]["trace"][k][:steps[b], b], outs[1]["trace"][k][:steps[b], b])
