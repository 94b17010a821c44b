"""The oracle against the closed-form fixtures in tests/golden (Section 4.2; Section 2; reading R9)."""

import json
import math
import os

import numpy as np

from oracle import onmt_oracle as O
from tests import _small

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")))


def test_length_penalty_values():
    for n, alpha, v in GOLDEN["length_penalty"]:
        assert abs(O.length_penalty(n, alpha) - v) < 1e-4


def test_zero_generator_values():
    for V, v in GOLDEN["neg_log_v"]:
        m = O.Model(1, 1, False, 2, 3, 3, V, {"W_s": np.zeros((V, 3)), "b_s": np.zeros(V)})
        lp = O.generator(m, np.ones((1, 3)))
        assert np.all(np.abs(lp - v) < 1e-4)


def test_all_zero_beam_values():
    g = GOLDEN["all_zero_beam"]
    w, ws, m = _small.model(seed=1, tgt_vocab=g["vocab"], src_vocab=g["vocab"])
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    for case in ("small_beam", "wide_beam"):
        for K in g[case]["K"]:
            res = O.beam_search(m, src, lens, K=K, max_len=g["max_len"])
            for b in range(len(lens)):
                assert res.tokens[b] == g[case]["tokens"]
                assert abs(res.raw[b] - g[case]["raw"]) < 1e-4
