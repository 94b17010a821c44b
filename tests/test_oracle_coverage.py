"""Pins for the coverage penalty of the oracle's beam search (Section 4.2: beam search with length and
attention coverage normalisation, citing GNMT; reading R17).

All-zero weights make attention uniform over the real source positions, so after t steps every position
holds t / n and the penalty has the closed form beta * n * log(min(t / n, 1)). A beam wide enough to keep
every hypothesis must return the exhaustive-search optimum of raw / lp + penalty.
"""

import math

import numpy as np
import pytest

from oracle import onmt_oracle as O
from workloads.configs import EOS_ID, PAD_ID
from tests import _small


@pytest.mark.parametrize("beta", [0.2, 1.0])
def test_zero_weights_wide_beam_closed_form(beta):
    # every candidate ties, so slot 0 keeps token 0 and EOS (among the first K flat indices) finishes at
    # every step t with raw -t ln V and coverage t / n; the search stops at the first step where the
    # pool's best reaches the live score -t ln V, or at max_len (where token 0 finishes first)
    V, T = 50, 6
    w, ws, m = _small.model(seed=1, tgt_vocab=V, src_vocab=V, len_lo=3, len_hi=9, batch=4)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=5, max_len=T, beta=beta)
    for b in range(len(lens)):
        n = int(lens[b])
        best, best_t = -math.inf, 0
        for t in range(1, T + 1):
            norm = -t * math.log(V) + beta * n * math.log(min(t / n, 1.0))
            if norm > best:
                best, best_t = norm, t
            if t == T or best >= -t * math.log(V):
                break
        expect = [PAD_ID] * T if best_t == T else [PAD_ID] * (best_t - 1) + [EOS_ID]
        assert res.tokens[b] == expect
        assert abs(res.raw[b] + best_t * math.log(V)) < 1e-12
        assert abs(res.norm[b] - best) < 1e-12


@pytest.mark.parametrize("beta", [0.3])
def test_zero_weights_small_beam_full_length(beta):
    # K = 1: token 0 at every step up to max_len; coverage t / n after t = 6 steps
    w, ws, m = _small.model(seed=1, tgt_vocab=50, src_vocab=50, len_lo=4, len_hi=10, batch=4)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=1, max_len=6, beta=beta)
    for b in range(len(lens)):
        n = int(lens[b])
        assert res.tokens[b] == [PAD_ID] * 6
        expect = -6 * math.log(50) + beta * n * math.log(min(6.0 / n, 1.0))
        assert abs(res.norm[b] - expect) < 1e-12


@pytest.mark.parametrize("beta,alpha", [(0.5, 0.0), (2.0, 0.6)])
def test_wide_beam_equals_brute_force_with_coverage(beta, alpha):
    w, ws, m = _small.model(seed=9, tgt_vocab=6, src_vocab=6, len_lo=2, len_hi=4,
                            scale={"W_s": 6.0, "b_s": 6.0, "W_a": 20.0})
    src, lens = _small.batch(w, seed=10)
    res = O.beam_search(m, src, lens, K=6 ** 3, max_len=3, alpha=alpha, beta=beta)
    for b in range(len(lens)):
        toks, raw, norm = O.brute_force(m, src[b], lens[b], max_len=3, alpha=alpha, beta=beta)
        assert abs(res.norm[b] - norm) < 1e-12
        assert res.tokens[b] == toks


def test_penalty_is_zero_when_covered_and_negative_otherwise():
    cov = np.array([1.2, 1.0, 3.0, 0.0])
    assert O.coverage_penalty(cov, 3, 0.7) == 0.0
    assert O.coverage_penalty(np.array([0.5, 2.0]), 2, 0.7) == pytest.approx(0.7 * math.log(0.5), abs=1e-15)
    assert O.coverage_penalty(np.array([0.5, 2.0]), 2, 0.0) == 0.0
