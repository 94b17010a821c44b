"""Pins for the oracle's teacher-forced scoring (Section 2: the training objective is the negative
log-likelihood under p(w_1:T | x) = prod_t p(w_t | w_<t, x)).

Pinned by: the uniform closed form (all-zero weights give every token log(1/V)); normalisation (the
probabilities of every one-token target sum to 1, and of every two-token target too, by the chain
rule); agreement with the beam search, whose 1-best path scores are checked against exhaustive search
elsewhere; and independence of the sentences of a batch (padding rows and other sentences do not
change a sentence's scores).
"""

import math
from itertools import product

import numpy as np
import pytest

from oracle import onmt_oracle as O
from tests import _small


def test_all_zero_weights_give_the_uniform_closed_form():
    w, ws, m = _small.model(seed=3, tgt_vocab=40, src_vocab=40, batch=3)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    rng = np.random.default_rng(4)
    tgt = rng.integers(0, 40, size=(3, 7))
    tgt_len = np.array([7, 1, 4])
    logp, nll = O.score_batch(m, src, lens, tgt, tgt_len)
    for b in range(3):
        np.testing.assert_allclose(logp[b, :tgt_len[b]], -math.log(40), atol=1e-12)
        assert np.all(logp[b, tgt_len[b]:] == 0.0)
        assert abs(nll[b] - tgt_len[b] * math.log(40)) < 1e-12


def test_probabilities_of_all_short_targets_sum_to_one():
    w, ws, m = _small.model(seed=7, tgt_vocab=6, src_vocab=6, scale={"W_s": 5.0, "b_s": 5.0})
    src, lens = _small.batch(w, seed=8)
    V = 6
    for T in (1, 2):
        seqs = np.array(list(product(range(V), repeat=T)))
        total = np.zeros(2)
        for b in range(2):
            srcb = np.repeat(src[b:b + 1], len(seqs), axis=0)
            lb = np.repeat(lens[b:b + 1], len(seqs))
            logp, nll = O.score_batch(m, srcb, lb, seqs, np.full(len(seqs), T))
            total[b] = np.exp(-nll).sum()
        np.testing.assert_allclose(total, 1.0, atol=1e-12)


@pytest.mark.parametrize("K,alpha", [(1, 0.0), (3, 0.6)])
def test_beam_output_scores_match(K, alpha):
    w, ws, m = _small.model(seed=21, enc_layers=2, dec_layers=2, emb=6, hidden=10, src_vocab=25,
                            tgt_vocab=25, len_lo=3, len_hi=7, batch=4, scale={"W_s": 8.0, "b_s": 8.0})
    src, lens = _small.batch(w, seed=22)
    res = O.beam_search(m, src, lens, K=K, max_len=8, alpha=alpha)
    T = max(len(t) for t in res.tokens)
    tgt = np.zeros((4, T), dtype=np.int64)
    for b, t in enumerate(res.tokens):
        tgt[b, :len(t)] = t
    tgt_len = np.array([len(t) for t in res.tokens])
    logp, nll = O.score_batch(m, src, lens, tgt, tgt_len)
    for b in range(4):
        np.testing.assert_allclose(logp[b, :tgt_len[b]], res.logps[b], atol=1e-12)
        assert abs(-nll[b] - res.raw[b]) < 1e-12


def test_sentences_are_scored_independently():
    w, ws, m = _small.model(seed=31, emb=6, hidden=10, src_vocab=20, tgt_vocab=20, len_lo=2, len_hi=6, batch=5,
                            scale={"W_a": 20.0})
    src, lens = _small.batch(w, seed=32)
    rng = np.random.default_rng(33)
    tgt = rng.integers(0, 20, size=(5, 6))
    tgt_len = np.array([6, 2, 5, 1, 3])
    logp, nll = O.score_batch(m, src, lens, tgt, tgt_len)
    for b in range(5):
        lb, nb = O.score_batch(m, src[b:b + 1], lens[b:b + 1], tgt[b:b + 1], tgt_len[b:b + 1])
        np.testing.assert_allclose(logp[b], lb[0], atol=1e-12)
        forced = O.score_forced(m, src[b], lens[b], tgt[b, :tgt_len[b]])
        np.testing.assert_allclose(logp[b, :tgt_len[b]], forced, atol=1e-12)
