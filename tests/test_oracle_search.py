"""Pins for the oracle's beam search (Section 2 item (d); Section 4.2 length normalisation).

The search is a heuristic, so it is pinned by special cases whose answer is
known independently: width 1 is greedy argmax decoding; a width that keeps
every hypothesis is exhaustive search; with all-zero weights every candidate
ties, which fixes the tie-break and the stop rule; teacher-forced rescoring of
the returned hypothesis must give its reported score.
"""

import math

import numpy as np
import pytest

from oracle import onmt_oracle as O
from workloads.configs import EOS_ID, PAD_ID
from tests import _small


def test_length_penalty_closed_form():
    assert abs(O.length_penalty(250, 0.6) - 9.4849) < 1e-4
    assert O.length_penalty(1, 0.6) == 1.0
    assert O.length_penalty(17, 0.0) == 1.0
    assert abs(O.length_penalty(7, 1.0) - 2.0) < 1e-15


@pytest.mark.parametrize("alpha", [0.0, 0.6])
def test_wide_beam_equals_brute_force(alpha):
    # V = 6, max_len = 3: 156 output sequences; K = 216 >= V^T keeps all of them.
    w, ws, m = _small.model(seed=31, scale={"W_s": 20.0, "b_s": 5.0})
    src, lens = _small.batch(w, seed=32)
    res = O.beam_search(m, src, lens, K=216, max_len=3, alpha=alpha)
    for b in range(src.shape[0]):
        seq, raw, norm = O.brute_force(m, src[b], lens[b], 3, alpha)
        assert res.tokens[b] == seq
        assert abs(res.raw[b] - raw) < 1e-12 and abs(res.norm[b] - norm) < 1e-12


def test_brute_force_scores_every_output_sequence_once(monkeypatch):
    # the sequences brute_force scores, recorded through score_forced, must be exactly the output
    # sequences of the search space: those whose first EOS ends them at n <= T (EOS-free prefixes of
    # length n - 1: (V-1)^(n-1) of them) and the EOS-free sequences of length T ((V-1)^T): 156 at V = 6,
    # T = 3, listed here by direct enumeration
    import itertools
    w, ws, m = _small.model(seed=31, scale={"W_s": 20.0, "b_s": 5.0})
    src, lens = _small.batch(w, seed=32)
    V, T = m.tgt_vocab, 3
    seen = []
    real = O.score_forced

    def counting(mm, s_row, n_src, target):
        seen.append(tuple(target))
        return real(mm, s_row, n_src, target)

    monkeypatch.setattr(O, "score_forced", counting)
    O.brute_force(m, src[0], lens[0], T)
    want = set()
    for n in range(1, T + 1):
        for seq in itertools.product(range(V), repeat=n):
            if EOS_ID not in seq[:-1] and (seq[-1] == EOS_ID or n == T):
                want.add(seq)
    assert len(want) == sum((V - 1) ** (k - 1) for k in range(1, T + 1)) + (V - 1) ** T == 156
    assert len(seen) == len(set(seen)) == 156
    assert set(seen) == want


@pytest.mark.parametrize("seed", [41, 42])
def test_width_one_is_greedy(seed):
    w, ws, m = _small.model(seed=seed, enc_layers=2, dec_layers=2, emb=6, hidden=10, src_vocab=40,
                            tgt_vocab=40, len_lo=3, len_hi=8, batch=4, scale={"W_s": 10.0, "b_s": 10.0})
    src, lens = _small.batch(w, seed=seed + 1)
    res = O.beam_search(m, src, lens, K=1, max_len=12)
    toks, raw = O.greedy(m, src, lens, 12)
    assert res.tokens == toks
    np.testing.assert_allclose(res.raw, raw, atol=1e-12)


@pytest.mark.parametrize("K,alpha", [(2, 0.0), (3, 0.6), (5, 0.6)])
def test_rescoring_and_monotone_scores(K, alpha):
    w, ws, m = _small.model(seed=51, enc_layers=2, dec_layers=2, emb=6, hidden=10, src_vocab=30,
                            tgt_vocab=30, len_lo=3, len_hi=8, batch=4, scale={"W_s": 8.0, "b_s": 8.0})
    src, lens = _small.batch(w, seed=52)
    res = O.beam_search(m, src, lens, K=K, max_len=10, alpha=alpha)
    for b in range(4):
        forced = O.score_forced(m, src[b], lens[b], res.tokens[b])
        np.testing.assert_allclose(forced, res.logps[b], atol=1e-12)
        assert abs(forced.sum() - res.raw[b]) < 1e-12
        assert np.all(np.asarray(res.logps[b]) <= 0)           # raw scores never increase
        n = len(res.tokens[b])
        assert abs(res.norm[b] - res.raw[b] / O.length_penalty(n, alpha)) < 1e-12
        if alpha == 0.0:
            assert res.norm[b] == res.raw[b]
        assert n == 10 or res.tokens[b][-1] == EOS_ID
        assert EOS_ID not in res.tokens[b][:-1]


@pytest.mark.parametrize("K,alpha", [(3, 0.0), (4, 0.6)])
def test_stop_rule_does_not_change_the_result(K, alpha):
    w, ws, m = _small.model(seed=61, emb=6, hidden=10, src_vocab=12, tgt_vocab=12, len_lo=3, len_hi=6,
                            batch=5, scale={"W_s": 15.0, "b_s": 15.0})
    src, lens = _small.batch(w, seed=62)
    a = O.beam_search(m, src, lens, K=K, max_len=9, alpha=alpha, stop_rule=True)
    b = O.beam_search(m, src, lens, K=K, max_len=9, alpha=alpha, stop_rule=False)
    assert a.tokens == b.tokens
    np.testing.assert_array_equal(a.raw, b.raw)
    assert (a.steps <= b.steps).all()


@pytest.mark.parametrize("K", [1, 2, 3])
def test_all_zero_weights_small_beam_outputs_pad(K):
    # every candidate ties; ties go to the smaller flat index, so slot 0 with token 0 always wins
    w, ws, m = _small.model(seed=1, tgt_vocab=50, src_vocab=50)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=K, max_len=6)
    for b in range(len(lens)):
        assert res.tokens[b] == [PAD_ID] * 6
        assert abs(res.raw[b] + 6 * math.log(50)) < 1e-12


@pytest.mark.parametrize("K", [4, 6])
def test_all_zero_weights_wide_beam_outputs_eos(K):
    # EOS (id 3) is among the first K flat indices at t = 1; it enters the pool with
    # norm = raw = -ln V, and the stop rule fires on equality.
    w, ws, m = _small.model(seed=1, tgt_vocab=50, src_vocab=50)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=K, max_len=6)
    for b in range(len(lens)):
        assert res.tokens[b] == [EOS_ID]
        assert abs(res.raw[b] + math.log(50)) < 1e-12
        assert res.steps[b] == 1


def test_replay_accepts_own_trace_and_rejects_a_wrong_one():
    w, ws, m = _small.model(seed=71, emb=6, hidden=10, src_vocab=30, tgt_vocab=30, len_lo=3, len_hi=7,
                            batch=3, scale={"W_s": 8.0, "b_s": 8.0})
    src, lens = _small.batch(w, seed=72)
    res = O.beam_search(m, src, lens, K=3, max_len=8, record=True)
    assert O.replay_verify(m, src, lens, 3, 8, 0.0, res.trace, tau=1e-9) == []
    bad = {k: [np.array(a) for a in v] for k, v in res.trace.items()}
    bad["tok"][2][1, 0] = (bad["tok"][2][1, 0] + 1) % 30       # plant a wrong token choice
    assert O.replay_verify(m, src, lens, 3, 8, 0.0, bad, tau=1e-9) != []
