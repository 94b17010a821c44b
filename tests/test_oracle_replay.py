"""Pins for the replay verifier: the step-by-step check of another implementation's beam decisions
(Section 2 item (d) beam search; Section 4.2 length normalisation; the near-tie reading R16).

The verifier must accept the oracle's own record of a search and reject records of the mistakes an
implementation can make in the bookkeeping that the per-step log-prob checks do not see: stopping a
sentence early or late, keeping a finished (EOS) hypothesis live, and returning a finished entry that
is not the best. Each mistake is planted here, on the CPU, by running the oracle's own search with the
mistake in place (or by editing its record) and replaying that record against the correct oracle.
"""

import numpy as np
import pytest

from oracle import onmt_oracle as O
from workloads.configs import EOS_ID, PAD_ID
from tests import _small


def _eos_model(seed=83, scale=10.0, eos_bias=1.0):
    # a small model with every weight scaled up (input-dependent outputs) and the EOS logit raised, so
    # that sentences finish at different steps (4 to 9 here), several hypotheses of one sentence enter
    # the finished pool, and the stop rule fires before max_len
    w, ws, m = _small.model(seed=seed, emb=6, hidden=10, src_vocab=20, tgt_vocab=20, len_lo=3, len_hi=7,
                            batch=6)
    for k in m.w:
        m.w[k] *= scale
    m.w["b_s"][EOS_ID] += eos_bias
    src, lens = _small.batch(w, seed=seed + 1)
    return w, m, src, lens


def _result(res, T):
    B = len(res.tokens)
    tok = np.full((B, T), PAD_ID, np.int64)
    for b, t in enumerate(res.tokens):
        tok[b, :len(t)] = t
    return {"tokens": tok, "len": np.array([len(t) for t in res.tokens]), "raw": res.raw, "norm": res.norm}


def _copy(trace):
    return {k: [np.array(a) for a in v] for k, v in trace.items()}


K, T = 3, 9


@pytest.mark.parametrize("alpha", [0.0, 0.6])
def test_replay_accepts_the_oracles_own_record(alpha):
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, alpha, record=True)
    assert (res.steps < T).any(), "the fixture must stop some sentence before max_len"
    bad = O.replay_verify(m, src, lens, K, T, alpha, res.trace, 1e-9, steps=res.steps, result=_result(res, T))
    assert bad == [], bad


def test_replay_rejects_an_early_finish_step():
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.0, record=True)
    steps = res.steps.copy()
    steps[1] -= 1
    bad = O.replay_verify(m, src, lens, K, T, 0.0, res.trace, 1e-9, steps=steps)
    assert any(s.startswith("b1: finished at step") for s in bad), bad


def test_replay_rejects_a_search_that_stops_early():
    # the implementation records nothing at the step where the sentence was still live
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.0, record=True)
    b = int(np.argmax(res.steps))
    tr = _copy(res.trace)
    last = int(res.steps[b])
    tr["slot"][last - 1][b, :] = -1
    tr["tok"][last - 1][b, :] = -1
    tr["cand"][last - 1][b, :] = -np.inf
    bad = O.replay_verify(m, src, lens, K, T, 0.0, tr, 1e-9)
    assert any(f"b{b} t{last}: nothing chosen" in s for s in bad), bad


@pytest.mark.parametrize("alpha", [0.0, 0.6])
def test_replay_rejects_a_search_without_the_stop_rule(alpha):
    w, m, src, lens = _eos_model()
    good = O.beam_search(m, src, lens, K, T, alpha, record=True)
    late = O.beam_search(m, src, lens, K, T, alpha, record=True, stop_rule=False)
    assert (late.steps > good.steps).any(), "the fixture must have a sentence the stop rule ends early"
    bad = O.replay_verify(m, src, lens, K, T, alpha, late.trace, 1e-9, steps=late.steps)
    for b in np.nonzero(late.steps > good.steps)[0]:
        assert any(s.startswith(f"b{b}: choices recorded after") for s in bad), bad
        assert any(s.startswith(f"b{b}: finished at step") for s in bad), bad


def test_replay_rejects_a_search_that_keeps_eos_live(monkeypatch):
    w, m, src, lens = _eos_model()
    with monkeypatch.context() as mp:
        mp.setattr(O, "EOS_ID", -1)            # the recorded search treats EOS as an ordinary token
        wrong = O.beam_search(m, src, lens, K, T, 0.0, record=True, stop_rule=False)
    chose_eos = [b for b in range(len(lens))
                 if any((wrong.trace["tok"][t][b] == EOS_ID).any() for t in range(T - 1))]
    assert chose_eos, "the fixture must choose EOS before the last step"
    bad = O.replay_verify(m, src, lens, K, T, 0.0, wrong.trace, 1e-9, steps=wrong.steps)
    for b in chose_eos:
        assert any(s.startswith(f"b{b} ") or s.startswith(f"b{b}:") for s in bad), (b, bad)


def test_replay_rejects_a_returned_entry_that_is_not_the_best():
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.6, record=True)
    # find a sentence with two finished entries and return the worse one
    tr = res.trace
    for b in range(len(lens)):
        entries = []
        hyp = {0: []}
        for t in range(1, int(res.steps[b]) + 1):
            nxt, j = {}, 0
            for r in range(K):
                k, tk, c = int(tr["slot"][t - 1][b, r]), int(tr["tok"][t - 1][b, r]), float(tr["cand"][t - 1][b, r])
                if k < 0:
                    continue
                seq = hyp[k] + [tk]
                if tk == EOS_ID or t == T:
                    entries.append((c / O.length_penalty(t, 0.6), c, seq))
                else:
                    nxt[j] = seq
                    j += 1
            hyp = nxt
        if len(entries) >= 2:
            break
    else:
        pytest.fail("the fixture must finish two hypotheses of one sentence")
    entries.sort(key=lambda e: -e[0])
    worse = entries[1]
    result = _result(res, T)
    result["tokens"][b, :] = PAD_ID
    result["tokens"][b, :len(worse[2])] = worse[2]
    result["len"] = result["len"].copy()
    result["len"][b] = len(worse[2])
    result["raw"] = res.raw.copy()
    result["raw"][b] = worse[1]
    result["norm"] = res.norm.copy()
    result["norm"][b] = worse[0]
    bad = O.replay_verify(m, src, lens, K, T, 0.6, tr, 1e-9, steps=res.steps, result=result)
    assert any(s.startswith(f"b{b}: returned hypothesis is not the pool's best") for s in bad), bad
    # and the correct result passes
    assert O.replay_verify(m, src, lens, K, T, 0.6, tr, 1e-9, steps=res.steps, result=_result(res, T)) == []


def test_replay_rejects_a_wrong_raw_score():
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.0, record=True)
    result = _result(res, T)
    result["raw"] = res.raw.copy()
    result["raw"][2] += 1e-6
    bad = O.replay_verify(m, src, lens, K, T, 0.0, res.trace, 1e-9, steps=res.steps, result=result)
    assert any(s.startswith("b2: returned raw") for s in bad), bad


def test_margins_separate_the_decisions():
    # the recorded margin of a sentence is at most every selection gap of its run, so perturbing the
    # log-probs by less than half of it cannot change the outputs (checked here by brute force: a search
    # on a model whose generator bias is shifted by a tiny amount in a token-dependent way)
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.6)
    assert np.isfinite(res.margin).all() and (res.margin >= 0).all()
    rng = np.random.default_rng(3)
    eps = 0.2 * res.margin.min() / T
    m2 = O.Model(m.enc_layers, m.dec_layers, m.bidirectional, m.emb, m.hidden, m.src_vocab, m.tgt_vocab,
                 {k: v.copy() for k, v in m.w.items()}, m.attn)
    m2.w["b_s"] += rng.uniform(-eps, eps, size=m2.w["b_s"].shape)
    res2 = O.beam_search(m2, src, lens, K, T, 0.6)
    assert res2.tokens == res.tokens


def test_margin_is_zero_when_candidates_tie():
    # all-zero weights: every candidate of a step has the same score, so the selection boundary is a tie
    w, ws, m = _small.model(seed=1, tgt_vocab=50, src_vocab=50)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=3, max_len=6)
    assert (res.margin == 0.0).all()
    # a beam that keeps every candidate has no selection boundary; what remains is the final argmax
    w, ws, m = _small.model(seed=31, scale={"W_s": 20.0, "b_s": 5.0})
    src, lens = _small.batch(w, seed=32)
    res = O.beam_search(m, src, lens, K=216, max_len=3)
    import itertools
    V = m.tgt_vocab
    for b in range(len(lens)):
        # every output sequence (first EOS ends it, or length 3 without EOS), scored from scratch
        norms = []
        for n in range(1, 4):
            for seq in itertools.product(range(V), repeat=n):
                if EOS_ID in seq[:-1] or (n < 3 and seq[-1] != EOS_ID):
                    continue
                norms.append(O.score_forced(m, src[b], lens[b], list(seq)).sum())
        assert len(norms) == 156
        top = sorted(norms, reverse=True)
        # the final argmax is one of the decisions; the stop rule's comparisons may be closer still
        assert 0 < res.margin[b] <= top[0] - top[1] + 1e-12


def test_prefix_agreement_accepts_itself_and_small_perturbations():
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.6, record=True)
    bad, n = O.prefix_agreement(res.trace, res.trace, range(len(lens)), K, 0.0)
    assert bad == [] and all(n[b] == res.steps[b] for b in n)
    # a model perturbed by far less than every margin chooses the same hypotheses at every step
    eps = 0.1 * res.margin.min() / T
    m2 = O.Model(m.enc_layers, m.dec_layers, m.bidirectional, m.emb, m.hidden, m.src_vocab, m.tgt_vocab,
                 {k: v.copy() for k, v in m.w.items()}, m.attn)
    m2.w["b_s"] += np.random.default_rng(4).uniform(-eps, eps, size=m2.w["b_s"].shape)
    res2 = O.beam_search(m2, src, lens, K, T, 0.6, record=True)
    bad, n = O.prefix_agreement(res.trace, res2.trace, range(len(lens)), K, 2 * eps * T)
    assert bad == [] and sum(n.values()) > 0


def test_prefix_agreement_rejects_a_different_choice_before_the_first_near_tie():
    w, m, src, lens = _eos_model()
    res = O.beam_search(m, src, lens, K, T, 0.6, record=True)
    b = int(np.argmax([res.trace["margin"][0][i] for i in range(len(lens))]))
    assert res.trace["margin"][0][b] > 1e-3
    wrong = _copy(res.trace)
    wrong["tok"][0][b, 1] = (wrong["tok"][0][b, 1] + 1) % 20
    bad, _ = O.prefix_agreement(res.trace, wrong, range(len(lens)), K, 1e-3)
    assert any(s.startswith(f"b{b} t1:") for s in bad), bad
    # the same change is accepted where the oracle's own first decision was a near-tie
    bad, n = O.prefix_agreement(res.trace, wrong, [b], K, res.trace["margin"][0][b] * 1.01)
    assert bad == [] and n[b] == 0
