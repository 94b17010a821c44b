"""GPU parity of the hypothesis filters and the unknown-word alignment (Section 4.2: beam search under a
limit on unknown words and word-level constraints on the search; OOV handling; readings R18, R19).
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import Setup, with_workload, translator_for

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _search(s, K, T, alpha=0.0, banned=(), max_unk=-1, align=True):
    B, S = s.src.shape
    buf = s.tr.search_buffers(B, S, K, T, alpha, banned=banned, max_unk=max_unk, align=align)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    out = {k: buf[k].cpu().numpy() for k in ("tok", "len", "raw", "norm", "tok_logp")}
    if align:
        out["align"] = buf["align"].cpu().numpy()
    return out


@pytest.fixture(scope="module")
def tiny_peaked():
    return Setup(W.get("tiny"), peaked=True)


@pytest.fixture(scope="module")
def default():
    return Setup(W.get("default"))


@pytest.fixture(scope="module")
def zero():
    w = with_workload(W.get("tiny"), tgt_vocab=50, src_vocab=50)
    s = Setup(w)
    s.tr = translator_for(w, {k: np.zeros_like(v) for k, v in s.weights.items()})
    for k in s.model.w:
        s.model.w[k][...] = 0.0
    return s


@pytest.mark.parametrize("banned,max_unk,K,want", [
    ((W.PAD_ID,), -1, 1, [W.UNK_ID] * 6), ((W.PAD_ID,), 0, 1, [2] * 6),
    ((W.PAD_ID, 2), 0, 1, [W.EOS_ID]), ((W.PAD_ID, 2, W.EOS_ID), 0, 1, [4] * 6),
    ((W.PAD_ID,), 2, 1, [W.UNK_ID, W.UNK_ID, 2, 2, 2, 2]), ((W.PAD_ID,), 2, 3, [W.EOS_ID])])
def test_filters_zero_weights_closed_form(zero, banned, max_unk, K, want):
    _case("filters_zero", banned=banned, max_unk=max_unk, K=K)
    # all candidates tie, so each slot takes the smallest allowed ids; with K = 3 EOS is among the first
    # three at step 1 and finishes with the live best's score, which ends the search
    out = _search(zero, K, 6, banned=banned, max_unk=max_unk)
    res = O.beam_search(zero.model, zero.src, zero.lens, K, 6, banned=banned, max_unk=max_unk)
    for b in range(zero.src.shape[0]):
        n = int(out["len"][b])
        assert list(out["tok"][b, :n]) == want == res.tokens[b]
        assert res.align[b] == [0] * n
        assert list(out["align"][b, :n]) == [0] * n          # uniform attention: position 0 on ties
        assert (out["align"][b, n:] == -1).all()


@pytest.mark.parametrize("banned,max_unk", [((), 0), ((5, 17, 300), -1), ((4, 5, 6, 7), 1)])
def test_filters_tiny_peaked_match_oracle(tiny_peaked, banned, max_unk):
    s = tiny_peaked
    w = s.w
    base = O.beam_search(s.model, s.src, s.lens, w.beam, w.max_len)
    banned = tuple(banned) + tuple(sorted({t for toks in base.tokens for t in toks[:1]}))
    _case("filters", banned=banned, max_unk=max_unk)
    out = _search(s, w.beam, w.max_len, banned=banned, max_unk=max_unk)
    res = O.beam_search(s.model, s.src, s.lens, w.beam, w.max_len, banned=banned, max_unk=max_unk)
    for b in range(s.src.shape[0]):
        n = int(out["len"][b])
        toks = list(out["tok"][b, :n])
        assert toks == res.tokens[b], b
        assert not set(toks) & set(banned)
        if max_unk >= 0:
            assert toks.count(W.UNK_ID) <= max_unk
        assert abs(out["raw"][b] - res.raw[b]) <= s.tau * n
        assert list(out["align"][b, :n]) == res.align[b]


def test_alignment_and_replacement_tiny_peaked(tiny_peaked):
    s = tiny_peaked
    w = s.w
    B, S = s.src.shape
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, 0.6, align=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    rep = s.tr.replace_unk(s.src_d, buf).cpu().numpy()          # onmt_replace_unk, on the device
    torch.cuda.synchronize()
    res = O.beam_search(s.model, s.src, s.lens, w.beam, w.max_len, alpha=0.6)
    n_unk = 0
    for b in range(B):
        n = int(buf["len"][b])
        assert list(buf["tok"][b, :n].cpu().numpy()) == res.tokens[b]
        assert list(buf["align"][b, :n].cpu().numpy()) == res.align[b]
        want = O.replace_unk(res.tokens[b], res.align[b], s.src[b])
        got = [("src", int(rep[b, t])) if rep[b, t] >= 0 else ("tgt", int(buf["tok"][b, t])) for t in range(n)]
        assert got == want
        assert (rep[b, n:] == -1).all()
        n_unk += sum(1 for k, _ in want if k == "src")
    print(f"  {n_unk} UNK outputs replaced", flush=True)


def test_replacement_of_every_unk():
    # a model that outputs UNK at most steps (the UNK bias raised), so that the device replacement covers
    # many positions; compared with the oracle's replacement along the oracle's own search
    w = with_workload(W.get("tiny"), tgt_vocab=60, src_vocab=60)
    s = Setup(w, peaked=True)
    s.weights["b_s"][W.UNK_ID] += 3.0
    s.model = O.model_from(w, s.weights)
    s.tr = translator_for(w, s.weights)
    B, S = s.src.shape
    _case("replace_unk", workload="tiny_unk")
    buf = s.tr.search_buffers(B, S, 2, 8, 0.0, align=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    rep = s.tr.replace_unk(s.src_d, buf).cpu().numpy()
    res = O.beam_search(s.model, s.src, s.lens, 2, 8, 0.0)
    n_unk = 0
    for b in range(B):
        n = int(buf["len"][b])
        toks = list(buf["tok"][b, :n].cpu().numpy())
        if toks != res.tokens[b]:
            continue
        want = O.replace_unk(res.tokens[b], res.align[b], s.src[b])
        got = [("src", int(rep[b, t])) if rep[b, t] >= 0 else ("tgt", int(toks[t])) for t in range(n)]
        assert got == want
        n_unk += sum(1 for k, _ in want if k == "src")
    assert n_unk > 0


def test_filters_default_sampled(default):
    s = default
    w = s.w
    banned = tuple(range(4, 104))            # the 100 most frequent target ids of the bounded Zipf law
    _case("filters", workload="default", n_banned=len(banned), max_unk=0)
    out = _search(s, w.beam, w.max_len, banned=banned, max_unk=0)
    for b in [0, 63]:
        n = int(out["len"][b])
        toks = list(out["tok"][b, :n])
        assert not set(toks) & set(banned)
        assert W.UNK_ID not in toks
        forced = O.score_forced(s.model, s.src[b], s.lens[b], toks)
        assert np.abs(forced - out["tok_logp"][b, :n]).max() <= s.tau
        assert ((out["align"][b, :n] >= 0) & (out["align"][b, :n] < s.lens[b])).all()
