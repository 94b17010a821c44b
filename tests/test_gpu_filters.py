"""GPU parity of the hypothesis filters and the unknown-word alignment (Section 4.2: beam search under
a limit on unknown words and
word-level constraints on the search; OOV handling; readings R18, R19).
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
    out = _search(s, w.beam, w.max_len, alpha=0.6)
    res = O.beam_search(s.model, s.src, s.lens, w.beam, w.max_len, alpha=0.6)
    for b in range(s.src.shape[0]):
        n = int(out["len"][b])
        assert list(out["tok"][b, :n]) == res.tokens[b]
        assert list(out["align"][b, :n]) == res.align[b]
        rep = s.tr.replace_unk(out["tok"][b, :n], out["align"][b, :n], s.src[b], W.UNK_ID)
        assert rep == O.replace_unk(res.tokens[b], res.align[b], s.src[b])


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
