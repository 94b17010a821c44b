"""Pins for the oracle's hypothesis filters and unknown-word replacement (Section 4.2: beam search under a
limit on unknown words and word-level constraints on the search, and OOV handling; readings R18,
R19).

A beam wide enough to keep every hypothesis must return the exhaustive-search optimum over the allowed
sequences; all-zero weights make every candidate tie (the smallest allowed id wins) and make attention
uniform (every token aligns to source position 0).
"""

import numpy as np
import pytest

from oracle import onmt_oracle as O
from workloads.configs import EOS_ID, PAD_ID, UNK_ID
from tests import _small


@pytest.mark.parametrize("banned,max_unk", [((2,), -1), ((4, 5), 0), ((), 1), ((0, 2), 0)])
def test_wide_beam_equals_brute_force_with_filters(banned, max_unk):
    w, ws, m = _small.model(seed=13, tgt_vocab=6, src_vocab=6, len_lo=2, len_hi=4,
                            scale={"W_s": 6.0, "b_s": 6.0})
    src, lens = _small.batch(w, seed=14)
    res = O.beam_search(m, src, lens, K=6 ** 3, max_len=3, banned=banned, max_unk=max_unk)
    for b in range(len(lens)):
        toks, raw, norm = O.brute_force(m, src[b], lens[b], max_len=3, banned=banned, max_unk=max_unk)
        assert res.tokens[b] == toks
        assert abs(res.norm[b] - norm) < 1e-12
        assert not set(res.tokens[b]) & set(banned)
        if max_unk >= 0:
            assert res.tokens[b].count(UNK_ID) <= max_unk


@pytest.mark.parametrize("banned,max_unk,want", [((PAD_ID,), -1, [UNK_ID] * 6), ((PAD_ID,), 0, [2] * 6),
                                                 ((PAD_ID, 2), 0, [EOS_ID]), ((PAD_ID, 2, EOS_ID), 0, [4] * 6)])
def test_zero_weights_smallest_allowed_id_wins(banned, max_unk, want):
    w, ws, m = _small.model(seed=1, tgt_vocab=50, src_vocab=50)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=1, max_len=6, banned=banned, max_unk=max_unk)
    for b in range(len(lens)):
        assert res.tokens[b] == want
        assert res.align[b] == [0] * len(want)


def test_unk_limit_counts_along_the_hypothesis():
    # UNK is the smallest allowed id once PAD is banned: exactly max_unk UNKs, then the next id
    w, ws, m = _small.model(seed=1, tgt_vocab=50, src_vocab=50)
    for k in m.w:
        m.w[k][...] = 0.0
    src, lens = _small.batch(w)
    res = O.beam_search(m, src, lens, K=1, max_len=6, banned=(PAD_ID,), max_unk=2)
    for b in range(len(lens)):
        assert res.tokens[b] == [UNK_ID, UNK_ID, 2, 2, 2, 2]


def test_alignment_follows_the_output_and_unk_replacement():
    w, ws, m = _small.model(seed=17, emb=6, hidden=10, src_vocab=30, tgt_vocab=30, len_lo=4, len_hi=8,
                            batch=3, scale={"W_a": 30.0, "W_s": 8.0, "b_s": 8.0})
    src, lens = _small.batch(w, seed=18)
    res = O.beam_search(m, src, lens, K=3, max_len=8)
    for b in range(3):
        toks = res.tokens[b]
        # recompute each step's attention along the output (teacher forcing) and take its argmax
        enc = O.encode(m, src[b:b + 1], lens[b:b + 1])
        st = O.init_state(m, enc, 1)
        prev = O.BOS_ID
        for t, tok in enumerate(toks):
            st, _, a = O.decode_step(m, enc, st, np.array([prev]), np.array([0]))
            assert res.align[b][t] == int(np.argmax(a[0, :lens[b]]))
            assert 0 <= res.align[b][t] < lens[b]
            prev = tok
        rep = O.replace_unk([UNK_ID] + toks, [1] + res.align[b], src[b])
        assert rep[0] == ("src", int(src[b, 1]))
        assert all(r[0] == ("src" if t == UNK_ID else "tgt") for r, t in zip(rep[1:], toks))
