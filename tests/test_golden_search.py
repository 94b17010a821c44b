"""The stored oracle searches (tests/golden/search_*.npz) are current: written from today's seeded inputs
by today's oracle (Section 2 item (d) beam search; Section 4.2 length normalisation).

The files are written by tests/golden/make_search_golden.py, which calls only the oracle. Here the cheap
parts are recomputed: the inputs of every file, the whole tiny workload at all three seeds, and one
sentence of the paper-default workload (2x500, beam 5, Table 2 shape).
"""

import os

import numpy as np
import pytest

import workloads as W
from oracle import onmt_oracle as O

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NAMES = ("tiny", "default", "larger", "greedy", "long")


def _load(name, seed):
    with np.load(os.path.join(HERE, f"search_{name}_seed{seed}.npz"), allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


@pytest.mark.parametrize("name", NAMES)
def test_golden_files_hold_todays_inputs(name):
    w = W.get(name)
    for off in (0, 1, 2):
        g = _load(name, 1000 + w.index + off)
        src, lens = W.make_batch(w, seed=1000 + w.index + off)
        np.testing.assert_array_equal(g["src"], src)
        np.testing.assert_array_equal(g["lens"], lens)
        B = w.batch
        assert g["tokens"].shape == (B, w.max_len)
        assert ((g["len"] >= 1) & (g["len"] <= w.max_len)).all()
        for b in range(B):
            assert (g["tokens"][b, g["len"][b]:] == W.PAD_ID).all()
        assert (g["steps"] >= g["len"]).all() and (g["margin"] >= 0).all()
        np.testing.assert_allclose(g["norm"], g["raw"] / O.length_penalty(g["len"], w.alpha), rtol=1e-12)


def _check(g, res, rows):
    # fp64 products over a different number of rows may round differently (BLAS blocking), hence 1e-9
    for i, b in enumerate(rows):
        assert res.tokens[i] == [int(x) for x in g["tokens"][b, :g["len"][b]]]
        assert abs(res.raw[i] - g["raw"][b]) < 1e-9 and abs(res.norm[i] - g["norm"][b]) < 1e-9
        assert res.steps[i] == g["steps"][b] and abs(res.margin[i] - g["margin"][b]) < 1e-9


def test_golden_tiny_recomputed():
    w = W.get("tiny")
    m = O.model_from(w, W.make_weights(w))
    for off in (0, 1, 2):
        g = _load("tiny", 1000 + w.index + off)
        res = O.beam_search(m, g["src"], g["lens"], w.beam, w.max_len, w.alpha)
        _check(g, res, range(w.batch))


@pytest.mark.slow
def test_golden_default_sentence_recomputed():
    w = W.get("default")
    m = O.model_from(w, W.make_weights(w))
    g = _load("default", 1000 + w.index + 1)
    res = O.beam_search(m, g["src"][:1], g["lens"][:1], w.beam, w.max_len, w.alpha)
    _check(g, res, [0])
