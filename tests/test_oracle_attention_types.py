"""Pins for the oracle's "dot" and "concat" attention types (Section 4.2 names general, dot product and
concatenation attention, citing Luong et al. 2015; reading R20).

dot: torch's scaled-dot-product attention with the memory as keys (scale 1) is an independent routine,
and dot equals "general" with W_a = I. concat: closed forms that a dropped tanh, a dropped or misplaced
v_a, or swapped query/memory halves of W_a would break: a query-only W_a gives uniform weights; a
memory-only W_a gives weights independent of the query; a saturating memory-only W_a gives scores
sum_a v_a sign(m_s[a]); a vanishing W_a makes log(a_s / a_0) / eps tend to v_a . W_m (m_s - m_0).
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import onmt_oracle as O
from tests import _small

H = 6


def _inputs(seed, N=5, S=7, Hm=H):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(N, H))
    mem = rng.normal(size=(N, S, Hm))
    lens = rng.integers(2, S + 1, size=N)
    lens[0] = S
    mask = np.arange(S)[None, :] < lens[:, None]
    mem = np.where(mask[..., None], mem, 0.0)
    return q, mem, mask, lens


def _model(attn, Hm=H, **w):
    rng = np.random.default_rng(77)
    w.setdefault("W_c", rng.normal(size=(H, Hm + H)))
    return O.Model(1, 1, False, 2, H, 3, 3, {k: np.asarray(v, np.float64) for k, v in w.items()}, attn)


@pytest.mark.parametrize("seed", [0, 1])
def test_dot_matches_torch_sdpa(seed):
    q, mem, mask, _ = _inputs(seed)
    m = _model("dot")
    a, ctx, ht = O.attention(m, q, mem, mask)
    tm = torch.from_numpy(mem)[:, None]
    bias = torch.from_numpy(np.where(mask, 0.0, -np.inf))[:, None, None, :]
    ref = F.scaled_dot_product_attention(torch.from_numpy(q)[:, None, None, :], tm, tm, attn_mask=bias,
                                         scale=1.0)[:, 0, 0]
    np.testing.assert_allclose(ctx, ref.numpy(), atol=1e-12)
    ref_ht = torch.tanh(F.linear(torch.cat([ref, torch.from_numpy(q)], -1), torch.from_numpy(m.w["W_c"])))
    np.testing.assert_allclose(ht, ref_ht.numpy(), atol=1e-12)
    assert (a[~mask] == 0).all() and np.all(np.abs(a.sum(1) - 1) <= 1e-12)


def test_dot_is_general_with_identity():
    q, mem, mask, _ = _inputs(2)
    a_dot, ctx_dot, _ = O.attention(_model("dot"), q, mem, mask)
    a_gen, ctx_gen, _ = O.attention(_model("general", W_a=np.eye(H)), q, mem, mask)
    np.testing.assert_allclose(a_dot, a_gen, atol=1e-14)
    np.testing.assert_allclose(ctx_dot, ctx_gen, atol=1e-14)


def _concat(Wq, Wm, v, Hm):
    return _model("concat", Hm=Hm, W_a=np.hstack([Wq, Wm]), v_a=v)


def test_concat_query_only_is_uniform():
    Hm = 4
    q, mem, mask, lens = _inputs(3, Hm=Hm)
    rng = np.random.default_rng(4)
    m = _concat(rng.normal(size=(H, H)), np.zeros((H, Hm)), rng.normal(size=H), Hm)
    a, ctx, _ = O.attention(m, q, mem, mask)
    for n in range(len(q)):
        np.testing.assert_allclose(a[n, :lens[n]], 1.0 / lens[n], atol=1e-14)
        np.testing.assert_allclose(ctx[n], mem[n, :lens[n]].mean(0), atol=1e-14)


def test_concat_memory_only_ignores_the_query():
    Hm = 4
    q, mem, mask, _ = _inputs(5, Hm=Hm)
    mem[:] = mem[0]
    mask[:] = mask[0]
    rng = np.random.default_rng(6)
    m = _concat(np.zeros((H, H)), rng.normal(size=(H, Hm)), rng.normal(size=H), Hm)
    a, _, _ = O.attention(m, q, mem, mask)
    assert np.ptp(a, axis=0).max() <= 1e-15          # every query row gets the same weights
    assert np.ptp(a[0, mask[0]]) > 1e-3               # ... which are not uniform


def test_concat_saturated_scores_are_signed_sums_of_v():
    Hm = 4
    q, mem, mask, lens = _inputs(7, Hm=Hm)
    mem = np.where(np.abs(mem) < 0.05, 0.05, mem) * mask[..., None]  # no entry near zero on real rows
    rng = np.random.default_rng(8)
    v = rng.normal(size=Hm)
    Wm = np.zeros((H, Hm))
    Wm[:Hm, :Hm] = 1e4 * np.eye(Hm)                  # unit a < Hm sees memory feature a, saturated
    m = _concat(np.zeros((H, H)), Wm, np.concatenate([v, [3.0, -2.0]]), Hm)
    a, _, _ = O.attention(m, q, mem, mask)
    for n in range(len(q)):
        e = [sum(v[j] * (1.0 if mem[n, s, j] > 0 else -1.0) for j in range(Hm)) for s in range(lens[n])]
        p = np.exp(np.array(e) - max(e))
        np.testing.assert_allclose(a[n, :lens[n]], p / p.sum(), atol=1e-13)


def test_concat_small_weights_are_linear_in_the_memory():
    Hm, eps = 4, 1e-5
    q, mem, mask, lens = _inputs(9, Hm=Hm)
    rng = np.random.default_rng(10)
    Wq, Wm, v = rng.normal(size=(H, H)), rng.normal(size=(H, Hm)), rng.normal(size=H)
    a, _, _ = O.attention(_concat(eps * Wq, eps * Wm, v, Hm), q, mem, mask)
    for n in range(len(q)):
        for s in range(1, lens[n]):
            slope = np.log(a[n, s] / a[n, 0]) / eps
            expect = sum(v[i] * sum(Wm[i, j] * (mem[n, s, j] - mem[n, 0, j]) for j in range(Hm)) for i in range(H))
            assert abs(slope - expect) <= 1e-6 * (1 + abs(expect))


@pytest.mark.parametrize("attn", ["dot", "concat"])
def test_wide_beam_equals_brute_force(attn):
    w, ws, m = _small.model(seed=9, tgt_vocab=6, src_vocab=6, len_lo=2, len_hi=4, attn=attn,
                            scale={"W_s": 6.0, "b_s": 6.0})
    src, lens = _small.batch(w, seed=10)
    res = O.beam_search(m, src, lens, K=6 ** 3, max_len=3)
    for b in range(len(lens)):
        toks, raw, norm = O.brute_force(m, src[b], lens[b], max_len=3)
        assert res.tokens[b] == toks
        assert abs(res.raw[b] - raw) < 1e-12


@pytest.mark.parametrize("attn", ["dot", "concat"])
def test_weight_specs_per_type(attn):
    w, ws, m = _small.model(attn=attn)
    names = list(ws)
    if attn == "dot":
        assert "W_a" not in names and "v_a" not in names
    else:
        assert ws["W_a"].shape == (w.hidden, 2 * w.hidden) and ws["v_a"].shape == (w.hidden,)
    assert names[-3:] == ["W_c", "W_s", "b_s"]
