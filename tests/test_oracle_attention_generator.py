"""Pins for the oracle's attention, generator and decoder step.

Section 2 (attention pooling, softmax layer), Section 2 item (c) (input
feeding), Section 4.2 ("general" attention), Figure 1(a) caption.
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import onmt_oracle as O
from tests import _small


def _attn_inputs(seed, N=5, S=7, H=6, Hm=6):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(N, H))
    mem = rng.normal(size=(N, S, Hm))
    lens = rng.integers(1, S + 1, size=N)
    mask = np.arange(S)[None, :] < lens[:, None]
    mem = np.where(mask[..., None], mem, 0.0)
    return q, mem, mask, lens


def _model_with(**w):
    m = O.Model(1, 1, False, 2, 6, 3, 3, {k: np.asarray(v, np.float64) for k, v in w.items()})
    return m


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_attention_matches_torch_sdpa(seed):
    # general score q^T W_a m_s == dot(q, key_s) with keys = m W_a^T; torch's SDPA with
    # scale 1 and a -inf mask is an independent softmax/weighted-sum routine.
    q, mem, mask, _ = _attn_inputs(seed, H=6, Hm=4)
    rng = np.random.default_rng(seed + 100)
    W_a, W_c = rng.normal(size=(6, 4)), rng.normal(size=(6, 10))
    m = _model_with(W_a=W_a, W_c=W_c)
    a, ctx, ht = O.attention(m, q, mem, mask)
    tq = torch.from_numpy(q)[:, None, None, :]                           # [N,1,1,H]
    tk = torch.from_numpy(mem @ W_a.T)[:, None]                           # [N,1,S,H]
    tv = torch.from_numpy(mem)[:, None]                                   # [N,1,S,Hm]
    bias = torch.from_numpy(np.where(mask, 0.0, -np.inf))[:, None, None, :]
    ref = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=bias, scale=1.0)[:, 0, 0]
    np.testing.assert_allclose(ctx, ref.numpy(), atol=1e-12)
    ref_a = torch.softmax(torch.from_numpy(np.einsum("nh,nsh->ns", q, mem @ W_a.T)) + bias[:, 0, 0], -1)
    np.testing.assert_allclose(a, ref_a.numpy(), atol=1e-13)
    ref_ht = torch.tanh(F.linear(torch.cat([ref, torch.from_numpy(q)], -1), torch.from_numpy(W_c)))
    np.testing.assert_allclose(ht, ref_ht.numpy(), atol=1e-12)


def test_attention_invariants():
    q, mem, mask, lens = _attn_inputs(4)
    rng = np.random.default_rng(5)
    m = _model_with(W_a=rng.normal(size=(6, 6)), W_c=rng.normal(size=(6, 12)))
    a, ctx, _ = O.attention(m, q, mem, mask)
    assert np.all(np.abs(a.sum(1) - 1) <= 1e-12)
    assert (a[~mask] == 0).all()                       # exactly zero on pads
    # one real position: weight 1, context = that row
    mask1 = np.zeros_like(mask)
    mask1[:, 0] = True
    a1, ctx1, _ = O.attention(m, q, mem, mask1)
    assert (a1[:, 0] == 1).all()
    np.testing.assert_array_equal(ctx1, mem[:, 0])


def test_attention_zero_wa_is_mean_of_real_rows():
    q, mem, mask, lens = _attn_inputs(6)
    m = _model_with(W_a=np.zeros((6, 6)), W_c=np.zeros((6, 12)))
    a, ctx, ht = O.attention(m, q, mem, mask)
    for n in range(len(q)):
        np.testing.assert_allclose(ctx[n], mem[n, :lens[n]].mean(0), atol=1e-14)
    assert (ht == 0).all()                             # W_c = 0 gives h_tilde = 0


def test_attention_concat_order_is_ctx_then_query():
    q, mem, mask, _ = _attn_inputs(7)
    I = np.eye(6)
    Z = np.zeros((6, 6))
    rng = np.random.default_rng(8)
    W_a = rng.normal(size=(6, 6))
    _, ctx, ht = O.attention(_model_with(W_a=W_a, W_c=np.hstack([I, Z])), q, mem, mask)
    np.testing.assert_allclose(ht, np.tanh(ctx), atol=1e-15)
    _, _, ht = O.attention(_model_with(W_a=W_a, W_c=np.hstack([Z, I])), q, mem, mask)
    np.testing.assert_allclose(ht, np.tanh(q), atol=1e-15)


def test_generator_invariants_and_torch():
    rng = np.random.default_rng(9)
    V, H = 50, 7
    W_s, b_s = rng.normal(size=(V, H)), rng.normal(size=V)
    h = rng.normal(size=(4, H))
    m = O.Model(1, 1, False, 2, H, 3, V, {"W_s": W_s, "b_s": b_s})
    lp = O.generator(m, h)
    ref = torch.log_softmax(F.linear(torch.from_numpy(h), torch.from_numpy(W_s), torch.from_numpy(b_s)), -1)
    np.testing.assert_allclose(lp, ref.numpy(), atol=1e-13)
    assert np.all(np.abs(np.log(np.exp(lp).sum(1))) < 1e-13)     # logsumexp(logp) == 0
    m0 = O.Model(1, 1, False, 2, H, 3, V, {"W_s": np.zeros((V, H)), "b_s": b_s})
    np.testing.assert_allclose(O.generator(m0, h), np.broadcast_to(torch.log_softmax(torch.from_numpy(b_s), 0).numpy(), (4, V)), atol=1e-14)
    mz = O.Model(1, 1, False, 2, H, 3, 50000, {"W_s": np.zeros((50000, H)), "b_s": np.zeros(50000)})
    lz = O.generator(mz, h[:1])
    assert np.all(np.abs(lz + math.log(50000)) < 1e-12)
    assert abs(math.log(50000) - 10.8198) < 1e-4 and abs(math.log(1000) - 6.9078) < 1e-4


def test_decoder_input_order_is_embedding_then_feed():
    # Zero the feed columns of decoder layer 1: the step must then ignore the feed vector.
    w, ws, m = _small.model(seed=12, emb=4, hidden=8, src_vocab=9, tgt_vocab=9)
    E, H = w.emb, w.hidden
    m.w["dec0_W"][:, E:E + H] = 0.0
    src, lens = _small.batch(w, seed=2)
    enc = O.encode(m, src, lens)
    st = O.init_state(m, enc, 1)
    st2 = O.State(st.h, st.c, np.random.default_rng(0).normal(size=st.feed.shape))
    rows = np.arange(src.shape[0])
    _, lp1, _ = O.decode_step(m, enc, st, np.full(len(rows), 5), rows)
    _, lp2, _ = O.decode_step(m, enc, st2, np.full(len(rows), 5), rows)
    np.testing.assert_array_equal(lp1, lp2)
    _, lp3, _ = O.decode_step(m, enc, st, np.full(len(rows), 6), rows)
    assert np.abs(lp3 - lp1).max() > 1e-6          # ...but not the embedding


def test_decode_step_matches_torch_composition():
    # One decoder step built from torch library pieces (LSTMCell stack, SDPA, linear, log_softmax).
    w, ws, m = _small.model(seed=21, enc_layers=2, dec_layers=2, emb=5, hidden=6, src_vocab=15, tgt_vocab=11,
                            len_lo=3, len_hi=6, batch=3)
    src, lens = _small.batch(w, seed=22)
    enc = O.encode(m, src, lens)
    st = O.init_state(m, enc, 2)
    rng = np.random.default_rng(1)
    st = O.State([rng.normal(size=a.shape) for a in st.h], [rng.normal(size=a.shape) for a in st.c],
                 rng.normal(size=st.feed.shape))
    prev = rng.integers(0, 11, size=6)
    rows = np.repeat(np.arange(3), 2)
    new, lp, a = O.decode_step(m, enc, st, prev, rows)
    T = lambda x: torch.from_numpy(np.asarray(x, np.float64))
    x = torch.cat([T(m.w["E_tgt"][prev]), T(st.feed)], -1)
    for l in range(2):
        Wl = m.w[f"dec{l}_W"]
        n_in = Wl.shape[1] - 6
        cell = torch.nn.LSTMCell(n_in, 6).double()
        with torch.no_grad():
            cell.weight_ih.copy_(T(Wl[:, :n_in]))
            cell.weight_hh.copy_(T(Wl[:, n_in:]))
            cell.bias_ih.copy_(T(m.w[f"dec{l}_b"]))
            cell.bias_hh.zero_()
            h, c = cell(x, (T(st.h[l]), T(st.c[l])))
        np.testing.assert_allclose(new.h[l], h.detach().numpy(), atol=1e-13)
        np.testing.assert_allclose(new.c[l], c.detach().numpy(), atol=1e-13)
        x = h.detach()
    mem = T(enc.memory[rows])
    bias = T(np.where(enc.mask[rows], 0.0, -np.inf))[:, None, None, :]
    ctx = F.scaled_dot_product_attention(x[:, None, None, :], (mem @ T(m.w["W_a"]).T)[:, None], mem[:, None],
                                         attn_mask=bias, scale=1.0)[:, 0, 0]
    ht = torch.tanh(F.linear(torch.cat([ctx, x], -1), T(m.w["W_c"])))
    np.testing.assert_allclose(new.feed, ht.numpy(), atol=1e-12)
    ref = torch.log_softmax(F.linear(ht, T(m.w["W_s"]), T(m.w["b_s"])), -1)
    np.testing.assert_allclose(lp, ref.numpy(), atol=1e-12)
