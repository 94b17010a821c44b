"""Pins for the oracle's LSTM cell and encoder (Section 2 items (a), (b); Tables 3-4 bi-RNN).

Each check ties the oracle to something other than itself: a closed form, a
library routine (torch's LSTMCell / packed LSTM on the CPU in float64), or an
invariance the definition implies.
"""

import math

import numpy as np
import pytest
import torch

from oracle.onmt_oracle import lstm_cell, run_direction, encode, sigmoid
from tests import _small

torch.set_default_dtype(torch.float64)


def test_closed_form_constant_bias():
    # All weight matrices 0, constant per-gate bias: i, f, g, o are constants,
    # so c_t = i*g*(1 - f^t)/(1 - f) and h_t = o*tanh(c_t).
    H, n_in, T = 3, 2, 7
    bias = np.array([0.3, -0.2, 0.7, 1.1])
    W = np.zeros((4 * H, n_in + H))
    b = np.repeat(bias, H)
    x = np.random.default_rng(0).normal(size=(1, T, n_in))
    real = np.ones((1, T), bool)
    out, h, c = run_direction(W, b, x, real, reverse=False)
    i, f, g, o = 1 / (1 + math.exp(-0.3)), 1 / (1 + math.exp(0.2)), math.tanh(0.7), 1 / (1 + math.exp(-1.1))
    for t in range(1, T + 1):
        ct = i * g * (1 - f ** t) / (1 - f)
        np.testing.assert_allclose(out[0, t - 1], o * math.tanh(ct), rtol=0, atol=1e-15)
    np.testing.assert_allclose(c[0], i * g * (1 - f ** T) / (1 - f), atol=1e-15)


def test_all_zero_weights_give_zero_state():
    W = np.zeros((8, 5))
    h, c = lstm_cell(W, np.zeros(8), np.ones((1, 3)), np.zeros((1, 2)), np.zeros((1, 2)))
    assert (h == 0).all() and (c == 0).all()


def test_hand_example_h1():
    # H = 1, one input: z_i = z_f = z_o = 0 (sigma = 1/2), z_g = atanh(1/2) (tanh = 1/2).
    # c' = 1/2 * c + 1/2 * 1/2, h' = 1/2 * tanh(c').
    W = np.zeros((4, 2))
    W[2, 0] = math.atanh(0.5)                    # g row, input column
    h, c = lstm_cell(W, np.zeros(4), np.array([[1.0]]), np.array([[0.0]]), np.array([[0.6]]))
    assert abs(c[0, 0] - 0.55) < 1e-15
    assert abs(h[0, 0] - 0.5 * math.tanh(0.55)) < 1e-15


def test_sigmoid_values():
    assert sigmoid(np.array(0.0)) == 0.5
    assert abs(sigmoid(np.array(math.log(3.0))) - 0.75) < 1e-15


@pytest.mark.parametrize("n_in,H", [(3, 4), (7, 5)])
def test_cell_matches_torch_lstmcell(n_in, H):
    rng = np.random.default_rng(n_in * 10 + H)
    W = rng.normal(size=(4 * H, n_in + H))
    b = rng.normal(size=4 * H)
    x, h, c = rng.normal(size=(6, n_in)), rng.normal(size=(6, H)), rng.normal(size=(6, H))
    cell = torch.nn.LSTMCell(n_in, H)                  # gate order (i, f, g, o)
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W[:, :n_in]))
        cell.weight_hh.copy_(torch.from_numpy(W[:, n_in:]))
        cell.bias_ih.copy_(torch.from_numpy(b))
        cell.bias_hh.zero_()
        th, tc = cell(torch.from_numpy(x), (torch.from_numpy(h), torch.from_numpy(c)))
    oh, oc = lstm_cell(W, b, x, h, c)
    np.testing.assert_allclose(oh, th.numpy(), atol=1e-13)
    np.testing.assert_allclose(oc, tc.numpy(), atol=1e-13)


@pytest.mark.parametrize("bi,layers", [(False, 1), (False, 2), (True, 2)])
def test_encoder_matches_torch_packed_lstm(bi, layers):
    # torch's packed (bi)LSTM is an independent implementation of the padded,
    # packed, stacked encoder: outputs [fwd ; bwd], zero at pads, h_n per layer/direction.
    w, ws, m = _small.model(seed=3, enc_layers=layers, dec_layers=layers, bidirectional=bi,
                            emb=5, hidden=6, src_vocab=20, len_lo=2, len_hi=7, batch=5)
    src, lens = _small.batch(w, seed=4)
    enc = encode(m, src, lens)
    Hd = w.enc_hidden
    lstm = torch.nn.LSTM(w.emb, Hd, num_layers=layers, bidirectional=bi, batch_first=True)
    with torch.no_grad():
        for l in range(layers):
            for d, sfx in (("fwd", ""), ("bwd", "_reverse"))[: 2 if bi else 1]:
                W = ws[f"enc{l}_{d}_W"].astype(np.float64)
                n_in = W.shape[1] - Hd
                getattr(lstm, f"weight_ih_l{l}{sfx}").copy_(torch.from_numpy(W[:, :n_in]))
                getattr(lstm, f"weight_hh_l{l}{sfx}").copy_(torch.from_numpy(W[:, n_in:]))
                getattr(lstm, f"bias_ih_l{l}{sfx}").copy_(torch.from_numpy(ws[f"enc{l}_{d}_b"].astype(np.float64)))
                getattr(lstm, f"bias_hh_l{l}{sfx}").zero_()
        x = torch.from_numpy(ws["E_src"].astype(np.float64)[src])
        packed = torch.nn.utils.rnn.pack_padded_sequence(x, torch.from_numpy(lens.astype(np.int64)),
                                                         batch_first=True, enforce_sorted=False)
        out, (hn, cn) = lstm(packed)
        out, _ = torch.nn.utils.rnn.pad_packed_sequence(out, batch_first=True, total_length=w.s_max)
    np.testing.assert_allclose(enc.memory, out.numpy(), atol=1e-13)
    ndir = 2 if bi else 1
    for l in range(layers):
        ref_h = torch.cat([hn[l * ndir + d] for d in range(ndir)], dim=-1).numpy()
        ref_c = torch.cat([cn[l * ndir + d] for d in range(ndir)], dim=-1).numpy()
        np.testing.assert_allclose(enc.final_h[l], ref_h, atol=1e-13)
        np.testing.assert_allclose(enc.final_c[l], ref_c, atol=1e-13)


def test_pad_invariance():
    # A sentence alone (no padding) gives the same memory and final state as inside a padded batch.
    w, ws, m = _small.model(seed=8, enc_layers=2, dec_layers=2, bidirectional=True, emb=5, hidden=6,
                            src_vocab=30, len_lo=2, len_hi=9, batch=4)
    src, lens = _small.batch(w, seed=9)
    full = encode(m, src, lens)
    for b in range(4):
        n = lens[b]
        alone = encode(m, src[b:b + 1, :n], lens[b:b + 1])
        np.testing.assert_allclose(full.memory[b, :n], alone.memory[0], atol=1e-14)
        assert (full.memory[b, n:] == 0).all()
        for l in range(2):
            np.testing.assert_allclose(full.final_h[l][b], alone.final_h[l][0], atol=1e-14)
            np.testing.assert_allclose(full.final_c[l][b], alone.final_c[l][0], atol=1e-14)


def test_backward_is_forward_on_reversed_input():
    rng = np.random.default_rng(2)
    W, b = rng.normal(size=(12, 5)) * 0.5, rng.normal(size=12) * 0.5
    x = rng.normal(size=(1, 6, 2))
    real = np.ones((1, 6), bool)
    ob, hb, cb = run_direction(W, b, x, real, reverse=True)
    of, hf, cf = run_direction(W, b, x[:, ::-1], real, reverse=False)
    np.testing.assert_allclose(ob, of[:, ::-1], atol=1e-15)
    np.testing.assert_allclose(hb, hf, atol=1e-15)
