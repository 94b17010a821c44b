"""Pin for the decoder's initial state (Figure 1(a) caption: the encoder's final time step initialises
the target RNN; Section 2 item (c): input feeding; readings R5 and R7).

The first decoder step is rebuilt from torch library pieces with no oracle code in the chain: torch's
packed (optionally bidirectional) multi-layer LSTM gives the encoder's final states h_n / c_n and its
outputs; decoder layer l starts from encoder layer l's final state ([forward ; backward] for a
bidirectional encoder), the input feed is zero, and the step is an LSTMCell stack, scaled dot-product
attention over the memory, tanh(W_c [ctx ; q]) and log_softmax. A slip in the layer order, the
direction order, the row replication across the beam or a non-zero initial feed changes the result.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from torch.nn.utils.rnn import pack_padded_sequence, pad_packed_sequence

from oracle import onmt_oracle as O
from workloads.configs import BOS_ID
from tests import _small


def _T(x):
    return torch.from_numpy(np.asarray(x, np.float64))


def _torch_encoder(m, src, lens):
    """torch.nn.LSTM over the packed batch: (memory [B, S, Hm] zero at pads, h_n, c_n [L * ndir, B, Hd])."""
    ndir = 2 if m.bidirectional else 1
    Hd = m.enc_hidden
    lstm = torch.nn.LSTM(m.emb, Hd, num_layers=m.enc_layers, bidirectional=m.bidirectional,
                         batch_first=True).double()
    with torch.no_grad():
        for l in range(m.enc_layers):
            for d, name in enumerate(("fwd", "bwd")[:ndir]):
                sfx = f"_l{l}" + ("_reverse" if d else "")
                W = m.w[f"enc{l}_{name}_W"]
                n_in = W.shape[1] - Hd
                getattr(lstm, "weight_ih" + sfx).copy_(_T(W[:, :n_in]))
                getattr(lstm, "weight_hh" + sfx).copy_(_T(W[:, n_in:]))
                getattr(lstm, "bias_ih" + sfx).copy_(_T(m.w[f"enc{l}_{name}_b"]))
                getattr(lstm, "bias_hh" + sfx).zero_()
        x = _T(m.w["E_src"][np.asarray(src)])
        packed = pack_padded_sequence(x, torch.from_numpy(np.asarray(lens, np.int64)), batch_first=True,
                                      enforce_sorted=False)
        out, (h_n, c_n) = lstm(packed)
        mem, _ = pad_packed_sequence(out, batch_first=True, total_length=src.shape[1])
    return mem, h_n, c_n


@pytest.mark.parametrize("bidirectional", [False, True])
def test_first_decoder_step_from_torch_packed_encoder(bidirectional):
    L, H, K = 2, 6, 2
    w, ws, m = _small.model(seed=91, enc_layers=L, dec_layers=L, bidirectional=bidirectional, emb=5,
                            hidden=H, src_vocab=15, tgt_vocab=11, len_lo=2, len_hi=6, batch=4,
                            scale={k: 8.0 for k in ("dec0_W", "dec1_W", "W_a", "W_c", "W_s")})
    src, lens = _small.batch(w, seed=92)
    B = src.shape[0]
    ndir = 2 if bidirectional else 1
    mem, h_n, c_n = _torch_encoder(m, src, lens)

    # the oracle: encoder, initial state replicated to K rows per sentence, one step from BOS
    enc = O.encode(m, src, lens)
    st = O.init_state(m, enc, K)
    rows = np.repeat(np.arange(B), K)
    new, lp, a = O.decode_step(m, enc, st, np.full(B * K, BOS_ID), rows)

    # torch: decoder layer l starts from encoder layer l's final state, directions concatenated; feed 0
    rep = lambda t: t.repeat_interleave(K, dim=0)
    h0 = [rep(torch.cat([h_n[l * ndir + d] for d in range(ndir)], -1)) for l in range(L)]
    c0 = [rep(torch.cat([c_n[l * ndir + d] for d in range(ndir)], -1)) for l in range(L)]
    x = torch.cat([_T(m.w["E_tgt"][np.full(B * K, BOS_ID)]), torch.zeros(B * K, H, dtype=torch.float64)], -1)
    with torch.no_grad():
        for l in range(L):
            Wl = m.w[f"dec{l}_W"]
            n_in = Wl.shape[1] - H
            cell = torch.nn.LSTMCell(n_in, H).double()
            cell.weight_ih.copy_(_T(Wl[:, :n_in]))
            cell.weight_hh.copy_(_T(Wl[:, n_in:]))
            cell.bias_ih.copy_(_T(m.w[f"dec{l}_b"]))
            cell.bias_hh.zero_()
            h, c = cell(x, (h0[l], c0[l]))
            np.testing.assert_allclose(new.h[l], h.numpy(), atol=1e-12)
            np.testing.assert_allclose(new.c[l], c.numpy(), atol=1e-12)
            x = h
        memr = rep(mem)
        mask = np.arange(src.shape[1])[None, :] < np.asarray(lens)[:, None]
        bias = _T(np.where(np.repeat(mask, K, 0), 0.0, -np.inf))[:, None, None, :]
        ctx = F.scaled_dot_product_attention(x[:, None, None, :], (memr @ _T(m.w["W_a"]).T)[:, None],
                                             memr[:, None], attn_mask=bias, scale=1.0)[:, 0, 0]
        ht = torch.tanh(F.linear(torch.cat([ctx, x], -1), _T(m.w["W_c"])))
        ref = torch.log_softmax(F.linear(ht, _T(m.w["W_s"]), _T(m.w["b_s"])), -1)
    np.testing.assert_allclose(enc.memory, mem.numpy(), atol=1e-12)
    np.testing.assert_allclose(new.feed, ht.numpy(), atol=1e-12)
    np.testing.assert_allclose(lp, ref.numpy(), atol=1e-12)
    # the state the pin starts from is not trivially symmetric: layers and sentences differ
    assert np.abs(h0[0].numpy() - h0[1].numpy()).max() > 1e-3
    assert np.abs(lp[0] - lp[K]).max() > 1e-6
