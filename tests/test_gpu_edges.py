"""GPU edge cases against the oracle: degenerate shapes (one-token sources, ragged length extremes in one
batch, a single sentence, a single decode step, beam 1 = greedy), the largest sizes the kernels support
(target vocabulary 131072 = 64 lanes x 16 generator tiles per lane in the beam step; beam 16 over a
1024-position source, the attention workgroups' LDS limit), and inputs the library must refuse before it
launches anything (Section 2's batched translation over padded sources; the C interface's conventions).
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import TAU, ATTN_TOL, with_workload, check_search, translator_for

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

TINY = W.get("tiny")


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


class Custom:
    """The peaked model of workload w on a seeded batch whose source lengths are given."""

    def __init__(self, w, lens, peaked=True, seed=77):
        self.w = w
        self.weights = W.make_weights(w, peaked=peaked)
        self.model = O.model_from(w, self.weights)
        src, _ = W.make_batch(w, seed=seed, batch=len(lens))
        lens = np.asarray(lens, np.int32)
        src[np.arange(w.s_max)[None, :] >= lens[:, None]] = W.PAD_ID
        self.src, self.lens = src, lens
        self.tr = translator_for(w, self.weights)
        self.src_d = torch.from_numpy(src).cuda()
        self.lens_d = torch.from_numpy(lens).cuda()
        self.tau = TAU[w.wdtype]


def _search(s, K, T, alpha=0.0):
    B, S = s.src.shape
    buf = s.tr.search_buffers(B, S, K, T, alpha, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    return buf


def _first_step(s, K):
    """Full log-distribution and attention of the first decoder step, GPU and oracle."""
    B, S = s.src.shape
    ws = s.tr.encode(s.src_d, s.lens_d)
    st = s.tr.decode_init(ws, B, S, K)
    tok = torch.full((B * K,), W.BOS_ID, dtype=torch.int32, device="cuda")
    _, logp, _, _, attn = s.tr.decode_step(ws, B, S, K, st, tok, None, mode=0, want_attn=True)
    torch.cuda.synchronize()
    enc = O.encode(s.model, s.src, s.lens)
    rows = np.repeat(np.arange(B), K)
    _, o_logp, o_attn = O.decode_step(s.model, enc, O.init_state(s.model, enc, K), np.full(B * K, W.BOS_ID), rows)
    return logp.cpu().numpy(), attn.cpu().numpy(), o_logp, o_attn


def test_one_token_sources():
    w = with_workload(TINY, len_lo=1, len_hi=1)
    s = Custom(w, [1, 1, 1])
    _case("one_token_sources", B=3)
    g_logp, g_attn, o_logp, o_attn = _first_step(s, 2)
    assert np.abs(g_logp - o_logp).max() <= s.tau
    assert (g_attn[:, 0] == 1.0).all()                  # one real position takes all the weight
    check_search(s, _search(s, w.beam, w.max_len), range(3), w.beam, w.max_len, 0.0)


def test_ragged_extremes_in_one_batch():
    s = Custom(TINY, [1, 10, 2, 9, 10])
    _case("ragged", lens=list(s.lens))
    g_logp, g_attn, o_logp, o_attn = _first_step(s, 3)
    assert np.abs(g_logp - o_logp).max() <= s.tau
    np.testing.assert_allclose(g_attn, o_attn, atol=ATTN_TOL["fp32"], rtol=0)
    assert (g_attn[np.arange(g_attn.shape[1])[None, :] >= np.repeat(s.lens, 3)[:, None]] == 0).all()
    check_search(s, _search(s, 4, 12, 0.6), range(5), 4, 12, 0.6)


def test_one_sentence():
    s = Custom(TINY, [7])
    _case("one_sentence")
    check_search(s, _search(s, 3, 12), [0], 3, 12, 0.0)


def test_one_decode_step():
    s = Custom(TINY, [3, 10, 5, 1])
    _case("max_decode_1")
    buf = _search(s, 2, 1)
    assert (buf["len"].cpu().numpy() == 1).all()
    check_search(s, buf, range(4), 2, 1, 0.0)


def test_beam_one_is_greedy():
    s = Custom(TINY, [4, 10, 6, 8])
    _case("beam_1_greedy")
    buf = _search(s, 1, 12)
    toks, _ = O.greedy(s.model, s.src, s.lens, 12)
    g_tok, g_len = buf["tok"].cpu().numpy(), buf["len"].cpu().numpy()
    for b in range(4):
        assert list(g_tok[b, :g_len[b]]) == toks[b]


def test_largest_vocabulary():
    w = with_workload(TINY, tgt_vocab=131072, max_len=4)
    s = Custom(w, [6, 10])
    _case("vocab_131072")
    g_logp, _, o_logp, _ = _first_step(s, 2)
    assert np.abs(g_logp - o_logp).max() <= s.tau
    check_search(s, _search(s, 16, 4), range(2), 16, 4, 0.0)


def test_beam_16_over_1024_positions():
    w = with_workload(TINY, len_lo=1024, len_hi=1024, max_len=3)
    s = Custom(w, [1024, 700])
    _case("beam_16_S_1024")
    check_search(s, _search(s, 16, 3), range(2), 16, 3, 0.0)
    # one position more does not fit the attention workgroup at beam 16
    w2 = with_workload(TINY, len_lo=1025, len_hi=1025, max_len=3)
    s2 = Custom(w2, [1025, 3])
    from paper_1805_11462_amd._lib import OnmtError
    with pytest.raises(OnmtError):
        _search(s2, 16, 3)


def test_invalid_inputs_are_refused():
    from paper_1805_11462_amd._lib import OnmtError
    s = Custom(TINY, [3, 5])
    B, S = s.src.shape
    _case("invalid_inputs")

    def search(src, lens, K=2, T=5):
        buf = s.tr.search_buffers(B, S, K, T, 0.0)
        s.tr.beam_search(torch.from_numpy(np.ascontiguousarray(src)).cuda(),
                         torch.from_numpy(np.asarray(lens, np.int32)).cuda(), buf)
        torch.cuda.synchronize()
        return buf

    for bad_lens in ([0, 5], [3, S + 1], [-1, 2]):
        with pytest.raises(OnmtError):
            search(s.src, bad_lens)
    for bad_id in (TINY.src_vocab, -3):
        bad = s.src.copy()
        bad[1, 0] = bad_id
        with pytest.raises(OnmtError):
            search(bad, s.lens)
    with pytest.raises(OnmtError):
        search(s.src, s.lens, K=17)
    # a decoder step fed a token outside the target vocabulary
    ws = s.tr.encode(s.src_d, s.lens_d)
    st = s.tr.decode_init(ws, B, S, 1)
    tok = torch.tensor([W.BOS_ID, TINY.tgt_vocab], dtype=torch.int32, device="cuda")
    with pytest.raises(OnmtError):
        s.tr.decode_step(ws, B, S, 1, st, tok, None, mode=0)
    # ids past a sentence's length are never read, so they may be anything; and after the refusals the
    # library still works
    ok = s.src.copy()
    ok[0, 4] = 99999
    buf = search(ok, s.lens)
    ref = search(s.src, s.lens)
    assert torch.equal(buf["tok"], ref["tok"])


def test_workspace_operands_past_the_descriptor_limit_are_refused():
    # the GEMMs read the memory bank and state rows through 2 GiB buffer descriptors: B * S_max source
    # positions (or B * beam rows) whose operands would reach 2 GiB are refused before anything is read
    # (the tiny workspace below would otherwise be refused as too small; no input buffer is touched)
    import ctypes
    from paper_1805_11462_amd import _lib
    s = Custom(TINY, [3, 5])
    lib = s.tr.lib
    _case("descriptor_limit")
    dummy = torch.zeros(64, dtype=torch.int32, device="cuda")
    ws = torch.zeros(1024, dtype=torch.uint8, device="cuda")
    B, S = 1 << 13, 1 << 10                       # 2^23 positions x 128 padded columns x 4 bytes = 4 GiB
    rc = lib.onmt_encode(s.tr.handle, ctypes.c_void_p(dummy.data_ptr()), ctypes.c_void_p(dummy.data_ptr()), B, S,
                         ctypes.c_void_p(ws.data_ptr()), 1024, None)
    assert rc == _lib.ONMT_EUNSUPPORTED and b"2 GiB" in lib.onmt_last_error()
    rc = lib.onmt_decode_init(s.tr.handle, ctypes.c_void_p(ws.data_ptr()), 1 << 18, 4, 16,
                              ctypes.c_void_p(ws.data_ptr()), None)
    assert rc == _lib.ONMT_EUNSUPPORTED
    # and a batch below the limit is unaffected
    buf = _search(s, 2, 4)
    assert (buf["len"].cpu().numpy() >= 1).all()


def test_kernel_timing_follows_the_kind_mask():
    # timing is a side channel: the searches' outputs do not change, and only the selected kinds are timed
    s = Custom(TINY, [3, 10, 5, 1])
    _case("kernel_timing_mask")
    K, T = 2, 6
    ref = _search(s, K, T)
    kinds = ("generator", "lstm", "attention", "output", "beam_step")
    for sel in (("lstm",), ("generator", "beam_step"), kinds):
        s.tr.profile(1, kinds=sel)
        for k in kinds:
            s.tr.profile_read(reset=True, kind=k)
        buf = _search(s, K, T)
        got = {k: s.tr.profile_read(reset=True, kind=k) for k in kinds}
        s.tr.profile(False)
        for k in kinds:
            n, ms = got[k]
            if k in sel:
                assert n > 0 and ms > 0, (sel, k)
            else:
                assert n == 0 and ms == 0, (sel, k)
        for key in ("tok", "len", "raw", "norm"):
            assert torch.equal(buf[key], ref[key]), key
    # every decode step runs each decoder layer once (the tiny model has one): as many LSTM launches as
    # generator launches
    s.tr.profile(1, kinds=("generator", "lstm"))
    _search(s, K, T)
    n_gen = s.tr.profile_read(reset=True, kind="generator")[0]
    n_lstm = s.tr.profile_read(reset=True, kind="lstm")[0]
    s.tr.profile(False)
    assert n_lstm == n_gen * TINY.dec_layers
