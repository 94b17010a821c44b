"""GPU parity of the dot and concat attention types (Section 4.2 names general, dot product and
concatenation attention; reading R20: dot q.m_s, concat v_a.tanh(W_a [q; m_s]), no biases).

Per type: the encoder's keys (concat: memory columns of W_a times the memory; dot: the memory itself),
three decoder steps (log-probs, attention weights and state against the oracle), the beam search on the
peaked tiny workload (every sentence) and on the default workload (sampled sentences, teacher-forced
rescoring and the replay of the GPU's decisions), and bf16 teacher-forced scores on the bidirectional
4-layer workload.
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import Setup, ATTN_TOL, with_workload, check_search

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

TYPES = ["dot", "concat"]


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


_cache = {}


def _setup(name, attn, peaked=False):
    key = (name, attn, peaked)
    if key not in _cache:
        _cache.clear()                    # one model on the device at a time
        _cache[key] = Setup(with_workload(W.get(name), attn=attn), peaked=peaked)
    return _cache[key]


@pytest.mark.parametrize("attn", TYPES)
@pytest.mark.parametrize("name", ["tiny", "default"])
def test_encoder_keys(name, attn):
    s = _setup(name, attn)
    B, S = s.src.shape
    _case("keys", workload=name, attn=attn)
    ws = s.tr.encode(s.src_d, s.lens_d)
    torch.cuda.synchronize()
    mem, keys, _, _ = s.tr.enc_views(ws, B, S)
    enc = O.encode(s.model, s.src, s.lens)
    np.testing.assert_allclose(mem.cpu().numpy(), enc.memory, atol=1e-5, rtol=0)
    if attn == "dot":
        assert keys.data_ptr() == mem.data_ptr()
    else:
        ref = enc.memory @ s.model.w["W_a"][:, s.w.hidden:].T
        np.testing.assert_allclose(keys.cpu().numpy()[enc.mask], ref[enc.mask], atol=1e-5, rtol=0)


@pytest.mark.parametrize("attn", TYPES)
@pytest.mark.parametrize("name,peaked", [("tiny", True), ("default", False)])
def test_decode_steps(name, peaked, attn):
    s = _setup(name, attn, peaked)
    w = s.w
    B, S = s.src.shape
    K = w.beam
    N = B * K
    _case("decode_step", workload=name, peaked=peaked, attn=attn)
    ws = s.tr.encode(s.src_d, s.lens_d)
    st = s.tr.decode_init(ws, B, S, K)
    enc = O.encode(s.model, s.src, s.lens)
    ost = O.init_state(s.model, enc, K)
    rows = np.repeat(np.arange(B), K)
    rng = np.random.default_rng(17)
    tok = np.full(N, W.BOS_ID, np.int32)
    parent = None
    for step in range(3):
        par_d = torch.from_numpy(parent).cuda() if parent is not None else None
        st, logp, _, _, attn_w = s.tr.decode_step(ws, B, S, K, st, torch.from_numpy(tok).cuda(), par_d, mode=0,
                                                  want_attn=True)
        torch.cuda.synchronize()
        o_new, o_logp, o_attn = O.decode_step(s.model, enc, ost if parent is None else ost.take(parent), tok, rows)
        err = np.abs(logp.cpu().numpy() - o_logp).max()
        print(f"  step {step}: max |logp - oracle| = {err:.3g}", flush=True)
        assert err <= s.tau
        np.testing.assert_allclose(attn_w.cpu().numpy(), o_attn, atol=ATTN_TOL[w.wdtype], rtol=0)
        np.testing.assert_allclose(s.tr.state_views(st, N)[2].cpu().numpy(), o_new.feed, atol=1e-5, rtol=0)
        parent = (rows * K + rng.integers(0, K, size=N)).astype(np.int32)
        tok = rng.integers(0, w.tgt_vocab, size=N).astype(np.int32)
        ost = o_new


@pytest.mark.parametrize("attn", TYPES)
def test_beam_search_tiny_peaked(attn):
    s = _setup("tiny", attn, peaked=True)
    w = s.w
    B, S = s.src.shape
    _case("beam_search", workload="tiny_peaked", attn=attn)
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, 0.6, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    mism = check_search(s, buf, range(B), w.beam, w.max_len, 0.6)
    print(f"  free-run token mismatches (replay-verified): {mism}", flush=True)


@pytest.mark.parametrize("attn", TYPES)
def test_beam_search_default_sampled(attn):
    s = _setup("default", attn)
    w = s.w
    B, S = s.src.shape
    _case("beam_search", workload="default", attn=attn)
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, w.alpha, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    g_len = buf["len"].cpu().numpy()
    assert (g_len >= 1).all() and (g_len <= w.max_len).all()
    check_search(s, buf, [0, 63], w.beam, w.max_len, w.alpha)


@pytest.mark.parametrize("attn", TYPES)
def test_score_larger_bf16_sampled(attn):
    s = _setup("larger", attn)
    B = s.src.shape[0]
    rng = np.random.default_rng(505)
    T = 12
    tgt = rng.integers(0, s.w.tgt_vocab, size=(B, T)).astype(np.int32)
    tgt_len = rng.integers(1, T + 1, size=B).astype(np.int32)
    tgt_len[2] = T
    _case("score", workload="larger", attn=attn)
    logp, nll = s.tr.score(s.src_d, s.lens_d, torch.from_numpy(tgt).cuda(), torch.from_numpy(tgt_len).cuda())
    torch.cuda.synchronize()
    rows = np.array([2])
    o_logp, o_nll = O.score_batch(s.model, s.src[rows], s.lens[rows], tgt[rows], tgt_len[rows])
    np.testing.assert_allclose(logp.cpu().numpy()[rows], o_logp, atol=s.tau, rtol=0)
    assert np.all(np.abs(nll.cpu().numpy()[rows] - o_nll) <= s.tau * tgt_len[rows])
