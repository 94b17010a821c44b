"""GPU parity of teacher-forced scoring (onmt_score) against the oracle's score_batch.

Per-token log-probs within 1e-4 (fp32) / 2e-2 (bf16) absolute; the NLL of a sentence within its length
times that. The scores of the beam search's own outputs must reproduce the search's per-token log-probs.
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import Setup, TAU

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _targets(B, T, V, seed):
    rng = np.random.default_rng(seed)
    tgt = rng.integers(0, V, size=(B, T)).astype(np.int32)
    tgt_len = rng.integers(1, T + 1, size=B).astype(np.int32)
    tgt_len[0] = T
    if B > 1:
        tgt_len[1] = 1
    return tgt, tgt_len


def _gpu_score(s, tgt, tgt_len):
    logp, nll = s.tr.score(s.src_d, s.lens_d, torch.from_numpy(tgt).cuda(), torch.from_numpy(tgt_len).cuda())
    torch.cuda.synchronize()
    return logp.cpu().numpy(), nll.cpu().numpy()


def _compare(s, tgt, tgt_len, g_logp, g_nll, rows):
    o_logp, o_nll = O.score_batch(s.model, s.src[rows], s.lens[rows], tgt[rows], tgt_len[rows])
    np.testing.assert_allclose(g_logp[rows], o_logp, atol=s.tau, rtol=0)
    assert np.all(np.abs(g_nll[rows] - o_nll) <= s.tau * tgt_len[rows]), (g_nll[rows], o_nll)


@pytest.fixture(scope="module")
def tiny_peaked():
    return Setup(W.get("tiny"), peaked=True)


@pytest.fixture(scope="module")
def default():
    return Setup(W.get("default"))


@pytest.fixture(scope="module")
def larger():
    return Setup(W.get("larger"))


def test_score_tiny_peaked_all_rows(tiny_peaked):
    s = tiny_peaked
    B = s.src.shape[0]
    tgt, tgt_len = _targets(B, 12, s.w.tgt_vocab, seed=101)
    _case("score", workload="tiny_peaked", B=B, T=12)
    g_logp, g_nll = _gpu_score(s, tgt, tgt_len)
    for b in range(B):
        assert np.all(g_logp[b, tgt_len[b]:] == 0.0)
    _compare(s, tgt, tgt_len, g_logp, g_nll, np.arange(B))


def test_score_default_sampled(default):
    s = default
    B = s.src.shape[0]
    tgt, tgt_len = _targets(B, 30, s.w.tgt_vocab, seed=202)
    _case("score", workload="default", B=B, T=30)
    g_logp, g_nll = _gpu_score(s, tgt, tgt_len)
    _compare(s, tgt, tgt_len, g_logp, g_nll, np.array([0, 1, 40]))


def test_score_larger_bf16_sampled(larger):
    s = larger
    B = s.src.shape[0]
    tgt, tgt_len = _targets(B, 16, s.w.tgt_vocab, seed=303)
    _case("score", workload="larger", B=B, T=16)
    g_logp, g_nll = _gpu_score(s, tgt, tgt_len)
    _compare(s, tgt, tgt_len, g_logp, g_nll, np.array([2]))


@pytest.mark.parametrize("which", ["tiny_peaked", "default"])
def test_score_of_beam_output_reproduces_search(which, request):
    s = request.getfixturevalue(which)
    w = s.w
    B, S = s.src.shape
    _case("score_beam_output", workload=which, B=B)
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, w.alpha)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    tok = buf["tok"].cpu().numpy()
    n = buf["len"].cpu().numpy()
    tok_logp = buf["tok_logp"].cpu().numpy()
    raw = buf["raw"].cpu().numpy()
    g_logp, g_nll = _gpu_score(s, tok, n)
    for b in range(B):
        np.testing.assert_allclose(g_logp[b, :n[b]], tok_logp[b, :n[b]], atol=s.tau, rtol=0)
        assert abs(-g_nll[b] - raw[b]) <= s.tau * n[b]


def test_score_rejects_bad_targets(tiny_peaked):
    from paper_1805_11462_amd._lib import OnmtError
    s = tiny_peaked
    B = s.src.shape[0]
    tgt, tgt_len = _targets(B, 5, s.w.tgt_vocab, seed=404)
    bad_len = tgt_len.copy()
    bad_len[0] = 0
    with pytest.raises(OnmtError):
        _gpu_score(s, tgt, bad_len)
    bad_tok = tgt.copy()
    bad_tok[1, 0] = s.w.tgt_vocab
    with pytest.raises(OnmtError):
        _gpu_score(s, bad_tok, tgt_len)
    # a token past a sentence's length is never read, so it may be anything
    ok_tok = tgt.copy()
    ok_tok[1, 3] = -7
    g_logp, _ = _gpu_score(s, ok_tok, tgt_len)
    assert np.isfinite(g_logp).all()
