"""Input validation on the device (ONMT_VALIDATE_DEVICE): the same results as host validation without a
stream sync per call, and bad inputs reported through onmt_device_status instead of refused up front.

Section 2 (the conditional model p(w_t | w_<t, x) evaluated step by step) and Section 4.1 (the batched GPU
translator behind a C interface): the decoder-step and encoder calls are meant to be chained on a stream
by a caller's own loop, so checking their device-resident inputs must not make the host wait.
"""

import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from paper_1805_11462_amd import _lib
from tests._gpu import Setup

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _status(tr):
    code = ctypes.c_int(99)
    _lib.check(tr.lib.onmt_device_status(tr.handle, ctypes.byref(code)))
    return code.value, tr.lib.onmt_last_error().decode()


def _steps(s, K, toks, parents):
    """Encoder + two decoder steps (full mode, with attention); returns every output on the host."""
    B, S = s.src.shape
    ws = s.tr.encode(s.src_d, s.lens_d)
    st = s.tr.decode_init(ws, B, S, K)
    # the encoder's outputs (its scratch regions differ: with device validation it steps over all S_max
    # positions, so its ping-pong state buffers end on a different side)
    out = [v.clone() for v in s.tr.enc_views(ws, B, S)]
    for tok, par in zip(toks, parents):
        st, logp, _, lse, attn = s.tr.decode_step(ws, B, S, K, st, tok, par, mode=0, want_attn=True)
        out += [st.clone(), logp.clone(), lse.clone(), attn.clone()]
    torch.cuda.synchronize()
    return [o.cpu() for o in out]


@pytest.fixture(scope="module")
def tiny_peaked():
    return Setup(W.get("tiny"), peaked=True)


def _inputs(s, K, seed=5):
    B = s.src.shape[0]
    N = B * K
    rng = np.random.default_rng(seed)
    toks = [torch.full((N,), W.BOS_ID, dtype=torch.int32, device="cuda"),
            torch.from_numpy(rng.integers(0, s.w.tgt_vocab, N).astype(np.int32)).cuda()]
    parents = [None, torch.from_numpy((np.repeat(np.arange(B), K) * K + rng.integers(0, K, N)).astype(np.int32)).cuda()]
    return toks, parents


def test_device_validation_gives_the_host_validated_results(tiny_peaked):
    s = tiny_peaked
    K = 3
    _case("device_validation_equal", workload="tiny_peaked", K=K)
    toks, parents = _inputs(s, K)
    host = _steps(s, K, toks, parents)
    _lib.check(s.tr.lib.onmt_set_validation(s.tr.handle, _lib.ONMT_VALIDATE_DEVICE))
    try:
        dev = _steps(s, K, toks, parents)
        assert _status(s.tr)[0] == _lib.ONMT_OK
        for a, b in zip(host, dev):
            assert torch.equal(a, b)
        # whole searches
        B, S = s.src.shape
        outs = []
        for mode in (_lib.ONMT_VALIDATE_HOST, _lib.ONMT_VALIDATE_DEVICE):
            _lib.check(s.tr.lib.onmt_set_validation(s.tr.handle, mode))
            buf = s.tr.search_buffers(B, S, 4, 10, 0.6)
            s.tr.beam_search(s.src_d, s.lens_d, buf)
            torch.cuda.synchronize()
            outs.append({k: buf[k].cpu() for k in ("tok", "len", "raw", "norm", "tok_logp")})
        for k in outs[0]:
            assert torch.equal(outs[0][k], outs[1][k]), k
        assert _status(s.tr)[0] == _lib.ONMT_OK
    finally:
        s.tr.lib.onmt_set_validation(s.tr.handle, _lib.ONMT_VALIDATE_HOST)


@pytest.mark.parametrize("what", ["len_zero", "len_past_s", "src_id", "prev_tok", "parent"])
def test_device_validation_reports_bad_inputs(tiny_peaked, what):
    s = tiny_peaked
    B, S = s.src.shape
    K = 2
    N = B * K
    _case("device_validation_bad", what=what)
    src, lens = s.src.copy(), s.lens.copy()
    if what == "len_zero":
        lens[1] = 0
    elif what == "len_past_s":
        lens[2] = S + 3
    elif what == "src_id":
        src[0, 0] = s.w.src_vocab + 5
    tok = torch.full((N,), W.BOS_ID, dtype=torch.int32, device="cuda")
    par = torch.arange(N, dtype=torch.int32, device="cuda")
    if what == "prev_tok":
        tok[3] = s.w.tgt_vocab
    elif what == "parent":
        par[1] = N + 7
    src_d = torch.from_numpy(src).cuda()
    lens_d = torch.from_numpy(lens).cuda()
    tr = s.tr
    _lib.check(tr.lib.onmt_set_validation(tr.handle, _lib.ONMT_VALIDATE_DEVICE))
    try:
        assert _status(tr)[0] == _lib.ONMT_OK          # nothing recorded yet
        ws = tr.encode(src_d, lens_d)                    # returns without waiting, and without an error
        st = tr.decode_init(ws, B, S, K)
        st2, logp, _, _, attn = tr.decode_step(ws, B, S, K, st, tok, par, mode=0, want_attn=True)
        torch.cuda.synchronize()
        code, msg = _status(tr)
        assert code == _lib.ONMT_EINVAL, what
        assert "device validation" in msg
        assert _status(tr)[0] == _lib.ONMT_OK          # the record was cleared
        # the bad value was replaced by a safe one: every output is finite and normalised
        lp = logp.cpu().numpy()
        assert np.isfinite(lp).all()
        assert np.abs(np.log(np.exp(lp.astype(np.float64)).sum(1))).max() < 1e-4
        a = attn.cpu().numpy()
        assert np.abs(a.sum(1) - 1).max() < 1e-5
    finally:
        tr.lib.onmt_set_validation(tr.handle, _lib.ONMT_VALIDATE_HOST)
    # host validation refuses the same inputs before launching anything
    if what in ("len_zero", "len_past_s", "src_id"):
        with pytest.raises(_lib.OnmtError):
            tr.encode(src_d, lens_d)
