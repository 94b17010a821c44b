"""GPU parity on model shapes the five workloads do not exercise (Section 2's encoder-decoder at other
sizes): hidden sizes that are not multiples of 32 (partial gate groups, padded K segments), vocabularies
that leave a ragged last generator tile, three stacked layers, bidirectional encoders with odd
per-direction widths, the concat attention type at such sizes, and a bf16 model whose hidden size is not
a multiple of 8 (its activations are split on load instead of read as pre-split planes). Each shape:
three decoder steps against the oracle (full log-distribution, attention, state) and a beam search whose
every sentence is checked by teacher-forced rescoring and the replay of its decisions. A bf16 model with
hidden 104 at 256 hypothesis rows runs the decoder layers' LDS-destination main loop (rows gathered by
beam parent, a segment width that is not a multiple of the 64-wide K stage).
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import Setup, TAU, ATTN_TOL, with_workload, check_search

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

TINY = W.get("tiny")
SHAPES = {
    "fp32_h100_v1003_3layers": dict(enc_layers=3, dec_layers=3, hidden=100, emb=36, src_vocab=700, tgt_vocab=1003),
    "fp32_bi_h72_v517": dict(enc_layers=2, dec_layers=2, bidirectional=True, hidden=72, emb=44, src_vocab=300,
                             tgt_vocab=517, beam=4),
    "fp32_concat_h100_v777": dict(hidden=100, emb=40, tgt_vocab=777, attn="concat"),
    "fp32_dot_bi_h64_v300": dict(bidirectional=True, hidden=64, emb=20, tgt_vocab=300, attn="dot"),
    "bf16_h104_v2049": dict(enc_layers=2, dec_layers=2, hidden=104, emb=48, tgt_vocab=2049, wdtype="bf16"),
    "bf16_h100_v1500_split_on_load": dict(hidden=100, emb=40, tgt_vocab=1500, wdtype="bf16"),
}


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


@pytest.fixture(scope="module", params=list(SHAPES))
def shape(request):
    w = with_workload(TINY, name=request.param, batch=5, **SHAPES[request.param])
    return Setup(w, peaked=True)


def test_decode_steps(shape):
    s = shape
    w = s.w
    B, S = s.src.shape
    K = w.beam
    N = B * K
    _case("decode_steps", shape=w.name)
    ws = s.tr.encode(s.src_d, s.lens_d)
    st = s.tr.decode_init(ws, B, S, K)
    enc = O.encode(s.model, s.src, s.lens)
    ost = O.init_state(s.model, enc, K)
    rows = np.repeat(np.arange(B), K)
    rng = np.random.default_rng(31)
    tok = np.full(N, W.BOS_ID, np.int32)
    parent = None
    for step in range(3):
        par_d = torch.from_numpy(parent).cuda() if parent is not None else None
        st, logp, _, _, attn = s.tr.decode_step(ws, B, S, K, st, torch.from_numpy(tok).cuda(), par_d, mode=0,
                                                want_attn=True)
        torch.cuda.synchronize()
        o_new, o_logp, o_attn = O.decode_step(s.model, enc, ost if parent is None else ost.take(parent), tok, rows)
        err = np.abs(logp.cpu().numpy() - o_logp).max()
        print(f"  step {step}: max |logp - oracle| = {err:.3g}", flush=True)
        assert err <= s.tau
        np.testing.assert_allclose(attn.cpu().numpy(), o_attn, atol=ATTN_TOL[w.wdtype], rtol=0)
        h, c, feed = s.tr.state_views(st, N)
        tol = 1e-5 if w.wdtype == "fp32" else 1e-2
        for l in range(w.dec_layers):
            np.testing.assert_allclose(h[l].cpu().numpy(), o_new.h[l], atol=tol, rtol=0)
        np.testing.assert_allclose(feed.cpu().numpy(), o_new.feed, atol=tol, rtol=0)
        parent = (rows * K + rng.integers(0, K, size=N)).astype(np.int32)
        tok = rng.integers(0, w.tgt_vocab, size=N).astype(np.int32)
        ost = o_new


def test_beam_search(shape):
    s = shape
    w = s.w
    B, S = s.src.shape
    _case("beam_search", shape=w.name)
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, 0.6, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    mism = check_search(s, buf, range(B), w.beam, w.max_len, 0.6)
    print(f"  free-run token mismatches (replay-verified): {mism}", flush=True)


def test_bf16_lds_path_256_rows():
    w = with_workload(TINY, name="bf16_h104_256rows", batch=64, beam=4, hidden=104, emb=48, tgt_vocab=1500,
                      wdtype="bf16")
    s = Setup(w, peaked=True)
    B, S = s.src.shape
    K = w.beam
    N = B * K
    assert N >= 256                                   # the decoder GEMMs use the 32-row bf16 tiles
    _case("bf16_lds_path", rows=N)
    ws = s.tr.encode(s.src_d, s.lens_d)
    st = s.tr.decode_init(ws, B, S, K)
    enc = O.encode(s.model, s.src, s.lens)
    ost = O.init_state(s.model, enc, K)
    rows = np.repeat(np.arange(B), K)
    rng = np.random.default_rng(5)
    tok = np.full(N, W.BOS_ID, np.int32)
    parent = None
    for step in range(3):
        par_d = torch.from_numpy(parent).cuda() if parent is not None else None
        st, logp, _, _, _ = s.tr.decode_step(ws, B, S, K, st, torch.from_numpy(tok).cuda(), par_d, mode=0)
        torch.cuda.synchronize()
        o_new, o_logp, _ = O.decode_step(s.model, enc, ost if parent is None else ost.take(parent), tok, rows)
        err = np.abs(logp.cpu().numpy() - o_logp).max()
        print(f"  step {step}: max |logp - oracle| = {err:.3g}", flush=True)
        assert err <= s.tau
        h, c, feed = s.tr.state_views(st, N)
        for l in range(w.dec_layers):
            np.testing.assert_allclose(h[l].cpu().numpy(), o_new.h[l], atol=1e-2, rtol=0)
        parent = (rows * K + rng.integers(0, K, size=N)).astype(np.int32)
        tok = rng.integers(0, w.tgt_vocab, size=N).astype(np.int32)
        ost = o_new

