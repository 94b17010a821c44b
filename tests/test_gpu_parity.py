"""GPU parity: the HIP path through the C ABI against the CPU oracle, element by element.

Tolerances: per-step log-probs within 1e-4 absolute (fp32 workloads) or 2e-2 (bf16 weights, fp32
accumulation); attention weights within 1e-5 / 1e-2. Token choices must be identical wherever the
oracle's selection gaps exceed twice the tolerance; elsewhere the step-by-step replay of the GPU's
decisions must pass (any choice within the tolerance is correct).
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


@pytest.fixture(scope="module")
def tiny():
    return Setup(W.get("tiny"))


@pytest.fixture(scope="module")
def tiny_peaked():
    return Setup(W.get("tiny"), peaked=True)


@pytest.fixture(scope="module")
def default():
    return Setup(W.get("default"))


def _print_case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


# ------------------------------------------------------------------ encoder
@pytest.mark.parametrize("which", ["tiny", "tiny_peaked", "default"])
def test_encoder_matches_oracle(which, request):
    s = request.getfixturevalue(which)
    _print_case("encoder", workload=s.w.name)
    B, S = s.src.shape
    ws = s.tr.encode(s.src_d, s.lens_d)
    torch.cuda.synchronize()
    mem, keys, fh, fc = s.tr.enc_views(ws, B, S)
    enc = O.encode(s.model, s.src, s.lens)
    np.testing.assert_allclose(mem.cpu().numpy(), enc.memory, atol=1e-5, rtol=0)
    mask = enc.mask
    assert (mem.cpu().numpy()[~mask] == 0).all()
    ref_keys = enc.memory @ s.model.w["W_a"].T
    np.testing.assert_allclose(keys.cpu().numpy()[mask], ref_keys[mask], atol=1e-5, rtol=0)
    for l in range(s.w.dec_layers):
        np.testing.assert_allclose(fh[l].cpu().numpy(), enc.final_h[l], atol=1e-5, rtol=0)
        np.testing.assert_allclose(fc[l].cpu().numpy(), enc.final_c[l], atol=1e-5, rtol=0)


# ------------------------------------------------------------------ decoder step
def _oracle_state(s, st_views, N):
    h, c, feed = st_views
    return O.State([h[l].cpu().numpy().astype(np.float64) for l in range(s.w.dec_layers)],
                   [c[l].cpu().numpy().astype(np.float64) for l in range(s.w.dec_layers)],
                   feed.cpu().numpy().astype(np.float64))


STATE_TOL = {"fp32": 1e-5, "bf16": 1e-3}     # decoder h, c and feed after a step


@pytest.mark.parametrize("which", ["tiny", "tiny_peaked", "default", "larger", "greedy", "long_src"])
def test_decode_steps_full_and_topk(which, request):
    s = request.getfixturevalue(which)
    w = s.w
    B, S = s.src.shape
    K = w.beam
    N = B * K
    _print_case("decode_step", workload=w.name, N=N)
    tr = s.tr
    ws = tr.encode(s.src_d, s.lens_d)
    st = tr.decode_init(ws, B, S, K)
    enc = O.encode(s.model, s.src, s.lens)
    ost = O.init_state(s.model, enc, K)
    rows = np.repeat(np.arange(B), K)
    rng = np.random.default_rng(7)
    tok = np.full(N, W.BOS_ID, np.int32)
    parent = None
    for step in range(3):
        tok_d = torch.from_numpy(tok).cuda()
        par_d = torch.from_numpy(parent).cuda() if parent is not None else None
        st_full, logp, _, lse, attn = tr.decode_step(ws, B, S, K, st, tok_d, par_d, mode=0, want_attn=True)
        st_topk, tv, ti, lse2, _ = tr.decode_step(ws, B, S, K, st, tok_d, par_d, mode=1)
        torch.cuda.synchronize()
        o_in = ost if parent is None else ost.take(parent)
        o_new, o_logp, o_attn = O.decode_step(s.model, enc, o_in, tok, rows)
        g_logp = logp.cpu().numpy()
        err = np.abs(g_logp - o_logp).max()
        a_err = np.abs(attn.cpu().numpy() - o_attn).max()
        print(f"  step {step}: max |logp - oracle| = {err:.3g}, max |attention - oracle| = {a_err:.3g}", flush=True)
        assert err <= s.tau
        np.testing.assert_allclose(attn.cpu().numpy(), o_attn, atol=ATTN_TOL[w.wdtype], rtol=0)
        assert (attn.cpu().numpy()[~enc.mask[rows]] == 0).all()     # exactly zero at pads
        # top-K mode: values within tau, ids exact where the oracle's sorted gaps exceed 2 tau
        o_sorted = np.argsort(-o_logp, axis=1, kind="stable")[:, :K + 1]
        g_ids = ti.cpu().numpy()
        g_val = tv.cpu().numpy()
        for r in range(N):
            np.testing.assert_allclose(g_val[r], o_logp[r, g_ids[r]], atol=s.tau, rtol=0)
            vals = o_logp[r, o_sorted[r]]
            for j in range(K):
                gap_ok = (j == 0 or vals[j - 1] - vals[j] > 2 * s.tau) and vals[j] - vals[j + 1] > 2 * s.tau
                if gap_ok:
                    assert g_ids[r, j] == o_sorted[r, j], (r, j)
        # full and top-K runs wrote the same state
        for a, b in zip(tr.state_views(st_full, N), tr.state_views(st_topk, N)):
            assert torch.equal(a, b)
        np.testing.assert_allclose(lse.cpu().numpy(), lse2.cpu().numpy(), atol=0, rtol=0)
        h, c, feed = tr.state_views(st_full, N)
        st_err = max([np.abs(h[l].cpu().numpy() - o_new.h[l]).max() for l in range(w.dec_layers)] +
                     [np.abs(c[l].cpu().numpy() - o_new.c[l]).max() for l in range(w.dec_layers)] +
                     [np.abs(feed.cpu().numpy() - o_new.feed).max()])
        print(f"  step {step}: max |state - oracle| = {st_err:.3g}", flush=True)
        stol = STATE_TOL[w.wdtype]
        for l in range(w.dec_layers):
            np.testing.assert_allclose(h[l].cpu().numpy(), o_new.h[l], atol=stol, rtol=0)
            np.testing.assert_allclose(c[l].cpu().numpy(), o_new.c[l], atol=stol, rtol=0)
        np.testing.assert_allclose(feed.cpu().numpy(), o_new.feed, atol=stol, rtol=0)
        # next step: random in-sentence parents and random tokens
        parent = (np.repeat(np.arange(B), K) * K + rng.integers(0, K, size=N)).astype(np.int32)
        tok = rng.integers(0, w.tgt_vocab, size=N).astype(np.int32)
        st = st_full
        ost = o_new


# ------------------------------------------------------------------ beam search
@pytest.mark.parametrize("which,alpha", [("tiny", 0.0), ("tiny", 0.6), ("tiny_peaked", 0.0), ("tiny_peaked", 0.6)])
def test_beam_search_tiny(which, alpha, request):
    s = request.getfixturevalue(which)
    w = s.w
    B, S = s.src.shape
    _print_case("beam_search", workload=w.name, alpha=alpha)
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, alpha, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    mism = check_search(s, buf, range(B), w.beam, w.max_len, alpha)
    print(f"  free-run token mismatches (replay-verified): {mism}", flush=True)


@pytest.mark.parametrize("K", [1, 3, 8, 16])
def test_beam_widths_tiny_peaked(tiny_peaked, K):
    s = tiny_peaked
    B, S = s.src.shape
    _print_case("beam_width", K=K)
    buf = s.tr.search_buffers(B, S, K, 9, 0.6, trace=True)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    check_search(s, buf, range(B), K, 9, 0.6)


def test_search_is_deterministic(tiny_peaked):
    s = tiny_peaked
    B, S = s.src.shape
    outs = []
    for _ in range(2):
        buf = s.tr.search_buffers(B, S, 4, 10, 0.6, trace=False)
        s.tr.beam_search(s.src_d, s.lens_d, buf)
        torch.cuda.synchronize()
        outs.append({k: buf[k].cpu().numpy() for k in ("tok", "len", "raw", "norm", "tok_logp")})
    for k in outs[0]:
        np.testing.assert_array_equal(outs[0][k], outs[1][k])


def test_all_zero_weights_tie_rules():
    # every candidate ties: the tie-break to the smaller flat index and the stop rule on equality
    w = with_workload(W.get("tiny"), tgt_vocab=50, src_vocab=50)
    s = Setup(w)
    s.weights = {k: np.zeros_like(v) for k, v in s.weights.items()}
    from tests._gpu import translator_for
    tr = translator_for(w, s.weights)
    B, S = s.src.shape
    for K, want in ((3, [W.PAD_ID] * 6), (4, [W.EOS_ID])):
        buf = tr.search_buffers(B, S, K, 6, 0.0)
        tr.beam_search(s.src_d, s.lens_d, buf)
        torch.cuda.synchronize()
        for b in range(B):
            n = int(buf["len"][b])
            assert list(buf["tok"][b, :n].cpu().numpy()) == want
            assert abs(buf["raw"][b].item() + len(want) * np.log(50)) < 1e-5


# ------------------------------------------------------------------ the other workloads (bf16 workloads at
# the bf16 tolerance); their whole searches are in test_gpu_search_all.py
@pytest.fixture(scope="module")
def larger():
    return Setup(W.get("larger"))


@pytest.fixture(scope="module")
def greedy():
    return Setup(W.get("greedy"))


@pytest.fixture(scope="module")
def long_src():
    return Setup(W.get("long"))


@pytest.mark.parametrize("which", ["larger", "greedy", "long_src"])
def test_encoder_other_workloads(which, request):
    s = request.getfixturevalue(which)
    _print_case("encoder", workload=s.w.name)
    B, S = s.src.shape
    ws = s.tr.encode(s.src_d, s.lens_d)
    torch.cuda.synchronize()
    mem, keys, fh, fc = s.tr.enc_views(ws, B, S)
    enc = O.encode(s.model, s.src, s.lens)
    tol = 1e-4 if s.w.wdtype == "fp32" else 2e-2
    err = np.abs(mem.cpu().numpy() - enc.memory).max()
    print(f"  max |memory - oracle| = {err:.3g} over all {B} sentences", flush=True)
    np.testing.assert_allclose(mem.cpu().numpy(), enc.memory, atol=tol, rtol=0)
    assert (mem.cpu().numpy()[~enc.mask] == 0).all()
    if s.w.attn == "general":
        np.testing.assert_allclose(keys.cpu().numpy()[enc.mask], (enc.memory @ s.model.w["W_a"].T)[enc.mask],
                                   atol=tol, rtol=0)
    for l in range(s.w.dec_layers):
        np.testing.assert_allclose(fh[l].cpu().numpy(), enc.final_h[l], atol=tol, rtol=0)
        np.testing.assert_allclose(fc[l].cpu().numpy(), enc.final_c[l], atol=tol, rtol=0)


# ------------------------------------------------------------------ generator precision (fp32 models)
def _bf16_terms(x, n):
    """x (float32 array) as n bf16 terms, RNE of the value and then of each remainder, as float64."""
    out, r = [], x.astype(np.float32)
    for _ in range(n):
        u = r.view(np.uint32).astype(np.uint64)
        t = (((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)).view(np.float32)
        out.append(t.astype(np.float64))
        r = (r - t).astype(np.float32)
    return out


@pytest.fixture(scope="module")
def default_peaked():
    return Setup(W.get("default"), peaked=True)


def test_generator_products_keep_fp32_accuracy(default_peaked):
    # The fp32 generator multiplies each fp32 weight and activation as three bf16 terms and keeps the six
    # term products down to 2^-16 of the leading one (Section 2 generator; fp32 workloads). On the GPU's
    # own attentional vector, its logits must match the fp64 generator's to fp32 rounding. Compared as
    # differences within a row (log-prob of every word minus that of word 0, so the row's log-sum-exp
    # cancels), with W_s scaled by 10 so that logits reach tens: an fp32 product errs by ~3e-6 there, the
    # cheaper three-product form (hi.hi + hi.lo + lo.hi) by ~2.4e-5, and the bound sits between them.
    s = default_peaked
    w = s.w
    B, S = s.src.shape
    K = w.beam
    N = B * K
    _print_case("generator_precision", workload=w.name, peaked=True, N=N)
    tr = s.tr
    ws = tr.encode(s.src_d, s.lens_d)
    st = tr.decode_init(ws, B, S, K)
    tok = torch.full((N,), W.BOS_ID, dtype=torch.int32, device="cuda")
    st_out, logp, _, _, _ = tr.decode_step(ws, B, S, K, st, tok, None, mode=0)
    torch.cuda.synchronize()
    feed = tr.state_views(st_out, N)[2].cpu().numpy()
    rows = slice(0, 64)                                  # 64 of the 320 rows: the fp64 reference over 50000 columns
    ref = O.generator(s.model, feed[rows].astype(np.float64))

    def dif(x):
        return x - x[:, :1]

    err = np.abs(dif(logp.cpu().numpy()[rows].astype(np.float64)) - dif(ref)).max()
    # the three-product form of the same operands, in fp64 otherwise
    a1, a2, _ = _bf16_terms(feed[rows], 3)
    w1, w2, _ = _bf16_terms(s.model.w["W_s"].astype(np.float32), 3)
    z3 = a1 @ w1.T + a1 @ w2.T + a2 @ w1.T + s.model.w["b_s"]
    err3 = np.abs(dif(z3) - dif(ref)).max()
    print(f"  max |logit difference - fp64| = {err:.3g}; three-product form: {err3:.3g}", flush=True)
    assert err <= 8e-6
    assert err3 > 8e-6
