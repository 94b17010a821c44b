"""GPU parity of the coverage penalty in beam search (Section 4.2 attention coverage normalisation; R17).

A finished hypothesis's normalised score is raw / lp(n) + beta * sum_i log(min(c_i, 1)). Checks: the GPU
search equals the oracle search on the peaked tiny workload; the GPU's reported norm matches the oracle's
penalty recomputed along the GPU's own output (teacher-forced attention sums); the all-zero-weight case
follows the closed form of the oracle pins; beta = 0 reproduces the plain search.
"""

import math

import numpy as np
import pytest
import torch

import workloads as W
from oracle import onmt_oracle as O
from tests._gpu import Setup, with_workload

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

CP_TOL = 2e-4      # attention weights carry fp32 rounding; the penalty sums logs of their running sums


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _search(s, K, T, alpha, beta):
    B, S = s.src.shape
    buf = s.tr.search_buffers(B, S, K, T, alpha, beta=beta)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    return {k: buf[k].cpu().numpy() for k in ("tok", "len", "raw", "norm", "tok_logp")}


def _check_norms(s, out, sentences, alpha, beta):
    for b in sentences:
        n = int(out["len"][b])
        toks = list(out["tok"][b, :n])
        cov = O.coverage_forced(s.model, s.src[b], s.lens[b], toks)
        cp = O.coverage_penalty(cov, s.lens[b], beta)
        expect = out["raw"][b] / O.length_penalty(n, alpha) + cp
        assert abs(out["norm"][b] - expect) <= CP_TOL * (1 + abs(cp)) + s.tau * n, (b, out["norm"][b], expect)


@pytest.fixture(scope="module")
def tiny_peaked():
    return Setup(W.get("tiny"), peaked=True)


@pytest.fixture(scope="module")
def default():
    return Setup(W.get("default"))


@pytest.mark.parametrize("beta,alpha", [(0.4, 0.0), (1.0, 0.6), (3.0, 0.0)])
def test_coverage_tiny_peaked_matches_oracle(tiny_peaked, beta, alpha):
    s = tiny_peaked
    w = s.w
    _case("coverage", workload="tiny_peaked", beta=beta, alpha=alpha)
    out = _search(s, w.beam, w.max_len, alpha, beta)
    res = O.beam_search(s.model, s.src, s.lens, w.beam, w.max_len, alpha, beta=beta)
    for b in range(s.src.shape[0]):
        n = int(out["len"][b])
        assert list(out["tok"][b, :n]) == res.tokens[b], b
        assert abs(out["norm"][b] - res.norm[b]) <= CP_TOL * (1 + abs(res.norm[b]))
    _check_norms(s, out, range(s.src.shape[0]), alpha, beta)


def test_coverage_zero_beta_is_the_plain_search(tiny_peaked):
    s = tiny_peaked
    w = s.w
    a = _search(s, w.beam, w.max_len, 0.6, 0.0)
    B, S = s.src.shape
    buf = s.tr.search_buffers(B, S, w.beam, w.max_len, 0.6)
    s.tr.beam_search(s.src_d, s.lens_d, buf)
    torch.cuda.synchronize()
    for k in a:
        np.testing.assert_array_equal(a[k], buf[k].cpu().numpy())


@pytest.mark.parametrize("beta", [0.2, 1.0])
def test_coverage_zero_weights_closed_form(beta):
    V, T, K = 50, 6, 5
    w = with_workload(W.get("tiny"), tgt_vocab=V, src_vocab=V)
    s = Setup(w)
    zero = {k: np.zeros_like(v) for k, v in s.weights.items()}
    from tests._gpu import translator_for
    s.tr = translator_for(w, zero)
    _case("coverage_zero_weights", beta=beta)
    out = _search(s, K, T, 0.0, beta)
    for b in range(s.src.shape[0]):
        n_src = int(s.lens[b])
        best, best_t = -math.inf, 0
        for t in range(1, T + 1):
            norm = -t * math.log(V) + beta * n_src * math.log(min(t / n_src, 1.0))
            if norm > best:
                best, best_t = norm, t
            if t == T or best >= -t * math.log(V):
                break
        expect = [W.PAD_ID] * T if best_t == T else [W.PAD_ID] * (best_t - 1) + [W.EOS_ID]
        n = int(out["len"][b])
        assert list(out["tok"][b, :n]) == expect
        assert abs(out["norm"][b] - best) <= 1e-4


def test_coverage_default_sampled(default):
    s = default
    w = s.w
    _case("coverage", workload="default", beta=0.2)
    out = _search(s, w.beam, w.max_len, w.alpha, 0.2)
    assert (out["len"] >= 1).all()
    _check_norms(s, out, [0, 63], w.alpha, 0.2)
