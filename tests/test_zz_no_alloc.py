"""onmt_decode_step_noalloc, the decoder step for callers that cannot allocate: the same outputs as
onmt_decode_step, bit for bit, from the library's built-in scratch array instead of a caller's step
workspace, on two calls in a row (the second with a smaller batch, so the array holds the first call's
contents when the second starts), and a refusal for steps that need more scratch than the array holds.

Section 2: one evaluation of p(w_t | w_<t, x) for every hypothesis row; Section 4.1: the batched GPU
translator behind a C interface.
"""

import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from paper_1805_11462_amd import _lib
from paper_1805_11462_amd.translator import _ptr, _stream
from tests._gpu import translator_for

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _case(name, **kw):
    print(f"[case] {name} " + " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _noalloc_step(tr, ws, B, S, K, st, tok, par, mode):
    N = B * K
    V = tr.cfg.tgt_vocab
    out_state = tr.new_state(N)
    logp = torch.empty(N, V if mode == 0 else K, dtype=torch.float32, device="cuda")
    ids = torch.empty(N, K, dtype=torch.int32, device="cuda") if mode == 1 else None
    lse = torch.empty(N, dtype=torch.float32, device="cuda")
    attn = torch.empty(N, S, dtype=torch.float32, device="cuda")
    _lib.check(tr.lib.onmt_decode_step_noalloc(tr.handle, _ptr(ws), B, S, K, _ptr(st), _ptr(out_state), _ptr(tok),
                                               _ptr(par), mode, _ptr(logp), _ptr(ids), _ptr(lse), _ptr(attn),
                                               _stream()))
    return out_state, logp, ids, lse, attn


@pytest.mark.parametrize("name", ["default", "larger"])
def test_noalloc_step_matches_the_workspace_step(name):
    w = W.get(name)
    weights = W.make_weights(w)
    tr = translator_for(w, weights)
    src, lens = W.make_batch(w)
    K = w.beam
    rng = np.random.default_rng(11)
    # two calls in a row: the whole batch, then its first 8 sentences
    for B in (src.shape[0], 8):
        _case("noalloc_step", workload=name, B=B, K=K)
        S = src.shape[1]
        N = B * K
        src_d = torch.from_numpy(np.ascontiguousarray(src[:B])).cuda()
        lens_d = torch.from_numpy(np.ascontiguousarray(lens[:B])).cuda()
        ws = tr.encode(src_d, lens_d)
        st = tr.decode_init(ws, B, S, K)
        tok = torch.full((N,), W.BOS_ID, dtype=torch.int32, device="cuda")
        par = None
        for step in range(2):
            for mode in (0, 1):
                ref = tr.decode_step(ws, B, S, K, st, tok, par, mode=mode, want_attn=True)
                got = _noalloc_step(tr, ws, B, S, K, st, tok, par, mode)
                torch.cuda.synchronize()
                # the state buffers' h, c and feed (the alignment padding after them is never written)
                for a, b in zip(tr.state_views(ref[0], N), tr.state_views(got[0], N)):
                    assert torch.equal(a, b), (name, B, step, mode, "state")
                for i, (a, b) in enumerate(zip(ref[1:], got[1:])):
                    if a is None:
                        assert b is None
                        continue
                    assert torch.equal(a, b), (name, B, step, mode, i + 1)
            code = ctypes.c_int(99)
            _lib.check(tr.lib.onmt_device_status(tr.handle, ctypes.byref(code)))
            assert code.value == _lib.ONMT_OK
            st = ref[0]
            tok = torch.from_numpy(rng.integers(0, w.tgt_vocab, N).astype(np.int32)).cuda()
            par = torch.from_numpy((np.repeat(np.arange(B), K) * K + rng.integers(0, K, N)).astype(np.int32)).cuda()
    tr.close()


def test_noalloc_step_refuses_steps_beyond_its_scratch():
    w = W.get("default")
    tr = translator_for(w, W.make_weights(w))
    B, S, K = 512, w.s_max, w.beam             # 2560 rows of generator partials: ~52 MB of scratch
    assert tr.lib.onmt_step_ws_bytes(tr.handle, B, S, K) > _lib.NOALLOC_SCRATCH_BYTES
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    p = ctypes.c_void_p(dummy.data_ptr())
    rc = tr.lib.onmt_decode_step_noalloc(tr.handle, p, B, S, K, p, ctypes.c_void_p(dummy.data_ptr() + 32), p, None, 0,
                                         p, None, None, None, None)
    assert rc == _lib.ONMT_EUNSUPPORTED
    assert b"scratch" in tr.lib.onmt_last_error()
    tr.close()
