"""The C-ABI library loads, exports every declared symbol and validates configs (no GPU needed)."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_1805_11462_amd import _lib
from paper_1805_11462_amd.translator import make_config
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "onmt.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(onmt_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound():
    lib = _lib.load()
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, f"{n} has no binding"
    assert set(_lib.SIGNATURES) == set(names)


def cfg_of(w):
    return make_config(w.enc_layers, w.dec_layers, w.bidirectional, w.emb, w.hidden, w.src_vocab, w.tgt_vocab,
                       w.wdtype, attn=w.attn)


@pytest.mark.parametrize("name,attn", [(n, "general") for n in W.WORKLOADS]
                         + [(n, a) for n in ("tiny", "larger") for a in ("dot", "concat")])
def test_weight_order_matches_the_shared_generator(name, attn):
    w = W.Workload(**{**W.get(name).as_dict(), "attn": attn})
    lib = _lib.load()
    cfg = cfg_of(w)
    specs = W.weight_specs(w)
    assert lib.onmt_num_weights(ctypes.byref(cfg)) == len(specs)
    for i, (_, shape) in enumerate(specs):
        assert lib.onmt_weight_numel(ctypes.byref(cfg), i) == int(np.prod(shape))
    assert lib.onmt_model_bytes(ctypes.byref(cfg)) > 0


@pytest.mark.parametrize("field,value,code", [
    ("dec_layers", 3, _lib.ONMT_EINVAL),        # encoder/decoder depth mismatch
    ("enc_layers", 0, _lib.ONMT_EINVAL),
    ("wdtype", 2, _lib.ONMT_EINVAL),
    ("emb", 30, _lib.ONMT_EUNSUPPORTED),        # not a multiple of 4
    ("eos_id", 50000, _lib.ONMT_EINVAL),
    ("tgt_vocab", 3, _lib.ONMT_EINVAL),
    ("attn_type", 3, _lib.ONMT_EINVAL),
    ("attn_type", -1, _lib.ONMT_EINVAL),
])
def test_invalid_configs_are_rejected(field, value, code):
    lib = _lib.load()
    cfg = cfg_of(W.get("default"))
    setattr(cfg, field, value)
    assert lib.onmt_num_weights(ctypes.byref(cfg)) == code
    assert lib.onmt_model_bytes(ctypes.byref(cfg)) == 0
    assert len(lib.onmt_last_error()) > 0


def test_bf16_needs_emb_multiple_of_8():
    lib = _lib.load()
    cfg = cfg_of(W.get("larger"))
    cfg.emb = 1004
    assert lib.onmt_num_weights(ctypes.byref(cfg)) == _lib.ONMT_EUNSUPPORTED


def test_null_handles_are_rejected_without_a_device():
    lib = _lib.load()
    assert lib.onmt_encode_ws_bytes(None, 4, 10) == 0
    assert lib.onmt_model_destroy(None) == _lib.ONMT_EINVAL
    assert lib.onmt_encode(None, None, None, 1, 1, None, 0, None) == _lib.ONMT_EINVAL
    assert lib.onmt_beam_search(None, None, None, 1, 1, None, None, 0, None, None, None, None, None, None,
                                None, None) == _lib.ONMT_EINVAL
    n = ctypes.c_int()
    ms = ctypes.c_double()
    assert lib.onmt_profile_read(None, ctypes.byref(n), ctypes.byref(ms), 0) == _lib.ONMT_EINVAL
    assert lib.onmt_profile_enable(None, 1, _lib.KERNEL_ALL) == _lib.ONMT_EINVAL


def test_model_create_rejects_bad_arguments_before_touching_memory():
    lib = _lib.load()
    cfg = cfg_of(W.get("tiny"))
    out = ctypes.c_void_p()
    n = lib.onmt_num_weights(ctypes.byref(cfg))
    arr = (ctypes.c_void_p * n)()
    # wrong count, NULL arrays, NULL buffer, too-small buffer: all rejected during validation
    assert lib.onmt_model_create(ctypes.byref(cfg), arr, n - 1, None, 0, None, ctypes.byref(out)) == _lib.ONMT_EINVAL
    assert lib.onmt_model_create(ctypes.byref(cfg), arr, n, None, 0, None, ctypes.byref(out)) == _lib.ONMT_EINVAL
    keep = [np.zeros(lib.onmt_weight_numel(ctypes.byref(cfg), i), np.float32) for i in range(n)]
    for i, a in enumerate(keep):
        arr[i] = a.ctypes.data
    assert lib.onmt_model_create(ctypes.byref(cfg), arr, n, None, 0, None, ctypes.byref(out)) == _lib.ONMT_EINVAL
    assert lib.onmt_model_create(ctypes.byref(cfg), arr, n, ctypes.c_void_p(256), 16, None,
                                 ctypes.byref(out)) == _lib.ONMT_ESIZE
    assert lib.onmt_model_create(ctypes.byref(cfg), arr, n, ctypes.c_void_p(8), 1 << 40, None,
                                 ctypes.byref(out)) == _lib.ONMT_EINVAL      # misaligned


def test_library_resolves_every_kernel_it_launches():
    # a kernel template whose host-side launch stub was not emitted would leave an undefined onmt:: symbol
    # in the shared library (the linker accepts it; the first launch would fail)
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    path = _lib.load()._name
    out = subprocess.run([nm, "-C", "--undefined-only", path], capture_output=True, text=True, check=True).stdout
    missing = [l for l in out.splitlines() if "onmt::" in l]
    assert missing == []


@pytest.mark.parametrize("wdtype,field,ok,too_big", [
    # E_src [src_vocab, emb]: 2^20 x 500 fp32 = 2.0e9 bytes fits, 2^20 x 512 = 2^31 does not
    ("fp32", "src_vocab_emb", (1 << 20, 500), (1 << 20, 512)),
    # the same table in bf16: 2^20 x 1016 fits, 2^20 x 1024 does not
    ("bf16", "src_vocab_emb", (1 << 20, 1016), (1 << 20, 1024)),
    # W_s [tgt_vocab, pad(hidden)]: fp32 models keep it in fp32 (131072 x 3968 fits; hidden 4000 pads to
    # 4096 columns = 2^31 bytes) besides its bf16 term planes, one descriptor each (131072 x 8064 x 2 bytes
    # fits, hidden 8100 pads to 8192 columns = 2^31 bytes)
    ("fp32", "tgt_vocab_hidden", (131072, 3968), (131072, 4000)),
    ("bf16", "tgt_vocab_hidden", (131072, 8064), (131072, 8100)),
])
def test_operands_past_the_descriptor_limit_are_refused(wdtype, field, ok, too_big):
    # buffer descriptors address at most 2 GiB: a config whose embedding table or packed weight matrix
    # reaches that is refused up front (ONMT_EUNSUPPORTED), never silently read as zeros
    lib = _lib.load()
    for (a, b), want_ok in ((ok, True), (too_big, False)):
        w = W.get("tiny")
        kw = {"src_vocab": a, "emb": b} if field == "src_vocab_emb" else {"tgt_vocab": a, "hidden": b}
        w = W.Workload(**{**w.as_dict(), "wdtype": wdtype, **kw})
        cfg = cfg_of(w)
        n = lib.onmt_num_weights(ctypes.byref(cfg))
        if want_ok:
            assert n > 0, lib.onmt_last_error()
            assert lib.onmt_model_bytes(ctypes.byref(cfg)) > 0
        else:
            assert n == _lib.ONMT_EUNSUPPORTED
            assert lib.onmt_model_bytes(ctypes.byref(cfg)) == 0
            assert b"2 GiB" in lib.onmt_last_error()
