"""ctypes binding of libonmt.so (argument marshalling only; every step runs in the HIP kernels).

The function names, argument order and structs mirror ``include/onmt.h``. Loading fails loudly if the
library has not been built (``python -m paper_1805_11462_amd.build``); there is no fallback path.
"""

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_int, c_int64, c_size_t, c_uint, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libonmt.so")

ONMT_OK, ONMT_EINVAL, ONMT_ESIZE, ONMT_EDEVICE, ONMT_EUNSUPPORTED = 0, -1, -2, -3, -4
ONMT_VALIDATE_HOST, ONMT_VALIDATE_DEVICE = 0, 1
KERNEL_KINDS = {"generator": 0, "lstm": 1, "attention": 2, "output": 3, "beam_step": 4}
KERNEL_ALL = (1 << len(KERNEL_KINDS)) - 1
NOALLOC_SCRATCH_BYTES = 16 << 20
ERROR_NAMES = {ONMT_EINVAL: "EINVAL", ONMT_ESIZE: "ESIZE", ONMT_EDEVICE: "EDEVICE", ONMT_EUNSUPPORTED: "EUNSUPPORTED"}


class OnmtConfig(ctypes.Structure):
    _fields_ = [(n, c_int) for n in ("enc_layers", "dec_layers", "bidirectional", "emb", "hidden", "src_vocab",
                                     "tgt_vocab", "wdtype", "pad_id", "unk_id", "bos_id", "eos_id",
                                     "attn_type")]


class OnmtSearchParams(ctypes.Structure):
    _fields_ = [("beam", c_int), ("max_len", c_int), ("alpha", c_double), ("check_every", c_int),
                ("beta", c_double), ("max_unk", c_int), ("banned", c_void_p), ("n_banned", c_int)]


class OnmtTrace(ctypes.Structure):
    _fields_ = [("slot", c_void_p), ("tok", c_void_p), ("cand", c_void_p), ("steps", c_void_p)]


# name -> (restype, argtypes), the full exported surface of include/onmt.h
SIGNATURES = {
    "onmt_last_error": (c_char_p, []),
    "onmt_num_weights": (c_int, [POINTER(OnmtConfig)]),
    "onmt_weight_numel": (c_int64, [POINTER(OnmtConfig), c_int]),
    "onmt_model_bytes": (c_size_t, [POINTER(OnmtConfig)]),
    "onmt_model_create": (c_int, [POINTER(OnmtConfig), POINTER(c_void_p), c_int, c_void_p, c_size_t, c_void_p,
                                  POINTER(c_void_p)]),
    "onmt_model_destroy": (c_int, [c_void_p]),
    "onmt_encode_ws_bytes": (c_size_t, [c_void_p, c_int, c_int]),
    "onmt_encode": (c_int, [c_void_p, c_void_p, c_void_p, c_int, c_int, c_void_p, c_size_t, c_void_p]),
    "onmt_state_bytes": (c_size_t, [c_void_p, c_int]),
    "onmt_step_ws_bytes": (c_size_t, [c_void_p, c_int, c_int, c_int]),
    "onmt_decode_init": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_void_p, c_void_p]),
    "onmt_decode_step": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "onmt_search_ws_bytes": (c_size_t, [c_void_p, c_int, c_int, POINTER(OnmtSearchParams)]),
    "onmt_beam_search": (c_int, [c_void_p, c_void_p, c_void_p, c_int, c_int, POINTER(OnmtSearchParams), c_void_p,
                                 c_size_t, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 POINTER(OnmtTrace), c_void_p]),
    "onmt_replace_unk": (c_int, [c_void_p, c_void_p, c_int, c_int, c_void_p, c_void_p, c_void_p, c_int, c_void_p,
                                 c_void_p]),
    "onmt_score_ws_bytes": (c_size_t, [c_void_p, c_int, c_int, c_int]),
    "onmt_score": (c_int, [c_void_p, c_void_p, c_void_p, c_int, c_int, c_void_p, c_void_p, c_int, c_void_p, c_size_t,
                           c_void_p, c_void_p, c_void_p]),
    "onmt_set_validation": (c_int, [c_void_p, c_int]),
    "onmt_device_status": (c_int, [c_void_p, POINTER(c_int)]),
    "onmt_decode_step_noalloc": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p,
                                         c_void_p, c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "onmt_profile_enable": (c_int, [c_void_p, c_int, c_uint]),
    "onmt_profile_read": (c_int, [c_void_p, POINTER(c_int), POINTER(c_double), c_int]),
    "onmt_profile_read_kernel": (c_int, [c_void_p, c_int, POINTER(c_int), POINTER(c_double), c_int]),
}

_lib = None


class OnmtError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


def load():
    """Load libonmt.so once; raises if it is missing (the product has no CPU path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_1805_11462_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def check(rc):
    if rc != ONMT_OK:
        raise OnmtError(rc, load().onmt_last_error().decode())
    return rc


def __getattr__(name):
    if name in SIGNATURES:
        return getattr(load(), name)
    raise AttributeError(name)
