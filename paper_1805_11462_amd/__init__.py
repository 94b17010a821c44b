"""MI355X (gfx950) beam-search translation with an attention-based LSTM encoder-decoder.

The compute lives in libonmt.so (HIP kernels behind the C ABI of include/onmt.h); this package holds
its sources (csrc/), the build script and a ctypes binding. Importing the binding requires the built
library; there is no CPU fallback.
"""

from . import _lib  # noqa: F401


def Translator(*args, **kwargs):
    from .translator import Translator as _T
    return _T(*args, **kwargs)


def make_config(*args, **kwargs):
    from .translator import make_config as _m
    return _m(*args, **kwargs)
