"""Device-memory plumbing around the C ABI: torch tensors hold the buffers, libonmt does the work.

Every call below only sizes buffers, allocates them as torch tensors on the current GPU, passes raw
pointers and the current HIP stream to the matching ``onmt_*`` function and returns the tensors.
"""

import ctypes

import numpy as np
import torch

from . import _lib
from ._lib import OnmtConfig, OnmtSearchParams, OnmtTrace, check


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _bytes(n, device):
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=device)


ATTN_TYPES = {"general": 0, "dot": 1, "concat": 2}


def make_config(enc_layers, dec_layers, bidirectional, emb, hidden, src_vocab, tgt_vocab, wdtype,
                pad_id=0, unk_id=1, bos_id=2, eos_id=3, attn="general"):
    return OnmtConfig(enc_layers, dec_layers, int(bool(bidirectional)), emb, hidden, src_vocab, tgt_vocab,
                      1 if wdtype in ("bf16", 1) else 0, pad_id, unk_id, bos_id, eos_id,
                      ATTN_TYPES[attn] if isinstance(attn, str) else int(attn))


class Translator:
    """A packed model on one GPU plus convenience wrappers of the ABI calls."""

    def __init__(self, cfg: OnmtConfig, weights, device="cuda"):
        lib = _lib.load()
        self.lib = lib
        self.cfg = cfg
        self.device = torch.device(device)
        n = lib.onmt_num_weights(ctypes.byref(cfg))
        if n < 0:
            check(n)
        if len(weights) != n:
            raise ValueError(f"expected {n} weight arrays, got {len(weights)}")
        host = []
        for i, w in enumerate(weights):
            a = np.ascontiguousarray(w, dtype=np.float32)
            want = lib.onmt_weight_numel(ctypes.byref(cfg), i)
            if a.size != want:
                raise ValueError(f"weight {i}: {a.size} elements, expected {want}")
            host.append(a)
        ptrs = (ctypes.c_void_p * n)(*[a.ctypes.data for a in host])
        nbytes = lib.onmt_model_bytes(ctypes.byref(cfg))
        self.wbuf = _bytes(nbytes, self.device)
        handle = ctypes.c_void_p()
        check(lib.onmt_model_create(ctypes.byref(cfg), ptrs, n, _ptr(self.wbuf), nbytes, _stream(),
                                    ctypes.byref(handle)))
        self.handle = handle

    def close(self):
        if self.handle:
            self.lib.onmt_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- encoder
    def encode(self, src, lens):
        B, S = src.shape
        n = self.lib.onmt_encode_ws_bytes(self.handle, B, S)
        ws = _bytes(n, self.device)
        check(self.lib.onmt_encode(self.handle, _ptr(src), _ptr(lens), B, S, _ptr(ws), n, _stream()))
        return ws

    def enc_views(self, ws, B, S):
        """(memory [B, S, Hm], keys [B, S, H], final_h [L, B, H], final_c [L, B, H]) inside an encoder
        workspace, following the library's documented carving order (256-byte aligned regions:
        lens, src, memory, keys, final_h, final_c; dot attention has no keys region, its keys are the
        memory)."""
        c = self.cfg
        Hm = c.hidden
        al = lambda x: (x + 255) // 256 * 256
        off = al(4 * B)
        off = al(off + 4 * B * S)
        mem = ws[off:off + 4 * B * S * Hm].view(torch.float32).view(B, S, Hm)
        off = al(off + 4 * B * S * Hm)
        if c.attn_type == ATTN_TYPES["dot"]:
            keys = mem
        else:
            keys = ws[off:off + 4 * B * S * c.hidden].view(torch.float32).view(B, S, c.hidden)
            off = al(off + 4 * B * S * c.hidden)
        L = c.dec_layers
        fh = ws[off:off + 4 * L * B * c.hidden].view(torch.float32).view(L, B, c.hidden)
        off = al(off + 4 * L * B * c.hidden)
        fc = ws[off:off + 4 * L * B * c.hidden].view(torch.float32).view(L, B, c.hidden)
        return mem, keys, fh, fc

    # ---------------------------------------------------------------- decoder
    def new_state(self, N):
        return _bytes(self.lib.onmt_state_bytes(self.handle, N), self.device)

    def state_views(self, st, N):
        """(h [L, N, H], c [L, N, H], feed [N, H]) of a decoder state buffer."""
        c = self.cfg
        L, H = c.dec_layers, c.hidden
        al = lambda x: (x + 255) // 256 * 256
        h = st[0:4 * L * N * H].view(torch.float32).view(L, N, H)
        o = al(4 * L * N * H)
        cc = st[o:o + 4 * L * N * H].view(torch.float32).view(L, N, H)
        o = al(o + 4 * L * N * H)
        feed = st[o:o + 4 * N * H].view(torch.float32).view(N, H)
        return h, cc, feed

    def decode_init(self, enc_ws, B, S, K):
        st = self.new_state(B * K)
        check(self.lib.onmt_decode_init(self.handle, _ptr(enc_ws), B, S, K, _ptr(st), _stream()))
        return st

    def decode_step(self, enc_ws, B, S, K, state_in, prev_tok, parent=None, mode=0, want_attn=False):
        N = B * K
        V = self.cfg.tgt_vocab
        out_state = self.new_state(N)
        if mode == 0:
            logp = torch.empty(N, V, dtype=torch.float32, device=self.device)
            ids = None
        else:
            logp = torch.empty(N, K, dtype=torch.float32, device=self.device)
            ids = torch.empty(N, K, dtype=torch.int32, device=self.device)
        lse = torch.empty(N, dtype=torch.float32, device=self.device)
        attn = torch.empty(N, S, dtype=torch.float32, device=self.device) if want_attn else None
        n = self.lib.onmt_step_ws_bytes(self.handle, B, S, K)
        ws = _bytes(n, self.device)
        check(self.lib.onmt_decode_step(self.handle, _ptr(enc_ws), B, S, K, _ptr(state_in), _ptr(out_state),
                                        _ptr(prev_tok), _ptr(parent), mode, _ptr(logp), _ptr(ids), _ptr(lse),
                                        _ptr(attn), _ptr(ws), n, _stream()))
        return out_state, logp, ids, lse, attn

    # ---------------------------------------------------------------- search
    def search_buffers(self, B, S, beam, max_len, alpha=0.0, check_every=0, trace=False, beta=0.0, max_unk=-1,
                       banned=(), align=False):
        """Allocate everything one onmt_beam_search call needs (reusable across calls)."""
        banned_arr = (ctypes.c_int32 * max(len(banned), 1))(*[int(x) for x in banned])
        p = OnmtSearchParams(beam, max_len, float(alpha), check_every, float(beta), int(max_unk),
                             ctypes.cast(banned_arr, ctypes.c_void_p) if len(banned) else None, len(banned))
        n = self.lib.onmt_search_ws_bytes(self.handle, B, S, ctypes.byref(p))
        d = self.device
        buf = {
            "params": p, "banned": banned_arr, "ws": _bytes(n, d), "ws_bytes": n,
            "tok": torch.empty(B, max_len, dtype=torch.int32, device=d),
            "len": torch.empty(B, dtype=torch.int32, device=d),
            "raw": torch.empty(B, dtype=torch.float64, device=d),
            "norm": torch.empty(B, dtype=torch.float64, device=d),
            "tok_logp": torch.empty(B, max_len, dtype=torch.float32, device=d),
            "align": torch.empty(B, max_len, dtype=torch.int32, device=d) if align else None,
            "trace": None,
        }
        if trace:
            buf["trace_slot"] = torch.empty(max_len, B, beam, dtype=torch.int32, device=d)
            buf["trace_tok"] = torch.empty(max_len, B, beam, dtype=torch.int32, device=d)
            buf["trace_cand"] = torch.empty(max_len, B, beam, dtype=torch.float64, device=d)
            buf["trace_steps"] = torch.empty(B, dtype=torch.int32, device=d)
            buf["trace"] = OnmtTrace(buf["trace_slot"].data_ptr(), buf["trace_tok"].data_ptr(),
                                     buf["trace_cand"].data_ptr(), buf["trace_steps"].data_ptr())
        return buf

    def beam_search(self, src, lens, buf):
        B, S = src.shape
        tr = ctypes.byref(buf["trace"]) if buf["trace"] is not None else None
        al = _ptr(buf["align"]) if buf.get("align") is not None else None
        check(self.lib.onmt_beam_search(self.handle, _ptr(src), _ptr(lens), B, S, ctypes.byref(buf["params"]),
                                        _ptr(buf["ws"]), buf["ws_bytes"], _ptr(buf["tok"]), _ptr(buf["len"]),
                                        _ptr(buf["raw"]), _ptr(buf["norm"]), _ptr(buf["tok_logp"]), al, tr,
                                        _stream()))
        return buf

    def replace_unk(self, src, buf):
        """Unknown-word replacement (Section 4.2 OOV handling) on the device for a search run with
        align=True: [B, max_len] int32, the source id at the aligned position of every UNK output token,
        -1 elsewhere (onmt_replace_unk)."""
        B, S = src.shape
        T = buf["tok"].shape[1]
        out = torch.empty(B, T, dtype=torch.int32, device=self.device)
        check(self.lib.onmt_replace_unk(self.handle, _ptr(src), B, S, _ptr(buf["tok"]), _ptr(buf["len"]),
                                        _ptr(buf["align"]), T, _ptr(out), _stream()))
        return out

    # ---------------------------------------------------------------- teacher-forced scoring
    def score_buffers(self, B, S, T):
        """Allocate what one onmt_score call needs (reusable across calls)."""
        n = self.lib.onmt_score_ws_bytes(self.handle, B, S, T)
        d = self.device
        return {"ws": _bytes(n, d), "ws_bytes": n, "T": T,
                "logp": torch.empty(B, T, dtype=torch.float32, device=d),
                "nll": torch.empty(B, dtype=torch.float64, device=d)}

    def score(self, src, lens, tgt, tgt_len, buf=None):
        """Per-token log-probs [B, T] and NLL [B] of the given targets (int32 device tensors)."""
        B, S = src.shape
        T = tgt.shape[1]
        if buf is None:
            buf = self.score_buffers(B, S, T)
        check(self.lib.onmt_score(self.handle, _ptr(src), _ptr(lens), B, S, _ptr(tgt), _ptr(tgt_len), T,
                                  _ptr(buf["ws"]), buf["ws_bytes"], _ptr(buf["logp"]), _ptr(buf["nll"]), _stream()))
        return buf["logp"], buf["nll"]

    # ---------------------------------------------------------------- timing
    def profile(self, every, kinds=("generator",)):
        """Time every ``every``-th launch of each listed kernel kind in later searches (0 or False: off)."""
        mask = 0
        for k in kinds:
            mask |= 1 << _lib.KERNEL_KINDS[k]
        check(self.lib.onmt_profile_enable(self.handle, int(every), mask))

    def profile_read(self, reset=True, kind="generator"):
        """(launches timed, their summed milliseconds) of one kernel kind since the last reset."""
        n = ctypes.c_int()
        ms = ctypes.c_double()
        check(self.lib.onmt_profile_read_kernel(self.handle, _lib.KERNEL_KINDS[kind], ctypes.byref(n),
                                                ctypes.byref(ms), 1 if reset else 0))
        return n.value, ms.value
