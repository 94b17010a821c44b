"""Seeded synthetic inputs shared by the oracle and the GPU path.

This module draws random numbers and lays them out; it contains none of the
method's arithmetic. It is the only code that both sides use.

Recipe (stands in for the paper's WMT15/WMT17 EN-DE BPE workloads, which are
not available here):

* weights: one ``numpy.random.Generator(PCG64(seed))`` stream, default seed 17,
  every tensor drawn as ``uniform(-0.1, 0.1)`` in the fixed order of
  :func:`weight_specs`, then cast to float32. bf16 workloads then round every
  weight to bfloat16 with round-to-nearest-even and keep it as float32, so both
  sides consume exactly the same values.
* source lengths: ``integers(len_lo, len_hi + 1, batch)`` from the data stream
  (seed ``1000 + workload index`` unless given), then tokens for all
  ``batch x s_max`` positions from a bounded Zipf law over ranks ``1..V-4``
  with ``P(r) ~ r^-s`` (inverse CDF), id ``3 + r``; positions at or beyond the
  length are set to the pad id 0.
"""

import numpy as np

from .configs import Workload, PAD_ID

WEIGHT_SEED = 17


def weight_specs(w: Workload):
    """(name, shape) of every weight tensor, in draw order and C-ABI order.

    Layouts are row-major. LSTM layer: ``W [4*Hl, in + Hl]`` with gate blocks
    (i, f, g, o) along rows and columns ``[input | recurrent]``; ``b [4*Hl]``.
    Attention: "general" ``W_a [H, Hm]``; "dot" no score weights; "concat" ``W_a [H, H + Hm]`` with
    columns ``[query | memory]`` and ``v_a [H]``. Then ``W_c [H, Hm + H]`` with columns ``[ctx | h]``.
    Generator: ``W_s [V, H]``, ``b_s [V]``.
    """
    H, Hd, E = w.hidden, w.enc_hidden, w.emb
    Hm = 2 * Hd if w.bidirectional else Hd
    specs = [("E_src", (w.src_vocab, E))]
    for l in range(w.enc_layers):
        n_in = E if l == 0 else Hm
        for d in (("fwd", "bwd") if w.bidirectional else ("fwd",)):
            specs.append((f"enc{l}_{d}_W", (4 * Hd, n_in + Hd)))
            specs.append((f"enc{l}_{d}_b", (4 * Hd,)))
    specs.append(("E_tgt", (w.tgt_vocab, E)))
    for l in range(w.dec_layers):
        n_in = E + H if l == 0 else H
        specs.append((f"dec{l}_W", (4 * H, n_in + H)))
        specs.append((f"dec{l}_b", (4 * H,)))
    if w.attn == "general":
        specs.append(("W_a", (H, Hm)))
    elif w.attn == "concat":
        specs += [("W_a", (H, H + Hm)), ("v_a", (H,))]
    elif w.attn != "dot":
        raise ValueError(f"unknown attention type {w.attn!r}")
    specs += [("W_c", (H, Hm + H)), ("W_s", (w.tgt_vocab, H)), ("b_s", (w.tgt_vocab,))]
    return specs


def round_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32 (finite inputs)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # no uint32 overflow for finite inputs: the largest finite pattern plus 0x8000 stays below 2^32
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def make_weights(w: Workload, seed: int = WEIGHT_SEED, peaked: bool = False):
    """Dict name -> float32 array, drawn in :func:`weight_specs` order.

    ``peaked`` (tests only) scales W_a (if any) by 30 and W_s, b_s by 10 after drawing,
    which makes attention non-uniform and widens the gaps between log-probs.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    out = {}
    for name, shape in weight_specs(w):
        out[name] = rng.uniform(-0.1, 0.1, size=shape).astype(np.float32)
    if peaked:
        if "W_a" in out:
            out["W_a"] = (out["W_a"] * np.float32(30.0)).astype(np.float32)
        out["W_s"] = (out["W_s"] * np.float32(10.0)).astype(np.float32)
        out["b_s"] = (out["b_s"] * np.float32(10.0)).astype(np.float32)
    if w.wdtype == "bf16":
        out = {k: round_bf16(v) for k, v in out.items()}
    return out


def zipf_cdf(n_ranks: int, s: float) -> np.ndarray:
    p = np.arange(1, n_ranks + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(p)
    c /= c[-1]
    c[-1] = 1.0
    return c


def make_batch(w: Workload, seed: int = None, batch: int = None):
    """(src int32 [B, s_max], lens int32 [B]) for workload ``w``."""
    if seed is None:
        seed = 1000 + w.index
    B = w.batch if batch is None else batch
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(w.len_lo, w.len_hi + 1, size=B).astype(np.int32)
    cdf = zipf_cdf(w.src_vocab - 4, w.zipf_s)
    u = rng.random(size=(B, w.s_max))
    ranks = np.searchsorted(cdf, u, side="right") + 1
    ranks = np.minimum(ranks, w.src_vocab - 4)
    src = (3 + ranks).astype(np.int32)
    pos = np.arange(w.s_max)[None, :]
    src[pos >= lens[:, None]] = PAD_ID
    return src, lens


def make_targets(w: Workload, seed: int = None, batch: int = None, T: int = None):
    """(tgt int32 [B, T], tgt_len int32 [B]) for teacher-forced scoring: bounded-Zipf target ids
    (same law as the source, ids 3 + r over the target vocabulary), every sentence T = max decode
    tokens long unless T is given. Seed 2000 + workload index unless given."""
    if seed is None:
        seed = 2000 + w.index
    B = w.batch if batch is None else batch
    T = w.max_len if T is None else T
    rng = np.random.Generator(np.random.PCG64(seed))
    cdf = zipf_cdf(w.tgt_vocab - 4, w.zipf_s)
    ranks = np.minimum(np.searchsorted(cdf, rng.random(size=(B, T)), side="right") + 1, w.tgt_vocab - 4)
    return (3 + ranks).astype(np.int32), np.full(B, T, dtype=np.int32)

