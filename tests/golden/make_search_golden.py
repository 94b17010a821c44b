"""Write the oracle's beam-search results for every sentence of the five workloads at three data seeds.

Section 2 item (d) (beam search) and Section 4.2 (length normalisation) define what is computed; the
oracle (plain fp64 NumPy) computes it. This script calls only ``oracle/`` and the seeded input
generators of ``workloads/``; nothing here comes from the HIP path. The GPU parity tests compare the
library's searches of the same seeded batches with these files: tokens must be identical wherever the
recorded decision margin exceeds twice the tolerance, and every sentence is replayed step by step.

Files: ``search_<workload>_seed<seed>.npz`` with ``src [B, S]``, ``lens [B]`` (the inputs, so a change of
the generators is caught), ``tokens [B, max_len]`` (pad-filled), ``len``, ``raw``, ``norm``, ``steps``
(finish step) and ``margin`` (smallest decision margin of the sentence's run), all per sentence, and the
search's record per step: ``trace_slot``, ``trace_tok`` ``[max_len, B, beam]`` by rank (-1 = nothing
chosen) and ``trace_margin [max_len, B]`` (that step's decision margin, inf once a sentence is done).

Usage: ``python tests/golden/make_search_golden.py [--workloads tiny,default,...] [--seeds 0,1,2]``
(seed offsets from the workload's data seed 1000 + index). The whole set takes about half an hour of
one CPU's NumPy.
"""

import argparse
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as W                       # noqa: E402
from oracle import onmt_oracle as O         # noqa: E402

NAMES = ("tiny", "default", "larger", "greedy", "long")
SEED_OFFSETS = (0, 1, 2)


def data_seed(w, offset):
    return 1000 + w.index + offset


def golden_path(name, seed):
    return os.path.join(HERE, f"search_{name}_seed{seed}.npz")


def make(name, offset):
    w = W.get(name)
    seed = data_seed(w, offset)
    weights = W.make_weights(w)
    m = O.model_from(w, weights)
    src, lens = W.make_batch(w, seed=seed)
    t0 = time.perf_counter()
    res = O.beam_search(m, src, lens, w.beam, w.max_len, w.alpha, record=True)
    B, K, T = src.shape[0], w.beam, w.max_len
    tok = np.full((B, T), W.PAD_ID, np.int32)
    for b, t in enumerate(res.tokens):
        tok[b, :len(t)] = t
    n_run = len(res.trace["slot"])
    tr_slot = np.full((T, B, K), -1, np.int32)
    tr_tok = np.full((T, B, K), -1, np.int32)
    tr_margin = np.full((T, B), np.inf)
    tr_slot[:n_run] = np.asarray(res.trace["slot"])
    tr_tok[:n_run] = np.asarray(res.trace["tok"])
    tr_margin[:n_run] = np.asarray(res.trace["margin"])
    np.savez_compressed(golden_path(name, seed), src=src, lens=lens, tokens=tok,
                        len=np.array([len(t) for t in res.tokens], np.int32), raw=res.raw, norm=res.norm,
                        steps=res.steps.astype(np.int32), margin=res.margin, trace_slot=tr_slot, trace_tok=tr_tok,
                        trace_margin=tr_margin)
    print(f"{name} seed {seed}: {B} sentences in {time.perf_counter() - t0:.0f} s, "
          f"median margin {np.median(res.margin):.3g}", flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", default=",".join(NAMES))
    ap.add_argument("--seeds", default=",".join(str(s) for s in SEED_OFFSETS), help="offsets from 1000 + index")
    a = ap.parse_args()
    for name in a.workloads.split(","):
        for off in a.seeds.split(","):
            make(name, int(off))


if __name__ == "__main__":
    main()
