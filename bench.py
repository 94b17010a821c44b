"""Throughput of batched beam-search translation on one MI355X, with roofline and CPU-oracle baselines.

One step = one onmt_beam_search call over the paper-default workload (2-layer 500-unit LSTM encoder and
input-feeding decoder, emb 500, general attention, vocab 50000, batch 64 with source lengths 10-50,
beam 5, max decode 100, fp32), i.e. encoder + every decoder step + beam bookkeeping + backtrack, with
the source batch and weights already resident in device memory.

Prints one JSON line: target tokens/s over the timed steps, the generator kernel's achieved fraction of
the fp32 MFMA peak (timed with HIP events on the library's stream inside the timed region), and the CPU
oracle's throughput on a bounded sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "target tokens/sec, beam-5 2×500 LSTM batch 64; MFMA util / HBM GB/s fraction"
PEAK_FP32_TFLOPS = 157.3
PEAK_BF16_TFLOPS = 2500.0
GEN_TIMING_PERIOD = 4
COUNTERS_FILE = os.path.join(ROOT, "profiles", "gen_gemm_default_counters.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="default")
    ap.add_argument("--mode", choices=["search", "score", "vendor"], default="search",
                    help="search: beam search (the headline metric); score: teacher-forced scoring of "
                         "max-decode-long synthetic targets; vendor: time the vendor GEMM library "
                         "(torch.matmul) at the workload's decoder GEMM shapes, for comparison with the "
                         "library's fused kernels")
    ap.add_argument("--attn", choices=["general", "dot", "concat"], default=None,
                    help="attention score type (default: the workload's, general)")
    ap.add_argument("--beta", type=float, default=0.0, help="coverage penalty weight of the search (0 = off)")
    ap.add_argument("--banned", type=int, default=0,
                    help="ban this many target ids (4, 4 + 7, 4 + 14, ...) from every hypothesis (0 = none)")
    ap.add_argument("--max-unk", type=int, default=-1, help="at most this many UNK tokens per hypothesis (-1 = no limit)")
    ap.add_argument("--align", action="store_true", help="also return attention-argmax alignments of the outputs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sentences", type=int, default=4)
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run one plain device-to-device copy of this many bytes (counter calibration)")
    return ap.parse_args()


def copy_calibration(nbytes):
    """One plain device copy of a known size, to scale rocprofv3's FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes}), flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("gemm.hip", "common.h", "kernels.h"):
        h.update(open(os.path.join(ROOT, "paper_1805_11462_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_counters(per_launch_flops_key):
    """HBM bytes per generator launch from committed rocprofv3 counters, if taken on the current kernel."""
    try:
        c = json.load(open(COUNTERS_FILE))
    except (OSError, ValueError):
        return None
    if c.get("kernel_source_hash") != kernel_source_hash() or c.get("workload") != per_launch_flops_key:
        return None
    return c.get("hbm_bytes_per_launch")


def cpu_threads():
    """Threads the oracle's BLAS actually uses on this host."""
    try:
        from threadpoolctl import threadpool_info
        return int(max([p.get("num_threads", 1) for p in threadpool_info()] or [1]))
    except Exception:
        return len(os.sched_getaffinity(0))


def banned_ids(w, n):
    return tuple(range(4, 4 + 7 * n, 7)) if n else ()


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def blas_vendor():
    try:
        import numpy as np
        cfg = np.show_config(mode="dicts")
        b = cfg["Build Dependencies"]["blas"]
        return f"{b.get('name', '?')} {b.get('version', '')}".strip()
    except Exception:
        return "unknown"


def cpu_baseline(w, weights, src, lens, n_sent, beta=0.0, banned=(), max_unk=-1):
    """The oracle on the first n_sent sentences of the same batch, on this host's cores: its fp32 mode
    (single-precision BLAS products, fp64 beam scores) is the timed baseline; the fp64 parity mode is
    timed on the same sentences and reported beside it."""
    import numpy as np
    from oracle import onmt_oracle as O
    threads = cpu_threads()
    out = {}
    for name, dt_ in (("fp32", np.float32), ("fp64", np.float64)):
        m = O.model_from(w, weights, dtype=dt_)
        t0 = time.perf_counter()
        res = O.beam_search(m, src[:n_sent], lens[:n_sent], w.beam, w.max_len, w.alpha, beta=beta, banned=banned,
                            max_unk=max_unk)
        dt = time.perf_counter() - t0
        out[name] = (int(sum(len(t) for t in res.tokens)), dt)
    toks, dt = out["fp32"]
    toks64, dt64 = out["fp64"]
    return {"value": round(toks / dt, 3), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n_sent} of the {src.shape[0]} sentences (full beam search incl. encoder), "
                      f"{toks} target tokens in {dt:.1f} s with the oracle's fp32 mode (fp64 beam scores)",
            "value_fp64": round(toks64 / dt64, 3), "cpu_model": cpu_model(), "blas": blas_vendor()}


KERNEL_KINDS = ("generator", "lstm", "attention", "output", "beam_step")
PEAK_HBM_GBS = 8000.0


def issued_mfma(w, achieved_tflops):
    """What the generator's matrix cores execute: its products run as bf16 MFMAs on bf16 term planes. fp32
    models: weights and activations as three bf16 terms each, six term products per fp32 product
    (fp32-accurate); bf16 models: two activation terms against the exact bf16 weights. `frac` is the issued
    bf16 MFMA rate against the bf16 dense peak."""
    products = 6 if w.wdtype == "fp32" else 2
    rate = achieved_tflops * products
    return {"mfma": "v_mfma_f32_16x16x32_bf16", "term_products": products, "achieved": round(rate, 1),
            "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(rate / PEAK_BF16_TFLOPS, 4)}


def kernel_fractions(w, lens, timed, peak_tflops):
    """Average launch time of every timed kernel kind (HIP events on the library's stream, every
    GEN_TIMING_PERIOD-th launch of each kind during one extra search after the timed region, so that the
    timed searches carry only the generator's event pairs) and its achieved fraction of the
    roofline that bounds it: algorithmic flops / time against the MFMA peak of the operand type for the
    GEMMs, algorithmic bytes / time against HBM for the attention, none for the (latency-bound) beam step.
    Per launch: generator 2 N V H flops; decoder LSTM layer 2 N 4H (2H) flops (input or feed half and
    recurrent half; the embedding rows of layer 1 come from a precomputed table); attentional output
    2 N H (Hm + H) flops; attention 4 bytes x (keys + memory of every real source position, H + Hm wide,
    plus the N query rows read and the N context rows written)."""
    import numpy as np
    N = w.batch * w.beam
    H, V = w.hidden, w.tgt_vocab
    Hm = H
    real = int(np.asarray(lens).sum())
    work = {"generator": ("mfma", 2.0 * N * V * H),
            "lstm": ("mfma", 2.0 * N * 4 * H * 2 * H),
            "attention": ("hbm", 4.0 * (real * (H + Hm) + N * H + N * Hm)),
            "output": ("mfma", 2.0 * N * H * (Hm + H)),
            "beam_step": ("latency", None)}
    out = {}
    for kind, (n, ms) in timed.items():
        if not n:
            continue
        us = ms * 1e3 / n
        bound, per = work[kind]
        e = {"launches_timed": n, "avg_launch_us": round(us, 2), "bound": bound}
        if bound == "mfma":
            ach = per / (us * 1e-6) / 1e12
            e.update({"flops_per_launch": per, "achieved": round(ach, 2), "unit": "TFLOP/s",
                      "peak": peak_tflops, "frac": round(ach / peak_tflops, 4)})
        elif bound == "hbm":
            ach = per / (us * 1e-6) / 1e9
            e.update({"bytes_per_launch": per, "achieved": round(ach, 1), "unit": "GB/s", "peak": PEAK_HBM_GBS,
                      "frac": round(ach / PEAK_HBM_GBS, 4)})
        out[kind] = e
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU design shards "
              f"sentences across GPUs and is not measured here", file=sys.stderr)
        sys.exit(2)
    if args.copy_bytes:
        copy_calibration(args.copy_bytes)
        return
    import numpy as np
    import torch

    import workloads as W
    from paper_1805_11462_amd.translator import Translator, make_config

    w = W.get(args.workload)
    if args.attn:
        w = W.Workload(**{**w.as_dict(), "attn": args.attn})
    if args.mode == "vendor":
        return bench_vendor(w)
    weights = W.make_weights(w)
    src, lens = W.make_batch(w)
    B, S = src.shape
    cfg = make_config(w.enc_layers, w.dec_layers, w.bidirectional, w.emb, w.hidden, w.src_vocab, w.tgt_vocab,
                      w.wdtype, attn=w.attn)
    tr = Translator(cfg, [weights[n] for n, _ in W.weight_specs(w)], device="cuda:0")
    src_d = torch.from_numpy(src).cuda()
    lens_d = torch.from_numpy(lens).cuda()
    if args.mode == "score":
        return bench_score(args, w, weights, tr, src, lens, src_d, lens_d)
    banned = banned_ids(w, args.banned)
    if banned and banned[-1] >= w.tgt_vocab:
        sys.exit(f"--banned {args.banned} reaches past the target vocabulary ({w.tgt_vocab})")
    buf = tr.search_buffers(B, S, w.beam, w.max_len, w.alpha, beta=args.beta, banned=banned,
                            max_unk=args.max_unk, align=args.align)

    for i in range(args.warmup):
        tr.beam_search(src_d, lens_d, buf)
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()

    # the generator's launch time is sampled on every GEN_TIMING_PERIOD-th launch of the timed searches
    tr.profile(GEN_TIMING_PERIOD, kinds=("generator",))
    for kind in KERNEL_KINDS:
        tr.profile_read(reset=True, kind=kind)
    tokens = 0
    step_s = []
    len_host = torch.empty(B, dtype=torch.int32, pin_memory=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ts = time.perf_counter()
        tr.beam_search(src_d, lens_d, buf)       # returns with its outputs written (stream synchronized)
        step_s.append(time.perf_counter() - ts)
        len_host.copy_(buf["len"])                 # target tokens of this step's 1-best outputs
        tokens += int(len_host.numpy().sum())
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    n_gen, gen_ms = tr.profile_read(reset=True, kind="generator")
    # every kind's launch time, sampled the same way on one more (untimed) search of the same batch
    tr.profile(GEN_TIMING_PERIOD, kinds=KERNEL_KINDS)
    tr.beam_search(src_d, lens_d, buf)
    torch.cuda.synchronize()
    timed = {kind: tr.profile_read(reset=True, kind=kind) for kind in KERNEL_KINDS}
    tr.profile(False)
    print(f"[bench] timed {args.steps} steps in {dt:.3f} s", file=sys.stderr, flush=True)

    N = B * w.beam
    gen_flops = 2.0 * N * w.tgt_vocab * w.hidden          # per generator launch (vocabulary projection)
    avg_gen_s = gen_ms / 1e3 / max(n_gen, 1)
    achieved = gen_flops / avg_gen_s / 1e12 if n_gen else 0.0
    peak = PEAK_BF16_TFLOPS if w.wdtype == "bf16" else PEAK_FP32_TFLOPS
    out = {
        "metric": METRIC,
        "value": round(tokens / dt, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.wdtype == "fp32" else "bf16",
        "data": "synthetic (seeded uniform(-0.1,0.1) weights, bounded-Zipf source tokens)",
        "config": {"workload": f"{w.name}: {w.enc_layers}x{w.hidden} LSTM enc/dec, emb {w.emb}, vocab {w.tgt_vocab}, "
                               f"batch {w.batch}, src len {w.len_lo}-{w.len_hi}, beam {w.beam}, "
                               f"max decode {w.max_len}, alpha {w.alpha}, {w.wdtype}, {w.attn} attention"
                               + (f", coverage beta {args.beta}" if args.beta else "")
                               + (f", {len(banned)} banned ids" if banned else "")
                               + (f", max {args.max_unk} UNK" if args.max_unk >= 0 else "")
                               + (", attention alignments" if args.align else ""),
                   "global_batch": B, "beam": w.beam, "max_decode": w.max_len,
                   "target_tokens_per_step": tokens // max(args.steps, 1)},
        "step_ms": {"min": round(min(step_s) * 1e3, 3), "median": round(sorted(step_s)[len(step_s) // 2] * 1e3, 3),
                    "max": round(max(step_s) * 1e3, 3)},
        "roofline": {"kernel": "k_gemm_gen_lds (generator GEMM + fused log-softmax/top-K partials)",
                     "bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": traffic_from_counters(w.name),
                     "launches_timed": n_gen, "avg_launch_us": round(avg_gen_s * 1e6, 2),
                     "flops_per_launch": gen_flops,
                     "issued": issued_mfma(w, achieved)},
    }
    out["kernels"] = kernel_fractions(w, lens, timed, peak)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, weights, src, lens, args.cpu_sentences, args.beta, banned,
                                           args.max_unk)
    print(json.dumps(out), flush=True)


def bench_vendor(w):
    """Plain GEMMs of the vendor library (torch.matmul, which runs hipBLASLt on ROCm) at the shapes of one
    decoder step's GEMMs: a reference for what a library GEMM takes at these shapes without the gathers and
    epilogues that the library's own kernels fuse in. bf16 workloads multiply several bf16 terms of each
    activation (two in the generator, three in the decoder layers and W_c), so the reference GEMM concatenates
    that many copies along K (A = [p0 | p1 | ...], W = [W | W | ...]): the same MFMA work. Not part of the
    translation path; prints one JSON line per shape."""
    import torch
    if not torch.cuda.is_available():
        sys.exit("--mode vendor needs a GPU")
    N = w.batch * w.beam
    H, E, V = w.hidden, w.emb, w.tgt_vocab
    Hm = w.hidden                     # memory width: a bidirectional encoder's directions have hidden / 2 units each
    bf16 = w.wdtype == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    # (name, M, N, K, activation terms of the library's bf16 product)
    shapes = [("generator", N, V, H, 2), ("decoder LSTM layer (feed or input ; h)", N, 4 * H, 2 * H, 3),
              ("attentional output W_c ([ctx ; h])", N, H, Hm + H, 3),
              ("square 8192 (what the library reaches on a large GEMM)", 8192, 8192, 8192, 1)]
    for name, M, Ncol, K, terms in shapes:
        rep = terms if bf16 else 1
        a = torch.randn(M, rep * K, device="cuda", dtype=dt)
        b = torch.randn(Ncol, rep * K, device="cuda", dtype=dt).t()
        out = torch.empty(M, Ncol, device="cuda", dtype=dt)
        for _ in range(5):
            torch.matmul(a, b, out=out)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        it = 50
        e0.record()
        for _ in range(it):
            torch.matmul(a, b, out=out)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / it
        flops = 2.0 * M * Ncol * K
        print(json.dumps({"vendor_gemm": name, "workload": w.name, "M": M, "N": Ncol, "K": K,
                          "operands": f"bf16, {rep} activation terms along K" if bf16 else "fp32",
                          "us": round(us, 2), "tflops": round(flops / us / 1e6, 1),
                          "frac_of_peak": round(flops / us / 1e6 / peak, 3),
                          "frac_counting_terms": round(rep * flops / us / 1e6 / peak, 3)}), flush=True)


def bench_score(args, w, weights, tr, src, lens, src_d, lens_d):
    """Teacher-forced scoring throughput: scored target tokens per second (same timing rules)."""
    import torch
    import workloads as W

    B, S = src.shape
    tgt, tgt_len = W.make_targets(w)
    T = tgt.shape[1]
    tgt_d = torch.from_numpy(tgt).cuda()
    tlen_d = torch.from_numpy(tgt_len).cuda()
    buf = tr.score_buffers(B, S, T)
    for i in range(args.warmup):
        tr.score(src_d, lens_d, tgt_d, tlen_d, buf)
    torch.cuda.synchronize()
    tr.profile(1)                                      # scoring launches the generator once per call
    tr.profile_read(reset=True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        tr.score(src_d, lens_d, tgt_d, tlen_d, buf)     # returns with its outputs written
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    n_gen, gen_ms = tr.profile_read(reset=True)
    tr.profile(False)
    tokens = int(tgt_len.sum()) * args.steps
    gen_flops = 2.0 * B * int(tgt_len.max()) * w.tgt_vocab * w.hidden    # one launch over all steps' rows
    avg_gen_s = gen_ms / 1e3 / max(n_gen, 1)
    achieved = gen_flops / avg_gen_s / 1e12 if n_gen else 0.0
    peak = PEAK_BF16_TFLOPS if w.wdtype == "bf16" else PEAK_FP32_TFLOPS
    out = {
        "metric": "teacher-forced target tokens/sec (per-token log-probs and NLL of given targets)",
        "value": round(tokens / dt, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(dt / args.steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if w.wdtype == "fp32" else "bf16",
        "data": "synthetic (seeded weights, bounded-Zipf source and target tokens)",
        "config": {"workload": f"{w.name} teacher-forced scoring, batch {B}, target length {T}",
                   "global_batch": B, "target_len": T},
        "roofline": {"kernel": "k_gemm_gen_lds (generator GEMM + fused log-softmax partials)", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None, "launches_timed": n_gen,
                     "avg_launch_us": round(avg_gen_s * 1e6, 2), "flops_per_launch": gen_flops,
                     "issued": issued_mfma(w, achieved)},
    }
    if not args.no_cpu_baseline:
        import numpy as np
        from oracle import onmt_oracle as O
        n = max(1, min(args.cpu_sentences, B))
        ct = {}
        for name, dt_ in (("fp32", np.float32), ("fp64", np.float64)):
            m = O.model_from(w, weights, dtype=dt_)
            t1 = time.perf_counter()
            O.score_batch(m, src[:n], lens[:n], tgt[:n], tgt_len[:n])
            ct[name] = time.perf_counter() - t1
        ntok = int(tgt_len[:n].sum())
        out["cpu_baseline"] = {"value": round(ntok / ct["fp32"], 3), "unit": "tokens/s",
                               "cores": cpu_threads(), "kind": "oracle",
                               "sample": f"{n} of the {B} sentences, {ntok} target tokens in {ct['fp32']:.1f} s "
                                         f"with the oracle's fp32 mode",
                               "value_fp64": round(ntok / ct["fp64"], 3), "cpu_model": cpu_model(),
                               "blas": blas_vendor()}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
