#!/usr/bin/env python3
"""Benchmark of the batched CTC beam-search step on one MI355X.

One *step* is one ``ctcbeam_decode`` launch: every frame of every utterance of
the workload (Algorithm 1 from initialisation to LM.Final, plus read-out).
Default workload: B=64 utterances, T=400 padded frames, V=1024 BPE tokens +
blank, beam K=8, 3-gram backoff LM (1024 unigrams, 300k bigrams, 1M trigrams),
alpha=0.5, beta=1.0 - synthetic, seeded, shaped like the paper's setting.

Prints ONE JSON line:
  value      = B*T / (mean launch time)   [decoded frames/s, padded frames]
  roofline   = algorithmic bytes per launch / mean launch time vs 8 TB/s HBM;
               the bytes come from the kernel's own counters (an untimed
               launch with statistics on): per utterance-frame 4*(V+1) for the
               log-prob row + 4*K back-pointers, per live beam-frame 12 B per
               LM/boosting chain state + 6 B per explicit continuation scanned,
               4 B per emitting winner; per utterance 8*V staging + 4*T + 4
               output bytes.
  cpu_baseline = the CPU oracle timed on a bounded sample of the same
               workload (a reported baseline, not a target): one warm-up and
               the median of 5 runs, on 1 thread and on up to 16 threads
               (one utterance each), with the host's CPU model and nproc.
  config.theta is null when there is no pruning (theta = +inf).

--mode nbest times the N-best entry point on the same workload (all K final
hypotheses out); --mode greedy times greedy decoding with the same LM fusion
(Algorithm 1 with one hypothesis; no back-pointers, LM / boosting rows
rebuilt once per emitted token, so its byte model counts one chain read per
emission instead of one per live beam-frame).  --batch overrides B (the
utterances are drawn from the same recipe).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "decoded frames/sec (B×T/s) at K=8, V=1024 + 3-gram LM; % HBM roofline"
METRIC_BY_MODE = {
    "beam": METRIC,
    "nbest": "decoded frames/sec (B×T/s), N-best output, K=8, V=1024 + 3-gram LM; % HBM roofline",
    "greedy": "decoded frames/sec (B×T/s), greedy + fusion, V=1024 + 3-gram LM; % HBM roofline",
}
KERNEL_SOURCES = {"beam": "ctcbeam_decode.inl", "nbest": "ctcbeam_decode.inl", "greedy": "ctcbeam_greedy.inl"}


def kernel_source_hash(mode: str = "beam") -> str:
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES[mode], "ctcbeam_internal.h"):
        with open(os.path.join(ROOT, "paper_2508_07315_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(stats, B: int, T: int, V: int, K: int, mode: str = "beam") -> int:
    """Bytes the method must move for one launch (see module docstring).
    K = 0 for greedy decoding (no back-pointers)."""
    W = V + 1
    s = stats.astype("int64")
    frames = int(s[:, 0].sum())
    per_frame = frames * (4 * W + 4 * K)
    chains = 12 * int(s[:, 2].sum()) + 6 * int(s[:, 3].sum()) + 12 * int(s[:, 4].sum()) + \
        6 * int(s[:, 5].sum())
    emit = 4 * int(s[:, 6].sum())
    outputs = K * (4 * T + 8) if mode == "nbest" else 4 * T + 4
    per_utt = B * (8 * V + outputs)
    return per_frame + chains + emit + per_utt


def load_traffic(workload: str, mode: str = "beam"):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_sha") != kernel_source_hash(mode):
        return None
    return d.get("hbm_bytes_per_launch")


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _usable_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(w, lp, lens, threads: int, mode: str = "beam", reps: int = 5):
    """The CPU oracle on the host cores, timed as one warm-up run, then the
    median of ``reps`` runs, (i) on one thread over
    one utterance and (ii) on ``threads`` threads over ``threads`` utterances
    (one per thread), wall time by time.perf_counter.  Frames/s counts padded
    frames (B*T), like the GPU metric."""
    import numpy as np

    import oracle
    import workloads as W
    lm = oracle.LM(W.lm_for(w.lm, w.V)) if w.lm is not None else None
    bt = None
    if w.boost is not None:
        off, tok = W.phrases_for(w.boost, w.V)
        bt = oracle.BT(w.V, off, tok)
    K = 1 if mode == "greedy" else w.K

    def timed(n_threads):
        idx = list(range(min(n_threads, w.B)))
        x, ln = np.ascontiguousarray(lp[idx]), lens[idx]
        ts = []
        for r in range(reps + 1):  # run 0 is the warm-up
            t0 = time.perf_counter()
            oracle.decode(x, ln, K, w.alpha, w.beta, w.boost_w, theta=w.theta, lm=lm, bt=bt,
                          n_threads=n_threads, want_nbest=mode == "nbest")
            if r > 0:
                ts.append(time.perf_counter() - t0)
        med = float(np.median(ts))
        return dict(threads=n_threads, utterances=len(idx), valid_frames=int(np.sum(ln)),
                    median_s=med, mean_s=float(np.mean(ts)), frames_per_s=len(idx) * w.T / med,
                    valid_frames_per_s=float(np.sum(ln)) / med)

    one = timed(1)
    many = timed(threads)
    return dict(value=many["frames_per_s"], unit="frames/s", cores=many["threads"], kind="oracle",
                sample=(f"utterances 0..{many['utterances'] - 1} of the {w.B} of the same workload "
                        f"(one per thread; {many['valid_frames']} valid frames, T={w.T} padded), "
                        f"one warm-up + median of {reps} runs; 1-thread figure on utterance 0"),
                threads_1=one, threads_n=many, nproc=os.cpu_count(), usable_cores=_usable_cores(),
                cpu_model=_cpu_model())


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, help="workload 1..6 (default 3)")
    ap.add_argument("--mode", choices=("beam", "nbest", "greedy"), default="beam")
    ap.add_argument("--batch", type=int, default=0, help="override the workload's B")
    ap.add_argument("--beam", type=int, default=0, help="override the workload's K")
    ap.add_argument("--logsumexp", action="store_true", help="log-sum-exp recombination variant")
    ap.add_argument("--boost-rollback", action="store_true",
                    help="end-of-utterance rollback of pending boosting")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=16,
                    help="threads (and utterances) of the multi-threaded CPU baseline, capped at "
                         "the usable host cores")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run a plain device copy of this many MiB three times "
                         "(calibrates rocprofv3 FETCH_SIZE/WRITE_SIZE against known bytes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU (asked for --gpus {args.gpus}); the decoder's utterances "
              "are independent and would be dealt across GPUs one shard each, which is not "
              "implemented", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2508_07315_amd as P
    import workloads as W

    P._load()  # no CPU fallback: fails loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    w = W.CONFIGS[args.config]
    if args.batch > 0 and args.batch != w.B:
        w = w.replace(B=args.batch, name=re.sub(r"_B\d+_", f"_B{args.batch}_", w.name))
    if args.beam > 0 and args.beam != w.K:
        w = w.replace(K=args.beam, name=re.sub(r"_K\d+", f"_K{args.beam}", w.name))
    t_setup = time.perf_counter()
    lens = W.make_lengths(w)
    lp = W.make_logprobs(w)
    lm = P.ctcbeam_lm_build(W.lm_for(w.lm, w.V)) if w.lm is not None else None
    bt = None
    if w.boost is not None:
        off, tok = W.phrases_for(w.boost, w.V)
        bt = P.ctcbeam_boost_build(w.V, off, tok)
    d_lp = torch.from_numpy(lp).to(dev)
    d_len = torch.from_numpy(lens).to(dev)
    B, T, V, K = w.B, w.T, w.V, w.K
    out_tok = torch.empty((B, T), dtype=torch.int32, device=dev)
    out_len = torch.empty((B,), dtype=torch.int32, device=dev)
    out_sc = torch.empty((B,), dtype=torch.float32, device=dev)
    ws = torch.empty((P.ctcbeam_workspace_bytes(B, T, K),), dtype=torch.uint8, device=dev)
    stats = torch.zeros((B, 8), dtype=torch.int64, device=dev)
    print(f"# setup {time.perf_counter() - t_setup:.1f} s: {w.name}", file=sys.stderr, flush=True)

    mode = args.mode
    if mode == "nbest":
        nb_tok = torch.empty((B, K, T), dtype=torch.int32, device=dev)
        nb_len = torch.empty((B, K), dtype=torch.int32, device=dev)
        nb_sc = torch.empty((B, K), dtype=torch.float32, device=dev)

    def launch(st=None):
        fl = dict(logsumexp=args.logsumexp, boost_rollback=args.boost_rollback)
        if mode == "beam":
            P.ctcbeam_decode_ex(d_lp, d_len, K, w.alpha, w.beta, w.boost_w, lm, bt, ws, out_tok,
                                out_len, out_sc, theta=w.theta, stats=st, **fl)
        elif mode == "nbest":
            P.ctcbeam_decode_nbest(d_lp, d_len, K, w.alpha, w.beta, w.boost_w, lm, bt, ws, nb_tok,
                                   nb_len, nb_sc, theta=w.theta, stats=st, **fl)
        else:
            P.ctcbeam_greedy_decode(d_lp, d_len, w.alpha, w.beta, w.boost_w, lm, bt, ws, out_tok,
                                    out_len, out_sc, stats=st, boost_rollback=args.boost_rollback)

    # untimed launch with the kernel's counters on: algorithmic bytes
    launch(stats)
    torch.cuda.synchronize()
    alg_bytes = algorithmic_bytes(stats.cpu().numpy(), B, T, V, 0 if mode == "greedy" else K, mode)
    status = P.ctcbeam_query_status(ws)
    for _ in range(args.warmup):
        launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        launch()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    k_ms = [e0.elapsed_time(e1) for e0, e1 in ev]
    mean_ms = float(np.mean(k_ms))
    ms_per_step = wall * 1e3 / args.steps
    value = B * T / (mean_ms * 1e-3)
    achieved = alg_bytes / (mean_ms * 1e-3) / 1e9
    traffic = load_traffic(w.name if mode == "beam" else f"{w.name}_{mode}", mode)
    result = {
        "metric": METRIC_BY_MODE[mode],
        "value": value,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "mode": mode,
                   "variants": [f for f, on in (("logsumexp", args.logsumexp),
                                                ("boost_rollback", args.boost_rollback)) if on], "B": B, "T": T, "V": V, "K": 1 if mode == "greedy" else K,
                   "lm": None if w.lm is None else f"{w.lm.order}-gram, {'/'.join(str(c) for c in w.lm.counts)} explicit n-grams",
                   "boost": None if w.boost is None else f"{w.boost.n_phrases} phrases",
                   "alpha": w.alpha, "beta": w.beta, "boost_w": w.boost_w,
                   "theta": None if math.isinf(w.theta) else w.theta,
                   "parallelism": "one wave per utterance" if mode == "greedy"
                   else "one workgroup per utterance"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic},
        "kernel_ms_mean": mean_ms,
        "kernel_ms_median": float(np.median(k_ms)),
        "kernel_ms_min": float(np.min(k_ms)),
        "algorithmic_bytes_per_launch": alg_bytes,
        "valid_frames_per_s": float(np.sum(lens)) / (mean_ms * 1e-3),
        "us_per_frame_step": mean_ms * 1e3 / T,
        "status_bits": status,
    }
    if args.copy_mib > 0:
        n = args.copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n * 4
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(
            w, lp, lens, max(1, min(args.cpu_threads, _usable_cores())), mode)
    print(json.dumps(result, allow_nan=False), flush=True)


if __name__ == "__main__":
    main()
