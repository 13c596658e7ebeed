"""Per-phase cycle profile of the decode kernel (profiling builds only).

Build the profiling flavour first (``python -m paper_2508_07315_amd.build_lib
--phase-clocks`` -> ``libctcbeam_phase.so``: the same kernels with s_memtime
counters at every phase boundary), then on a GPU:

    python -m paper_2508_07315_amd.phase_profile --config 3 [--beam K] [--theta 12]
    python -m paper_2508_07315_amd.phase_profile --config 3 --mode greedy

Prints, per phase of the frame step (beam search: fill, barrier A,
candidates, barrier B, bound, filter, barrier C, rank, barrier D, and the update
as prune + recombination, new state, chunk plan and the rest; greedy:
scoring, the wave's best, the exchange barrier, the decision, chain headers +
fold, continuations, log-prob row loads), the mean cycles per frame of each
wave, averaged over the utterances (weighted by their frames), and the mean
chunks (refills) per frame.  Inputs are the seeded workloads of ``workloads``.
"""
from __future__ import annotations

import argparse
import math
import os
import sys

# (counter word, name); the beam update is split into prune + recombination,
# new state, chunk plan and the rest (one slot per lane; two slots per lane
# count the whole update under "upd rest")
PHASES = {"beam": [(0, "fill"), (1, "bar A"), (2, "cand"), (3, "bar B"), (14, "bound"), (4, "filter"), (5, "bar C"),
                   (6, "rank"), (7, "bar D"), (11, "upd merge"), (12, "upd state"), (13, "upd plan"),
                   (8, "upd rest")],
          "greedy": list(enumerate(["score", "best", "barrier", "decide", "hdr+fold", "arcs", "rows"]))}
WAVES = 8
WORDS = 20


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--beam", type=int, default=0, help="beam size (default: the workload's)")
    ap.add_argument("--theta", type=float, default=math.inf)
    ap.add_argument("--batch", type=int, default=0)
    ap.add_argument("--mode", choices=("beam", "greedy"), default="beam")
    args = ap.parse_args(argv)

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import numpy as np
    import torch

    import paper_2508_07315_amd as P
    import workloads as W

    lib = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libctcbeam_phase.so")
    if not os.path.exists(lib):
        raise SystemExit(f"{lib} is missing: python -m paper_2508_07315_amd.build_lib --phase-clocks")
    P.LIB_PATH = lib  # the profiling flavour of the same C ABI

    w = W.CONFIGS[args.config]
    if args.beam:
        w = w.replace(K=args.beam)
    if args.batch:
        w = w.replace(B=args.batch)
    lm = P.ctcbeam_lm_build(W.lm_for(w.lm, w.V)) if w.lm is not None else None
    bt = P.ctcbeam_boost_build(w.V, *W.phrases_for(w.boost, w.V)) if w.boost is not None else None
    dev = torch.device("cuda", 0)
    lp = torch.from_numpy(W.make_logprobs(w)).to(dev)
    lens = torch.from_numpy(W.make_lengths(w)).to(dev)
    B = w.B
    buf = torch.zeros(B * 8 + B * WAVES * WORDS, dtype=torch.int64, device=dev)
    stats = buf[: B * 8].view(B, 8)
    theta = args.theta if not math.isinf(args.theta) else w.theta
    for _ in range(2):  # the second launch is measured (the first warms caches and code)
        buf.zero_()
        if args.mode == "greedy":
            P.ctcbeam_greedy_decode(lp, lens, w.alpha, w.beta, w.boost_w, lm, bt, stats=stats)
        else:
            P.ctcbeam_decode_ex(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=theta,
                                stats=stats)
        torch.cuda.synchronize()
    ph = buf[B * 8:].view(B, WAVES, WORDS).cpu().numpy().astype(np.float64)
    frames = ph[:, 0, 9]
    chunks = ph[:, 0, 10]
    nf = frames.sum()
    what = "refills" if args.mode == "greedy" else "chunks"
    print(f"{w.name} {args.mode} K={1 if args.mode == 'greedy' else w.K} theta={theta}: {int(nf)} frames, "
          f"{chunks.sum() / max(nf, 1):.2f} {what}/frame")
    print("cycles per frame by wave (mean over utterances, weighted by frames)")
    print("phase     " + " ".join(f"{'w%d' % q:>7s}" for q in range(WAVES)) + "     mean")
    tot = np.zeros(WAVES)
    for k, name in PHASES[args.mode]:
        per = ph[:, :, k].sum(axis=0) / max(nf, 1)
        tot += per
        print(f"{name:9s} " + " ".join(f"{v:7.0f}" for v in per) + f"  {per.mean():7.0f}")
    print(f"{'total':9s} " + " ".join(f"{v:7.0f}" for v in tot) + f"  {tot.mean():7.0f}")
    if args.mode == "beam":
        per = lambda k: ph[:, 0, k].sum() / max(nf, 1)
        print(f"ranks per frame {per(15):.2f} (block or merge-tree ranks of more than 64 entries "
              f"{per(16):.2f}), pool overflows per frame {per(17):.3f}")


if __name__ == "__main__":
    main()
