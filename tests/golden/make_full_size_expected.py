"""Write the oracle's full-size outputs for the GPU parity tests.

Runs only the CPU oracle (``oracle/``) on the seeded inputs of ``workloads/``
at the workloads' full sizes and stores, per (workload, theta):

* the 1-best result of every utterance: transcript lengths, scores, and the
  transcripts concatenated (int16);
* greedy decoding with the same fusion (K = 1): the 1-best result only;
* the N-best result of every utterance: lengths and scores [B, K], and per
  row a 64-bit BLAKE2b digest of the int32 transcript (rows are compared by
  digest, which keeps the files small);
* a SHA-256 fingerprint of the inputs (log-probs, lengths, n-gram arrays,
  phrase list) so that a test on changed inputs fails instead of comparing
  against stale values.

Usage: python tests/golden/make_full_size_expected.py [case ...]
(cases like ``cfg3_inf``, ``cfg4_12``, ``cfg3_greedy``; default: all).  Several cases take
minutes each on 8 host threads (the 4-gram + boosting workload about 15).
"""
from __future__ import annotations

import hashlib
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as W  # noqa: E402

OUT_DIR = os.path.join(HERE, "full")
# (workload, theta): every workload at theta = inf, the LM workloads also at
# the paper's theta = 12 (Sec. IV-D); the paper-scale workload only at 12
CASES = [(1, math.inf), (2, math.inf), (3, math.inf), (3, 12.0), (4, math.inf), (4, 12.0),
         (5, math.inf), (5, 12.0), (6, 12.0)]
# greedy decoding with the same fusion (the search with K = 1; theta has no
# effect with one hypothesis)
GREEDY_CASES = [2, 3, 4, 5, 6]


def case_name(cfg: int, theta: float) -> str:
    return f"cfg{cfg}_{'inf' if math.isinf(theta) else int(theta)}"


def greedy_name(cfg: int) -> str:
    return f"cfg{cfg}_greedy"


def row_digest(tokens: np.ndarray) -> np.uint64:
    d = hashlib.blake2b(np.ascontiguousarray(tokens, dtype=np.int32).tobytes(), digest_size=8)
    return np.frombuffer(d.digest(), dtype="<u8")[0]


def input_fingerprint(w: W.Workload, lp: np.ndarray, lens: np.ndarray) -> str:
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(lp).tobytes())
    h.update(np.ascontiguousarray(lens, dtype=np.int32).tobytes())
    if w.lm is not None:
        arr = W.lm_for(w.lm, w.V)
        for part in ("ids", "log10_prob", "log10_bow"):
            for a in arr[part]:
                if a is not None:
                    h.update(np.ascontiguousarray(a).tobytes())
    if w.boost is not None:
        off, tok = W.phrases_for(w.boost, w.V)
        h.update(np.ascontiguousarray(off, dtype=np.int32).tobytes())
        h.update(np.ascontiguousarray(tok, dtype=np.int32).tobytes())
    return h.hexdigest()


def make_case(cfg: int, theta: float, n_threads: int, greedy: bool = False) -> str:
    w = W.CONFIGS[cfg]
    K = 1 if greedy else w.K
    t0 = time.time()
    lens = W.make_lengths(w)
    lp = W.make_logprobs(w)
    olm = oracle.LM(W.lm_for(w.lm, w.V)) if w.lm is not None else None
    obt = oracle.BT(w.V, *W.phrases_for(w.boost, w.V)) if w.boost is not None else None
    fp = input_fingerprint(w, lp, lens)
    t1 = time.time()
    r = oracle.decode(lp, lens, K, w.alpha, w.beta, w.boost_w, theta=theta, lm=olm, bt=obt,
                      n_threads=n_threads, want_nbest=not greedy)
    t2 = time.time()
    flat = np.concatenate([r["tokens"][b, : r["lengths"][b]] for b in range(w.B)]).astype(np.int16)
    out = dict(workload=np.array(w.name), theta=np.float64(theta), K=np.int32(K),
               fingerprint=np.array(fp), lengths=r["lengths"], scores=r["scores"],
               tokens_flat=flat)
    if not greedy:
        dig = np.zeros((w.B, w.K), dtype=np.uint64)
        for b in range(w.B):
            for k in range(w.K):
                dig[b, k] = row_digest(r["nbest_tokens"][b, k, : r["nbest_lengths"][b, k]])
        out.update(nbest_lengths=r["nbest_lengths"], nbest_scores=r["nbest_scores"],
                   nbest_digest=dig)
    name = greedy_name(cfg) if greedy else case_name(cfg, theta)
    path = os.path.join(OUT_DIR, name + ".npz")
    np.savez_compressed(path, **out)
    print(f"{name}: inputs {t1 - t0:.1f} s, oracle {t2 - t1:.1f} s "
          f"({int(lens.sum())} frames, {n_threads} threads) -> {os.path.relpath(path, ROOT)}",
          flush=True)
    return path


def main(argv):
    os.makedirs(OUT_DIR, exist_ok=True)
    want = set(argv)
    n_threads = max(1, os.cpu_count() or 1)
    for cfg, theta in CASES:
        if want and case_name(cfg, theta) not in want:
            continue
        make_case(cfg, theta, n_threads)
    for cfg in GREEDY_CASES:
        if want and greedy_name(cfg) not in want:
            continue
        make_case(cfg, math.inf, n_threads, greedy=True)


if __name__ == "__main__":
    main(sys.argv[1:])
