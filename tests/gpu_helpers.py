"""Shared helpers of the GPU tests: run the HIP decoder through the C ABI and
the CPU oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import math
import os
import sys
import time
from functools import lru_cache

import numpy as np

import oracle
import paper_2508_07315_amd as P
import workloads as W

SCORE_TOL = 1e-4   # |score_gpu - score_oracle| bound; tokens must be identical


def log(*a):
    print(f"[{time.strftime('%H:%M:%S')}]", *a, flush=True)
    sys.stdout.flush()


def device():
    import torch
    assert torch.cuda.is_available(), "GPU test without a GPU"
    return torch.device("cuda:0")


@lru_cache(maxsize=4)
def gpu_lm(spec: W.LMSpec, V: int):
    return P.ctcbeam_lm_build(W.lm_for(spec, V))


@lru_cache(maxsize=4)
def oracle_lm(spec: W.LMSpec, V: int):
    return oracle.LM(W.lm_for(spec, V))


@lru_cache(maxsize=4)
def gpu_boost(spec: W.BoostSpec, V: int):
    off, tok = W.phrases_for(spec, V)
    return P.ctcbeam_boost_build(V, off, tok)


@lru_cache(maxsize=4)
def oracle_bt(spec: W.BoostSpec, V: int):
    off, tok = W.phrases_for(spec, V)
    return oracle.BT(V, off, tok)


def run_gpu(lp: np.ndarray, lens: np.ndarray, K: int, alpha=0.0, beta=0.0, boost_w=0.0,
            lm=None, boost=None, theta=math.inf, stats=False, stream=None):
    import torch
    dev = device()
    d_lp = torch.from_numpy(np.ascontiguousarray(lp)).to(dev)
    d_len = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    st = torch.zeros((lp.shape[0], 8), dtype=torch.int64, device=dev) if stats else None
    tok, ln, sc, ws = P.ctcbeam_decode_ex(d_lp, d_len, K, alpha, beta, boost_w, lm, boost,
                                          theta=theta, stats=st, stream=stream)
    torch.cuda.synchronize()
    out = dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy(),
               status=P.ctcbeam_query_status(ws))
    if stats:
        out["stats"] = st.cpu().numpy()
    return out


def compare(gpu: dict, ref: dict, rows=None, ref_rows=None, what=""):
    """Tokens bit-exact, scores within SCORE_TOL (both -inf allowed)."""
    rows = range(gpu["tokens"].shape[0]) if rows is None else rows
    ref_rows = rows if ref_rows is None else ref_rows
    worst = 0.0
    for g, r in zip(rows, ref_rows):
        gt, rt = gpu["tokens"][g], ref["tokens"][r]
        assert gpu["lengths"][g] == ref["lengths"][r], f"{what} utt {g}: length {gpu['lengths'][g]} vs {ref['lengths'][r]}"
        if not np.array_equal(gt, rt):
            bad = int(np.nonzero(gt != rt)[0][0])
            raise AssertionError(f"{what} utt {g}: tokens differ at {bad}: gpu {gt[max(0, bad-3):bad+3]} "
                                 f"oracle {rt[max(0, bad-3):bad+3]}")
        gs, rs = float(gpu["scores"][g]), float(ref["scores"][r])
        if math.isinf(rs) or math.isinf(gs):
            assert gs == rs, f"{what} utt {g}: score {gs} vs {rs}"
        else:
            d = abs(gs - rs)
            worst = max(worst, d)
            assert d <= SCORE_TOL, f"{what} utt {g}: score {gs} vs {rs}"
    return worst


def handles(w: W.Workload):
    lm = gpu_lm(w.lm, w.V) if w.lm is not None else None
    bt = gpu_boost(w.boost, w.V) if w.boost is not None else None
    olm = oracle_lm(w.lm, w.V) if w.lm is not None else None
    obt = oracle_bt(w.boost, w.V) if w.boost is not None else None
    return lm, bt, olm, obt


def oracle_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))
