"""GPU parity of the semantic variants (CTCBEAM_FLAG_LOGSUMEXP,
CTCBEAM_FLAG_BOOST_ROLLBACK, and in the fuzzing CTCBEAM_FLAG_REPEAT_SCORE)
against the CPU oracle with the same flags.

Bar: tokens bit-exact, scores within 1e-4 (both sides run the same fp32
log-sum-exp steps, so the difference is expected to be 0).

* the workloads at reduced sizes, 1-best and N-best, theta = inf and 12,
  both recombination code paths (K <= 16 and K > 16);
* exhaustive inputs (K >= (V+1)^T) with log-sum-exp, where every alignment
  is kept and merged;
* rollback for the beam, N-best and greedy entry points;
* fuzzing over shapes, LM, boosting, theta and flags; unknown flag bits.
"""
import ctypes
import math

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import compare, device, handles, log, oracle_threads

pytestmark = pytest.mark.gpu

REDUCED = {
    2: dict(B=6, T=120, lengths=("uniform", 40, 120)),
    3: dict(B=6, T=120, lengths=("uniform", 40, 120)),
    4: dict(B=3, T=80, lengths=("uniform", 40, 80)),
    5: dict(B=3, T=60, lengths=("uniform", 30, 60)),
}


def _dev(lp, lens):
    import torch
    dev = device()
    return (torch.from_numpy(np.ascontiguousarray(lp)).to(dev),
            torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev))


def run(lp, lens, K, alpha=0.0, beta=0.0, boost_w=0.0, lm=None, bt=None, theta=math.inf,
        nbest=False, greedy=False, **flags):
    import torch
    d_lp, d_len = _dev(lp, lens)
    if greedy:
        tok, ln, sc, ws = P.ctcbeam_greedy_decode(d_lp, d_len, alpha, beta, boost_w, lm, bt,
                                                  boost_rollback=flags.get("boost_rollback", False))
    elif nbest:
        tok, ln, sc, ws = P.ctcbeam_decode_nbest(d_lp, d_len, K, alpha, beta, boost_w, lm, bt,
                                                 theta=theta, **flags)
    else:
        tok, ln, sc, ws = P.ctcbeam_decode_ex(d_lp, d_len, K, alpha, beta, boost_w, lm, bt,
                                              theta=theta, **flags)
    torch.cuda.synchronize()
    return dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy(),
                status=P.ctcbeam_query_status(ws))


def compare_nbest(g, r, what):
    np.testing.assert_array_equal(g["lengths"], r["nbest_lengths"], err_msg=what)
    np.testing.assert_array_equal(g["tokens"], r["nbest_tokens"], err_msg=what)
    gs, rs = g["scores"], r["nbest_scores"]
    inf = np.isinf(gs) | np.isinf(rs)
    np.testing.assert_array_equal(gs[inf], rs[inf], err_msg=what)
    assert np.all(np.abs(gs[~inf].astype(np.float64) - rs[~inf]) <= 1e-4), what


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_logsumexp_reduced(cfg):
    w = W.CONFIGS[cfg].replace(**REDUCED[cfg])
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    for th in (math.inf, 12.0):
        log(f"logsumexp cfg{cfg} B={w.B} T={w.T} K={w.K} theta={th}")
        g = run(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th, logsumexp=True)
        r = oracle.decode(lp, lens, w.K, w.alpha, w.beta, w.boost_w, theta=th, lm=olm, bt=obt,
                          n_threads=oracle_threads(), want_nbest=True, logsumexp=True)
        compare(g, r, what=f"lse cfg{cfg} theta={th}")
        assert g["status"] == 0
        gn = run(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th, nbest=True,
                 logsumexp=True)
        compare_nbest(gn, r, what=f"lse nbest cfg{cfg} theta={th}")


@pytest.mark.parametrize("V", [1, 2, 3])
def test_logsumexp_exhaustive(V):
    for T in (2, 3):
        if (V + 1) ** T > 64:
            continue
        rng = np.random.default_rng(700 + 10 * V + T)
        D = W.random_logprobs(rng, 1, T, V, scale=1.5)
        arrays = W.random_small_lm(rng, 3, V, density=0.5)
        lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
        g = run(D, np.array([T]), 64, 0.6, 0.4, lm=lm, nbest=True, logsumexp=True)
        r = oracle.decode(D, np.array([T]), 64, 0.6, 0.4, lm=olm, want_nbest=True, logsumexp=True)
        compare_nbest(g, r, what=f"lse exhaustive V={V} T={T}")


@pytest.mark.parametrize("cfg", [4, 5])
def test_boost_rollback(cfg):
    w = W.CONFIGS[cfg].replace(**REDUCED[cfg])
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log(f"rollback cfg{cfg} B={w.B} T={w.T} K={w.K}")
    r = oracle.decode(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                      n_threads=oracle_threads(), want_nbest=True, boost_rollback=True)
    g = run(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, boost_rollback=True)
    compare(g, r, what=f"rollback cfg{cfg}")
    gn = run(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, nbest=True, boost_rollback=True)
    compare_nbest(gn, r, what=f"rollback nbest cfg{cfg}")
    r1 = oracle.decode(lp, lens, 1, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                       n_threads=oracle_threads(), boost_rollback=True)
    gg = run(lp, lens, 1, w.alpha, w.beta, w.boost_w, lm, bt, greedy=True, boost_rollback=True)
    compare(gg, r1, what=f"rollback greedy cfg{cfg}")


def _phrases(V, rng, n):
    lens = rng.integers(1, 5, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), toks.astype(np.int32)


@pytest.mark.parametrize("seed", range(16))
def test_variants_fuzz(seed):
    rng = np.random.default_rng(13000 + seed)
    V = int(rng.choice([1, 2, 3, 7, 31, 200, 513, 1024]))
    K = int(rng.choice([2, 3, 8, 16, 17, 33, 64]))
    B = int(rng.integers(1, 6))
    T = int(rng.integers(1, 40))
    lens = rng.integers(0, T + 1, size=B)
    lens[rng.integers(0, B)] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 3.0)))
    theta = float(rng.choice([math.inf, 5.0, 12.0]))
    alpha, beta, bw = float(rng.uniform(0, 1)), float(rng.uniform(-1, 2)), float(rng.uniform(0, 2))
    lm = bt = olm = obt = None
    if rng.random() < 0.7:
        arrays = W.random_small_lm(rng, int(rng.integers(1, 5)), V, density=0.4) if V <= 8 else \
            W.make_lm(3, V, [min(3 * V, (V + 1) ** 2), 2 * V], int(rng.integers(0, 1 << 30)))
        lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    if rng.random() < 0.6:
        off, toks = _phrases(V, rng, int(rng.integers(1, 20)))
        bt, obt = P.ctcbeam_boost_build(V, off, toks), oracle.BT(V, off, toks)
    flags = dict(logsumexp=bool(rng.random() < 0.8), boost_rollback=bool(rng.random() < 0.5),
                 repeat_score=bool(rng.random() < 0.5))
    log(f"variants fuzz {seed}: B={B} T={T} V={V} K={K} theta={theta} {flags}")
    g = run(lp, lens, K, alpha, beta, bw, lm, bt, theta=theta, **flags)
    r = oracle.decode(lp, lens, K, alpha, beta, bw, theta=theta, lm=olm, bt=obt,
                      n_threads=oracle_threads(), **flags)
    compare(g, r, what=f"variants fuzz {seed}")
    assert g["status"] == 0


def test_unknown_flag_bits_are_rejected():
    import torch
    d_lp, d_len = _dev(np.zeros((1, 3, 5), dtype=np.float32), np.array([3]))
    lib = P._load()
    ws = torch.empty((P.ctcbeam_workspace_bytes(1, 3, 2),), dtype=torch.uint8, device=device())
    tok = torch.empty((1, 3), dtype=torch.int32, device=device())
    sc = torch.empty((1,), dtype=torch.float32, device=device())
    o = P._Opts()
    o.prune_theta = math.inf
    o.flags = 16
    rc = lib.ctcbeam_decode_ex(ctypes.c_void_p(d_lp.data_ptr()), ctypes.c_void_p(d_len.data_ptr()),
                               1, 3, 4, 2, 0.0, 0.0, 0.0, None, None, ctypes.c_void_p(ws.data_ptr()),
                               ws.numel(), ctypes.c_void_p(tok.data_ptr()), None,
                               ctypes.c_void_p(sc.data_ptr()), None, ctypes.byref(o))
    assert rc == 1 and b"flag" in lib.ctcbeam_last_error()
