"""GPU parity for beams above 64 (up to 128, the largest beam of the paper's
Fig. "beam_size_vs_wer"): the kernel then keeps two beam slots per lane.
Against the CPU oracle: tokens bit-exact, scores within 1e-4.

* exhaustive pins (K = 128 >= (V+1)^T): the brute-force best fold and, for
  N-best, every recombination key's best fold;
* the workloads at reduced sizes with K = 65, 96, 128 (theta = inf, 12);
  the paper-scale 6-gram + boosting workload at K = 128;
* N-best and log-sum-exp recombination at K = 128, fuzzing over K in 65..128;
* beams above 64 with more than 1024 tokens are rejected (return 2).
"""
import ctypes
import math

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import compare, device, handles, log, oracle_threads, run_gpu
from oracle_helpers import brute_force, brute_force_keys

pytestmark = pytest.mark.gpu


def _nbest(lp, lens, K, alpha=0.0, beta=0.0, boost_w=0.0, lm=None, bt=None, theta=math.inf, **kw):
    import torch
    dev = device()
    d_lp = torch.from_numpy(np.ascontiguousarray(lp)).to(dev)
    d_len = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    tok, ln, sc, ws = P.ctcbeam_decode_nbest(d_lp, d_len, K, alpha, beta, boost_w, lm, bt,
                                             theta=theta, **kw)
    torch.cuda.synchronize()
    return dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy(),
                status=P.ctcbeam_query_status(ws))


def _compare_nbest(g, r, what):
    np.testing.assert_array_equal(g["lengths"], r["nbest_lengths"], err_msg=what)
    np.testing.assert_array_equal(g["tokens"], r["nbest_tokens"], err_msg=what)
    gs, rs = g["scores"], r["nbest_scores"]
    inf = np.isinf(gs) | np.isinf(rs)
    np.testing.assert_array_equal(gs[inf], rs[inf], err_msg=what)
    assert np.all(np.abs(gs[~inf].astype(np.float64) - rs[~inf]) <= 1e-4), what


@pytest.mark.parametrize("V,T", [(4, 3), (1, 7), (2, 4)])
def test_exhaustive_k128(V, T):
    rng = np.random.default_rng(5100 + 10 * V + T)
    D = W.random_logprobs(rng, 1, T, V, scale=1.5)
    arrays = W.random_small_lm(rng, 3, V, density=0.5)
    lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    best, arg = brute_force(D[0], V, alpha=0.6, beta=0.4, lm=olm)
    g = run_gpu(D, np.array([T]), 128, 0.6, 0.4, lm=lm)
    assert g["scores"][0] == best
    assert tuple(g["tokens"][0, : g["lengths"][0]].tolist()) in arg
    keys = brute_force_keys(D[0], V, alpha=0.6, beta=0.4, lm=olm)
    gn = _nbest(D, np.array([T]), 128, 0.6, 0.4, lm=lm)
    sc, ln, tk = gn["scores"][0], gn["lengths"][0], gn["tokens"][0]
    live = int(np.sum(sc != -np.inf))
    assert live == len(keys)
    got = sorted(((float(sc[r]), tuple(tk[r, : ln[r]].tolist())) for r in range(live)),
                 key=lambda e: (-e[0], e[1]))
    want = sorted(((float(s), k[0]) for k, s in keys.items()), key=lambda e: (-e[0], e[1]))
    assert got == want


@pytest.mark.parametrize("cfg,K", [(3, 65), (3, 96), (3, 128), (5, 128), (2, 100)])
def test_large_beam_reduced(cfg, K):
    w = W.CONFIGS[cfg].replace(B=3, T=90, lengths=("uniform", 40, 90), K=K)
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    for th in (math.inf, 12.0):
        log(f"large beam cfg{cfg} K={K} theta={th}")
        g = run_gpu(lp, lens, K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th)
        r = oracle.decode(lp, lens, K, w.alpha, w.beta, w.boost_w, theta=th, lm=olm, bt=obt,
                          n_threads=oracle_threads(), want_nbest=True, logsumexp=False)
        compare(g, r, what=f"cfg{cfg} K={K} theta={th}")
        assert g["status"] == 0
        if K == 128 and th == 12.0:
            gn = _nbest(lp, lens, K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th)
            _compare_nbest(gn, r, what=f"nbest cfg{cfg} K={K}")


def test_paper_scale_k128():
    w = W.CONFIGS[6].replace(B=2, T=80, lengths=("uniform", 50, 80), K=128)
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log("6-gram + boosting, K=128")
    g = run_gpu(lp, lens, 128, w.alpha, w.beta, w.boost_w, lm, bt, theta=w.theta)
    r = oracle.decode(lp, lens, 128, w.alpha, w.beta, w.boost_w, theta=w.theta, lm=olm, bt=obt,
                      n_threads=oracle_threads())
    compare(g, r, what="6-gram K=128")
    assert g["status"] == 0


def test_logsumexp_k128():
    w = W.CONFIGS[3].replace(B=3, T=70, lengths=("uniform", 30, 70), K=128)
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    gn = _nbest(lp, lens, 128, w.alpha, w.beta, w.boost_w, lm, bt, logsumexp=True)
    r = oracle.decode(lp, lens, 128, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                      n_threads=oracle_threads(), want_nbest=True, logsumexp=True)
    _compare_nbest(gn, r, what="lse nbest K=128")


def _phrases(V, rng, n):
    lens = rng.integers(1, 5, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), toks.astype(np.int32)


@pytest.mark.parametrize("seed", range(12))
def test_large_beam_fuzz(seed):
    rng = np.random.default_rng(15000 + seed)
    V = int(rng.choice([1, 2, 5, 31, 200, 513, 1024]))
    K = int(rng.integers(65, 129))
    B = int(rng.integers(1, 5))
    T = int(rng.integers(1, 30))
    lens = rng.integers(0, T + 1, size=B)
    lens[rng.integers(0, B)] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 3.0)))
    for b in range(B):
        lp[b, lens[b]:] = np.nan   # padding is never read
    theta = float(rng.choice([math.inf, 5.0, 12.0]))
    alpha, beta, bw = float(rng.uniform(0, 1)), float(rng.uniform(-1, 2)), float(rng.uniform(0, 2))
    lm = bt = olm = obt = None
    if rng.random() < 0.7:
        arrays = W.random_small_lm(rng, int(rng.integers(1, 5)), V, density=0.4) if V <= 8 else \
            W.make_lm(3, V, [min(3 * V, (V + 1) ** 2), 2 * V], int(rng.integers(0, 1 << 30)))
        lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    if rng.random() < 0.5:
        off, toks = _phrases(V, rng, int(rng.integers(1, 20)))
        bt, obt = P.ctcbeam_boost_build(V, off, toks), oracle.BT(V, off, toks)
    flags = dict(logsumexp=bool(rng.random() < 0.3), boost_rollback=bool(rng.random() < 0.3))
    log(f"large beam fuzz {seed}: B={B} T={T} V={V} K={K} theta={theta} {flags}")
    import torch
    dev = device()
    tok, ln, sc, ws = P.ctcbeam_decode_ex(torch.from_numpy(lp).to(dev),
                                          torch.from_numpy(lens.astype(np.int32)).to(dev), K,
                                          alpha, beta, bw, lm, bt, theta=theta, **flags)
    torch.cuda.synchronize()
    g = dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy())
    r = oracle.decode(lp, lens, K, alpha, beta, bw, theta=theta, lm=olm, bt=obt,
                      n_threads=oracle_threads(), **flags)
    compare(g, r, what=f"large beam fuzz {seed}")
    assert P.ctcbeam_query_status(ws) == 0


def test_wide_vocabulary_large_beam_rejected():
    import torch
    dev = device()
    lp = torch.zeros((1, 3, 1026), dtype=torch.float32, device=dev)
    ln = torch.full((1,), 3, dtype=torch.int32, device=dev)
    with pytest.raises(P.CtcbeamError) as e:
        P.ctcbeam_decode_ex(lp, ln, 65)
    assert e.value.code == 2
    P.ctcbeam_decode_ex(lp, ln, 64)   # K = 64 stays supported at any V
    torch.cuda.synchronize()
