"""GPU parity of the LM key-row cache (one row per LM state kept across
frames; used with an LM and no boosting when one chunk holds the beam:
V of 513..1024 with K <= 8, up to 2048 with K <= 4, up to 4096 with K <= 2).

The cache changes which frames fill which rows, never a score: the decoder
with the cache and with CTCBEAM_FLAG_NO_ROW_CACHE must agree bit for bit, and
both match the CPU oracle (tokens bit-exact, scores within 1e-4).

* the 3-gram workload at reduced size and at full size (B=64, T=400: the
  6-bit row generation wraps six times per utterance);
* 1-best and N-best, max and log-sum-exp recombination, theta = inf and 12;
* fuzzing over V (all three row counts), LM order 2..6 and K;
* the full-size comparison of the two paths (no oracle: too slow there);
* an LM of more than 2^23 states (the paper-scale 6-gram) takes the refill
  path with the same results.
"""
import math

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import compare, device, handles, log, oracle_threads

pytestmark = pytest.mark.gpu


def _run(lp, lens, K, alpha, beta, lm, theta=math.inf, nbest=False, **kw):
    import torch
    dev = device()
    d_lp = torch.from_numpy(np.ascontiguousarray(lp)).to(dev)
    d_len = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    f = P.ctcbeam_decode_nbest if nbest else P.ctcbeam_decode_ex
    tok, ln, sc, ws = f(d_lp, d_len, K, alpha, beta, 0.0, lm, None, theta=theta, **kw)
    torch.cuda.synchronize()
    return dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy(),
                status=P.ctcbeam_query_status(ws))


def _same(a, b, what):
    for k in ("tokens", "lengths"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=f"{what}: {k}")
    np.testing.assert_array_equal(a["scores"].view(np.uint32), b["scores"].view(np.uint32),
                                  err_msg=f"{what}: score bits")
    assert a["status"] == 0 and b["status"] == 0, what


def _compare_nbest(g, r, what):
    np.testing.assert_array_equal(g["lengths"], r["nbest_lengths"], err_msg=what)
    np.testing.assert_array_equal(g["tokens"], r["nbest_tokens"], err_msg=what)
    gs, rs = g["scores"], r["nbest_scores"]
    inf = np.isinf(gs) | np.isinf(rs)
    np.testing.assert_array_equal(gs[inf], rs[inf], err_msg=what)
    assert np.all(np.abs(gs[~inf].astype(np.float64) - rs[~inf]) <= 1e-4), what


@pytest.mark.parametrize("K", [1, 2, 5, 8])
def test_row_cache_reduced(K):
    w = W.CONFIGS[3].replace(B=4, T=160, lengths=("uniform", 70, 160), K=K)
    lm, _, olm, _ = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    for th in (math.inf, 12.0):
        log(f"row cache cfg3 K={K} theta={th}")
        g = _run(lp, lens, K, w.alpha, w.beta, lm, theta=th)
        g0 = _run(lp, lens, K, w.alpha, w.beta, lm, theta=th, row_cache=False)
        _same(g, g0, f"cache vs refill K={K} theta={th}")
        r = oracle.decode(lp, lens, K, w.alpha, w.beta, 0.0, theta=th, lm=olm,
                          n_threads=oracle_threads(), want_nbest=True)
        compare(g, r, what=f"row cache K={K} theta={th}")
        gn = _run(lp, lens, K, w.alpha, w.beta, lm, theta=th, nbest=True)
        _compare_nbest(gn, r, what=f"row cache nbest K={K} theta={th}")


def test_row_cache_logsumexp():
    w = W.CONFIGS[3].replace(B=3, T=120, lengths=("uniform", 60, 120))
    lm, _, olm, _ = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    g = _run(lp, lens, 8, w.alpha, w.beta, lm, nbest=True, logsumexp=True)
    g0 = _run(lp, lens, 8, w.alpha, w.beta, lm, nbest=True, logsumexp=True, row_cache=False)
    _same(g, g0, "lse cache vs refill")
    r = oracle.decode(lp, lens, 8, w.alpha, w.beta, 0.0, lm=olm, n_threads=oracle_threads(),
                      want_nbest=True, logsumexp=True)
    _compare_nbest(g, r, what="lse nbest row cache")


def test_row_cache_full_size_matches_refill():
    w = W.CONFIGS[3]
    lm, _, _, _ = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log(f"row cache full size B={w.B} T={w.T}")
    g = _run(lp, lens, w.K, w.alpha, w.beta, lm)
    g0 = _run(lp, lens, w.K, w.alpha, w.beta, lm, row_cache=False)
    _same(g, g0, "full-size cache vs refill")


@pytest.mark.parametrize("seed", range(10))
def test_row_cache_fuzz(seed):
    rng = np.random.default_rng(17000 + seed)
    V = int(rng.choice([600, 1024, 1500, 2048, 3000]))
    kmax = 8 if V <= 1024 else (4 if V <= 2048 else 2)
    K = int(rng.integers(1, kmax + 1))
    B = int(rng.integers(1, 4))
    T = int(rng.integers(1, 90))
    lens = rng.integers(0, T + 1, size=B)
    lens[rng.integers(0, B)] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 3.0)))
    theta = float(rng.choice([math.inf, 5.0, 12.0]))
    alpha, beta = float(rng.uniform(0, 1)), float(rng.uniform(-1, 2))
    order = int(rng.integers(2, 7))
    counts = [min(3 * V, (V + 1) ** 2)] + [2 * V] * (order - 2)
    arrays = W.make_lm(order, V, counts, int(rng.integers(0, 1 << 30)))
    lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    lse = bool(rng.random() < 0.3)
    log(f"row cache fuzz {seed}: B={B} T={T} V={V} K={K} order={order} theta={theta} lse={lse}")
    g = _run(lp, lens, K, alpha, beta, lm, theta=theta, logsumexp=lse)
    g0 = _run(lp, lens, K, alpha, beta, lm, theta=theta, logsumexp=lse, row_cache=False)
    _same(g, g0, f"fuzz {seed} cache vs refill")
    r = oracle.decode(lp, lens, K, alpha, beta, 0.0, theta=theta, lm=olm,
                      n_threads=oracle_threads(), logsumexp=lse)
    compare(g, r, what=f"row cache fuzz {seed}")


def test_large_lm_takes_the_refill_path():
    # the 6-gram of the paper-scale workload numbers 8.5 M LM states, above
    # the 2^23 a cached entry can name: small beams without boosting refill
    # their rows every frame; results as with the flag, and the oracle's
    w = W.CONFIGS[6].replace(B=2, T=80, lengths=("uniform", 50, 80), K=8, boost=None, boost_w=0.0)
    lm, _, olm, _ = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log("6-gram without boosting, K=8 (LM above 2^23 states)")
    g = _run(lp, lens, 8, w.alpha, w.beta, lm, theta=w.theta)
    g0 = _run(lp, lens, 8, w.alpha, w.beta, lm, theta=w.theta, row_cache=False)
    _same(g, g0, "large LM default vs refill flag")
    r = oracle.decode(lp, lens, 8, w.alpha, w.beta, 0.0, theta=w.theta, lm=olm,
                      n_threads=oracle_threads())
    compare(g, r, what="large LM K=8")
