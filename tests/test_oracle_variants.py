"""Pins of the oracle's semantic variants (flags): log-sum-exp recombination
and the end-of-utterance rollback of pending boosting.

* lse32 against fp64 log(exp(a) + exp(b)): within half an ulp of the result
  plus two ulp of the log1p term, exact identities;
* log-sum-exp search, exhaustive (K >= (V+1)^T, no pruning): every live
  N-best row's score is the log of the summed probability of all alignments
  of its key (the closed form of merging by sum), within 2e-5 relative;
* rollback, exhaustive: the best score equals the brute-force maximum of
  fold + w * (-pending) over all alignments, bit for bit.
"""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import brute_force, brute_force_keys_logsum

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _ulp(x):
    return float(np.spacing(np.float32(abs(x))))


def test_lse32_against_fp64():
    rng = np.random.default_rng(0)
    a = rng.uniform(-200, 5, size=4000).astype(np.float32)
    d = np.concatenate([rng.uniform(-90, 0, size=2000), rng.uniform(-3, 0, size=2000)])
    b = (a + d).astype(np.float32)
    worst = 0.0
    for x, y in zip(a, b):
        got = float(oracle.lse32(x, y))
        ref = np.logaddexp(np.float64(x), np.float64(y))
        # the final a + log1p(.) is rounded once; the log1p term carries a
        # few ulp of its own (cancellation near 0 makes ulp(ref) the wrong
        # yardstick for that part)
        lterm = ref - max(float(x), float(y))
        bound = 0.5 * _ulp(ref) + 2.0 * _ulp(lterm)
        worst = max(worst, abs(got - ref) / bound)
        assert abs(got - ref) <= bound, (x, y, got, ref)
    # symmetric, identities
    for x, y in zip(a[:200], b[:200]):
        assert oracle.lse32(x, y) == oracle.lse32(y, x)
    assert oracle.lse32(-7.5, -np.inf) == np.float32(-7.5)
    assert oracle.lse32(-np.inf, -np.inf) == -np.inf
    assert abs(float(oracle.lse32(-2.0, -2.0)) - (-2.0 + math.log(2.0))) <= 2 * _ulp(-2.0 + math.log(2.0))


def _phrases(V, rng, n=3):
    lens = rng.integers(1, 4, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]), toks


CASES = [(V, T) for V in (1, 2, 3) for T in (1, 2, 3, 4) if (V + 1) ** T <= 256]


@pytest.mark.parametrize("V,T", CASES)
@pytest.mark.parametrize("mode", ["plain", "lm", "lm_bt"])
def test_logsumexp_search_sums_over_alignments(V, T, mode):
    rng = np.random.default_rng(3000 + 100 * V + 10 * T + len(mode))
    D = W.random_logprobs(rng, 1, T, V, scale=1.5)[0]
    kw = dict(beta=0.4)
    if "lm" in mode:
        kw["lm"] = oracle.LM(W.random_small_lm(rng, 3, V, density=0.5))
        kw["alpha"] = 0.6
    if "bt" in mode:
        off, toks = _phrases(V, rng)
        kw["bt"] = oracle.BT(V, off, toks)
        kw["boost_w"] = 1.2
    ref = brute_force_keys_logsum(D, V, **kw)
    K = (V + 1) ** T
    out = oracle.decode(D[None], np.array([T]), K, kw.get("alpha", 0.0), kw["beta"],
                        kw.get("boost_w", 0.0), lm=kw.get("lm"), bt=kw.get("bt"),
                        want_nbest=True, logsumexp=True)
    sc, ln, tk = out["nbest_scores"][0], out["nbest_lengths"][0], out["nbest_tokens"][0]
    live = int(np.sum(sc != -np.inf))
    assert live == len(ref)
    got = {}
    for r in range(live):
        got.setdefault(tuple(tk[r, : ln[r]].tolist()), []).append(float(sc[r]))
    want = {}
    for (y, _), v in ref.items():
        want.setdefault(y, []).append(v)
    assert set(got) == set(want)
    for y in want:
        g, w_ = sorted(got[y]), sorted(want[y])
        for x, r in zip(g, w_):
            assert abs(x - r) <= 2e-5 * max(1.0, abs(r)), (y, g, w_)
    # the 1-best is the key with the largest summed probability
    best = max(ref.values())
    assert abs(float(out["scores"][0]) - best) <= 2e-5 * max(1.0, abs(best))


def test_logsumexp_differs_from_max_only_by_merges():
    """Without any recombination (K = 1) the flag changes nothing."""
    rng = np.random.default_rng(8)
    D = W.random_logprobs(rng, 3, 20, 5)
    a = oracle.decode(D, np.array([20, 11, 0]), 1, beta=0.3)
    b = oracle.decode(D, np.array([20, 11, 0]), 1, beta=0.3, logsumexp=True)
    for k in ("tokens", "lengths", "scores"):
        np.testing.assert_array_equal(a[k], b[k])


@pytest.mark.parametrize("V,T", [(1, 4), (2, 3), (2, 4), (3, 3)])
def test_boost_rollback_exhaustive(V, T):
    rng = np.random.default_rng(4000 + 10 * V + T)
    for _ in range(3):
        D = W.random_logprobs(rng, 1, T, V, scale=1.5)[0]
        off, toks = _phrases(V, rng, 4)
        bt = oracle.BT(V, off, toks)
        lm = oracle.LM(W.random_small_lm(rng, 2, V, density=0.5))
        kw = dict(alpha=0.5, beta=0.3, boost_w=1.7, lm=lm, bt=bt)
        best, arg = brute_force(D, V, rollback=True, **kw)
        out = oracle.decode(D[None], np.array([T]), (V + 1) ** T, 0.5, 0.3, 1.7, lm=lm, bt=bt,
                            boost_rollback=True)
        assert out["scores"][0] == best
        assert tuple(out["tokens"][0, : out["lengths"][0]].tolist()) in arg
