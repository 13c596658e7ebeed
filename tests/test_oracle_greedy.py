"""Pins of the oracle's single-hypothesis search with fusion (greedy decoding
with LM / boosting, the greedy rows of Table II): Algorithm 1 with K = 1
against a separately written sequential search (``greedy_fused``) that scores
every label of every frame with the candidate fold and keeps the first
maximum.  The plain case (no fusion) is pinned against textbook greedy CTC in
test_oracle_search.py."""
import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import brute_force, greedy_fused

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _phrases(V, rng, n):
    lens = rng.integers(1, 4, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]), toks


@pytest.mark.parametrize("seed", range(24))
def test_greedy_fused_matches_sequential_search(seed):
    rng = np.random.default_rng(500 + seed)
    V = int(rng.choice([1, 2, 3, 5, 9, 17]))
    T = int(rng.integers(1, 25))
    D = W.random_logprobs(rng, 1, T, V, scale=float(rng.uniform(0.5, 3.0)))[0]
    mode = seed % 4   # plain+beta, lm, bt, lm+bt
    kw = dict(beta=float(rng.uniform(-1, 2)))
    if mode in (1, 3):
        kw["lm"] = oracle.LM(W.random_small_lm(rng, int(rng.integers(1, 5)), V, density=0.5))
        kw["alpha"] = float(rng.uniform(0.1, 1.0))
    if mode in (2, 3):
        off, toks = _phrases(V, rng, int(rng.integers(1, 6)))
        kw["bt"] = oracle.BT(V, off, toks)
        kw["boost_w"] = float(rng.uniform(0.2, 2.0))
    y, s = greedy_fused(D, T, V, **kw)
    out = oracle.decode(D[None], np.array([T]), 1, kw.get("alpha", 0.0), kw["beta"],
                        kw.get("boost_w", 0.0), lm=kw.get("lm"), bt=kw.get("bt"))
    assert out["scores"][0] == s
    assert out["tokens"][0, : out["lengths"][0]].tolist() == y


def test_greedy_fused_is_a_lower_bound_of_the_exhaustive_search():
    """The greedy path is one alignment, so its score never exceeds the best
    over all alignments; with one dominant label per frame they agree."""
    rng = np.random.default_rng(9)
    V, T = 2, 5
    lm = oracle.LM(W.random_small_lm(rng, 3, V, density=0.5))
    for _ in range(6):
        D = W.random_logprobs(rng, 1, T, V, scale=2.0)[0]
        y, s = greedy_fused(D, T, V, alpha=0.5, beta=0.3, lm=lm)
        best, _ = brute_force(D, V, alpha=0.5, beta=0.3, lm=lm)
        assert s <= best
        Dp = np.full_like(D, -30.0)
        lab = rng.integers(0, V + 1, size=T)
        Dp[np.arange(T), lab] = -0.01
        y, s = greedy_fused(Dp, T, V, alpha=0.5, beta=0.3, lm=lm)
        best, arg = brute_force(Dp, V, alpha=0.5, beta=0.3, lm=lm)
        assert s == best and tuple(y) in arg


def test_greedy_fused_dead_frame_and_empty():
    rng = np.random.default_rng(4)
    V, T = 4, 6
    D = W.random_logprobs(rng, 2, T, V)
    D[1, 3, :] = -np.inf
    lm = oracle.LM(W.random_small_lm(rng, 2, V))
    out = oracle.decode(D, np.array([0, T]), 1, 0.5, 0.2, lm=lm)
    y0, s0 = greedy_fused(D[0], 0, V, alpha=0.5, beta=0.2, lm=lm)
    assert y0 == [] and out["scores"][0] == s0 and out["lengths"][0] == 0
    y1, s1 = greedy_fused(D[1], T, V, alpha=0.5, beta=0.2, lm=lm)
    assert y1 == [] and s1 == -np.inf
    assert out["scores"][1] == -np.inf and out["lengths"][1] == 0
