"""Pins of the oracle's search (beam search steps of Algorithm 1).

* exhaustive: with K >= (V+1)^T and no pruning nothing is dropped, so the
  best score must equal the maximum over all alignments of the same fp32
  fold, bit for bit (max-merge recombination is exact Viterbi);
* greedy: K = 1 with alpha = beta = w = 0 is greedy CTC decoding.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import brute_force, greedy

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _phrases(V, rng, n=3):
    lens = rng.integers(1, 4, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    off = np.concatenate([[0], np.cumsum(lens)])
    return off, toks


CASES = []
for V in (1, 2, 3):
    for T in (1, 2, 3, 4, 5):
        if (V + 1) ** T > 1024:
            continue
        CASES.append((V, T))


@pytest.mark.parametrize("V,T", CASES)
@pytest.mark.parametrize("mode", ["plain", "beta", "lm", "bt", "lm_bt"])
def test_exhaustive_matches_brute_force(V, T, mode):
    rng = np.random.default_rng(100 * V + 10 * T + len(mode))
    D = W.random_logprobs(rng, 1, T, V, scale=1.5)[0]
    kw = {}
    lm = bt = None
    if mode in ("beta", "lm", "lm_bt"):
        kw["beta"] = 0.7
    if mode in ("lm", "lm_bt"):
        lm = oracle.LM(W.random_small_lm(rng, 3, V, density=0.5))
        kw["alpha"] = 0.6
        kw["lm"] = lm
    if mode in ("bt", "lm_bt"):
        off, toks = _phrases(V, rng)
        bt = oracle.BT(V, off, toks)
        kw["boost_w"] = 1.3
        kw["bt"] = bt
    best, arg = brute_force(D, V, **kw)
    K = (V + 1) ** T
    out = oracle.decode(D[None], np.array([T]), K, alpha=kw.get("alpha", 0.0),
                        beta=kw.get("beta", 0.0), boost_w=kw.get("boost_w", 0.0),
                        lm=lm, bt=bt)
    assert out["scores"][0] == best, (out["scores"][0], best)
    got = tuple(out["tokens"][0, : out["lengths"][0]].tolist())
    assert got in arg
    if len(arg) == 1:
        assert got == next(iter(arg))


def test_exhaustive_with_padding_and_batch():
    """Same pin with a batch of ragged lengths inside a padded tensor."""
    rng = np.random.default_rng(7)
    V, T = 2, 5
    D = W.random_logprobs(rng, 3, T, V, scale=2.0)
    lens = np.array([5, 3, 0])
    out = oracle.decode(D, lens, (V + 1) ** T, beta=0.4)
    for b in range(3):
        best, arg = brute_force(D[b, : lens[b]], V, beta=0.4)
        assert out["scores"][b] == best
        assert tuple(out["tokens"][b, : out["lengths"][b]].tolist()) in arg


@pytest.mark.parametrize("cfg", [1, 2])
def test_greedy_equivalence(cfg):
    w = W.CONFIGS[cfg]
    idx = list(range(min(w.B, 4)))
    D = W.make_logprobs(w, idx)
    lens = W.make_lengths(w)[idx]
    out = oracle.decode(D, lens, 1)
    for i, b in enumerate(idx):
        toks, s = greedy(D[i], lens[i], w.V)
        assert out["scores"][i] == s
        assert out["tokens"][i, : out["lengths"][i]].tolist() == toks
        assert (out["tokens"][i, out["lengths"][i]:] == -1).all()


def test_greedy_equivalence_with_ties():
    """Rows with exactly tied maxima: the lowest label wins (index order)."""
    rng = np.random.default_rng(3)
    V, T = 5, 40
    D = np.log(np.full((1, T, V + 1), 1.0 / (V + 1), dtype=np.float64)).astype(np.float32)
    # a few frames with a unique peak, the rest fully tied
    for t in rng.choice(T, size=10, replace=False):
        D[0, t, rng.integers(0, V + 1)] = -0.5
    out = oracle.decode(D, np.array([T]), 1)
    toks, s = greedy(D[0], T, V)
    assert out["scores"][0] == s
    assert out["tokens"][0, : out["lengths"][0]].tolist() == toks


def test_empty_utterance():
    """L = 0: empty transcript; score 0, or alpha * LM(</s> | <s>) with an LM."""
    rng = np.random.default_rng(5)
    V = 4
    D = W.random_logprobs(rng, 1, 3, V)
    out = oracle.decode(D, np.array([0]), 3)
    assert out["lengths"][0] == 0 and out["scores"][0] == 0.0
    lm = oracle.LM(W.random_small_lm(rng, 2, V))
    out = oracle.decode(D, np.array([0]), 3, alpha=0.5, lm=lm)
    assert out["scores"][0] == np.float32(np.float32(0.5) * np.float32(lm.score([], V)))


def test_all_minus_inf_frame_gives_empty_output():
    V, T = 3, 4
    D = np.zeros((1, T, V + 1), dtype=np.float32) - 1.0
    D[0, 2, :] = -np.inf
    out = oracle.decode(D, np.array([T]), 4, beta=0.5)
    assert out["scores"][0] == -np.inf and out["lengths"][0] == 0
    assert (out["tokens"][0] == -1).all()


def test_lengths_clamped():
    rng = np.random.default_rng(9)
    D = W.random_logprobs(rng, 2, 6, 3)
    a = oracle.decode(D, np.array([9, -2]), 4)
    b = oracle.decode(D, np.array([6, 0]), 4)
    np.testing.assert_array_equal(a["tokens"], b["tokens"])
    np.testing.assert_array_equal(a["scores"], b["scores"])


def test_theta_pruning_keeps_window():
    """After every frame each alive slot is within theta of the best one."""
    w = W.CONFIGS[1]
    D = W.make_logprobs(w)
    lens = W.make_lengths(w)
    out = oracle.decode(D, lens, 4, beta=0.5, theta=3.0, want_trace=True)
    ss = out["slot_scores"]
    for b in range(w.B):
        for t in range(lens[b]):
            row = ss[b, t]
            alive = row[np.isfinite(row)]
            assert len(alive) >= 1
            assert alive.min() >= np.float32(row[0] - np.float32(3.0))


def test_merge_key_includes_blank_flag():
    """Merging on the transcript alone loses the exact best path: with V = 1,
    beta = 1 and rows (a -1, _ -10), (a -1, _ -1.1), (a -1, _ -10) the best
    alignment is "a _ a" -> "a a" at -1.1; "a|a" and "a|_" share the
    transcript "a" after frame 1 but must not be merged."""
    D = np.array([[[-1.0, -10.0], [-1.0, -1.1], [-1.0, -10.0]]], dtype=np.float32)
    best, arg = brute_force(D[0], 1, beta=1.0)
    assert arg == {(0, 0)}
    out = oracle.decode(D, np.array([3]), 8, beta=1.0)
    assert out["scores"][0] == best
    assert out["tokens"][0, : out["lengths"][0]].tolist() == [0, 0]
