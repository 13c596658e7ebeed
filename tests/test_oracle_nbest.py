"""Pins of the oracle's N-best output (every slot's final hypothesis, the
batched-hypotheses result of Algorithm 1), an adjacent row of the hot path.

* exhaustive: with K >= (V+1)^T and no pruning nothing is dropped and every
  recombination key (collapsed transcript, ends-in-blank) keeps its best
  alignment, so the live N-best entries are exactly the keys' best folds over
  all alignments, in descending order of score;
* the first entry is the 1-best output; scores never increase down the list;
  dead slots come last, empty and at -inf.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import brute_force_keys

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _phrases(V, rng, n=3):
    lens = rng.integers(1, 4, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    off = np.concatenate([[0], np.cumsum(lens)])
    return off, toks


CASES = [(V, T) for V in (1, 2, 3) for T in (1, 2, 3, 4) if (V + 1) ** T <= 256]


@pytest.mark.parametrize("V,T", CASES)
@pytest.mark.parametrize("mode", ["plain", "beta", "lm", "bt", "lm_bt"])
def test_exhaustive_nbest_matches_brute_force(V, T, mode):
    rng = np.random.default_rng(1000 + 100 * V + 10 * T + len(mode))
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
    keys = brute_force_keys(D, V, **kw)
    K = (V + 1) ** T
    out = oracle.decode(D[None], np.array([T]), K, alpha=kw.get("alpha", 0.0),
                        beta=kw.get("beta", 0.0), boost_w=kw.get("boost_w", 0.0),
                        lm=lm, bt=bt, want_nbest=True)
    sc = out["nbest_scores"][0]
    ln = out["nbest_lengths"][0]
    tk = out["nbest_tokens"][0]
    live = int(np.sum(sc != -np.inf))
    assert live == len(keys)
    got = sorted(((float(sc[r]), tuple(tk[r, : ln[r]].tolist())) for r in range(live)),
                 key=lambda e: (-e[0], e[1]))
    want = sorted(((float(s), k[0]) for k, s in keys.items()), key=lambda e: (-e[0], e[1]))
    assert got == want
    assert np.all(np.diff(sc[:live]) <= 0)


def _check_structure(out, T):
    sc, ln, tk = out["nbest_scores"], out["nbest_lengths"], out["nbest_tokens"]
    B, K = sc.shape
    for b in range(B):
        live = sc[b] != -np.inf
        n = int(live.sum())
        assert np.all(live[:n]) and not np.any(live[n:])
        assert np.all(np.diff(sc[b, :n]) <= 0)
        assert np.all(ln[b, n:] == 0)
        for r in range(K):
            assert np.all(tk[b, r, ln[b, r]:] == -1)
            assert np.all(tk[b, r, : ln[b, r]] >= 0)
        # the first entry is the 1-best output
        assert sc[b, 0] == out["scores"][b] or (np.isneginf(sc[b, 0]) and np.isneginf(out["scores"][b]))
        assert ln[b, 0] == out["lengths"][b]
        assert np.array_equal(tk[b, 0], out["tokens"][b])


@pytest.mark.parametrize("cfg,theta", [(1, np.inf), (2, np.inf), (3, np.inf), (3, 12.0), (5, 12.0)])
def test_nbest_structure_and_first_entry(cfg, theta):
    w = W.CONFIGS[cfg]
    idx = list(range(min(w.B, 3)))
    lens = np.minimum(W.make_lengths(w)[idx], 60).astype(np.int32)
    D = np.ascontiguousarray(W.make_logprobs(w, idx)[:, :60])
    lm = oracle.LM(W.lm_for(w.lm, w.V)) if w.lm else None
    bt = None
    if w.boost:
        off, toks = W.phrases_for(w.boost, w.V)
        bt = oracle.BT(w.V, off, toks)
    out = oracle.decode(D, lens, w.K, w.alpha, w.beta, w.boost_w, theta=theta, lm=lm, bt=bt,
                        n_threads=3, want_nbest=True)
    _check_structure(out, D.shape[1])


def test_nbest_empty_and_dead():
    """L = 0 keeps only the initial beam; a -inf frame kills every slot."""
    rng = np.random.default_rng(5)
    V, T, K = 4, 6, 5
    D = W.random_logprobs(rng, 2, T, V)
    D[1, 2, :] = -np.inf
    out = oracle.decode(D, np.array([0, T]), K, beta=0.3, want_nbest=True)
    assert out["nbest_scores"][0, 0] == 0.0 and np.all(np.isneginf(out["nbest_scores"][0, 1:]))
    assert np.all(out["nbest_lengths"][0] == 0)
    assert np.all(np.isneginf(out["nbest_scores"][1]))
    _check_structure(out, T)
