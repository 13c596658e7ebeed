"""Pins of the oracle's repeat-scoring variant (flag bit 2): a frame that
repeats the beam's last frame label (a token, Sec. III-C's alternative of
scoring repeated emissions at every occurrence) adds again the fl(alpha*LM)
and fl(w*BT) terms the token received when it was emitted; no beta, no state
change.

* exhaustive (K >= (V+1)^T, no pruning): every live N-best row's score equals
  the best fp32 fold over all alignments of its recombination key, each
  alignment folded by ``fold_alignment(..., repeat=True)`` (a per-alignment
  re-scoring written apart from the search), bit for bit; the repeat terms
  depend only on the transcript, so max-merge recombination stays exact;
* without an LM and boosting the flag changes nothing (there are no terms to
  repeat);
* with an LM the flag changes the scores of hypotheses that hold a token over
  several frames, and only of those.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import brute_force_keys, fold_alignment

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _phrases(V, rng, n=3):
    lens = rng.integers(1, 4, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    off = np.concatenate([[0], np.cumsum(lens)])
    return off, toks


CASES = [(V, T) for V in (1, 2, 3) for T in (2, 3, 4, 5) if (V + 1) ** T <= 256]


def _setup(mode, V, rng):
    kw = dict(beta=0.7)
    lm = bt = None
    if mode in ("lm", "lm_bt"):
        lm = oracle.LM(W.random_small_lm(rng, 3, V, density=0.5))
        kw.update(alpha=0.6, lm=lm)
    if mode in ("bt", "lm_bt"):
        off, toks = _phrases(V, rng)
        bt = oracle.BT(V, off, toks)
        kw.update(boost_w=1.3, bt=bt)
    return kw, lm, bt


@pytest.mark.parametrize("V,T", CASES)
@pytest.mark.parametrize("mode", ["lm", "bt", "lm_bt"])
def test_repeat_score_exhaustive_nbest(V, T, mode):
    rng = np.random.default_rng(5000 + 100 * V + 10 * T + len(mode))
    for _ in range(2):
        D = W.random_logprobs(rng, 1, T, V, scale=1.5)[0]
        kw, lm, bt = _setup(mode, V, rng)
        keys = brute_force_keys(D, V, repeat=True, **kw)
        K = (V + 1) ** T
        out = oracle.decode(D[None], np.array([T]), K, alpha=kw.get("alpha", 0.0),
                            beta=kw["beta"], boost_w=kw.get("boost_w", 0.0), lm=lm, bt=bt,
                            want_nbest=True, repeat_score=True)
        sc, ln, tk = out["nbest_scores"][0], out["nbest_lengths"][0], out["nbest_tokens"][0]
        live = int(np.sum(sc != -np.inf))
        assert live == len(keys)
        got = sorted(((float(sc[r]), tuple(tk[r, : ln[r]].tolist())) for r in range(live)),
                     key=lambda e: (-e[0], e[1]))
        want = sorted(((float(s), k[0]) for k, s in keys.items()), key=lambda e: (-e[0], e[1]))
        assert got == want
        # the 1-best is the best of them
        assert out["scores"][0] == max(s for s, _ in want)


def test_repeat_score_without_fusion_changes_nothing():
    rng = np.random.default_rng(5100)
    D = W.random_logprobs(rng, 4, 40, 6, scale=2.0)
    lens = np.array([40, 33, 1, 0])
    a = oracle.decode(D, lens, 4, beta=0.4, want_nbest=True)
    b = oracle.decode(D, lens, 4, beta=0.4, want_nbest=True, repeat_score=True)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])


def test_repeat_terms_apply_to_held_tokens_only():
    """Re-scoring single alignments: the flag adds the emitted token's terms
    once per extra frame it is held, and nothing to an alignment whose
    tokens are separated by blanks."""
    rng = np.random.default_rng(5200)
    V = 3
    lm = oracle.LM(W.random_small_lm(rng, 3, V, density=0.5))
    D = W.random_logprobs(rng, 1, 6, V, scale=1.5)[0]
    kw = dict(alpha=0.6, beta=0.7, lm=lm)
    spaced = [0, V, 1, V, 2, V]
    assert fold_alignment(D, spaced, V, repeat=True, **kw) == fold_alignment(D, spaced, V, **kw)
    held = [0, 0, 0, 1, 1, V]
    s1, y1 = fold_alignment(D, held, V, repeat=True, **kw)
    s0, y0 = fold_alignment(D, held, V, **kw)
    assert y1 == y0 == [0, 1]
    assert s1 != s0
    # the 1-best of the search with the flag differs from the default search
    # somewhere on a random batch with an LM
    D = W.random_logprobs(rng, 8, 30, V, scale=1.0)
    lens = np.full(8, 30)
    a = oracle.decode(D, lens, 4, 0.6, 0.7, lm=lm, want_nbest=True)
    b = oracle.decode(D, lens, 4, 0.6, 0.7, lm=lm, want_nbest=True, repeat_score=True)
    assert np.any(a["nbest_scores"] != b["nbest_scores"])
