"""Invariants of the oracle's beam search (Algorithm 1 update/recombination):

* after every frame: no two live slots share (collapsed transcript,
  ends-in-blank); live scores do not increase with the slot index; each
  survivor is the lowest index of its group (RecombineHypotheses);
* self-consistency: re-scoring the returned alignment reproduces the returned
  score bit for bit, and collapsing it gives the returned tokens;
* invariances: batch permutation, NaN in padded frames, alpha = 0 with an LM
  equals no LM, an empty phrase list equals no boosting.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import collapse, fold_alignment, transcripts_from_trace


def _small_setup(seed=0, V=12, T=30, B=3, K=6):
    rng = np.random.default_rng(seed)
    D = W.random_logprobs(rng, B, T, V, scale=1.5)
    lens = np.array([T, T - 7, T // 2][:B])
    lm = oracle.LM(W.random_small_lm(rng, 3, V, density=0.2))
    lens_p = rng.integers(1, 4, size=5)
    off = np.concatenate([[0], np.cumsum(lens_p)])
    toks = rng.integers(0, V, size=int(lens_p.sum()))
    bt = oracle.BT(V, off, toks)
    return D, lens, lm, bt, K


@pytest.mark.parametrize("use_lm,use_bt", [(False, False), (True, False), (True, True)])
def test_dedup_invariants(use_lm, use_bt):
    D, lens, lm, bt, K = _small_setup()
    W_ = D.shape[2]
    out = oracle.decode(D, lens, K, alpha=0.4, beta=0.6, boost_w=1.1,
                        lm=lm if use_lm else None, bt=bt if use_bt else None, want_trace=True)
    for b in range(D.shape[0]):
        for t in range(lens[b]):
            sc = out["slot_scores"][b, t]
            keys = transcripts_from_trace(out["bp_index"][b], W_, t, K)
            live = [j for j in range(K) if np.isfinite(sc[j])]
            seen = {}
            for j in live:
                y, last = keys[j]
                key = (y, last == W_ - 1)
                assert key not in seen, (b, t, j)
                seen[key] = j
            for a_, c_ in zip(live, live[1:]):
                assert sc[a_] >= sc[c_]
            # every dead slot whose key matches a live one lost to a lower index
            assert live == sorted(live)


@pytest.mark.parametrize("use_lm,use_bt", [(False, False), (True, False), (True, True), (False, True)])
def test_self_consistency(use_lm, use_bt):
    D, lens, lm, bt, K = _small_setup(seed=1)
    kw = dict(alpha=0.4, beta=0.6, boost_w=1.1)
    out = oracle.decode(D, lens, K, lm=lm if use_lm else None, bt=bt if use_bt else None,
                        want_align=True, **kw)
    V = D.shape[2] - 1
    for b in range(D.shape[0]):
        al = out["align"][b, : lens[b]]
        assert (out["align"][b, lens[b]:] == -1).all()
        s, y = fold_alignment(D[b], al, V, lm=lm if use_lm else None,
                              bt=bt if use_bt else None, **kw)
        assert s == out["scores"][b]
        assert y == collapse(al, V) == out["tokens"][b, : out["lengths"][b]].tolist()


def test_batch_permutation_and_padding_nan():
    D, lens, lm, bt, K = _small_setup(seed=2)
    kw = dict(alpha=0.4, beta=0.6, boost_w=1.1, lm=lm, bt=bt)
    ref = oracle.decode(D, lens, K, **kw)
    perm = np.array([2, 0, 1])
    out = oracle.decode(D[perm], lens[perm], K, **kw)
    np.testing.assert_array_equal(out["tokens"], ref["tokens"][perm])
    np.testing.assert_array_equal(out["scores"], ref["scores"][perm])
    Dn = D.copy()
    for b in range(D.shape[0]):
        Dn[b, lens[b]:] = np.nan
    out = oracle.decode(Dn, lens, K, **kw)
    np.testing.assert_array_equal(out["tokens"], ref["tokens"])
    np.testing.assert_array_equal(out["scores"], ref["scores"])


def test_alpha_zero_equals_no_lm():
    D, lens, lm, bt, K = _small_setup(seed=3)
    a = oracle.decode(D, lens, K, alpha=0.0, beta=0.3, lm=lm)
    b = oracle.decode(D, lens, K, beta=0.3)
    np.testing.assert_array_equal(a["tokens"], b["tokens"])
    np.testing.assert_array_equal(a["scores"], b["scores"])


def test_empty_phrase_list_equals_no_boosting():
    D, lens, lm, bt, K = _small_setup(seed=4)
    V = D.shape[2] - 1
    empty = oracle.BT(V, np.zeros(1, np.int32), np.zeros(0, np.int32))
    a = oracle.decode(D, lens, K, beta=0.3, boost_w=2.0, bt=empty)
    b = oracle.decode(D, lens, K, beta=0.3)
    np.testing.assert_array_equal(a["tokens"], b["tokens"])
    np.testing.assert_array_equal(a["scores"], b["scores"])


def test_counters_are_consistent():
    """Instrumentation used by the byte model: frames, live beams, LM chain
    states/arcs, boosting chain nodes/arcs, emitting winners."""
    D, lens, lm, bt, K = _small_setup(seed=5)
    out = oracle.decode(D, lens, K, alpha=0.4, beta=0.6, boost_w=1.1, lm=lm, bt=bt,
                        want_counters=True)
    c = out["counters"]
    np.testing.assert_array_equal(c[:, 0], lens)
    assert (c[:, 1] >= c[:, 0]).all() and (c[:, 1] <= K * c[:, 0]).all()
    assert (c[:, 2] >= c[:, 1]).all()   # the unigram-context level always exists
    assert (c[:, 6] <= K * c[:, 0]).all()
