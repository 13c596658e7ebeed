"""Pins of the oracle's threshold pruning and of its byte-model counters.

Pruning (Algorithm 1, threshold pruning: a kept candidate scoring below the
frame's best minus theta becomes -inf; theta = 12 in Sec. IV-D):

* two-sided, per slot: every slot's pre-prune candidate score is recomputed
  from the trace with the fp32 fold of Eq. 1 written out here (the parent's
  score, its transcript's LM score and boosting step), and the slot must be
  dead exactly when that score is below fl(x0 - theta) or when it loses the
  recombination to a live lower slot, and otherwise hold that score;
* theta = 0 on tie-free inputs leaves one live hypothesis per frame, which is
  the K = 1 search (itself pinned against a separate sequential search);
* theta above every frame's score spread prunes nothing: equal to theta = inf.

Counters (the roofline's byte model): hand-counted values for one short
decode on the toy ARPA model (tests/golden/toy3_counters.json), and a
recount from the trace with continuation counts taken straight from the
n-gram arrays.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads as W
from oracle_helpers import F32, NEG_INF, transcripts_from_trace

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _setup(seed, V=10, T=24, B=3, K=6, with_bt=True):
    rng = np.random.default_rng(seed)
    D = W.random_logprobs(rng, B, T, V, scale=1.5)
    lens = np.array([T, T - 5, T // 2][:B])
    lm = oracle.LM(W.random_small_lm(rng, 3, V, density=0.3))
    bt = None
    if with_bt:
        lens_p = rng.integers(1, 4, size=6)
        off = np.concatenate([[0], np.cumsum(lens_p)])
        toks = rng.integers(0, V, size=int(lens_p.sum()))
        bt = oracle.BT(V, off, toks)
    return D, lens, lm, bt, K


def _pre_prune_scores(D, out, b, t, K, kw, lm, bt):
    """Candidate score of every slot at frame t before pruning, from the
    parent's slot score after frame t-1: x = s + D[c]; for an emitting label
    x += beta, += fl(alpha * LM), += fl(w * BT) (Eq. 1, Alg. 1 line order)."""
    Wl = D.shape[2]
    V = Wl - 1
    if t == 0:
        prev = [F32(0.0)] + [NEG_INF] * (K - 1)
        keys = [((), V)] * K
    else:
        prev = [F32(v) for v in out["slot_scores"][b, t - 1]]
        keys = transcripts_from_trace(out["bp_index"][b], Wl, t - 1, K)
    xs = []
    for j in range(K):
        i = int(out["bp_index"][b, t, j])
        p, c = i // Wl, i % Wl
        s = prev[p]
        y, last = keys[p]
        x = F32(s + F32(D[b, t, c]))
        if c != V and c != last and s != NEG_INF:
            x = F32(x + F32(kw["beta"]))
            if lm is not None:
                x = F32(x + F32(F32(kw["alpha"]) * F32(lm.score(list(y), c))))
            if bt is not None:
                _, q = bt.run(list(y))
                sc, _ = bt.step(q, c)
                x = F32(x + F32(F32(kw["boost_w"]) * F32(sc)))
        xs.append(x)
    return xs


@pytest.mark.parametrize("theta", [0.75, 1.5, 3.0])
@pytest.mark.parametrize("with_bt", [False, True])
def test_prune_two_sided_per_slot(theta, with_bt):
    D, lens, lm, bt, K = _setup(seed=11 + int(theta * 4), with_bt=with_bt)
    kw = dict(alpha=0.45, beta=0.8, boost_w=1.2 if with_bt else 0.0)
    out = oracle.decode(D, lens, K, theta=theta, lm=lm, bt=bt, want_trace=True, **kw)
    Wl = D.shape[2]
    V = Wl - 1
    th = F32(theta)
    n_pruned = n_window = 0
    for b in range(D.shape[0]):
        for t in range(lens[b]):
            xs = _pre_prune_scores(D, out, b, t, K, kw, lm, bt)
            lim = F32(xs[0] - th)
            keys = transcripts_from_trace(out["bp_index"][b], Wl, t, K)
            live = []
            for j in range(K):
                x = xs[j]
                if x != NEG_INF and x < lim:
                    n_pruned += 1
                    want = NEG_INF
                elif x == NEG_INF:
                    want = NEG_INF
                else:
                    y, last = keys[j]
                    key = (y, last == V)
                    if any(k == key for k in live):
                        want = NEG_INF  # recombination loser
                    else:
                        live.append(key)
                        want = x
                        if j > 0 and x < F32(xs[0] - F32(th * F32(0.5))):
                            n_window += 1  # kept, though below best - theta/2
                got = F32(out["slot_scores"][b, t, j])
                assert (got == want) or (np.isnan(got) and np.isnan(want)), (b, t, j, got, want)
    # the inputs exercise both sides of the threshold
    assert n_pruned > 0
    assert n_window > 0


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_theta_zero_is_single_hypothesis(seed):
    """theta = 0: every slot but the best scores below it (no ties), so only
    one hypothesis lives and the search is the K = 1 search."""
    D, lens, lm, bt, _ = _setup(seed=seed)
    kw = dict(alpha=0.45, beta=0.8, boost_w=1.2, lm=lm, bt=bt)
    a = oracle.decode(D, lens, 6, theta=0.0, want_trace=True, **kw)
    b = oracle.decode(D, lens, 1, **kw)
    np.testing.assert_array_equal(a["tokens"], b["tokens"])
    np.testing.assert_array_equal(a["lengths"], b["lengths"])
    np.testing.assert_array_equal(a["scores"], b["scores"])
    for bb in range(D.shape[0]):
        for t in range(lens[bb]):
            assert np.isfinite(a["slot_scores"][bb, t, 0])
            assert not np.isfinite(a["slot_scores"][bb, t, 1:]).any()


def test_theta_above_spread_prunes_nothing():
    D, lens, lm, bt, K = _setup(seed=21)
    kw = dict(alpha=0.45, beta=0.8, boost_w=1.2)
    ref = oracle.decode(D, lens, K, lm=lm, bt=bt, want_trace=True, **kw)
    spread = 0.0
    for b in range(D.shape[0]):
        for t in range(lens[b]):
            xs = [x for x in _pre_prune_scores(D, ref, b, t, K, kw, lm, bt) if x != NEG_INF]
            spread = max(spread, float(xs[0] - min(xs)))
    above = oracle.decode(D, lens, K, theta=spread * 1.01 + 1e-3, lm=lm, bt=bt, want_trace=True, **kw)
    for k in ("tokens", "lengths", "scores", "bp_index", "slot_scores"):
        np.testing.assert_array_equal(above[k], ref[k])
    # and a threshold inside the spread does prune
    inside = oracle.decode(D, lens, K, theta=spread * 0.5, lm=lm, bt=bt, want_trace=True, **kw)
    assert not np.array_equal(inside["slot_scores"], ref["slot_scores"])


def _toy_golden():
    g = json.load(open(os.path.join(GOLD, "toy3_counters.json")))
    lm = oracle.LM(W.read_arpa(os.path.join(GOLD, "toy3.arpa"), V=3))
    ph = [[0, 1, 2], [1, 2]]
    off = np.array([0, 3, 5], np.int32)
    bt = oracle.BT(3, off, np.array(sum(ph, []), np.int32))
    D = np.array(g["logprob_rows"], np.float32)[None]
    return g, lm, bt, D


def test_counters_hand_counted_toy():
    g, lm, bt, D = _toy_golden()
    out = oracle.decode(D, np.array([4]), 2, alpha=0.5, beta=0.0, boost_w=1.0, lm=lm, bt=bt,
                        want_counters=True)
    e = g["expected_counters"]
    c = out["counters"][0]
    names = ["frames", "alive_beam_frames", "lm_states", "lm_arcs", "bt_nodes", "bt_arcs",
             "emitting_winners"]
    assert {n: int(c[i]) for i, n in enumerate(names)} == e
    assert out["tokens"][0, : out["lengths"][0]].tolist() == g["expected_tokens"]
    assert abs(float(out["scores"][0]) - g["expected_score_approx"]) < 2e-3


def test_counters_recount_from_trace():
    """LM chain states / arcs recounted per alive slot from the trace, with
    each context's explicit continuations counted from the n-gram arrays."""
    rng = np.random.default_rng(31)
    V, T, K = 9, 20, 5
    arrays = W.random_small_lm(rng, 3, V, density=0.35)
    lm = oracle.LM(arrays)
    entries = set()
    n_cont = {}
    for m, ids in enumerate(arrays["ids"], start=1):
        for g in np.asarray(ids).reshape(-1, m).tolist():
            entries.add(tuple(g))
            if m >= 2:
                n_cont[tuple(g[:-1])] = n_cont.get(tuple(g[:-1]), 0) + 1
    D = W.random_logprobs(rng, 2, T, V, scale=1.5)
    lens = np.array([T, 13])
    kw = dict(alpha=0.5, beta=0.4)
    out = oracle.decode(D, lens, K, lm=lm, want_trace=True, want_counters=True, **kw)
    Wl = V + 1
    for b in range(2):
        states = arcs = alive = emits = 0
        for t in range(lens[b]):
            if t == 0:
                prev_keys, prev_s = [((), V)], [0.0]
            else:
                prev_keys = transcripts_from_trace(out["bp_index"][b], Wl, t - 1, K)
                prev_s = out["slot_scores"][b, t - 1]
            for (y, _), s in zip(prev_keys, prev_s):
                if not np.isfinite(s):
                    continue
                alive += 1
                hist = (V + 1,) + tuple(y)
                ctx = hist[-min(2, len(hist)):]
                for ln_ in range(1, len(ctx) + 1):
                    suf = ctx[-ln_:]
                    if suf in entries:
                        states += 1
                        arcs += n_cont.get(suf, 0)
            for j in range(K):
                i = int(out["bp_index"][b, t, j])
                p, c = i // Wl, i % Wl
                # an emitting winner counts when its score is finite (theta =
                # inf: the parent is alive; recombination does not undo it)
                if c != V and c != prev_keys[p][1] and np.isfinite(prev_s[p]):
                    emits += 1
        cnt = out["counters"][b]
        assert (int(cnt[0]), int(cnt[1]), int(cnt[2]), int(cnt[3])) == (lens[b], alive, states, arcs)
        assert int(cnt[6]) == emits
