"""Pins of the oracle's n-gram LM (backoff evaluation, Sec. II "NGPU-LM";
ARPA input, Sec. IV-A).

* hand-worked values on a toy 3-gram ARPA file (tests/golden);
* normalisation: for a backoff model whose weights are set so that every
  context's distribution sums to one, sum_c P(c|h) = 1 for every history,
  seen or unseen - a dropped or misplaced backoff term breaks this;
* fp32 fold order: the value equals the innermost-first fp32 sum of the
  converted entries along the backoff path;
* the order of the input arrays does not matter.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")
LN10 = np.log(10.0)


def test_toy_arpa_hand_values():
    lm_arrays = W.read_arpa(os.path.join(GOLD, "toy3.arpa"), V=3)
    lm = oracle.LM(lm_arrays)
    exp = json.load(open(os.path.join(GOLD, "toy3_expected.json")))
    for case in exp["cases"]:
        got = lm.score(case["y"], case["c"])
        assert abs(got - case["log10"] * LN10) < 1e-5, case


def _normalised_lm(rng, V, order):
    """Random backoff LM with backoff weights chosen so each context's
    distribution over tokens + </s> sums to one (worked in float64)."""
    EOS, BOS = V, V + 1
    n_cont = V + 1
    p1 = rng.dirichlet(np.ones(n_cont))
    ids = [np.arange(V + 2)[:, None]]
    logp = [np.concatenate([np.log10(p1), [-99.0]])]
    prob = {(i,): p1[i] for i in range(n_cont)}

    def P(h, w):  # float64 reference for building the weights only
        h = tuple(h)
        while True:
            if h + (w,) in prob:
                return prob[h + (w,)]
            if not h:
                raise KeyError
            b = bow.get(h, 1.0)
            return b * P(h[1:], w)

    bow = {}
    for m in range(2, order + 1):
        prev = [tuple(r) for r in ids[-1].tolist() if r[-1] != EOS]
        rows, vals = [], []
        for h in prev:
            k = rng.integers(1, n_cont)  # explicit continuations of h
            ws = rng.choice(n_cont, size=k, replace=False)
            if m > 2:  # keep suffix closure
                ws = [w for w in ws if h[1:] + (w,) in prob]
                if not ws:
                    continue
            mass = rng.uniform(0.3, 0.9)
            share = rng.dirichlet(np.ones(len(ws))) * mass
            for w, s in zip(ws, share):
                rows.append(h + (int(w),))
                vals.append(s)
        for r, v in zip(rows, vals):
            prob[r] = v
        # backoff weights of the contexts h (entries of order m-1)
        for h in prev:
            seen = [r for r in rows if r[:-1] == h]
            m_h = sum(prob[r] for r in seen)
            lower = sum(P(h[1:], r[-1]) for r in seen)
            bow[h] = (1.0 - m_h) / (1.0 - lower)
        arr = np.asarray(rows, dtype=np.int32).reshape(-1, m)
        order_idx = np.lexsort(arr.T[::-1]) if len(arr) else np.zeros(0, int)
        ids.append(arr[order_idx])
        logp.append(np.log10(np.asarray(vals))[order_idx])
    bows = []
    for m in range(1, order):
        bows.append(np.asarray([np.log10(bow.get(tuple(r), 1.0)) for r in ids[m - 1].tolist()],
                               dtype=np.float32))
    bows[0][EOS] = 0.0
    return dict(order=order, V=V, ids=[np.asarray(a, dtype=np.int32) for a in ids],
                log10_prob=[np.asarray(a, dtype=np.float32) for a in logp],
                log10_bow=bows + [None])


@pytest.mark.parametrize("order", [2, 3, 4])
def test_normalisation(order):
    rng = np.random.default_rng(40 + order)
    V = 5
    lm = oracle.LM(_normalised_lm(rng, V, order))
    for _ in range(60):
        y = rng.integers(0, V, size=rng.integers(0, 7)).tolist()
        tot = sum(np.exp(np.float64(lm.score(y, c))) for c in range(V + 1))
        assert abs(tot - 1.0) < 2e-5, (y, tot)


def test_fold_order_is_innermost_first():
    """P(c | a b) for a model where c is only a unigram: the fp32 value must be
    ((p(c) + bo(b)) + bo(a b)) with every entry converted on its own."""
    V = 3
    lm_arrays = dict(order=3, V=V,
                     ids=[np.arange(V + 2, dtype=np.int32)[:, None],
                          np.array([[0, 1]], dtype=np.int32),
                          np.array([[0, 1, 0]], dtype=np.int32)],
                     log10_prob=[np.array([-0.7, -0.31, -1.13, -0.9, -99], dtype=np.float32),
                                 np.array([-0.123], dtype=np.float32),
                                 np.array([-0.05], dtype=np.float32)],
                     log10_bow=[np.array([-0.3, -0.77, -0.21, 0.0, -0.4], dtype=np.float32),
                                np.array([-0.61], dtype=np.float32), None])
    lm = oracle.LM(lm_arrays)

    def ln(v):
        return np.float32(np.float64(np.float32(v)) * np.float64(LN10))

    want = np.float32(np.float32(ln(-1.13) + ln(-0.77)) + ln(-0.61))
    assert np.float32(lm.backoff([0, 1], 2)) == want
    # history truncation: <s> 0 1 -> context (0, 1)
    assert np.float32(lm.score([0, 1], 2)) == want
    # a context that is no entry adds nothing: P(2 | 2 1) = p(2) + bo(1)
    assert np.float32(lm.backoff([2, 1], 2)) == np.float32(ln(-1.13) + ln(-0.77))
    # explicit trigram
    assert np.float32(lm.score([0, 1], 0)) == ln(-0.05)


def test_array_order_invariance():
    rng = np.random.default_rng(11)
    V = 6
    a = W.random_small_lm(rng, 3, V, density=0.4)
    b = dict(a)
    perm_ids, perm_p, perm_b = [], [], []
    for m in range(3):
        p = rng.permutation(a["ids"][m].shape[0])
        perm_ids.append(a["ids"][m][p])
        perm_p.append(a["log10_prob"][m][p])
        perm_b.append(None if a["log10_bow"][m] is None else a["log10_bow"][m][p])
    b.update(ids=perm_ids, log10_prob=perm_p, log10_bow=perm_b)
    la, lb = oracle.LM(a), oracle.LM(b)
    for _ in range(200):
        y = rng.integers(0, V, size=rng.integers(0, 5)).tolist()
        c = int(rng.integers(0, V + 1))
        assert la.score(y, c) == lb.score(y, c)


def test_arpa_roundtrip(tmp_path):
    rng = np.random.default_rng(12)
    V = 7
    a = W.random_small_lm(rng, 3, V, density=0.3)
    path = str(tmp_path / "m.arpa")
    W.write_arpa(a, path)
    b = W.read_arpa(path, V)
    la, lb = oracle.LM(a), oracle.LM(b)
    for _ in range(200):
        y = rng.integers(0, V, size=rng.integers(0, 5)).tolist()
        c = int(rng.integers(0, V + 1))
        assert la.score(y, c) == lb.score(y, c)
