"""GPU parity of fill groups: with beams over one chunk (K above 16 / labels
per lane) and no row cache, beams in the same LM state read one LM row and
beams with the same boosting list one boosting row, filled once for a group
of consecutive chunks.  Sharing changes which rows are filled, never a score,
so the results must equal the CPU oracle's (tokens bit-exact, scores within
1e-4).

* 5- and 6-gram LMs of a few thousand n-grams (most hypotheses back off to
  short, shared states) with K = 9..128 (one and two beam slots per lane),
  vocabularies of 300, 400, 1024, 1500 and 3000 tokens (one, two, four and
  eight labels per lane), with and without boosting, theta = inf and 12,
  1-best and N-best.  At 3000 tokens a group holds one boosting list, so an
  LM state whose beams hold several lists is split over groups list by list;
* log-sum-exp recombination and repeat scoring on the same path;
* a witness that the final beams do share LM states (the longest suffix of
  <s> + tokens that is an n-gram of the model), so that shared rows are what
  these cases run.
"""
import math

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import compare, device, handles, log, oracle_bt, oracle_lm, oracle_threads

pytestmark = pytest.mark.gpu


def _workload(order, V, K, boost, seed):
    counts = tuple([min(3 * V, (V + 1) ** 2)] + [2 * V] * (order - 2))
    # above 2048 tokens a group holds one list: many Zipf phrases put the
    # beams of one LM state in several boosting states
    spec = W.BoostSpec(5000, 2, 4, "zipf", seed + 2) if V > 2048 else W.BoostSpec(300, 2, 5, "uniform", seed + 2)
    return W.CONFIGS[6].replace(
        B=3, T=90, V=V, K=K, lengths=("uniform", 40, 90), seed=seed,
        lm=W.LMSpec(order=order, counts=counts, seed=seed + 1),
        boost=spec if boost else None,
        boost_w=1.5 if boost else 0.0)


def _run(lp, lens, K, w, lm, bt, theta, nbest=False, **kw):
    import torch
    dev = device()
    d_lp = torch.from_numpy(np.ascontiguousarray(lp)).to(dev)
    d_len = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    f = P.ctcbeam_decode_nbest if nbest else P.ctcbeam_decode_ex
    tok, ln, sc, ws = f(d_lp, d_len, K, w.alpha, w.beta, w.boost_w, lm, bt, theta=theta, **kw)
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


def _lm_state(entries, order, bos, toks):
    """Longest suffix of <s> + toks, at most order-1 long, that is an n-gram."""
    y = (bos,) + tuple(int(t) for t in toks)
    for L in range(min(order - 1, len(y)), 0, -1):
        if y[-L:] in entries[L - 1]:
            return y[-L:]
    return ()


@pytest.mark.parametrize("order,V,K,boost", [
    (5, 1024, 16, False), (5, 1024, 64, True), (6, 1024, 40, True), (6, 1024, 64, False),
    (6, 1024, 9, True), (6, 300, 33, True), (5, 1500, 64, False), (5, 1500, 24, True),
    (6, 1024, 100, True), (5, 1024, 128, False), (6, 400, 77, True),
    (5, 3000, 24, True), (5, 3000, 64, True)])
def test_shared_rows(order, V, K, boost):
    w = _workload(order, V, K, boost, 31000 + 97 * order + K)
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    for th in (math.inf, 12.0):
        log(f"shared rows order={order} V={V} K={K} boost={boost} theta={th}")
        r = oracle.decode(lp, lens, K, w.alpha, w.beta, w.boost_w, theta=th, lm=olm, bt=obt,
                          n_threads=oracle_threads(), want_nbest=True)
        g = _run(lp, lens, K, w, lm, bt, th)
        assert g["status"] == 0
        compare(g, r, what=f"order={order} V={V} K={K} boost={boost} theta={th}")
        gn = _run(lp, lens, K, w, lm, bt, th, nbest=True)
        _compare_nbest(gn, r, what=f"nbest order={order} V={V} K={K} theta={th}")


@pytest.mark.parametrize("seed", range(3))
def test_shared_rows_random_logits(seed):
    # flat logits keep many distinct hypotheses alive
    rng = np.random.default_rng(32000 + seed)
    V = int(rng.choice([200, 700, 1024]))
    order = int(rng.integers(5, 8 if V <= 500 else 7))  # LM ids need (V+2)^order < 2^62
    K = int(rng.integers(9, 129))
    w = _workload(order, V, K, bool(rng.random() < 0.5), 32100 + seed)
    lm, bt, olm, obt = handles(w)
    B, T = 2, int(rng.integers(20, 70))
    lens = rng.integers(0, T + 1, size=B)
    lens[0] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 2.5)))
    lse = bool(rng.random() < 0.5)
    log(f"shared rows fuzz {seed}: order={order} V={V} K={K} T={T} lse={lse}")
    r = oracle.decode(lp, lens, K, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                      n_threads=oracle_threads(), want_nbest=True, logsumexp=lse)
    gn = _run(lp, lens, K, w, lm, bt, math.inf, nbest=True, logsumexp=lse)
    assert gn["status"] == 0
    _compare_nbest(gn, r, what=f"fuzz {seed}")


@pytest.mark.parametrize("boost", [False, True])
def test_shared_rows_repeat_score(boost):
    w = _workload(6, 1024, 32, boost, 33000 + int(boost))
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log(f"shared rows repeat scoring boost={boost}")
    r = oracle.decode(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                      n_threads=oracle_threads(), want_nbest=True, repeat_score=True)
    g = _run(lp, lens, w.K, w, lm, bt, math.inf, repeat_score=True)
    compare(g, r, what=f"repeat boost={boost}")
    gn = _run(lp, lens, w.K, w, lm, bt, math.inf, nbest=True, repeat_score=True)
    _compare_nbest(gn, r, what=f"repeat nbest boost={boost}")


def test_final_beams_share_lm_states():
    w = _workload(6, 1024, 64, False, 34000)
    lm, _, olm, _ = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    gn = _run(lp, lens, w.K, w, lm, None, math.inf, nbest=True)
    arrays = W.lm_for(w.lm, w.V)
    entries = [set(map(tuple, ids.tolist())) for ids in arrays["ids"][: w.lm.order - 1]]
    shared = 0
    for b in range(w.B):
        live = [r for r in range(w.K) if gn["scores"][b, r] != -np.inf]
        states = {_lm_state(entries, w.lm.order, w.V + 1, gn["tokens"][b, r, : gn["lengths"][b, r]])
                  for r in live}
        log(f"utterance {b}: {len(live)} beams, {len(states)} LM states")
        shared += len(live) - len(states)
    assert shared > 0
    r = oracle.decode(lp, lens, w.K, w.alpha, w.beta, 0.0, lm=olm, n_threads=oracle_threads(),
                      want_nbest=True)
    _compare_nbest(gn, r, what="witness workload")


def test_wide_vocabulary_splits_states_over_groups():
    # Witness for the (5, 3000, 64, boosting) case above: in some frames of
    # the oracle's search the live beams of one LM state sit in two boosting
    # states, more than a group holds at 3000 tokens (one list), so the plan
    # splits that state over groups list by list.
    import collections
    order, V, K = 5, 3000, 64
    w = _workload(order, V, K, True, 31000 + 97 * order + K)
    olm, obt = oracle_lm(w.lm, w.V), oracle_bt(w.boost, w.V)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    r = oracle.decode(lp, lens, K, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                      n_threads=oracle_threads(), want_trace=True)
    arrays = W.lm_for(w.lm, w.V)
    entries = [set(map(tuple, ids.tolist())) for ids in arrays["ids"][: order - 1]]
    bp, ss, Wd = r["bp_index"], r["slot_scores"], V + 1
    split = 0
    for b in range(w.B):
        ys = [[] for _ in range(K)]
        last = [V] * K
        for t in range(int(lens[b])):
            nys, nlast = [], []
            for j in range(K):
                p, c = divmod(int(bp[b, t, j]), Wd)
                y = list(ys[p])
                if c != V and c != last[p]:
                    y.append(c)
                nys.append(y)
                nlast.append(c)
            ys, last = nys, nlast
            by_state = collections.defaultdict(set)
            for j in range(K):
                if np.isfinite(ss[b, t, j]):
                    q = tuple(obt.run(ys[j])[1])
                    if q:
                        by_state[_lm_state(entries, order, V + 1, ys[j])].add(q)
            split += any(len(v) >= 2 for v in by_state.values())
    log(f"frames with an LM state in two boosting states: {split}")
    assert split > 0
