"""Test-side helpers: independent reference computations used to pin the oracle.

Nothing here is imported by the decoder package.  The fold below re-scores a
single given alignment; the exhaustive search over all alignments is a
different method from beam search, so agreement is a real pin.
"""
from __future__ import annotations

import itertools

import numpy as np

F32 = np.float32
NEG_INF = F32(-np.inf)


def collapse(align, V):
    """CTC collapse of a frame-label sequence: merge repeats, drop blanks (= V)."""
    out = []
    prev = V
    for c in align:
        c = int(c)
        if c != V and c != prev:
            out.append(c)
        prev = c
    return out


def fold_alignment(D, align, V, alpha=0.0, beta=0.0, boost_w=0.0, lm=None, bt=None,
                   rollback=False, repeat=False):
    """fp32 score of one alignment: the per-frame left fold of the candidate
    score (Alg. 1 score update, Eq. 1), then LM.Final (and, with rollback, the
    pending boosting taken back).  With repeat, a frame that repeats the
    previous frame's token adds that token's LM and boosting terms again
    (the terms it got when it was emitted; no beta).  D: [T, V+1] fp32."""
    s = F32(0.0)
    last = V
    y = []
    q = []
    terms = []  # the LM and boosting terms of the last emitted token
    for t, c in enumerate(align):
        c = int(c)
        x = F32(s + F32(D[t, c]))
        emit = c != V and c != last
        if emit:
            x = F32(x + F32(beta))
            terms = []
            if lm is not None:
                al = F32(F32(alpha) * F32(lm.score(y, c)))
                x = F32(x + al)
                terms.append(al)
            if bt is not None:
                sc, q2 = bt.step(q, c)
                wb = F32(F32(boost_w) * F32(sc))
                x = F32(x + wb)
                terms.append(wb)
                q = q2
            y.append(c)
        elif repeat and c != V:
            for v in terms:
                x = F32(x + v)
        last = c
        s = x
    if lm is not None:
        s = F32(s + F32(F32(alpha) * F32(lm.score(y, V))))
    if rollback and bt is not None and s != NEG_INF:
        s = F32(s + F32(F32(boost_w) * F32(-bt.pot(q))))
    return s, y


def brute_force(D, V, **kw):
    """Max over all (V+1)^T alignments of fold_alignment.  Returns
    (best score, set of transcripts attaining it)."""
    T = D.shape[0]
    best = NEG_INF
    arg = set()
    for align in itertools.product(range(V + 1), repeat=T):
        s, y = fold_alignment(D, align, V, **kw)
        if s > best:
            best = s
            arg = {tuple(y)}
        elif s == best:
            arg.add(tuple(y))
    return best, arg


def brute_force_keys_logsum(D, V, **kw):
    """For every recombination key (collapsed transcript, ends-in-blank) the
    log of the summed probability of all its alignments, in fp64 from the
    fp32 fold of each alignment: {key: log sum exp(fold)}."""
    T = D.shape[0]
    acc = {}
    for align in itertools.product(range(V + 1), repeat=T):
        s, y = fold_alignment(D, align, V, **kw)
        if s == NEG_INF:
            continue
        key = (tuple(y), (align[-1] if T else V) == V)
        acc.setdefault(key, []).append(float(s))
    out = {}
    for key, v in acc.items():
        m = max(v)
        out[key] = m + float(np.log(np.sum(np.exp(np.array(v) - m))))
    return out


def greedy(D, L, V):
    """Greedy CTC: per-frame argmax (lowest index on ties), collapse; score is
    the fp32 left fold of the per-frame maxima."""
    s = F32(0.0)
    align = []
    for t in range(L):
        c = int(np.argmax(D[t]))
        s = F32(s + F32(D[t, c]))
        align.append(c)
    return collapse(align, V), s


def greedy_fused(D, L, V, alpha=0.0, beta=0.0, boost_w=0.0, lm=None, bt=None):
    """Greedy decoding with fusion written as its own sequential search: at
    every frame score each label with the candidate fold of Eq. 1 (the same
    steps as fold_alignment), keep the first maximum (lowest label), then
    LM.Final.  A frame whose best candidate is -inf ends the hypothesis
    (empty transcript, -inf).  Returns (transcript, score)."""
    s = F32(0.0)
    last = V
    y, q = [], []
    for t in range(L):
        best, arg, arg_q = NEG_INF, -1, None
        for c in range(V + 1):
            x = F32(s + F32(D[t, c]))
            q2 = q
            if c != V and c != last:
                x = F32(x + F32(beta))
                if lm is not None:
                    x = F32(x + F32(F32(alpha) * F32(lm.score(y, c))))
                if bt is not None:
                    sc, q2 = bt.step(q, c)
                    x = F32(x + F32(F32(boost_w) * F32(sc)))
            if x > best:
                best, arg, arg_q = x, c, q2
        if best == NEG_INF:
            return [], NEG_INF
        if arg != V and arg != last:
            y.append(arg)
            q = arg_q
        last = arg
        s = best
    if lm is not None:
        s = F32(s + F32(F32(alpha) * F32(lm.score(y, V))))
    return y, s


def transcripts_from_trace(bp_index, W, t, K):
    """Collapsed transcript and last label of every slot after frame t,
    rebuilt by walking the backpointers."""
    V = W - 1
    res = []
    for j in range(K):
        labels = []
        jj = j
        for tt in range(t, -1, -1):
            i = int(bp_index[tt, jj])
            labels.append(i % W)
            jj = i // W
        labels.reverse()
        res.append((tuple(collapse(labels, V)), labels[-1]))
    return res


def brute_force_keys(D, V, **kw):
    """Best fp32 fold over all (V+1)^T alignments for every recombination key
    (collapsed transcript, ends-in-blank flag): {key: best score}."""
    T = D.shape[0]
    best = {}
    for align in itertools.product(range(V + 1), repeat=T):
        s, y = fold_alignment(D, align, V, **kw)
        key = (tuple(y), (align[-1] if T else V) == V)
        if key not in best or s > best[key]:
            best[key] = s
    return best
