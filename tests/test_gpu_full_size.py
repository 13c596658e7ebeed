"""GPU parity at full size on every utterance of every workload.

The oracle needs minutes per workload at these sizes (about 15 for the
4-gram + boosting one on 8 host threads), so its outputs were written once
by ``tests/golden/make_full_size_expected.py``, which runs only the oracle
on the seeded inputs of ``workloads/``.  Each stored case carries a SHA-256
fingerprint of its inputs; the test recomputes it and fails if the inputs
changed.

Per case (workload, theta in {inf, 12}): one 1-best launch and one N-best
launch of the whole batch, in the configuration the benchmark times.
* 1-best: every utterance's transcript bit-exact, score within 1e-4;
* N-best: every row's length exact, its transcript bit-exact (compared by
  a 64-bit digest of the int32 row), its score within 1e-4.
"""
import math
import os
import sys

import numpy as np
import pytest

import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import SCORE_TOL, device, handles, log

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
from make_full_size_expected import CASES, case_name, input_fingerprint, row_digest  # noqa: E402

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden", "full")


def _scores_match(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    inf = np.isinf(r) | np.isinf(g)
    d = np.abs(np.where(inf, 0.0, g) - np.where(inf, 0.0, r))
    ok = np.where(inf, g == r, d <= SCORE_TOL)
    return ok, float(np.max(d, initial=0.0))


@pytest.mark.parametrize("cfg,theta", CASES, ids=[case_name(c, t) for c, t in CASES])
def test_full_size_every_utterance(cfg, theta):
    import torch
    path = os.path.join(GOLD, case_name(cfg, theta) + ".npz")
    ref = np.load(path, allow_pickle=False)
    w = W.CONFIGS[cfg]
    assert str(ref["workload"]) == w.name
    log(f"{case_name(cfg, theta)}: B={w.B} T={w.T} K={w.K}: building inputs")
    lens = W.make_lengths(w)
    lp = W.make_logprobs(w)
    assert input_fingerprint(w, lp, lens) == str(ref["fingerprint"]), \
        "inputs differ from those the stored oracle outputs were computed on"
    lm, bt, _, _ = handles(w)
    dev = device()
    d_lp = torch.from_numpy(lp).to(dev)
    d_len = torch.from_numpy(lens).to(dev)
    del lp
    log("  1-best launch")
    tok, ln, sc, ws = P.ctcbeam_decode_ex(d_lp, d_len, w.K, w.alpha, w.beta, w.boost_w, lm, bt,
                                          theta=theta)
    torch.cuda.synchronize()
    assert P.ctcbeam_query_status(ws) == 0
    tok, ln, sc = tok.cpu().numpy(), ln.cpu().numpy(), sc.cpu().numpy()
    np.testing.assert_array_equal(ln, ref["lengths"])
    flat = ref["tokens_flat"].astype(np.int32)
    off = np.concatenate([[0], np.cumsum(ref["lengths"])])
    for b in range(w.B):
        n = int(ln[b])
        if not np.array_equal(tok[b, :n], flat[off[b]:off[b + 1]]):
            bad = int(np.nonzero(tok[b, :n] != flat[off[b]:off[b + 1]])[0][0])
            raise AssertionError(f"utt {b}: tokens differ at {bad}")
        assert (tok[b, n:] == -1).all(), f"utt {b}: not -1 padded"
    ok, worst = _scores_match(sc, ref["scores"])
    assert ok.all(), f"scores differ at utterances {np.nonzero(~ok)[0].tolist()}"
    log(f"  1-best: {w.B} utterances equal, max |score diff| {worst:.3g}")

    log("  N-best launch")
    ntok, nln, nsc, ws = P.ctcbeam_decode_nbest(d_lp, d_len, w.K, w.alpha, w.beta, w.boost_w,
                                                lm, bt, theta=theta)
    torch.cuda.synchronize()
    assert P.ctcbeam_query_status(ws) == 0
    ntok, nln, nsc = ntok.cpu().numpy(), nln.cpu().numpy(), nsc.cpu().numpy()
    np.testing.assert_array_equal(nln, ref["nbest_lengths"])
    ok, worst = _scores_match(nsc, ref["nbest_scores"])
    assert ok.all(), f"N-best scores differ at {np.argwhere(~ok)[:5].tolist()}"
    dig = ref["nbest_digest"]
    for b in range(w.B):
        for k in range(w.K):
            n = int(nln[b, k])
            assert row_digest(ntok[b, k, :n]) == dig[b, k], f"utt {b} rank {k}: transcript differs"
            assert (ntok[b, k, n:] == -1).all()
    # row 0 is the 1-best result
    np.testing.assert_array_equal(nln[:, 0], ln)
    log(f"  N-best: {w.B}x{w.K} rows equal, max |score diff| {worst:.3g}")
    del d_lp
    torch.cuda.empty_cache()
