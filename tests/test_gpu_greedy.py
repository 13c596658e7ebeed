"""GPU parity of greedy decoding with fusion (Algorithm 1 with one hypothesis,
the greedy rows of Table II) through the C ABI, against the CPU oracle at
K = 1.

Bar: tokens bit-exact; scores within 1e-4 absolute (the fp32 fold is the
same on both sides, so the difference is expected to be 0).

* the five workloads at reduced sizes (every utterance); workloads 2-6 at
  full size (every utterance against the oracle's stored outputs and against
  the beam kernel at K = 1);
* fuzzing over B, T, V (across the 256 / 1024 / 4096 label-per-lane
  classes), LM order, boosting and lengths (0, T, ragged, NaN padding);
* a -inf frame, fully tied rows, L = 0 / T = 0, clamped lengths, counters.
"""
import math
import os
import sys

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import SCORE_TOL, compare, device, handles, log, oracle_threads, run_gpu

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
from make_full_size_expected import GREEDY_CASES, greedy_name, input_fingerprint  # noqa: E402

GOLD = os.path.join(os.path.dirname(__file__), "golden", "full")

pytestmark = pytest.mark.gpu

REDUCED = {
    1: dict(),
    2: dict(B=8, T=200, lengths=("uniform", 80, 200)),
    3: dict(B=8, T=200, lengths=("uniform", 80, 200)),
    4: dict(B=4, T=160, lengths=("uniform", 60, 160)),
    5: dict(B=4, T=120, lengths=("uniform", 40, 120)),
}


def run_greedy(lp, lens, alpha=0.0, beta=0.0, boost_w=0.0, lm=None, boost=None, stats=False):
    import torch
    dev = device()
    d_lp = torch.from_numpy(np.ascontiguousarray(lp)).to(dev)
    d_len = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    st = torch.zeros((lp.shape[0], 8), dtype=torch.int64, device=dev) if stats else None
    tok, ln, sc, ws = P.ctcbeam_greedy_decode(d_lp, d_len, alpha, beta, boost_w, lm, boost, stats=st)
    torch.cuda.synchronize()
    out = dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy(),
               status=P.ctcbeam_query_status(ws))
    if stats:
        out["stats"] = st.cpu().numpy()
    return out


def _oracle(w, lp, lens, olm, obt):
    return oracle.decode(lp, lens, 1, w.alpha, w.beta, w.boost_w, lm=olm, bt=obt,
                         n_threads=oracle_threads())


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_greedy_config_reduced(cfg):
    w = W.CONFIGS[cfg].replace(**REDUCED[cfg])
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log(f"greedy cfg{cfg} reduced B={w.B} T={w.T}")
    g = run_greedy(lp, lens, w.alpha, w.beta, w.boost_w, lm, bt)
    r = _oracle(w, lp, lens, olm, obt)
    worst = compare(g, r, what=f"greedy cfg{cfg}")
    assert g["status"] == 0
    log(f"  ok, max |score diff| = {worst}")


@pytest.mark.parametrize("cfg", GREEDY_CASES)
def test_greedy_full_size(cfg):
    """Every utterance at full size against the oracle's stored K = 1 outputs
    (tests/golden/make_full_size_expected.py), and against the beam kernel
    with one hypothesis, bit for bit."""
    w = W.CONFIGS[cfg]
    ref = np.load(os.path.join(GOLD, greedy_name(cfg) + ".npz"), allow_pickle=False)
    assert str(ref["workload"]) == w.name
    log(f"greedy cfg{cfg} full size B={w.B} T={w.T}")
    lm, bt, _, _ = handles(w)
    lens = W.make_lengths(w)
    lp = W.make_logprobs(w)
    assert input_fingerprint(w, lp, lens) == str(ref["fingerprint"])
    g = run_greedy(lp, lens, w.alpha, w.beta, w.boost_w, lm, bt)
    assert g["status"] == 0
    np.testing.assert_array_equal(g["lengths"], ref["lengths"])
    flat = ref["tokens_flat"].astype(np.int32)
    off = np.concatenate([[0], np.cumsum(ref["lengths"])])
    for b in range(w.B):
        n = int(g["lengths"][b])
        assert np.array_equal(g["tokens"][b, :n], flat[off[b]:off[b + 1]]), f"utt {b}"
        assert (g["tokens"][b, n:] == -1).all()
        gs, rs = float(g["scores"][b]), float(ref["scores"][b])
        assert (gs == rs) if (math.isinf(gs) or math.isinf(rs)) else abs(gs - rs) <= SCORE_TOL
    k1 = run_gpu(lp, lens, 1, w.alpha, w.beta, w.boost_w, lm, bt)
    for k in ("tokens", "lengths", "scores"):
        np.testing.assert_array_equal(g[k], k1[k])


def _phrases(V, rng, n):
    lens = rng.integers(1, 5, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), toks.astype(np.int32)


FUZZ_V = [1, 2, 3, 63, 64, 65, 255, 256, 257, 1000, 1023, 1024, 1025, 2048, 4095, 4096]


@pytest.mark.parametrize("seed", range(24))
def test_greedy_fuzz(seed):
    rng = np.random.default_rng(11000 + seed)
    V = int(FUZZ_V[seed % len(FUZZ_V)])
    B = int(rng.integers(1, 7))
    T = int(rng.integers(1, 70))
    lens = rng.integers(0, T + 1, size=B)
    lens[rng.integers(0, B)] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 3.0)))
    for b in range(B):
        lp[b, lens[b]:] = np.nan   # padding is never read
    use_lm = rng.random() < 0.7
    use_bt = rng.random() < 0.5
    alpha, beta, bw = float(rng.uniform(0, 1)), float(rng.uniform(-1, 2)), float(rng.uniform(0, 2))
    lm = bt = olm = obt = None
    if use_lm:
        order = int(rng.integers(1, 6))
        if V <= 8:
            arrays = W.random_small_lm(rng, order, V, density=0.5)
        else:
            counts = [min(int(rng.integers(V, 4 * V)), (V + 1) ** 2) for _ in range(order - 1)]
            arrays = W.make_lm(order, V, counts, int(rng.integers(0, 1 << 30)))
        lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    if use_bt:
        off, toks = _phrases(V, rng, int(rng.integers(1, 40)))
        bt, obt = P.ctcbeam_boost_build(V, off, toks), oracle.BT(V, off, toks)
    log(f"greedy fuzz {seed}: B={B} T={T} V={V} lm={use_lm} bt={use_bt}")
    g = run_greedy(lp, lens, alpha, beta, bw, lm, bt)
    r = oracle.decode(lp, lens, 1, alpha, beta, bw, lm=olm, bt=obt, n_threads=oracle_threads())
    compare(g, r, what=f"greedy fuzz {seed}")
    assert g["status"] == 0


def test_greedy_edges_and_counters():
    rng = np.random.default_rng(12)
    arrays = W.random_small_lm(rng, 3, 6)
    lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    # a -inf frame kills the hypothesis: empty transcript, -inf
    lp = W.random_logprobs(rng, 3, 15, 6)
    lp[1, 7, :] = -np.inf
    lens = np.array([15, 15, 0])
    g = run_greedy(lp, lens, 0.5, 0.3, lm=lm, stats=True)
    r = oracle.decode(lp, lens, 1, 0.5, 0.3, lm=olm)
    compare(g, r, what="greedy edges")
    assert g["scores"][1] == -np.inf and g["lengths"][1] == 0 and (g["tokens"][1] == -1).all()
    st = g["stats"]
    assert st[0, 0] == 15 and st[0, 1] == 15 and st[0, 6] == g["lengths"][0]
    assert st[0, 7] == 1 + g["lengths"][0]     # one refill at the start, one per emission
    assert st[2, 0] == 0 and st[2, 7] == 0
    # clamped lengths are flagged
    g = run_greedy(lp, np.array([-3, 40, 5]), 0.5, 0.3, lm=lm)
    r = oracle.decode(lp, np.array([0, 15, 5]), 1, 0.5, 0.3, lm=olm)
    compare(g, r, what="greedy clamp")
    assert g["status"] & 1
    # empty time axis
    lp0 = np.zeros((2, 0, 7), dtype=np.float32)
    g = run_greedy(lp0, np.array([0, 0]), 0.5, lm=lm)
    r = oracle.decode(lp0, np.array([0, 0]), 1, 0.5, lm=olm)
    compare(g, r, what="greedy T=0")
    # constant rows: every label ties, the lowest index wins
    for V in (300, 1024, 1500):
        lp = np.full((2, 7, V + 1), -math.log(V + 1), dtype=np.float32)
        lp[1, 3, 5] = -0.5
        g = run_greedy(lp, np.array([7, 7]), beta=0.25)
        r = oracle.decode(lp, np.array([7, 7]), 1, beta=0.25)
        compare(g, r, what=f"greedy ties V={V}")
