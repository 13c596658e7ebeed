"""GPU parity: the HIP decoder (through the C ABI) against the CPU oracle.

Bar: output tokens bit-exact; scores within 1e-4 absolute (the fp32 fold is
the same on both sides, so the difference is expected to be 0).

* the five workloads at reduced sizes, every utterance compared, with and
  without pruning (theta = 12, the paper's setting);
* full size, every utterance: tests/test_gpu_full_size.py;
* exhaustive pins on the GPU (T <= 3, V <= 3, K = 64 >= (V+1)^T);
* fuzzing over B, T, V, K, lengths (0, T, out of range), NaN padding,
  LM order, boosting lists and theta;
* determinism, batch permutation, streams, byte-model counters, edge cases.
"""
import math

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import (compare, device, handles, log, oracle_threads, run_gpu)
from oracle_helpers import brute_force

pytestmark = pytest.mark.gpu

REDUCED = {
    1: dict(),
    2: dict(B=8, T=160, lengths=("uniform", 60, 160)),
    3: dict(B=8, T=160, lengths=("uniform", 60, 160)),
    4: dict(B=4, T=100, lengths=("uniform", 50, 100)),
    5: dict(B=4, T=60, lengths=("uniform", 30, 60)),
}


def _oracle(w, lp, lens, olm, obt, theta=math.inf, **kw):
    return oracle.decode(lp, lens, w.K, w.alpha, w.beta, w.boost_w, theta=theta, lm=olm, bt=obt,
                         n_threads=oracle_threads(), **kw)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_config_reduced(cfg):
    w = W.CONFIGS[cfg].replace(**REDUCED[cfg])
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    thetas = [math.inf] + ([12.0] if cfg >= 3 else [])
    for th in thetas:
        log(f"cfg{cfg} reduced B={w.B} T={w.T} K={w.K} theta={th}")
        g = run_gpu(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th)
        r = _oracle(w, lp, lens, olm, obt, theta=th)
        worst = compare(g, r, what=f"cfg{cfg} theta={th}")
        assert g["status"] == 0
        log(f"  ok, max |score diff| = {worst}")


def _phrases(V, rng, n):
    lens = rng.integers(1, 5, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), toks.astype(np.int32)


@pytest.mark.parametrize("V", [1, 2, 3])
@pytest.mark.parametrize("mode", ["plain", "beta", "lm", "bt", "lm_bt"])
def test_exhaustive_on_gpu(V, mode):
    for T in (1, 2, 3):
        if (V + 1) ** T > 64:
            continue
        rng = np.random.default_rng(1000 * V + 10 * T + len(mode))
        D = W.random_logprobs(rng, 1, T, V, scale=1.5)
        kw = {}
        lm = bt = olm = obt = None
        beta = 0.7 if mode in ("beta", "lm", "lm_bt") else 0.0
        alpha = 0.6 if "lm" in mode else 0.0
        w_ = 1.3 if "bt" in mode else 0.0
        if "lm" in mode:
            arrays = W.random_small_lm(rng, 3, V, density=0.5)
            lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
            kw["lm"] = olm
        if "bt" in mode:
            off, toks = _phrases(V, rng, 3)
            bt, obt = P.ctcbeam_boost_build(V, off, toks), oracle.BT(V, off, toks)
            kw["bt"] = obt
        best, arg = brute_force(D[0], V, alpha=alpha, beta=beta, boost_w=w_, **kw)
        g = run_gpu(D, np.array([T]), 64, alpha, beta, w_, lm, bt)
        assert g["scores"][0] == best, (V, T, mode, g["scores"][0], best)
        assert tuple(g["tokens"][0, : g["lengths"][0]].tolist()) in arg
        r = oracle.decode(D, np.array([T]), 64, alpha, beta, w_, lm=olm, bt=obt)
        compare(g, r, what=f"exhaustive V={V} T={T} {mode}")


FUZZ_V = [1, 2, 3, 7, 31, 64, 100, 511, 512, 513, 700, 1024, 1100]
FUZZ_K = [1, 2, 3, 4, 5, 8, 16, 32, 64]


def _fuzz_lm(rng, V):
    order = int(rng.integers(1, 5))
    if V <= 8:
        return W.random_small_lm(rng, order, V, density=0.4)
    counts = [int(rng.integers(V, 4 * V)) for _ in range(order - 1)]
    counts = [min(c, (V + 1) * (V + 1)) for c in counts]
    return W.make_lm(order, V, counts, int(rng.integers(0, 1 << 30)))


@pytest.mark.parametrize("seed", range(40))
def test_fuzz(seed):
    rng = np.random.default_rng(7000 + seed)
    V = int(rng.choice(FUZZ_V))
    K = int(rng.choice(FUZZ_K))
    B = int(rng.integers(1, 9))
    T = int(rng.integers(1, 40))
    lens = rng.integers(0, T + 1, size=B)
    lens[rng.integers(0, B)] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 3.0)))
    for b in range(B):
        lp[b, lens[b]:] = np.nan   # padding is never read
    use_lm = rng.random() < 0.6
    use_bt = rng.random() < 0.5
    theta = float(rng.choice([math.inf, math.inf, 5.0, 12.0]))
    alpha, beta, bw = float(rng.uniform(0, 1)), float(rng.uniform(-1, 2)), float(rng.uniform(0, 2))
    lm = bt = olm = obt = None
    if use_lm:
        arrays = _fuzz_lm(rng, V)
        lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    if use_bt:
        off, toks = _phrases(V, rng, int(rng.integers(1, 30)))
        bt, obt = P.ctcbeam_boost_build(V, off, toks), oracle.BT(V, off, toks)
    log(f"fuzz {seed}: B={B} T={T} V={V} K={K} lm={use_lm} bt={use_bt} theta={theta}")
    g = run_gpu(lp, lens, K, alpha, beta, bw, lm, bt, theta=theta)
    r = oracle.decode(lp, lens, K, alpha, beta, bw, theta=theta, lm=olm, bt=obt, n_threads=oracle_threads())
    compare(g, r, what=f"fuzz {seed}")
    assert g["status"] == 0


def test_determinism_permutation_and_streams():
    import torch
    w = W.CONFIGS[3].replace(**REDUCED[3])
    lm, bt, _, _ = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    a = run_gpu(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt)
    b = run_gpu(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt)
    for k in ("tokens", "lengths", "scores"):
        np.testing.assert_array_equal(a[k], b[k])
    perm = np.random.default_rng(0).permutation(w.B)
    c = run_gpu(lp[perm], lens[perm], w.K, w.alpha, w.beta, w.boost_w, lm, bt)
    for k in ("tokens", "lengths", "scores"):
        np.testing.assert_array_equal(c[k], a[k][perm])
    s = torch.cuda.Stream(device=device())
    d = run_gpu(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, stream=s.cuda_stream)
    for k in ("tokens", "lengths", "scores"):
        np.testing.assert_array_equal(d[k], a[k])


@pytest.mark.parametrize("cfg", [3, 5])
def test_byte_model_counters_match_oracle(cfg):
    w = W.CONFIGS[cfg].replace(**REDUCED[cfg])
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    g = run_gpu(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, stats=True)
    r = _oracle(w, lp, lens, olm, obt, want_counters=True)
    np.testing.assert_array_equal(g["stats"][:, :7], r["counters"][:, :7])


def test_lengths_out_of_range_are_clamped_and_flagged():
    rng = np.random.default_rng(1)
    B, T, V, K = 3, 20, 9, 4
    lp = W.random_logprobs(rng, B, T, V)
    g = run_gpu(lp, np.array([-4, T + 7, 5]), K, beta=0.3)
    r = oracle.decode(lp, np.array([0, T, 5]), K, beta=0.3)
    compare(g, r, what="clamp")
    assert g["status"] & 1


def test_all_minus_inf_frame_and_ties():
    rng = np.random.default_rng(2)
    # a frame of -inf kills every beam: empty transcript, score -inf
    lp = W.random_logprobs(rng, 2, 12, 6)
    lp[0, 5, :] = -np.inf
    g = run_gpu(lp, np.array([12, 12]), 4, beta=0.5)
    r = oracle.decode(lp, np.array([12, 12]), 4, beta=0.5)
    compare(g, r, what="-inf frame")
    assert g["scores"][0] == -np.inf and g["lengths"][0] == 0
    # constant rows: every label ties, index order decides (exercises the
    # exact fallback of the selection when the survivor buffer overflows)
    for V, K in [(600, 8), (1024, 16), (300, 64), (33, 64)]:
        lp = np.full((2, 6, V + 1), -math.log(V + 1), dtype=np.float32)
        lp[1, 2, 5] = -0.5
        g = run_gpu(lp, np.array([6, 6]), K, beta=0.25)
        r = oracle.decode(lp, np.array([6, 6]), K, beta=0.25)
        compare(g, r, what=f"ties V={V} K={K}")


def test_zero_lengths_and_empty_time_axis():
    rng = np.random.default_rng(3)
    arrays = W.random_small_lm(rng, 3, 4)
    lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    lp = W.random_logprobs(rng, 3, 5, 4)
    g = run_gpu(lp, np.array([0, 0, 0]), 3, alpha=0.5, lm=lm)
    r = oracle.decode(lp, np.array([0, 0, 0]), 3, alpha=0.5, lm=olm)
    compare(g, r, what="L=0")
    lp0 = np.zeros((2, 0, 5), dtype=np.float32)
    g = run_gpu(lp0, np.array([0, 0]), 3, alpha=0.5, lm=lm)
    r = oracle.decode(lp0, np.array([0, 0]), 3, alpha=0.5, lm=olm)
    compare(g, r, what="T=0")


def test_query_status_reads_the_batch_size_from_the_workspace():
    """ctcbeam_query_status takes the workspace alone: the decode records its
    batch size in the workspace header.  A reused workspace reports the last
    decode (an empty batch included); a never-used one is rejected."""
    import torch
    dev = device()
    rng = np.random.default_rng(4)
    B, T, V, K = 3, 20, 9, 4
    lp = torch.from_numpy(W.random_logprobs(rng, B, T, V)).to(dev)
    ws = torch.zeros(P.ctcbeam_workspace_bytes(B, T, K), dtype=torch.uint8, device=dev)
    with pytest.raises(P.CtcbeamError) as e:
        P.ctcbeam_query_status(ws)
    assert e.value.code == 1
    bad = torch.tensor([-4, T + 7, 5], dtype=torch.int32, device=dev)
    P.ctcbeam_decode_ex(lp, bad, K, beta=0.3, workspace=ws)
    assert P.ctcbeam_query_status(ws) & 1
    # a smaller batch in the same workspace: only its own status words count
    ok = torch.tensor([T], dtype=torch.int32, device=dev)
    P.ctcbeam_decode_ex(lp[2:], ok, K, beta=0.3, workspace=ws)
    assert P.ctcbeam_query_status(ws) == 0
    P.ctcbeam_decode_ex(lp, bad, K, beta=0.3, workspace=ws)
    assert P.ctcbeam_query_status(ws) & 1
    empty = torch.zeros((0, T, V + 1), dtype=torch.float32, device=dev)
    P.ctcbeam_decode_ex(empty, torch.zeros(0, dtype=torch.int32, device=dev), K, workspace=ws)
    assert P.ctcbeam_query_status(ws) == 0
    # the greedy kernel records the header too
    P.ctcbeam_greedy_decode(lp, bad, beta=0.3, workspace=ws)
    assert P.ctcbeam_query_status(ws) & 1
    torch.cuda.synchronize()
