"""GPU parity of the N-best output (every beam slot's final hypothesis, the
batched-hypotheses result of Algorithm 1) against the CPU oracle.

Bar: every row's tokens and length bit-exact, in the same order; scores
within 1e-4 absolute (both -inf allowed).

* the five workloads at reduced sizes, with and without pruning;
* full size, every utterance of every workload: tests/test_gpu_full_size.py;
* exhaustive pins on the GPU: with K >= (V+1)^T the live rows are exactly
  the recombination keys' best folds over all alignments;
* row 0 equals the 1-best entry point's output; fuzzing over B, T, V, K,
  lengths, LM, boosting and theta; L = 0, T = 0, a -inf frame, K = 1.
"""
import math

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import SCORE_TOL, device, handles, log, oracle_threads, run_gpu
from oracle_helpers import brute_force_keys

pytestmark = pytest.mark.gpu

REDUCED = {
    1: dict(),
    2: dict(B=6, T=120, lengths=("uniform", 40, 120)),
    3: dict(B=6, T=120, lengths=("uniform", 40, 120)),
    4: dict(B=3, T=80, lengths=("uniform", 40, 80)),
    5: dict(B=3, T=60, lengths=("uniform", 30, 60)),
}


def run_nbest(lp, lens, K, alpha=0.0, beta=0.0, boost_w=0.0, lm=None, boost=None,
              theta=math.inf):
    import torch
    dev = device()
    d_lp = torch.from_numpy(np.ascontiguousarray(lp)).to(dev)
    d_len = torch.from_numpy(np.ascontiguousarray(lens, dtype=np.int32)).to(dev)
    tok, ln, sc, ws = P.ctcbeam_decode_nbest(d_lp, d_len, K, alpha, beta, boost_w, lm, boost,
                                             theta=theta)
    torch.cuda.synchronize()
    return dict(tokens=tok.cpu().numpy(), lengths=ln.cpu().numpy(), scores=sc.cpu().numpy(),
                status=P.ctcbeam_query_status(ws))


def compare_nbest(g, r, rows=None, ref_rows=None, what=""):
    rows = range(g["tokens"].shape[0]) if rows is None else rows
    ref_rows = rows if ref_rows is None else ref_rows
    worst = 0.0
    for gb, rb in zip(rows, ref_rows):
        gl, rl = g["lengths"][gb], r["nbest_lengths"][rb]
        assert np.array_equal(gl, rl), f"{what} utt {gb}: lengths {gl} vs {rl}"
        gt, rt = g["tokens"][gb], r["nbest_tokens"][rb]
        if not np.array_equal(gt, rt):
            row, col = (int(x[0]) for x in np.nonzero(gt != rt))
            raise AssertionError(f"{what} utt {gb} row {row}: tokens differ at {col}: "
                                 f"gpu {gt[row, max(0, col-3):col+3]} oracle {rt[row, max(0, col-3):col+3]}")
        gs, rs = g["scores"][gb], r["nbest_scores"][rb]
        inf = np.isinf(gs) | np.isinf(rs)
        assert np.array_equal(gs[inf], rs[inf]), f"{what} utt {gb}: scores {gs} vs {rs}"
        if (~inf).any():
            d = float(np.max(np.abs(gs[~inf].astype(np.float64) - rs[~inf])))
            worst = max(worst, d)
            assert d <= SCORE_TOL, f"{what} utt {gb}: scores {gs} vs {rs}"
    return worst


def _oracle(w, lp, lens, olm, obt, theta=math.inf):
    return oracle.decode(lp, lens, w.K, w.alpha, w.beta, w.boost_w, theta=theta, lm=olm, bt=obt,
                         n_threads=oracle_threads(), want_nbest=True)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_nbest_config_reduced(cfg):
    w = W.CONFIGS[cfg].replace(**REDUCED[cfg])
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    for th in [math.inf] + ([12.0] if cfg >= 3 else []):
        log(f"nbest cfg{cfg} reduced B={w.B} T={w.T} K={w.K} theta={th}")
        g = run_nbest(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th)
        r = _oracle(w, lp, lens, olm, obt, theta=th)
        worst = compare_nbest(g, r, what=f"nbest cfg{cfg} theta={th}")
        assert g["status"] == 0
        # row 0 is the 1-best entry point's result
        one = run_gpu(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=th)
        np.testing.assert_array_equal(g["tokens"][:, 0], one["tokens"])
        np.testing.assert_array_equal(g["lengths"][:, 0], one["lengths"])
        np.testing.assert_array_equal(g["scores"][:, 0], one["scores"])
        log(f"  ok, max |score diff| = {worst}")


def _phrases(V, rng, n):
    lens = rng.integers(1, 5, size=n)
    toks = rng.integers(0, V, size=int(lens.sum()))
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), toks.astype(np.int32)


@pytest.mark.parametrize("V", [1, 2, 3])
@pytest.mark.parametrize("mode", ["plain", "lm", "lm_bt"])
def test_nbest_exhaustive_on_gpu(V, mode):
    for T in (1, 2, 3):
        if (V + 1) ** T > 64:
            continue
        rng = np.random.default_rng(2000 + 100 * V + 10 * T + len(mode))
        D = W.random_logprobs(rng, 1, T, V, scale=1.5)
        kw = {}
        lm = bt = olm = obt = None
        beta = 0.7 if mode != "plain" else 0.0
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
        keys = brute_force_keys(D[0], V, alpha=alpha, beta=beta, boost_w=w_, **kw)
        g = run_nbest(D, np.array([T]), 64, alpha, beta, w_, lm, bt)
        sc, ln, tk = g["scores"][0], g["lengths"][0], g["tokens"][0]
        live = int(np.sum(sc != -np.inf))
        assert live == len(keys), (V, T, mode, live, len(keys))
        got = sorted(((float(sc[r]), tuple(tk[r, : ln[r]].tolist())) for r in range(live)),
                     key=lambda e: (-e[0], e[1]))
        want = sorted(((float(s), k[0]) for k, s in keys.items()), key=lambda e: (-e[0], e[1]))
        assert got == want, (V, T, mode)
        r = oracle.decode(D, np.array([T]), 64, alpha, beta, w_, lm=olm, bt=obt, want_nbest=True)
        compare_nbest(g, r, what=f"nbest exhaustive V={V} T={T} {mode}")


FUZZ_V = [1, 2, 3, 7, 31, 100, 512, 513, 1024]
FUZZ_K = [1, 2, 3, 5, 8, 16, 33, 64]


@pytest.mark.parametrize("seed", range(16))
def test_nbest_fuzz(seed):
    rng = np.random.default_rng(9000 + seed)
    V = int(rng.choice(FUZZ_V))
    K = int(rng.choice(FUZZ_K))
    B = int(rng.integers(1, 7))
    T = int(rng.integers(1, 30))
    lens = rng.integers(0, T + 1, size=B)
    lens[rng.integers(0, B)] = T
    lp = W.random_logprobs(rng, B, T, V, scale=float(rng.uniform(0.5, 3.0)))
    for b in range(B):
        lp[b, lens[b]:] = np.nan   # padding is never read
    use_lm = rng.random() < 0.6
    use_bt = rng.random() < 0.5
    theta = float(rng.choice([math.inf, 5.0, 12.0]))
    alpha, beta, bw = float(rng.uniform(0, 1)), float(rng.uniform(-1, 2)), float(rng.uniform(0, 2))
    lm = bt = olm = obt = None
    if use_lm:
        arrays = W.random_small_lm(rng, int(rng.integers(1, 5)), V, density=0.4) if V <= 8 else \
            W.make_lm(3, V, [min(3 * V, (V + 1) ** 2), 2 * V], int(rng.integers(0, 1 << 30)))
        lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    if use_bt:
        off, toks = _phrases(V, rng, int(rng.integers(1, 20)))
        bt, obt = P.ctcbeam_boost_build(V, off, toks), oracle.BT(V, off, toks)
    log(f"nbest fuzz {seed}: B={B} T={T} V={V} K={K} lm={use_lm} bt={use_bt} theta={theta}")
    g = run_nbest(lp, lens, K, alpha, beta, bw, lm, bt, theta=theta)
    r = oracle.decode(lp, lens, K, alpha, beta, bw, theta=theta, lm=olm, bt=obt,
                      n_threads=oracle_threads(), want_nbest=True)
    compare_nbest(g, r, what=f"nbest fuzz {seed}")
    assert g["status"] == 0


def test_nbest_edges():
    rng = np.random.default_rng(11)
    arrays = W.random_small_lm(rng, 3, 4)
    lm, olm = P.ctcbeam_lm_build(arrays), oracle.LM(arrays)
    # L = 0 (only the initial beam), a -inf frame (every slot dead), full length
    lp = W.random_logprobs(rng, 3, 8, 4)
    lp[1, 3, :] = -np.inf
    lens = np.array([0, 8, 8])
    for K in (1, 3, 7):
        g = run_nbest(lp, lens, K, 0.5, 0.4, lm=lm)
        r = oracle.decode(lp, lens, K, 0.5, 0.4, lm=olm, want_nbest=True)
        compare_nbest(g, r, what=f"nbest edges K={K}")
        assert np.all(np.isneginf(g["scores"][1])) and np.all(g["lengths"][1] == 0)
        assert np.all(g["tokens"][1] == -1)
        assert np.all(np.isneginf(g["scores"][0, 1:])) and np.all(g["lengths"][0] == 0)
    # empty time axis
    lp0 = np.zeros((2, 0, 5), dtype=np.float32)
    g = run_nbest(lp0, np.array([0, 0]), 3, 0.5, lm=lm)
    r = oracle.decode(lp0, np.array([0, 0]), 3, 0.5, lm=olm, want_nbest=True)
    compare_nbest(g, r, what="nbest T=0")
    # constant rows: every label ties and index order decides the slots
    for V, K in [(600, 8), (33, 64)]:
        lp = np.full((2, 6, V + 1), -math.log(V + 1), dtype=np.float32)
        lp[1, 2, 5] = -0.5
        g = run_nbest(lp, np.array([6, 6]), K, beta=0.25)
        r = oracle.decode(lp, np.array([6, 6]), K, beta=0.25, want_nbest=True)
        compare_nbest(g, r, what=f"nbest ties V={V} K={K}")


def test_nbest_argument_errors():
    import torch
    dev = device()
    lp = torch.zeros((1, 4, 5), dtype=torch.float32, device=dev)
    ln = torch.full((1,), 4, dtype=torch.int32, device=dev)
    lib = P._load()
    import ctypes
    ws = torch.empty((P.ctcbeam_workspace_bytes(1, 4, 2),), dtype=torch.uint8, device=dev)
    sc = torch.empty((1, 2), dtype=torch.float32, device=dev)
    rc = lib.ctcbeam_decode_nbest(ctypes.c_void_p(lp.data_ptr()), ctypes.c_void_p(ln.data_ptr()),
                                  1, 4, 4, 2, 0.0, 0.0, 0.0, None, None,
                                  ctypes.c_void_p(ws.data_ptr()), ws.numel(), None, None,
                                  ctypes.c_void_p(sc.data_ptr()), None, None)
    assert rc == 1 and b"null output" in lib.ctcbeam_last_error()
