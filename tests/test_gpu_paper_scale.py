"""GPU parity at paper scale: a subword 6-gram LM with 11 M n-grams (the paper
decodes with KenLM 6-grams, Sec. IV-A), 1000 boosted phrases, theta = 12
(Sec. IV-D), beams 4-64 (Fig. "beam_size_vs_wer"; K = 8 fills all rows of a
chunk, K = 4 and 8 with the fold kept in the rows of one chunk, 16 and 64
across chunks), through the C ABI against
the CPU oracle.  Tokens bit-exact, scores within 1e-4.
"""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from gpu_helpers import compare, handles, log, oracle_threads, run_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("K", [4, 8, 16, 64])
def test_six_gram_reduced(K):
    w = W.CONFIGS[6].replace(B=3, T=120, lengths=("uniform", 60, 120), K=K)
    log(f"6-gram: building inputs (K={K})")
    lm, bt, olm, obt = handles(w)
    lp = W.make_logprobs(w)
    lens = W.make_lengths(w)
    log(f"6-gram B={w.B} T={w.T} K={K} theta={w.theta}")
    g = run_gpu(lp, lens, K, w.alpha, w.beta, w.boost_w, lm, bt, theta=w.theta)
    r = oracle.decode(lp, lens, K, w.alpha, w.beta, w.boost_w, theta=w.theta, lm=olm, bt=obt,
                      n_threads=oracle_threads())
    compare(g, r, what=f"6-gram K={K}")
    assert g["status"] == 0
