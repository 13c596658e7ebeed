"""The entry point that allocates nothing (ctcbeam_decode_noalloc) against
ctcbeam_decode_ex on the same inputs: tokens and lengths bit-exact, scores
within 1e-4 (the same kernels run, so they are expected to be identical).
Two calls in a row on the shared per-device array, the second with a smaller
input; a request above the array's size is rejected with code 2."""
import ctypes
import math

import numpy as np
import pytest

import paper_2508_07315_amd as P
import workloads as W
from gpu_helpers import SCORE_TOL, device, handles, log

pytestmark = pytest.mark.gpu


def _check_same(a, b, what):
    ta, la, sa = (x.cpu().numpy() for x in a)
    tb, lb, sb = (x.cpu().numpy() for x in b)
    np.testing.assert_array_equal(la, lb, err_msg=what)
    np.testing.assert_array_equal(ta, tb, err_msg=what)
    fin = np.isfinite(sb)
    assert np.array_equal(np.isfinite(sa), fin), what
    assert np.all(np.abs(sa[fin].astype(np.float64) - sb[fin]) <= SCORE_TOL), what


def _case(w, theta):
    import torch
    dev = device()
    lm, bt, _, _ = handles(w)
    lp = torch.from_numpy(W.make_logprobs(w)).to(dev)
    lens = torch.from_numpy(W.make_lengths(w)).to(dev)
    B, T = w.B, w.T
    outs = (torch.empty((B, T), dtype=torch.int32, device=dev),
            torch.empty((B,), dtype=torch.int32, device=dev),
            torch.empty((B,), dtype=torch.float32, device=dev))
    torch.cuda.synchronize()
    got = P.ctcbeam_decode_noalloc(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, *outs,
                                   theta=theta)
    ref = P.ctcbeam_decode_ex(lp, lens, w.K, w.alpha, w.beta, w.boost_w, lm, bt, theta=theta)[:3]
    torch.cuda.synchronize()
    return got, ref


def test_noalloc_matches_decode_ex_two_calls():
    import torch
    big = W.CONFIGS[3].replace(B=16, T=240, lengths=("uniform", 120, 240))
    small = W.CONFIGS[3].replace(B=5, T=90, lengths=("uniform", 30, 90))
    log(f"noalloc: call 1 B={big.B} T={big.T} K={big.K}")
    got, ref = _case(big, math.inf)
    _check_same(got, ref, "first call")
    log(f"noalloc: call 2 B={small.B} T={small.T} K={small.K} theta=12")
    got, ref = _case(small, 12.0)
    _check_same(got, ref, "second, smaller call")
    # a boosting workload with a larger beam through the same array
    w5 = W.CONFIGS[5].replace(B=3, T=60, lengths=("uniform", 30, 60))
    log(f"noalloc: call 3 B={w5.B} T={w5.T} K={w5.K} with boosting")
    got, ref = _case(w5, math.inf)
    _check_same(got, ref, "boosting call")
    torch.cuda.synchronize()


def test_noalloc_rejects_sizes_above_the_array():
    import torch
    dev = device()
    lib = P._load()
    B, T, K, V = 64, 9000, 8, 7  # 18.4 MB of back-pointers > 16 MiB
    assert P.ctcbeam_workspace_bytes(B, T, K) > P.NOALLOC_MAX_WORKSPACE
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the size check comes first
    rc = lib.ctcbeam_decode_noalloc(fake, fake, B, T, V, K, 0.0, 0.0, 0.0, None, None, fake, None,
                                    fake, None, None)
    assert rc == 2
    assert b"no-allocation limit" in lib.ctcbeam_last_error()
    torch.cuda.synchronize()
