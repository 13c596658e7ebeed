"""CPU oracle for the batched CTC beam-search step - TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The decoder package never does, and
this package never imports the decoder: the two share no code.

The arithmetic lives in ``ctc_oracle.cpp`` (plain C++17, fp32, no FMA
contraction); this module builds it with g++ and marshals numpy arrays
through ctypes.  Every function cites, in the C++ source, the part of the
paper it follows (Algorithm 1, Eq. 1, Sec. II "NGPU-LM", Sec. III-B).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ctc_oracle.cpp")
_LIB = os.path.join(_HERE, "libctc_oracle.so")
_lib = None

CXXFLAGS = ["-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
            "-pthread"]


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["g++", *CXXFLAGS, _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.oracle_lm_new.restype = P
    lib.oracle_lm_new.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, P]
    lib.oracle_lm_free.argtypes = [P]
    lib.oracle_lm_score.restype = ctypes.c_float
    lib.oracle_lm_score.argtypes = [P, i32p, ctypes.c_int, ctypes.c_int]
    lib.oracle_lm_backoff.restype = ctypes.c_float
    lib.oracle_lm_backoff.argtypes = [P, i32p, ctypes.c_int, ctypes.c_int]
    lib.oracle_bt_new.restype = P
    lib.oracle_bt_new.argtypes = [ctypes.c_int, ctypes.c_int, P, P]
    lib.oracle_bt_free.argtypes = [P]
    lib.oracle_bt_run.restype = ctypes.c_int
    lib.oracle_bt_run.argtypes = [P, i32p, ctypes.c_int, i32p, ctypes.POINTER(ctypes.c_int)]
    lib.oracle_bt_step.restype = ctypes.c_int
    lib.oracle_bt_step.argtypes = [P, i32p, ctypes.c_int, ctypes.c_int, i32p,
                                   ctypes.POINTER(ctypes.c_int)]
    lib.oracle_bt_pot.restype = ctypes.c_int
    lib.oracle_bt_pot.argtypes = [P, i32p, ctypes.c_int]
    lib.oracle_decode.restype = ctypes.c_int
    lib.oracle_decode.argtypes = [P, P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                  ctypes.c_int, P, P, ctypes.c_int, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_lse32.restype = ctypes.c_float
    lib.oracle_lse32.argtypes = [ctypes.c_float, ctypes.c_float]
    _lib = lib
    return lib


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _ip(seq):
    arr = _i32(np.asarray(seq, dtype=np.int32).reshape(-1))
    return arr, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def lse32(a: float, b: float) -> np.float32:
    """The oracle's fp32 log(exp(a) + exp(b)) (log-sum-exp recombination)."""
    return np.float32(_load().oracle_lse32(float(a), float(b)))


class LM:
    """Backoff n-gram model over ARPA-style arrays (see ``workloads.make_lm``)."""

    def __init__(self, arrays: dict):
        lib = _load()
        order, V = int(arrays["order"]), int(arrays["V"])
        self._keep = []
        ids = [np.ascontiguousarray(a, dtype=np.int32) for a in arrays["ids"]]
        pr = [np.ascontiguousarray(a, dtype=np.float32) for a in arrays["log10_prob"]]
        bo = [None if a is None else np.ascontiguousarray(a, dtype=np.float32)
              for a in arrays["log10_bow"]]
        counts = np.asarray([a.shape[0] for a in ids], dtype=np.int64)
        ids_p = (ctypes.c_void_p * order)(*[_ptr(a) for a in ids])
        pr_p = (ctypes.c_void_p * order)(*[_ptr(a) for a in pr])
        bo_p = (ctypes.c_void_p * order)(*[_ptr(a) for a in bo])
        self._h = lib.oracle_lm_new(order, V, _ptr(counts), ids_p, pr_p, bo_p)
        if not self._h:
            raise ValueError("oracle rejected the n-gram arrays")
        self.order, self.V = order, V

    def score(self, y, c: int) -> float:
        """ln P(c | <s> y) as fp32 (returned as a Python float)."""
        arr, p = _ip(y)
        return float(np.float32(_load().oracle_lm_score(self._h, p, len(arr), int(c))))

    def backoff(self, h, c: int) -> float:
        arr, p = _ip(h)
        return float(np.float32(_load().oracle_lm_backoff(self._h, p, len(arr), int(c))))

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.oracle_lm_free(self._h)
            self._h = None


class BT:
    """Phrase-boosting tree over a CSR phrase list."""

    def __init__(self, V: int, offsets, tokens):
        lib = _load()
        self._off = _i32(offsets)
        self._tok = _i32(tokens)
        n = len(self._off) - 1
        self._h = lib.oracle_bt_new(int(V), n, _ptr(self._off), _ptr(self._tok))
        if not self._h:
            raise ValueError("oracle rejected the phrase list")
        self.V = V

    def run(self, seq):
        """(total score, final state) of reading seq from the root."""
        arr, p = _ip(seq)
        st = np.zeros(max(1, len(arr)), dtype=np.int32)
        n = ctypes.c_int(0)
        s = _load().oracle_bt_run(self._h, p, len(arr),
                                  st.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                  ctypes.byref(n))
        return int(s), st[: n.value].tolist()

    def step(self, q, c: int):
        arr, p = _ip(q)
        st = np.zeros(len(arr) + 1, dtype=np.int32)
        n = ctypes.c_int(0)
        s = _load().oracle_bt_step(self._h, p, len(arr), int(c),
                                   st.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                   ctypes.byref(n))
        return int(s), st[: n.value].tolist()

    def pot(self, q) -> int:
        arr, p = _ip(q)
        return int(_load().oracle_bt_pot(self._h, p, len(arr)))

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.oracle_bt_free(self._h)
            self._h = None


def decode(logprobs: np.ndarray, lengths, K: int, alpha: float = 0.0, beta: float = 0.0,
           boost_w: float = 0.0, theta: float = math.inf, lm: Optional[LM] = None,
           bt: Optional[BT] = None, n_threads: int = 1, want_align: bool = False,
           want_trace: bool = False, want_counters: bool = False, want_nbest: bool = False,
           logsumexp: bool = False, boost_rollback: bool = False,
           repeat_score: bool = False) -> dict:
    """Run the oracle on host arrays.  logprobs: fp32 [B, T, V+1] (blank = V).

    want_nbest adds every slot's final hypothesis ordered by final score
    (lowest slot on ties; dead slots last, empty, -inf): nbest_tokens
    [B, K, T] (-1 padded), nbest_lengths [B, K], nbest_scores [B, K].
    logsumexp merges recombined hypotheses with lse32 instead of max;
    boost_rollback takes back the pending boosting of unfinished phrases at
    the end of the utterance; repeat_score adds the LM and boosting terms of
    a token again at every frame that repeats it."""
    lib = _load()
    flags = (1 if logsumexp else 0) | (2 if boost_rollback else 0) | (4 if repeat_score else 0)
    lp = np.ascontiguousarray(logprobs, dtype=np.float32)
    B, T, W = lp.shape
    V = W - 1
    ln = _i32(lengths)
    assert ln.shape == (B,)
    toks = np.empty((B, T), dtype=np.int32)
    lens = np.empty(B, dtype=np.int32)
    scores = np.empty(B, dtype=np.float32)
    align = np.empty((B, T), dtype=np.int32) if want_align else None
    bp = np.full((B, T, K), -1, dtype=np.int32) if want_trace else None
    ss = np.full((B, T, K), np.nan, dtype=np.float32) if want_trace else None
    cnt = np.zeros((B, 8), dtype=np.int64) if want_counters else None
    nbt = np.empty((B, K, T), dtype=np.int32) if want_nbest else None
    nbl = np.empty((B, K), dtype=np.int32) if want_nbest else None
    nbs = np.empty((B, K), dtype=np.float32) if want_nbest else None
    rc = lib.oracle_decode(_ptr(lp), _ptr(ln), B, T, V, int(K), float(alpha), float(beta),
                           float(boost_w), float(theta), int(flags), lm._h if lm else None,
                           bt._h if bt else None, int(n_threads), _ptr(toks), _ptr(lens),
                           _ptr(scores), _ptr(align), _ptr(bp), _ptr(ss), _ptr(cnt),
                           _ptr(nbt), _ptr(nbl), _ptr(nbs))
    if rc != 0:
        raise ValueError(f"oracle_decode returned {rc}")
    out = dict(tokens=toks, lengths=lens, scores=scores)
    if want_align:
        out["align"] = align
    if want_trace:
        out["bp_index"] = bp
        out["slot_scores"] = ss
    if want_counters:
        out["counters"] = cnt
    if want_nbest:
        out["nbest_tokens"] = nbt
        out["nbest_lengths"] = nbl
        out["nbest_scores"] = nbs
    return out
