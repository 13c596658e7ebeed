"""ctcbeam - MI355X-native batched CTC beam search with n-gram LM fusion and
phrase boosting (the per-frame step of FlexCTC, arXiv 2508.07315, Algorithm 1).

This module is a thin ctypes binding over the C ABI declared in
``include/ctcbeam.h`` and implemented by ``libctcbeam.so`` (host builders in
``csrc/ctcbeam_host.cpp``, gfx950 kernels in ``csrc/ctcbeam_decode.inl`` and
``csrc/ctcbeam_greedy.inl``, compiled per vocabulary class by the
``csrc/*.hip`` units).  It only marshals arguments: every step of the search
runs in the HIP kernels.  PyTorch supplies device memory and streams; each
call runs with the inputs' device current, and tensors the binding allocates
are recorded on the launch stream when it is not torch's current stream.

If the shared library has not been built, importing the binding's entry
points raises; build it with ``python -m paper_2508_07315_amd.build_lib`` (or
``__graft_entry__.build()``).  There is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libctcbeam.so")
_lib = None

MAX_K = 128           # CTCBEAM_MAX_K (beams above 64 need V <= 1024)
MAX_V = 4096
MAX_ORDER = 8


class CtcbeamError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"ctcbeam error {code}: {msg}")
        self.code = code


def library_path() -> str:
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2508_07315_amd.build_lib` "
            "(the decoder has no CPU fallback)")
    # torch first: its HIP runtime and the system one share a SONAME, so the
    # first loaded serves the whole process; it must be the one that owns
    # torch's device memory and streams
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    I = ctypes.c_int
    F = ctypes.c_float
    lib.ctcbeam_last_error.restype = ctypes.c_char_p
    lib.ctcbeam_last_error.argtypes = []
    for name in ("ctcbeam_lm_build", "ctcbeam_lm_build_host"):
        fn = getattr(lib, name)
        fn.restype = I
        fn.argtypes = [I, I, P, P, P, P, ctypes.POINTER(P)]
    for name in ("ctcbeam_lm_build_arpa", "ctcbeam_lm_build_arpa_host"):
        fn = getattr(lib, name)
        fn.restype = I
        fn.argtypes = [ctypes.c_char_p, I, ctypes.POINTER(P)]
    lib.ctcbeam_lm_free.restype = None
    lib.ctcbeam_lm_free.argtypes = [P]
    for name in ("ctcbeam_boost_build", "ctcbeam_boost_build_host"):
        fn = getattr(lib, name)
        fn.restype = I
        fn.argtypes = [I, I, P, P, ctypes.POINTER(P)]
    lib.ctcbeam_boost_free.restype = None
    lib.ctcbeam_boost_free.argtypes = [P]
    lib.ctcbeam_workspace_bytes.restype = ctypes.c_size_t
    lib.ctcbeam_workspace_bytes.argtypes = [I, I, I]
    dec = [P, P, I, I, I, I, F, F, F, P, P, P, ctypes.c_size_t, P, P, P, P]
    lib.ctcbeam_decode.restype = I
    lib.ctcbeam_decode.argtypes = dec
    lib.ctcbeam_decode_ex.restype = I
    lib.ctcbeam_decode_ex.argtypes = dec + [P]
    lib.ctcbeam_decode_nbest.restype = I
    lib.ctcbeam_decode_nbest.argtypes = dec + [P]
    lib.ctcbeam_greedy_decode.restype = I
    lib.ctcbeam_greedy_decode.argtypes = [P, P, I, I, I, F, F, F, P, P, P, ctypes.c_size_t, P, P, P, P, P]
    lib.ctcbeam_decode_noalloc.restype = I
    lib.ctcbeam_decode_noalloc.argtypes = [P, P, I, I, I, I, F, F, F, P, P, P, P, P, P, P]
    lib.ctcbeam_query_status.restype = I
    lib.ctcbeam_query_status.argtypes = [P, P, ctypes.POINTER(ctypes.c_uint32)]
    lib.ctcbeam_lm_tables.restype = I
    lib.ctcbeam_lm_tables.argtypes = [P, P]
    lib.ctcbeam_boost_tables.restype = I
    lib.ctcbeam_boost_tables.argtypes = [P, P]
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        raise CtcbeamError(rc, _load().ctcbeam_last_error().decode())


class _Opts(ctypes.Structure):
    _fields_ = [("prune_theta", ctypes.c_float), ("stats", ctypes.c_void_p),
                ("flags", ctypes.c_int), ("reserved", ctypes.c_int * 3)]


FLAG_LOGSUMEXP = 1        # CTCBEAM_FLAG_LOGSUMEXP
FLAG_BOOST_ROLLBACK = 2   # CTCBEAM_FLAG_BOOST_ROLLBACK
FLAG_NO_ROW_CACHE = 4     # CTCBEAM_FLAG_NO_ROW_CACHE
FLAG_REPEAT_SCORE = 8     # CTCBEAM_FLAG_REPEAT_SCORE


def _opts(theta, stats, B, logsumexp, boost_rollback, row_cache=True, device=None,
          repeat_score=False):
    """ctcbeam_opts by reference, or None when every option is at its default."""
    import torch
    flags = (FLAG_LOGSUMEXP if logsumexp else 0) | (FLAG_BOOST_ROLLBACK if boost_rollback else 0) | \
        (0 if row_cache else FLAG_NO_ROW_CACHE) | (FLAG_REPEAT_SCORE if repeat_score else 0)
    if (theta is None or math.isinf(theta)) and stats is None and flags == 0:
        return None
    o = _Opts()
    o.prune_theta = float(theta if theta is not None else math.inf)
    o.stats = None if stats is None else _dptr(stats, torch.int64, "stats", (B, 8), device).value
    o.flags = flags
    return o


class _LmView(ctypes.Structure):
    _fields_ = [("order", ctypes.c_int), ("vocab_size", ctypes.c_int), ("nlev", ctypes.c_int),
                ("n_states", ctypes.c_int64), ("n_arcs", ctypes.c_int64),
                ("states", ctypes.c_void_p), ("arcs", ctypes.c_void_p),
                ("unigram", ctypes.c_void_p)]


class _BoostView(ctypes.Structure):
    _fields_ = [("vocab_size", ctypes.c_int), ("n_nodes", ctypes.c_int64),
                ("n_list", ctypes.c_int64), ("nodes", ctypes.c_void_p),
                ("list", ctypes.c_void_p), ("root_key", ctypes.c_void_p)]


class LM:
    """Owning wrapper of a ``ctcbeam_lm*`` handle."""

    def __init__(self, handle: int, vocab_size: int):
        self._h = ctypes.c_void_p(handle)
        self.vocab_size = vocab_size

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h and self._h.value:
            _load().ctcbeam_lm_free(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Boost:
    """Owning wrapper of a ``ctcbeam_boost*`` handle."""

    def __init__(self, handle: int, vocab_size: int):
        self._h = ctypes.c_void_p(handle)
        self.vocab_size = vocab_size

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h and self._h.value:
            _load().ctcbeam_boost_free(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _lm_args(arrays: dict):
    order = int(arrays["order"])
    ids = [np.ascontiguousarray(a, dtype=np.int32) for a in arrays["ids"]]
    pr = [np.ascontiguousarray(a, dtype=np.float32) for a in arrays["log10_prob"]]
    bo = [None if a is None else np.ascontiguousarray(a, dtype=np.float32)
          for a in arrays["log10_bow"]]
    counts = np.asarray([a.shape[0] for a in ids], dtype=np.int64)
    ptr = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p).value  # noqa: E731
    keep = (ids, pr, bo, counts)
    ids_p = (ctypes.c_void_p * order)(*[ptr(a) for a in ids])
    pr_p = (ctypes.c_void_p * order)(*[ptr(a) for a in pr])
    bo_p = (ctypes.c_void_p * order)(*[ptr(a) for a in bo])
    return order, counts.ctypes.data_as(ctypes.c_void_p), ids_p, pr_p, bo_p, keep


def ctcbeam_lm_build(arrays: dict, host_only: bool = False) -> LM:
    """Build an LM from ARPA-style arrays: dict(order, V, ids=[int32 [n_m, m]],
    log10_prob=[f32 [n_m]], log10_bow=[f32 [n_m] or None])."""
    lib = _load()
    order, counts, ids_p, pr_p, bo_p, keep = _lm_args(arrays)
    out = ctypes.c_void_p()
    fn = lib.ctcbeam_lm_build_host if host_only else lib.ctcbeam_lm_build
    _check(fn(order, int(arrays["V"]), counts, ids_p, pr_p, bo_p, ctypes.byref(out)))
    del keep
    return LM(out.value, int(arrays["V"]))


def ctcbeam_lm_build_host(arrays: dict) -> LM:
    return ctcbeam_lm_build(arrays, host_only=True)


def ctcbeam_lm_build_arpa(path: str, vocab_size: int, host_only: bool = False) -> LM:
    lib = _load()
    fn = lib.ctcbeam_lm_build_arpa_host if host_only else lib.ctcbeam_lm_build_arpa
    out = ctypes.c_void_p()
    _check(fn(path.encode(), int(vocab_size), ctypes.byref(out)))
    return LM(out.value, int(vocab_size))


def ctcbeam_lm_build_arpa_host(path: str, vocab_size: int) -> LM:
    return ctcbeam_lm_build_arpa(path, vocab_size, host_only=True)


def ctcbeam_boost_build(vocab_size: int, offsets, tokens, host_only: bool = False) -> Boost:
    lib = _load()
    off = np.ascontiguousarray(offsets, dtype=np.int32)
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    if tok.size == 0:
        tok = np.zeros(1, dtype=np.int32)
    out = ctypes.c_void_p()
    fn = lib.ctcbeam_boost_build_host if host_only else lib.ctcbeam_boost_build
    _check(fn(int(vocab_size), int(off.shape[0] - 1), off.ctypes.data_as(ctypes.c_void_p),
              tok.ctypes.data_as(ctypes.c_void_p), ctypes.byref(out)))
    return Boost(out.value, int(vocab_size))


def ctcbeam_boost_build_host(vocab_size: int, offsets, tokens) -> Boost:
    return ctcbeam_boost_build(vocab_size, offsets, tokens, host_only=True)


def ctcbeam_lm_tables(lm: LM) -> dict:
    """Copies of the LM's host tables (see ``ctcbeam_lm_view``)."""
    v = _LmView()
    _check(_load().ctcbeam_lm_tables(lm.handle, ctypes.byref(v)))

    def arr(ptr, n, dt):
        if n == 0:
            return np.zeros(0, dtype=dt)
        return np.ctypeslib.as_array(ctypes.cast(ptr, ctypes.POINTER(
            ctypes.c_uint32 if dt == np.uint32 else ctypes.c_float)), shape=(n,)).copy()

    states = arr(v.states, v.n_states * v.nlev * 3, np.uint32).reshape(v.n_states, v.nlev, 3)
    arcs = arr(v.arcs, v.n_arcs * 3, np.uint32).reshape(v.n_arcs, 3)
    uni = arr(v.unigram, v.vocab_size + 1, np.float32)
    return dict(order=v.order, V=v.vocab_size, nlev=v.nlev, states=states, arcs=arcs, unigram=uni)


def ctcbeam_boost_tables(bt: Boost) -> dict:
    v = _BoostView()
    _check(_load().ctcbeam_boost_tables(bt.handle, ctypes.byref(v)))

    def arr(ptr, n):
        if n == 0:
            return np.zeros(0, dtype=np.uint32)
        return np.ctypeslib.as_array(ctypes.cast(ptr, ctypes.POINTER(ctypes.c_uint32)),
                                     shape=(n,)).copy()

    return dict(V=v.vocab_size, nodes=arr(v.nodes, v.n_nodes * 4).reshape(v.n_nodes, 4),
                list=arr(v.list, v.n_list * 2).reshape(v.n_list, 2),
                root_key=arr(v.root_key, v.vocab_size))


def ctcbeam_workspace_bytes(B: int, T: int, K: int) -> int:
    return int(_load().ctcbeam_workspace_bytes(int(B), int(T), int(K)))


def _dptr(t, dtype, name, shape=None, device=None):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the inputs on {device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _shape(logprobs):
    if logprobs.dim() != 3:
        raise ValueError("logprobs must be [B, T, V+1]")
    B, T, W = (int(x) for x in logprobs.shape)
    return B, T, W - 1, logprobs.device


def _stream_handle(stream, dev):
    """(raw hipStream_t, torch stream object or None) for ``stream``: None
    (torch's current stream on dev), a torch.cuda.Stream, or a raw handle."""
    import torch
    if stream is None:
        return torch.cuda.current_stream(dev).cuda_stream, None
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream, stream
    return int(stream), None


def _launch(call, dev, stream, owned):
    """Run ``call(raw_stream)`` (one C entry point, returning its code) with
    the inputs' device current.  Tensors the binding allocated (``owned``)
    are recorded on the launch stream when it is not torch's current stream,
    so the caching allocator does not hand their memory to other work before
    the kernel is done with it."""
    import torch
    with torch.cuda.device(dev):
        raw, obj = _stream_handle(stream, dev)
        _check(call(ctypes.c_void_p(raw)))
        if owned and raw != torch.cuda.current_stream(dev).cuda_stream:
            rec = obj if obj is not None else torch.cuda.ExternalStream(raw, device=dev)
            for t in owned:
                t.record_stream(rec)


def _handles(lm, boost):
    return (lm.handle if lm is not None else None, boost.handle if boost is not None else None)


def _alloc(t, shape, dtype, dev, owned):
    import torch
    if t is None:
        t = torch.empty(shape, dtype=dtype, device=dev)
        owned.append(t)
    return t


def ctcbeam_decode_ex(logprobs, lengths, K: int, alpha: float = 0.0, beta: float = 0.0,
                      boost_w: float = 0.0, lm: Optional[LM] = None,
                      boost: Optional[Boost] = None, workspace=None, out_tokens=None,
                      out_lengths=None, out_scores=None, stream=None,
                      theta: float = math.inf, stats=None, logsumexp: bool = False,
                      boost_rollback: bool = False, row_cache: bool = True,
                      repeat_score: bool = False):
    """Enqueue one decode on ``stream`` (default: torch's current stream on the
    inputs' device; a torch.cuda.Stream or a raw hipStream_t handle).

    logprobs: float32 [B, T, V+1] device tensor (blank = V); lengths: int32 [B].
    Outputs are allocated when not given.  ``row_cache=False`` sets
    CTCBEAM_FLAG_NO_ROW_CACHE (same results); ``repeat_score=True`` sets
    CTCBEAM_FLAG_REPEAT_SCORE.  Returns (tokens [B,T] int32
    with -1 padding, lengths [B] int32, scores [B] float32, workspace uint8)."""
    import torch
    lib = _load()
    B, T, V, dev = _shape(logprobs)
    owned = []
    out_tokens = _alloc(out_tokens, (B, T), torch.int32, dev, owned)
    out_lengths = _alloc(out_lengths, (B,), torch.int32, dev, owned)
    out_scores = _alloc(out_scores, (B,), torch.float32, dev, owned)
    workspace = _alloc(workspace, (max(ctcbeam_workspace_bytes(B, T, K), 1),), torch.uint8, dev, owned)
    o = _opts(theta, stats, B, logsumexp, boost_rollback, row_cache, dev, repeat_score)
    args = (_dptr(logprobs, torch.float32, "logprobs", None, dev),
            _dptr(lengths, torch.int32, "lengths", (B,), dev),
            B, T, V, int(K), float(alpha), float(beta), float(boost_w), *_handles(lm, boost),
            _dptr(workspace, torch.uint8, "workspace", None, dev), int(workspace.numel()),
            _dptr(out_tokens, torch.int32, "out_tokens", (B, T), dev),
            _dptr(out_lengths, torch.int32, "out_lengths", (B,), dev),
            _dptr(out_scores, torch.float32, "out_scores", (B,), dev))
    _launch(lambda st: lib.ctcbeam_decode_ex(*args, st, None if o is None else ctypes.byref(o)),
            dev, stream, owned)
    return out_tokens, out_lengths, out_scores, workspace


def ctcbeam_decode(logprobs, lengths, K: int, alpha: float = 0.0, beta: float = 0.0,
                   boost_w: float = 0.0, lm: Optional[LM] = None, boost: Optional[Boost] = None,
                   workspace=None, out_tokens=None, out_lengths=None, out_scores=None,
                   stream=None):
    """``ctcbeam_decode_ex`` without options (no pruning, no statistics)."""
    return ctcbeam_decode_ex(logprobs, lengths, K, alpha, beta, boost_w, lm, boost, workspace,
                             out_tokens, out_lengths, out_scores, stream)


def ctcbeam_decode_nbest(logprobs, lengths, K: int, alpha: float = 0.0, beta: float = 0.0,
                         boost_w: float = 0.0, lm: Optional[LM] = None,
                         boost: Optional[Boost] = None, workspace=None, nbest_tokens=None,
                         nbest_lengths=None, nbest_scores=None, stream=None,
                         theta: float = math.inf, stats=None, logsumexp: bool = False,
                         boost_rollback: bool = False, row_cache: bool = True,
                         repeat_score: bool = False):
    """Enqueue one N-best decode on ``stream`` (as for ``ctcbeam_decode_ex``).

    Same inputs as ``ctcbeam_decode_ex``.  Returns (tokens [B,K,T] int32 with
    -1 padding, lengths [B,K] int32, scores [B,K] float32 descending,
    workspace uint8); row 0 of each utterance is the 1-best result."""
    import torch
    lib = _load()
    B, T, V, dev = _shape(logprobs)
    K = int(K)
    owned = []
    nbest_tokens = _alloc(nbest_tokens, (B, K, T), torch.int32, dev, owned)
    nbest_lengths = _alloc(nbest_lengths, (B, K), torch.int32, dev, owned)
    nbest_scores = _alloc(nbest_scores, (B, K), torch.float32, dev, owned)
    workspace = _alloc(workspace, (max(ctcbeam_workspace_bytes(B, T, K), 1),), torch.uint8, dev, owned)
    o = _opts(theta, stats, B, logsumexp, boost_rollback, row_cache, dev, repeat_score)
    args = (_dptr(logprobs, torch.float32, "logprobs", None, dev),
            _dptr(lengths, torch.int32, "lengths", (B,), dev),
            B, T, V, K, float(alpha), float(beta), float(boost_w), *_handles(lm, boost),
            _dptr(workspace, torch.uint8, "workspace", None, dev), int(workspace.numel()),
            _dptr(nbest_tokens, torch.int32, "nbest_tokens", (B, K, T), dev),
            _dptr(nbest_lengths, torch.int32, "nbest_lengths", (B, K), dev),
            _dptr(nbest_scores, torch.float32, "nbest_scores", (B, K), dev))
    _launch(lambda st: lib.ctcbeam_decode_nbest(*args, st, None if o is None else ctypes.byref(o)),
            dev, stream, owned)
    return nbest_tokens, nbest_lengths, nbest_scores, workspace


def ctcbeam_greedy_decode(logprobs, lengths, alpha: float = 0.0, beta: float = 0.0,
                          boost_w: float = 0.0, lm: Optional[LM] = None,
                          boost: Optional[Boost] = None, workspace=None, out_tokens=None,
                          out_lengths=None, out_scores=None, stream=None, stats=None,
                          boost_rollback: bool = False, repeat_score: bool = False):
    """Enqueue one greedy decode with fusion (Algorithm 1 with one hypothesis)
    on ``stream``.  Returns (tokens [B,T] int32 with -1 padding, lengths [B],
    scores [B], workspace uint8)."""
    import torch
    lib = _load()
    B, T, V, dev = _shape(logprobs)
    owned = []
    out_tokens = _alloc(out_tokens, (B, T), torch.int32, dev, owned)
    out_lengths = _alloc(out_lengths, (B,), torch.int32, dev, owned)
    out_scores = _alloc(out_scores, (B,), torch.float32, dev, owned)
    workspace = _alloc(workspace, (max(ctcbeam_workspace_bytes(B, 0, 1), 1),), torch.uint8, dev, owned)
    o = _opts(math.inf, stats, B, False, boost_rollback, True, dev, repeat_score)
    args = (_dptr(logprobs, torch.float32, "logprobs", None, dev),
            _dptr(lengths, torch.int32, "lengths", (B,), dev),
            B, T, V, float(alpha), float(beta), float(boost_w), *_handles(lm, boost),
            _dptr(workspace, torch.uint8, "workspace", None, dev), int(workspace.numel()),
            _dptr(out_tokens, torch.int32, "out_tokens", (B, T), dev),
            _dptr(out_lengths, torch.int32, "out_lengths", (B,), dev),
            _dptr(out_scores, torch.float32, "out_scores", (B,), dev))
    _launch(lambda st: lib.ctcbeam_greedy_decode(*args, st, None if o is None else ctypes.byref(o)),
            dev, stream, owned)
    return out_tokens, out_lengths, out_scores, workspace


NOALLOC_MAX_WORKSPACE = 16 << 20   # CTCBEAM_NOALLOC_MAX_WORKSPACE


def ctcbeam_decode_noalloc(logprobs, lengths, K: int, alpha: float = 0.0, beta: float = 0.0,
                           boost_w: float = 0.0, lm: Optional[LM] = None,
                           boost: Optional[Boost] = None, out_tokens=None, out_lengths=None,
                           out_scores=None, stream=None, theta: float = math.inf, stats=None,
                           logsumexp: bool = False, boost_rollback: bool = False,
                           row_cache: bool = True, repeat_score: bool = False):
    """``ctcbeam_decode_ex`` through the entry point that allocates nothing:
    the workspace is the library's fixed per-device array (calls that overlap
    on one device race).  Pass the outputs to keep the call allocation-free
    (they are allocated here when not given).  Returns (tokens, lengths,
    scores)."""
    import torch
    lib = _load()
    B, T, V, dev = _shape(logprobs)
    owned = []
    out_tokens = _alloc(out_tokens, (B, T), torch.int32, dev, owned)
    out_lengths = _alloc(out_lengths, (B,), torch.int32, dev, owned)
    out_scores = _alloc(out_scores, (B,), torch.float32, dev, owned)
    o = _opts(theta, stats, B, logsumexp, boost_rollback, row_cache, dev, repeat_score)
    args = (_dptr(logprobs, torch.float32, "logprobs", None, dev),
            _dptr(lengths, torch.int32, "lengths", (B,), dev),
            B, T, V, int(K), float(alpha), float(beta), float(boost_w), *_handles(lm, boost),
            _dptr(out_tokens, torch.int32, "out_tokens", (B, T), dev),
            _dptr(out_lengths, torch.int32, "out_lengths", (B,), dev),
            _dptr(out_scores, torch.float32, "out_scores", (B,), dev))
    _launch(lambda st: lib.ctcbeam_decode_noalloc(*args, st, None if o is None else ctypes.byref(o)),
            dev, stream, owned)
    return out_tokens, out_lengths, out_scores


def ctcbeam_query_status(workspace, stream=None) -> int:
    """Status bits (ORed over utterances) of the last decode that used
    ``workspace``; synchronises ``stream`` (default: torch's current one)."""
    import torch
    dev = workspace.device
    bits = ctypes.c_uint32(0)
    with torch.cuda.device(dev):
        raw, _ = _stream_handle(stream, dev)
        _check(_load().ctcbeam_query_status(ctypes.c_void_p(workspace.data_ptr()),
                                            ctypes.c_void_p(raw), ctypes.byref(bits)))
    return int(bits.value)


def decode(logprobs, lengths, K: int, **kw):
    """Convenience: returns (tokens, lengths, scores) device tensors."""
    tok, ln, sc, _ = ctcbeam_decode_ex(logprobs, lengths, K, **kw)
    return tok, ln, sc


def decode_nbest(logprobs, lengths, K: int, **kw):
    """Convenience: returns N-best (tokens [B,K,T], lengths [B,K], scores [B,K])."""
    tok, ln, sc, _ = ctcbeam_decode_nbest(logprobs, lengths, K, **kw)
    return tok, ln, sc
