"""CPU tests of the C-ABI library's host side (no GPU needed).

* the library loads and exports every function declared in include/ctcbeam.h;
* the LM builder's tables, walked by a test-side reader that follows the
  kernel's fill rule (highest-order explicit arc wins, backoff weights of the
  higher orders added innermost first), reproduce the oracle's LM value for
  every token and </s> at many histories - bit for bit;
* the boosting builder's merged continuation lists reproduce the oracle's
  per-token boosting scores along random token streams;
* invalid inputs are rejected with the documented codes before any device
  call.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
import paper_2508_07315_amd as P
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
F32 = np.float32


@pytest.fixture(scope="session", autouse=True)
def built_library():
    if not os.path.exists(P.library_path()):
        from paper_2508_07315_amd import build_lib
        build_lib.build()
    return P.library_path()


def test_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "ctcbeam.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    names = set(re.findall(r"\b(ctcbeam_[a-z_]+)\s*\(", hdr))
    assert len(names) >= 15, names
    lib = ctypes.CDLL(P.library_path())
    missing = [n for n in sorted(names) if not hasattr(lib, n)]
    assert not missing, missing


def test_flag_values_match_the_header():
    # the binding's option bits are the header's CTCBEAM_FLAG_* values
    hdr = open(os.path.join(ROOT, "include", "ctcbeam.h")).read()
    flags = {m.group(1): int(m.group(2)) for m in re.finditer(r"#define CTCBEAM_FLAG_(\w+)\s+(\d+)", hdr)}
    assert flags == {"LOGSUMEXP": P.FLAG_LOGSUMEXP, "BOOST_ROLLBACK": P.FLAG_BOOST_ROLLBACK,
                     "NO_ROW_CACHE": P.FLAG_NO_ROW_CACHE,
                     "REPEAT_SCORE": P.FLAG_REPEAT_SCORE}, flags
    assert len(set(flags.values())) == len(flags)
    assert all(v & (v - 1) == 0 for v in flags.values())  # one bit each


# ---------------------------------------------------------------------------
# LM tables
# ---------------------------------------------------------------------------
class LmWalker:
    def __init__(self, tab):
        self.t = tab
        self.V = tab["V"]
        self.nlev = tab["nlev"]

    def level(self, s, l):
        rec = self.t["states"][s, l]
        return int(rec[0]), int(rec[1] & 0x7FFFFFFF), bool(rec[1] >> 31), rec[2:3].view(np.float32)[0]

    def arc(self, begin, cnt, c):
        a = self.t["arcs"][begin: begin + cnt]
        hit = np.nonzero(a[:, 2] == c)[0]
        if len(hit) == 0:
            return None
        row = a[hit[0]]
        return row[0:1].view(np.float32)[0], int(row[1])

    def value(self, s, c):
        bos = [self.level(s, l)[3] for l in range(self.nlev)]
        for l in range(self.nlev - 1, -1, -1):
            b, n, _, _ = self.level(s, l)
            a = self.arc(b, n, c)
            if a is not None:
                v = F32(a[0])
                for l2 in range(l + 1, self.nlev):
                    v = F32(v + bos[l2])
                return v
        v = F32(self.t["unigram"][c])
        for l in range(self.nlev):
            v = F32(v + bos[l])
        return v

    def next(self, s, c):
        for l in range(self.nlev - 1, -1, -1):
            b, n, _, _ = self.level(s, l)
            a = self.arc(b, n, c)
            if a is not None:
                return a[1]
        return c

    def state(self, y):
        s = self.V
        for c in y:
            s = self.next(s, c)
        return s


@pytest.mark.parametrize("order,V,density", [(1, 5, 0.5), (2, 6, 0.5), (3, 5, 0.4), (4, 4, 0.5)])
def test_lm_tables_match_oracle_small(order, V, density):
    rng = np.random.default_rng(order * 10 + V)
    arrays = W.random_small_lm(rng, order, V, density=density)
    ref = oracle.LM(arrays)
    walker = LmWalker(P.ctcbeam_lm_tables(P.ctcbeam_lm_build_host(arrays)))
    for _ in range(150):
        y = rng.integers(0, V, size=int(rng.integers(0, 8))).tolist()
        s = walker.state(y)
        for c in range(V + 1):
            assert walker.value(s, c) == F32(ref.score(y, c)), (y, c)


def test_lm_tables_match_oracle_3gram_config():
    """The 3-gram LM of the B=64 workload (300k bigrams, 1M trigrams)."""
    w = W.CONFIGS[3]
    arrays = W.lm_for(w.lm, w.V)
    ref = oracle.LM(arrays)
    tab = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_host(arrays))
    assert tab["states"].shape == (1025 + 300_000 - np.sum(arrays["ids"][1][:, 1] == w.V), 2, 3)
    walker = LmWalker(tab)
    rng = np.random.default_rng(0)
    bigrams = arrays["ids"][1]
    for _ in range(6):
        # follow explicit bigrams so the history reaches trigram contexts
        a = int(rng.integers(0, w.V))
        y = [a]
        for _ in range(4):
            nxt = bigrams[(bigrams[:, 0] == y[-1]) & (bigrams[:, 1] < w.V)][:, 1]
            y.append(int(rng.choice(nxt)) if len(nxt) else int(rng.integers(0, w.V)))
        s = walker.state(y)
        cs = rng.choice(w.V + 1, size=64, replace=False)
        for c in cs:
            assert walker.value(s, int(c)) == F32(ref.score(y, int(c))), (y, c)


def test_arpa_builder_matches_arrays():
    V = 3
    path = os.path.join(ROOT, "tests", "golden", "toy3.arpa")
    a = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_arpa_host(path, V))
    b = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_host(W.read_arpa(path, V)))
    for k in ("states", "arcs", "unigram"):
        np.testing.assert_array_equal(a[k], b[k])
    ref = oracle.LM(W.read_arpa(path, V))
    walker = LmWalker(a)
    for y in ([], [0], [0, 1], [0, 1, 2], [2, 2, 1]):
        for c in range(V + 1):
            assert walker.value(walker.state(y), c) == F32(ref.score(y, c))


def test_arpa_reader_formatting_and_errors(tmp_path):
    """The ARPA reader takes CRLF line ends, blank lines, tabs and skips
    n-grams with a word outside the vocabulary; a line with too few fields
    is an error.  A large file is parsed in parallel parts and still equals
    the array build."""
    V = 40
    arrays = W.make_lm(3, V, [600, 900], 77)
    clean = tmp_path / "clean.arpa"
    W.write_arpa(arrays, str(clean))
    text = clean.read_text()
    lines = text.split("\n")
    messy = []
    for i, ln in enumerate(lines):
        if ln and ln[0] not in "\\n" and i % 7 == 0:
            ln = ln.replace(" ", "\t", 1)
        messy.append(ln + ("\r" if i % 3 == 0 else ""))
        if i % 11 == 0:
            messy.append("")
    # an n-gram with an unknown word, inside the 2-gram section
    k = next(i for i, ln in enumerate(messy) if ln.rstrip("\r") == "\\2-grams:")
    messy.insert(k + 1, "-1.5 99999 3 -0.2")
    path = tmp_path / "messy.arpa"
    path.write_text("\n".join(messy))
    a = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_arpa_host(str(path), V))
    b = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_host(arrays))
    for key in ("states", "arcs", "unigram"):
        np.testing.assert_array_equal(a[key], b[key])
    bad = tmp_path / "bad.arpa"
    bad.write_text(text.replace("\\2-grams:\n", "\\2-grams:\n-1.0 5\n", 1))
    with pytest.raises(P.CtcbeamError) as e:
        P.ctcbeam_lm_build_arpa_host(str(bad), V)
    assert e.value.code == 1 and "malformed" in str(e.value)
    # several MB: parsed in parts, identical to the array build
    big = W.make_lm(3, 1024, [60000, 150000], 78)
    bigp = tmp_path / "big.arpa"
    W.write_arpa(big, str(bigp))
    a = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_arpa_host(str(bigp), 1024))
    b = P.ctcbeam_lm_tables(P.ctcbeam_lm_build_host(big))
    for key in ("states", "arcs", "unigram"):
        np.testing.assert_array_equal(a[key], b[key])


# ---------------------------------------------------------------------------
# Boosting tables
# ---------------------------------------------------------------------------
def bt_step(tab, q, c):
    lb, lc, potw, _ = (int(x) for x in tab["nodes"][q])
    pot = potw & 0xFF
    lst = tab["list"][lb: lb + lc]
    hit = np.nonzero(lst[:, 0] == c)[0]
    key = int(lst[hit[0], 1]) if len(hit) else int(tab["root_key"][c])
    pre = (key >> 20) & 63
    return pre - pot, key & 0xFFFFF


def _stream(rng, phrases, V, n):
    out = []
    while len(out) < n:
        if rng.random() < 0.6 and phrases:
            p = phrases[int(rng.integers(0, len(phrases)))]
            cut = int(rng.integers(1, len(p) + 1))
            out.extend(p[:cut])
        else:
            out.append(int(rng.integers(0, V)))
    return out[:n]


@pytest.mark.parametrize("seed", range(6))
def test_boost_tables_match_oracle(seed):
    rng = np.random.default_rng(seed)
    V = int(rng.integers(3, 9))
    n = int(rng.integers(1, 12))
    phrases = [rng.integers(0, V, size=int(rng.integers(1, 6))).tolist() for _ in range(n)]
    off = np.concatenate([[0], np.cumsum([len(p) for p in phrases])]).astype(np.int32)
    toks = np.asarray([t for p in phrases for t in p], dtype=np.int32)
    ref = oracle.BT(V, off, toks)
    tab = P.ctcbeam_boost_tables(P.ctcbeam_boost_build_host(V, off, toks))
    for _ in range(20):
        seq = _stream(rng, phrases, V, 30)
        q_ref, q = [], 0
        for c in seq:
            s_ref, q_ref = ref.step(q_ref, c)
            s, q = bt_step(tab, q, c)
            assert s == s_ref
            assert (int(tab["nodes"][q][2]) & 0xFF) == ref.pot(q_ref)


def test_boost_tables_config5_phrases():
    w = W.CONFIGS[5]
    off, toks = W.phrases_for(w.boost, w.V)
    ref = oracle.BT(w.V, off, toks)
    tab = P.ctcbeam_boost_tables(P.ctcbeam_boost_build_host(w.V, off, toks))
    phrases = [toks[off[i]: off[i + 1]].tolist() for i in range(len(off) - 1)]
    rng = np.random.default_rng(1)
    seq = _stream(rng, phrases, w.V, 400)
    q_ref, q = [], 0
    for c in seq:
        s_ref, q_ref = ref.step(q_ref, c)
        s, q = bt_step(tab, q, c)
        assert s == s_ref


# ---------------------------------------------------------------------------
# Argument checking (no device call is reached)
# ---------------------------------------------------------------------------
def _err(fn, *a):
    with pytest.raises(P.CtcbeamError) as e:
        fn(*a)
    return e.value.code


def test_lm_builder_rejects_bad_models():
    rng = np.random.default_rng(3)
    V = 4
    good = W.random_small_lm(rng, 3, V, density=0.5)
    assert P.ctcbeam_lm_build_host(good) is not None

    def variant(**kw):
        d = {k: (list(v) if isinstance(v, list) else v) for k, v in good.items()}
        d.update(kw)
        return d

    # a token without a unigram
    ids1 = good["ids"][0]
    keep = ids1[:, 0] != 2
    bad = variant(ids=[ids1[keep]] + good["ids"][1:],
                  log10_prob=[good["log10_prob"][0][keep]] + good["log10_prob"][1:],
                  log10_bow=[good["log10_bow"][0][keep]] + good["log10_bow"][1:])
    assert _err(P.ctcbeam_lm_build_host, bad) == 1
    # duplicate bigram
    i2 = good["ids"][1]
    bad = variant(ids=[good["ids"][0], np.concatenate([i2, i2[:1]]), good["ids"][2]],
                  log10_prob=[good["log10_prob"][0], np.concatenate([good["log10_prob"][1], [-1.0]]).astype(np.float32),
                              good["log10_prob"][2]],
                  log10_bow=[good["log10_bow"][0], np.concatenate([good["log10_bow"][1], [0.0]]).astype(np.float32), None])
    assert _err(P.ctcbeam_lm_build_host, bad) == 1
    # a trigram whose context is not a bigram
    present = {tuple(r) for r in i2.tolist()}
    ctx = next((a, b) for a in range(V) for b in range(V) if (a, b) not in present)
    bad = variant(ids=[good["ids"][0], i2, np.concatenate([good["ids"][2], [[ctx[0], ctx[1], 0]]]).astype(np.int32)],
                  log10_prob=[good["log10_prob"][0], good["log10_prob"][1],
                              np.concatenate([good["log10_prob"][2], [-1.0]]).astype(np.float32)])
    assert _err(P.ctcbeam_lm_build_host, bad) == 1
    # </s> inside an n-gram, <s> not first
    bad = variant(ids=[good["ids"][0], np.concatenate([i2, [[V, 1]]]).astype(np.int32), good["ids"][2]],
                  log10_prob=[good["log10_prob"][0], np.concatenate([good["log10_prob"][1], [-1.0]]).astype(np.float32),
                              good["log10_prob"][2]],
                  log10_bow=[good["log10_bow"][0], np.concatenate([good["log10_bow"][1], [0.0]]).astype(np.float32), None])
    assert _err(P.ctcbeam_lm_build_host, bad) == 1
    bad["ids"][1][-1] = [1, V + 1]
    assert _err(P.ctcbeam_lm_build_host, bad) == 1
    # order and vocabulary limits
    big = W.random_small_lm(rng, 2, 3)
    big["V"] = P.MAX_V + 1
    assert _err(P.ctcbeam_lm_build_host, big) == 2


def test_boost_builder_rejects_bad_lists():
    assert _err(P.ctcbeam_boost_build_host, 4, [0, 2], [1, 4]) == 1       # token out of range
    assert _err(P.ctcbeam_boost_build_host, 4, [0, 2, 1], [1, 2]) == 1    # decreasing offsets
    assert _err(P.ctcbeam_boost_build_host, 4, [0, 63], [1] * 63) == 2    # phrase too long
    # empty list and empty phrases are fine
    P.ctcbeam_boost_build_host(4, [0], [])
    P.ctcbeam_boost_build_host(4, [0, 0, 2], [1, 2])


def test_decode_rejects_bad_arguments_before_any_device_call():
    lib = ctypes.CDLL(P.library_path())
    P._load()
    fake = ctypes.c_void_p(0x1000)
    null = ctypes.c_void_p(None)
    ws = P.ctcbeam_workspace_bytes(2, 3, 4)
    dec = P._load().ctcbeam_decode_ex

    def call(B=2, T=3, V=5, K=4, lm=None, bt=None, ws_bytes=ws, lp=fake, opts=None, alpha=0.0,
             wsp=fake):
        return dec(lp, fake, B, T, V, K, alpha, 0.0, 0.0, lm, bt, wsp, ws_bytes, fake, null, fake,
                   null, opts)

    assert call(K=0) == 1
    assert call(K=P.MAX_K + 1) == 2
    assert call(K=65, V=1025, ws_bytes=P.ctcbeam_workspace_bytes(2, 3, 65)) == 2  # wide V, K > 64
    assert call(V=0) == 1
    assert call(V=P.MAX_V + 1) == 2
    assert call(B=-1) == 1
    assert call(ws_bytes=ws - 1) == 1
    assert call(lp=null) == 1
    assert call(alpha=float("nan")) == 1
    # B = 0 without a workspace: nothing to do, nothing launched (with one,
    # a one-thread kernel records the empty batch in its header)
    assert call(B=0, wsp=null) == 0
    rng = np.random.default_rng(0)
    lm = P.ctcbeam_lm_build_host(W.random_small_lm(rng, 2, 5))
    assert call(lm=lm.handle) == 1            # host-only handle
    lm6 = P.ctcbeam_lm_build_host(W.random_small_lm(rng, 2, 6))
    assert call(lm=lm6.handle) == 1           # vocabulary mismatch
    o = P._Opts()
    o.prune_theta = -1.0
    assert call(opts=ctypes.byref(o)) == 1
    assert b"prune_theta" in P._load().ctcbeam_last_error()
    assert P.ctcbeam_workspace_bytes(64, 400, 8) >= 64 * 400 * 8 * 4
    del lib


def test_workspace_bytes_formula():
    for B, T, K in [(1, 1, 1), (64, 400, 8), (128, 1000, 16), (3, 0, 5)]:
        n = P.ctcbeam_workspace_bytes(B, T, K)
        assert n >= B * T * K * 4 + B * 4
        assert n - B * T * K * 4 <= 4 * B + 256 + 256  # status words + header
    assert P.ctcbeam_workspace_bytes(0, 0, 1) == 256  # the header alone


def test_query_status_signature_matches_the_boundary():
    """ctcbeam_query_status(const void* workspace, hipStream_t stream,
    uint32_t* bits): the batch size comes from the workspace header."""
    hdr = open(os.path.join(ROOT, "include", "ctcbeam.h")).read()
    m = re.search(r"int\s+ctcbeam_query_status\s*\(([^)]*)\)", hdr)
    assert m, "ctcbeam_query_status is not declared"
    params = [" ".join(a.split()) for a in m.group(1).split(",")]
    assert params == ["const void* workspace", "hipStream_t stream", "uint32_t* bits"], params
    lib = P._load()
    assert len(lib.ctcbeam_query_status.argtypes) == 3
    # no device call is made for a null workspace
    bits = ctypes.c_uint32(7)
    assert lib.ctcbeam_query_status(None, None, ctypes.byref(bits)) == 1
