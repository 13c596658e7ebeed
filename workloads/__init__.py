"""Seeded synthetic inputs for the batched CTC beam-search frame step.

This module only *draws inputs*: CTC log-probabilities, valid lengths,
backoff n-gram tables (as ARPA-style arrays of log10 values) and boosting
phrase lists.  It holds none of the decoder's arithmetic, so both the CPU
oracle and the HIP path can be fed from it without sharing any code.

The shapes follow the paper's workloads: a BPE vocabulary of 1024 tokens plus
blank (Sec. IV-A "Models"), batches of 32-128 utterances and beams of 4-128
(Tables "tab:custom"/"tab:strategies", Figs. "batch_size_vs_rtfx" and
"beam_size_vs_wer"), ~1000 boosted phrases (Sec. IV-B "Datasets"), subword
n-gram LMs used through ARPA files (Sec. IV-A).  The datasets, the trained
acoustic model and the paper's KenLM files are not available; these seeded
draws stand in for them.

Conventions shared with the decoder's interface:
  * labels 0..V-1 are tokens, label V is blank; a frame row has W = V+1 values;
  * LM ids: 0..V-1 tokens, V = ``</s>``, V+1 = ``<s>``.

Random streams (numpy ``default_rng``):
  * config i's lengths: ``default_rng(1000+i)``; utterance b's logits:
    ``default_rng([1000+i, b+1])`` (so any subset of utterances can be drawn
    on its own);
  * config i's LM: ``default_rng(2000+i)``; phrases: ``default_rng(3000+i)``.
"""
from __future__ import annotations

import dataclasses
import math
from functools import lru_cache
from typing import Optional, Sequence

import numpy as np

ZIPF_S = 1.1


# ----------------------------------------------------------------------------
# Workload descriptions
# ----------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LMSpec:
    order: int
    counts: tuple          # explicit n-gram counts for orders 2..order
    seed: int


@dataclasses.dataclass(frozen=True)
class BoostSpec:
    n_phrases: int
    min_len: int
    max_len: int
    token_dist: str        # "uniform" or "zipf"
    seed: int


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    T: int
    V: int
    K: int
    logits: str            # "gauss3" (N(0,3^2)) or "peaky" (blank/peak recipe)
    lengths: tuple         # ("fixed", (l0, l1, ...)) or ("uniform", lo, hi)
    seed: int              # logprob/length seed (1000+i)
    alpha: float = 0.0
    beta: float = 0.0
    boost_w: float = 0.0
    theta: float = math.inf
    lm: Optional[LMSpec] = None
    boost: Optional[BoostSpec] = None

    @property
    def W(self) -> int:
        return self.V + 1

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


LM3 = LMSpec(order=3, counts=(300_000, 1_000_000), seed=2003)
LM4 = LMSpec(order=4, counts=(500_000, 3_000_000, 6_000_000), seed=2004)
# paper-scale subword 6-gram (Sec. IV-A uses KenLM 6-grams): 11.0 M n-grams
LM6 = LMSpec(order=6, counts=(500_000, 2_000_000, 3_000_000, 3_000_000, 2_500_000), seed=2006)

CONFIGS = {
    1: Workload("cfg1_B2_T50_V32_K4", B=2, T=50, V=32, K=4, logits="gauss3",
                lengths=("fixed", (50, 37)), seed=1001),
    2: Workload("cfg2_B32_T400_V1024_K8", B=32, T=400, V=1024, K=8, logits="peaky",
                lengths=("uniform", 200, 400), seed=1002),
    3: Workload("cfg3_B64_T400_V1024_K8_lm3", B=64, T=400, V=1024, K=8, logits="peaky",
                lengths=("uniform", 200, 400), seed=1003, alpha=0.5, beta=1.0, lm=LM3),
    4: Workload("cfg4_B128_T1000_V1024_K16_lm4_pb1000", B=128, T=1000, V=1024, K=16,
                logits="peaky", lengths=("uniform", 500, 1000), seed=1004,
                alpha=0.5, beta=1.0, boost_w=1.0, lm=LM4,
                boost=BoostSpec(1000, 2, 6, "uniform", 3004)),
    5: Workload("cfg5_B64_T400_V1024_K64_lm3_pb5000", B=64, T=400, V=1024, K=64,
                logits="peaky", lengths=("uniform", 100, 400), seed=1005,
                alpha=0.5, beta=1.0, boost_w=1.5, lm=LM3,
                boost=BoostSpec(5000, 2, 8, "zipf", 3005)),
    # paper scale (Sec. V-C, Fig. "beam_size_vs_wer": batch 32, LM + PB,
    # beams 4..128; Sec. IV-D: theta = 12): a 6-gram with 11 M n-grams
    6: Workload("cfg6_B32_T400_V1024_K16_lm6_pb1000", B=32, T=400, V=1024, K=16,
                logits="peaky", lengths=("uniform", 200, 400), seed=1006,
                alpha=0.5, beta=1.0, boost_w=1.0, theta=12.0, lm=LM6,
                boost=BoostSpec(1000, 2, 6, "uniform", 3006)),
}


# ----------------------------------------------------------------------------
# Log-probabilities and lengths
# ----------------------------------------------------------------------------
def make_lengths(w: Workload) -> np.ndarray:
    kind = w.lengths[0]
    if kind == "fixed":
        out = np.asarray(w.lengths[1], dtype=np.int32)
        assert out.shape == (w.B,)
        return out
    lo, hi = w.lengths[1], w.lengths[2]
    rng = np.random.default_rng(w.seed)
    return rng.integers(lo, hi + 1, size=w.B).astype(np.int32)


def _log_softmax64(x: np.ndarray) -> np.ndarray:
    m = x.max(axis=-1, keepdims=True)
    s = np.log(np.exp(x - m).sum(axis=-1, keepdims=True))
    return x - m - s


def make_utterance_logprobs(w: Workload, b: int) -> np.ndarray:
    """fp32 [T, V+1] log-probabilities of utterance b (drawn in fp64)."""
    rng = np.random.default_rng([w.seed, b + 1])
    T, V, W = w.T, w.V, w.V + 1
    if w.logits == "gauss3":
        logits = rng.normal(0.0, 3.0, size=(T, W))
    elif w.logits == "peaky":
        logits = rng.normal(0.0, 2.0, size=(T, W))
        blank_frame = rng.random(T) < 0.7
        peak = rng.integers(0, V, size=T)
        logits[blank_frame, V] += 4.0
        nb = ~blank_frame
        logits[np.nonzero(nb)[0], peak[nb]] += 3.0
    else:
        raise ValueError(w.logits)
    return _log_softmax64(logits).astype(np.float32)


def make_logprobs(w: Workload, utterances: Optional[Sequence[int]] = None) -> np.ndarray:
    """fp32 [n, T, V+1] for the given utterance indices (default: all B)."""
    idx = range(w.B) if utterances is None else utterances
    out = np.empty((len(idx), w.T, w.V + 1), dtype=np.float32)
    for i, b in enumerate(idx):
        out[i] = make_utterance_logprobs(w, b)
    return out


# ----------------------------------------------------------------------------
# Backoff n-gram LM (ARPA-style arrays, log10 values)
# ----------------------------------------------------------------------------
def _zipf_weights(n: int, rng: np.random.Generator) -> np.ndarray:
    """Zipf(1.1) weights over a seeded random ranking of n items (sum 1)."""
    rank = rng.permutation(n)
    z = (rank + 1.0) ** (-ZIPF_S)
    return z / z.sum()


def _waterfill(r: np.ndarray, caps: np.ndarray, total: int) -> np.ndarray:
    """Integer counts ~ proportional to r, capped at caps, summing to total
    (or to caps.sum() if that is smaller)."""
    caps = caps.astype(np.int64)
    total = int(min(total, caps.sum()))
    if total == 0:
        return np.zeros_like(caps)
    lo, hi = 0.0, float(total) / float(r[caps > 0].min()) + 1.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if np.minimum(caps, mid * r).sum() >= total:
            hi = mid
        else:
            lo = mid
    c = np.minimum(caps, np.floor(hi * r)).astype(np.int64)
    deficit = total - int(c.sum())
    order = np.argsort(-r, kind="stable")
    while deficit > 0:
        room = order[c[order] < caps[order]]
        take = room[:deficit]
        c[take] += 1
        deficit -= len(take)
    while deficit < 0:  # can only happen through floor rounding at the caps
        over = order[::-1][c[order[::-1]] > 0][: -deficit]
        c[over] -= 1
        deficit += len(over)
    return c


def _encode(ids: np.ndarray, base: int) -> np.ndarray:
    """Integer code of each row of ids (row-major digits in `base`)."""
    code = np.zeros(ids.shape[0], dtype=np.int64)
    for j in range(ids.shape[1]):
        code = code * base + ids[:, j].astype(np.int64)
    return code


def _race_topk(rng, ctxs, group_start, group_len, items, weights, counts, chunk=8_000_000):
    """Exponential-race (Efraimidis-Spirakis) selection: for each context in
    ctxs (ascending) keep the counts[ctx] admissible items with the largest
    log(u)/weight keys.  Processed in chunks of contexts to bound memory."""
    out_c, out_i = [], []
    lens_all = group_len[ctxs]
    bounds = [0]
    acc = 0
    for j, n in enumerate(lens_all.tolist()):
        acc += n
        if acc >= chunk:
            bounds.append(j + 1)
            acc = 0
    if bounds[-1] != len(ctxs):
        bounds.append(len(ctxs))
    for a, b in zip(bounds[:-1], bounds[1:]):
        cs = ctxs[a:b]
        lens = group_len[cs]
        tot = int(lens.sum())
        if tot == 0:
            continue
        seg0 = np.repeat(np.cumsum(lens) - lens, lens)
        ctx_rep = np.repeat(cs, lens)
        within = np.arange(tot) - seg0
        it = items[np.repeat(group_start[cs], lens) + within]
        key = np.log(rng.random(tot)) / weights[it]
        order = np.lexsort((-key, ctx_rep))
        rank = within  # ctx_rep is already grouped in ascending context order
        keep = rank < np.repeat(counts[cs], lens)
        out_c.append(ctx_rep[order][keep])
        out_i.append(it[order][keep])
    if not out_c:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    return np.concatenate(out_c), np.concatenate(out_i)


def _sample_without_replacement(rng, n_ctx, group_start, group_len, items, weights,
                                counts, max_rounds=32):
    """For each context i pick counts[i] distinct items out of
    items[group_start[i] : group_start[i]+group_len[i]], Zipf-weighted without
    replacement (draws proportional to weight among the items not yet taken).
    Contexts that take their whole admissible set take it directly; contexts
    that take more than a quarter of it use an exponential race; the rest use
    batched draws with rejection of repeats (the same distribution), and any
    context still short after max_rounds is redone with the race."""
    counts = counts.astype(np.int64)
    picks_ctx, picks_item = [], []
    full = (counts >= group_len) & (counts > 0)
    fi = np.nonzero(full)[0]
    if len(fi):
        lens = group_len[fi]
        ctx = np.repeat(fi, lens)
        within = np.arange(len(ctx)) - np.repeat(np.cumsum(lens) - lens, lens)
        picks_ctx.append(ctx)
        picks_item.append(items[np.repeat(group_start[fi], lens) + within])
    dense = (~full) & (counts > 0) & (4 * counts > group_len)
    di = np.nonzero(dense)[0]
    if len(di):
        c, i = _race_topk(rng, di, group_start, group_len, items, weights, counts)
        picks_ctx.append(c)
        picks_item.append(i)
    todo = np.nonzero((~full) & (~dense) & (counts > 0))[0]
    if len(todo):
        cw = np.concatenate([[0.0], np.cumsum(weights[items].astype(np.float64))])
        base = int(items.max()) + 1
        acc = np.zeros(0, dtype=np.int64)
        got = np.zeros(n_ctx, dtype=np.int64)
        for _ in range(max_rounds):
            need = counts[todo] - got[todo]
            sel = need > 0
            if not sel.any():
                break
            ctx = np.repeat(todo[sel], need[sel])
            g0 = group_start[ctx]
            g1 = g0 + group_len[ctx]
            u = cw[g0] + rng.random(len(ctx)) * (cw[g1] - cw[g0])
            pos = np.clip(np.searchsorted(cw, u, side="right") - 1, g0, g1 - 1)
            code = ctx.astype(np.int64) * base + items[pos]
            _, first = np.unique(code, return_index=True)
            code = code[np.sort(first)]
            code = code[~np.isin(code, acc)]
            acc = np.concatenate([acc, code])
            got += np.bincount(code // base, minlength=n_ctx)
        short = todo[(counts[todo] - got[todo]) > 0]
        if len(short):
            acc = acc[~np.isin(acc // base, short)]
            c, i = _race_topk(rng, short, group_start, group_len, items, weights, counts)
            picks_ctx.append(c)
            picks_item.append(i)
        picks_ctx.append(acc // base)
        picks_item.append(acc % base)
    if not picks_ctx:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    return np.concatenate(picks_ctx), np.concatenate(picks_item)


def make_lm(order: int, V: int, counts: Sequence[int], seed: int) -> dict:
    """Synthetic backoff n-gram model as ARPA-style arrays.

    Recipe: unigrams for the V tokens and ``</s>`` get Zipf(1.1) probabilities
    over a seeded ranking; ``<s>`` gets log10 -99.  For order m >= 2 the
    explicit continuations per context are allocated by Zipf(1.1) over a
    seeded context ranking, capped at the admissible continuations and
    water-filled; they are drawn Zipf-weighted without replacement.  The model
    is suffix-closed ((h1..hm, w) admissible only if (h2..hm, w) exists) and
    prefix-closed (contexts are existing entries).  log10 p(w|h) =
    log10(m_h z_w / sum_{S_h} z) with m_h ~ U[0.5, 0.95]; log10 backoff
    weights ~ U[-1, 0] for every entry that can be a context.

    Returns dict(order, V, ids=[int32 [n_m, m]], log10_prob=[f32 [n_m]],
    log10_bow=[f32 [n_m]] for m < order (None for the top order)).
    """
    assert order >= 1 and len(counts) == order - 1
    rng = np.random.default_rng(seed)
    EOS, BOS = V, V + 1
    base = V + 2
    assert base ** order < 2 ** 62, "code space too small for this order/V"
    z = _zipf_weights(V + 1, rng)            # continuation weights (tokens + </s>)
    ids = [np.arange(V + 2, dtype=np.int32)[:, None]]
    p1 = np.empty(V + 2, dtype=np.float64)
    p1[: V + 1] = np.log10(z)
    p1[BOS] = -99.0
    probs = [p1]
    bows = []
    for m in range(2, order + 1):
        prev = ids[-1]                       # (m-1)-gram entries, sorted
        is_ctx = prev[:, -1] != EOS
        ctx = prev[is_ctx]
        n_ctx = ctx.shape[0]
        if m == 2:
            items = np.arange(V + 1, dtype=np.int64)
            group_start = np.zeros(n_ctx, dtype=np.int64)
            group_len = np.full(n_ctx, V + 1, dtype=np.int64)
        else:
            # admissible continuations of h = continuations of h[1:] at order m-1
            items = prev[:, -1].astype(np.int64)
            gcode = _encode(prev[:, :-1], base)          # sorted (entries are sorted)
            ucode, ustart, ulen = np.unique(gcode, return_index=True, return_counts=True)
            scode = _encode(ctx[:, 1:], base)
            j = np.searchsorted(ucode, scode)
            j = np.clip(j, 0, len(ucode) - 1)
            found = ucode[j] == scode
            group_start = np.where(found, ustart[j], 0).astype(np.int64)
            group_len = np.where(found, ulen[j], 0).astype(np.int64)
        r = _zipf_weights(n_ctx, rng)
        cnt = _waterfill(r, group_len, counts[m - 2])
        if m == 2:
            # dense rows: exponential-race keys (Efraimidis-Spirakis), one row per context
            keys = np.log(rng.random((n_ctx, V + 1))) / z[None, :]
            order_idx = np.argsort(-keys, axis=1, kind="stable")
            pc = np.repeat(np.arange(n_ctx), cnt)
            within = np.arange(len(pc)) - np.repeat(np.cumsum(cnt) - cnt, cnt)
            pi = order_idx[pc, within]
        else:
            pc, pi = _sample_without_replacement(rng, n_ctx, group_start, group_len,
                                                 items, z, cnt)
        new = np.concatenate([ctx[pc], pi[:, None].astype(np.int32)], axis=1).astype(np.int32)
        srt = np.lexsort(new.T[::-1])
        new = new[srt]
        pc = pc[srt]
        mh = rng.uniform(0.5, 0.95, size=n_ctx)
        zw = z[new[:, -1]]
        zsum = np.bincount(pc, weights=zw, minlength=n_ctx)
        probs.append(np.log10(mh[pc] * zw / zsum[pc]))
        ids.append(new)
    for m in range(1, order):
        e = ids[m - 1]
        bo = rng.uniform(-1.0, 0.0, size=e.shape[0])
        bo[e[:, -1] == EOS] = 0.0
        bows.append(bo.astype(np.float32))
    return dict(order=order, V=V, ids=ids,
                log10_prob=[p.astype(np.float32) for p in probs],
                log10_bow=bows + [None])


@lru_cache(maxsize=4)
def lm_for(spec: LMSpec, V: int) -> dict:
    return make_lm(spec.order, V, spec.counts, spec.seed)


def write_arpa(lm: dict, path: str) -> None:
    """Write the arrays as an ARPA text file (words "0".."V-1", "<s>", "</s>")."""
    V = lm["V"]

    def word(i):
        return "</s>" if i == V else ("<s>" if i == V + 1 else str(int(i)))

    with open(path, "w") as f:
        f.write("\n\\data\\\n")
        for m, e in enumerate(lm["ids"], start=1):
            f.write(f"ngram {m}={e.shape[0]}\n")
        for m, e in enumerate(lm["ids"], start=1):
            f.write(f"\n\\{m}-grams:\n")
            p = lm["log10_prob"][m - 1]
            bo = lm["log10_bow"][m - 1]
            for i in range(e.shape[0]):
                words = " ".join(word(x) for x in e[i])
                if bo is not None:
                    f.write(f"{float(p[i])!r}\t{words}\t{float(bo[i])!r}\n")
                else:
                    f.write(f"{float(p[i])!r}\t{words}\n")
        f.write("\n\\end\\\n")


# ----------------------------------------------------------------------------
# Boosting phrases
# ----------------------------------------------------------------------------
def make_phrases(V: int, spec: BoostSpec):
    """CSR phrase list: (offsets int32 [n+1], tokens int32)."""
    rng = np.random.default_rng(spec.seed)
    lens = rng.integers(spec.min_len, spec.max_len + 1, size=spec.n_phrases)
    n = int(lens.sum())
    if spec.token_dist == "uniform":
        toks = rng.integers(0, V, size=n)
    elif spec.token_dist == "zipf":
        w = _zipf_weights(V, rng)
        toks = rng.choice(V, size=n, p=w)
    else:
        raise ValueError(spec.token_dist)
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return offsets, toks.astype(np.int32)


@lru_cache(maxsize=4)
def phrases_for(spec: BoostSpec, V: int):
    return make_phrases(V, spec)


# ----------------------------------------------------------------------------
# Small random cases for fuzzing and exhaustive tests
# ----------------------------------------------------------------------------
def random_logprobs(rng: np.random.Generator, B: int, T: int, V: int, scale: float = 2.0):
    x = rng.normal(0.0, scale, size=(B, T, V + 1))
    return _log_softmax64(x).astype(np.float32)


def random_small_lm(rng: np.random.Generator, order: int, V: int, density: float = 0.5) -> dict:
    """A small prefix-closed backoff model with arbitrary log10 values, for
    exhaustive tests (every token, </s> and <s> have unigrams)."""
    EOS, BOS = V, V + 1
    ids = [np.arange(V + 2, dtype=np.int32)[:, None]]
    p = [rng.uniform(-3.0, -0.1, size=V + 2)]
    p[0][BOS] = -99.0
    for m in range(2, order + 1):
        prev = ids[-1]
        ctx = prev[prev[:, -1] != EOS]
        rows = []
        for h in ctx:
            for w in range(V + 1):
                if rng.random() < density:
                    rows.append(np.concatenate([h, [w]]))
        arr = np.asarray(rows, dtype=np.int32).reshape(-1, m)
        if arr.shape[0]:
            arr = arr[np.lexsort(arr.T[::-1])]
        ids.append(arr)
        p.append(rng.uniform(-3.0, -0.1, size=arr.shape[0]))
    bows = []
    for m in range(1, order):
        e = ids[m - 1]
        bo = rng.uniform(-1.0, 0.0, size=e.shape[0])
        bo[e[:, -1] == EOS] = 0.0
        bows.append(bo.astype(np.float32))
    return dict(order=order, V=V, ids=ids, log10_prob=[x.astype(np.float32) for x in p],
                log10_bow=bows + [None])


def read_arpa(path: str, V: int) -> dict:
    """Parse an ARPA file whose words are "0".."V-1", "<s>", "</s>" into the
    array layout of ``make_lm`` (n-grams containing other words are skipped)."""
    def wid(w):
        if w == "</s>":
            return V
        if w == "<s>":
            return V + 1
        i = int(w)
        if not 0 <= i < V:
            raise ValueError(w)
        return i

    rows = {}
    order = 0
    cur = 0
    with open(path) as f:
        for raw in f:
            line = raw.strip()
            if not line or line == "\\data\\" or line == "\\end\\":
                continue
            if line.startswith("ngram "):
                order = max(order, int(line.split()[1].split("=")[0]))
                continue
            if line.startswith("\\") and line.endswith("-grams:"):
                cur = int(line[1:].split("-")[0])
                rows.setdefault(cur, [])
                continue
            parts = line.split()
            p = float(parts[0])
            try:
                g = [wid(w) for w in parts[1:1 + cur]]
            except ValueError:
                continue
            bo = float(parts[1 + cur]) if len(parts) > 1 + cur else 0.0
            rows[cur].append((g, p, bo))
    ids, probs, bows = [], [], []
    for m in range(1, order + 1):
        r = rows.get(m, [])
        ids.append(np.asarray([g for g, _, _ in r], dtype=np.int32).reshape(-1, m))
        probs.append(np.asarray([p for _, p, _ in r], dtype=np.float32))
        bows.append(np.asarray([b for _, _, b in r], dtype=np.float32) if m < order else None)
    return dict(order=order, V=V, ids=ids, log10_prob=probs, log10_bow=bows)
