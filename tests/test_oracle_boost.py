"""Pins of the oracle's phrase-boosting tree (Sec. III-B: Aho-Corasick prefix
tree, boosting spread over the nodes by depth; Alg. 1 BT(<0>) start state and
PB state update).  Closed forms of the tree's rules:

* a phrase read exactly earns |p|;
* a proper prefix of length m followed by a token that continues nothing
  earns 0 in total (+m, then -m);
* phrases separated by tokens that start nothing earn sum |p_i|;
* an empty phrase list, or tokens that start no phrase, earn 0;
* nested "ab" inside "abcd", read as "a b c x", earns 2 (the completed "ab"
  stays banked, the pending "c" is rolled back);
* a token is never counted twice: the total never exceeds the number of
  tokens read and never drops below 0.
"""
import numpy as np

import oracle


def _bt(V, phrases):
    lens = [len(p) for p in phrases]
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    toks = np.asarray([t for p in phrases for t in p], dtype=np.int32)
    return oracle.BT(V, off, toks)


def test_exact_phrase():
    bt = _bt(10, [[1, 2, 3], [4, 5]])
    assert bt.run([1, 2, 3])[0] == 3
    assert bt.run([4, 5])[0] == 2


def test_prefix_then_break_rolls_back():
    bt = _bt(10, [[1, 2, 3, 4]])
    for m in (1, 2, 3):
        s, q = bt.run([1, 2, 3, 4][:m] + [9])
        assert s == 0 and q == []
    # step-by-step: +1 per matched token, then -m
    assert [bt.step([1, 2][:i], c)[0] for i, c in enumerate([1, 2])] == [1, 1]
    assert bt.step([1, 2], 9)[0] == -2


def test_separated_phrases_add_up():
    bt = _bt(10, [[1, 2], [3, 4, 5], [6]])
    assert bt.run([1, 2, 9, 3, 4, 5, 8, 6, 7])[0] == 2 + 3 + 1
    assert bt.run([1, 2, 3, 4, 5, 6])[0] == 2 + 3 + 1


def test_empty_list_and_unrelated_tokens():
    bt = _bt(10, [])
    assert bt.run([1, 2, 3, 4])[0] == 0
    bt = _bt(10, [[1, 2]])
    assert bt.run([7, 8, 9, 0])[0] == 0


def test_nested_phrase_break():
    bt = _bt(10, [[1, 2], [1, 2, 3, 4]])
    assert bt.run([1, 2, 3, 9])[0] == 2
    assert bt.run([1, 2, 3, 4])[0] == 4
    assert bt.pot([1, 2]) == 0 and bt.pot([1, 2, 3]) == 1


def test_overlap_continues_from_a_suffix():
    # "1 2 3" fails at 9 after "1 2"; the suffix "2" is itself a prefix of "2 9"
    bt = _bt(10, [[1, 2, 3], [2, 9]])
    s, q = bt.run([1, 2, 9])
    # +1 +1 for "1 2"; on 9: back off to "2" (pot 1 - pot 2 = -1), then +1 for "2 9"
    assert s == 2 and q == [2, 9]


def test_no_double_counting_bounds():
    rng = np.random.default_rng(0)
    V = 4
    for _ in range(50):
        n = int(rng.integers(1, 6))
        phrases = [rng.integers(0, V, size=int(rng.integers(1, 4))).tolist() for _ in range(n)]
        bt = _bt(V, phrases)
        seq = rng.integers(0, V, size=int(rng.integers(1, 12))).tolist()
        total = 0
        q = []
        for i, c in enumerate(seq):
            s, q = bt.step(q, c)
            total += s
            assert 0 <= total <= i + 1
            assert bt.pot(q) <= total


def test_completed_phrase_restarts_at_root():
    """Tokens of a banked phrase never start another phrase: with "1 2" and
    "2 3", reading "1 2 3" earns 2 ("1 2" banked; "3" starts nothing)."""
    bt = _bt(10, [[1, 2], [2, 3]])
    assert bt.run([1, 2, 3])[0] == 2
    # the pending tail of a longer match can start one: "1 2 3 x" with
    # "1 2", "1 2 3 4" and "3 9": "3" is pending when 9 arrives, and "3 9"
    # completes, so all four tokens end up banked
    bt = _bt(10, [[1, 2], [1, 2, 3, 4], [3, 9]])
    assert bt.run([1, 2, 3, 9])[0] == 4
