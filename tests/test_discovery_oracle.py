"""Pins for the f-gram discovery oracle (Algorithm 3 and the minimum count of
Section 3.1): a dictionary count over tuples, hand-counted corpora, and the
window-count identity."""
from collections import Counter

import numpy as np
from hypothesis import given, settings, HealthCheck, strategies as st

from oracle import discovery


def counter_candidates(X, K, min_count):
    c = Counter()
    for row in np.asarray(X).tolist():
        for n in range(2, K + 1):
            for t in range(n - 1, len(row)):
                c[tuple(row[t - n + 1:t + 1])] += 1
    return {g: k for g, k in c.items() if len(g) == 2 or k >= min_count}


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(st.integers(1, 4), st.integers(0, 30), st.integers(2, 6), st.integers(2, 5),
       st.integers(1, 4), st.integers(0, 10 ** 6))
def test_candidates_match_dictionary_count(B, T, V, K, min_count, seed):
    X = np.random.default_rng(seed).integers(0, V, size=(B, T)).astype(np.int32)
    got = discovery.candidates(X, K, min_count)
    assert dict(got) == counter_candidates(X, K, min_count)
    counts = [c for _, c in got]
    assert counts == sorted(counts, reverse=True)


def test_hand_counted_corpus():
    # row 0: a b c a b c a ; row 1: b c a  (a=1, b=2, c=3)
    X = [[1, 2, 3, 1, 2, 3, 1], [2, 3, 1, 0, 0, 0, 0]]
    X = np.array(X, dtype=np.int32)
    cands = dict(discovery.candidates(X[:, :], 3, 1))
    # bigrams in row 0: ab bc ca ab bc ca ; row 1: bc ca a0 00 00 00
    assert cands[(1, 2)] == 2 and cands[(2, 3)] == 3 and cands[(3, 1)] == 3
    assert cands[(1, 0)] == 1 and cands[(0, 0)] == 3
    # trigrams: abc bca cab abc bca (row 0); bca ca0 a00 000 000 (row 1)
    assert cands[(1, 2, 3)] == 2 and cands[(2, 3, 1)] == 3 and cands[(3, 1, 2)] == 1
    assert cands[(0, 0, 0)] == 2
    # no n-gram crosses rows: (1, 2, 3) would gain one from "... 1 | 2 3 ..."
    top = discovery.discover(X, 3, 3, 1)
    assert sorted(c for _, c in top) == [3, 3, 3]
    # the minimum count drops rare trigrams, never bigrams
    c2 = dict(discovery.candidates(X, 3, 2))
    assert (3, 1, 2) not in c2 and (1, 0) in c2 and (2, 3, 1) in c2


def test_window_count_identity():
    X = np.random.default_rng(1).integers(0, 50, size=(5, 40)).astype(np.int32)
    for n in range(2, 6):
        _, counts = discovery.count_ngrams(X, n)
        assert counts.sum() == 5 * (40 - n + 1)
