"""Independent checks used to pin the oracle (pure Python / numpy).

* ``brute_force`` scans the whole f-gram list for every (b, t, n): no hashing,
  no early exit, tiny inputs only.
* ``check_invariants`` verifies properties that characterise the longest-suffix
  result uniquely (Algorithm 1's choice of j): the matched length range, that
  the matched suffix is an f-gram with that id, that no longer suffix within
  the window is an f-gram, and the identity fallback.
"""
import numpy as np


def brute_force(fgrams, lengths, ids, X, max_n):
    X = np.asarray(X)
    B, T = X.shape
    out = np.empty((B, T), dtype=np.int64)
    lens = np.empty((B, T), dtype=np.int64)
    entries = [(tuple(int(v) for v in fgrams[k][:lengths[k]]), int(ids[k]))
               for k in range(len(lengths))]
    for b in range(B):
        for t in range(T):
            best_n, best_id = 1, int(X[b, t])
            # every admissible length, every f-gram; keep the longest hit
            for n in range(2, max_n + 1):
                if n > t + 1:
                    break
                window = tuple(int(v) for v in X[b, t - n + 1:t + 1])
                for g, i in entries:
                    if g == window and n > best_n:
                        best_n, best_id = n, i
            out[b, t], lens[b, t] = best_id, best_n
    return out, lens


def fgram_dict(fgrams, lengths, ids):
    d = {}
    for k in range(len(lengths)):
        d[np.asarray(fgrams[k][:lengths[k]], dtype=np.int32).tobytes()] = int(ids[k])
    return d


def check_invariants(X, ids, lens, max_n, fdict, planted_end=None):
    """Raise AssertionError on the first violated invariant."""
    X = np.asarray(X, dtype=np.int32)
    B, T = X.shape
    for b in range(B):
        row = X[b]
        for t in range(T):
            L = int(lens[b, t])
            top = min(max_n, t + 1)
            # I1: length range
            assert L == 1 or 2 <= L <= top, (b, t, L)
            if L >= 2:
                # I2: the matched suffix is an f-gram carrying that id
                key = row[t - L + 1:t + 1].tobytes()
                assert fdict.get(key) == int(ids[b, t]), (b, t, L)
            else:
                # I4: fallback to the token's own row
                assert int(ids[b, t]) == int(row[t]), (b, t)
            # I3: no longer suffix inside the window is an f-gram
            for n in range(max(L + 1, 2), top + 1):
                assert row[t - n + 1:t + 1].tobytes() not in fdict, (b, t, n)
            # I5: a whole planted f-gram ending here bounds L from below
            if planted_end is not None:
                g = int(planted_end[b, t])
                if 2 <= g <= max_n:
                    assert L >= g, (b, t, g, L)
