"""CPU oracle for f-gram discovery (test infrastructure only).

Only the tests and the benchmark's CPU-baseline leg use this module; the
product path never does.  It shares no code with the GPU library.

What it computes: Algorithm 3 of "Scaling Embedding Layers in Language
Models": count every n-gram, n = 2..K, over all token sequences; order all of
them by count, highest first (ties in any order); the f-gram set is the first
S.  Section 3.1 adds a minimum count (5 in the paper) from the second scan on:
n-grams with n >= 3 below it are never kept; 2-grams are all kept.  With a
minimum count of 1 this is Algorithm 3 exactly.  n-grams never cross from one
sequence into the next.
"""
from __future__ import annotations

import numpy as np


def count_ngrams(X: np.ndarray, n: int):
    """All distinct n-grams of the rows of X with their counts.

    Returns (grams [m, n] int32, counts [m] int64), grams sorted
    lexicographically (np.unique order).
    """
    X = np.asarray(X, dtype=np.int32)
    B, T = X.shape
    if T < n or B == 0:
        return np.zeros((0, n), dtype=np.int32), np.zeros(0, dtype=np.int64)
    windows = np.stack([X[:, j:T - n + 1 + j] for j in range(n)], axis=-1).reshape(-1, n)
    grams, counts = np.unique(windows, axis=0, return_counts=True)
    return grams.astype(np.int32), counts.astype(np.int64)


def candidates(X: np.ndarray, K: int, min_count: int = 1):
    """Every n-gram that may enter the f-gram set, with its count, ordered by
    count (highest first; equal counts in an unspecified order).

    Returns a list of (tuple_of_tokens, count).
    """
    out = []
    for n in range(2, K + 1):
        grams, counts = count_ngrams(X, n)
        keep = counts >= (min_count if n >= 3 else 1)
        out.extend((tuple(int(v) for v in g), int(c)) for g, c in zip(grams[keep], counts[keep]))
    out.sort(key=lambda gc: -gc[1])
    return out


def discover(X: np.ndarray, K: int, S: int, min_count: int = 1):
    """One valid top-S f-gram set: list of (tokens, count)."""
    return candidates(X, K, min_count)[:S]
