"""Pins for the CPU oracle: each test checks it against something other than itself.

* a hand-worked example of Algorithm 1 (tests/golden/alg1_worked_example.json);
* a brute-force linear scan over the f-gram list on random tiny inputs;
* the invariants that characterise the longest-suffix result (Algorithm 1);
* closed forms: identity when the window is 1 or the set is empty, and
  all-bigram / all-trigram sets whose ids are an explicit function of the
  tokens;
* the gather against numpy fancy indexing, byte for byte.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, HealthCheck, strategies as st

import oracle
from checks import brute_force, check_invariants, fgram_dict
from workloads import CONFIGS, make_workload, scaled, table_rows

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "alg1_worked_example.json")


def pad(rows, width):
    out = np.full((len(rows), width), -1, dtype=np.int32)
    for k, r in enumerate(rows):
        out[k, :len(r)] = r
    return out


def test_worked_example_alg1():
    g = json.load(open(GOLDEN))
    rows = g["fgrams"]
    o = oracle.OracleTable(pad(rows, 4), [len(r) for r in rows], g["ids"])
    X = np.array(g["tokens"], dtype=np.int32)
    for max_n, exp in g["expected"].items():
        ids, ml = o.lookup(X, int(max_n))
        assert ids.tolist() == exp["ids"], max_n
        assert ml.tolist() == exp["len"], max_n


@st.composite
def tiny_instance(draw):
    vocab = draw(st.integers(2, 8))
    kmax = draw(st.integers(2, 5))
    pool = draw(st.lists(
        st.lists(st.integers(0, vocab - 1), min_size=2, max_size=kmax),
        max_size=60, unique_by=tuple))
    B = draw(st.integers(1, 3))
    T = draw(st.integers(0, 40))
    X = draw(st.lists(st.lists(st.integers(0, vocab - 1), min_size=T, max_size=T),
                      min_size=B, max_size=B))
    max_n = draw(st.integers(1, 6))
    ids = draw(st.permutations(list(range(100, 100 + len(pool)))))
    return pool, list(ids), np.array(X, dtype=np.int32).reshape(B, T), max_n, kmax


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(tiny_instance())
def test_oracle_matches_brute_force(inst):
    pool, ids, X, max_n, kmax = inst
    fg = pad(pool, kmax)
    ln = np.array([len(r) for r in pool], dtype=np.int32)
    o = oracle.OracleTable(fg, ln, ids)
    got_ids, got_len = o.lookup(X, max_n)
    exp_ids, exp_len = brute_force(fg, ln, ids, X, max_n)
    assert np.array_equal(got_ids, exp_ids)
    assert np.array_equal(got_len, exp_len)


@pytest.mark.parametrize("name,kw", [
    ("tiny", {}),
    ("c2_1m", dict(n_fgrams=20_000, B=4, T=1024)),
    ("c3_10m_k5", dict(n_fgrams=30_000, B=2, T=2048)),
    ("c5_decode", dict(n_fgrams=20_000, B=16, T=128)),
])
def test_invariants_on_configs(name, kw):
    cfg = scaled(CONFIGS[name], **kw)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    ids, ml = o.lookup(w.tokens, cfg.max_n)
    check_invariants(w.tokens, ids, ml, cfg.max_n, fgram_dict(w.fgrams, w.lengths, w.ids),
                     planted_end=w.planted_end)
    # the workload really exercises matches of every admissible length
    assert set(np.unique(ml)) >= set(range(1, cfg.max_n + 1))


def test_window_one_and_empty_set_are_identity():
    w = make_workload(scaled(CONFIGS["tiny"], B=4, T=300))
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    ids, ml = o.lookup(w.tokens, 1)
    assert np.array_equal(ids, w.tokens) and (ml == 1).all()
    empty = oracle.OracleTable(np.zeros((0, 3), np.int32), [], [])
    ids, ml = empty.lookup(w.tokens, 3)
    assert np.array_equal(ids, w.tokens) and (ml == 1).all()


def test_all_bigrams_and_trigrams_closed_form():
    V = 6
    a, b, c = np.meshgrid(np.arange(V), np.arange(V), np.arange(V), indexing="ij")
    bi = np.stack([a[:, :, 0].ravel(), b[:, :, 0].ravel()], 1)
    tri = np.stack([a.ravel(), b.ravel(), c.ravel()], 1)
    fg = pad(list(bi) + list(tri), 3)
    ln = np.array([2] * len(bi) + [3] * len(tri), dtype=np.int32)
    # id of bigram (x, y) = V + x*V + y ; trigram (x, y, z) = V + V^2 + (x*V + y)*V + z
    ids = np.concatenate([V + bi[:, 0] * V + bi[:, 1],
                          V + V * V + (tri[:, 0] * V + tri[:, 1]) * V + tri[:, 2]]).astype(np.int32)
    rng = np.random.default_rng(5)
    X = rng.integers(0, V, size=(3, 50)).astype(np.int32)
    o = oracle.OracleTable(fg, ln, ids)
    got2, l2 = o.lookup(X, 2)
    assert (l2[:, 0] == 1).all() and (l2[:, 1:] == 2).all()
    assert np.array_equal(got2[:, 0], X[:, 0])
    assert np.array_equal(got2[:, 1:], V + X[:, :-1] * V + X[:, 1:])
    got3, l3 = o.lookup(X, 3)
    assert (l3[:, 1] == 2).all() and (l3[:, 2:] == 3).all()
    assert np.array_equal(got3[:, 2:], V + V * V + (X[:, :-2] * V + X[:, 1:-1]) * V + X[:, 2:])
    # a wider window than the longest f-gram changes nothing
    got9, l9 = o.lookup(X, 9)
    assert np.array_equal(got9, got3) and np.array_equal(l9, l3)


def test_build_order_does_not_matter():
    w = make_workload(scaled(CONFIGS["tiny"], B=4, T=256))
    perm = np.random.default_rng(1).permutation(len(w.lengths))
    a = oracle.OracleTable(w.fgrams, w.lengths, w.ids).lookup(w.tokens, 3)
    b = oracle.OracleTable(w.fgrams[perm], w.lengths[perm], w.ids[perm]).lookup(w.tokens, 3)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_build_rejects_invalid_sets():
    fg = pad([[1, 2], [2, 3]], 3)
    with pytest.raises(oracle.OracleError) as e:
        oracle.OracleTable(pad([[1, 2], [1, 2]], 3), [2, 2], [10, 11])
    assert e.value.code == oracle.OR_DUPLICATE
    with pytest.raises(oracle.OracleError) as e:
        oracle.OracleTable(fg, [2, 1], [10, 11])
    assert e.value.code == oracle.OR_BAD_LENGTH
    with pytest.raises(oracle.OracleError) as e:
        oracle.OracleTable(fg, [2, 4], [10, 11])
    assert e.value.code == oracle.OR_BAD_LENGTH
    with pytest.raises(oracle.OracleError) as e:
        oracle.OracleTable(fg, [2, 2], [10, -1])
    assert e.value.code == oracle.OR_BAD_ID
    # same tokens, different lengths are different f-grams
    o = oracle.OracleTable(pad([[1, 2, 3], [1, 2, 3]], 3), [2, 3], [10, 11])
    assert len(o) == 2


def test_gather_equals_fancy_indexing_bytes():
    cfg = CONFIGS["tiny"]
    E = table_rows(cfg, range(cfg.n_rows)).numpy()
    # plant special bit patterns: -0.0, +inf, a NaN with payload, a denormal
    E.view(np.uint32)[3, :4] = [0x80000000, 0x7F800000, 0x7FC01234, 0x00000001]
    rng = np.random.default_rng(0)
    ids = rng.integers(0, cfg.n_rows, size=(5, 77)).astype(np.int32)
    ids[0, :4] = 3
    out = oracle.gather(ids, E)
    assert out.tobytes() == E[ids].tobytes()
    # bf16 rows (stored as uint16) and an odd row width
    Eh = rng.integers(0, 1 << 16, size=(50, 7), dtype=np.uint16)
    ih = rng.integers(0, 50, size=300).astype(np.int32)
    assert oracle.gather(ih, Eh).tobytes() == Eh[ih].tobytes()


def test_gather_rejects_bad_rows():
    E = np.zeros((10, 4), np.float32)
    for bad in (-1, 10):
        with pytest.raises(oracle.OracleError) as e:
            oracle.gather(np.array([0, bad], np.int32), E)
        assert e.value.code == oracle.OR_BAD_ROW


def test_query_count_bound():
    # at most max_n - 1 dictionary queries per token (Section 4.3: up to four for K = 5)
    cfg = scaled(CONFIGS["c3_10m_k5"], n_fgrams=5000, B=2, T=512)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    o.lookup(w.tokens, 5)
    assert o.queries <= cfg.n_tok * 4
    T = cfg.T
    exact_max = cfg.B * sum(max(0, min(5, t + 1) - 1) for t in range(T))
    assert o.queries <= exact_max
