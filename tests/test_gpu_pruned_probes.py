"""Suffix entries and pruned probing against the oracle.

Tables with f-grams of length 4 or more hold an entry, flagged as extending,
for the last three tokens of each such f-gram (a marker when those three
tokens are not an f-gram themselves), and for the last five tokens of each
f-gram of length 6 or more; lookups probe lengths 4-5 (6-7) only where that
entry exists.  The oracle probes every length, so equal results show that no
pruned probe could have hit.  Cases: a marker-only suffix, an f-gram that is
also a flagged suffix (its id must come back without the flag), a length-5
marker gating lengths 6-7, windows shorter than the table's K, ids next to the
reserved value, dense small-vocabulary tables in which most suffixes collide,
and every path that probes (lookup, tagging, fused embed, pipelined step,
decode).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S
from gpu_util import as_bytes, build_gpu, dev
from workloads import CONFIGS, make_workload, scaled

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _clean_error_word():
    S.check()
    yield
    assert S.check() == S.scone.OK, "a test left a device error behind"


def pad(rows, width):
    out = np.full((len(rows), width), -1, dtype=np.int32)
    for k, r in enumerate(rows):
        out[k, :len(r)] = r
    return out


def check_lookup(fgrams, ids, X, max_len, max_ns):
    fg = pad(fgrams, max_len)
    ln = [len(r) for r in fgrams]
    o = oracle.OracleTable(fg, ln, ids)
    tb = build_gpu(fg, ln, ids)
    Xn = np.asarray(X, dtype=np.int32)
    for max_n in max_ns:
        exp_ids, exp_len = o.lookup(Xn, max_n)
        got_ids, got_len = S.lookup(tb, dev(Xn), max_n, want_len=True)
        S.check_ok()
        np.testing.assert_array_equal(got_ids.cpu().numpy(), exp_ids, err_msg=f"max_n {max_n}")
        np.testing.assert_array_equal(got_len.cpu().numpy(), exp_len, err_msg=f"max_n {max_n}")
    return tb, o


def test_marker_only_suffix():
    # [2, 3, 4] is not an f-gram, but the 4-gram ending with it must be found
    check_lookup([[1, 2, 3, 4]], [100], [[9, 1, 2, 3, 4, 2, 3, 4]], 4, [2, 3, 4, 5])


def test_fgram_that_is_also_a_flagged_suffix():
    fgrams = [[2, 3, 4], [1, 2, 3, 4], [3, 4]]
    ids = [50, 100, 60]
    X = [[1, 2, 3, 4, 7, 2, 3, 4, 0, 3, 4]]
    tb, o = check_lookup(fgrams, ids, X, 5, [2, 3, 4, 5])
    got = S.lookup(tb, dev(np.asarray(X, dtype=np.int32)), 5)[0].cpu().numpy().ravel()
    assert got[3] == 100 and got[7] == 50 and got[10] == 60


def test_length_five_marker_gates_six_and_seven():
    fgrams = [[1, 2, 3, 4, 5, 6, 7], [9, 4, 5, 6, 7, 8], [5, 6, 7], [4, 5, 6, 7]]
    ids = [200, 210, 70, 80]
    X = [[1, 2, 3, 4, 5, 6, 7, 0, 9, 4, 5, 6, 7, 8, 3, 4, 5, 6, 7, 2, 3, 4, 5, 6, 7]]
    check_lookup(fgrams, ids, X, 7, [2, 3, 4, 5, 6, 7])


def test_ids_next_to_the_reserved_value():
    top = 2**31 - 2
    fgrams = [[2, 3, 4], [1, 2, 3, 4], [5, 6]]
    ids = [top, top - 1, top - 2]
    tb, _ = check_lookup(fgrams, ids, [[1, 2, 3, 4, 8, 2, 3, 4, 5, 6]], 4, [3, 4])
    got = S.lookup(tb, dev(np.array([[1, 2, 3, 4, 8, 2, 3, 4]], dtype=np.int32)), 4)[0]
    assert got.cpu().numpy().ravel()[[3, 7]].tolist() == [top - 1, top]
    with pytest.raises(S.SconeError) as e:
        build_gpu(pad([[1, 2, 3, 4]], 4), [4], [2**31 - 1])
    assert e.value.code == S.scone.EID


@pytest.mark.parametrize("max_len,V,n", [(4, 6, 600), (5, 8, 3000), (6, 5, 2500), (7, 6, 6000)])
def test_dense_tables_all_paths(max_len, V, n):
    """A small vocabulary makes most suffixes shared: many f-grams end in the
    same three (five) tokens, and many of those suffixes are f-grams too."""
    cfg = scaled(CONFIGS["tiny"], V=V, n_fgrams=n, max_len=max_len, max_n=max_len, B=3, T=700,
                 d=256)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    tb = build_gpu(w.fgrams, w.lengths, w.ids, max_load=0.9)   # the sizing must leave room
    X = dev(w.tokens)
    E = torch.arange(cfg.n_rows * 64, dtype=torch.int32, device="cuda").view(cfg.n_rows, 64)
    table = E.cpu().view(torch.uint8).numpy()
    for max_n in range(1, max_len + 1):
        exp_ids, exp_len = o.lookup(w.tokens, max_n)
        ids, lens = S.lookup(tb, X, max_n, want_len=True)
        hist = torch.zeros(S.scone.MAX_FGRAM_LEN + 1, dtype=torch.int64, device="cuda")
        tag_len, _ = S.tag(tb, X, max_n, hist=hist)
        fid = torch.empty_like(X)
        out = S.embed(tb, X, max_n, E, fgram_ids=fid)
        nxt = torch.empty_like(X)
        S.embed_pipelined(tb, X, max_n, nxt, None, E)
        S.check_ok()
        msg = f"K {max_len} max_n {max_n}"
        np.testing.assert_array_equal(ids.cpu().numpy(), exp_ids, err_msg=msg)
        np.testing.assert_array_equal(lens.cpu().numpy(), exp_len, err_msg=msg)
        np.testing.assert_array_equal(tag_len.cpu().numpy(), exp_len, err_msg=msg)
        np.testing.assert_array_equal(fid.cpu().numpy(), exp_ids, err_msg=msg)
        np.testing.assert_array_equal(nxt.cpu().numpy(), exp_ids, err_msg=msg)
        assert as_bytes(out).tobytes() == oracle.gather(exp_ids, table).tobytes(), msg
        counts = np.bincount(exp_len.ravel(), minlength=S.scone.MAX_FGRAM_LEN + 1)
        assert hist.cpu().numpy().tolist() == counts.tolist(), msg
        if max_n == max_len:
            assert (exp_len >= 4).mean() > 0.2, "the case must exercise the pruned rounds"

    # decode: one position per step, every length probed in one round
    Sq, T = w.tokens.shape
    cap = max_len - 1
    ctx = torch.zeros((Sq, cap), dtype=torch.int32, device="cuda")
    ctx_len = torch.zeros(Sq, dtype=torch.int32, device="cuda")
    out = torch.empty((Sq, 64), dtype=torch.int32, device="cuda")
    fid = torch.empty(Sq, dtype=torch.int32, device="cuda")
    exp_ids, _ = o.lookup(w.tokens, max_len)
    got = np.empty_like(exp_ids)
    for t in range(T):
        S.decode_step(tb, ctx, ctx_len, X[:, t].contiguous(), max_len, E, out, fgram_ids=fid)
        got[:, t] = fid.cpu().numpy()
    S.check_ok()
    np.testing.assert_array_equal(got, exp_ids)


def literal_probe_count(fgrams, X, max_n, max_len):
    """Keys the tile lookup probes, walked position by position from its rule:
    with a window of w = min(max_n, K, t + 1) tokens, lengths 2 and 3 where
    they fit (only 2 when the window is capped at 2); 4 and 5 where they fit
    and the length-3 suffix ends some f-gram of length 4 or more; 6 and 7
    where, in addition, the length-5 suffix (which must fit) ends one of
    length 6 or more."""
    ends = {3: set(), 5: set()}
    for g in fgrams:
        for n in (3, 5):
            if len(g) >= n + 1:
                ends[n].add(tuple(g[-n:]))
    cap = min(max_n, max_len)
    total = 0
    for row in np.asarray(X):
        for t in range(len(row)):
            w = min(cap, t + 1)
            if cap <= 2:
                total += int(w >= 2)
                continue
            total += int(w >= 2) + int(w >= 3)
            go4 = w >= 3 and tuple(row[t - 2:t + 1]) in ends[3]
            if go4:
                total += int(w >= 4) + int(w >= 5)
                if cap >= 6 and w >= 5 and tuple(row[t - 4:t + 1]) in ends[5]:
                    total += int(w >= 6) + int(w >= 7)
    return total


@pytest.mark.parametrize("max_len,V,n", [(5, 6, 300), (7, 4, 400), (3, 5, 100), (5, 40, 2000)])
def test_device_probe_count_matches_the_schedule(max_len, V, n):
    """scone_lookup_counted's device count equals the literal walk of the
    pruned schedule, and its ids and lengths equal scone_lookup's."""
    rng = np.random.default_rng(max_len * 100 + V)
    X = rng.integers(0, V, size=(3, 257)).astype(np.int32)
    fgrams, seen = [], set()
    while len(fgrams) < n:
        L = int(rng.integers(2, max_len + 1))
        if rng.random() < 0.5:                      # windows of X, so every length hits
            b, t = int(rng.integers(3)), int(rng.integers(L - 1, X.shape[1]))
            g = tuple(int(v) for v in X[b, t - L + 1:t + 1])
        else:
            g = tuple(int(v) for v in rng.integers(0, V, size=L))
        if g not in seen:
            seen.add(g)
            fgrams.append(list(g))
    ids = list(range(1000, 1000 + len(fgrams)))
    fg = pad(fgrams, max_len)
    tb = build_gpu(fg, [len(g) for g in fgrams], ids)
    Xd = dev(X)
    for max_n in sorted({2, 3, max_len, max_len + 2}):
        want_ids, want_len = S.lookup(tb, Xd, max_n, want_len=True)
        got_ids, got_len, probes = S.lookup_counted(tb, Xd, max_n)
        S.check_ok()
        assert torch.equal(got_ids, want_ids) and torch.equal(got_len, want_len), max_n
        assert probes == literal_probe_count(fgrams, X, max_n, max_len), max_n
