"""GPU f-gram discovery against the discovery oracle.

Equal counts at the cut may be broken either way (Algorithm 3 breaks ties
arbitrarily), so a result is checked for what is unique: its size, that every
f-gram is a real candidate with the oracle's count, and that no candidate
counting more than the smallest kept count was left out.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import discovery
import paper_2502_01637_amd as S
from gpu_util import build_gpu, dev
from workloads import CONFIGS, make_workload, scaled, query_batches, zipf_cdf, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _clean_error_word():
    S.check()
    yield
    assert S.check() == S.scone.OK


def check_top_s(fg, ln, ct, cands, Sn):
    fg, ln, ct = fg.cpu().numpy(), ln.cpu().numpy(), ct.cpu().numpy()
    want = min(Sn, len(cands))
    assert len(ln) == want
    got = {}
    for row, L, c in zip(fg, ln, ct):
        assert 2 <= L <= fg.shape[1] and (row[L:] == -1).all()
        got[tuple(int(v) for v in row[:L])] = int(c)
    assert len(got) == want, "duplicate f-grams in the output"
    oc = dict(cands)
    for g, c in got.items():
        assert oc.get(g) == c, (g, c, oc.get(g))
    if want and want < len(cands):
        cmin = min(got.values())
        for g, c in cands:
            if c > cmin:
                assert g in got, (g, c, cmin)
            else:
                break
    return got


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("K,min_count", [(2, 1), (3, 1), (5, 2), (7, 1), (4, 3)])
def test_discovery_small_random(seed, K, min_count):
    rng = np.random.default_rng(seed * 31 + K)
    V = int(rng.integers(2, 7))
    B, T = int(rng.integers(1, 5)), int(rng.integers(1, 80))
    X = rng.integers(0, V, size=(B, T)).astype(np.int32)
    cands = discovery.candidates(X, K, min_count)
    for Sn in (1, 7, 50, 10 ** 6):
        fg, ln, ct = S.discover_fgrams(dev(X), K, Sn, min_count)
        check_top_s(fg, ln, ct, cands, Sn)


def test_discovery_zipf_corpus_and_round_trip():
    cfg = scaled(CONFIGS["c3_10m_k5"], n_fgrams=20_000, B=16, T=2048)
    w = make_workload(cfg)
    X = np.concatenate(query_batches(w, 2))
    cands = discovery.candidates(X, 5, 5)
    fg, ln, ct = S.discover_fgrams(dev(X), 5, 5000, 5)
    got = check_top_s(fg, ln, ct, cands, 5000)
    assert set(len(g) for g in got) >= {2, 3}
    # the discovered set is a valid f-gram set: it builds and serves lookups
    ids = np.arange(cfg.V, cfg.V + len(ln), dtype=np.int32)
    fg_np, ln_np = fg.cpu().numpy(), ln.cpu().numpy()
    tb = build_gpu(fg_np, ln_np, ids)
    o = oracle.OracleTable(fg_np, ln_np, ids)
    exp_ids, exp_len = o.lookup(w.tokens, 5)
    got_ids, got_len = S.lookup(tb, dev(w.tokens), 5, want_len=True)
    S.check_ok()
    np.testing.assert_array_equal(got_ids.cpu().numpy(), exp_ids)
    np.testing.assert_array_equal(got_len.cpu().numpy(), exp_len)


def test_discovery_threshold_above_the_histogram():
    """A small S over a corpus whose top n-grams count in the tens of
    thousands: the count threshold lies above the exact range of the device
    histogram, so the search over the pooled counts decides it."""
    rng = np.random.default_rng(31)
    X = zipf_tokens(rng, zipf_cdf(40), (16, 125_000)).astype(np.int32)
    for K, Sn, mc in [(3, 3, 5), (2, 10, 1), (3, 40, 5)]:
        cands = discovery.candidates(X, K, mc)
        assert cands[Sn - 1][1] >= 4096
        fg, ln, ct = S.discover_fgrams(dev(X), K, Sn, mc)
        check_top_s(fg, ln, ct, cands, Sn)


def test_discovery_edges_and_errors():
    X = np.array([[65535, 65535, 65535, 0, 65535, 65535]], dtype=np.int32)
    cands = discovery.candidates(X, 4, 1)
    fg, ln, ct = S.discover_fgrams(dev(X), 4, 100, 1)
    check_top_s(fg, ln, ct, cands, 100)
    # sequences shorter than every n-gram: nothing to find
    fg, ln, ct = S.discover_fgrams(dev(np.zeros((3, 1), np.int32)), 3, 10, 1)
    assert len(ln) == 0
    with pytest.raises(S.SconeError) as e:
        S.discover_fgrams(dev(np.array([[1, 70000, 2]], np.int32)), 3, 10, 1)
    assert e.value.code == S.scone.ETOKEN
    with pytest.raises(S.SconeError) as e:
        S.discover_fgrams(dev(np.array([[1, 2, 2]], np.int32)), 3, 10, 0)
    assert e.value.code == S.scone.EINVAL


def test_workspace_paths_agree():
    """The call with no workspace (it allocates its own), with a caller's
    workspace reused across calls, and through the binding all give the same
    top-S set; a short or misaligned workspace is an argument error."""
    import ctypes
    rng = np.random.default_rng(21)
    cdf = zipf_cdf(500)
    X = zipf_tokens(rng, cdf, (8, 700)).astype(np.int32)
    K, Sn, mc = 4, 300, 2
    cands = discovery.candidates(X, K, mc)
    Xd = dev(X)
    B, T = X.shape
    L = S.scone.lib()
    need = S.discover_workspace_bytes(B, T, K)
    assert need > 0
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")

    def call(workspace, nbytes):
        fg = torch.empty((Sn, K), dtype=torch.int32, device="cuda")
        ln = torch.empty(Sn, dtype=torch.int32, device="cuda")
        ct = torch.empty(Sn, dtype=torch.int32, device="cuda")
        n = ctypes.c_int64()
        rc = L.scone_discover_fgrams(Xd.data_ptr(), B, T, K, mc, Sn, fg.data_ptr(), ln.data_ptr(),
                                     ct.data_ptr(), ctypes.byref(n), workspace, nbytes, None)
        return rc, fg[:n.value], ln[:n.value], ct[:n.value]

    results = [call(None, 0), call(ws.data_ptr(), need), call(ws.data_ptr(), need),
               (S.scone.OK,) + tuple(S.discover_fgrams(Xd, K, Sn, mc))]
    for rc, fg, ln, ct in results:
        assert rc == S.scone.OK
        check_top_s(fg, ln, ct, cands, Sn)
    assert call(ws.data_ptr(), need - 1)[0] == S.scone.EINVAL
    assert call(ws.data_ptr() + 16, need)[0] == S.scone.EINVAL


# Random corpora (seeds 70000 + case): vocabularies of 2 to 30,000, K 2-7,
# minimum counts 1-5, three values of S each.  SCONE_DISCOVERY_SWEEP sets the
# number of cases (1,000 take under a minute).
DISC_CASES = int(os.environ.get("SCONE_DISCOVERY_SWEEP", "20"))


@pytest.mark.parametrize("case", range(DISC_CASES))
def test_random_corpora(case):
    rng = np.random.default_rng(70000 + case)
    V = int(rng.choice([2, 3, 7, 50, 1000, 30000]))
    K = int(rng.integers(2, 8))
    mc = int(rng.integers(1, 6))
    B, T = int(rng.integers(1, 9)), int(rng.integers(1, 2500))
    X = rng.integers(0, V, size=(B, T)).astype(np.int32)
    cands = discovery.candidates(X, K, mc)
    for Sn in (1, int(rng.integers(2, 300)), 10 ** 6):
        fg, ln, ct = S.discover_fgrams(dev(X), K, Sn, mc)
        check_top_s(fg, ln, ct, cands, Sn)
