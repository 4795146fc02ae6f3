"""GPU path (through the C ABI) against the CPU oracle, bit for bit.

Ids and match lengths are compared element by element with the oracle on the
same seeded inputs; gathered rows are compared as raw bytes with the
oracle's memcpy gather.  Sizes span several workgroup tiles with ragged
tails; the edge cases cover empty inputs, window 1, windows wider than the
table's K, 7-token f-grams (32-byte slots), extreme token values, unaligned
row widths and every error the library reports.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S
from gpu_util import as_bytes, build_gpu, dev, device_rows
from workloads import CONFIGS, make_workload, scaled, table_rows

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "alg1_worked_example.json")


@pytest.fixture(autouse=True)
def _clean_error_word():
    if torch.cuda.is_available():
        S.check()
    yield
    if torch.cuda.is_available():
        assert S.check() == S.scone.OK, "a test left a device error behind"


def pad(rows, width, fill=-1):
    out = np.full((len(rows), width), fill, dtype=np.int32)
    for k, r in enumerate(rows):
        out[k, :len(r)] = r
    return out


def compare_lookup(w_fgrams, w_lengths, w_ids, X, max_n, max_load=0.5):
    o = oracle.OracleTable(w_fgrams, w_lengths, w_ids)
    exp_ids, exp_len = o.lookup(X, max_n)
    tb = build_gpu(w_fgrams, w_lengths, w_ids, max_load)
    ids, ml = S.lookup(tb, dev(X), max_n, want_len=True)
    S.check_ok()
    np.testing.assert_array_equal(ids.cpu().numpy(), exp_ids)
    np.testing.assert_array_equal(ml.cpu().numpy(), exp_len)
    return tb, exp_ids


def test_worked_example_through_gpu():
    g = json.load(open(GOLDEN))
    fg = pad(g["fgrams"], 4)
    ln = [len(r) for r in g["fgrams"]]
    tb = build_gpu(fg, ln, g["ids"])
    X = dev(np.array(g["tokens"], dtype=np.int32))
    for max_n, exp in g["expected"].items():
        ids, ml = S.lookup(tb, X, int(max_n), want_len=True)
        assert ids.cpu().tolist() == exp["ids"], max_n
        assert ml.cpu().tolist() == exp["len"], max_n


def test_tiny_full_parity():
    cfg = CONFIGS["tiny"]
    w = make_workload(cfg)
    tb, exp_ids = compare_lookup(w.fgrams, w.lengths, w.ids, w.tokens, cfg.max_n)
    E = device_rows(cfg)
    ids, _ = S.lookup(tb, dev(w.tokens), cfg.max_n)
    out = S.gather(ids, E)
    S.check_ok()
    exp = oracle.gather(exp_ids, E.cpu().numpy())
    assert as_bytes(out).tobytes() == exp.tobytes()


@pytest.mark.parametrize("max_len", [2, 3, 5, 6, 7])
@pytest.mark.parametrize("shape", [(1, 1), (3, 7), (2, 257), (5, 1000), (1, 4099)])
def test_lookup_shapes_and_windows(max_len, shape):
    V = 6  # tiny vocabulary: dense overlaps, every length matches somewhere
    possible = sum(V ** n for n in range(2, max_len + 1))
    cfg = scaled(CONFIGS["tiny"], V=V, n_fgrams=min(400, possible // 2), max_len=max_len,
                 B=shape[0], T=shape[1], coverage=0.5)
    w = make_workload(cfg, seed=11 * max_len + shape[1])
    for max_n in sorted({1, 2, max_len - 1, max_len, max_len + 3}):
        if max_n >= 1:
            compare_lookup(w.fgrams, w.lengths, w.ids, w.tokens, max_n)


def test_extreme_tokens_and_long_fgrams():
    hi = 65535
    rows = [[hi, 0], [0, hi, hi], [hi] * 7, [1, 2, 3, 4, 5, 6, 7], [7, 6, 5, 4, 3, 2],
            [hi, hi, hi, hi, hi, hi], [0, 0]]
    fg = pad(rows, 7)
    ln = [len(r) for r in rows]
    ids = [70000 + k for k in range(len(rows))]
    X = np.array([[hi] * 9 + [0, hi, hi] + [1, 2, 3, 4, 5, 6, 7, 6, 5, 4, 3, 2] + [0] * 4],
                 dtype=np.int32)
    X = np.concatenate([X, X[:, ::-1]])
    for max_n in range(1, 10):
        compare_lookup(fg, ln, ids, X, max_n)


def test_build_order_invariance():
    cfg = scaled(CONFIGS["c3_10m_k5"], n_fgrams=50_000, B=4, T=3000)
    w = make_workload(cfg)
    perm = np.random.default_rng(3).permutation(len(w.lengths))
    a = build_gpu(w.fgrams, w.lengths, w.ids)
    b = build_gpu(w.fgrams[perm], w.lengths[perm], w.ids[perm])
    X = dev(w.tokens)
    ia, la = S.lookup(a, X, 5, want_len=True)
    ib, lb = S.lookup(b, X, 5, want_len=True)
    assert torch.equal(ia, ib) and torch.equal(la, lb)


@pytest.mark.parametrize("max_load", [0.05, 0.5, 0.9])
def test_load_factors(max_load):
    cfg = scaled(CONFIGS["c2_1m"], n_fgrams=30_000, B=3, T=777)
    w = make_workload(cfg)
    tb, _ = compare_lookup(w.fgrams, w.lengths, w.ids, w.tokens, 3, max_load=max_load)
    assert tb.n == 30_000 and tb.capacity >= 30_000 / max_load
    assert tb.capacity & (tb.capacity - 1) == 0
    assert tb.entries == tb.n          # K = 3: no suffix markers


def test_table_entries_count_suffix_markers():
    """entries = the f-grams plus one marker per distinct length-3 suffix of an
    f-gram of length >= 4 that is not itself an f-gram, plus the extra copies
    that concurrent inserts of one marker may leave (at most one slot per long
    f-gram in all; a few percent of the markers on this Zipf set, whose
    frequent suffixes are shared by many f-grams)."""
    cfg = scaled(CONFIGS["c3_10m_k5"], n_fgrams=40_000, B=2, T=100)
    w = make_workload(cfg)
    tb = build_gpu(w.fgrams, w.lengths, w.ids, max_load=0.25)
    fgrams = {tuple(r[:L]) for r, L in zip(w.fgrams.tolist(), w.lengths.tolist())}
    long_ = [tuple(r[L - 3:L]) for r, L in zip(w.fgrams.tolist(), w.lengths.tolist()) if L >= 4]
    markers = {s for s in long_ if s not in fgrams}
    assert tb.n == len(fgrams)
    assert tb.n + len(markers) <= tb.entries <= tb.n + len(long_)
    assert tb.entries <= tb.n + len(markers) + max(8, len(markers) // 10)


def test_empty_inputs():
    tb = build_gpu(np.zeros((0, 3), np.int32), [], [])
    assert tb.n == 0
    X = dev(np.array([[5, 6, 7]], dtype=np.int32))
    ids, ml = S.lookup(tb, X, 3, want_len=True)
    assert ids.cpu().tolist() == [[5, 6, 7]] and ml.cpu().tolist() == [[1, 1, 1]]
    for B, T in [(0, 5), (4, 0), (0, 0)]:
        ids, _ = S.lookup(tb, torch.zeros((B, T), dtype=torch.int32, device="cuda"), 3)
        assert ids.shape == (B, T)
    E = torch.zeros((10, 8), dtype=torch.float32, device="cuda")
    out = S.gather(torch.zeros(0, dtype=torch.int32, device="cuda"), E)
    assert out.shape == (0, 8)


@pytest.mark.parametrize("row_bytes", [1, 2, 3, 6, 12, 16, 48, 256, 1024, 2048, 4096, 4100,
                                       8192])
@pytest.mark.parametrize("offset", [0, 1, 4])
def test_gather_row_widths_and_alignment(row_bytes, offset):
    rng = np.random.default_rng(row_bytes + offset)
    n_rows, n_tok = 300, 1537
    table = rng.integers(0, 256, size=(n_rows, row_bytes), dtype=np.uint8)
    ids = rng.integers(0, n_rows, size=n_tok).astype(np.int32)
    exp = oracle.gather(ids, table)
    E = dev(table)
    buf = torch.empty(n_tok * row_bytes + offset, dtype=torch.uint8, device="cuda")
    out = buf[offset:].view(n_tok, row_bytes)
    S.gather(dev(ids), E, out=out)
    S.check_ok()
    assert out.cpu().numpy().tobytes() == exp.tobytes()


def test_gather_keeps_special_bit_patterns():
    E = torch.randn(64, 32, dtype=torch.float32)
    E.view(torch.int32)[5, :5] = torch.tensor([0x80000000 - 2**32, 0x7F800000, 0x7FC01234,
                                               0xFFC00001 - 2**32, 1], dtype=torch.int32)
    Eb = torch.randn(64, 48).to(torch.bfloat16)
    Eb.view(torch.int16)[7, :3] = torch.tensor([-32768, 0x7FC1, 0x7F81], dtype=torch.int16)
    ids = np.array([5, 7, 5, 0, 63], dtype=np.int32)
    for T in (E, Eb):
        out = S.gather(dev(ids), T.cuda())
        S.check_ok()
        exp = oracle.gather(ids, T.view(torch.uint8).numpy())
        assert as_bytes(out).tobytes() == exp.tobytes()


def test_host_rows_gather():
    cfg = scaled(CONFIGS["tiny"], d=96)
    w = make_workload(cfg)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    host = S.HostRows(cfg.n_rows, (cfg.d,), torch.float32)
    try:
        host.tensor().copy_(table_rows(cfg, range(cfg.n_rows)))
        ids, _ = S.lookup(tb, dev(w.tokens), cfg.max_n)
        out = S.gather(ids, host)
        S.check_ok()
        o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
        exp_ids, _ = o.lookup(w.tokens, cfg.max_n)
        exp = oracle.gather(exp_ids, host.tensor().numpy())
        assert as_bytes(out).tobytes() == exp.tobytes()
    finally:
        host.close()


# ------------------------------------------------------------- errors ------

def raises_code(code, fn, *a, **kw):
    with pytest.raises(S.SconeError) as e:
        fn(*a, **kw)
    assert e.value.code == code, (e.value.code, code)


def test_build_errors():
    fg = pad([[1, 2], [2, 3], [3, 4, 5]], 3)
    raises_code(S.scone.EDUP, build_gpu, pad([[1, 2], [9, 9], [1, 2]], 3), [2, 2, 2], [10, 11, 12])
    raises_code(S.scone.ELEN, build_gpu, fg, [2, 1, 3], [10, 11, 12])
    raises_code(S.scone.ELEN, build_gpu, fg, [2, 2, 4], [10, 11, 12])
    raises_code(S.scone.EID, build_gpu, fg, [2, 2, 3], [10, -11, 12])
    raises_code(S.scone.ETOKEN, build_gpu, pad([[1, 70000]], 3), [2], [10])
    raises_code(S.scone.ETOKEN, build_gpu, pad([[-1, 2]], 3), [2], [10])
    raises_code(S.scone.EINVAL, build_gpu, fg, [2, 2, 3], [10, 11, 12], max_load=0.95)
    raises_code(S.scone.EINVAL, build_gpu, pad([[1, 2]], 8), [2], [10])
    # many duplicates among many keys, one key repeated once
    rng = np.random.default_rng(0)
    base = rng.integers(0, 60000, size=(20000, 3)).astype(np.int32)
    base = np.unique(base, axis=0)
    dup = np.concatenate([base, base[1234:1235]])
    raises_code(S.scone.EDUP, build_gpu, dup, np.full(len(dup), 3), np.arange(len(dup)) + 5)


def test_lookup_and_gather_errors_raise_through_check():
    tb = build_gpu(pad([[1, 2]], 3), [2], [10])
    X = dev(np.array([[1, 2, 65536, 3]], dtype=np.int32))
    ids, _ = S.lookup(tb, X, 3)
    assert S.check() == S.scone.ETOKEN
    assert S.check() == S.scone.OK  # cleared
    X = dev(np.array([[1, 2, -5]], dtype=np.int32))
    S.lookup(tb, X, 3)
    assert S.check() == S.scone.ETOKEN
    E = torch.arange(40, dtype=torch.float32, device="cuda").view(10, 4) + 1
    out = S.gather(dev(np.array([1, 10, 3, -1], dtype=np.int32)), E)
    assert S.check() == S.scone.EROW
    got = out.cpu()
    assert torch.equal(got[0], E[1].cpu()) and torch.equal(got[2], E[3].cpu())
    assert (got[1] == 0).all() and (got[3] == 0).all()
    # the same through the one-wavefront-per-row path (2 KiB rows)
    Eb = torch.arange(8 * 1024, dtype=torch.int16, device="cuda").view(8, 1024).to(torch.bfloat16)
    out = S.gather(dev(np.array([7, 8, 0, -3, 2], dtype=np.int32)), Eb)
    assert S.check() == S.scone.EROW
    got = out.cpu()
    assert torch.equal(got[0], Eb[7].cpu()) and torch.equal(got[2], Eb[0].cpu())
    assert (got[1].view(torch.int16) == 0).all() and (got[3].view(torch.int16) == 0).all()
    empty_rows = torch.zeros((0, 4), dtype=torch.float32, device="cuda")
    S.gather(dev(np.array([0], dtype=np.int32)), empty_rows)
    assert S.check() == S.scone.EROW
    raises_code(S.scone.EINVAL, S.lookup, tb, X, 0)


# ------------------------------------------------------- fused and decode --

@pytest.mark.parametrize("case", ["tiny", "c2_small", "c3_small", "k7_small", "odd_rows"])
@pytest.mark.parametrize("outputs", [True, False])
def test_embed_matches_oracle(case, outputs):
    if case == "tiny":
        cfg = CONFIGS["tiny"]
    elif case == "c2_small":
        cfg = scaled(CONFIGS["c2_1m"], n_fgrams=20_000, B=3, T=1500)
    elif case == "c3_small":
        cfg = scaled(CONFIGS["c3_10m_k5"], n_fgrams=40_000, B=2, T=2100, d=512)
    elif case == "k7_small":
        cfg = scaled(CONFIGS["tiny"], V=40, n_fgrams=3000, max_len=7, max_n=7, B=3, T=700, d=24)
    else:
        cfg = scaled(CONFIGS["tiny"], d=7, B=5, T=333)  # 28-byte rows: byte path
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    exp_ids, exp_len = o.lookup(w.tokens, cfg.max_n)
    E = device_rows(cfg)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    ids = torch.empty((cfg.B, cfg.T), dtype=torch.int32, device="cuda") if outputs else None
    ml = torch.empty((cfg.B, cfg.T), dtype=torch.int8, device="cuda") if outputs else None
    out = S.embed(tb, dev(w.tokens), cfg.max_n, E, fgram_ids=ids, match_len=ml)
    S.check_ok()
    exp = oracle.gather(exp_ids, E.cpu().view(torch.uint8).numpy())
    assert as_bytes(out).tobytes() == exp.tobytes()
    if outputs:
        np.testing.assert_array_equal(ids.cpu().numpy(), exp_ids)
        np.testing.assert_array_equal(ml.cpu().numpy(), exp_len)


def test_embed_errors_and_rowless_table():
    tb = build_gpu(pad([[1, 2]], 3), [2], [10])
    E = torch.arange(12 * 8, dtype=torch.float32, device="cuda").view(12, 8)
    X = dev(np.array([[1, 2, 11, 3]], dtype=np.int32))
    out = S.embed(tb, X, 3, E)
    S.check_ok()
    assert torch.equal(out[0, 1], E[10]) and torch.equal(out[0, 2], E[11])
    small = E[:5].contiguous()          # ids 10 and 11 fall outside
    ids = torch.empty((1, 4), dtype=torch.int32, device="cuda")
    out = S.embed(tb, X, 3, small, fgram_ids=ids)
    assert S.check() == S.scone.EROW
    assert ids.cpu().tolist() == [[1, 10, 11, 3]]
    assert (out[0, 1] == 0).all() and torch.equal(out[0, 0], small[1])
    S.embed(tb, dev(np.array([[1, 70000]], dtype=np.int32)), 3, E)
    assert S.check() == S.scone.ETOKEN
    out = S.embed(tb, X, 3, E[:0], fgram_ids=ids)
    assert S.check() == S.scone.EROW
    assert ids.cpu().tolist() == [[1, 10, 11, 3]] and (out == 0).all()


def decode_all(tb, X, max_n, E, cap, host=None):
    """Feed X[:, s] step by step; returns per-step ids, lens and rows."""
    Sq, steps = X.shape
    Xd = dev(X)
    ctx = torch.full((Sq, cap), -7, dtype=torch.int32, device="cuda")
    clen = torch.zeros(Sq, dtype=torch.int32, device="cuda")
    rows = E if host is None else host
    ids, lens, outs = [], [], []
    for s in range(steps):
        i = torch.empty(Sq, dtype=torch.int32, device="cuda")
        m = torch.empty(Sq, dtype=torch.int8, device="cuda")
        o = torch.empty((Sq, E.shape[1]), dtype=E.dtype, device="cuda")
        S.decode_step(tb, ctx, clen, Xd[:, s].contiguous(), max_n, rows, o, fgram_ids=i,
                      match_len=m)
        ids.append(i)
        lens.append(m)
        outs.append(o)
    S.check_ok()
    return (torch.stack(ids, 1).cpu().numpy(), torch.stack(lens, 1).cpu().numpy(),
            torch.stack(outs, 1))


@pytest.mark.parametrize("max_len,max_n,cap", [(3, 3, 2), (3, 3, 6), (5, 5, 4), (7, 7, 6),
                                               (3, 1, 0), (3, 9, 2)])
def test_decode_equals_prefill(max_len, max_n, cap):
    cfg = scaled(CONFIGS["c5_decode"], V=50 if max_len > 3 else 32768,
                 n_fgrams=4000 if max_len > 3 else 20_000, max_len=max_len, max_n=max_n, B=37,
                 T=40, d=64)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    exp_ids, exp_len = o.lookup(w.tokens, max_n)
    E = device_rows(cfg)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    ids, lens, outs = decode_all(tb, w.tokens, max_n, E, cap)
    np.testing.assert_array_equal(ids, exp_ids)
    np.testing.assert_array_equal(lens, exp_len)
    exp = oracle.gather(exp_ids, E.cpu().view(torch.uint8).numpy())
    assert as_bytes(outs).tobytes() == exp.tobytes()


def test_decode_host_rows_and_errors():
    cfg = scaled(CONFIGS["c5_decode"], n_fgrams=5000, B=16, T=12, d=128)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    exp_ids, _ = o.lookup(w.tokens, 3)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    host = S.HostRows(cfg.n_rows, (cfg.d,), torch.bfloat16)
    try:
        host.tensor().copy_(table_rows(cfg, range(cfg.n_rows)))
        E = torch.empty((1, cfg.d), dtype=torch.bfloat16, device="cuda")  # shape carrier only
        ids, _, outs = decode_all(tb, w.tokens, 3, E, 2, host=host)
        np.testing.assert_array_equal(ids, exp_ids)
        exp = oracle.gather(exp_ids, host.tensor().view(torch.uint8).numpy())
        assert as_bytes(outs).tobytes() == exp.tobytes()
    finally:
        host.close()
    ctx = torch.zeros((2, 2), dtype=torch.int32, device="cuda")
    clen = torch.zeros(2, dtype=torch.int32, device="cuda")
    out = torch.empty((2, 4), dtype=torch.float32, device="cuda")
    rows = torch.zeros((10, 4), dtype=torch.float32, device="cuda")
    raises_code(S.scone.EINVAL, S.decode_step, tb, ctx[:, :1].contiguous(), clen,
                dev(np.array([1, 2], np.int32)), 3, rows, out)  # context too short for max_n 3
    S.decode_step(tb, ctx, clen, dev(np.array([1, 70000], np.int32)), 3, rows, out)
    assert S.check() == S.scone.ETOKEN  # also EROW: token 70000 is not a row; lowest code wins


@pytest.mark.parametrize("max_len,max_n,d,T", [(3, 3, 1024, 8190), (5, 5, 2048, 4099),
                                               (3, 2, 1024, 8192), (7, 7, 512, 8191),
                                               (7, 6, 2048, 2053), (3, 3, 64, 9000)])
def test_embed_many_tiles_per_workgroup(max_len, max_n, d, T):
    # enough tiles that each resident workgroup walks several of them, with a
    # ragged last tile in most rows
    V = 32768 if max_len <= 5 else 60
    cfg = scaled(CONFIGS["c2_1m"], V=V, n_fgrams=30_000, max_len=max_len, max_n=max_n, d=d,
                 B=8, T=T)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    exp_ids, exp_len = o.lookup(w.tokens, max_n)
    E = device_rows(cfg)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    ids = torch.empty((cfg.B, cfg.T), dtype=torch.int32, device="cuda")
    ml = torch.empty((cfg.B, cfg.T), dtype=torch.int8, device="cuda")
    out = S.embed(tb, dev(w.tokens), max_n, E, fgram_ids=ids, match_len=ml)
    S.check_ok()
    np.testing.assert_array_equal(ids.cpu().numpy(), exp_ids)
    np.testing.assert_array_equal(ml.cpu().numpy(), exp_len)
    # rows: compare against the generator's rows for the oracle's ids
    exp_rows = table_rows(cfg, torch.from_numpy(exp_ids.reshape(-1).astype(np.int64)).cuda(),
                          device="cuda")
    assert torch.equal(out.view(-1, d).view(torch.int16), exp_rows.view(torch.int16))
    # and a sample of positions through the oracle's own gather
    rng = np.random.default_rng(0)
    pos = rng.integers(0, cfg.n_tok, size=512)
    sample_ids = exp_ids.reshape(-1)[pos]
    uniq, inv = np.unique(sample_ids, return_inverse=True)
    compact = table_rows(cfg, uniq).view(torch.uint8).numpy()
    exp = oracle.gather(inv.astype(np.int32), compact)
    got = out.view(cfg.n_tok, -1)[torch.from_numpy(pos).cuda()].cpu().view(torch.uint8).numpy()
    assert got.tobytes() == exp.tobytes()


# ----------------------------------------------------- split placement ----

@pytest.mark.parametrize("d,n_near,n_far,n_tok", [(64, 40, 500, 3000), (1024, 1000, 3000, 777),
                                                  (8, 3, 7, 1), (2048, 32768, 20000, 4100)])
def test_gather_split_matches_concatenated_table(d, n_near, n_far, n_tok):
    rng = np.random.default_rng(d + n_tok)
    table = rng.integers(-30000, 30000, size=(n_near + n_far, d), dtype=np.int16)
    # Zipf-like ids: many repeats among the far rows
    ids = np.minimum(rng.zipf(1.3, size=n_tok) - 1, n_near + n_far - 1).astype(np.int32)
    ids[::3] = rng.integers(0, n_near + n_far, size=len(ids[::3]))
    near = dev(table[:n_near]).view(torch.bfloat16)
    far = S.HostRows(n_far, (d,), torch.bfloat16)
    try:
        far.tensor().view(torch.int16).copy_(torch.from_numpy(table[n_near:]))
        ws = torch.empty(S.split_workspace_bytes(n_tok, 2 * d), dtype=torch.uint8, device="cuda")
        nu = torch.zeros(1, dtype=torch.int32, device="cuda")
        for _ in range(2):  # the workspace is reused across calls
            out = S.gather_split(dev(ids), near, far, ws, n_unique=nu)
            S.check_ok()
            assert out.cpu().view(torch.int16).numpy().tobytes() == \
                oracle.gather(ids, table).tobytes()
            assert int(nu.item()) == len(np.unique(ids[ids >= n_near]))
    finally:
        far.close()


def test_gather_split_errors():
    near = torch.zeros((4, 8), dtype=torch.float32, device="cuda") + 1
    far = S.HostRows(3, (8,), torch.float32)
    try:
        far.tensor().fill_(2)
        ids = dev(np.array([0, 5, 7, -1, 6], dtype=np.int32))
        ws = torch.empty(S.split_workspace_bytes(5, 32), dtype=torch.uint8, device="cuda")
        out = S.gather_split(ids, near, far, ws)
        assert S.check() == S.scone.EROW
        got = out.cpu()
        assert (got[0] == 1).all() and (got[1] == 2).all() and (got[4] == 2).all()
        assert (got[2] == 0).all() and (got[3] == 0).all()
        raises_code(S.scone.EINVAL, S.gather_split, ids, near, far, ws[:100])
    finally:
        far.close()


# ------------------------------------------------------- pre-scan tagger --

@pytest.mark.parametrize("name,max_n", [("tiny", 3), ("c3_10m_k5", 5), ("c3_10m_k5", 3)])
def test_tag_lengths_and_histogram(name, max_n):
    cfg = scaled(CONFIGS[name], n_fgrams=min(CONFIGS[name].n_fgrams, 40_000), B=7, T=3001)
    w = make_workload(cfg)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    _, exp_len = o.lookup(w.tokens, max_n)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    hist = torch.zeros(S.scone.MAX_FGRAM_LEN + 1, dtype=torch.int64, device="cuda")
    ml, _ = S.tag(tb, dev(w.tokens), max_n, hist=hist)
    S.tag(tb, dev(w.tokens), max_n, hist=hist, want_len=False)  # accumulates
    S.check_ok()
    np.testing.assert_array_equal(ml.cpu().numpy(), exp_len)
    expected = 2 * np.bincount(exp_len.reshape(-1).astype(np.int64),
                               minlength=S.scone.MAX_FGRAM_LEN + 1)
    np.testing.assert_array_equal(hist.cpu().numpy(), expected)
    raises_code(S.scone.EINVAL, S.tag, tb, dev(w.tokens), max_n, want_len=False)


# ------------------------------------------------------------ HIP graphs --

def test_graph_capture_replays_match_eager():
    """lookup + gather, the fused kernel, the split gather and a pipelined step
    captured once and replayed several times, with eager work and syncs
    between replays."""
    # 1 KiB rows: the pipelined step and the gather take their one-wavefront-per-row kernels
    cfg = scaled(CONFIGS["c2_1m"], n_fgrams=20_000, B=4, T=1000, d=512)
    w = make_workload(cfg)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    E = device_rows(cfg)
    X = dev(w.tokens)
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    exp_ids, _ = o.lookup(w.tokens, cfg.max_n)
    exp = oracle.gather(exp_ids, E.cpu().view(torch.uint8).numpy())
    ids = torch.empty((cfg.B, cfg.T), dtype=torch.int32, device="cuda")
    out_a = torch.empty((cfg.B, cfg.T, cfg.d), dtype=E.dtype, device="cuda")
    out_b = torch.empty_like(out_a)
    out_c = torch.empty_like(out_a)
    out_d = torch.empty_like(out_a)
    nxt = torch.empty_like(ids)
    near = E[:cfg.V].contiguous()
    far = S.HostRows(cfg.n_fgrams, (cfg.d,), E.dtype)
    try:
        far.tensor().copy_(E[cfg.V:].cpu())
        ws = torch.empty(S.split_workspace_bytes(cfg.n_tok, cfg.row_bytes), dtype=torch.uint8,
                         device="cuda")
        # eager once (also initialises the library's error word outside capture)
        S.lookup(tb, X, cfg.max_n, fgram_ids=ids)
        S.gather(ids, E, out=out_a)
        S.check_ok()
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            S.lookup(tb, X, cfg.max_n, fgram_ids=ids)
            S.gather(ids, E, out=out_a)
            S.embed(tb, X, cfg.max_n, E, out=out_b)
            S.gather_split(ids, near, far, ws, out=out_c)
            S.embed_pipelined(tb, X, cfg.max_n, nxt, ids, E, out=out_d)
        for r in range(4):
            for t in (ids, nxt, out_a, out_b, out_c, out_d):
                t.view(torch.uint8).fill_(0xA5)      # eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            S.check_ok()
            np.testing.assert_array_equal(ids.cpu().numpy(), exp_ids)
            np.testing.assert_array_equal(nxt.cpu().numpy(), exp_ids)
            for t in (out_a, out_b, out_c, out_d):
                assert as_bytes(t).tobytes() == exp.tobytes(), r
    finally:
        far.close()
