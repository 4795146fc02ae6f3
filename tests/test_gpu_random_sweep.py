"""Seeded random sweep of the whole inference path against the oracle.

Each case draws a vocabulary, an f-gram set (half taken from windows of the
query stream itself, so every length hits; half random), a query matrix with
ragged tails, a window max_n on either side of K and a row table of an odd or
even width, then checks every call through the C ABI against the CPU oracle:
lookup ids and lengths, the tagger's lengths and histogram, the gather and the
fused kernel byte for byte, a two-batch pipelined stream, decoding step by step
against prefill, and the split placement.  The sweep is deterministic (fixed seeds) and prints the case
it is on.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S
from gpu_util import as_bytes, build_gpu, dev

pytestmark = pytest.mark.gpu


def draw_case(rng):
    K = int(rng.integers(2, 8))
    V = int(rng.choice([3, 17, 300, 5000, 65536]))
    B = int(rng.integers(1, 5))
    T = int(rng.integers(0, 700))
    X = rng.integers(0, V, size=(B, T)).astype(np.int32)
    # f-grams: windows of X (so matches of every length exist) and random ones
    want = int(rng.integers(1, 3000))
    seen, rows = set(), []
    for _ in range(want):
        n = int(rng.integers(2, K + 1))
        if T >= n and rng.random() < 0.5:
            b, t = int(rng.integers(B)), int(rng.integers(n - 1, T))
            g = tuple(int(v) for v in X[b, t - n + 1:t + 1])
        else:
            g = tuple(int(v) for v in rng.integers(0, V, size=n))
        if g not in seen:
            seen.add(g)
            rows.append(g)
    fg = np.full((len(rows), K), -1, dtype=np.int32)
    for k, g in enumerate(rows):
        fg[k, :len(g)] = g
    lengths = np.array([len(g) for g in rows], dtype=np.int32)
    ids = (V + rng.permutation(len(rows))).astype(np.int32)
    max_n = int(rng.choice([1, 2, K, K, K + 2]))
    row_bytes = int(rng.choice([4, 12, 16, 40, 256, 2048, 4112]))
    max_load = float(rng.choice([0.3, 0.5, 0.9]))
    return K, V, X, fg, lengths, ids, max_n, row_bytes, max_load


# Blocks of 15 cases (seeds 9000 + case); SCONE_SWEEP_BLOCKS widens the sweep
# (700 blocks = 10,500 cases, about eight minutes on one MI355X).
BLOCKS = int(os.environ.get("SCONE_SWEEP_BLOCKS", "4"))


@pytest.mark.parametrize("block", range(BLOCKS))
def test_random_sweep(block):
    for case in range(block * 15, block * 15 + 15):
        rng = np.random.default_rng(9000 + case)
        K, V, X, fg, lengths, ids, max_n, row_bytes, max_load = draw_case(rng)
        B, T = X.shape
        what = (f"case {case}: K={K} V={V} B={B} T={T} f-grams={len(lengths)} max_n={max_n} "
                f"row_bytes={row_bytes} max_load={max_load}")
        print(what, flush=True)
        o = oracle.OracleTable(fg, lengths, ids)
        exp_ids, exp_len = o.lookup(X, max_n)
        n_rows = V + len(lengths)
        table = rng.integers(0, 256, size=(n_rows, row_bytes), dtype=np.uint8)
        E = dev(table)
        exp_rows = oracle.gather(exp_ids, table)

        tb = build_gpu(fg, lengths, ids, max_load)
        Xd = dev(X)
        got_ids, got_len = S.lookup(tb, Xd, max_n, want_len=True)
        hist = torch.zeros(S.scone.MAX_FGRAM_LEN + 1, dtype=torch.int64, device="cuda")
        tag_len, _ = S.tag(tb, Xd, max_n, hist=hist)
        out = S.gather(got_ids, E)
        fused = S.embed(tb, Xd, max_n, E)
        S.check_ok()
        np.testing.assert_array_equal(got_ids.cpu().numpy(), exp_ids, err_msg=what)
        np.testing.assert_array_equal(got_len.cpu().numpy(), exp_len, err_msg=what)
        np.testing.assert_array_equal(tag_len.cpu().numpy(), exp_len, err_msg=what)
        h = hist.cpu().numpy()
        assert h[0] == 0 and h.sum() == B * T, what
        np.testing.assert_array_equal(h[1:K + 1],
                                      np.bincount(exp_len.ravel(), minlength=K + 1)[1:K + 1],
                                      err_msg=what)
        assert as_bytes(out).tobytes() == exp_rows.tobytes(), what
        assert as_bytes(fused).tobytes() == exp_rows.tobytes(), what

        # pipelined step, a stream of two batches (X, then X reversed along T):
        # step 0 looks up X; step 1 looks up the second batch while gathering
        # X's rows, on the case's row width (one launch for 1/2/4/8 KiB rows,
        # the two kernels otherwise) and on a random width of whole KiB
        X2 = np.ascontiguousarray(X[:, ::-1])
        exp_ids2, _ = o.lookup(X2, max_n)
        rng2 = np.random.default_rng(19000 + case)
        rb2 = int(rng2.choice([1024, 2048, 4096, 8192]))
        table2 = rng2.integers(0, 256, size=(n_rows, rb2), dtype=np.uint8)
        for tab, Et, exp_r in ((table, E, exp_rows),
                               (table2, dev(table2), oracle.gather(exp_ids, table2))):
            p0 = torch.empty((B, T), dtype=torch.int32, device="cuda")
            p1 = torch.empty((B, T), dtype=torch.int32, device="cuda")
            S.embed_pipelined(tb, Xd, max_n, p0, None, Et)
            pout = S.embed_pipelined(tb, dev(X2), max_n, p1, p0, Et)
            S.check_ok()
            np.testing.assert_array_equal(p0.cpu().numpy(), exp_ids, err_msg=what)
            np.testing.assert_array_equal(p1.cpu().numpy(), exp_ids2, err_msg=what)
            assert as_bytes(pout).tobytes() == exp_r.tobytes(), what

        if row_bytes % 16 == 0 and B * T > 0:
            # split placement: token rows in HBM, f-gram rows in pinned host memory
            far = S.HostRows(len(lengths), (row_bytes,), torch.uint8)
            try:
                far.tensor().copy_(torch.from_numpy(table[V:]))
                ws = torch.empty(S.split_workspace_bytes(B * T, row_bytes), dtype=torch.uint8,
                                 device="cuda")
                split = S.gather_split(got_ids, E[:V].contiguous(), far, ws)
                S.check_ok()
                assert as_bytes(split).tobytes() == exp_rows.tobytes(), what
            finally:
                far.close()

        if B * T > 0 and max_n >= 1 and T <= 64:
            # decoding: one step per position, context of max(min(max_n, K) - 1, 0)
            cap = max(min(max_n, K) - 1, 0)
            ctx = torch.zeros((B, cap), dtype=torch.int32, device="cuda")
            clen = torch.zeros(B, dtype=torch.int32, device="cuda")
            for t in range(T):
                step_out = torch.empty((B, row_bytes), dtype=torch.uint8, device="cuda")
                sid = torch.empty(B, dtype=torch.int32, device="cuda")
                S.decode_step(tb, ctx, clen, Xd[:, t].contiguous(), max_n, E, step_out,
                              fgram_ids=sid)
                np.testing.assert_array_equal(sid.cpu().numpy(), exp_ids[:, t], err_msg=what)
                assert as_bytes(step_out).tobytes() == exp_rows[:, t].tobytes(), what
            S.check_ok()
        tb.close()
