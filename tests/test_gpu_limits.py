"""Indices past 32 bits.

A lookup and a tagging pass over more than 2^31 positions, and gathers whose
outputs hold more than 2^31 copy units (34 GB of 4 KiB rows on the
one-wavefront-per-row path and in the pipelined step, 4.3 GB of 50-byte rows
on the flat path, which moves them as 2-byte units).  Positions are sampled
at random, at both ends of every row and on both sides of the 2^31 boundary,
and compared with the oracle: a lookup position through the oracle's lookup
of the window that ends there (a window never reaches before its row's
start), a gathered row through the oracle's memcpy gather.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S
from gpu_util import build_gpu
from workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu

BOUNDARY = 1 << 31


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    gc.collect()
    if torch.cuda.is_available():
        torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def tiny():
    w = make_workload(CONFIGS["tiny"])
    return w, oracle.OracleTable(w.fgrams, w.lengths, w.ids)


def oracle_at(o, X, b, t, K, max_n):
    """Oracle (id, length) at positions (b[i], t[i]) of the device tensor X
    [B, T], each from the window of at most K tokens that ends there."""
    T = X.shape[1]
    ids = np.empty(len(b), dtype=np.int32)
    lens = np.empty(len(b), dtype=np.int8)
    full = t >= K - 1
    if full.any():
        f = torch.from_numpy(b[full] * T + t[full]).cuda()
        idx = f[:, None] + torch.arange(-(K - 1), 1, device="cuda")[None, :]
        win = X.view(-1)[idx].cpu().numpy()
        i, l = o.lookup(win, max_n)
        ids[full], lens[full] = i[:, -1], l[:, -1]
    for k in np.nonzero(~full)[0]:
        win = X[b[k], :t[k] + 1].cpu().numpy()[None, :]
        i, l = o.lookup(win, max_n)
        ids[k], lens[k] = i[0, -1], l[0, -1]
    return ids, lens


def test_lookup_and_tag_past_2_31_positions(tiny):
    w, o = tiny
    cfg = CONFIGS["tiny"]
    B, T = 2, (1 << 30) + 1024                      # 2^31 + 2048 positions
    base = torch.from_numpy(np.ascontiguousarray(w.tokens.reshape(-1))).cuda()
    X = torch.empty((B, T), dtype=torch.int32, device="cuda")
    reps = T // base.numel() + 1
    X[0] = base.repeat(reps)[:T]
    X[1] = torch.roll(base, 37).repeat(reps)[:T]
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    ids, lens = S.lookup(tb, X, cfg.max_n, want_len=True)
    hist = torch.zeros(S.scone.MAX_FGRAM_LEN + 1, dtype=torch.int64, device="cuda")
    tag_len, _ = S.tag(tb, X, cfg.max_n, hist=hist)
    S.check_ok()
    assert int(hist.sum().item()) == B * T
    assert torch.equal(tag_len, lens)
    for n in range(1, cfg.max_len + 1):
        assert int(hist[n].item()) == int((lens == n).sum().item())

    rng = np.random.default_rng(7)
    K = cfg.max_len
    b = [rng.integers(0, B, size=3000)]
    t = [rng.integers(0, T, size=3000)]
    for row in range(B):                             # both ends of each row
        b.append(np.full(2 * K + 64, row))
        t.append(np.concatenate([np.arange(K + 32), np.arange(T - K - 32, T)]))
    flat = np.arange(BOUNDARY - 64, BOUNDARY + 64)   # both sides of 2^31
    b.append(flat // T)
    t.append(flat % T)
    b, t = np.concatenate(b).astype(np.int64), np.concatenate(t).astype(np.int64)
    exp_ids, exp_lens = oracle_at(o, X, b, t, K, cfg.max_n)
    sel = torch.from_numpy(b * T + t).cuda()
    assert np.array_equal(ids.view(-1)[sel].cpu().numpy(), exp_ids)
    assert np.array_equal(lens.view(-1)[sel].cpu().numpy(), exp_lens)
    assert (exp_lens > 1).mean() > 0.3                # the sample sees matches


def sample_positions(n_tok, unit_row, rng):
    return np.unique(np.concatenate([
        rng.integers(0, n_tok, size=2000), np.arange(64), np.arange(n_tok - 64, n_tok),
        np.arange(unit_row - 64, unit_row + 64)]))


def rows_equal_oracle(out, ids, table, pos):
    exp = oracle.gather(ids[torch.from_numpy(pos).cuda()].cpu().numpy(),
                        table.cpu().view(torch.uint8).numpy())
    got = out[torch.from_numpy(pos).cuda()].cpu().view(torch.uint8).numpy()
    return got.tobytes() == exp.tobytes()


def test_gather_wave_rows_past_2_31_units():
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    table = torch.randint(-32768, 32768, (10000, 2048), dtype=torch.int16, device="cuda",
                          generator=g)                 # 4 KiB rows: 256 units each
    n_tok = BOUNDARY // 256 + 12_392                 # 34.4 GB of output
    ids = torch.randint(0, 10000, (n_tok,), dtype=torch.int32, device="cuda", generator=g)
    out = S.gather(ids, table)
    S.check_ok()
    pos = sample_positions(n_tok, BOUNDARY // 256, np.random.default_rng(3))
    assert rows_equal_oracle(out, ids, table, pos)


def test_gather_flat_units_past_2_31():
    g = torch.Generator(device="cuda")
    g.manual_seed(12)
    table = torch.randint(-32768, 32768, (10000, 25), dtype=torch.int16, device="cuda",
                          generator=g)                 # 50-byte rows: 25 two-byte units
    n_tok = BOUNDARY // 25 + 5_000                   # 4.3 GB of output
    ids = torch.randint(0, 10000, (n_tok,), dtype=torch.int32, device="cuda", generator=g)
    out = S.gather(ids, table)
    S.check_ok()
    pos = sample_positions(n_tok, BOUNDARY // 25, np.random.default_rng(4))
    assert rows_equal_oracle(out, ids, table, pos)


def test_pipelined_step_past_2_31_units(tiny):
    w, o = tiny
    cfg = CONFIGS["tiny"]
    g = torch.Generator(device="cuda")
    g.manual_seed(13)
    table = torch.randint(-32768, 32768, (11000, 2048), dtype=torch.int16, device="cuda",
                          generator=g)
    n_tok = BOUNDARY // 256 + 12_392
    cur = torch.randint(0, 11000, (n_tok,), dtype=torch.int32, device="cuda", generator=g)
    tb = build_gpu(w.fgrams, w.lengths, w.ids)
    X = torch.from_numpy(w.tokens).cuda()
    nxt = torch.empty_like(X)
    out = S.embed_pipelined(tb, X, cfg.max_n, nxt, cur, table)
    S.check_ok()
    exp_ids, _ = o.lookup(w.tokens, cfg.max_n)
    assert np.array_equal(nxt.cpu().numpy(), exp_ids)
    pos = sample_positions(n_tok, BOUNDARY // 256, np.random.default_rng(5))
    assert rows_equal_oracle(out, cur, table, pos)
