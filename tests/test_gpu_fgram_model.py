"""Parity of the precompute of F (scone_fgram_model_forward) with the oracle.

Tolerance, from the arithmetic.  The oracle is float64 on the bf16 parameter
values.  The kernels keep the residual stream in float32 and round to bf16 at
five points per layer (the two LayerNorm outputs, q/k/v, the attention output
and the GELU output, the inputs of the matrix products) plus the output row.
Each rounding has relative error at most u = 2^-9 and about u/sqrt(3) rms;
the linear maps carry a relative error through unchanged and the residual
sums add independent errors in quadrature, so an output row's relative rms
error is about

    eps(L) = u * sqrt((5 L + 2) / 3)          (L = number of layers).

The bar: every row's relative L2 error at most 3 eps(L), and every element
within 12 eps(L) times its row's rms.  A dropped bias or gain (0.1 relative
with the "unit" parameters), a wrong mask, position or head split moves rows
by far more.
"""
import os

import numpy as np
import pytest
import torch

import paper_2502_01637_amd as S
from oracle import fgram_model as orc
from workloads import CONFIGS, make_workload
from workloads.fgram_model import (GPT2_128M, ModelConfig, make_params, make_token_rows,
                                   bf16_bits_to_f64)
from gpu_util import dev

pytestmark = pytest.mark.gpu

U = 2.0 ** -9


def eps(n_layers):
    return U * np.sqrt((5 * n_layers + 2) / 3)


def assert_close(got, ref, n_layers, what=""):
    got = np.asarray(got, dtype=np.float64)
    e = eps(n_layers)
    err = got - ref
    row = np.linalg.norm(err, axis=1) / np.linalg.norm(ref, axis=1)
    rms = np.sqrt((ref ** 2).mean(axis=1, keepdims=True))
    el = np.abs(err) / rms
    assert np.isfinite(got).all(), what
    assert row.max() <= 3 * e, f"{what}: row error {row.max():.5f} > {3 * e:.5f}"
    assert el.max() <= 12 * e, f"{what}: element error {el.max():.5f} > {12 * e:.5f}"


def random_fgrams(rng, V, N, K, lengths=None):
    if lengths is None:
        lengths = rng.integers(2, K + 1, size=N)
    lengths = np.asarray(lengths, dtype=np.int32)
    fg = rng.integers(0, V, size=(len(lengths), K)).astype(np.int32)
    for i, n in enumerate(lengths):
        fg[i, n:] = -1
    return fg, lengths


def bf16_dev(bits):
    return torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)


def run(cfg, fg, lengths, row_ids, T_bits, params_bits, n_rows):
    model = S.FgramModel(params_bits, cfg.d, cfg.n_heads, cfg.d_ff, cfg.n_layers, cfg.max_len)
    rows = torch.zeros((n_rows, cfg.d), dtype=torch.bfloat16, device="cuda")
    S.precompute_fgram_rows(model, dev(fg), dev(lengths), dev(row_ids), bf16_dev(T_bits), rows)
    return rows


def as_f64(rows_t):
    return rows_t.float().cpu().numpy().astype(np.float64)


CASES = [
    # d, heads, d_ff, layers, K, N: several GEMM tiles, ragged tails, every length
    (ModelConfig(512, 8, 1024, 2, 7), 3000),
    (ModelConfig(512, 4, 1536, 3, 3), 2000),    # 128-wide heads, d_ff not a power of two
    (ModelConfig(1024, 16, 4096, 1, 5), 500),
    (ModelConfig(1536, 12, 1024, 1, 4), 300),   # d = 3 * 512, 128-wide heads
    (ModelConfig(512, 8, 512, 0, 6), 700),      # no layers: LNf(T + pos)
]


@pytest.mark.parametrize("cfg,N", CASES, ids=[f"d{c.d}h{c.n_heads}f{c.d_ff}L{c.n_layers}K{c.max_len}"
                                            for c, _ in CASES])
def test_forward_matches_oracle(cfg, N):
    rng = np.random.default_rng(cfg.d + cfg.n_layers)
    V = 500
    P = make_params(cfg, seed=11)
    T = make_token_rows(V, cfg.d, seed=12)
    fg, lengths = random_fgrams(rng, V, N, cfg.max_len)
    row_ids = (rng.permutation(N) + 7).astype(np.int32)   # scattered, not in order
    rows = run(cfg, fg, lengths, row_ids, T, P, N + 7)
    ref = orc.forward(fg, lengths, bf16_bits_to_f64(T),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, cfg.n_layers, cfg.n_heads)
    got = as_f64(rows)
    assert_close(got[row_ids], ref, cfg.n_layers, "rows")
    untouched = np.setdiff1d(np.arange(N + 7), row_ids)
    assert not got[untouched].any()


def test_tiny_and_empty_buckets():
    """Buckets of 1, 2 and 3 f-grams (products with M < 16) next to empty
    lengths; 128-wide heads so the attention takes its other lane grouping."""
    cfg = ModelConfig(512, 4, 768, 2, 7)
    rng = np.random.default_rng(10)
    V = 200
    P = make_params(cfg, seed=71)
    T = make_token_rows(V, cfg.d, seed=72)
    lengths = np.array([7, 2, 5, 5, 7, 5], dtype=np.int32)   # no 3, 4 or 6
    fg, lengths = random_fgrams(rng, V, len(lengths), cfg.max_len, lengths)
    ids = np.array([5, 0, 3, 1, 4, 2], dtype=np.int32)
    got = as_f64(run(cfg, fg, lengths, ids, T, P, 6))
    ref = orc.forward(fg, lengths, bf16_bits_to_f64(T),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, cfg.n_layers, cfg.n_heads)
    assert_close(got[ids], ref, cfg.n_layers, "tiny buckets")


def test_several_chunks_per_length():
    """More than 65536 tokens of one length: the bucket runs in several chunks."""
    cfg = ModelConfig(512, 8, 512, 1, 3)
    rng = np.random.default_rng(5)
    V = 1000
    N = 70000
    P = make_params(cfg, seed=21)
    T = make_token_rows(V, cfg.d, seed=22)
    lengths = np.where(rng.random(N) < 0.5, 2, 3).astype(np.int32)
    fg, lengths = random_fgrams(rng, V, N, cfg.max_len, lengths)
    row_ids = np.arange(N, dtype=np.int32)
    got = as_f64(run(cfg, fg, lengths, row_ids, T, P, N))
    sample = np.sort(rng.choice(N, 1500, replace=False))
    sample = np.union1d(sample, [0, N - 1])
    ref = orc.forward(fg[sample], lengths[sample], bf16_bits_to_f64(T),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, cfg.n_layers, cfg.n_heads)
    assert_close(got[sample], ref, cfg.n_layers, "sampled rows")


def test_bit_identical_under_permutation_and_repeat():
    """Each f-gram's arithmetic does not depend on where it sits in a chunk."""
    cfg = ModelConfig(512, 8, 1024, 2, 5)
    rng = np.random.default_rng(6)
    V = 300
    P = make_params(cfg, seed=31)
    T = make_token_rows(V, cfg.d, seed=32)
    fg, lengths = random_fgrams(rng, V, 1500, cfg.max_len)
    ids = np.arange(1500, dtype=np.int32)
    a = run(cfg, fg, lengths, ids, T, P, 1500).view(torch.int16).cpu().numpy()
    b = run(cfg, fg, lengths, ids, T, P, 1500).view(torch.int16).cpu().numpy()
    perm = rng.permutation(1500)
    c = run(cfg, fg[perm], lengths[perm], ids[perm], T, P, 1500).view(torch.int16).cpu().numpy()
    assert np.array_equal(a, b)
    assert np.array_equal(a, c)


def test_unified_table_end_to_end():
    """Token rows T are the first V rows of the table; F is precomputed into the
    f-gram rows; lookup + gather then return F(longest f-gram) per position."""
    cfg = ModelConfig(512, 8, 1024, 2, 3)
    rng = np.random.default_rng(7)
    V, N = 400, 2000
    P = make_params(cfg, seed=41)
    fg, lengths = random_fgrams(rng, V, N, cfg.max_len)
    keep = []
    seen = set()
    for i, (r, n) in enumerate(zip(fg.tolist(), lengths)):
        t = tuple(r[:n])
        if t not in seen:
            seen.add(t)
            keep.append(i)
    fg, lengths = fg[keep], lengths[keep]
    N = len(keep)
    ids = (V + np.arange(N)).astype(np.int32)
    table_rows = torch.zeros((V + N, cfg.d), dtype=torch.bfloat16, device="cuda")
    T_bits = make_token_rows(V, cfg.d, seed=42)
    table_rows[:V].copy_(bf16_dev(T_bits))
    model = S.FgramModel(P, cfg.d, cfg.n_heads, cfg.d_ff, cfg.n_layers, cfg.max_len)
    S.precompute_fgram_rows(model, dev(fg), dev(lengths), dev(ids), table_rows[:V], table_rows)
    ref = orc.forward(fg, lengths, bf16_bits_to_f64(T_bits),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, cfg.n_layers, cfg.n_heads)
    got = as_f64(table_rows)
    assert_close(got[V:], ref, cfg.n_layers, "F rows")
    assert np.array_equal(table_rows[:V].view(torch.int16).cpu().numpy(), T_bits.view(np.int16))
    # the inference path over a token stream with planted f-grams
    X = rng.integers(0, V, size=(4, 300)).astype(np.int32)
    for b in range(4):
        for t in range(0, 290, 10):
            g = rng.integers(N)
            X[b, t:t + lengths[g]] = fg[g, :lengths[g]]
    tb = S.build_fgram_table(dev(fg), dev(lengths), dev(ids))
    fid, _ = S.lookup(tb, dev(X), cfg.max_len, want_len=True)
    out = S.gather(fid, table_rows)
    S.check_ok()
    fid = fid.cpu().numpy()
    assert (fid >= V).any()
    exp = table_rows.view(torch.int16).cpu().numpy()[fid]
    assert np.array_equal(out.view(torch.int16).cpu().numpy(), exp)


def test_errors():
    cfg = ModelConfig(512, 8, 512, 1, 3)
    rng = np.random.default_rng(8)
    V, N = 100, 50
    P = make_params(cfg, seed=51)
    T = make_token_rows(V, cfg.d, seed=52)
    fg, lengths = random_fgrams(rng, V, N, cfg.max_len)
    ids = np.arange(N, dtype=np.int32)
    model = S.FgramModel(P, cfg.d, cfg.n_heads, cfg.d_ff, cfg.n_layers, cfg.max_len)
    Tt = bf16_dev(T)

    def call(fg_, ln_, id_, n_rows=N):
        rows = torch.zeros((n_rows, cfg.d), dtype=torch.bfloat16, device="cuda")
        S.precompute_fgram_rows(model, dev(fg_), dev(ln_), dev(id_), Tt, rows)
        return rows

    bad = lengths.copy(); bad[7] = 1
    with pytest.raises(S.SconeError) as e:
        call(fg, bad, ids)
    assert e.value.code == S.scone.ELEN
    bad = lengths.copy(); bad[3] = 4
    with pytest.raises(S.SconeError) as e:
        call(fg, bad, ids)
    assert e.value.code == S.scone.ELEN
    badf = fg.copy(); badf[5, 0] = V
    with pytest.raises(S.SconeError) as e:
        call(badf, lengths, ids)
    assert e.value.code == S.scone.ETOKEN
    badf = fg.copy(); badf[6, 1] = -3
    with pytest.raises(S.SconeError) as e:
        call(badf, lengths, ids)
    assert e.value.code == S.scone.ETOKEN
    badi = ids.copy(); badi[9] = N
    with pytest.raises(S.SconeError) as e:
        call(fg, lengths, badi)
    assert e.value.code == S.scone.EROW
    # pads past the length are ignored, whatever they hold
    padded = fg.copy()
    for i, n in enumerate(lengths):
        padded[i, n:] = 10 ** 6
    a = call(fg, lengths, ids).view(torch.int16).cpu().numpy()
    b = call(padded, lengths, ids).view(torch.int16).cpu().numpy()
    assert np.array_equal(a, b)
    # empty input is a no-op
    rows = torch.zeros((4, cfg.d), dtype=torch.bfloat16, device="cuda")
    S.precompute_fgram_rows(model, dev(np.zeros((0, 3), np.int32)), dev(np.zeros(0, np.int32)),
                            dev(np.zeros(0, np.int32)), Tt, rows)
    assert not rows.any()


def test_full_size_gpt2_128m_on_1m_fgrams():
    """The 1M f-gram set of the d = 1024 workload through the 6-layer 128M-shape
    f-gram model, every row written; a sample checked against the oracle."""
    cfg = GPT2_128M
    wcfg = CONFIGS["c2_1m"]
    w = make_workload(wcfg)
    P = make_params(cfg, seed=61)
    T = make_token_rows(wcfg.V, cfg.d, seed=62)
    fg = np.ascontiguousarray(w.fgrams[:, :cfg.max_len])
    rows = run(cfg, fg, w.lengths, w.ids, T, P, wcfg.n_rows)
    got_bits = rows.view(torch.int16)
    assert not got_bits[:wcfg.V].any()          # token rows untouched
    written = (got_bits[wcfg.V:] != 0).any(dim=1)
    assert bool(written.all())
    rng = np.random.default_rng(9)
    sample = rng.choice(len(w.ids), 48, replace=False)
    ref = orc.forward(fg[sample], w.lengths[sample], bf16_bits_to_f64(T),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, cfg.n_layers, cfg.n_heads)
    got = as_f64(rows[torch.from_numpy(w.ids[sample].astype(np.int64)).cuda()])
    assert_close(got, ref, cfg.n_layers, "sampled rows")


# Random model shapes (seeds 50000 + case): widths that are not multiples of
# 256, fc2 depths down to two 64-deep slabs, 0-2 layers, 1 to 5,000 f-grams.
# SCONE_MODEL_SWEEP sets the number of cases (1,000 take about four minutes).
MODEL_CASES = int(os.environ.get("SCONE_MODEL_SWEEP", "6"))


@pytest.mark.parametrize("case", range(MODEL_CASES))
def test_random_model_shapes(case):
    rng = np.random.default_rng(50000 + case)
    d = int(rng.choice([512, 1024, 1536, 2048]))
    dh = int(rng.choice([64, 128]))
    d_ff = int(rng.choice([128, 384, 512, 1024, 2048, 4096]))
    layers = int(rng.integers(0, 3))
    K = int(rng.integers(2, 8))
    N = int(rng.choice([1, 2, 7, 15, 16, 17, 255, 256, 257, 1000, 3000,
                        int(rng.integers(1, 5000))]))
    V = int(rng.choice([5, 300, 5000]))
    cfg = ModelConfig(d, d // dh, d_ff, layers, K)
    P = make_params(cfg, seed=case)
    T = make_token_rows(V, d, seed=case + 1)
    fg, lengths = random_fgrams(rng, V, N, K)
    row_ids = (rng.permutation(N) + 3).astype(np.int32)
    got = as_f64(run(cfg, fg, lengths, row_ids, T, P, N + 3))
    sample = np.sort(rng.choice(N, min(N, 200), replace=False))
    ref = orc.forward(fg[sample], lengths[sample], bf16_bits_to_f64(T),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, layers, d // dh)
    assert_close(got[row_ids[sample]], ref, layers, f"case {case}")
    assert not got[[0, 1, 2]].any()
