"""The seeded generator: determinism, distinct f-grams, coverage, table bits."""
import numpy as np
import torch

from workloads import CONFIGS, make_workload, scaled, table_rows, fill_table, torch_dtype
from checks import fgram_dict


def test_deterministic_and_distinct():
    cfg = scaled(CONFIGS["c3_10m_k5"], n_fgrams=40_000, B=4, T=1024)
    a, b = make_workload(cfg), make_workload(cfg)
    for f in ("fgrams", "lengths", "ids", "tokens", "planted"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    assert len(fgram_dict(a.fgrams, a.lengths, a.ids)) == cfg.n_fgrams
    assert a.lengths.min() >= 2 and a.lengths.max() <= 5
    assert (a.fgrams[np.arange(5)[None, :] >= a.lengths[:, None]] == -1).all()
    assert a.tokens.min() >= 0 and a.tokens.max() < cfg.V
    assert np.array_equal(a.ids, cfg.V + np.arange(cfg.n_fgrams))
    c = make_workload(cfg, seed=7)
    assert not np.array_equal(a.tokens, c.tokens)


def test_planted_coverage_near_target():
    for name in ("c2_1m", "c3_10m_k5"):
        cfg = scaled(CONFIGS[name], n_fgrams=50_000, B=8, T=2048)
        w = make_workload(cfg)
        assert abs(w.planted.mean() - cfg.coverage) < 0.03, name


def test_table_rows_match_full_fill_and_stats():
    cfg = scaled(CONFIGS["c2_1m"], n_fgrams=3000, d=256)
    full = torch.empty((cfg.n_rows, cfg.d), dtype=torch_dtype(cfg))
    fill_table(cfg, full, chunk_elems=100_003)
    rows = [0, 1, 17, cfg.n_rows - 1]
    assert torch.equal(table_rows(cfg, rows), full[rows])
    f = full.float()
    assert abs(f.std().item() - cfg.std) < 0.002 and abs(f.mean().item()) < 0.001
    tiny = CONFIGS["tiny"]
    t = table_rows(tiny, range(tiny.n_rows))
    assert t.dtype == torch.float32 and abs(t.std().item() - 1.0) < 0.01
    # different seeds give different tables
    assert not torch.equal(table_rows(cfg, rows, seed=1), table_rows(cfg, rows, seed=2))
