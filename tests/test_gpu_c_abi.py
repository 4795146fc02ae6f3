"""The C ABI from plain C: paper_2502_01637_amd/examples/scone_embed.c (C99,
HIP runtime and libscone.so only, built by the package's build step) builds
the dictionary, looks up and gathers on the GPU; its outputs are compared
with the oracle bit for bit."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2502_01637_amd import _build
from workloads import CONFIGS, make_workload, scaled

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,row_bytes", [("tiny", 256), ("c3_10m_k5", 4112)])
def test_plain_c_program_matches_oracle(tmp_path, name, row_bytes):
    if not os.path.exists(_build.EXAMPLE):
        pytest.fail(f"{_build.EXAMPLE} is missing: run the package build first")
    cfg = scaled(CONFIGS[name], n_fgrams=5000, B=3, T=777)
    w = make_workload(cfg)
    K = w.fgrams.shape[1]
    n_rows = cfg.V + len(w.ids)
    rows = np.random.default_rng(5).integers(0, 256, size=(n_rows, row_bytes), dtype=np.uint8)
    d = tmp_path
    (d / "meta.txt").write_text(f"{len(w.ids)} {K} {cfg.B} {cfg.T} {cfg.max_n} {n_rows} "
                                f"{row_bytes}\n")
    for fname, arr in (("fgrams.bin", w.fgrams), ("lengths.bin", w.lengths),
                       ("ids.bin", w.ids), ("tokens.bin", w.tokens), ("rows.bin", rows)):
        np.ascontiguousarray(arr).tofile(d / fname)
    r = subprocess.run([_build.EXAMPLE, str(d)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    o = oracle.OracleTable(w.fgrams, w.lengths, w.ids)
    exp_ids, exp_len = o.lookup(w.tokens, cfg.max_n)
    got_ids = np.fromfile(d / "ids_out.bin", dtype=np.int32).reshape(cfg.B, cfg.T)
    got_len = np.fromfile(d / "len_out.bin", dtype=np.int8).reshape(cfg.B, cfg.T)
    np.testing.assert_array_equal(got_ids, exp_ids)
    np.testing.assert_array_equal(got_len, exp_len)
    got = np.fromfile(d / "out.bin", dtype=np.uint8)
    assert got.tobytes() == oracle.gather(exp_ids, rows).tobytes()
