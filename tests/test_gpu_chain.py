"""The offline steps and the inference path chained on the GPU, each stage
checked against its oracle: f-gram discovery on a corpus (Algorithm 3 with
Section 3.1's minimum count), ids V, V+1, ... in discovery order, F
precomputed by the f-gram model into the f-gram rows of the unified table
(Section 3.2), the dictionary built from the discovered set, then lookup +
gather and the fused kernel over the same corpus (Algorithm 1)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_01637_amd as S
from oracle import discovery, fgram_model as orc
from gpu_util import as_bytes, dev
from test_gpu_discovery import check_top_s
from test_gpu_fgram_model import assert_close, bf16_dev
from workloads import zipf_cdf, zipf_tokens
from workloads.fgram_model import ModelConfig, make_params, make_token_rows, bf16_bits_to_f64

pytestmark = pytest.mark.gpu


def test_discover_precompute_embed_chain():
    rng = np.random.default_rng(77)
    V, K, Sn, min_count = 400, 4, 2500, 2
    X = zipf_tokens(rng, zipf_cdf(V), (8, 1500)).astype(np.int32)
    Xd = dev(X)

    # 1. discovery
    fg_d, ln_d, ct_d = S.discover_fgrams(Xd, K, Sn, min_count)
    got = check_top_s(fg_d, ln_d, ct_d, discovery.candidates(X, K, min_count), Sn)
    n = len(got)
    assert n == Sn
    fg = fg_d.cpu().numpy()
    ln = ln_d.cpu().numpy()
    ids = (V + np.arange(n)).astype(np.int32)

    # 2. precompute F into rows V .. V+n-1 of the unified table
    cfg = ModelConfig(512, 8, 1024, 2, K)
    P = make_params(cfg, seed=78)
    T_bits = make_token_rows(V, cfg.d, seed=79)
    rows = torch.zeros((V + n, cfg.d), dtype=torch.bfloat16, device="cuda")
    rows[:V].copy_(bf16_dev(T_bits))
    model = S.FgramModel(P, cfg.d, cfg.n_heads, cfg.d_ff, cfg.n_layers, cfg.max_len)
    S.precompute_fgram_rows(model, fg_d, ln_d, dev(ids), rows[:V], rows)
    ref = orc.forward(fg, ln, bf16_bits_to_f64(T_bits),
                      {k: bf16_bits_to_f64(v) for k, v in P.items()}, cfg.n_layers, cfg.n_heads)
    assert_close(rows[V:].float().cpu().numpy().astype(np.float64), ref, cfg.n_layers, "F")

    # 3. dictionary from the discovered set; lookup + gather and the fused kernel
    tb = S.build_fgram_table(fg_d, ln_d, dev(ids))
    o = oracle.OracleTable(fg, ln, ids)
    for max_n in (2, K):
        exp_ids, exp_len = o.lookup(X, max_n)
        fid, ml = S.lookup(tb, Xd, max_n, want_len=True)
        out = S.gather(fid, rows)
        fused = S.embed(tb, Xd, max_n, rows)
        S.check_ok()
        np.testing.assert_array_equal(fid.cpu().numpy(), exp_ids)
        np.testing.assert_array_equal(ml.cpu().numpy(), exp_len)
        table = rows.view(torch.uint8).cpu().numpy()
        exp = oracle.gather(exp_ids, table)
        assert as_bytes(out).tobytes() == exp.tobytes()
        assert as_bytes(fused).tobytes() == exp.tobytes()
        # a frequent corpus: most positions past the first few match an f-gram
        assert (exp_len[:, K:] > 1).mean() > 0.5
