"""Pins for the f-gram model oracle (precomputing F, Section 3.2).

The oracle is pinned to code it does not share:

* torch's own pre-LayerNorm encoder layer (nn.TransformerEncoderLayer with
  norm_first, GELU, a causal mask) plus nn.LayerNorm, run in float64 on a
  right-padded batch, the way the paper batches f-grams (implementation
  appendix): the last real token's output must equal the oracle's, for any
  pad content;
* closed forms: with no layers the output is LN_f(T(last) + P(n-1)); with
  zero query and key weights attention is the plain mean of the values over
  the prefix, and with zero first MLP weights the MLP adds only its output
  bias.

Each check takes the oracle module as an argument so that the mutant tests
can run it against a copy with one planted mistake.
"""
import numpy as np
import torch

from oracle import fgram_model as orc_module
from workloads.fgram_model import (ModelConfig, make_params, make_token_rows,
                                   bf16_bits_to_f64)


def _f64(bits):
    return {k: bf16_bits_to_f64(v) for k, v in bits.items()}


def _fgrams(rng, V, N, K, lo=2):
    lengths = rng.integers(lo, K + 1, size=N).astype(np.int32)
    fg = rng.integers(0, V, size=(N, K)).astype(np.int32)
    for i, n in enumerate(lengths):
        fg[i, n:] = -1
    return fg, lengths


def torch_reference(fg, lengths, T, P, cfg, pad_token=0):
    """nn.TransformerEncoderLayer stack over the right-padded batch."""
    N, K = fg.shape
    d = cfg.d
    layers = []
    for l in range(cfg.n_layers):
        p = f"l{l}."
        m = torch.nn.TransformerEncoderLayer(d, cfg.n_heads, cfg.d_ff, dropout=0.0,
                                             activation="gelu", batch_first=True,
                                             norm_first=True, layer_norm_eps=1e-5,
                                             dtype=torch.float64)
        with torch.no_grad():
            m.self_attn.in_proj_weight.copy_(torch.from_numpy(P[p + "w_qkv"]))
            m.self_attn.in_proj_bias.copy_(torch.from_numpy(P[p + "b_qkv"]))
            m.self_attn.out_proj.weight.copy_(torch.from_numpy(P[p + "w_o"]))
            m.self_attn.out_proj.bias.copy_(torch.from_numpy(P[p + "b_o"]))
            m.linear1.weight.copy_(torch.from_numpy(P[p + "w_fc1"]))
            m.linear1.bias.copy_(torch.from_numpy(P[p + "b_fc1"]))
            m.linear2.weight.copy_(torch.from_numpy(P[p + "w_fc2"]))
            m.linear2.bias.copy_(torch.from_numpy(P[p + "b_fc2"]))
            m.norm1.weight.copy_(torch.from_numpy(P[p + "ln1_g"]))
            m.norm1.bias.copy_(torch.from_numpy(P[p + "ln1_b"]))
            m.norm2.weight.copy_(torch.from_numpy(P[p + "ln2_g"]))
            m.norm2.bias.copy_(torch.from_numpy(P[p + "ln2_b"]))
        m.train()  # dropout is 0; keeps the plain (non-fused) code path
        layers.append(m)
    lnf = torch.nn.LayerNorm(d, eps=1e-5, dtype=torch.float64)
    with torch.no_grad():
        lnf.weight.copy_(torch.from_numpy(P["lnf_g"]))
        lnf.bias.copy_(torch.from_numpy(P["lnf_b"]))
    tok = np.where(fg >= 0, fg, pad_token)
    x = torch.from_numpy(T[tok] + P["pos"][:K])
    mask = torch.nn.Transformer.generate_square_subsequent_mask(K, dtype=torch.float64)
    with torch.no_grad():
        for m in layers:
            x = m(x, src_mask=mask, is_causal=True)
        last = x[torch.arange(N), torch.from_numpy(lengths.astype(np.int64) - 1)]
        return lnf(last).numpy()


def _case(seed, cfg, V=50, N=40):
    rng = np.random.default_rng(seed)
    P = _f64(make_params(cfg, seed))
    T = bf16_bits_to_f64(make_token_rows(V, cfg.d, seed + 1))
    fg, lengths = _fgrams(rng, V, N, cfg.max_len)
    return fg, lengths, T, P


def check_matches_torch_encoder(orc):
    for seed, cfg in [(1, ModelConfig(d=32, n_heads=4, d_ff=64, n_layers=2, max_len=5)),
                      (2, ModelConfig(d=64, n_heads=2, d_ff=96, n_layers=3, max_len=7)),
                      (3, ModelConfig(d=16, n_heads=1, d_ff=48, n_layers=1, max_len=3))]:
        fg, lengths, T, P = _case(seed, cfg)
        got = orc.forward(fg, lengths, T, P, cfg.n_layers, cfg.n_heads)
        for pad in (0, 7):
            ref = torch_reference(fg, lengths, T, P, cfg, pad_token=pad)
            np.testing.assert_allclose(got, ref, rtol=1e-9, atol=1e-9)


def check_no_layers_closed_form(orc):
    cfg = ModelConfig(d=24, n_heads=3, d_ff=32, n_layers=0, max_len=6)
    fg, lengths, T, P = _case(4, cfg)
    got = orc.forward(fg, lengths, T, P, 0, cfg.n_heads)
    for i, n in enumerate(lengths):
        x = torch.from_numpy(T[fg[i, n - 1]] + P["pos"][n - 1])
        ref = torch.nn.functional.layer_norm(x, (cfg.d,), torch.from_numpy(P["lnf_g"]),
                                             torch.from_numpy(P["lnf_b"]), eps=1e-5)
        np.testing.assert_allclose(got[i], ref.numpy(), rtol=1e-12, atol=1e-12)


def check_uniform_attention_closed_form(orc):
    """Zero query/key weights and biases: every score is 0, so the softmax over
    j <= i is uniform; zero first MLP layer: GELU(0) = 0."""
    cfg = ModelConfig(d=32, n_heads=4, d_ff=64, n_layers=1, max_len=5)
    fg, lengths, T, P = _case(5, cfg)
    d = cfg.d
    P["l0.w_qkv"][:2 * d] = 0.0
    P["l0.b_qkv"][:2 * d] = 0.0
    P["l0.w_fc1"][:] = 0.0
    P["l0.b_fc1"][:] = 0.0
    got = orc.forward(fg, lengths, T, P, 1, cfg.n_heads)
    ln = torch.nn.functional.layer_norm
    t = {k: torch.from_numpy(v) for k, v in P.items()}
    for i, n in enumerate(lengths):
        h0 = torch.from_numpy(T[fg[i, :n]] + P["pos"][:n])
        a = ln(h0, (d,), t["l0.ln1_g"], t["l0.ln1_b"], eps=1e-5)
        v = a @ t["l0.w_qkv"][2 * d:].T + t["l0.b_qkv"][2 * d:]
        o = v.mean(dim=0)          # the last position sees all n tokens
        h = h0[n - 1] + o @ t["l0.w_o"].T + t["l0.b_o"] + t["l0.b_fc2"]
        ref = ln(h, (d,), t["lnf_g"], t["lnf_b"], eps=1e-5)
        np.testing.assert_allclose(got[i], ref.numpy(), rtol=1e-12, atol=1e-12)


def check_order_and_grouping_invariance(orc):
    cfg = ModelConfig(d=32, n_heads=2, d_ff=64, n_layers=2, max_len=4)
    fg, lengths, T, P = _case(6, cfg, N=30)
    got = orc.forward(fg, lengths, T, P, cfg.n_layers, cfg.n_heads)
    perm = np.random.default_rng(0).permutation(len(lengths))
    got_p = orc.forward(fg[perm], lengths[perm], T, P, cfg.n_layers, cfg.n_heads)
    np.testing.assert_allclose(got_p, got[perm], rtol=1e-12, atol=1e-12)
    one = np.stack([orc.forward(fg[i:i + 1], lengths[i:i + 1], T, P, cfg.n_layers,
                                cfg.n_heads)[0] for i in range(len(lengths))])
    np.testing.assert_allclose(one, got, rtol=1e-12, atol=1e-12)


def test_matches_torch_encoder():
    check_matches_torch_encoder(orc_module)


def test_no_layers_closed_form():
    check_no_layers_closed_form(orc_module)


def test_uniform_attention_closed_form():
    check_uniform_attention_closed_form(orc_module)


def test_order_and_grouping_invariance():
    check_order_and_grouping_invariance(orc_module)


def test_round_bf16_known_values():
    r = orc_module.round_bf16
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: ties go to the even mantissa (1.0)
    assert r(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert r(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    assert r(np.array([-2.5]))[0] == -2.5
    assert r(np.array([1.0 + 2.0 ** -8 + 2.0 ** -20]))[0] == 1.0 + 2.0 ** -7
