"""CPU oracle for precomputing the f-gram embedding layer (test infrastructure only).

Only the tests and the benchmark's CPU-baseline leg use this module; the
product path never does.  It shares no code with the GPU library.

What it computes.  Section 3.2: at inference the f-gram layer F is a cache of
the f-gram model's outputs, one row per f-gram; during training the same
model maps the token embeddings of an f-gram to one vector, the output at the
f-gram's final token (Algorithm 1, training branch).  So

    F(w) = A_fgram(T(w_0), ..., T(w_{n-1}))   for every f-gram w of length n.

The paper fixes only part of A_fgram: a transformer whose sizes are those of
its main-model tables, with absolute position embeddings whose number of
positions equals the longest f-gram, f-grams of a batch right-padded to the
longest one, bfloat16 parameters (implementation appendix).  The remaining
choices are readings:

* a GPT-2 style decoder block, pre-LayerNorm:
      h += Attn(LN1(h)) ;  h += W2 GELU(W1 LN2(h) + b1) + b2
  with causal multi-head self-attention (scores scaled by 1/sqrt(head_dim),
  biases on every linear map), exact (erf) GELU, LayerNorm epsilon 1e-5;
* position p (0 = the f-gram's oldest token) adds position row p;
* a final LayerNorm on the last token's hidden state gives the output.

Because attention is causal and padding is on the right, the final token never
sees pad positions, so padding an f-gram changes nothing: this oracle
processes each length on its own, unpadded.  Arithmetic is float64 on the
bf16 parameter values; the caller rounds the result if it wants bf16.
"""
from __future__ import annotations

from typing import Dict

import numpy as np
from scipy.special import erf

LN_EPS = 1e-5


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray) -> np.ndarray:
    """LayerNorm over the last axis: (x - mean) / sqrt(var + eps) * g + b,
    var the biased (population) variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS) * g + b


def gelu(x: np.ndarray) -> np.ndarray:
    """x * Phi(x), Phi the standard normal CDF."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q, k, v [G, H, n, dh] -> [G, H, n, dh]; position i attends to j <= i."""
    n, dh = q.shape[-2], q.shape[-1]
    s = q @ np.swapaxes(k, -1, -2) / np.sqrt(dh)
    future = np.triu(np.ones((n, n), dtype=bool), k=1)
    s = np.where(future, -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v


def forward_group(tokens: np.ndarray, tok_emb: np.ndarray, P: Dict[str, np.ndarray],
                  n_layers: int, n_heads: int) -> np.ndarray:
    """tokens [G, n] (all f-grams of one length n) -> outputs [G, d]."""
    G, n = tokens.shape
    d = tok_emb.shape[1]
    dh = d // n_heads
    h = tok_emb[tokens] + P["pos"][:n]                       # [G, n, d]
    for l in range(n_layers):
        p = f"l{l}."
        a = layer_norm(h, P[p + "ln1_g"], P[p + "ln1_b"])
        qkv = a @ P[p + "w_qkv"].T + P[p + "b_qkv"]         # [G, n, 3d]
        q, k, v = (qkv[..., i * d:(i + 1) * d].reshape(G, n, n_heads, dh).transpose(0, 2, 1, 3)
                   for i in range(3))
        o = causal_attention(q, k, v).transpose(0, 2, 1, 3).reshape(G, n, d)
        h = h + o @ P[p + "w_o"].T + P[p + "b_o"]
        a = layer_norm(h, P[p + "ln2_g"], P[p + "ln2_b"])
        f = gelu(a @ P[p + "w_fc1"].T + P[p + "b_fc1"])
        h = h + f @ P[p + "w_fc2"].T + P[p + "b_fc2"]
    return layer_norm(h[:, n - 1], P["lnf_g"], P["lnf_b"])


def forward(fgrams: np.ndarray, lengths: np.ndarray, tok_emb: np.ndarray,
            params: Dict[str, np.ndarray], n_layers: int, n_heads: int) -> np.ndarray:
    """F rows for every f-gram: fgrams [N, K] (oldest token first, padded),
    lengths [N]; tok_emb [V, d] and params as float64 arrays -> [N, d] float64."""
    fgrams = np.asarray(fgrams)
    lengths = np.asarray(lengths)
    out = np.zeros((len(lengths), tok_emb.shape[1]), dtype=np.float64)
    for n in np.unique(lengths):
        sel = np.nonzero(lengths == n)[0]
        out[sel] = forward_group(fgrams[sel, :n], tok_emb, params, n_layers, n_heads)
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value (ties to even) of float64 values, via float32."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)
