"""Seeded random parameters for an f-gram transformer (A_fgram of Section 3.2).

No trained weights exist here, so the parameters are random.  This module only
draws them; it holds none of the forward arithmetic, so the GPU library and the
CPU oracle are both fed from it without sharing code.

The parameter set follows the model readings used throughout: absolute
position embeddings with one row per position up to the longest f-gram
(implementation appendix), then a stack of pre-LayerNorm decoder blocks, then a
final LayerNorm.  Linear weights are stored [out_features, in_features] and
applied as y = x W^T + b.  Every value is bf16-representable (the paper trains
in bfloat16) and is handed out as raw bf16 bit patterns (uint16).

Two scale recipes:

* "unit" (tests): weights N(0, 1/fan_in), biases and LayerNorm offsets
  N(0, 0.1^2), LayerNorm gains 1 + N(0, 0.1^2), positions N(0, 1), so that
  every term of the forward moves the output by a visible amount;
* "gpt2" (benchmark): the customary GPT-2 initialisation, weights and
  positions N(0, 0.02^2), zero biases, unit gains.  Only the timing matters
  there; the values do not change the work done.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List

import numpy as np


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    d: int          # d_model
    n_heads: int
    d_ff: int       # feed-forward width
    n_layers: int
    max_len: int    # longest f-gram, = number of position rows

    @property
    def head_dim(self) -> int:
        return self.d // self.n_heads


# The WebText 128M main-model shape (d_model 1024, ffw 4096, 6 layers; the
# appendix's WebText model table) used as a 1x f-gram model, 64-wide heads.
GPT2_128M = ModelConfig(d=1024, n_heads=16, d_ff=4096, n_layers=6, max_len=3)


def layer_param_names(layer: int) -> List[str]:
    p = f"l{layer}."
    return [p + s for s in ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                            "ln2_g", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2")]


def param_names(cfg: ModelConfig) -> List[str]:
    """All parameter names in the library's packing order."""
    names = ["pos"]
    for l in range(cfg.n_layers):
        names += layer_param_names(l)
    return names + ["lnf_g", "lnf_b"]


def param_shape(cfg: ModelConfig, name: str):
    d, f = cfg.d, cfg.d_ff
    base = name.split(".")[-1]
    return {"pos": (cfg.max_len, d), "ln1_g": (d,), "ln1_b": (d,), "w_qkv": (3 * d, d),
            "b_qkv": (3 * d,), "w_o": (d, d), "b_o": (d,), "ln2_g": (d,), "ln2_b": (d,),
            "w_fc1": (f, d), "b_fc1": (f,), "w_fc2": (d, f), "b_fc2": (d,),
            "lnf_g": (d,), "lnf_b": (d,)}[base]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32) \
        .astype(np.float64)


def make_params(cfg: ModelConfig, seed: int, recipe: str = "unit") -> Dict[str, np.ndarray]:
    """name -> uint16 bf16 bits of the given shape."""
    if cfg.d % cfg.n_heads:
        raise ValueError("d must be a multiple of n_heads")
    rng = np.random.Generator(np.random.PCG64(seed))
    out = {}
    for name in param_names(cfg):
        shape = param_shape(cfg, name)
        base = name.split(".")[-1]
        if recipe == "unit":
            if base.startswith("w_"):
                v = rng.standard_normal(shape, dtype=np.float32) / np.float32(np.sqrt(shape[1]))
            elif base == "pos":
                v = rng.standard_normal(shape, dtype=np.float32)
            elif base.endswith("_g"):
                v = 1.0 + 0.1 * rng.standard_normal(shape, dtype=np.float32)
            else:
                v = 0.1 * rng.standard_normal(shape, dtype=np.float32)
        elif recipe == "gpt2":
            if base.startswith("w_") or base == "pos":
                v = 0.02 * rng.standard_normal(shape, dtype=np.float32)
            elif base.endswith("_g"):
                v = np.ones(shape, dtype=np.float32)
            else:
                v = np.zeros(shape, dtype=np.float32)
        else:
            raise ValueError(recipe)
        out[name] = f32_to_bf16_bits(v.astype(np.float32))
    return out


def make_token_rows(vocab: int, d: int, seed: int, std: float = 1.0) -> np.ndarray:
    """[vocab, d] token embedding rows T as uint16 bf16 bits."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return f32_to_bf16_bits((std * rng.standard_normal((vocab, d), dtype=np.float32))
                            .astype(np.float32))
