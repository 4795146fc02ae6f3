"""The f-gram model oracle's pins catch plausible mistakes.

Each case copies the oracle's source, plants one mistake (attention that sees
the future, a wrong score scale, the tanh GELU, positions counted from the
newest token, the first token's output instead of the last, a dropped bias or
LayerNorm ...), loads it as a module and runs the pins against it: at least
one must fail.
"""
import importlib.util
import os
import sys

import pytest

import oracle.fgram_model as orc
import test_fgram_model_oracle as pins

SRC = open(orc.__file__).read()

MUTANTS = {
    "bidirectional": ("s = np.where(future, -np.inf, s)", "pass"),
    "score_scale_dh": ("/ np.sqrt(dh)", "/ dh"),
    "tanh_gelu": ("0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))",
                  "0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))"),
    "positions_reversed": ('P["pos"][:n]', 'P["pos"][:n][::-1]'),
    "first_token_output": ("h[:, n - 1]", "h[:, 0]"),
    "no_final_ln": ('return layer_norm(h[:, n - 1], P["lnf_g"], P["lnf_b"])',
                    "return h[:, n - 1]"),
    "no_out_bias": ('o @ P[p + "w_o"].T + P[p + "b_o"]', 'o @ P[p + "w_o"].T'),
    "post_ln": ('h = h + f @ P[p + "w_fc2"].T + P[p + "b_fc2"]',
                'h = layer_norm(h + f @ P[p + "w_fc2"].T + P[p + "b_fc2"], P[p + "ln2_g"], '
                'P[p + "ln2_b"])'),
    "unbiased_variance": ("var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)",
                          "var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)"),
    "qk_swapped": ("for i in range(3))", "for i in (1, 0, 2))"),
    "w_not_transposed": ('a @ P[p + "w_fc1"].T', 'a @ P[p + "w_fc1"].T[::-1]'),
    "no_mlp_residual": ('h = h + f @ P[p + "w_fc2"].T', 'h = f @ P[p + "w_fc2"].T'),
}

PINS = [pins.check_matches_torch_encoder, pins.check_no_layers_closed_form,
        pins.check_uniform_attention_closed_form, pins.check_order_and_grouping_invariance]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    assert SRC.count(old) >= 1, name
    path = tmp_path / f"mutant_{name}.py"
    path.write_text(SRC.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    failed = []
    for pin in PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
