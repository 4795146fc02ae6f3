"""The oracle's pins catch plausible mistakes.

Each case copies the oracle source, plants one mistake (a dropped length, a
shifted window, a wrong probe order, a transposed operand ...), compiles it on
the CPU and runs the pin tests against the mutant: at least one must fail.
"""
import ctypes
import os
import subprocess

import pytest

import oracle
import test_oracle_pins as pins

SRC = open(os.path.join(os.path.dirname(oracle.__file__), "scone_oracle.cpp")).read()

MUTANTS = {
    "no_bigrams": ("for (int64_t n = top; n >= 2; --n)", "for (int64_t n = top; n >= 3; --n)"),
    "window_shift": ("key_of(row + (t - n + 1), (int32_t)n)", "key_of(row + (t - n), (int32_t)n)"),
    "shortest_first": ("for (int64_t n = top; n >= 2; --n)", "for (int64_t n = 2; n <= top; ++n)"),
    "no_early_exit": ("id = it->second; len = (int32_t)n; break;", "id = it->second; len = (int32_t)n;"),
    "crosses_rows": ("int64_t top = max_n < t + 1 ? (int64_t)max_n : t + 1;",
                     "int64_t top = max_n < b * T + t + 1 ? (int64_t)max_n : b * T + t + 1;"),
    "window_too_short": ("int64_t top = max_n < t + 1 ? (int64_t)max_n : t + 1;",
                         "int64_t top = max_n - 1 < t + 1 ? (int64_t)max_n - 1 : t + 1;"),
    "len_off_by_one": ("len = (int32_t)n; break;", "len = (int32_t)n - 1; break;"),
    "gather_transposed": ("table + r * row_bytes", "table + k * row_bytes"),
    "gather_bound": ("r >= n_rows", "r > n_rows"),
    "no_dup_check": ("if (!ins.second) { delete s; return OR_DUPLICATE; }", ""),
    "accepts_unigrams": ("if (len < 2 || len > stride)", "if (len < 1 || len > stride)"),
}

PINS = [
    pins.test_worked_example_alg1,
    pins.test_all_bigrams_and_trigrams_closed_form,
    pins.test_build_rejects_invalid_sets,
    pins.test_gather_equals_fancy_indexing_bytes,
    pins.test_gather_rejects_bad_rows,
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path, monkeypatch):
    old, new = MUTANTS[name]
    assert SRC.count(old) >= 1, name
    src = tmp_path / "mutant.cpp"
    src.write_text(SRC.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-shared", "-fPIC", "-o", str(so), str(src)])
    monkeypatch.setattr(oracle, "_lib", oracle.bind(ctypes.CDLL(str(so))))
    failed = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, oracle.OracleError, pytest.fail.Exception):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
