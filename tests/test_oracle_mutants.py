"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a text
substitution), builds it with the same flags into a temporary library, and
runs the pins of ``test_oracle_pins`` against it: at least one pin must
fail.  Mistakes are planted on the CPU only, in the oracle, never in the
GPU library.
"""

import itertools
import os

import numpy as np
import pytest

import oracle
import test_oracle_pins as pins

F32_BODY_START = "int oracle_step_f32("
F64_BODY_START = "int oracle_step_f64("

# (name, which function, old text, new text)
MUTANTS = [
    ("sum_right_fold", "f32",
     "float s = grads[0 * (size_t)num_keys + k][i];\n            for (int j = 1; j < num_workers; ++j)\n                s = s + grads[(size_t)j * num_keys + k][i];",
     "float s = grads[(size_t)(num_workers - 1) * num_keys + k][i];\n            for (int j = num_workers - 2; j >= 0; --j)\n                s = s + grads[(size_t)j * num_keys + k][i];"),
    ("sum_is_mean", "f32",
     "float d = fmaf(wd, w[i], s);", "float d = fmaf(wd, w[i], s / (float)num_workers);"),
    ("worker_key_index_swapped", "f32",
     "s = s + grads[(size_t)j * num_keys + k][i];", "s = s + grads[(size_t)k * num_workers + j][i];"),
    ("weight_decay_dropped", "f32", "float d = fmaf(wd, w[i], s);", "float d = s;"),
    ("weight_decay_unfused", "f32", "float d = fmaf(wd, w[i], s);", "float d = wd * w[i]; d = d + s;"),
    ("weight_decay_sign", "f32", "float d = fmaf(wd, w[i], s);", "float d = fmaf(-wd, w[i], s);"),
    ("momentum_unfused", "f32", "float m1 = fmaf(mu, m[i], d);", "float m1 = mu * m[i]; m1 = m1 + d;"),
    ("momentum_dampened", "f32", "float m1 = fmaf(mu, m[i], d);", "float m1 = fmaf(mu, m[i], (1.0f - mu) * d);"),
    ("nesterov_uses_old_momentum", "f32", "float u = nesterov ? fmaf(mu, m1, d) : m1;",
     "float u = nesterov ? fmaf(mu, m[i], d) : m1;"),
    ("nesterov_unfused", "f32", "float u = nesterov ? fmaf(mu, m1, d) : m1;",
     "float u = m1; if (nesterov) { u = mu * m1; u = u + d; }"),
    ("nesterov_flag_ignored", "f32", "float u = nesterov ? fmaf(mu, m1, d) : m1;", "float u = fmaf(mu, m1, d);"),
    ("update_sign", "f32", "w[i] = fmaf(-lr, u, w[i]);", "w[i] = fmaf(lr, u, w[i]);"),
    ("update_unfused", "f32", "w[i] = fmaf(-lr, u, w[i]);", "{ float t = lr * u; w[i] = w[i] - t; }"),
    ("momentum_not_stored", "f32", "m[i] = m1;", "m[i] = d;"),
    ("update_with_gradient_not_momentum", "f32", "float u = nesterov ? fmaf(mu, m1, d) : m1;",
     "float u = nesterov ? fmaf(mu, m1, d) : d;"),
    ("f64_weight_decay_dropped", "f64", "double d = fma(wd, w[i], s);", "double d = s;"),
    ("f64_nesterov_uses_old_momentum", "f64", "double u = nesterov ? fma(mu, m1, d) : m1;",
     "double u = nesterov ? fma(mu, m[i], d) : m1;"),
    ("f64_momentum_sign", "f64", "double m1 = fma(mu, m[i], d);", "double m1 = fma(-mu, m[i], d);"),
]


def _plant(src, which, old, new):
    start = src.index(F32_BODY_START if which == "f32" else F64_BODY_START)
    end = src.index(F64_BODY_START) if which == "f32" else len(src)
    body = src[start:end]
    assert body.count(old) == 1, f"mutation anchor not unique: {old!r}"
    return src[:start] + body.replace(old, new) + src[end:]


def _pin_calls():
    """Every pin as a callable of the oracle object, with its parameters."""
    calls = []
    for mode in ("nesterov", "plain"):
        calls.append((f"worked_example[{mode}]", lambda o, mode=mode: pins.test_worked_example(o, mode)))
    for case in pins.ROUNDING_CASES:
        calls.append((f"rounding[{case[0]}]", lambda o, case=case: pins.test_rounding_points(o, case)))
    for n in (1, 2, 3, 8, 16):
        calls.append((f"identical[{n}]", lambda o, n=n: pins.test_identical_gradients_sum_exactly(o, n)))
    for nest in (True, False):
        calls.append((f"zero_grad[{nest}]", lambda o, nest=nest: pins.test_zero_gradient_closed_form(o, nest)))
        calls.append((f"torch_sgd[{nest}]", lambda o, nest=nest: pins.test_against_torch_sgd(o, nest)))
        calls.append((f"lr0[{nest}]", lambda o, nest=nest: pins.test_zero_lr_leaves_weights_and_updates_momentum(o, nest)))
    calls.append(("zero_grad_by_hand", pins.test_zero_gradient_single_step_by_hand))
    calls.append(("indexing", pins.test_key_and_worker_indexing))
    calls.append(("dyadic_plain_sgd", pins.test_plain_sgd_on_dyadic_values_is_exact))
    calls.append(("mu0_flag", pins.test_zero_momentum_makes_nesterov_flag_irrelevant))
    for n, nest in itertools.product((1, 3, 16), (True, False)):
        calls.append((f"exact_rational[{n},{nest}]",
                      lambda o, n=n, nest=nest: pins.test_exact_rational_bruteforce(o, n, nest)))
    return calls


def test_unmutated_copy_passes_every_pin(tmp_path):
    lib = oracle.build(force=True, src=oracle.SRC, out=str(tmp_path / "libref.so"))
    o = oracle.OracleLib(lib)
    for name, call in _pin_calls():
        call(o)


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, mutant):
    name, which, old, new = mutant
    with open(oracle.SRC) as f:
        src = f.read()
    mutated = _plant(src, which, old, new)
    cpath = tmp_path / f"{name}.c"
    cpath.write_text(mutated)
    lib = oracle.build(force=True, src=str(cpath), out=str(tmp_path / f"lib{name}.so"))
    o = oracle.OracleLib(lib)
    caught = []
    for pin_name, call in _pin_calls():
        try:
            call(o)
        except AssertionError:
            caught.append(pin_name)
    assert caught, f"no pin caught the planted mistake {name}"
