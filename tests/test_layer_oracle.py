"""Pins of the layer oracle (CPU only), and planted mistakes that the pins must
catch. See layer_pins.py for what each pin fixes."""
import os
import types

import pytest

from oracle import layer_oracle
from tests import layer_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "layer_oracle.py")


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(check):
    check(layer_oracle)


# (name, exact text in the layer oracle, replacement)
MUTATIONS = [
    ("rope_frequency_exponent", "base ** (-2.0 * np.arange(half) / D)", "base ** (-1.0 * np.arange(half) / D)"),
    ("rope_sin_sign", "[x1 * c - x2 * s, x1 * s + x2 * c]", "[x1 * c + x2 * s, x1 * s + x2 * c]"),
    ("rope_positions_one_based", "np.arange(T, dtype=np.float64)[:, None]",
     "np.arange(1, T + 1, dtype=np.float64)[:, None]"),
    ("rope_interleaved_pairs", "x1, x2 = x[..., : D // 2], x[..., D // 2:]\n    return np.concatenate(",
     "x1, x2 = x[..., 0::2], x[..., 1::2]\n    return np.concatenate("),
    ("rope_transpose_is_forward", "[g1 * c + g2 * s, -g1 * s + g2 * c]", "[g1 * c - g2 * s, g1 * s + g2 * c]"),
    ("givens_sign", "out[:, a] = c * I[:, a] - s * I[:, b]", "out[:, a] = c * I[:, a] + s * I[:, b]"),
    ("pairing_B_no_wrap", "(2 * p + 1, (2 * p + 2) % H)", "(2 * p + 1, min(2 * p + 2, H - 1))"),
    ("givens_dI_not_transposed", "dI[:, a] = c * dIt[:, a] + s * dIt[:, b]",
     "dI[:, a] = c * dIt[:, a] - s * dIt[:, b]"),
    ("dtheta_sign", "np.sum(dIt[:, a] * (-s * I[:, a] - c * I[:, b]))",
     "np.sum(dIt[:, a] * (s * I[:, a] - c * I[:, b]))"),
    ("layer_bwd_skips_rope_on_dq", 'dq = rope_transpose(r["dq"], rope_base) if rope_base else r["dq"]',
     'dq = r["dq"]'),
]


def _load_mutant(old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor must occur once: {old!r}"
    mod = types.ModuleType("layer_oracle_mutant")
    mod.__file__ = SRC
    mod.__package__ = "oracle"  # its relative import reaches the real operator oracle
    exec(compile(text.replace(old, new), SRC + " (mutant)", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(name, old, new):
    mod = _load_mutant(old, new)
    caught = []
    for check in pins.ALL_CHECKS:
        try:
            check(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(check.__name__)
    assert caught, f"planted mistake {name} passed every pin"
