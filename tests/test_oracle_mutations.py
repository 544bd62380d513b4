"""Plant plausible mistakes in copies of the oracle (on the CPU) and check
that at least one pin catches each of them."""
import importlib.util
import os
import sys
import types

import pytest

from tests import oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "relation_oracle.py")

# (name, exact text in the oracle, replacement)
MUTATIONS = [
    ("silu_drops_U_factor", "E = U * expit(U)", "E = expit(U)"),
    ("self_temperature_inverted", "expit(U[np.arange(nb), rows] / tau_s)",
     "expit(U[np.arange(nb), rows] * tau_s)"),
    ("count_correction_sign", "(E - lam * np.log(ione)[:, None])[below]",
     "(E + lam * np.log(ione)[:, None])[below]"),
    ("count_index_zero_based_shift", "ione = (rows + 1).astype(np.float64)            # one-based count",
     "ione = (rows + 2).astype(np.float64)            # one-based"),
    ("U_transposed_operands", "U = s * (q[rows] @ k.T)", "U = s * (k[rows] @ q.T)"),
    ("missing_scale", "U = s * (q[rows] @ k.T)", "U = (q[rows] @ k.T)"),
    ("transport_uses_keys", "Y[b0:b1] = Ft @ v ", "Y[b0:b1] = Ft @ k "),
    ("exchange_only_keeps_self", "            Ft[np.arange(b1 - b0), rr] = 0.0\n",
     "            Ft[np.arange(b1 - b0), rr] = Ft[np.arange(b1 - b0), rr]\n"),
    ("exchange_only_grad_keeps_self_flow", "            H[np.arange(nb), rr] = 0.0\n", "            pass\n"),
    ("exchange_only_dv_keeps_self", "            Ft[np.arange(nb), rr] = 0.0\n", "            pass\n"),
    ("exchange_mass_includes_self", "        below = np.arange(T)[None, :] < rr[:, None]\n        g[b0:b1]",
     "        below = np.arange(T)[None, :] <= rr[:, None]\n        g[b0:b1]"),
    ("self_grad_drops_tau", "dU[diag] = dR[diag] * Sb * (1.0 - Sb) / tau_s",
     "dU[diag] = dR[diag] * Sb * (1.0 - Sb)"),
    ("dk_transposed", "dk += s * (dU.T @ q[rr])", "dk += s * (dU @ q[rr])"),
    ("silu_grad_drops_term", "return sg + U * sg * (1.0 - sg)", "return sg"),
    ("dlam_sign", "dlam += float(-(np.log(ione)", "dlam += float((np.log(ione)"),
    ("factorised_dS_sign", "dS = -g * (1.0 - g) * c ", "dS = g * (1.0 - g) * c "),
    ("factorised_dv_drops_self", "dv = (1.0 - g)[:, None] * G + (g[:, None] * pi).T @ G",
     "dv = (g[:, None] * pi).T @ G"),
]


def _load_mutant(old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor must occur once: {old!r}"
    text = text.replace(old, new)
    mod = types.ModuleType("relation_oracle_mutant")
    mod.__file__ = SRC
    exec(compile(text, SRC + " (mutant)", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(name, old, new):
    mod = _load_mutant(old, new)
    caught = []
    for check in pins.ALL_CHECKS:
        try:
            check(mod)
        except (AssertionError, ValueError, IndexError, FloatingPointError):
            caught.append(check.__name__)
    assert caught, f"planted mistake {name} passed every pin"
