"""Each plausible mistake planted in a copy of the C oracle (on the CPU) must
fail at least one pin; otherwise the pins would not pin the oracle."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from oracle_pins import ALL_PINS, TOL

SRC = os.path.join(os.path.dirname(oracle.__file__), "swila_oracle.c")
STATE_IDX = "((((size_t)b * H + h) * J + j) * Dk + i) * Dv + d"

# name -> (text in the oracle, replacement, replace every occurrence?)
MUTATIONS = {
    "half_dropped_in_estep": ("exp(-0.5 * delta[j] * delta[j] - shift)",
                              "exp(-1.0 * delta[j] * delta[j] - shift)", False),
    "estep_shift_ignored": ("num[j] = prior[j] * exp(-0.5 * delta[j] * delta[j] - shift);",
                            "num[j] = prior[j] * exp(-0.5 * delta[j] * delta[j] - shift * j);",
                            False),
    "delta_sign_flipped": ("delta[j] = vt[d] - pred;", "delta[j] = pred - vt[d];", False),
    "prediction_with_query": ("pred += w[i] * kt[i];", "pred += w[i] * qt[i];", False),
    "prior_dropped": ("num[j] = prior[j] * exp(", "num[j] = 1.0 * exp(", False),
    "responsibility_unnormalised": ("double r = num[j] / Z;", "double r = num[j];", False),
    "beta_dropped": ("w[i] += beta * r * delta[j] * kt[i];", "w[i] += r * delta[j] * kt[i];", False),
    "update_along_query": ("w[i] += beta * r * delta[j] * kt[i];",
                           "w[i] += beta * r * delta[j] * qt[i];", False),
    "sigmoid_sign_flipped": ("1.0 / (1.0 + exp(-lbt[", "1.0 / (1.0 + exp(lbt[", False),
    "retrieval_with_key": ("y += w[i] * qt[i];", "y += w[i] * kt[i];", False),
    "query_prior_from_key_logits": ("lqt[", "lkt[", True),
    "query_prior_unnormalised": ("double pq = exp(lqt[(size_t)j * Dv + d] - m) / z;",
                                 "double pq = exp(lqt[(size_t)j * Dv + d] - m);", False),
    "initial_state_transposed": (STATE_IDX, "((((size_t)b * H + h) * J + j) * Dv + d) * Dk + i", False),
}


def _mutant(tmp_path, name):
    old, new, every = MUTATIONS[name]
    src = open(SRC).read()
    assert old in src, "mutation %s no longer matches the oracle source" % name
    src = src.replace(old, new) if every else src.replace(old, new, 1)
    c = tmp_path / ("%s.c" % name)
    so = tmp_path / ("%s.so" % name)
    c.write_text(src)
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-std=c11", "-pthread", "-o", str(so), str(c),
                    "-lm"], check=True)
    return oracle.load_library(str(so))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(tmp_path, name):
    lib = _mutant(tmp_path, name)

    def fwd(*args, **kw):
        return oracle.forward(*args, lib=lib, **kw)

    caught = []
    for pin, fn in ALL_PINS.items():
        try:
            err = fn(fwd)
        except (FloatingPointError, ValueError, np.linalg.LinAlgError):
            err = np.inf
        if not err < TOL:
            caught.append(pin)
    assert caught, "mutation %s passed every pin" % name
