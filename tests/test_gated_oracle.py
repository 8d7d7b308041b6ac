"""Gated SwiLA (Sec. 3.4, App. B.4) in the fp64 oracle: every pin holds, and
each plausible mistake planted in a copy of the oracle's gated code fails at
least one pin."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from gated_pins import GATED_PINS, TOL

SRC = os.path.join(os.path.dirname(oracle.__file__), "swila_oracle.c")


@pytest.mark.parametrize("name", sorted(GATED_PINS))
def test_gated_pin(name):
    err = GATED_PINS[name](oracle.forward)
    assert err < TOL, "%s: %.3e" % (name, err)


PRE = "if (a->decay && !a->post_decay)"
POST = "if (a->decay && a->post_decay) {   /* gated, post-decay */"
# name -> list of (text in the oracle, replacement)
MUTATIONS = {
    "decay_after_prediction": [(PRE, "if (0)"), (POST, "if (a->decay) {")],
    "decay_sign_flipped": [("for (int i = 0; i < Dk; ++i) w[i] *= 1.0 / (1.0 + exp(-dl[i]));\n                }\n\n",
                            "for (int i = 0; i < Dk; ++i) w[i] *= 1.0 / (1.0 + exp(dl[i]));\n                }\n\n")],
    "decay_of_component_0": [("const double *dl = a->decay + (row * J + j) * (size_t)Dk;\n                    for",
                              "const double *dl = a->decay + (row * J + 0) * (size_t)Dk;\n                    for")],
    "decay_on_update_too": [(POST, "if (a->decay) {")],
    "decay_by_key_index_reversed": [("w[i] *= 1.0 / (1.0 + exp(-dl[i]));\n                }\n\n",
                                     "w[i] *= 1.0 / (1.0 + exp(-dl[Dk - 1 - i]));\n                }\n\n")],
}


def _mutant(tmp_path, name):
    src = open(SRC).read()
    for old, new in MUTATIONS[name]:
        assert old in src, "mutation %s no longer matches the oracle source" % name
        src = src.replace(old, new, 1)
    c = tmp_path / ("%s.c" % name)
    so = tmp_path / ("%s.so" % name)
    c.write_text(src)
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-std=c11", "-pthread", "-o", str(so), str(c),
                    "-lm"], check=True)
    return oracle.load_library(str(so))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_gated_mutation_is_caught(tmp_path, name):
    lib = _mutant(tmp_path, name)

    def fwd(*args, **kw):
        return oracle.forward(*args, lib=lib, **kw)

    caught = []
    for pin, fn in GATED_PINS.items():
        try:
            err = fn(fwd)
        except (FloatingPointError, ValueError):
            err = np.inf
        if not err < TOL:
            caught.append(pin)
    assert caught, "mutation %s passed every gated pin" % name
