"""Temporal SwiLA (Sec. 3.3, App. B.3) in the fp64 oracle: every pin holds, and
each plausible mistake planted in a copy of the oracle's temporal code fails at
least one pin."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from temporal_pins import TEMPORAL_PINS, TOL

SRC = os.path.join(os.path.dirname(oracle.__file__), "swila_oracle.c")


@pytest.mark.parametrize("name", sorted(TEMPORAL_PINS))
def test_temporal_pin(name):
    err = TEMPORAL_PINS[name](oracle.forward)
    assert err < TOL, "%s: %.3e" % (name, err)


# name -> (text in the oracle, replacement, replace every occurrence?)
MUTATIONS = {
    "key_prior_carried_not_posterior": ("if (temporal) rprev[(size_t)j * Dv + d] = r;",
                                        "if (temporal) rprev[(size_t)j * Dv + d] = prior[j];",
                                        False),
    "key_gate_swapped": ("prior[j] = (1.0 - g) * rprev[(size_t)j * Dv + d] + g * prior[j];",
                         "prior[j] = g * rprev[(size_t)j * Dv + d] + (1.0 - g) * prior[j];", False),
    "key_gate_from_query_logit": ("exp(-a->gk[row * Dv + d])", "exp(-a->gq[row * Dv + d])", False),
    "query_gate_swapped": ("*rq = (1.0 - gq) * *rq + gq * pq;",
                           "*rq = gq * *rq + (1.0 - gq) * pq;", False),
    "query_prior_not_used": ("pq = *rq;", "(void)pq;", False),
    "uniform_start_zero": (": 1.0 / J;", ": 0.0;", True),
    "prior_parts_swapped": ("a->prior_out[p] = rprev[(size_t)j * Dv + d];",
                            "a->prior_out[p] = rho[(size_t)j * Dv + d];", False),
    "query_prior_not_carried": ("double *rq = rho + (size_t)j * Dv + d;",
                                "double tmp_rq = 1.0 / J; double *rq = &tmp_rq;", False),
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
def test_temporal_mutation_is_caught(tmp_path, name):
    lib = _mutant(tmp_path, name)

    def fwd(*args, **kw):
        return oracle.forward(*args, lib=lib, **kw)

    caught = []
    for pin, fn in TEMPORAL_PINS.items():
        try:
            err = fn(fwd)
        except (FloatingPointError, ValueError):
            err = np.inf
        if not err < TOL:
            caught.append(pin)
    assert caught, "mutation %s passed every temporal pin" % name
