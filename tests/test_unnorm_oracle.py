"""The unnormalised-responsibility variant (App. D.2) in the fp64 oracles: every
pin holds; each plausible mistake planted in a copy of the C oracle's variant
code fails at least one pin; and the App. D iteration of the variant, whose
Jacobian is exact, reaches its sequential trajectory (App. D.1)."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads
from oracle import newton
from unnorm_pins import TOL, UNNORM_PINS

SRC = os.path.join(os.path.dirname(oracle.__file__), "swila_oracle.c")
NAMES = workloads.NAMES


@pytest.mark.parametrize("name", sorted(UNNORM_PINS))
def test_unnorm_pin(name):
    err = UNNORM_PINS[name](oracle.forward)
    assert err < TOL, "%s: %.3e" % (name, err)


VARIANT = "if (a->unnormalized) r = prior[j] * exp(-0.5 * delta[j] * delta[j]);"

# name -> (text in the oracle, replacement, replace every occurrence?)
MUTATIONS = {
    "prior_dropped": (VARIANT, "if (a->unnormalized) r = exp(-0.5 * delta[j] * delta[j]);", False),
    "half_dropped": (VARIANT, "if (a->unnormalized) r = prior[j] * exp(-delta[j] * delta[j]);",
                     False),
    "still_normalised": (VARIANT, "if (a->unnormalized) r = num[j] / Z;", False),
    "shifted_numerator": (VARIANT, "if (a->unnormalized) r = num[j];", False),
    "prior_logits_unnormalised": (VARIANT,
                                  "if (a->unnormalized) r = prior[j] * z * exp(-0.5 * delta[j] * delta[j]);",
                                  False),
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
def test_unnorm_mutation_is_caught(tmp_path, name):
    lib = _mutant(tmp_path, name)

    def fwd(*args, **kw):
        return oracle.forward(*args, lib=lib, **kw)

    caught = []
    for pin, fn in UNNORM_PINS.items():
        try:
            err = fn(fwd)
        except (FloatingPointError, ValueError):
            err = np.inf
        if not err < TOL:
            caught.append(pin)
    assert caught, "mutation %s passed every pin" % name


def _inp(B, H, T, Dk, Dv, J, seed, state_std=0.3):
    return workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="f32", seed=seed, state_std=state_std)


def _f64(inp):
    return [np.asarray(inp[n], dtype=np.float64) for n in NAMES]


# the fixed point is the variant's own sequential trajectory, with the exact
# Jacobian and with the clamped one (App. D.1-D.2); ragged last chunk
@pytest.mark.parametrize("g_clamp", [None, "stable"])
def test_unnorm_fixed_point_is_sequential(g_clamp):
    inp = _inp(1, 2, 13, 4, 3, 3, seed=61)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"], unnormalized=True)
    o, S, _ = newton.newton_forward(*args, inp["state"], chunk=5, iters=13, g_clamp=g_clamp,
                                    unnormalized=True)
    assert np.max(np.abs(o - seq["o"])) < 1e-10
    assert np.max(np.abs(S - seq["state"])) < 1e-10


# after i sweeps the first i predictions are exact (App. D.1)
def test_unnorm_first_i_steps_exact():
    inp = _inp(1, 1, 10, 3, 2, 2, seed=62)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"], unnormalized=True, want_delta=True)
    exact_pred = args[2][0, :, 0][:, None, :] - seq["delta"][0, :, 0]
    _, _, heads = newton.newton_forward(*args, inp["state"], chunk=4, iters=10, unnormalized=True)
    preds = heads[(0, 0)]["preds"]
    for i in range(1, 11):
        assert np.max(np.abs(preds[i][:i] - exact_pred[:i])) < 1e-10, i


# With the exact Jacobian the iteration is Newton's method on the trajectory:
# once close, each sweep squares the error (quadratic convergence), which the
# normalised form's quasi-Newton sweeps do not do in general.
def test_unnorm_newton_converges_quadratically():
    inp = _inp(1, 1, 48, 8, 4, 3, seed=63, state_std=0.1)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"], unnormalized=True, want_delta=True)
    exact = args[2][0, :, 0][:, None, :] - seq["delta"][0, :, 0]
    _, _, heads = newton.newton_forward(*args, inp["state"], chunk=16, iters=12,
                                        unnormalized=True)
    errs = [np.max(np.abs(p - exact)) for p in heads[(0, 0)]["preds"]]
    assert errs[-1] < 1e-12
    close = [i for i in range(len(errs) - 1) if 1e-12 < errs[i] < 1e-2 and errs[i + 1] > 1e-13]
    assert close, errs
    for i in close:
        assert errs[i + 1] <= 10.0 * errs[i] ** 2, (i, errs)
