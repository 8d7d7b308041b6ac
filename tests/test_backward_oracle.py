"""The gradient oracle (``oracle.backward``) against its pins, and each plausible
mistake planted in a copy of it failing at least one pin."""
import inspect

import pytest

import oracle.backward as ob
from backward_pins import BACKWARD_PINS


@pytest.mark.parametrize("name", sorted(BACKWARD_PINS))
def test_backward_pin(name):
    pin, bar = BACKWARD_PINS[name]
    err = pin(ob.backward)
    assert err < bar, "%s: %.3e" % (name, err)


# name -> (text in the oracle, replacement)
MUTATIONS = {
    "no_exponent_term": ("ddelta = ddelta - delta * da", "ddelta = ddelta"),
    "exponent_term_sign": ("ddelta = ddelta - delta * da", "ddelta = ddelta + delta * da"),
    "pred_sign": ("dpred = -ddelta", "dpred = ddelta"),
    "softmax_jacobian_no_mean": ("da = r * (dr - (r * dr).sum(axis=0, keepdims=True))",
                                 "da = r * dr"),
    "sigmoid_derivative": ("dbeta * beta * (1.0 - beta)", "dbeta * beta"),
    "query_prior_no_mean": ("piq * (dpiq - (piq * dpiq).sum(axis=0, keepdims=True))",
                            "piq * dpiq"),
    "retrieval_with_old_state": ('np.einsum("jd,jdi->i", dy, w_t)',
                                 'np.einsum("jd,jdi->i", dy, w_prev[t])'),
    "key_grad_new_state": ('np.einsum("jd,jdi->i", dpred, w_prev[t])',
                           'np.einsum("jd,jdi->i", dpred, w_t)'),
    "update_grad_dropped": ('out["k"][b, t, h] += np.einsum("jd,jdi->i", c, G)', "pass"),
    "query_term_after_dc": ("                G = G + dy[:, :, None] * qt[None, None, :]\n", ""),
    "carry_misses_prediction": ("G = G + dpred[:, :, None] * kt[None, None, :]", "G = G"),
    "value_grad_one_component": ('out["v"][b, t, h] = ddelta.sum(axis=0)',
                                 'out["v"][b, t, h] = ddelta[0]'),
}


def _mutant(old, new):
    src = inspect.getsource(ob.backward)     # the code, not the module docstring
    assert src.count(old) == 1, old
    src = src.replace(old, new, 1)
    if "G = G + dy" in old:
        # move the query term after dc instead of dropping it
        src = src.replace("dc = G @ kt\n", "dc = G @ kt\n" + old, 1)
    ns = dict(vars(ob))
    exec(compile(src, "oracle_backward_mutant", "exec"), ns)
    return ns["backward"]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_backward_mutation_caught(name):
    bwd = _mutant(*MUTATIONS[name])
    worst = {}
    for pin_name, (pin, bar) in BACKWARD_PINS.items():
        try:
            err = pin(bwd)
        except Exception as e:  # a mutant that breaks outright is caught too
            err = float("inf")
            worst[pin_name] = repr(e)
        if not err < bar:
            return
        worst[pin_name] = err
    pytest.fail("mutation %s passed every pin: %s" % (name, worst))
