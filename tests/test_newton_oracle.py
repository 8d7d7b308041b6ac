"""The App. D chunkwise quasi-Newton oracle (NumPy) against what fixes it:
the sequential recurrence (independently pinned C oracle), the finite-difference
Jacobian, and the structural facts App. D states.  CPU only."""
import numpy as np
import pytest
import scipy.special

import oracle
import workloads
from oracle import newton
from oracle_pins import NAMES


def _inp(B, H, T, Dk, Dv, J, seed, state_std=0.3):
    return workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="f32", seed=seed, state_std=state_std)


def _f64(inp):
    return [np.asarray(inp[n], dtype=np.float64) for n in NAMES]


# P11 -- the fixed point is the sequential trajectory (App. D.1: the iteration
#        converges, whatever the Jacobian approximation); ragged last chunk.
@pytest.mark.parametrize("chunk", [4, 5, 13])
def test_fixed_point_is_sequential(chunk):
    inp = _inp(1, 2, 13, 4, 3, 3, seed=31)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"])
    o, S, _ = newton.newton_forward(*args, inp["state"], chunk=chunk, iters=13)
    assert np.max(np.abs(o - seq["o"])) < 1e-10
    assert np.max(np.abs(S - seq["state"])) < 1e-10


# P12 -- after i sweeps the first i predictions are exact (App. D.1: at most T
#        iterations).
def test_first_i_steps_exact():
    inp = _inp(1, 1, 10, 3, 2, 2, seed=32)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"], want_delta=True)
    exact_pred = args[2][0, :, 0][:, None, :] - seq["delta"][0, :, 0]     # v - delta
    _, _, heads = newton.newton_forward(*args, inp["state"], chunk=4, iters=10)
    preds = heads[(0, 0)]["preds"]
    for i in range(1, 11):
        assert np.max(np.abs(preds[i][:i] - exact_pred[:i])) < 1e-10, i
    assert np.max(np.abs(preds[10] - exact_pred)) < 1e-10


# P13 -- one component: r = 1, g = beta and the linearisation is exact, so a
#        single sweep gives the delta-rule trajectory.
def test_one_component_converges_in_one_sweep():
    inp = _inp(2, 2, 16, 5, 4, 1, seed=33)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"])
    o, S, _ = newton.newton_forward(*args, inp["state"], chunk=6, iters=1)
    assert np.max(np.abs(o - seq["o"])) < 1e-10
    assert np.max(np.abs(S - seq["state"])) < 1e-10


# P14 -- eq. jacobian: d f / d w_{jd} = I - g k k^T, with g from eq.
#        jacobian_coeff, against central differences of one step of the C oracle
#        with respect to one component's weights.
def test_jacobian_coefficient_matches_finite_differences():
    B, H, Dk, Dv, J = 1, 1, 3, 2, 3
    inp = _inp(B, H, 1, Dk, Dv, J, seed=34, state_std=0.8)
    args = _f64(inp)
    S0 = np.asarray(inp["state"], dtype=np.float64)
    k = args[1][0, 0, 0]
    v = args[2][0, 0, 0]
    beta = scipy.special.expit(args[3][0, 0, 0])
    prior = scipy.special.softmax(args[4][0, 0, 0], axis=0)
    pred = np.einsum("jid,i->jd", S0[0, 0], k)
    g, _, _, _ = newton.linearise(pred[None], v[None], beta[None], prior[None])
    eps = 1e-6
    for j in range(J):
        for d in range(Dv):
            Jac = np.zeros((Dk, Dk))
            for i in range(Dk):
                Sp, Sm = S0.copy(), S0.copy()
                Sp[0, 0, j, i, d] += eps
                Sm[0, 0, j, i, d] -= eps
                fp = oracle.forward(*args, Sp)["state"][0, 0, j, :, d]
                fm = oracle.forward(*args, Sm)["state"][0, 0, j, :, d]
                Jac[:, i] = (fp - fm) / (2 * eps)
            expect = np.eye(Dk) - g[0, j, d] * np.outer(k, k)
            assert np.max(np.abs(Jac - expect)) < 1e-7, (j, d)


# P15 -- every sweep solves its linear recurrence exactly, so the iterates do
#        not depend on the chunk size; chunk = T is one dense system per column.
def test_chunk_size_invariance():
    inp = _inp(1, 1, 12, 4, 3, 3, seed=35)
    args = _f64(inp)
    runs = []
    for c in (1, 3, 5, 12):
        _, _, heads = newton.newton_forward(*args, inp["state"], chunk=c, iters=4)
        runs.append(heads[(0, 0)]["preds"])
    for other in runs[1:]:
        for a, b in zip(runs[0], other):
            assert np.max(np.abs(a - b)) < 1e-10


# A clamp of g changes the path, not the fixed point (App. D.2).
def test_clamped_jacobian_same_fixed_point():
    inp = _inp(1, 1, 9, 3, 2, 2, seed=36)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"])
    o, S, _ = newton.newton_forward(*args, inp["state"], chunk=4, iters=9, g_clamp=(0.0, 1.0))
    assert np.max(np.abs(o - seq["o"])) < 1e-10
    assert np.max(np.abs(S - seq["state"])) < 1e-10


# The "stable" clamp, g_t in [0, 2 / |k_t|^2]: keys of norm^2 up to ~3 so that
# the upper bound binds; the fixed point is still the sequential trajectory and
# the first i predictions are exact after i sweeps (App. D.1-D.2).
def _scaled_keys(inp, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    k = np.asarray(inp["k"], dtype=np.float64)
    scale = np.sqrt(rng.uniform(0.5, 3.0, size=k.shape[:3] + (1,)))
    inp = dict(inp)
    inp["k"] = k / np.linalg.norm(k, axis=-1, keepdims=True) * scale
    return inp


def test_stable_clamp_fixed_point_and_exact_prefix():
    inp = _scaled_keys(_inp(1, 1, 12, 4, 3, 3, seed=37, state_std=0.2), seed=38)
    args = _f64(inp)
    seq = oracle.forward(*args, inp["state"], want_delta=True)
    exact_pred = args[2][0, :, 0][:, None, :] - seq["delta"][0, :, 0]
    o, S, heads = newton.newton_forward(*args, inp["state"], chunk=5, iters=12,
                                        g_clamp="stable")
    preds = heads[(0, 0)]["preds"]
    for i in range(1, 13):
        assert np.max(np.abs(preds[i][:i] - exact_pred[:i])) < 1e-9, i
    assert np.max(np.abs(o - seq["o"])) < 1e-9
    assert np.max(np.abs(S - seq["state"])) < 1e-9


def test_stable_clamp_bounds():
    inp = _scaled_keys(_inp(1, 1, 40, 6, 5, 4, seed=39), seed=40)
    k = np.asarray(inp["k"], dtype=np.float64)[0, :, 0]
    kk = np.einsum("ti,ti->t", k, k)
    rng = np.random.Generator(np.random.PCG64(41))
    pred = rng.standard_normal((40, 4, 5)) * 3.0          # far from any fixed point
    v = rng.standard_normal((40, 5))
    beta = rng.uniform(0.0, 1.0, (40, 4, 5))
    prior = scipy.special.softmax(rng.standard_normal((40, 4, 5)), axis=1)
    g0, _, _, _ = newton.linearise(pred, v, beta, prior)
    g, p, delta, r = newton.linearise(pred, v, beta, prior, "stable", kk=kk)
    hi = (2.0 / kk)[:, None, None]
    assert (g0 < 0).any() and (g0 > hi).any()              # both bounds are exercised
    assert np.all(g >= 0) and np.all(g <= hi)
    inside = (g0 >= 0) & (g0 <= hi)
    assert np.array_equal(g[inside], g0[inside])
    # p keeps its definition with the clamped g (eq. effective_input)
    assert np.allclose(p, g * pred + beta * r * delta, rtol=0, atol=1e-12)
