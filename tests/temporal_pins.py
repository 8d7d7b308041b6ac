"""Pins for the Temporal SwiLA form of the fp64 oracle (Sec. 3.3, App. B.3):
reductions to the plain recurrence, closed forms of the prior recursions, and
relations between the oracle's outputs that the paper's definitions fix.

Every pin takes ``fwd`` (a callable with the signature of ``oracle.forward``)
and returns the largest absolute deviation it found; the tests require a value
below ``TOL``.  The same pins run against deliberately broken copies of the
oracle's temporal code, each of which must fail at least one of them.
"""
from __future__ import annotations

import numpy as np
import scipy.special

import workloads

TOL = 1e-10
NAMES = workloads.NAMES
SAT = 40.0     # sigmoid(40) rounds to 1 in fp64
OFF = -800.0   # sigmoid(-800) is exactly 0 in fp64


def _case(B, H, T, D, J, seed, state_std=0.3, prior_state=True, gate_scale=1.0):
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="f32", seed=seed, state_std=state_std)
    tmp = workloads.temporal_inputs(B, H, T, D, J, dtype="f32", seed=seed,
                                    gate_scale=gate_scale, prior_state=prior_state)
    args = [np.asarray(inp[n], dtype=np.float64) for n in NAMES]
    return inp, tmp, args


# T1 -- gates saturated at 1: both priors are the new softmax priors at every
#       token, which is the plain recurrence (Sec. 3.2) exactly.
def pin_t_saturated_gates(fwd):
    inp, tmp, args = _case(2, 2, 12, 6, 3, seed=101)
    B, T, H, D = args[2].shape
    g = np.full((B, T, H, D), SAT)
    plain = fwd(*args, inp["state"])
    temp = fwd(*args, inp["state"], gate_k_logit=g, gate_q_logit=g, prior_in=tmp["prior"])
    return max(np.abs(plain["o"] - temp["o"]).max(), np.abs(plain["state"] - temp["state"]).max())


# T2 -- one component: every prior is 1, so any gates leave the plain
#       recurrence unchanged (up to the rounding of (1-g) + g).
def pin_t_single_component(fwd):
    inp, tmp, args = _case(2, 2, 10, 5, 1, seed=102, prior_state=False)
    plain = fwd(*args, inp["state"])
    temp = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"])
    return max(np.abs(plain["o"] - temp["o"]).max(), np.abs(plain["state"] - temp["state"]).max())


# T3 -- query gate closed: the query prior stays at its initial value, so the
#       one-token output is sum_j rho0_j (W_1 q)_j with W_1 the returned state.
def pin_t_frozen_query_prior(fwd):
    inp, tmp, args = _case(2, 3, 1, 6, 3, seed=103)
    B, T, H, D = args[2].shape
    J = args[3].shape[3]
    rho0 = tmp["prior"].astype(np.float64)[:, :, 1]                 # [B,H,J,D]
    gq = np.full((B, T, H, D), OFF)
    r = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=gq, prior_in=tmp["prior"])
    y = np.einsum("bhjid,bhi->bhjd", r["state"], args[0][:, 0])      # W_1 q per (j, d)
    o = (rho0 * y).sum(axis=2)                                      # [B,H,D]
    err = np.abs(r["o"][:, 0] - o).max()
    err = max(err, np.abs(r["prior"][:, :, 1] - rho0).max())
    # and with no prior state the frozen prior is uniform
    r = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=gq)
    y = np.einsum("bhjid,bhi->bhjd", r["state"], args[0][:, 0])
    return max(err, np.abs(r["o"][:, 0] - y.mean(axis=2)).max())


# T4 -- constant query logits and gate g: rhobar_T = pi + (1 - g)^T (rho0 - pi),
#       the solution of the linear recursion.
def pin_t_query_prior_closed_form(fwd):
    inp, tmp, args = _case(1, 2, 9, 4, 3, seed=104)
    B, T, H, D = args[2].shape
    J = args[3].shape[3]
    lq = np.repeat(args[5][:, :1], T, axis=1)                        # same logits every token
    args[5] = lq
    gl = 0.3
    gq = np.full((B, T, H, D), gl)
    r = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=gq, prior_in=tmp["prior"])
    g = 1.0 / (1.0 + np.exp(-gl))
    pi = scipy.special.softmax(lq[:, 0], axis=2)                     # [B,H,J,D]
    rho0 = tmp["prior"].astype(np.float64)[:, :, 1]
    want = pi + (1.0 - g) ** T * (rho0 - pi)
    return np.abs(r["prior"][:, :, 1] - want).max()


def _e_step_relation(fwd, gk, seed):
    """Largest deviation from r_t ~ ((1-g_t) r_{t-1} + g_t pi^k_t) exp(-delta_t^2/2),
    with r_0 the input prior state, using the oracle's own r and delta."""
    inp, tmp, args = _case(2, 2, 10, 5, 3, seed=seed)
    if gk is None:
        gk = tmp["gk"]
    r = fwd(*args, inp["state"], gate_k_logit=gk, gate_q_logit=tmp["gq"], prior_in=tmp["prior"],
            want_resp=True, want_delta=True)
    resp, delta = r["resp"], r["delta"]                               # [B,T,H,J,D]
    T = resp.shape[1]
    g = scipy.special.expit(np.asarray(gk, dtype=np.float64))        # sigmoid, [B,T,H,D]
    pik = scipy.special.softmax(args[4], axis=3)
    prev = tmp["prior"].astype(np.float64)[:, :, 0]                  # r_0 [B,H,J,D]
    err = 0.0
    for t in range(T):
        rbar = (1.0 - g[:, t, :, None]) * prev + g[:, t, :, None] * pik[:, t]
        lik = np.exp(-0.5 * delta[:, t] ** 2)
        want = rbar * lik / (rbar * lik).sum(axis=2, keepdims=True)
        err = max(err, np.abs(resp[:, t] - want).max())
        prev = resp[:, t]
    err = max(err, np.abs(r["prior"][:, :, 0] - resp[:, -1]).max())
    return err


# T5 -- key gate closed: the key prior of each token is the previous token's
#       responsibilities (a pure filter), checked on the oracle's r and delta.
def pin_t_key_filter(fwd):
    B, T, H, D = 2, 10, 2, 5
    return _e_step_relation(fwd, np.full((B, T, H, D), OFF), seed=105)


# T6 -- general gates: the key prior is the gated mixture of the previous
#       responsibilities and pi^k = softmax(key-prior logits).
def pin_t_key_mixture(fwd):
    return _e_step_relation(fwd, None, seed=106)


# T7 -- the prior state carries everything: two calls chained through
#       (state, prior state) equal one call over the whole sequence.
def pin_t_state_passing(fwd):
    inp, tmp, args = _case(2, 2, 11, 4, 3, seed=107)
    whole = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"],
                prior_in=tmp["prior"])
    c = 5
    a = fwd(*[x[:, :c] for x in args], inp["state"], gate_k_logit=tmp["gk"][:, :c],
            gate_q_logit=tmp["gq"][:, :c], prior_in=tmp["prior"])
    b = fwd(*[x[:, c:] for x in args], a["state"], gate_k_logit=tmp["gk"][:, c:],
            gate_q_logit=tmp["gq"][:, c:], prior_in=a["prior"])
    o = np.concatenate([a["o"], b["o"]], axis=1)
    return max(np.abs(o - whole["o"]).max(), np.abs(b["state"] - whole["state"]).max(),
               np.abs(b["prior"] - whole["prior"]).max())


# T8 -- the retrieval uses the running query prior: o_t = sum_j rhobar_tj (W_t q_t)_j
#       with W_t and rhobar_t taken from the outputs of each prefix.
def pin_t_retrieval_prior(fwd):
    inp, tmp, args = _case(1, 2, 6, 4, 3, seed=108)
    T = args[0].shape[1]
    whole = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"],
                prior_in=tmp["prior"])
    err = 0.0
    for t in range(1, T + 1):
        p = fwd(*[x[:, :t] for x in args], inp["state"], gate_k_logit=tmp["gk"][:, :t],
                gate_q_logit=tmp["gq"][:, :t], prior_in=tmp["prior"])
        y = np.einsum("bhjid,bhi->bhjd", p["state"], args[0][:, t - 1])
        o = (p["prior"][:, :, 1] * y).sum(axis=2)
        err = max(err, np.abs(whole["o"][:, t - 1] - o).max())
    return err


# T9 -- both parts of the returned prior state are distributions over j
#       (given an input prior state that is one).
def pin_t_prior_state_valid(fwd):
    inp, tmp, args = _case(2, 2, 8, 5, 4, seed=109, gate_scale=3.0)
    prior = tmp["prior"].astype(np.float64)
    prior /= prior.sum(axis=3, keepdims=True)
    r = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"], prior_in=prior)
    p = r["prior"]
    err = np.abs(p.sum(axis=3) - 1.0).max()
    if p.min() < 0 or p.max() > 1:
        err = max(err, 1.0)
    return err


TEMPORAL_PINS = {
    "saturated_gates": pin_t_saturated_gates,
    "single_component": pin_t_single_component,
    "frozen_query_prior": pin_t_frozen_query_prior,
    "query_prior_closed_form": pin_t_query_prior_closed_form,
    "key_filter": pin_t_key_filter,
    "key_mixture": pin_t_key_mixture,
    "state_passing": pin_t_state_passing,
    "retrieval_prior": pin_t_retrieval_prior,
    "prior_state_valid": pin_t_prior_state_valid,
}
