"""Pins for the unnormalised-responsibility variant of the fp64 oracle
(App. D.2: the responsibilities of eq. responsibility without their
denominator, r = pi^k exp(-delta^2/2)), each computed by a route other than the
oracle's own formulas.

Every pin takes ``fwd`` (a callable with the signature of ``oracle.forward``)
and returns the largest absolute deviation it found; the tests require a value
below ``TOL``.  The same pins run against deliberately broken copies of the
oracle's variant code, each of which must fail at least one of them.
"""
from __future__ import annotations

import numpy as np
import scipy.special
import torch

import workloads

TOL = 1e-10
NAMES = workloads.NAMES


def _inp(B, H, T, Dk, Dv, J, seed, state_std=0.0):
    return workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="f32", seed=seed, state_std=state_std)


def _args(inp, t0=0, t1=None):
    return [np.asarray(inp[n], dtype=np.float64)[:, t0:t1] for n in NAMES]


# U1 -- the update is beta times the gradient of the mixture likelihood itself,
#       sum_j pi_j exp(-delta_j^2/2) (eq. loglik without its logarithm), from
#       torch autograd in fp64; the retrieval is eq. retrieval on the new state.
def pin_u_likelihood_gradient(fwd):
    inp = _inp(2, 2, 6, 3, 4, 3, seed=51, state_std=0.7)
    T = inp["q"].shape[1]
    B, _, H, Dk = inp["q"].shape
    J, Dv = inp["lb"].shape[3], inp["lb"].shape[4]
    states = [np.asarray(inp["state"], dtype=np.float64)]
    for t in range(1, T + 1):
        states.append(fwd(*_args(inp, 0, t), inp["state"], unnormalized=True)["state"])
    out = fwd(*_args(inp), inp["state"], unnormalized=True)
    q, k, v, lb, lk, lq = (torch.from_numpy(x) for x in _args(inp))
    err = 0.0
    for t in range(T):
        W = torch.tensor(states[t], dtype=torch.float64, requires_grad=True)
        pred = torch.einsum("bhjid,bhi->bhjd", W, k[:, t])
        prior = torch.softmax(lk[:, t], dim=2)
        lik = (prior * torch.exp(-0.5 * (v[:, t][:, :, None, :] - pred) ** 2)).sum()
        (grad,) = torch.autograd.grad(lik, W)
        beta = torch.sigmoid(lb[:, t])[:, :, :, None, :]
        err = max(err, np.max(np.abs(states[t] + (beta * grad).numpy() - states[t + 1])))
        prior_q = torch.softmax(lq[:, t], dim=2).numpy()
        o = np.einsum("bhjd,bhjid,bhi->bhd", prior_q, states[t + 1], q[:, t].numpy())
        err = max(err, np.max(np.abs(o - out["o"][:, t])))
    return err


# U2 -- one step from the same state: the variant's r is the normalised r
#       times the normaliser Z_d = sum_j pi^k_jd exp(-delta_jd^2/2), so its state
#       change is Z_d times that of the plain recurrence (whose oracle is pinned
#       on its own), column by column.
def pin_u_scaled_plain_step(fwd):
    inp = _inp(2, 3, 1, 5, 6, 4, seed=52, state_std=0.6)
    args = _args(inp)
    s0 = np.asarray(inp["state"], dtype=np.float64)
    plain = fwd(*args, inp["state"], want_delta=True, want_resp=True)
    unn = fwd(*args, inp["state"], unnormalized=True, want_resp=True)
    pk = scipy.special.softmax(args[4][:, 0], axis=2)                 # [B,H,J,Dv]
    Z = (pk * np.exp(-0.5 * plain["delta"][:, 0] ** 2)).sum(axis=2)   # [B,H,Dv]
    err = np.max(np.abs(unn["state"] - s0 - Z[:, :, None, None, :] * (plain["state"] - s0)))
    err = max(err, np.max(np.abs(unn["resp"][:, 0] - Z[:, :, None, :] * plain["resp"][:, 0])))
    return err


def _orthonormal_keys(rng, B, T, H, Dk):
    k = np.zeros((B, T, H, Dk))
    for b in range(B):
        for h in range(H):
            Qm, _ = np.linalg.qr(rng.standard_normal((Dk, Dk)))
            k[b, :, h] = Qm[:T]
    return k


# U3 -- orthonormal keys and a zero initial state: every prediction is zero, so
#       delta = v and r = pi^k exp(-v^2/2); the output is the brute-force O(T^2)
#       sum o_td = sum_j pi^q_tjd sum_{s<=t} beta_sjd r_sjd v_sd (q_t.k_s).
def pin_u_orthonormal(fwd):
    rng = np.random.Generator(np.random.PCG64(53))
    B, T, H, Dk, Dv, J = 2, 6, 2, 8, 5, 3
    inp = _inp(B, H, T, Dk, Dv, J, seed=53)
    inp["k"] = _orthonormal_keys(rng, B, T, H, Dk)
    out = fwd(*_args(inp), None, unnormalized=True, want_resp=True)
    q, k, v, lb, lk, lq = _args(inp)
    beta = scipy.special.expit(lb)
    pq = scipy.special.softmax(lq, axis=3)
    r = scipy.special.softmax(lk, axis=3) * np.exp(-0.5 * v[:, :, :, None, :] ** 2)
    err = np.max(np.abs(out["resp"] - r))
    for b in range(B):
        for h in range(H):
            A = np.tril(q[b, :, h] @ k[b, :, h].T)                     # (q_t.k_s), s <= t
            for j in range(J):
                c = beta[b, :, h, j] * r[b, :, h, j] * v[b, :, h]       # [T, Dv]
                o_j = pq[b, :, h, j] * (A @ c)
                if j == 0:
                    o = o_j
                else:
                    o = o + o_j
            err = max(err, np.max(np.abs(o - out["o"][b, :, h])))
    return err


# U4 -- App. D.2: without the denominator no term couples the components, and
#       one step's Jacobian in w_{jd} is I - g k k^T with g = beta r (1 - delta^2)
#       exactly.  Central differences of one step of the oracle, over every
#       component's weights: the diagonal blocks match, the others vanish.
def pin_u_exact_jacobian(fwd):
    B, H, Dk, Dv, J = 1, 1, 3, 2, 3
    inp = _inp(B, H, 1, Dk, Dv, J, seed=54, state_std=0.8)
    args = _args(inp)
    S0 = np.asarray(inp["state"], dtype=np.float64)
    k = args[1][0, 0, 0]
    v = args[2][0, 0, 0]
    beta = scipy.special.expit(args[3][0, 0, 0])
    prior = scipy.special.softmax(args[4][0, 0, 0], axis=0)
    pred = np.einsum("jid,i->jd", S0[0, 0], k)
    delta = v[None, :] - pred
    g = beta * prior * np.exp(-0.5 * delta ** 2) * (1.0 - delta ** 2)
    eps = 1e-6
    err = 0.0
    for d in range(Dv):
        for jin in range(J):
            for i in range(Dk):
                Sp, Sm = S0.copy(), S0.copy()
                Sp[0, 0, jin, i, d] += eps
                Sm[0, 0, jin, i, d] -= eps
                fp = fwd(*args, Sp, unnormalized=True)["state"][0, 0, :, :, d]
                fm = fwd(*args, Sm, unnormalized=True)["state"][0, 0, :, :, d]
                col = (fp - fm) / (2 * eps)                            # [J, Dk]
                for jout in range(J):
                    expect = np.zeros(Dk)
                    if jout == jin:
                        expect = np.eye(Dk)[:, i] - g[jin, d] * k * k[i]
                    err = max(err, np.max(np.abs(col[jout] - expect)))
    # central differences carry O(eps^2) truncation and O(1e-16/eps) rounding:
    # deviations within that accuracy (1e-7) count as none
    return err if err > 1e-7 else 0.0


UNNORM_PINS = {
    "U1_likelihood_gradient": pin_u_likelihood_gradient,
    "U2_scaled_plain_step": pin_u_scaled_plain_step,
    "U3_orthonormal": pin_u_orthonormal,
    "U4_exact_jacobian": pin_u_exact_jacobian,
}
