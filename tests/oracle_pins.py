"""Pins for the fp64 oracle: checks against what the paper and the mathematics
fix, each computed by a route other than the oracle's own formulas.

Every pin takes ``fwd`` (a callable with the signature of ``oracle.forward``)
and returns the largest absolute deviation it found; the tests require a value
below ``TOL``.  The same pins are run against deliberately broken copies of
the oracle to show that a plausible mistake fails at least one of them.
"""
from __future__ import annotations

import json
import os

import numpy as np
import scipy.linalg
import scipy.special
import scipy.stats
import torch

import workloads

TOL = 1e-10
NAMES = workloads.NAMES
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_examples.json")


def _inp(B, H, T, Dk, Dv, J, seed, state_std=0.0, logit_scale=1.0):
    return workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="f32", seed=seed,
                                state_std=state_std, logit_scale=logit_scale)


def _args(inp, t0=0, t1=None):
    return [np.asarray(inp[n], dtype=np.float64)[:, t0:t1] for n in NAMES]


def _prefix_states(fwd, inp):
    """State after each prefix of the sequence: S[0] = initial, S[t] after t tokens."""
    T = inp["q"].shape[1]
    B, _, H, Dk = inp["q"].shape
    J, Dv = inp["lb"].shape[3], inp["lb"].shape[4]
    s0 = inp["state"] if inp["state"] is not None else np.zeros((B, H, J, Dk, Dv))
    states = [np.asarray(s0, dtype=np.float64)]
    for t in range(1, T + 1):
        states.append(fwd(*_args(inp, 0, t), inp["state"])["state"])
    return states


# P1 -- responsibilities are a distribution over j for every (t, d)  (eq. responsibility)
def pin_resp_normalised(fwd):
    inp = _inp(2, 2, 16, 4, 5, 3, seed=11, state_std=0.3)
    r = fwd(*_args(inp), inp["state"], want_resp=True)["resp"]
    err = np.max(np.abs(r.sum(axis=3) - 1.0))
    if r.min() < 0 or r.max() > 1:
        err = max(err, 1.0)
    return err


# P2 -- the E-step is Bayes' rule with unit-variance Gaussian likelihoods
#       (eq. molr_gen_model), evaluated with scipy's normal density on the
#       predictions of the oracle's own state outputs.
def pin_bayes_estep(fwd):
    inp = _inp(2, 2, 6, 3, 4, 3, seed=12, state_std=0.7)
    S = _prefix_states(fwd, inp)
    r = fwd(*_args(inp), inp["state"], want_resp=True)["resp"]
    q, k, v, lb, lk, lq = _args(inp)
    err = 0.0
    for t in range(k.shape[1]):
        pred = np.einsum("bhjid,bhi->bhjd", S[t], k[:, t])
        like = scipy.stats.norm.pdf(v[:, t][:, :, None, :], loc=pred, scale=1.0)
        prior = scipy.special.softmax(lk[:, t], axis=2)
        post = prior * like / (prior * like).sum(axis=2, keepdims=True)
        err = max(err, np.max(np.abs(post - r[:, t])))
    # errors so large that every density underflows in fp64: Bayes' rule in log
    # space (scipy's normal log-density and a softmax over j)
    inp = _inp(1, 2, 5, 3, 4, 3, seed=20, state_std=3.0, logit_scale=5.0)
    inp["v"] = inp["v"] * np.float32(60.0)
    S = _prefix_states(fwd, inp)
    r = fwd(*_args(inp), inp["state"], want_resp=True)["resp"]
    q, k, v, lb, lk, lq = _args(inp)
    for t in range(k.shape[1]):
        pred = np.einsum("bhjid,bhi->bhjd", S[t], k[:, t])
        logpost = (scipy.special.log_softmax(lk[:, t], axis=2)
                   + scipy.stats.norm.logpdf(v[:, t][:, :, None, :], loc=pred, scale=1.0))
        post = scipy.special.softmax(logpost, axis=2)
        err = max(err, np.max(np.abs(post - r[:, t])))
    return err


# P3 -- the update is beta times the gradient of the marginal log-likelihood
#       (eq. loglik, eq. recurrence, App. B.1); the gradient comes from torch
#       autograd in fp64, not from the closed form r*delta*k.  The retrieval is
#       checked on the returned state (eq. retrieval).
def pin_em_gradient(fwd):
    inp = _inp(2, 2, 6, 3, 4, 3, seed=13, state_std=0.7)
    S = _prefix_states(fwd, inp)
    out = fwd(*_args(inp), inp["state"])
    q, k, v, lb, lk, lq = (torch.from_numpy(x) for x in _args(inp))
    err = 0.0
    for t in range(k.shape[1]):
        W = torch.tensor(S[t], dtype=torch.float64, requires_grad=True)
        pred = torch.einsum("bhjid,bhi->bhjd", W, k[:, t])
        log_prior = torch.log_softmax(lk[:, t], dim=2)
        log_like = torch.distributions.Normal(pred, 1.0).log_prob(v[:, t][:, :, None, :])
        ll = torch.logsumexp(log_prior + log_like, dim=2).sum()
        (grad,) = torch.autograd.grad(ll, W)
        beta = torch.sigmoid(lb[:, t])[:, :, :, None, :]
        expect = S[t] + (beta * grad).numpy()
        err = max(err, np.max(np.abs(expect - S[t + 1])))
        prior_q = torch.softmax(lq[:, t], dim=2).numpy()
        o = np.einsum("bhjd,bhjid,bhi->bhd", prior_q, S[t + 1], q[:, t].numpy())
        err = max(err, np.max(np.abs(o - out["o"][:, t])))
    return err


def _deltanet_ut(K, Q, V, beta, w0):
    """Delta rule with per-output-dim learning rates in the closed UT form:
    u = (I + diag(beta) tril(K K^T, -1))^{-1} diag(beta) (v - K w0), one dense
    triangular solve per output dim; o_t = q_t.w0 + sum_{s<=t} (q_t.k_s) u_s;
    final w = w0 + K^T u.  K, Q [T,Dk]; V, beta [T,Dv]; w0 [Dk,Dv]."""
    w0 = np.asarray(w0, dtype=np.float64)
    T = K.shape[0]
    G = K @ K.T
    A_incl = np.tril(Q @ K.T)
    O = Q @ w0
    W = w0.copy()
    for d in range(V.shape[1]):
        Lmat = np.eye(T) + beta[:, d][:, None] * np.tril(G, -1)
        u = scipy.linalg.solve_triangular(Lmat, beta[:, d] * (V[:, d] - K @ w0[:, d]), lower=True)
        O[:, d] += A_incl @ u
        W[:, d] += K.T @ u
    return O, W


# P4 -- one component is the delta rule (Sec. 4.1): compare with the O(T^2)
#       closed form, from a non-zero initial state.
def pin_deltanet(fwd):
    inp = _inp(2, 2, 24, 5, 6, 1, seed=14, state_std=0.5)
    out = fwd(*_args(inp), inp["state"])
    q, k, v, lb, lk, lq = _args(inp)
    err = 0.0
    for b in range(2):
        for h in range(2):
            beta = scipy.special.expit(lb[b, :, h, 0])
            O, W = _deltanet_ut(k[b, :, h], q[b, :, h], v[b, :, h], beta, inp["state"][b, h, 0])
            err = max(err, np.max(np.abs(O - out["o"][b, :, h])),
                      np.max(np.abs(W - out["state"][b, h, 0])))
    return err


def _orthonormal_keys(rng, B, T, H, Dk):
    k = np.zeros((B, T, H, Dk))
    for b in range(B):
        for h in range(H):
            Qm, _ = np.linalg.qr(rng.standard_normal((Dk, Dk)))
            k[b, :, h] = Qm[:T]
    return k


# P5 -- orthonormal keys and a zero initial state make every prediction zero,
#       so delta = v and r = pi^k exactly; the output is then the brute-force sum
#       o_td = sum_j pi^q_tjd sum_{s<=t} beta_sjd pi^k_sjd v_sd (q_t.k_s).  With
#       one component and beta = 1 this is causal linear attention.
def pin_orthonormal(fwd):
    rng = np.random.Generator(np.random.PCG64(15))
    B, T, H, Dk, Dv, J = 2, 6, 2, 8, 5, 3
    inp = _inp(B, H, T, Dk, Dv, J, seed=15)
    inp["k"] = _orthonormal_keys(rng, B, T, H, Dk)
    out = fwd(*_args(inp), None, want_resp=True)
    q, k, v, lb, lk, lq = _args(inp)
    beta = scipy.special.expit(lb)
    pk = scipy.special.softmax(lk, axis=3)
    pq = scipy.special.softmax(lq, axis=3)
    err = np.max(np.abs(out["resp"] - pk))
    for b in range(B):
        for h in range(H):
            for t in range(T):
                for d in range(Dv):
                    o = 0.0
                    for j in range(J):
                        acc = sum(beta[b, s, h, j, d] * pk[b, s, h, j, d] * v[b, s, h, d]
                                  * np.dot(q[b, t, h], k[b, s, h]) for s in range(t + 1))
                        o += pq[b, t, h, j, d] * acc
                    err = max(err, abs(o - out["o"][b, t, h, d]))
    # one component, beta = 1: causal linear attention o_t = sum_{s<=t} (q_t.k_s) v_s
    inp1 = _inp(B, H, T, Dk, Dv, 1, seed=16)
    inp1["k"] = k
    inp1["lb"] = np.full_like(inp1["lb"], 40.0)
    out1 = fwd(*_args(inp1), None)
    q1, _, v1 = (np.asarray(inp1[n], dtype=np.float64) for n in ("q", "k", "v"))
    for b in range(B):
        for h in range(H):
            A = np.tril(q1[b, :, h] @ k[b, :, h].T)
            err = max(err, np.max(np.abs(A @ v1[b, :, h] - out1["o"][b, :, h])))
    return err


# P6 -- identical components (same initial weights, same beta and key-prior
#       logits for every j) stay identical, each takes 1/J of the responsibility,
#       and the layer is the delta rule with rate beta/J whatever pi^q is.
def pin_symmetric_components(fwd):
    B, T, H, Dk, Dv, J = 1, 20, 2, 4, 3, 3
    inp = _inp(B, H, T, Dk, Dv, J, seed=17, state_std=0.5)
    for n in ("lb", "lk"):
        inp[n] = np.repeat(inp[n][:, :, :, :1], J, axis=3)
    inp["state"] = np.repeat(inp["state"][:, :, :1], J, axis=2)
    out = fwd(*_args(inp), inp["state"], want_resp=True)
    q, k, v, lb, lk, lq = _args(inp)
    err = np.max(np.abs(out["resp"] - 1.0 / J))
    for b in range(B):
        for h in range(H):
            beta = scipy.special.expit(lb[b, :, h, 0]) / J
            O, W = _deltanet_ut(k[b, :, h], q[b, :, h], v[b, :, h], beta, inp["state"][b, h, 0])
            err = max(err, np.max(np.abs(O - out["o"][b, :, h])))
            for j in range(J):
                err = max(err, np.max(np.abs(W - out["state"][b, h, j])))
    return err


# P7 -- relabelling the components permutes the state and leaves o unchanged.
def pin_permutation(fwd):
    inp = _inp(2, 2, 12, 4, 5, 4, seed=18, state_std=0.4)
    perm = np.array([2, 0, 3, 1])
    a = fwd(*_args(inp), inp["state"])
    p = dict(inp)
    for n in ("lb", "lk", "lq"):
        p[n] = inp[n][:, :, :, perm]
    p["state"] = inp["state"][:, :, perm]
    b = fwd(*_args(p), p["state"])
    return max(np.max(np.abs(a["o"] - b["o"])), np.max(np.abs(a["state"][:, :, perm] - b["state"])))


# P8 -- closed-form cases worked by hand from the definitions.
def pin_hand_examples(fwd):
    doc = json.load(open(GOLDEN))
    err = 0.0
    for c in doc["cases"]:
        arr = {n: np.asarray(c[key], dtype=np.float64)[None, :, None]
               for n, key in zip(NAMES, ("q", "k", "v", "beta_logit", "prior_k_logit",
                                         "prior_q_logit"))}
        W0 = None if c["W0"] is None else np.asarray(c["W0"], dtype=np.float64)[None, None]
        out = fwd(*(arr[n] for n in NAMES), W0, want_resp=True)
        e = c["expect"]
        err = max(err,
                  np.max(np.abs(out["o"][0, :, 0] - np.asarray(e["o"]))),
                  np.max(np.abs(out["state"][0, 0] - np.asarray(e["state"]))),
                  np.max(np.abs(out["resp"][0, :, 0] - np.asarray(e["resp"]))))
    return err


# P9 -- a fixed-size state is all the history there is: running the sequence in
#       two pieces, passing the state, equals one run.
def pin_state_passing(fwd):
    inp = _inp(2, 3, 17, 4, 6, 2, seed=19, state_std=0.3)
    whole = fwd(*_args(inp), inp["state"])
    first = fwd(*_args(inp, 0, 7), inp["state"])
    second = fwd(*_args(inp, 7, None), first["state"])
    return max(np.max(np.abs(np.concatenate([first["o"], second["o"]], axis=1) - whole["o"])),
               np.max(np.abs(second["state"] - whole["state"])))


ALL_PINS = {
    "P1_resp_normalised": pin_resp_normalised,
    "P2_bayes_estep": pin_bayes_estep,
    "P3_em_gradient": pin_em_gradient,
    "P4_deltanet": pin_deltanet,
    "P5_orthonormal": pin_orthonormal,
    "P6_symmetric_components": pin_symmetric_components,
    "P7_permutation": pin_permutation,
    "P8_hand_examples": pin_hand_examples,
    "P9_state_passing": pin_state_passing,
}
