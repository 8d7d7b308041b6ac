"""Pins for the gradient oracle (``oracle.backward``): the exact gradient of the
plain forward of Sec. 3.2.

Every pin takes ``bwd`` (a callable with the signature of
``oracle.backward.backward``) and returns the largest deviation it found, to be
compared with the pin's own bar.  None of them uses ``bwd``'s arithmetic to make
its expected value: the first checks every gradient entry against central
finite differences of the C forward oracle, the rest check facts that follow
from the definition alone.
"""
from __future__ import annotations

import numpy as np

import oracle
import workloads

NAMES = workloads.NAMES       # q, k, v, lb, lk, lq


def _case(B, H, T, Dk, Dv, J, seed, state_std=0.4):
    inp = workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="f32", seed=seed, state_std=state_std)
    x = {n: np.asarray(inp[n], np.float64) for n in NAMES}
    x["state"] = None if inp["state"] is None else np.asarray(inp["state"], np.float64)
    rng = np.random.default_rng(seed + 1)
    go = rng.standard_normal(x["v"].shape)
    gs = rng.standard_normal((B, H, J, Dk, Dv))
    return x, go, gs


def _loss(x, go, gs):
    r = oracle.forward(*(x[n] for n in NAMES), x["state"])
    return float((go * r["o"]).sum() + (gs * r["state"]).sum())


# B1 -- every entry of every gradient equals the central difference of the
#       forward oracle's loss (step 1e-5, truncation error ~1e-10 here).
FD_BAR = 1e-6


def pin_b_finite_differences(bwd):
    x, go, gs = _case(1, 2, 5, 4, 3, 3, seed=301)
    g = bwd(*(x[n] for n in NAMES), x["state"], go, gs)
    eps = 1e-5
    err = 0.0
    for n in NAMES + ("state",):
        a = x[n]
        it = np.nditer(a, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            old = a[i]
            a[i] = old + eps
            lp = _loss(x, go, gs)
            a[i] = old - eps
            lm = _loss(x, go, gs)
            a[i] = old
            fd = (lp - lm) / (2 * eps)
            err = max(err, abs(fd - g[n][i]) / max(1.0, abs(fd)))
    return err


# B2 -- adding one constant to the J logits of a (t, d) changes neither softmax:
#       the logit gradients sum to zero over j.
def pin_b_softmax_shift(bwd):
    x, go, gs = _case(2, 2, 9, 8, 6, 4, seed=302)
    g = bwd(*(x[n] for n in NAMES), x["state"], go, gs)
    return max(np.abs(g["lk"].sum(axis=3)).max(), np.abs(g["lq"].sum(axis=3)).max())


# B3 -- J = 1: both priors are identically 1, so their logits have no gradient,
#       and r = 1 makes the update the delta rule w += beta delta k.
def pin_b_single_component(bwd):
    x, go, gs = _case(1, 2, 7, 5, 4, 1, seed=303)
    g = bwd(*(x[n] for n in NAMES), x["state"], go, gs)
    return max(np.abs(g["lk"]).max(), np.abs(g["lq"]).max())


# B4 -- beta = 0 (logit -800): the state never moves, o_td = sum_j pi^q_jd
#       w0_jd . q_t, so dk = dv = 0, dlb = dlk = 0, dq_t = sum_jd pi^q do w0_jd,
#       dW_0 = grad_state + sum_t (pi^q do) q_t.
def pin_b_frozen_state(bwd):
    x, go, gs = _case(2, 1, 6, 4, 3, 3, seed=304)
    x["lb"] = np.full_like(x["lb"], -800.0)
    with np.errstate(over="ignore"):     # sigmoid(-800) = 1 / (1 + inf) = 0
        g = bwd(*(x[n] for n in NAMES), x["state"], go, gs)
    e = np.exp(x["lq"] - x["lq"].max(axis=3, keepdims=True))
    piq = e / e.sum(axis=3, keepdims=True)                           # [B,T,H,J,Dv]
    dy = piq * go[:, :, :, None, :]
    dq = np.einsum("bthjd,bhjid->bthi", dy, x["state"])
    dw0 = gs + np.einsum("bthjd,bthi->bhjid", dy, x["q"])
    return max(np.abs(g["k"]).max(), np.abs(g["v"]).max(), np.abs(g["lb"]).max(),
               np.abs(g["lk"]).max(), np.abs(g["q"] - dq).max(), np.abs(g["state"] - dw0).max())


# B5 -- the gradient is linear in (grad_o, grad_state): the pair's sum gives the
#       sum of the gradients of each alone.
def pin_b_linear_in_seed(bwd):
    x, go, gs = _case(1, 2, 8, 6, 5, 2, seed=305)
    args = [x[n] for n in NAMES] + [x["state"]]
    a = bwd(*args, go, None)
    b = bwd(*args, np.zeros_like(go), gs)
    ab = bwd(*args, go, gs)
    return max(np.abs(ab[n] - a[n] - b[n]).max() for n in NAMES + ("state",))


# B6 -- T = 1 with zero initial state: pred = 0, delta = v, r = softmax_j(lk -
#       v^2/2) (independent of j through delta, so r = pi^k), and
#       o_d = (k . q) v_d sum_j pi^q_j beta_j pi^k_j.  The value gradient in closed
#       form: do_d (k . q) sum_j pi^q_j beta_j pi^k_j.
def pin_b_first_token(bwd):
    x, go, gs = _case(2, 2, 1, 4, 3, 3, seed=306, state_std=0.0)
    g = bwd(*(x[n] for n in NAMES), None, go, None)

    def sm(z):
        e = np.exp(z - z.max(axis=3, keepdims=True))
        return e / e.sum(axis=3, keepdims=True)

    pik, piq = sm(x["lk"]), sm(x["lq"])
    beta = 1.0 / (1.0 + np.exp(-x["lb"]))
    kq = (x["k"] * x["q"]).sum(axis=3)                                 # [B,1,H]
    s = (piq * beta * pik).sum(axis=3)                                 # [B,1,H,Dv]
    dv = go * kq[..., None] * s
    return np.abs(g["v"] - dv).max()


BACKWARD_PINS = {
    "finite_differences": (pin_b_finite_differences, FD_BAR),
    "softmax_shift": (pin_b_softmax_shift, 1e-12),
    "single_component": (pin_b_single_component, 1e-12),
    "frozen_state": (pin_b_frozen_state, 1e-12),
    "linear_in_seed": (pin_b_linear_in_seed, 1e-12),
    "first_token": (pin_b_first_token, 1e-12),
}
