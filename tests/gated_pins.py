"""Pins for the Gated SwiLA form of the fp64 oracle (Sec. 3.4, App. B.4): the
state decays by a per-key-dimension gate before the prediction (eq. pre-decay).

Every pin takes ``fwd`` (a callable with the signature of ``oracle.forward``)
and returns the largest absolute deviation it found (``TOL`` is the bar).  The
same pins run against deliberately broken copies of the oracle's gated code.
"""
from __future__ import annotations

import numpy as np
import scipy.special

import workloads

TOL = 1e-10
NAMES = workloads.NAMES
SAT = 40.0     # sigmoid(40) rounds to 1 in fp64
OFF = -800.0   # sigmoid(-800) is exactly 0 in fp64


def _case(B, H, T, D, J, seed, state_std=0.3):
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="f32", seed=seed, state_std=state_std)
    dec = workloads.gated_inputs(B, H, T, D, J, dtype="f32", seed=seed)["decay"]
    args = [np.asarray(inp[n], dtype=np.float64) for n in NAMES]
    return inp, np.asarray(dec, np.float64), args


# G1 -- decay gate saturated at 1: the plain recurrence exactly.
def pin_g_saturated(fwd):
    inp, dec, args = _case(2, 2, 12, 6, 3, seed=201)
    plain = fwd(*args, inp["state"])
    gated = fwd(*args, inp["state"], decay_logit=np.full_like(dec, SAT))
    return max(np.abs(plain["o"] - gated["o"]).max(),
               np.abs(plain["state"] - gated["state"]).max())


# G2 -- decay gate closed: the state forgets everything before each token, so
#       every component predicts 0, r = pi^k (equal errors cancel in eq.
#       responsibility), w_{t,jd} = beta r v_d k_t, and o_td = v_td (k_t . q_t)
#       sum_j pi^q beta pi^k.
def pin_g_closed(fwd):
    inp, dec, args = _case(2, 2, 7, 5, 3, seed=202)
    q, k, v, lb, lk, lq = args
    r = fwd(*args, inp["state"], decay_logit=np.full_like(dec, OFF))
    beta = scipy.special.expit(lb)
    pik = scipy.special.softmax(lk, axis=3)
    piq = scipy.special.softmax(lq, axis=3)
    kq = (k * q).sum(axis=3)                                        # [B,T,H]
    o = v * kq[..., None] * (piq * beta * pik).sum(axis=3)          # [B,T,H,D]
    w = beta[:, -1] * pik[:, -1] * v[:, -1][:, :, None]             # [B,H,J,D]
    state = w[:, :, :, None, :] * k[:, -1][:, :, None, :, None]     # [B,H,J,Dk,D]
    return max(np.abs(r["o"] - o).max(), np.abs(r["state"] - state).max())


# G3 -- J = 1, the affine-map form of App. B.4 with the decay as a right
#       diagonal scaling: W_t = W_{t-1} Diag(a_t) (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,
#       rows of W indexing output dims (one beta per output dim: a row scaling).
def pin_g_affine_map(fwd):
    inp, dec, args = _case(2, 2, 9, 5, 1, seed=203)
    q, k, v, lb, lk, lq = args
    r = fwd(*args, inp["state"], decay_logit=dec)
    B, T, H, D = v.shape
    a = scipy.special.expit(dec[:, :, :, 0])                        # [B,T,H,Dk]
    beta = scipy.special.expit(lb[:, :, :, 0])                      # [B,T,H,Dv]
    err = 0.0
    for b in range(B):
        for h in range(H):
            W = np.asarray(inp["state"], np.float64)[b, h, 0].T.copy()   # [Dv, Dk]
            for t in range(T):
                kt, vt, bt = k[b, t, h], v[b, t, h], beta[b, t, h]
                Wd = W @ np.diag(a[b, t, h])
                W = Wd - np.diag(bt) @ Wd @ np.outer(kt, kt) + np.outer(bt * vt, kt)
                err = max(err, np.abs(r["o"][b, t, h] - W @ q[b, t, h]).max())
            err = max(err, np.abs(r["state"][b, h, 0].T - W).max())
    return err


# G4 -- J = 1: eq. post-decay with (alpha, beta, v) equals eq. pre-decay with
#       (alpha, beta / alpha, alpha v) for a scalar decay (App. B.4).
def pin_g_pre_post_equivalence(fwd):
    inp, dec, args = _case(1, 2, 10, 6, 1, seed=204)
    q, k, v, lb, lk, lq = args
    B, T, H, D = v.shape
    rng = np.random.default_rng(204)
    alpha = rng.uniform(0.6, 0.95, size=(B, T, H))
    beta_post = rng.uniform(0.05, 0.5, size=(B, T, H, 1, D))
    dl = np.broadcast_to(scipy.special.logit(alpha)[:, :, :, None, None], (B, T, H, 1, D)).copy()
    post = fwd(q, k, v, scipy.special.logit(beta_post), lk, lq, inp["state"], decay_logit=dl,
               post_decay=True)
    beta_pre = beta_post / alpha[:, :, :, None, None]
    v_pre = v * alpha[:, :, :, None]
    pre = fwd(q, k, v_pre, scipy.special.logit(beta_pre), lk, lq, inp["state"], decay_logit=dl)
    return max(np.abs(post["o"] - pre["o"]).max(), np.abs(post["state"] - pre["state"]).max())


# G5 -- the E-step sees the decayed state: delta_t = v_t - (a_t (.) W_{t-1}) . k_t,
#       with W_{t-1} from the outputs of each prefix, and r from those errors.
def pin_g_decayed_errors(fwd):
    inp, dec, args = _case(1, 2, 6, 4, 3, seed=205)
    q, k, v, lb, lk, lq = args
    T = v.shape[1]
    whole = fwd(*args, inp["state"], decay_logit=dec, want_resp=True, want_delta=True)
    W = np.asarray(inp["state"], np.float64)                         # [B,H,J,Dk,Dv]
    a = scipy.special.expit(dec)                                     # [B,T,H,J,Dk]
    pik = scipy.special.softmax(lk, axis=3)
    err = 0.0
    for t in range(T):
        Wd = W * a[:, t][..., None]                                  # decay along Dk
        pred = np.einsum("bhjid,bhi->bhjd", Wd, k[:, t])
        delta = v[:, t][:, :, None, :] - pred                        # [B,H,J,D]
        lik = pik[:, t] * np.exp(-0.5 * delta ** 2)
        want_r = lik / lik.sum(axis=2, keepdims=True)
        err = max(err, np.abs(whole["delta"][:, t] - delta).max(),
                  np.abs(whole["resp"][:, t] - want_r).max())
        W = fwd(*[x[:, :t + 1] for x in args], inp["state"], decay_logit=dec[:, :t + 1])["state"]
    return err


# G6 -- two chained calls equal one.
def pin_g_state_passing(fwd):
    inp, dec, args = _case(2, 2, 11, 4, 3, seed=206)
    whole = fwd(*args, inp["state"], decay_logit=dec)
    c = 6
    a = fwd(*[x[:, :c] for x in args], inp["state"], decay_logit=dec[:, :c])
    b = fwd(*[x[:, c:] for x in args], a["state"], decay_logit=dec[:, c:])
    o = np.concatenate([a["o"], b["o"]], axis=1)
    return max(np.abs(o - whole["o"]).max(), np.abs(b["state"] - whole["state"]).max())


# G7 -- the decay composes with the temporal priors: a saturated decay gate
#       leaves the temporal form unchanged.
def pin_g_with_temporal(fwd):
    inp, dec, args = _case(1, 2, 8, 4, 3, seed=207)
    B, T, H, D = args[2].shape
    tmp = workloads.temporal_inputs(B, H, T, D, 3, dtype="f32", seed=207, prior_state=True)
    t0 = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"],
             prior_in=tmp["prior"])
    t1 = fwd(*args, inp["state"], gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"],
             prior_in=tmp["prior"], decay_logit=np.full_like(dec, SAT))
    return max(np.abs(t0["o"] - t1["o"]).max(), np.abs(t0["prior"] - t1["prior"]).max())


GATED_PINS = {
    "saturated": pin_g_saturated,
    "closed": pin_g_closed,
    "affine_map": pin_g_affine_map,
    "pre_post_equivalence": pin_g_pre_post_equivalence,
    "decayed_errors": pin_g_decayed_errors,
    "state_passing": pin_g_state_passing,
    "with_temporal": pin_g_with_temporal,
}
