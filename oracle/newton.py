"""Chunkwise parallel quasi-Newton evaluation of the SwiLA recurrence, App. D.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  NumPy fp64, explicit loops over the
mixture component j and output dimension d so that every equation can be
checked by eye; meant for small shapes.

The iteration (App. D.1, eq. unif) refines a guess of the whole trajectory
w_{1:T}.  Each step linearises the recurrence around the previous iterate:

  g_t = beta_t r_t [1 - delta_t^2 (1 - r_t)]                    eq. jacobian_coeff
  p_t = g_t k_t^T w^{(i)}_{t-1} + beta_t r_t delta_t            eq. effective_input
  w^{(i+1)}_t = (I - g_t k_t k_t^T) w^{(i+1)}_{t-1} + k_t p_t   eq. linearized

and solves that linear recurrence chunk by chunk (App. D.3):

  Lambda_{s,t} = -g_s k_s^T k_t  (s > t), 0 otherwise          eq. lambda
  M = (I - Lambda)^{-1} diag(g) K                               eq. aggregate_transition
  Hh = (I - Lambda)^{-1} p                                      eq. aggregate_history
  w_{[n+1]} = w_{[n]} + K^T (Hh - M w_{[n]})                    eq. boundary
  O = K w_{[n]} + (K K^T . L) (Hh - M w_{[n]})                  eq. parallel_output

Readings taken where the appendix is silent:
* g, p, Lambda, M, Hh carry the output index d as well as j: g depends on d
  (eq. jacobian_coeff), so each (j, d) column has its own triangular system.
* eq. parallel_output with the strict mask L yields k_s^T w_{s-1}, the
  predictions; the recurrence depends on the iterate only through them, so the
  iteration carries the predictions from one sweep to the next.
* The initial guess is w^{(0)}_t = W_0 for every t.
* The layer output after an iteration is eq. retrieval evaluated on the
  trajectory of that iteration's linear solve.
* ``g_clamp`` (default off) optionally clips g into an interval; the fixed point
  does not depend on the Jacobian approximation (App. D.2).  ``"stable"``
  clips g_t into [0, 2 / |k_t|^2], the widest interval in which every
  linearised transition I - g k k^T has spectral radius at most 1 (its only
  eigenvalue other than 1 is 1 - g |k|^2).  Without such a clip, g < 0 makes
  transitions expansive and the iterates of long sequences overflow before
  they converge.
* ``unnormalized`` runs App. D.2's variant of the recurrence whose
  responsibilities drop the denominator of eq. responsibility,
  r = pi^k exp(-delta^2/2).  Each (j, d) column is then a recurrence of its own,
  and its Jacobian I - g k k^T with g = beta r (1 - delta^2) is exact (the
  derivative of r delta along w is -r (1 - delta^2) k^T), so the iteration is
  Newton's method proper; its fixed point is the sequential trajectory of the
  same variant.
"""
from __future__ import annotations

import numpy as np


def _softmax_j(x):
    m = x.max(axis=0, keepdims=True)
    e = np.exp(x - m)
    return e / e.sum(axis=0, keepdims=True)


def linearise(pred, v, beta, prior_k, g_clamp=None, kk=None, unnormalized=False):
    """Jacobian coefficient g (eq. jacobian_coeff) and effective input p
    (eq. effective_input) around predictions ``pred`` = k_t^T w^{(i)}_{t-1}.
    pred, beta, prior_k [T,J,Dv]; v [T,Dv]; kk [T] = |k_t|^2 (needed for
    g_clamp="stable").  With ``unnormalized``, r has no denominator and g is
    the exact coefficient of that variant (App. D.2).  Returns (g, p, delta, r)."""
    delta = v[:, None, :] - pred
    num = prior_k * np.exp(-0.5 * delta ** 2)
    if unnormalized:
        r = num
        g = beta * r * (1.0 - delta ** 2)
    else:
        r = num / num.sum(axis=1, keepdims=True)
        g = beta * r * (1.0 - delta ** 2 * (1.0 - r))
    if isinstance(g_clamp, str):
        if g_clamp != "stable":
            raise ValueError("g_clamp must be None, (lo, hi) or 'stable'")
        with np.errstate(divide="ignore"):
            hi = 2.0 / np.asarray(kk, dtype=np.float64)          # inf for a zero key
        g = np.minimum(np.maximum(g, 0.0), hi[:, None, None])
    elif g_clamp is not None:
        g = np.clip(g, g_clamp[0], g_clamp[1])
    p = g * pred + beta * r * delta
    return g, p, delta, r


def newton_head(q, k, v, lb, lk, lq, W0=None, *, chunk, iters, g_clamp=None, tol=None,
                unnormalized=False):
    """One head.  q, k [T,Dk]; v [T,Dv]; logits [T,J,Dv]; W0 [J,Dv,Dk] (paper
    layout: W0[j, d] is w_{jd}) or None.

    Returns a dict: ``o`` [T,Dv], ``W`` [J,Dv,Dk] (the final state),
    ``preds`` list of [T,J,Dv] predictions k_t^T w_{t-1} per iterate (entry 0 is
    the initial guess), ``iters`` the number of sweeps run.
    """
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    lb, lk, lq = (np.asarray(x, dtype=np.float64) for x in (lb, lk, lq))
    T, Dk = k.shape
    Dv = v.shape[1]
    J = lb.shape[1]
    W0 = np.zeros((J, Dv, Dk)) if W0 is None else np.asarray(W0, dtype=np.float64)
    beta = 1.0 / (1.0 + np.exp(-lb))                            # App. B.2
    prior_k = np.stack([_softmax_j(lk[t]) for t in range(T)])   # [T,J,Dv]
    prior_q = np.stack([_softmax_j(lq[t]) for t in range(T)])

    # initial guess: every state equals W_0, so pred_t = k_t^T W_0
    pred = np.einsum("ti,jdi->tjd", k, W0)
    preds = [pred.copy()]
    traj = np.broadcast_to(W0, (T, J, Dv, Dk)).copy()
    W_end = W0.copy()
    n_run = 0
    for _ in range(iters):
        # linearisation around the current iterate (App. D.2)
        g, p, _, _ = linearise(pred, v, beta, prior_k, g_clamp, kk=np.einsum("ti,ti->t", k, k),
                               unnormalized=unnormalized)

        new_pred = np.zeros_like(pred)
        Wb = W0.copy()                      # boundary state w_[n]
        for n0 in range(0, T, chunk):
            idx = np.arange(n0, min(n0 + chunk, T))
            Kc = k[idx]                      # [c, Dk]
            c = len(idx)
            G = Kc @ Kc.T
            L = np.tril(np.ones((c, c)), -1)
            W_next = Wb.copy()
            for j in range(J):
                for d in range(Dv):
                    gc = g[idx, j, d]
                    Lam = -(gc[:, None] * G) * L                     # eq. lambda
                    A = np.eye(c) - Lam
                    M = np.linalg.solve(A, gc[:, None] * Kc)         # eq. aggregate_transition
                    Hh = np.linalg.solve(A, p[idx, j, d])            # eq. aggregate_history
                    x = Hh - M @ Wb[j, d]
                    W_next[j, d] = Wb[j, d] + Kc.T @ x               # eq. boundary
                    new_pred[idx, j, d] = Kc @ Wb[j, d] + (G * L) @ x  # eq. parallel_output
                    traj[idx, j, d] = Wb[j, d] + np.cumsum(x[:, None] * Kc, axis=0)
            Wb = W_next
        W_end = Wb
        change = np.max(np.abs(new_pred - pred)) if T else 0.0
        pred = new_pred
        preds.append(pred.copy())
        n_run += 1
        if tol is not None and change <= tol:
            break

    # eq. retrieval on the final trajectory
    o = np.einsum("tjd,tjdi,ti->td", prior_q, traj, q)
    return {"o": o, "W": W_end, "preds": preds, "iters": n_run}


def newton_forward(q, k, v, lb, lk, lq, state_in=None, *, chunk, iters, g_clamp=None, tol=None,
                   unnormalized=False):
    """All heads, in the library's layouts: q, k [B,T,H,Dk]; v [B,T,H,Dv];
    logits [B,T,H,J,Dv]; state [B,H,J,Dk,Dv].  Returns (o [B,T,H,Dv],
    state [B,H,J,Dk,Dv], per-head result dicts)."""
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    B, T, H, Dk = q.shape
    Dv = v.shape[3]
    J = lb.shape[3]
    o = np.zeros((B, T, H, Dv))
    S = np.zeros((B, H, J, Dk, Dv))
    heads = {}
    for b in range(B):
        for h in range(H):
            W0 = None
            if state_in is not None:
                W0 = np.transpose(np.asarray(state_in, dtype=np.float64)[b, h], (0, 2, 1))
            res = newton_head(q[b, :, h], k[b, :, h], v[b, :, h], lb[b, :, h], lk[b, :, h],
                              lq[b, :, h], W0, chunk=chunk, iters=iters, g_clamp=g_clamp, tol=tol,
                              unnormalized=unnormalized)
            o[b, :, h] = res["o"]
            S[b, h] = np.transpose(res["W"], (0, 2, 1))
            heads[(b, h)] = res
    return o, S, heads
