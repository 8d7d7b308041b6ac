"""Gradient of the plain SwiLA forward -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.

A plain fp64 NumPy implementation of reverse-mode differentiation through the
recurrence of Sec. 3.2 (eq. recurrence, eq. responsibility, eq. retrieval) with
beta and the priors formed from logits as in App. B.2.  The paper trains SwiLA
with automatic differentiation through its sequential evaluation and states no
backward formulas; what is computed here is the exact gradient of that forward,
written out by the chain rule, one token at a time, in reverse.  Only the tests,
the smoke check and the CPU-baseline leg of the benchmark may use it; it shares
nothing with the GPU library.

Per (b, h), with w_{t,jd} in R^{Dk} the regression weight of component j for
output dim d after token t, the forward is

    pred_{tjd}  = w_{t-1,jd} . k_t,        delta_{tjd} = v_{td} - pred_{tjd}
    r_{t.d}     = softmax_j(lk_{tjd} - delta_{tjd}^2 / 2)
                  (pi^k = softmax_j(lk); its normaliser cancels in r)
    beta_{tjd}  = sigmoid(lb_{tjd}),       c_{tjd} = beta r delta
    w_{t,jd}    = w_{t-1,jd} + c_{tjd} k_t
    y_{tjd}     = w_{t,jd} . q_t,          o_{td} = sum_j softmax_j(lq_{t.d})_j y_{tjd}

and for a scalar loss L with dL/do = grad_o and dL/dw_T = grad_state, the
reverse sweep carries G = dL/dw_t:

    dy = pi^q do;  dlq = pi^q (do y - sum_j pi^q do y);  G += dy q_t;  dq_t = sum dy w_t
    dc = G . k_t;  dk_t += sum c G
    dbeta = dc r delta -> dlb = dbeta beta (1 - beta)
    dr = dc beta delta;  da = r (dr - sum_j r dr);  dlk = da
    ddelta = dc beta r - delta da;  dv_t = sum_j ddelta;  dpred = -ddelta
    G += dpred k_t  (now dL/dw_{t-1});  dk_t += sum dpred w_{t-1}

and dL/dw_0 is G after token 0.

Layouts as the forward: q, k [B,T,H,Dk]; v, o [B,T,H,Dv]; logits
[B,T,H,J,Dv]; state [B,H,J,Dk,Dv] with element (b,h,j,i,d) = (w_{jd})_i.
"""
from __future__ import annotations

import numpy as np


def _softmax_j(x):
    """Softmax over axis 0 (the component axis of a [J, Dv] array)."""
    m = x.max(axis=0, keepdims=True)
    e = np.exp(x - m)
    return e / e.sum(axis=0, keepdims=True)


def backward(q, k, v, lb, lk, lq, state_in, grad_o, grad_state=None):
    """Gradients of L = sum(grad_o * o) + sum(grad_state * state_out) with respect
    to every input of the plain forward.  Returns a dict with q, k, v, lb, lk,
    lq (shaped like the inputs) and state (dL/dW_0, [B,H,J,Dk,Dv]); every value
    is fp64."""
    q, k, v, lb, lk, lq, grad_o = (np.asarray(x, np.float64)
                                   for x in (q, k, v, lb, lk, lq, grad_o))
    B, T, H, Dk = q.shape
    Dv = v.shape[3]
    J = lb.shape[3]
    out = {n: np.zeros_like(x) for n, x in
           (("q", q), ("k", k), ("v", v), ("lb", lb), ("lk", lk), ("lq", lq))}
    out["state"] = np.zeros((B, H, J, Dk, Dv))
    for b in range(B):
        for h in range(H):
            # w[j, d, :] = w_{jd}
            if state_in is None:
                w = np.zeros((J, Dv, Dk))
            else:
                w = np.asarray(state_in, np.float64)[b, h].transpose(0, 2, 1).copy()
            # forward, keeping what the reverse sweep needs
            w_prev, delta_t, r_t, beta_t, c_t, piq_t, y_t = [], [], [], [], [], [], []
            for t in range(T):
                kt, qt = k[b, t, h], q[b, t, h]
                w_prev.append(w.copy())
                delta = v[b, t, h][None, :] - w @ kt                      # [J, Dv]
                r = _softmax_j(lk[b, t, h] - 0.5 * delta ** 2)
                beta = 1.0 / (1.0 + np.exp(-lb[b, t, h]))
                c = beta * r * delta
                w = w + c[:, :, None] * kt[None, None, :]
                piq = _softmax_j(lq[b, t, h])
                y = w @ qt
                delta_t.append(delta); r_t.append(r); beta_t.append(beta)
                c_t.append(c); piq_t.append(piq); y_t.append(y)
            # reverse sweep; w is w_T here
            if grad_state is None:
                G = np.zeros((J, Dv, Dk))
            else:
                G = np.asarray(grad_state, np.float64)[b, h].transpose(0, 2, 1).copy()
            for t in reversed(range(T)):
                kt, qt, do = k[b, t, h], q[b, t, h], grad_o[b, t, h]
                delta, r, beta, c = delta_t[t], r_t[t], beta_t[t], c_t[t]
                piq, y = piq_t[t], y_t[t]
                w_t = w_prev[t] + c[:, :, None] * kt[None, None, :]
                # retrieval o = sum_j pi^q y, y = w_t . q
                dy = piq * do[None, :]
                dpiq = y * do[None, :]
                out["lq"][b, t, h] = piq * (dpiq - (piq * dpiq).sum(axis=0, keepdims=True))
                G = G + dy[:, :, None] * qt[None, None, :]
                out["q"][b, t, h] += np.einsum("jd,jdi->i", dy, w_t)
                # update w_t = w_{t-1} + c k
                dc = G @ kt
                out["k"][b, t, h] += np.einsum("jd,jdi->i", c, G)
                # c = beta r delta
                dbeta = dc * r * delta
                out["lb"][b, t, h] = dbeta * beta * (1.0 - beta)
                dr = dc * beta * delta
                ddelta = dc * beta * r
                # r = softmax_j(lk - delta^2 / 2)
                da = r * (dr - (r * dr).sum(axis=0, keepdims=True))
                out["lk"][b, t, h] = da
                ddelta = ddelta - delta * da
                # delta = v - w_{t-1} . k
                out["v"][b, t, h] = ddelta.sum(axis=0)
                dpred = -ddelta
                G = G + dpred[:, :, None] * kt[None, None, :]
                out["k"][b, t, h] += np.einsum("jd,jdi->i", dpred, w_prev[t])
            out["state"][b, h] = G.transpose(0, 2, 1)
    return out
