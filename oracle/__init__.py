"""SwiLA reference oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.

Plain, slow, fp64 CPU implementations of what the SwiLA hot path computes,
written from the paper:

* ``forward`` / ``decode_step`` -- the recurrence, E-step and retrieval of
  Sec. 3.2 (eq. recurrence, eq. responsibility, eq. retrieval), with beta and
  the two priors produced from logits as App. B.2 states; with gate logits,
  the temporal priors of Temporal SwiLA (Sec. 3.3, App. B.3).  Backed by the C
  file ``swila_oracle.c`` next to this module (compiled here with gcc on first
  use).
* ``newton`` (submodule) -- the chunkwise parallel quasi-Newton iteration of
  App. D (eqs. jacobian_coeff, effective_input, lambda, aggregate_transition,
  aggregate_history, boundary, parallel_output) in NumPy fp64.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU library
and never calls it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "swila_oracle.c")
_LIB = os.path.join(_HERE, "libswila_oracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (fp64, no fast-math) and return the path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(
            ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
             "-std=c11", "-pthread", "-o", tmp, _SRC, "-lm"],
            check=True)
        os.replace(tmp, _LIB)
    return _LIB


def load_library(path):
    """ctypes handle of a compiled oracle at ``path`` (the tests also load
    deliberately broken copies to check that the pins catch them)."""
    lib = ctypes.CDLL(path)
    dp = ctypes.POINTER(ctypes.c_double)
    lib.swila_oracle_forward.argtypes = [ctypes.c_int] * 6 + [dp] * 11 + [ctypes.c_int]
    lib.swila_oracle_forward.restype = ctypes.c_int
    lib.swila_oracle_forward_ext.argtypes = ([ctypes.c_int] * 6 + [dp] * 9 + [ctypes.c_int] * 2
                                             + [dp] * 7 + [ctypes.c_int])
    lib.swila_oracle_forward_ext.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            _lib = load_library(build())
    return _lib


def _f64(x):
    return None if x is None else np.ascontiguousarray(x, dtype=np.float64)


def _ptr(x):
    if x is None:
        return None
    return x.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def forward(q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in=None, *,
            gate_k_logit=None, gate_q_logit=None, prior_in=None, decay_logit=None,
            post_decay: bool = False, unnormalized: bool = False, nthreads: int = 0,
            want_resp: bool = False, want_delta: bool = False, lib=None):
    """Run the recurrence over a whole sequence.

    Shapes: q, k [B,T,H,Dk]; v [B,T,H,Dv]; the three logit tensors
    [B,T,H,J,Dv]; state_in None (zeros) or [B,H,J,Dk,Dv].  Inputs of any float
    dtype are upcast exactly to fp64.  Returns a dict with ``o`` [B,T,H,Dv],
    ``state`` [B,H,J,Dk,Dv] and, on request, ``resp`` (the key-side
    responsibilities r) and ``delta`` (the prediction errors), both
    [B,T,H,J,Dv].

    Temporal SwiLA (App. B.3): with ``gate_k_logit`` and ``gate_q_logit``
    ([B,T,H,Dv], both or neither) the priors are the running mixtures of the
    previous responsibilities (key side) or previous prior (query side) with
    the new softmax priors; ``prior_in`` is the carried prior state
    [B,H,2,J,Dv] (part 0: r_{t-1}, part 1: rhobar_{t-1}) or None (uniform 1/J),
    and the result then also holds ``prior``, the final prior state.

    Gated SwiLA (App. B.4): with ``decay_logit`` [B,T,H,J,Dk] the state decays by
    a = sigmoid(decay_logit), one gate per key dimension and component, before
    the prediction (eq. pre-decay), or after it with ``post_decay`` (eq.
    post-decay).  It combines with the temporal priors.

    ``unnormalized`` (App. D.2): the variant whose responsibilities drop the
    denominator of eq. responsibility, r = pi^k exp(-delta^2/2); plain form only.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    lb, lk, lq = _f64(beta_logit), _f64(prior_k_logit), _f64(prior_q_logit)
    B, T, H, Dk = q.shape
    Dv = v.shape[3]
    J = lb.shape[3]
    assert k.shape == (B, T, H, Dk) and v.shape == (B, T, H, Dv)
    for x in (lb, lk, lq):
        assert x.shape == (B, T, H, J, Dv)
    s_in = _f64(state_in)
    if s_in is not None:
        assert s_in.shape == (B, H, J, Dk, Dv)
    o = np.zeros((B, T, H, Dv))
    s_out = np.zeros((B, H, J, Dk, Dv))
    resp = np.zeros((B, T, H, J, Dv)) if want_resp else None
    delta = np.zeros((B, T, H, J, Dv)) if want_delta else None
    temporal = gate_k_logit is not None or gate_q_logit is not None
    dec = _f64(decay_logit)
    if dec is not None:
        assert dec.shape == (B, T, H, J, Dk)
    if unnormalized and (temporal or dec is not None):
        raise ValueError("the unnormalised variant is defined for the plain form only")
    if temporal or dec is not None or unnormalized:
        gk, gq, p_in = _f64(gate_k_logit), _f64(gate_q_logit), _f64(prior_in)
        p_out = None
        if temporal:
            assert gk is not None and gq is not None, "both gate logits are needed"
            assert gk.shape == (B, T, H, Dv) and gq.shape == (B, T, H, Dv)
            if p_in is not None:
                assert p_in.shape == (B, H, 2, J, Dv)
            p_out = np.zeros((B, H, 2, J, Dv))
        else:
            assert prior_in is None, "prior_in needs the gate logits"
        rc = (lib or _load()).swila_oracle_forward_ext(
            B, H, T, Dk, Dv, J, _ptr(q), _ptr(k), _ptr(v), _ptr(lb), _ptr(lk), _ptr(lq),
            _ptr(gk), _ptr(gq), _ptr(dec), int(bool(post_decay)), int(bool(unnormalized)),
            _ptr(s_in), _ptr(p_in),
            _ptr(s_out), _ptr(p_out), _ptr(o), _ptr(resp), _ptr(delta), int(nthreads))
    else:
        assert prior_in is None, "prior_in needs the gate logits"
        rc = (lib or _load()).swila_oracle_forward(
            B, H, T, Dk, Dv, J, _ptr(q), _ptr(k), _ptr(v), _ptr(lb), _ptr(lk), _ptr(lq),
            _ptr(s_in), _ptr(s_out), _ptr(o), _ptr(resp), _ptr(delta), int(nthreads))
    if rc != 0:
        raise FloatingPointError("oracle failed with status %d" % rc)
    out = {"o": o, "state": s_out}
    if temporal:
        out["prior"] = p_out
    if want_resp:
        out["resp"] = resp
    if want_delta:
        out["delta"] = delta
    return out


def decode_step(q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in, *,
                gate_k_logit=None, gate_q_logit=None, prior_in=None, decay_logit=None,
                nthreads: int = 0):
    """One token per sequence: q, k [B,H,Dk]; v [B,H,Dv]; logits [B,H,J,Dv];
    state_in [B,H,J,Dk,Dv].  Returns (o [B,H,Dv], state [B,H,J,Dk,Dv]), plus
    the prior state [B,H,2,J,Dv] for the temporal form (gate logits [B,H,Dv]);
    decay_logit [B,H,J,Dk] for the gated form.  This is ``forward`` with T = 1."""
    temporal = gate_k_logit is not None
    gates = {}
    if temporal:
        gates = dict(gate_k_logit=np.asarray(gate_k_logit)[:, None],
                     gate_q_logit=np.asarray(gate_q_logit)[:, None], prior_in=prior_in)
    if decay_logit is not None:
        gates["decay_logit"] = np.asarray(decay_logit)[:, None]
    r = forward(*(np.asarray(x)[:, None] for x in
                  (q, k, v, beta_logit, prior_k_logit, prior_q_logit)),
                state_in, nthreads=nthreads, **gates)
    if temporal:
        return r["o"][:, 0], r["state"], r["prior"]
    return r["o"][:, 0], r["state"]
