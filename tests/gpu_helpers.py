"""Helpers for GPU parity tests: move seeded inputs to the device, run the
library, and measure the error against the fp64 oracle per (b, h)."""
from __future__ import annotations

import numpy as np

import workloads

NAMES = workloads.NAMES
TOL_F32 = 1e-4     # fp32 inputs
TOL_BF16 = 2e-2    # bf16 inputs, fp32 state and accumulation


def tol_for(dtype):
    return TOL_F32 if dtype == "f32" else TOL_BF16


def torch_dtype(dtype):
    import torch
    return torch.float32 if dtype == "f32" else torch.bfloat16


def to_device(inp, dtype, device="cuda"):
    return workloads.to_torch(inp, device, torch_dtype(dtype))


def gpu_forward(inp, dtype, *, out_dtype=None, resp=False, state_out=True, algo="auto"):
    import paper_2609_39034_amd as sw
    import torch
    dev = to_device(inp, dtype)
    od = None if out_dtype is None else torch_dtype(out_dtype)
    res = sw.forward(*(dev[n] for n in NAMES), dev["state"], out_dtype=od, resp=resp,
                     state_out=state_out, algo=algo)
    torch.cuda.synchronize()
    return [None if x is None else x.float().cpu().numpy().astype(np.float64) for x in res]


def head_rel_err(x, y, kind):
    """max |x - y| / max(max |y|, 1e-6) per (b, h); ``kind`` is 'o'
    ([B,T,H,Dv]), 'state' ([B,H,J,Dk,Dv]) or 'resp' ([B,T,H,J,Dv]).  Returns the
    worst head's value."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    assert x.shape == y.shape, (x.shape, y.shape)
    if kind == "o":
        xs, ys = np.moveaxis(x, 2, 1), np.moveaxis(y, 2, 1)   # [B,H,T,Dv]
    elif kind == "resp":
        xs, ys = np.moveaxis(x, 2, 1), np.moveaxis(y, 2, 1)   # [B,H,T,J,Dv]
    else:
        xs, ys = x, y
    B, H = xs.shape[:2]
    xs = xs.reshape(B, H, -1)
    ys = ys.reshape(B, H, -1)
    num = np.abs(xs - ys).max(axis=2) if xs.shape[2] else np.zeros((B, H))
    den = np.maximum(np.abs(ys).max(axis=2) if ys.shape[2] else np.zeros((B, H)), 1e-6)
    return float((num / den).max())


def range_edge_inputs(case, seed, B=1, H=2, T=40, Dk=64, Dv=32, J=4):
    """bf16 inputs that put the E-step's softmax sum at the edges of the fp32
    range.  Keys are distinct signed basis vectors (orthonormal, exact in bf16,
    T <= Dk), so every update is orthogonal to the later keys and the prediction
    of token t is exactly W_0[j, :, d] . k_t: the errors delta_tjd are set
    through W_0.
      "band":   the largest e^{-delta^2/2} of each (t, d) lies in
                [2^-125, 2^-111] (|delta| in [12.4, 13.1]) and the other
                components are 0.02 to 2 higher in |delta|, so many of their
                terms fall below 2^-126 while their r is far from 0; equal
                key-prior logits.
      "logits": one component's key-prior logit is 86 to 88 and its |delta|
                below 1.5, so the sum reaches 2^124 .. 2^127 and its
                reciprocal is at or below the smallest normal fp32.
    Returns the dict of ``workloads.iid_inputs`` (state = W_0)."""
    assert T <= Dk
    rng = np.random.Generator(np.random.PCG64(seed))
    f32 = np.float32
    q = workloads.round_bf16(rng.standard_normal((B, T, H, Dk), dtype=f32))
    lb = workloads.round_bf16(rng.standard_normal((B, T, H, J, Dv), dtype=f32))
    lq = workloads.round_bf16(rng.standard_normal((B, T, H, J, Dv), dtype=f32))
    k = np.zeros((B, T, H, Dk), f32)
    W0 = (rng.standard_normal((B, H, J, Dk, Dv)) * 0.1).astype(f32)
    v = np.zeros((B, T, H, Dv), f32)
    lk = np.zeros((B, T, H, J, Dv), f32)
    for b in range(B):
        for h in range(H):
            perm = rng.permutation(Dk)[:T]
            sgn = rng.choice([-1.0, 1.0], size=T)
            for t in range(T):
                k[b, t, h, perm[t]] = sgn[t]
                lead = rng.integers(0, J, size=Dv)
                if case == "band":
                    vt = workloads.round_bf16(rng.choice([-1.0, 1.0], size=Dv) *
                                              rng.uniform(6.0, 10.0, size=Dv).astype(f32))
                    dl = rng.uniform(12.4, 13.1, size=Dv)
                    mag = dl[None, :] + rng.uniform(0.02, 2.0, size=(J, Dv))
                    mag[lead, np.arange(Dv)] = dl
                else:
                    vt = workloads.round_bf16(rng.standard_normal(Dv).astype(f32))
                    mag = rng.uniform(0.0, 1.5, size=(J, Dv))
                    lt = rng.standard_normal((J, Dv)).astype(f32)
                    lt[lead, np.arange(Dv)] = rng.choice([86.0, 86.5, 87.0, 87.5, 88.0], size=Dv)
                    lk[b, t, h] = workloads.round_bf16(lt)
                delta = rng.choice([-1.0, 1.0], size=(J, Dv)) * mag
                v[b, t, h] = vt
                # pred_tjd = sgn_t W0[j, perm_t, d] = v_td - delta_tjd
                W0[b, h, :, perm[t], :] = ((vt[None, :] - delta) * sgn[t]).astype(f32)
    return {"q": q, "k": k, "v": v, "lb": lb, "lk": lk, "lq": lq, "state": W0}
