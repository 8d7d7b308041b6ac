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
