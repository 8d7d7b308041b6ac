"""Seeded synthetic inputs for the SwiLA layer.

This module only draws and lays out inputs; it holds none of the method's
arithmetic.  Both the GPU path (tests, benchmark) and the fp64 oracle consume
exactly the values produced here: bf16 inputs are returned as float32 arrays
whose every value is exactly representable in bf16 (round-to-nearest-even is
applied here, once), so converting them to bfloat16 or to float64 is exact.

Layouts (row-major):
  q, k   [B, T, H, Dk]        v  [B, T, H, Dv]
  lb, lk, lq (beta logit, key-prior logits, query-prior logits) [B, T, H, J, Dv]
  state  [B, H, J, Dk, Dv]    element (b,h,j,i,d) is weight i of component j
                              for output dimension d

Workload recipes (the five standard configurations):
  1 tiny      B=1  H=1  T=64     D=16  J=2  fp32  i.i.d. N(0,1), k L2-normalised
  2 small     B=4  H=8  T=2048   D=64  J=4  bf16  same draws
  3 lm        B=8  H=16 T=4096   D=128 J=4  bf16  N(0,1) projections of random
              token embeddings (vocabulary 32000, width 1024)
  4 decode    B=256 H=16 D=128 J=4, 512 one-token steps, bf16 N(0,1) inputs,
              fp32 initial state N(0, 0.1^2)
  5 recall    B=2  H=8  T=16384  D=128 J=8  bf16  projections of a token stream in
              which 1024 key/value tokens per sequence recur at random offsets
              and later occurrences query the stored key
Seeds default to 1000 + configuration number; draw order q, k, v, lb, lk, lq,
state.
"""
from __future__ import annotations

import numpy as np

CONFIGS = {
    1: dict(name="tiny", B=1, H=1, T=64, Dk=16, Dv=16, J=2, dtype="f32", kind="iid"),
    2: dict(name="small", B=4, H=8, T=2048, Dk=64, Dv=64, J=4, dtype="bf16", kind="iid"),
    3: dict(name="lm", B=8, H=16, T=4096, Dk=128, Dv=128, J=4, dtype="bf16", kind="lm"),
    4: dict(name="decode", B=256, H=16, T=1, Dk=128, Dv=128, J=4, dtype="bf16",
            kind="decode", steps=512, state_std=0.1),
    5: dict(name="recall", B=2, H=8, T=16384, Dk=128, Dv=128, J=8, dtype="bf16", kind="recall"),
}

NAMES = ("q", "k", "v", "lb", "lk", "lq")


def round_bf16_reference(x):
    """Round float32 values to the nearest bfloat16 (ties to even) by bit
    arithmetic; the result is returned as float32.  Inputs must be finite."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def round_bf16(x):
    """Round float32 values to the nearest bfloat16 (ties to even), returned as
    float32: torch's multi-threaded conversion, which the tests check against
    ``round_bf16_reference``."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _finish(x, dtype):
    if not isinstance(x, np.ndarray):          # a CPU torch tensor
        import torch
        x = x.contiguous()
        if dtype == "bf16":
            x = x.to(torch.bfloat16).to(torch.float32)
        return x.numpy()
    x = np.ascontiguousarray(x, dtype=np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def _l2norm_last(x):
    if not isinstance(x, np.ndarray):          # a CPU torch tensor
        import torch
        n = x.to(torch.float64).pow(2).sum(dim=-1, keepdim=True).sqrt().clamp_min(1e-12)
        return (x / n).to(torch.float32)
    n = np.sqrt((x.astype(np.float64) ** 2).sum(axis=-1, keepdims=True))
    return (x / np.maximum(n, 1e-12)).astype(np.float32)


def iid_inputs(B, H, T, Dk, Dv, J, *, dtype="bf16", seed=0, state_std=0.0,
               normalize_k=True, logit_scale=1.0):
    """Independent N(0,1) draws; k L2-normalised per (b, t, h) before rounding.
    Returns a dict with q, k, v, lb, lk, lq and ``state`` (None when
    state_std == 0, i.e. a zero initial state)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    q = rng.standard_normal((B, T, H, Dk), dtype=np.float32)
    k = rng.standard_normal((B, T, H, Dk), dtype=np.float32)
    v = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    lb = rng.standard_normal((B, T, H, J, Dv), dtype=np.float32) * np.float32(logit_scale)
    lk = rng.standard_normal((B, T, H, J, Dv), dtype=np.float32) * np.float32(logit_scale)
    lq = rng.standard_normal((B, T, H, J, Dv), dtype=np.float32) * np.float32(logit_scale)
    state = None
    if state_std > 0:
        state = (rng.standard_normal((B, H, J, Dk, Dv), dtype=np.float32)
                 * np.float32(state_std))
    if normalize_k:
        k = _l2norm_last(k)
    out = {n: _finish(x, dtype) for n, x in zip(NAMES, (q, k, v, lb, lk, lq))}
    out["state"] = state
    return out


def temporal_inputs(B, H, T, Dv, J, *, dtype="bf16", seed=0, gate_scale=1.0,
                    prior_state=False):
    """Extra inputs of Temporal SwiLA: the key- and query-side gate logits
    ``gk``, ``gq`` [B, T, H, Dv], i.i.d. N(0, gate_scale^2) (rounded like the
    other inputs), and, when ``prior_state`` is set, a carried prior state
    ``prior`` [B, H, 2, J, Dv] fp32 whose two parts are probability vectors
    over J (normalised exponentials of N(0,1) draws).  Drawn from their own
    generator, so the base inputs of the same seed are unchanged."""
    rng = np.random.Generator(np.random.PCG64(seed + 7919))
    gk = rng.standard_normal((B, T, H, Dv), dtype=np.float32) * np.float32(gate_scale)
    gq = rng.standard_normal((B, T, H, Dv), dtype=np.float32) * np.float32(gate_scale)
    out = {"gk": _finish(gk, dtype), "gq": _finish(gq, dtype), "prior": None}
    if prior_state:
        e = np.exp(rng.standard_normal((B, H, 2, J, Dv)))
        out["prior"] = (e / e.sum(axis=3, keepdims=True)).astype(np.float32)
    return out


def gated_inputs(B, H, T, Dk, J, *, dtype="bf16", seed=0, mean=2.0, scale=1.0):
    """Extra input of Gated SwiLA: decay logits ``decay`` [B, T, H, J, Dk],
    i.i.d. N(mean, scale^2) (sigmoid(2) = 0.88 keeps most of the state per
    token), rounded like the other inputs.  Drawn from their own generator."""
    rng = np.random.Generator(np.random.PCG64(seed + 104729))
    d = rng.standard_normal((B, T, H, J, Dk), dtype=np.float32) * np.float32(scale) + np.float32(mean)
    return {"decay": _finish(d, dtype)}


def _project_tokens(rng, ids, vocab, width, H, Dk, Dv, J, dtype, chunk_tokens=4096):
    """q, k, v and the three logit tensors as linear projections of random token
    embeddings E ~ N(0,1) [vocab, width] with weights N(0, 1/width), so every
    projected value is close to N(0,1).  ids: [B, T] integer token ids.
    Returns CPU torch float32 tensors."""
    import torch
    B, T = ids.shape
    E = torch.from_numpy(rng.standard_normal((vocab, width), dtype=np.float32))
    widths = [H * Dk, H * Dk, H * Dv, H * J * Dv, H * J * Dv, H * J * Dv]
    scale = np.float32(1.0 / np.sqrt(width))
    thetas = [torch.from_numpy(rng.standard_normal((width, w), dtype=np.float32) * scale)
              for w in widths]
    shapes = [(B, T, H, Dk), (B, T, H, Dk), (B, T, H, Dv),
              (B, T, H, J, Dv), (B, T, H, J, Dv), (B, T, H, J, Dv)]
    outs = [torch.empty((B * T, w), dtype=torch.float32) for w in widths]
    flat_ids = torch.from_numpy(ids.reshape(-1))
    for a in range(0, flat_ids.numel(), chunk_tokens):
        sl = slice(a, min(a + chunk_tokens, flat_ids.numel()))
        X = E[flat_ids[sl]]
        for o, th in zip(outs, thetas):
            torch.matmul(X, th, out=o[sl])
    return [o.reshape(s) for o, s in zip(outs, shapes)]


def lm_inputs(B=8, H=16, T=4096, Dk=128, Dv=128, J=4, *, dtype="bf16", seed=1003,
              vocab=32000, width=1024):
    """LM-shaped forward inputs: token ids uniform over the vocabulary, N(0,1)
    embeddings projected by random N(0, 1/width) weights; k L2-normalised per
    (token, head)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ids = rng.integers(0, vocab, size=(B, T))
    q, k, v, lb, lk, lq = _project_tokens(rng, ids, vocab, width, H, Dk, Dv, J, dtype)
    k = _l2norm_last(k)
    out = {n: _finish(x, dtype) for n, x in zip(NAMES, (q, k, v, lb, lk, lq))}
    out["state"] = None
    return out


def recall_inputs(B=2, H=8, T=16384, Dk=128, Dv=128, J=8, *, dtype="bf16", seed=1005,
                  vocab=8192, width=1024, pairs=1024, repeats=8, query_noise=0.1):
    """Recall-shaped long-context inputs.  Per sequence, ``pairs`` distinct token
    ids each recur at ``repeats`` random positions (the rest are random filler
    tokens); every token's q, k, v and logits are projections of its embedding,
    so recurring tokens carry the same key, value and logits.  At the second and
    later occurrences of a pair token, the query is that token's normalised key
    plus ``query_noise`` * N(0,1), so those positions query a stored key."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ids = rng.integers(0, vocab, size=(B, T))
    occ = np.zeros((B, T), dtype=bool)          # a later occurrence of a pair token
    for b in range(B):
        pair_ids = rng.choice(vocab, size=pairs, replace=False)
        pos = rng.choice(T, size=pairs * repeats, replace=False).reshape(pairs, repeats)
        pos.sort(axis=1)
        for p in range(pairs):
            ids[b, pos[p]] = pair_ids[p]
            occ[b, pos[p, 1:]] = True
    import torch
    q, k, v, lb, lk, lq = _project_tokens(rng, ids, vocab, width, H, Dk, Dv, J, dtype)
    k = _l2norm_last(k)
    noise = torch.from_numpy(rng.standard_normal((B, T, H, Dk), dtype=np.float32)
                             * np.float32(query_noise))
    q = torch.where(torch.from_numpy(occ)[:, :, None, None], k + noise, q)
    out = {n: _finish(x, dtype) for n, x in zip(NAMES, (q, k, v, lb, lk, lq))}
    out["state"] = None
    return out


def config_inputs(cfg, seed=None):
    """Inputs of standard configuration ``cfg`` (1, 2, 3 or 5; decode inputs for
    configuration 4 come from ``decode_initial_state`` and ``decode_step_inputs``)."""
    c = CONFIGS[cfg]
    seed = 1000 + cfg if seed is None else seed
    if c["kind"] == "iid":
        return iid_inputs(c["B"], c["H"], c["T"], c["Dk"], c["Dv"], c["J"],
                          dtype=c["dtype"], seed=seed)
    if c["kind"] == "lm":
        return lm_inputs(c["B"], c["H"], c["T"], c["Dk"], c["Dv"], c["J"],
                         dtype=c["dtype"], seed=seed)
    if c["kind"] == "recall":
        return recall_inputs(c["B"], c["H"], c["T"], c["Dk"], c["Dv"], c["J"],
                             dtype=c["dtype"], seed=seed)
    raise ValueError("configuration %d has no whole-sequence inputs" % cfg)


def decode_initial_state(B=256, H=16, Dk=128, Dv=128, J=4, *, std=0.1, seed=1004):
    """fp32 initial states N(0, std^2), [B, H, J, Dk, Dv]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.standard_normal((B, H, J, Dk, Dv), dtype=np.float32) * np.float32(std)


def decode_step_inputs_torch(step, B=256, H=16, Dk=128, Dv=128, J=4, *, seed=1004,
                             device="cuda", dtype=None):
    """Fresh N(0,1) inputs of one decode step, drawn with torch's counter-based
    generator on ``device`` (seeded by seed and step, so any step can be redrawn);
    k L2-normalised in fp32 before rounding.  Returns a dict of tensors with
    q, k [B,H,Dk], v [B,H,Dv], lb, lk, lq [B,H,J,Dv]."""
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1_000_003 + int(step))
    f = dict(device=device, dtype=torch.float32, generator=g)
    q = torch.randn((B, H, Dk), **f)
    k = torch.randn((B, H, Dk), **f)
    v = torch.randn((B, H, Dv), **f)
    lb = torch.randn((B, H, J, Dv), **f)
    lk = torch.randn((B, H, J, Dv), **f)
    lq = torch.randn((B, H, J, Dv), **f)
    k = k / k.norm(dim=-1, keepdim=True).clamp_min(1e-12)
    return {n: x.to(dtype) for n, x in zip(NAMES, (q, k, v, lb, lk, lq))}


def to_torch(inputs, device, dtype):
    """Move a dict of float32 arrays (values exact in ``dtype``) to ``device``."""
    import torch
    out = {}
    for n in NAMES:
        out[n] = torch.from_numpy(np.ascontiguousarray(inputs[n])).to(device=device, dtype=dtype)
    st = inputs.get("state")
    out["state"] = None if st is None else torch.from_numpy(np.ascontiguousarray(st)).to(device)
    return out
