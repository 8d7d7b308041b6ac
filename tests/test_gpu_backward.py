"""Parity of the backward pass (swila_backward, the exact gradient of the plain
forward of Sec. 3.2) through the C ABI with the fp64 gradient oracle.

Bar as for the forward: per (b, h), max|gpu - oracle| / max|oracle| <= 1e-4
for fp32 inputs and <= 2e-2 for bf16 inputs, on every gradient (q, k, v, the
three logit tensors and the initial state).
"""
import numpy as np
import pytest

import oracle.backward as ob
import workloads
from gpu_helpers import NAMES, head_rel_err, to_device, tol_for, torch_dtype

pytestmark = pytest.mark.gpu

GRADS = ("q", "k", "v", "lb", "lk", "lq")
KIND = {"q": "o", "k": "o", "v": "o", "lb": "resp", "lk": "resp", "lq": "resp"}


def _seeds(B, H, T, Dv, Dk, J, dtype, seed, with_gs):
    """dL/do (rounded to the output dtype) and dL/dW_T (or None)."""
    import torch
    rng = np.random.default_rng(seed + 17)
    go = rng.standard_normal((B, T, H, Dv)).astype(np.float32)
    go_dev = torch.from_numpy(go).to("cuda", torch_dtype(dtype))
    go = go_dev.float().cpu().numpy().astype(np.float64)
    gs = None
    if with_gs:
        gs = rng.standard_normal((B, H, J, Dk, Dv)).astype(np.float32)
    return go_dev, go, gs


def _run(B, H, T, Dk, Dv, J, dtype, std, with_gs, seed, heads=None):
    import torch
    import paper_2609_39034_amd as sw
    inp = workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype=dtype, seed=seed, state_std=std)
    dev = to_device(inp, dtype)
    go_dev, go, gs = _seeds(B, H, T, Dv, Dk, J, dtype, seed, with_gs)
    gs_dev = None if gs is None else torch.from_numpy(gs).cuda()
    res = sw.backward(*(dev[n] for n in NAMES), dev["state"], go_dev, gs_dev)
    torch.cuda.synchronize()
    got = dict(zip(GRADS + ("state",), (x.cpu().numpy().astype(np.float64) for x in res)))
    if heads is None:
        ref = ob.backward(*(inp[n] for n in NAMES), inp["state"], go, gs)
        return got, ref
    errs = {}
    for b, h in heads:
        sub = [inp[n][b:b + 1, :, h:h + 1] for n in NAMES]
        st = None if inp["state"] is None else inp["state"][b:b + 1, h:h + 1]
        g1 = None if gs is None else gs[b:b + 1, h:h + 1]
        ref = ob.backward(*sub, st, go[b:b + 1, :, h:h + 1], g1)
        for n in GRADS:
            e = head_rel_err(got[n][b:b + 1, :, h:h + 1], ref[n], KIND[n])
            errs[n] = max(errs.get(n, 0.0), e)
        e = head_rel_err(got["state"][b:b + 1, h:h + 1], ref["state"], "state")
        errs["state"] = max(errs.get("state", 0.0), e)
    return errs


def _errs(got, ref):
    e = {n: head_rel_err(got[n], ref[n], KIND[n]) for n in GRADS}
    e["state"] = head_rel_err(got["state"], ref["state"], "state")
    return e


CASES = [
    # B, H, T, Dk, Dv, J, dtype, state_std, grad_state
    (1, 1, 64, 16, 16, 2, "f32", 0.0, False),
    (2, 3, 50, 64, 64, 4, "f32", 0.3, True),       # a ragged second chunk
    (2, 2, 77, 128, 128, 4, "bf16", 0.1, True),    # three chunks, ragged
    (1, 2, 33, 128, 64, 8, "f32", 0.2, False),
    (2, 1, 17, 32, 16, 3, "f32", 0.5, True),       # J = 3: tiles of 12 columns
    (1, 3, 21, 16, 32, 1, "f32", 0.5, True),
    (3, 1, 40, 64, 32, 2, "bf16", 0.0, False),
    (1, 1, 1, 128, 128, 4, "f32", 0.2, True),      # one token
    (2, 2, 96, 32, 128, 8, "bf16", 0.1, True),
    (1, 2, 130, 64, 64, 4, "f32", 0.1, True),      # five chunks, two staging rounds each
    (1, 2, 45, 32, 16, 1, "f32", 0.2, True),       # reverse blocks of 8 dims, half a tile
    (2, 1, 70, 64, 16, 2, "bf16", 0.1, False),     # the same with two components
    (1, 2, 75, 64, 32, 3, "bf16", 0.2, True),      # J = 3 on the matrix cores: padded columns
    (2, 1, 40, 16, 32, 4, "bf16", 0.0, True),      # Dk = 16: dq, dk tiles on two waves
]


@pytest.mark.parametrize("B,H,T,Dk,Dv,J,dtype,std,gs", CASES)
def test_backward(B, H, T, Dk, Dv, J, dtype, std, gs):
    got, ref = _run(B, H, T, Dk, Dv, J, dtype, std, gs, seed=700 + T + J)
    e = _errs(got, ref)
    tol = tol_for(dtype)
    print(" ".join("%s %.2e" % kv for kv in e.items()), "(tol %.0e)" % tol)
    assert all(v <= tol for v in e.values()), e


@pytest.mark.parametrize("dtype,go_dtype", [("bf16", "f32"), ("f32", "bf16")])
def test_backward_grad_o_dtype_differs(dtype, go_dtype):
    """dL/do in the other dtype than the inputs (it carries the forward's output
    dtype): the gradients against the oracle fed the same rounded dL/do."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, T, Dk, Dv, J = 2, 2, 37, 64, 32, 4
    inp = workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype=dtype, seed=731, state_std=0.1)
    dev = to_device(inp, dtype)
    rng = np.random.default_rng(732)
    go_dev = torch.from_numpy(rng.standard_normal((B, T, H, Dv)).astype(np.float32)).to(
        "cuda", torch_dtype(go_dtype))
    go = go_dev.float().cpu().numpy().astype(np.float64)
    res = sw.backward(*(dev[n] for n in NAMES), dev["state"], go_dev, None)
    torch.cuda.synchronize()
    got = dict(zip(GRADS + ("state",), (x.cpu().numpy().astype(np.float64) for x in res)))
    ref = ob.backward(*(inp[n] for n in NAMES), inp["state"], go, None)
    e = _errs(got, ref)
    tol = tol_for(dtype)
    print(" ".join("%s %.2e" % kv for kv in e.items()), "(tol %.0e)" % tol)
    assert all(v <= tol for v in e.values()), e


def test_backward_empty_sequence():
    """T = 0: dL/dW_0 = dL/dW_T; nothing else is written."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, D, J = 2, 2, 32, 4
    z = lambda *s: torch.zeros(*s, device="cuda")
    gs = torch.randn(B, H, J, D, D, device="cuda")
    res = sw.backward(z(B, 0, H, D), z(B, 0, H, D), z(B, 0, H, D), z(B, 0, H, J, D),
                      z(B, 0, H, J, D), z(B, 0, H, J, D), None, z(B, 0, H, D), gs)
    torch.cuda.synchronize()
    assert torch.equal(res[-1], gs)
    res = sw.backward(z(B, 0, H, D), z(B, 0, H, D), z(B, 0, H, D), z(B, 0, H, J, D),
                      z(B, 0, H, J, D), z(B, 0, H, J, D), None, z(B, 0, H, D), None)
    torch.cuda.synchronize()
    assert float(res[-1].abs().max()) == 0.0


def test_backward_frozen_state():
    """beta = 0 (logit -800): the state never moves, so the key, value, beta and
    key-prior gradients are exactly zero."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, T, D, J = 2, 2, 45, 64, 4
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="f32", seed=91, state_std=0.3)
    dev = to_device(inp, "f32")
    dev["lb"] = torch.full_like(dev["lb"], -800.0)
    go = torch.randn(B, T, H, D, device="cuda")
    dq, dk, dv, dlb, dlk, dlq, ds = sw.backward(*(dev[n] for n in NAMES), dev["state"], go)
    torch.cuda.synchronize()
    for x in (dk, dv, dlb, dlk):
        assert float(x.abs().max()) == 0.0
    assert float(dq.abs().max()) > 0.0


def test_backward_config2_every_head():
    """The standard bf16 training batch (B=4 H=8 T=2048 Dk=Dv=64 J=4, zero initial
    state) as the benchmark runs it; the oracle on every (b, h), one after another
    (about 0.7 s each), the worst error over the heads per gradient."""
    c = workloads.CONFIGS[2]
    heads = [(b, h) for b in range(c["B"]) for h in range(c["H"])]
    errs = _run(c["B"], c["H"], c["T"], c["Dk"], c["Dv"], c["J"], "bf16", 0.0, False,
                seed=1002, heads=heads)
    print(" ".join("%s %.2e" % kv for kv in errs.items()))
    assert all(v <= 2e-2 for v in errs.values()), errs


def test_backward_lm_batch_sampled_head():
    """The LM-shaped batch (B=8 H=16 T=4096 Dk=Dv=128 J=4, bf16; 128 chunks of 32
    tokens and 64-lane reverse blocks), the oracle on one sampled head (the
    oracle keeps every token's state: about 2 GB at this size)."""
    import torch
    import paper_2609_39034_amd as sw
    c = workloads.CONFIGS[3]
    B, H, T, Dk, Dv, J = (c[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    inp = workloads.config_inputs(3)
    dev = to_device(inp, "bf16")
    go_dev, go, _ = _seeds(B, H, T, Dv, Dk, J, "bf16", 1003, False)
    res = sw.backward(*(dev[n] for n in NAMES), None, go_dev, None)
    torch.cuda.synchronize()
    b, h = 5, 11
    got = [x[b:b + 1, :, h:h + 1].cpu().numpy().astype(np.float64) for x in res[:6]]
    ref = ob.backward(*(inp[n][b:b + 1, :, h:h + 1] for n in NAMES), None,
                      go[b:b + 1, :, h:h + 1], None)
    errs = {n: head_rel_err(g, ref[n], KIND[n]) for n, g in zip(GRADS, got)}
    errs["state"] = head_rel_err(res[6][b:b + 1, h:h + 1].cpu().numpy(), ref["state"], "state")
    print(" ".join("%s %.2e" % kv for kv in errs.items()))
    assert all(v <= 2e-2 for v in errs.values()), errs
