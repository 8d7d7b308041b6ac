"""swila_forward_noalloc (the entry point for callers that cannot allocate)
through the C ABI against swila_forward on the same inputs: two calls in a
row, the second smaller, for the App. D form (which uses the library's device
scratch array) and the exact chunk scan; a call beyond the scratch limit is
rejected before anything is enqueued.

Bar: the App. D form runs the same kernels on the same inputs, only the
scratch differs, so the outputs, final state and sweep counts must be identical;
against the oracle's bar that is within 2e-2 a fortiori."""
import numpy as np
import pytest

import workloads
from gpu_helpers import NAMES, head_rel_err, to_device

pytestmark = pytest.mark.gpu


def _both(inp, algo, **kw):
    import torch
    import paper_2609_39034_amd as sw
    dev = to_device(inp, "bf16")
    B, T, H, Dk = inp["q"].shape
    J, Dv = inp["lb"].shape[3], inp["lb"].shape[4]
    it_a = torch.full((2,), -5, dtype=torch.int32, device="cuda")
    it_b = torch.full((2,), -5, dtype=torch.int32, device="cuda")
    o_a, s_a = sw.forward(*(dev[n] for n in NAMES), dev["state"], algo=algo, iters_out=it_a, **kw)
    o_b = torch.empty((B, T, H, Dv), device="cuda", dtype=torch.bfloat16)
    s_b = torch.empty((B, H, J, Dk, Dv), device="cuda", dtype=torch.float32)
    sw.forward_noalloc(*(dev[n] for n in NAMES), dev["state"], o_b, state_out=s_b, algo=algo,
                       iters_out=it_b, **kw)
    torch.cuda.synchronize()
    return o_a, s_a, it_a, o_b, s_b, it_b


@pytest.mark.parametrize("algo", ["newton", "chunk"])
def test_noalloc_matches_forward_twice(algo):
    import torch
    kw = dict(max_iters=64, tol=1e-3) if algo == "newton" else {}
    for shape, seed in (((2, 4, 300, 64, 64, 4), 900), ((1, 2, 70, 32, 32, 4), 901)):
        inp = workloads.iid_inputs(*shape, dtype="bf16", seed=seed, state_std=0.1)
        o_a, s_a, it_a, o_b, s_b, it_b = _both(inp, algo, **kw)
        eo = head_rel_err(o_b.float().cpu().numpy(), o_a.float().cpu().numpy(), "o")
        es = head_rel_err(s_b.cpu().numpy(), s_a.cpu().numpy(), "state")
        print("%s %s: o %.3e state %.3e sweeps %s / %s" % (algo, shape, eo, es,
                                                           it_a.tolist(), it_b.tolist()))
        assert torch.equal(o_a, o_b) and torch.equal(s_a, s_b)
        if algo == "newton":
            assert torch.equal(it_a, it_b) and int(it_a[1]) == 0


def test_noalloc_rejects_beyond_scratch():
    import torch
    import paper_2609_39034_amd as sw
    # B*H*J*Dv*16*ceil(T/16)*4 = 4*8*4*64*2064*4 > 64 MiB: rejected before any launch
    inp = workloads.iid_inputs(4, 8, 2050, 64, 64, 4, dtype="bf16", seed=902)
    dev = to_device(inp, "bf16")
    o = torch.empty((4, 2050, 8, 64), device="cuda", dtype=torch.bfloat16)
    with pytest.raises(sw.SwilaError) as e:
        sw.forward_noalloc(*(dev[n] for n in NAMES), None, o, algo="newton")
    assert e.value.code == sw.EUNSUPPORTED and "scratch" in str(e.value)
    # the largest call within the limit (exactly 64 MiB of predictions) runs
    inp = workloads.iid_inputs(4, 8, 2048, 64, 64, 4, dtype="bf16", seed=903)
    dev = to_device(inp, "bf16")
    o = torch.empty((4, 2048, 8, 64), device="cuda", dtype=torch.bfloat16)
    it = torch.zeros(2, dtype=torch.int32, device="cuda")
    sw.forward_noalloc(*(dev[n] for n in NAMES), None, o, algo="newton", iters_out=it, tol=1e-3,
                       max_iters=64)
    o_ref, _ = sw.forward(*(dev[n] for n in NAMES), None, algo="newton", tol=1e-3, max_iters=64)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and int(it[1]) == 0
    assert np.isfinite(o.float().cpu().numpy()).all()
