"""Parity of the Gated SwiLA path (Sec. 3.4, App. B.4, eq. pre-decay with one
gate per key dimension) through the C ABI with the fp64 oracle: the
token-by-token scan and the decode step, alone and with the temporal priors.

Bar as for the plain form: per (b, h), max|gpu - oracle| / max|oracle| <= 1e-4
for fp32 inputs and <= 2e-2 for bf16 inputs (outputs, final state,
responsibilities, prior state).
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_helpers import NAMES, head_rel_err, to_device, tol_for, torch_dtype

pytestmark = pytest.mark.gpu


def _t(x, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda", torch_dtype(dtype))


CASES = [
    # B, H, T, Dk, Dv, J, dtype, state_std, temporal, decay mean
    (1, 1, 64, 16, 16, 2, "f32", 0.0, False, 2.0),
    (2, 3, 50, 64, 128, 4, "f32", 0.3, False, 1.0),
    (2, 2, 37, 128, 128, 4, "bf16", 0.1, False, 2.0),
    (1, 2, 33, 128, 64, 8, "f32", 0.2, True, 2.0),
    (2, 1, 17, 32, 16, 3, "f32", 0.5, False, 0.0),
    (1, 3, 21, 16, 32, 1, "f32", 0.5, True, 3.0),
    (3, 1, 40, 64, 32, 2, "bf16", 0.0, True, 2.0),
    (1, 1, 1, 128, 128, 4, "f32", 0.2, False, 2.0),
    (2, 2, 16, 32, 128, 8, "bf16", 0.1, False, 1.0),
    # 256 heads: grids of at least 256 blocks keep 16 (J <= 4) or 8 key rows per
    # lane; the grids above have fewer blocks and take 4 rows per lane
    (16, 16, 21, 64, 64, 4, "bf16", 0.1, False, 2.0),
    (16, 16, 18, 64, 64, 4, "f32", 0.2, True, 2.0),
    (8, 32, 19, 128, 128, 8, "bf16", 0.1, False, 2.0),
    # J = 16 (J * Dk <= 1024: its gate tile fits LDS)
    (1, 2, 37, 64, 64, 16, "f32", 0.1, False, 2.0),
    (2, 1, 20, 16, 32, 16, "bf16", 0.2, True, 1.0),
]


@pytest.mark.parametrize("B,H,T,Dk,Dv,J,dtype,std,temporal,mean", CASES)
def test_gated_forward(B, H, T, Dk, Dv, J, dtype, std, temporal, mean):
    import torch
    import paper_2609_39034_amd as sw
    seed = 400 + T + J
    inp = workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype=dtype, seed=seed, state_std=std)
    dec = workloads.gated_inputs(B, H, T, Dk, J, dtype=dtype, seed=seed, mean=mean)["decay"]
    dev = to_device(inp, dtype)
    kw, okw = {}, {}
    if temporal:
        tmp = workloads.temporal_inputs(B, H, T, Dv, J, dtype=dtype, seed=seed, prior_state=True)
        kw = dict(gate_k_logit=_t(tmp["gk"], dtype), gate_q_logit=_t(tmp["gq"], dtype),
                  prior_in=torch.from_numpy(tmp["prior"]).cuda())
        okw = dict(gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"], prior_in=tmp["prior"])
    res = sw.forward_gated(*(dev[n] for n in NAMES), _t(dec, dtype), dev["state"], resp=True, **kw)
    torch.cuda.synchronize()
    res = [x.float().cpu().numpy().astype(np.float64) for x in res]
    ref = oracle.forward(*(inp[n] for n in NAMES), inp["state"], decay_logit=dec, want_resp=True,
                         **okw)
    tol = tol_for(dtype)
    eo, es = head_rel_err(res[0], ref["o"], "o"), head_rel_err(res[1], ref["state"], "state")
    er = head_rel_err(res[-1], ref["resp"], "resp")
    ep = float(np.abs(res[2] - ref["prior"]).max()) if temporal else 0.0
    print("o %.3e state %.3e resp %.3e prior %.3e (tol %.0e)" % (eo, es, er, ep, tol))
    assert eo <= tol and es <= tol and er <= tol and ep <= tol


def test_gated_saturated_equals_plain():
    """A decay gate at 1 (logit 40) gives the plain recurrence."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, T, D, J = 2, 2, 45, 64, 4
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="f32", seed=79, state_std=0.2)
    dev = to_device(inp, "f32")
    dec = torch.full((B, T, H, J, D), 40.0, device="cuda")
    o_g, s_g = sw.forward_gated(*(dev[n] for n in NAMES), dec, dev["state"])
    o_p, s_p = sw.forward(*(dev[n] for n in NAMES), dev["state"], algo="recurrent")
    torch.cuda.synchronize()
    eo = head_rel_err(o_g.cpu().numpy(), o_p.cpu().numpy().astype(np.float64), "o")
    es = head_rel_err(s_g.cpu().numpy(), s_p.cpu().numpy().astype(np.float64), "state")
    print("o %.3e state %.3e" % (eo, es))
    assert eo <= 1e-6 and es <= 1e-6


DECODE = [
    # B, H, Dk, Dv, J, dtype, steps, temporal
    (4, 3, 64, 64, 4, "f32", 3, False),
    (3, 2, 128, 128, 4, "bf16", 4, True),
    (2, 2, 32, 16, 3, "f32", 3, True),
    (2, 1, 16, 32, 8, "bf16", 2, False),
    (5, 2, 128, 64, 1, "f32", 2, False),
    (2, 2, 128, 128, 16, "bf16", 3, True),
    (3, 1, 64, 32, 16, "f32", 2, False),
]


@pytest.mark.parametrize("B,H,Dk,Dv,J,dtype,steps,temporal", DECODE)
def test_gated_decode_steps(B, H, Dk, Dv, J, dtype, steps, temporal):
    """Consecutive gated decode steps, state (and prior state) in place, equal the
    oracle's forward over those tokens."""
    import torch
    import paper_2609_39034_amd as sw
    seed = 600 + Dk + J
    inp = workloads.iid_inputs(B, H, steps, Dk, Dv, J, dtype=dtype, seed=seed, state_std=0.1)
    dec = workloads.gated_inputs(B, H, steps, Dk, J, dtype=dtype, seed=seed)["decay"]
    dev = to_device(inp, dtype)
    st = dev["state"].clone()
    okw = {}
    pr = None
    if temporal:
        tmp = workloads.temporal_inputs(B, H, steps, Dv, J, dtype=dtype, seed=seed,
                                        prior_state=True)
        pr = torch.from_numpy(tmp["prior"]).cuda()
        okw = dict(gate_k_logit=tmp["gk"], gate_q_logit=tmp["gq"], prior_in=tmp["prior"])
    outs = []
    for t in range(steps):
        x = [dev[n][:, t].contiguous() for n in NAMES]
        kw = {}
        if temporal:
            kw = dict(gate_k_logit=_t(tmp["gk"][:, t], dtype), gate_q_logit=_t(tmp["gq"][:, t], dtype),
                      prior_in=pr)
        res = sw.decode_step_gated(*x, _t(dec[:, t], dtype), st, **kw)
        outs.append(res[0].float())
    torch.cuda.synchronize()
    ref = oracle.forward(*(inp[n] for n in NAMES), inp["state"], decay_logit=dec, **okw)
    o = torch.stack(outs, dim=1).cpu().numpy()
    tol = tol_for(dtype)
    eo, es = head_rel_err(o, ref["o"], "o"), head_rel_err(st.cpu().numpy(), ref["state"], "state")
    ep = float(np.abs(pr.cpu().numpy() - ref["prior"]).max()) if temporal else 0.0
    print("o %.3e state %.3e prior %.3e (tol %.0e)" % (eo, es, ep, tol))
    assert eo <= tol and es <= tol and ep <= tol


def test_gated_config2_every_head():
    """The c2 batch, as the benchmark times it, through the gated form (decay
    logits N(2,1)); the oracle on every head."""
    import torch
    import paper_2609_39034_amd as sw
    inp = workloads.config_inputs(2)
    c = workloads.CONFIGS[2]
    B, H, T, Dk, J = c["B"], c["H"], c["T"], c["Dk"], c["J"]
    dec = workloads.gated_inputs(B, H, T, Dk, J, dtype="bf16", seed=1002)["decay"]
    dev = to_device(inp, "bf16")
    o, s, r = sw.forward_gated(*(dev[n] for n in NAMES), _t(dec, "bf16"), None, resp=True)
    torch.cuda.synchronize()
    o, s, r = (x.float().cpu().numpy().astype(np.float64) for x in (o, s, r))
    ref = oracle.forward(*(inp[n] for n in NAMES), None, decay_logit=dec, want_resp=True)
    eo = head_rel_err(o, ref["o"], "o")
    es = head_rel_err(s, ref["state"], "state")
    er = head_rel_err(r, ref["resp"], "resp")
    print("worst head: o %.3e state %.3e resp %.3e" % (eo, es, er))
    assert eo <= 2e-2 and es <= 2e-2 and er <= 2e-2


def test_gated_empty_sequence_copies_states():
    """T = 0 through the gated forward: the states are copied, nothing else."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, D, J = 2, 3, 32, 4
    q = torch.empty((B, 0, H, D), device="cuda")
    lb = torch.empty((B, 0, H, J, D), device="cuda")
    dec = torch.empty((B, 0, H, J, D), device="cuda")
    s0 = torch.randn((B, H, J, D, D), device="cuda")
    o, s = sw.forward_gated(q, q, q, lb, lb, lb, dec, s0)
    torch.cuda.synchronize()
    assert o.numel() == 0 and torch.equal(s, s0)
