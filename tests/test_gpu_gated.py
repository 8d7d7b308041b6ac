"""Parity of the Gated SwiLA path (Sec. 3.4, App. B.4, eq. pre-decay with one
gate per key dimension) through the C ABI with the fp64 oracle: the
token-by-token scan and the decode step, alone and with the temporal priors,
and the chunk form on the matrix cores (bf16 inputs, J <= 4, J * Dk <= 512),
including chunks whose gates decay past the factorised Gram products.

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
    res = sw.forward_gated(*(dev[n] for n in NAMES), _t(dec, dtype), dev["state"], resp=True,
                           algo="recurrent", **kw)
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


@pytest.mark.parametrize("algo", ["chunk", "recurrent"])
def test_gated_config2_every_head(algo):
    """The c2 batch, as the benchmark times it, through the gated form (decay
    logits N(2,1)) on either algorithm; the oracle on every head."""
    import torch
    import paper_2609_39034_amd as sw
    inp = workloads.config_inputs(2)
    c = workloads.CONFIGS[2]
    B, H, T, Dk, J = c["B"], c["H"], c["T"], c["Dk"], c["J"]
    dec = workloads.gated_inputs(B, H, T, Dk, J, dtype="bf16", seed=1002)["decay"]
    dev = to_device(inp, "bf16")
    o, s, r = sw.forward_gated(*(dev[n] for n in NAMES), _t(dec, "bf16"), None, resp=True,
                               algo=algo)
    torch.cuda.synchronize()
    o, s, r = (x.float().cpu().numpy().astype(np.float64) for x in (o, s, r))
    ref = oracle.forward(*(inp[n] for n in NAMES), None, decay_logit=dec, want_resp=True)
    eo = head_rel_err(o, ref["o"], "o")
    es = head_rel_err(s, ref["state"], "state")
    er = head_rel_err(r, ref["resp"], "resp")
    print("%s, worst head: o %.3e state %.3e resp %.3e" % (algo, eo, es, er))
    assert eo <= 2e-2 and es <= 2e-2 and er <= 2e-2


# ---- the chunk form (bf16 inputs, J <= 4, J * Dk <= 512)
CHUNK_CASES = [
    # B, H, T, Dk, Dv, J, state_std, decay mean
    (1, 2, 37, 64, 64, 4, 0.1, 2.0),     # ragged third chunk
    (2, 1, 16, 32, 16, 2, 0.0, 1.0),     # one whole chunk
    (1, 1, 1, 16, 16, 1, 0.3, 2.0),      # one token
    (2, 2, 50, 16, 32, 3, 0.2, 0.0),     # J = 3 (padded lanes), a = 1/2 on average
    (1, 3, 70, 128, 64, 2, 0.1, 2.0),    # Dk = 128
    (1, 2, 45, 128, 128, 1, 0.2, 3.0),   # J = 1
    (2, 2, 64, 32, 128, 4, 0.1, 2.0),    # Dv = 128, whole chunks
    (1, 1, 33, 64, 16, 4, 0.3, -1.0),    # strong decay (some chunks past the factorised form)
    (8, 8, 40, 64, 64, 4, 0.1, 2.0),     # 256 blocks of 16 output dims
    (4, 16, 29, 64, 32, 2, 0.2, 2.0),    # 256 blocks of 8 output dims
    (1, 2, 37, 128, 128, 4, 0.1, 2.0),   # J * Dk = 512
    (2, 2, 50, 128, 64, 3, 0.2, 1.0),    # J = 3, Dk = 128
    (8, 16, 20, 128, 128, 4, 0.1, 2.0),  # 1024 blocks of 16 output dims, J * Dk = 512
]


def _chunk_case(B, H, T, Dk, Dv, J, std, mean, seed, dec=None):
    import torch
    import paper_2609_39034_amd as sw
    inp = workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="bf16", seed=seed, state_std=std)
    if dec is None:
        dec = workloads.gated_inputs(B, H, T, Dk, J, dtype="bf16", seed=seed, mean=mean)["decay"]
    dev = to_device(inp, "bf16")
    res = sw.forward_gated(*(dev[n] for n in NAMES), _t(dec, "bf16"), dev["state"], resp=True,
                           algo="chunk")
    torch.cuda.synchronize()
    res = [x.float().cpu().numpy().astype(np.float64) for x in res]
    ref = oracle.forward(*(inp[n] for n in NAMES), inp["state"], decay_logit=dec, want_resp=True)
    eo, es = head_rel_err(res[0], ref["o"], "o"), head_rel_err(res[1], ref["state"], "state")
    er = head_rel_err(res[2], ref["resp"], "resp")
    print("chunk form: o %.3e state %.3e resp %.3e" % (eo, es, er))
    return eo, es, er


@pytest.mark.parametrize("B,H,T,Dk,Dv,J,std,mean", CHUNK_CASES)
def test_gated_chunk_forward(B, H, T, Dk, Dv, J, std, mean):
    eo, es, er = _chunk_case(B, H, T, Dk, Dv, J, std, mean, seed=700 + T + J + Dk)
    assert eo <= 2e-2 and es <= 2e-2 and er <= 2e-2


@pytest.mark.parametrize("J,Dk", [(4, 64), (2, 128), (1, 16), (4, 128)])
def test_gated_chunk_deep_decay(J, Dk):
    """Eight tokens of gate logit -8 (a = 3.4e-4, log a = -8) in the second chunk
    take its cumulative log gate to about -64, past the factorised Gram
    products: that chunk forms them with the per-pair exponent, the others do
    not."""
    B, H, T, Dv = 1, 2, 56, 32
    dec = workloads.gated_inputs(B, H, T, Dk, J, dtype="bf16", seed=770)["decay"]
    dec[:, 20:28] = -8.0
    eo, es, er = _chunk_case(B, H, T, Dk, Dv, J, 0.2, 2.0, seed=771, dec=dec)
    assert eo <= 2e-2 and es <= 2e-2 and er <= 2e-2


def test_gated_chunk_all_chunks_deep():
    """Gate logits around -4 everywhere: every chunk past the factorised form."""
    eo, es, er = _chunk_case(2, 1, 48, 32, 32, 2, 0.1, -4.0, seed=772)
    assert eo <= 2e-2 and es <= 2e-2 and er <= 2e-2


def test_gated_chunk_saturated_equals_plain_chunk():
    """Gate logits of 40 (a = 1 in fp32): the gated chunk form gives the plain
    chunk scan's result, up to the rounding of two different kernels."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, T, D, J = 2, 2, 45, 64, 4
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="bf16", seed=773, state_std=0.2)
    dev = to_device(inp, "bf16")
    dec = torch.full((B, T, H, J, D), 40.0, device="cuda", dtype=torch.bfloat16)
    o_g, s_g = sw.forward_gated(*(dev[n] for n in NAMES), dec, dev["state"], algo="chunk")
    o_p, s_p = sw.forward(*(dev[n] for n in NAMES), dev["state"], algo="chunk")
    torch.cuda.synchronize()
    eo = head_rel_err(o_g.float().cpu().numpy(), o_p.float().cpu().numpy().astype(np.float64), "o")
    es = head_rel_err(s_g.cpu().numpy(), s_p.cpu().numpy().astype(np.float64), "state")
    print("o %.3e state %.3e" % (eo, es))
    assert eo <= 1e-2 and es <= 1e-3


def test_gated_chunk_state_chaining():
    """Two calls, the second starting from the first's final state, equal one
    call over the whole sequence (the split falls inside a chunk)."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, T, D, J = 1, 2, 53, 64, 4
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="bf16", seed=774, state_std=0.1)
    dec = _t(workloads.gated_inputs(B, H, T, D, J, dtype="bf16", seed=774)["decay"], "bf16")
    dev = to_device(inp, "bf16")
    o, s = sw.forward_gated(*(dev[n] for n in NAMES), dec, dev["state"], algo="chunk")
    cut = 21
    first = [dev[n][:, :cut].contiguous() for n in NAMES]
    second = [dev[n][:, cut:].contiguous() for n in NAMES]
    o1, s1 = sw.forward_gated(*first, dec[:, :cut].contiguous(), dev["state"], algo="chunk")
    o2, s2 = sw.forward_gated(*second, dec[:, cut:].contiguous(), s1, algo="chunk")
    torch.cuda.synchronize()
    oc = torch.cat([o1, o2], dim=1).float().cpu().numpy().astype(np.float64)
    eo = head_rel_err(oc, o.float().cpu().numpy().astype(np.float64), "o")
    es = head_rel_err(s2.cpu().numpy(), s.cpu().numpy().astype(np.float64), "state")
    print("o %.3e state %.3e" % (eo, es))
    assert eo <= 1e-2 and es <= 1e-3


def test_gated_auto_picks_the_chunk_form():
    """SWILA_ALGO_AUTO on a shape the chunk form takes gives its result exactly."""
    import torch
    import paper_2609_39034_amd as sw
    B, H, T, D, J = 1, 2, 40, 64, 4
    inp = workloads.iid_inputs(B, H, T, D, D, J, dtype="bf16", seed=775, state_std=0.1)
    dec = _t(workloads.gated_inputs(B, H, T, D, J, dtype="bf16", seed=775)["decay"], "bf16")
    dev = to_device(inp, "bf16")
    oa, sa = sw.forward_gated(*(dev[n] for n in NAMES), dec, dev["state"])
    oc, sc = sw.forward_gated(*(dev[n] for n in NAMES), dec, dev["state"], algo="chunk")
    torch.cuda.synchronize()
    assert torch.equal(oa, oc) and torch.equal(sa, sc)


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
