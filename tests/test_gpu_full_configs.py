"""Oracle parity on every head of the standard and the largest configurations,
in the launch shape the benchmark times, through the C ABI.

  c2  B=4  H=8  T=2048  Dk=Dv=64  J=4  the standard training batch
  c3  B=8  H=16 T=4096  Dk=Dv=128 J=4  LM-shaped projections
  c5  B=2  H=8  T=16384 Dk=Dv=128 J=8  recall-shaped long context
  c4  B=256 H=16 Dk=Dv=128 J=4, 512 in-place decode steps from N(0, 0.1^2)

For c2, c3 and c5: the plain forward (outputs, final state, responsibilities), the
App. D form run to convergence (its fixed point is the sequential trajectory,
App. D.1), the temporal form (App. B.3; gate logits N(0,1)) and the gated form
(App. B.4; decay logits N(2,1)), each against the fp64 oracle on the whole
batch.  For c4: every sequence over all 512 steps.

Bar: per (b, h), max|gpu - oracle| / max|oracle| <= 2e-2 (bf16 inputs, fp32
state and accumulation).  Each test prints its worst head's errors.
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_helpers import NAMES, TOL_BF16, head_rel_err, to_device

pytestmark = pytest.mark.gpu

_cache = {}


def _inputs(cfg):
    """Inputs of configuration cfg; the inputs and oracle results of any other
    configuration are dropped first (they take several GB of host memory)."""
    for key in [k for k in _cache if k[0] != cfg]:
        del _cache[key]
    if (cfg, "inp") not in _cache:
        _cache[(cfg, "inp")] = workloads.config_inputs(cfg)
    return _cache[(cfg, "inp")]


def _plain_oracle(cfg):
    if (cfg, "plain") not in _cache:
        inp = _inputs(cfg)
        _cache[(cfg, "plain")] = oracle.forward(*(inp[n] for n in NAMES), inp["state"],
                                                want_resp=True)
    return _cache[(cfg, "plain")]


def _np(x):
    return x.float().cpu().numpy().astype(np.float64)


def _report(cfg, form, **errs):
    print("c%d %s, worst head: %s" % (cfg, form, " ".join("%s %.3e" % kv for kv in errs.items())),
          flush=True)
    for name, e in errs.items():
        assert e <= TOL_BF16, (name, e)


@pytest.mark.parametrize("cfg", [2, 3, 5])
class TestEveryHead:
    def test_plain(self, cfg):
        import torch
        import paper_2609_39034_amd as sw
        inp = _inputs(cfg)
        dev = to_device(inp, "bf16")
        o, s, r = sw.forward(*(dev[n] for n in NAMES), dev["state"], resp=True)
        torch.cuda.synchronize()
        ref = _plain_oracle(cfg)
        _report(cfg, "forward", o=head_rel_err(_np(o), ref["o"], "o"),
                state=head_rel_err(_np(s), ref["state"], "state"),
                resp=head_rel_err(_np(r), ref["resp"], "resp"))

    def test_newton_converges_to_sequential(self, cfg):
        import torch
        import paper_2609_39034_amd as sw
        inp = _inputs(cfg)
        dev = to_device(inp, "bf16")
        it = torch.zeros(2, dtype=torch.int32, device="cuda")
        o, s = sw.forward(*(dev[n] for n in NAMES), dev["state"], algo="newton", max_iters=256,
                          tol=1e-3, iters_out=it)
        torch.cuda.synchronize()
        sweeps, unconverged = (int(x) for x in it.cpu())
        print("c%d App. D: %d sweeps, %d blocks unconverged" % (cfg, sweeps, unconverged))
        assert unconverged == 0
        ref = _plain_oracle(cfg)
        _report(cfg, "App. D", o=head_rel_err(_np(o), ref["o"], "o"),
                state=head_rel_err(_np(s), ref["state"], "state"))

    def test_temporal(self, cfg):
        import torch
        import paper_2609_39034_amd as sw
        inp = _inputs(cfg)
        c = workloads.CONFIGS[cfg]
        B, H, T, Dv, J = c["B"], c["H"], c["T"], c["Dv"], c["J"]
        tmp = workloads.temporal_inputs(B, H, T, Dv, J, dtype="bf16", seed=1000 + cfg)
        dev = to_device(inp, "bf16")
        gk = torch.from_numpy(tmp["gk"]).to("cuda", torch.bfloat16)
        gq = torch.from_numpy(tmp["gq"]).to("cuda", torch.bfloat16)
        o, s, p, r = sw.forward_temporal(*(dev[n] for n in NAMES), gk, gq, dev["state"], None,
                                         resp=True)
        torch.cuda.synchronize()
        ref = oracle.forward(*(inp[n] for n in NAMES), inp["state"], gate_k_logit=tmp["gk"],
                             gate_q_logit=tmp["gq"], want_resp=True)
        ep = float(np.abs(_np(p) - ref["prior"]).max())
        _report(cfg, "temporal", o=head_rel_err(_np(o), ref["o"], "o"),
                state=head_rel_err(_np(s), ref["state"], "state"),
                resp=head_rel_err(_np(r), ref["resp"], "resp"), prior=ep)

    def test_gated(self, cfg):
        import torch
        import paper_2609_39034_amd as sw
        inp = _inputs(cfg)
        c = workloads.CONFIGS[cfg]
        B, H, T, Dk, J = c["B"], c["H"], c["T"], c["Dk"], c["J"]
        dec = workloads.gated_inputs(B, H, T, Dk, J, dtype="bf16", seed=1000 + cfg)["decay"]
        dev = to_device(inp, "bf16")
        dd = torch.from_numpy(dec).to("cuda", torch.bfloat16)
        o, s, r = sw.forward_gated(*(dev[n] for n in NAMES), dd, dev["state"], resp=True)
        torch.cuda.synchronize()
        ref = oracle.forward(*(inp[n] for n in NAMES), inp["state"], decay_logit=dec,
                             want_resp=True)
        _report(cfg, "gated", o=head_rel_err(_np(o), ref["o"], "o"),
                state=head_rel_err(_np(s), ref["state"], "state"),
                resp=head_rel_err(_np(r), ref["resp"], "resp"))


# ---------------------------------------------------------------- c4 decode
_GROUPS = 8


@pytest.fixture(scope="module")
def decode_run():
    """The whole c4 workload on the GPU: 512 in-place decode steps of all 256
    sequences; every step's inputs (drawn on the device) and outputs are kept
    on the host (bf16), with the initial and final states."""
    import torch
    import paper_2609_39034_amd as sw
    _cache.clear()
    c = workloads.CONFIGS[4]
    B, H, Dk, Dv, J, steps = c["B"], c["H"], c["Dk"], c["Dv"], c["J"], c["steps"]
    s0 = workloads.decode_initial_state(B, H, Dk, Dv, J)
    st = torch.from_numpy(s0).cuda()
    shapes = {"q": (H, Dk), "k": (H, Dk), "v": (H, Dv), "lb": (H, J, Dv), "lk": (H, J, Dv),
              "lq": (H, J, Dv)}
    rec = {n: torch.empty((B, steps) + shapes[n], dtype=torch.bfloat16) for n in NAMES}
    outs = torch.empty((B, steps, H, Dv), dtype=torch.bfloat16)
    for t in range(steps):
        x = workloads.decode_step_inputs_torch(t, B, H, Dk, Dv, J)
        o, _ = sw.decode_step(*(x[n] for n in NAMES), st, state_out=st)
        for n in NAMES:
            rec[n][:, t] = x[n].cpu()
        outs[:, t] = o.cpu()
    torch.cuda.synchronize()
    assert torch.isfinite(st).all()
    return {"s0": s0, "inputs": rec, "o": outs, "state": st.cpu().numpy()}


@pytest.mark.parametrize("group", range(_GROUPS))
def test_decode_every_sequence(decode_run, group):
    """Sequences [32 g, 32 g + 32) of c4 over all 512 steps against the oracle's
    forward over those tokens from the same initial states."""
    B = decode_run["o"].shape[0]
    sl = slice(group * B // _GROUPS, (group + 1) * B // _GROUPS)
    args = [decode_run["inputs"][n][sl].float().numpy() for n in NAMES]
    ref = oracle.forward(*args, decode_run["s0"][sl])
    eo = head_rel_err(decode_run["o"][sl].float().numpy(), ref["o"], "o")
    es = head_rel_err(decode_run["state"][sl], ref["state"], "state")
    print("c4 sequences %d..%d, worst head: o %.3e state %.3e" % (sl.start, sl.stop - 1, eo, es),
          flush=True)
    assert eo <= TOL_BF16 and es <= TOL_BF16
