"""Benchmark of the SwiLA hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config 3] [--no-decode] [--no-cpu-baseline]

A step is one swila_forward call over the whole batch of the LM-shaped
workload (B=8, H=16, T=4096, Dk=Dv=128, J=4, bf16 inputs, fp32 state), inputs
resident in HBM.  value = B*T / seconds per step (tokens/s).  The same run
also times:
  "c2", "c5", "c1"  the forward on the other whole-sequence workloads (c1 in us);
  "temporal", "gated"  the temporal (App. B.3) and gated (App. B.4) forms on the
                    headline batch;
  "newton", "newton_c5"  the App. D form on the c2 and c5 batches;
  "backward"        the gradient of the plain forward on the c2 batch;
  "decode"          the batched decode workload (B=256, H=16, D=128, J=4, 512
                    one-token steps, state updated in place);
  "cpu_baseline"    the fp64 oracle on the host cores (whole headline batch), with
                    single-thread figures for c1 and c2.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("SwiLA fwd tokens/sec at B·H·T·D·K; decode steps/sec; "
          "% HBM/MFMA roofline")
PEAK_HBM = 8.0e12          # B/s, MI355X HBM3E
PEAK_VALU_F32 = 157.3e12   # FLOP/s, MI355X fp32 vector (packed); unpacked FMA is half
PEAK_MFMA_BF16 = 2.5e15    # FLOP/s, MI355X dense bf16 matrix
PEAK_MFMA_F32 = 157.3e12   # FLOP/s, MI355X dense fp32 matrix

# Counter-measured HBM bytes per launch (FETCH_SIZE and WRITE_SIZE, each scaled by
# what the counter reads for a plain copy of known size), keyed by the kernel's
# source, the workload it ran and the digest of the source at measurement.
MEASURED_TRAFFIC = {
    ("scan_pipe.hip", "forward B=8 H=16 T=4096 Dk=Dv=128 J=4",
     "69a737312b74bd8f3dedd808d43ac8367b2dbf9b21ccca372790ce9b8cebd952"): 2185222850,
    ("scan_pipe.hip", "forward B=4 H=8 T=2048 Dk=Dv=64 J=4",
     "69a737312b74bd8f3dedd808d43ac8367b2dbf9b21ccca372790ce9b8cebd952"): 136707495,
    ("scan_pipe.hip", "forward B=2 H=8 T=16384 Dk=Dv=128 J=8",
     "69a737312b74bd8f3dedd808d43ac8367b2dbf9b21ccca372790ce9b8cebd952"): 2797221636,
    ("scan_pipe_temporal.hip", "temporal B=8 H=16 T=4096 Dk=Dv=128 J=4",
     "41604fc349b073c09ba91bf77ad77b546ac62f0e66f6d17093fb967cc91b2027"): 2450471795,
    ("scan_gated_chunk.hip", "gated B=8 H=16 T=4096 Dk=Dv=128 J=4",
     "3521c3b9f68a659ea24c176dfcb5d3ac4e3060cceb8b7219c8ae445ec250cf44"): 2720938128,
    ("decode.hip", "decode B=256 H=16 Dk=Dv=128 J=4",
     "a4c73fb2a97e003cf707dbe2b81c1b57afaee61077b4cfc79a6a3f9889745265"): 2166168222,
    ("scan_gated_chunk.hip", "gated B=4 H=8 T=2048 Dk=Dv=64 J=4",
     "3521c3b9f68a659ea24c176dfcb5d3ac4e3060cceb8b7219c8ae445ec250cf44"): 170459080,
}


def workload_key(kind, B, H, T, Dk, Dv, J):
    """The MEASURED_TRAFFIC key of a workload: its kind and sizes."""
    dims = "Dk=Dv=%d" % Dk if Dk == Dv else "Dk=%d Dv=%d" % (Dk, Dv)
    if kind == "decode":
        return "decode B=%d H=%d %s J=%d" % (B, H, dims, J)
    return "%s B=%d H=%d T=%d %s J=%d" % (kind, B, H, T, dims, J)


def measured_traffic(source, workload):
    """Counter-measured HBM bytes per launch of the kernel in ``source`` on
    ``workload`` (a ``workload_key``), or None when that source has changed since
    the counters were taken or the workload was not measured."""
    try:
        digest = kernel_source_digest(source)
    except OSError:
        return None
    return MEASURED_TRAFFIC.get((source, workload, digest))


def kernel_source_digest(source):
    """sha256 over the code of ``source`` and, recursively and once each, of the
    local headers and fragments it includes (``#include "..."``), in include
    order.  Comments and blank lines are left out, so that a change to the
    comments alone keeps the digest (and the measurements filed under it)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2609_39034_amd", "csrc")
    h = hashlib.sha256()
    seen = set()

    def code(text):
        text = re.sub(rb"/\*.*?\*/", b"", text, flags=re.S)
        text = re.sub(rb"//[^\n]*", b"", text)
        return b"\n".join(l.rstrip() for l in text.split(b"\n") if l.strip())

    def add(name):
        path = os.path.join(csrc, name)
        if name in seen or not os.path.exists(path):
            return
        seen.add(name)
        text = open(path, "rb").read()
        h.update(code(text))
        for inc in re.findall(rb'^\s*#include\s+"([^"]+)"', text, re.M):
            add(inc.decode())

    add(source)
    if source not in seen:
        raise OSError("no such kernel source: %s" % source)
    return h.hexdigest()


def forward_alg_bytes(B, H, T, Dk, Dv, J, in_bytes=2, out_bytes=2, state_in=False,
                      state_out=True):
    """Bytes the forward must move at least once: q, k, v, three logit tensors,
    the output, and the state (read if given, written if kept)."""
    per_token_head = in_bytes * (2 * Dk + Dv) + in_bytes * 3 * J * Dv + out_bytes * Dv
    state = 4 * J * Dk * Dv * B * H
    return B * H * T * per_token_head + state * (int(state_in) + int(state_out))


def forward_alg_flops(B, H, T, Dk, Dv, J):
    """Two length-Dk dots (w.k, w.q) and one rank-one update per (t, j, d):
    3 * Dk * J * Dv fused multiply-adds per token and head, 2 FLOP each."""
    return 2 * 3 * Dk * J * Dv * B * H * T


def decode_alg_bytes(B, H, Dk, Dv, J, in_bytes=2, out_bytes=2):
    """Per step: the state read and written once, one token of inputs, output."""
    return (2 * 4 * J * Dk * Dv + in_bytes * (2 * Dk + Dv + 3 * J * Dv) + out_bytes * Dv) * B * H


def host_cores():
    """(threads the oracle uses, cores visible to this process).  The threads
    are the visible cores, capped by OMP_NUM_THREADS when it is set: a GPU
    box grants one GPU's job that many cores of the host."""
    try:
        visible = len(os.sched_getaffinity(0))
    except AttributeError:
        visible = os.cpu_count() or 1
    n = visible
    try:
        cap = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        cap = 0
    if cap > 0:
        n = min(n, cap)
    return max(1, n), visible


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_forward(sw, torch, dev, steps, warmup, o, s_out, algo, **kw):
    names = ("q", "k", "v", "lb", "lk", "lq")
    args = [dev[n] for n in names]
    for _ in range(warmup):
        sw.forward(*args, dev["state"], o=o, state_out=s_out, algo=algo, **kw)
    torch.cuda.synchronize()
    # One pair of HIP events on the launch stream brackets the timed calls:
    # the device time per call, gaps between back-to-back launches included.
    # (A pair around every call would put two event records, about 4 us of
    # host time each, into every step of a launch that takes microseconds.)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(steps):
        sw.forward(*args, dev["state"], o=o, state_out=s_out, algo=algo, **kw)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    kern = e0.elapsed_time(e1) / steps / 1e3
    return wall, kern


def newton_alg_flops(B, H, T, Dk, Dv, J, sweeps, chunk=16):
    """Matrix-core work of the App. D form as this library evaluates it, each
    product counted once (the bf16 high/residual split counts against it).
    Per sweep, per chunk of C tokens and head (N = J * Dv columns):
    Q S and K S (2 C Dk N), the state update K^T X (C Dk N), the two C x C by
    C x N products of the forward substitution and the retrieval (2 C^2 N),
    and the three C x C Gram products (3 C^2 Dk).  The initial guess K W_0
    (Dk N per token) is counted once.  2 FLOP per multiply-add."""
    nch = (T + chunk - 1) // chunk
    per_chunk = 3 * chunk * Dk * J * Dv + 2 * chunk * chunk * J * Dv + 3 * chunk * chunk * Dk
    return 2 * B * H * (sweeps * nch * per_chunk + T * Dk * J * Dv)


def bench_newton(sw, torch, dev, cfg, steps, warmup, o, s_out, tol, unnormalized=False,
                 clamp=True):
    B, H, T, Dk, Dv, J = (cfg[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    batch = "B=%d H=%d T=%d Dk=Dv=%d J=%d" % (B, H, T, Dk, J)
    ws = torch.empty(sw.forward_workspace_bytes(B, H, T, Dk, Dv, J, algo="newton"),
                     device="cuda", dtype=torch.uint8)
    it = torch.zeros(2, device="cuda", dtype=torch.int32)
    wall, kern = time_forward(sw, torch, dev, steps, warmup, o, s_out, "newton", workspace=ws,
                              tol=tol, max_iters=256, iters_out=it, unnormalized=unnormalized,
                              clamp=clamp)
    sweeps, unconverged = (int(x) for x in it.cpu())
    nflop = newton_alg_flops(B, H, T, Dk, Dv, J, sweeps)
    form = ("App. D.2's unnormalised-responsibility variant" if unnormalized
            else "App. D chunkwise quasi-Newton")
    jac = ("g clamped to [0, 2/|k|^2]" if clamp
           else "g unclamped (the exact Jacobian: Newton's method proper)")
    return {
        "workload": "%s, %s, bf16 inputs, tol %g (relative change of the predictions), %s"
                    % (form, batch, tol, jac),
        "tokens_per_s": B * T / wall, "ms_per_step": wall * 1e3, "sweeps": sweeps,
        "unconverged_blocks": unconverged,
        "roofline": {"bound": "mfma", "achieved": nflop / kern / 1e12,
                     "peak": PEAK_MFMA_BF16 / 1e12, "unit": "TFLOP/s",
                     "frac": nflop / kern / PEAK_MFMA_BF16, "traffic": None,
                     "kernel": "scan_pipe_kernel (Newton mode)", "kernel_ms": kern * 1e3,
                     "alg_flop_per_launch": nflop},
    }


def bench_decode(sw, torch, workloads, steps_total, warmup):
    c = workloads.CONFIGS[4]
    B, H, Dk, Dv, J = c["B"], c["H"], c["Dk"], c["Dv"], c["J"]
    st = torch.from_numpy(workloads.decode_initial_state(B, H, Dk, Dv, J)).cuda()
    inputs = [workloads.decode_step_inputs_torch(t, B, H, Dk, Dv, J) for t in range(steps_total)]
    o = torch.empty((B, H, Dv), device="cuda", dtype=torch.bfloat16)
    names = ("q", "k", "v", "lb", "lk", "lq")
    for t in range(warmup):
        sw.decode_step(*(inputs[t % steps_total][n] for n in names), st, state_out=st, o=o)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps_total)]
    t0 = time.perf_counter()
    for t in range(steps_total):
        ev[t][0].record(stream)
        sw.decode_step(*(inputs[t][n] for n in names), st, state_out=st, o=o)
        ev[t][1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps_total
    kern = sum(a.elapsed_time(b) for a, b in ev) / steps_total / 1e3
    nbytes = decode_alg_bytes(B, H, Dk, Dv, J)
    assert torch.isfinite(st).all().item()
    return {
        "workload": "batched decode B=%d H=%d Dk=Dv=%d J=%d, %d one-token steps, bf16 inputs, "
                    "fp32 state N(0,0.1^2) updated in place" % (B, H, Dk, J, steps_total),
        "steps_per_s": 1.0 / wall, "tokens_per_s": B / wall, "ms_per_step": wall * 1e3,
        "roofline": {"bound": "hbm", "achieved": nbytes / kern / 1e9, "peak": PEAK_HBM / 1e9,
                     "unit": "GB/s", "frac": nbytes / kern / PEAK_HBM,
                     "traffic": measured_traffic("decode.hip",
                                                 workload_key("decode", B, H, 1, Dk, Dv, J)),
                     "kernel": "decode_kernel",
                     "kernel_ms": kern * 1e3, "alg_bytes_per_launch": nbytes},
    }


def temporal_alg_bytes(B, H, T, Dk, Dv, J, in_bytes=2, out_bytes=2, state_in=False,
                       state_out=True, prior_in=False, prior_out=True):
    """The forward's bytes plus the two gate-logit tensors (one value per token,
    head and output dim each) and the fp32 prior state [B,H,2,J,Dv]."""
    prior = 4 * 2 * J * Dv * B * H
    return (forward_alg_bytes(B, H, T, Dk, Dv, J, in_bytes, out_bytes, state_in, state_out)
            + 2 * in_bytes * Dv * B * H * T + prior * (int(prior_in) + int(prior_out)))


def bench_temporal(sw, torch, workloads, dev, cfg, seed, steps, warmup, o, s_out, algo, tdt):
    """Temporal SwiLA (App. B.3) on the same batch: N(0,1) gate logits, uniform
    initial priors, final prior state kept."""
    B, H, T, Dk, Dv, J = (cfg[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    tmp = workloads.temporal_inputs(B, H, T, Dv, J, dtype=cfg["dtype"], seed=seed)
    gk = torch.from_numpy(tmp["gk"]).to("cuda", tdt)
    gq = torch.from_numpy(tmp["gq"]).to("cuda", tdt)
    p_out = torch.empty((B, H, 2, J, Dv), device="cuda", dtype=torch.float32)
    names = ("q", "k", "v", "lb", "lk", "lq")
    args = [dev[n] for n in names]

    def step():
        sw.forward_temporal(*args, gk, gq, dev["state"], None, o=o, state_out=s_out,
                            prior_out=p_out, algo=algo)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        step()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    kern = sum(a.elapsed_time(b) for a, b in ev) / steps / 1e3
    bf16 = cfg["dtype"] == "bf16"
    eb = 2 if bf16 else 4
    chunk = algo == "chunk" or (algo == "auto" and bf16)
    nbytes = temporal_alg_bytes(B, H, T, Dk, Dv, J, eb, eb, dev["state"] is not None, True)
    return {
        "workload": "Temporal SwiLA (App. B.3), B=%d H=%d T=%d Dk=Dv=%d J=%d, N(0,1) gate "
                    "logits, uniform initial priors, final prior state kept" % (B, H, T, Dk, J),
        "tokens_per_s": B * T / wall, "ms_per_step": wall * 1e3,
        "algo": "chunk_exact" if chunk else "recurrent",
        "roofline": {"bound": "hbm", "achieved": nbytes / kern / 1e9, "peak": PEAK_HBM / 1e9,
                     "unit": "GB/s", "frac": nbytes / kern / PEAK_HBM,
                     "traffic": (measured_traffic("scan_pipe_temporal.hip",
                                                  workload_key("temporal", B, H, T, Dk, Dv, J))
                                 if chunk else None),
                     "kernel": ("scan_pipe_kernel (temporal mode)" if chunk
                                else "scan_direct_kernel (temporal)"),
                     "kernel_ms": kern * 1e3, "alg_bytes_per_launch": nbytes},
    }


def backward_alg_flops(B, H, T, Dk, Dv, J):
    """Multiply-adds of the gradient per token, head, component and output dim,
    each Dk long: the forward's three (the state and errors are recomputed), the
    reverse recurrence's three (dy q and dpred k into dL/dw, dc = dL/dw . k), the
    query and key gradients' three (dy . w_t, c . dL/dw, dpred . w_{t-1}) and the
    retrieval y = w_t . q for the query-prior gradient.  2 FLOP each."""
    return 2 * 10 * Dk * J * Dv * B * H * T


def backward_alg_bytes(B, H, T, Dk, Dv, J, in_bytes=2, go_bytes=2):
    """The forward's inputs and dL/do read once; the six fp32 input gradients
    written once; dL/dW_0 written (zero initial state: no state read)."""
    per_token_head = (in_bytes * (2 * Dk + Dv + 3 * J * Dv) + go_bytes * Dv
                      + 4 * (2 * Dk + Dv + 3 * J * Dv))
    return B * H * T * per_token_head + 4 * J * Dk * Dv * B * H


def bench_backward(sw, torch, dev, cfg, steps, warmup):
    """The backward pass (swila_backward) on the same batch: dL/do ~ N(0,1) in the
    input dtype, no state gradient.  One step is one call: the forward
    recompute, the reverse scan and the chunk pass."""
    B, H, T, Dk, Dv, J = (cfg[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    names = ("q", "k", "v", "lb", "lk", "lq")
    args = [dev[n] for n in names]
    g = torch.Generator(device="cuda")
    g.manual_seed(4242)
    go = torch.randn((B, T, H, Dv), device="cuda", generator=g).to(dev["q"].dtype)
    ws = torch.empty(sw.backward_workspace_bytes(B, H, T, Dk, Dv, J), device="cuda",
                     dtype=torch.uint8)

    def step():
        return sw.backward(*args, dev["state"], go, None, workspace=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        step()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    kern = sum(a.elapsed_time(b) for a, b in ev) / steps / 1e3
    eb = dev["q"].element_size()
    nflop = backward_alg_flops(B, H, T, Dk, Dv, J)
    nbytes = backward_alg_bytes(B, H, T, Dk, Dv, J, eb, eb)
    return {
        "workload": "backward of the plain forward (exact gradient), B=%d H=%d T=%d Dk=Dv=%d "
                    "J=%d, dL/do N(0,1), zero initial state, no final-state gradient"
                    % (B, H, T, Dk, J),
        "tokens_per_s": B * T / wall, "ms_per_step": wall * 1e3,
        # its products run on the matrix cores in fp32 (the chunk pass) or as
        # split bf16 products with fp32 accumulation: the fp32 matrix peak
        "roofline": {"bound": "mfma", "achieved": nflop / kern / 1e12,
                     "peak": PEAK_MFMA_F32 / 1e12, "unit": "TFLOP/s",
                     "frac": nflop / kern / PEAK_MFMA_F32, "traffic": None,
                     "kernel": "swila_backward (forward recompute, reverse scan, chunk pass)",
                     "kernel_ms": kern * 1e3, "alg_flop_per_launch": nflop,
                     "alg_bytes_per_launch": nbytes},
    }


def gated_chunk_form(cfg):
    """Whether SWILA_ALGO_AUTO runs the gated form in chunks on the matrix cores
    (bf16 inputs, J <= 4, J * Dk <= 512, no temporal priors)."""
    return cfg["dtype"] == "bf16" and cfg["J"] <= 4 and cfg["J"] * cfg["Dk"] <= 512


def bench_gated(sw, torch, workloads, dev, cfg, seed, steps, warmup, o, s_out, tdt):
    """Gated SwiLA (App. B.4, eq. pre-decay, one gate per key dimension) on the
    same batch: decay logits N(2, 1), SWILA_ALGO_AUTO (the chunk form on the
    matrix cores where it applies, else the token-by-token scan)."""
    B, H, T, Dk, Dv, J = (cfg[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    dec = workloads.gated_inputs(B, H, T, Dk, J, dtype=cfg["dtype"], seed=seed)["decay"]
    dec = torch.from_numpy(dec).to("cuda", tdt)
    names = ("q", "k", "v", "lb", "lk", "lq")
    args = [dev[n] for n in names]

    def step():
        sw.forward_gated(*args, dec, dev["state"], o=o, state_out=s_out)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        step()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    kern = sum(a.elapsed_time(b) for a, b in ev) / steps / 1e3
    eb = 2 if cfg["dtype"] == "bf16" else 4
    nbytes = (forward_alg_bytes(B, H, T, Dk, Dv, J, eb, eb, dev["state"] is not None, True)
              + eb * J * Dk * B * H * T)
    # the method's FMAs plus the decay: one multiply per state element and token
    nflop = forward_alg_flops(B, H, T, Dk, Dv, J) + J * Dk * Dv * B * H * T
    chunk = gated_chunk_form(cfg)
    key = workload_key("gated", B, H, T, Dk, Dv, J)
    alu = {"bound": "alu", "achieved": nflop / kern / 1e12, "peak": PEAK_VALU_F32 / 1e12,
           "unit": "TFLOP/s", "frac": nflop / kern / PEAK_VALU_F32,
           "kernel_ms": kern * 1e3, "alg_flop_per_launch": nflop, "alg_bytes_per_launch": nbytes}
    hbm = {"bound": "hbm", "achieved": nbytes / kern / 1e9, "peak": PEAK_HBM / 1e9,
           "unit": "GB/s", "frac": nbytes / kern / PEAK_HBM, "kernel_ms": kern * 1e3,
           "alg_bytes_per_launch": nbytes}
    if chunk:
        # the Dk-long products run on the matrix cores: the HBM roofline, as for
        # the plain chunk scan, with the fp32-ALU figure beside it
        roof = dict(hbm, kernel="scan_gated_chunk_kernel",
                    traffic=measured_traffic("scan_gated_chunk.hip", key))
        other = dict(alu, kernel="scan_gated_chunk_kernel")
    else:
        roof = dict(alu, kernel="scan_direct_kernel (gated)",
                    traffic=measured_traffic("scan_direct_dk%d.hip" % Dk, key))
        other = None
    return {
        "workload": "Gated SwiLA (App. B.4, pre-decay, one gate per key dim), B=%d H=%d T=%d "
                    "Dk=Dv=%d J=%d, decay logits N(2,1), %s"
                    % (B, H, T, Dk, J, "chunks of 16 tokens on the matrix cores" if chunk
                       else "token-by-token scan"),
        "tokens_per_s": B * T / wall, "ms_per_step": wall * 1e3,
        "algo": "chunk_exact" if chunk else "recurrent",
        "roofline": roof, "roofline_other": other,
    }


def newton_study(sw, torch, workloads, steps, tol):
    """The paper's only chunked measurement (App. D.2): batch 16, T = 4096, 8 heads,
    D = 64, J = 4, synthetic N(0,1) inputs.  Runs the exact chunk scan, the App. D
    form, and App. D.2's unnormalised-responsibility variant (clamped and with
    its exact Jacobian unclamped) to tolerance on the same batch.  The variant is
    a different recurrence: only the normalised form is compared with the exact
    chunk scan."""
    B, H, T, Dk, Dv, J = 16, 8, 4096, 64, 64, 4
    inp = workloads.iid_inputs(B, H, T, Dk, Dv, J, dtype="bf16", seed=1042)
    dev = workloads.to_torch(inp, "cuda", torch.bfloat16)
    o = torch.empty((B, T, H, Dv), device="cuda", dtype=torch.bfloat16)
    s_out = torch.empty((B, H, J, Dk, Dv), device="cuda", dtype=torch.float32)
    wall_x, kern_x = time_forward(sw, torch, dev, steps, 1, o, s_out, "chunk")
    o_x, s_x = o.float().clone(), s_out.clone()
    cfg = {"B": B, "H": H, "T": T, "Dk": Dk, "Dv": Dv, "J": J}
    res = bench_newton(sw, torch, dev, cfg, steps, 1, o, s_out, tol)
    torch.cuda.synchronize()
    diff_o = ((o.float() - o_x).abs().amax() / o_x.abs().amax()).item()
    diff_s = ((s_out - s_x).abs().amax() / s_x.abs().amax()).item()
    res.update({
        "workload": "App. D study: B=16 H=8 T=4096 Dk=Dv=64 J=4, bf16 N(0,1) inputs, tol %g"
                    % tol,
        "exact_chunk_ms": wall_x * 1e3, "exact_chunk_kernel_ms": kern_x * 1e3,
        "newton_over_exact": res["ms_per_step"] / (wall_x * 1e3),
        "max_rel_diff_vs_exact": {"o": diff_o, "state": diff_s},
    })
    variants = {}
    for name, clamp in (("unnormalized_clamped", True), ("unnormalized_exact_jacobian", False)):
        v = bench_newton(sw, torch, dev, cfg, steps, 1, o, s_out, tol, unnormalized=True,
                         clamp=clamp)
        variants[name] = {x: v[x] for x in ("workload", "ms_per_step", "sweeps",
                                             "unconverged_blocks")}
        variants[name]["mfma_frac"] = v["roofline"]["frac"]
    res["variants"] = variants
    return res


def cpu_baseline(workloads, inp, cfg):
    """The fp64 oracle on the host cores: the whole headline batch on every
    thread granted, then c1 and c2 on one thread."""
    import oracle
    n, visible = host_cores()
    names = ("q", "k", "v", "lb", "lk", "lq")
    oracle.build()
    t0 = time.perf_counter()
    oracle.forward(*(inp[x] for x in names), inp["state"], nthreads=n)
    dt = time.perf_counter() - t0
    B, T = cfg["B"], cfg["T"]
    single = {}
    for c in (1, 2):
        x = workloads.config_inputs(c)
        t1 = time.perf_counter()
        oracle.forward(*(x[y] for y in names), x["state"], nthreads=1)
        d1 = time.perf_counter() - t1
        cc = workloads.CONFIGS[c]
        single["c%d" % c] = {"tokens_per_s": cc["B"] * cc["T"] / d1, "seconds": d1,
                             "us_per_call": d1 * 1e6}
    return {"value": B * T / dt, "unit": "tokens/s", "cores": n, "kind": "oracle",
            "sample": "the whole benchmark batch (B=%d H=%d T=%d Dk=Dv=%d J=%d), fp64, %d "
                      "threads, %.1f s" % (B, cfg["H"], T, cfg["Dk"], cfg["J"], n, dt),
            "cores_visible": visible, "cpu_model": cpu_model(),
            "single_thread": single}


def bench_forward(sw, torch, workloads, cfg_id, steps, warmup, algo, inp=None):
    """One swila_forward over the whole batch of workload cfg_id: wall time per
    step, kernel time from HIP events on the launch stream, and the HBM and
    fp32-ALU rooflines of the dominant kernel."""
    cfg = workloads.CONFIGS[cfg_id]
    B, H, T, Dk, Dv, J = (cfg[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    bf16 = cfg["dtype"] == "bf16"
    tdt = torch.bfloat16 if bf16 else torch.float32
    inp = workloads.config_inputs(cfg_id) if inp is None else inp
    dev = workloads.to_torch(inp, "cuda", tdt)
    o = torch.empty((B, T, H, Dv), device="cuda", dtype=tdt)
    s_out = torch.empty((B, H, J, Dk, Dv), device="cuda", dtype=torch.float32)
    wall, kern = time_forward(sw, torch, dev, steps, warmup, o, s_out, algo)
    chunk = algo == "chunk" or (algo == "auto" and bf16 and J <= 8)
    kname, ksrc = (("scan_pipe_kernel", "scan_pipe.hip") if chunk
                   else ("scan_direct_kernel", "scan_direct_dk%d.hip" % Dk))
    eb = 2 if bf16 else 4
    nbytes = forward_alg_bytes(B, H, T, Dk, Dv, J, eb, eb, dev["state"] is not None, True)
    nflop = forward_alg_flops(B, H, T, Dk, Dv, J)
    hbm = {"bound": "hbm", "achieved": nbytes / kern / 1e9, "peak": PEAK_HBM / 1e9,
           "unit": "GB/s", "frac": nbytes / kern / PEAK_HBM,
           "traffic": measured_traffic(ksrc, workload_key("forward", B, H, T, Dk, Dv, J)),
           "kernel": kname, "kernel_ms": kern * 1e3, "alg_bytes_per_launch": nbytes}
    alu = {"bound": "alu", "achieved": nflop / kern / 1e12, "peak": PEAK_VALU_F32 / 1e12,
           "unit": "TFLOP/s", "frac": nflop / kern / PEAK_VALU_F32, "kernel": kname,
           "kernel_ms": kern * 1e3, "alg_flop_per_launch": nflop}
    # The chunk scan runs the method's Dk-long products on the matrix cores,
    # where they take microseconds: its binding roofline is HBM.  The
    # token-by-token scan is bound by its fp32 FMAs on the vector ALUs.
    roof, other = (hbm, alu) if chunk else (alu, hbm)
    res = {
        "workload": "SwiLA forward, %s: B=%d H=%d T=%d Dk=Dv=%d J=%d, %s inputs, fp32 state, "
                    "zero initial state, seeded" % (cfg["name"], B, H, T, Dk, J, cfg["dtype"]),
        "B": B, "H": H, "T": T, "Dk": Dk, "Dv": Dv, "J": J,
        "algo": "chunk_exact" if chunk else "recurrent",
        "tokens_per_s": B * T / wall, "ms_per_step": wall * 1e3, "us_per_step": wall * 1e6,
        "roofline": roof, "roofline_other": other,
    }
    return res, dev, o, s_out, wall


ARITH = ("fp32 state, fp32 scalar recurrence and E-step; the Dk-long products on bf16 "
         "matrix cores with each fp32 operand split into a bf16 high part and a bf16 "
         "residual (hi*hi + hi*lo + lo*hi, about 2^-16 relative per product), fp32 "
         "accumulation; bf16 inputs and output")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 5])
    ap.add_argument("--algo", default="auto", choices=["auto", "chunk", "recurrent"])
    ap.add_argument("--decode-steps", type=int, default=512)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-newton", action="store_true")
    ap.add_argument("--no-temporal", action="store_true")
    ap.add_argument("--no-gated", action="store_true")
    ap.add_argument("--no-backward", action="store_true")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the c1, c2 and c5 forward lines")
    ap.add_argument("--newton-study", action="store_true",
                    help="only the App. D measurement at B=16 H=8 T=4096 D=64 J=4")
    ap.add_argument("--newton-tol", type=float, default=1e-3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy 1 GiB device-to-device (scales HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the SwiLA path has no cross-GPU step; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_39034_amd as sw
    import workloads

    if args.copy_calibration:
        x = torch.ones(1 << 28, device="cuda")
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        # the same copy timed: what a plain stream reaches on this GPU
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(20):
            y.copy_(x)
        e1.record()
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) / 20 / 1e3
        print(json.dumps({"copy_bytes_read": x.numel() * 4, "copy_bytes_written": y.numel() * 4,
                          "copy_ms": sec * 1e3, "copy_GBps": 2 * x.numel() * 4 / sec / 1e9}))
        return
    sw.load_library()
    if args.newton_study:
        print(json.dumps({"newton_study": newton_study(sw, torch, workloads, args.steps,
                                                        args.newton_tol)}), flush=True)
        return
    cfg = workloads.CONFIGS[args.config]
    B, H, T, Dk, Dv, J = (cfg[x] for x in ("B", "H", "T", "Dk", "Dv", "J"))
    bf16 = cfg["dtype"] == "bf16"
    tdt = torch.bfloat16 if bf16 else torch.float32
    inp = workloads.config_inputs(args.config)
    head, dev, o, s_out, wall = bench_forward(sw, torch, workloads, args.config, args.steps,
                                              args.warmup, args.algo, inp=inp)
    chunk = head["algo"] == "chunk_exact"
    out = {
        "metric": METRIC, "value": B * T / wall, "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32+bf16x3" if chunk else "f32",
        "arith": ARITH if chunk else "fp32 throughout on the vector ALUs",
        "io_dtype": "bf16" if bf16 else "f32", "data": "synthetic",
        "config": {"workload": head["workload"], "B": B, "H": H, "T": T, "Dk": Dk, "Dv": Dv,
                   "J": J, "algo": head["algo"]},
        "roofline": head["roofline"], "roofline_other": head["roofline_other"],
        "head_tokens_per_s": B * H * T / wall,
    }
    print("headline forward done: %.3f ms" % (wall * 1e3), file=sys.stderr, flush=True)
    if not args.no_temporal:
        out["temporal"] = bench_temporal(sw, torch, workloads, dev, cfg, 1000 + args.config,
                                         args.steps, args.warmup, o, s_out, args.algo, tdt)
    if not args.no_gated:
        out["gated"] = bench_gated(sw, torch, workloads, dev, cfg, 1000 + args.config,
                                   args.steps, args.warmup, o, s_out, tdt)
    print("temporal and gated done", file=sys.stderr, flush=True)
    if args.config in (2, 5) and not args.no_newton:
        out["newton" if args.config == 2 else "newton_c5"] = bench_newton(
            sw, torch, dev, cfg, args.steps, args.warmup, o, s_out, args.newton_tol)
    if args.config == 2 and not args.no_backward:
        out["backward"] = bench_backward(sw, torch, dev, cfg, args.steps, args.warmup)
    del dev, o, s_out
    if not args.no_other_configs:
        for c in (1, 2, 5):
            if c == args.config:
                continue
            res, dv, oc, sc, _ = bench_forward(sw, torch, workloads, c, args.steps, args.warmup,
                                               args.algo)
            out["c%d" % c] = res
            if c in (2, 5) and not args.no_newton:
                key = "newton" if c == 2 else "newton_c5"
                out[key] = bench_newton(sw, torch, dv, workloads.CONFIGS[c], args.steps,
                                        args.warmup, oc, sc, args.newton_tol)
            if c == 2 and not args.no_backward:
                out["backward"] = bench_backward(sw, torch, dv, workloads.CONFIGS[c], args.steps,
                                                 args.warmup)
            if c == 2 and not args.no_gated:
                out["gated_c2"] = bench_gated(sw, torch, workloads, dv, workloads.CONFIGS[c],
                                              1000 + c, args.steps, args.warmup, oc, sc,
                                              torch.bfloat16)
            del dv, oc, sc
            torch.cuda.empty_cache()
            print("c%d done" % c, file=sys.stderr, flush=True)
    if not args.no_decode:
        out["decode"] = bench_decode(sw, torch, workloads, args.decode_steps, args.warmup)
        print("decode done", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(workloads, inp, cfg)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
