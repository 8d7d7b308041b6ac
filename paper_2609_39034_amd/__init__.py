"""SwiLA hot path for MI355X (gfx950): Python binding of libswila.so.

The binding only marshals arguments: it checks tensors, allocates outputs
with torch (device memory), and calls the C ABI declared in
``include/swila.h`` with raw device pointers and the current HIP stream.
Every step of the layer runs in the library's HIP kernels.  There is no
fallback: if ``libswila.so`` is missing or fails to load, importing the
library raises.

Entry points (names as in the C ABI):
  ``forward``            whole sequences       -> swila_forward
  ``forward_noalloc``    the same, allocating nothing -> swila_forward_noalloc
  ``decode_step``        one token per sequence -> swila_decode_step
  ``forward_temporal``, ``decode_step_temporal``  Temporal SwiLA (App. B.3)
                                                -> swila_forward_temporal, ...
  ``forward_gated``, ``decode_step_gated``      Gated SwiLA (App. B.4)
                                                -> swila_forward_gated, ...
  ``state_init``         initial state          -> swila_state_init
  ``state_bytes``, ``forward_workspace_bytes``, ``version``
"""
from __future__ import annotations

import ctypes
import os

__all__ = ["forward", "forward_noalloc", "NOALLOC_SCRATCH_BYTES", "decode_step", "forward_temporal", "decode_step_temporal",
           "forward_gated", "decode_step_gated", "backward", "backward_workspace_bytes",
           "state_init", "state_bytes", "forward_workspace_bytes",
           "version", "library_path", "SwilaError", "F32", "BF16", "ALGO_AUTO",
           "ALGO_RECURRENT", "ALGO_CHUNK_EXACT", "ALGO_NEWTON", "FLAG_NEWTON_NO_CLAMP",
           "FLAG_NEWTON_SYNC", "FLAG_UNNORMALIZED", "ENOTCONVERGED"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libswila.so")

F32, BF16 = 0, 1
ALGO_AUTO, ALGO_RECURRENT, ALGO_CHUNK_EXACT, ALGO_NEWTON = 0, 1, 2, 3
_ALGOS = {"auto": ALGO_AUTO, "recurrent": ALGO_RECURRENT, "chunk": ALGO_CHUNK_EXACT,
          "newton": ALGO_NEWTON}
FLAG_NEWTON_NO_CLAMP, FLAG_NEWTON_SYNC, FLAG_UNNORMALIZED = 1, 2, 4

OK, EINVAL, EUNSUPPORTED, EHIP, ENOTCONVERGED = 0, -1, -2, -3, -4


class SwilaError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("swila error %d: %s" % (code, msg))
        self.code = code


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "H", "T", "Dk", "Dv", "J")]


class Opts(ctypes.Structure):
    _fields_ = [("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("algo", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("max_iters", ctypes.c_int32), ("tol", ctypes.c_float),
                ("flags", ctypes.c_uint32)]


class Temporal(ctypes.Structure):
    _fields_ = [("gate_k_logit", ctypes.c_void_p), ("gate_q_logit", ctypes.c_void_p),
                ("prior_in", ctypes.c_void_p), ("prior_out", ctypes.c_void_p)]


class Gated(ctypes.Structure):
    _fields_ = [("decay_logit", ctypes.c_void_p)]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """The ctypes handle of libswila.so (loaded once).  Raises if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError("libswila.so is not built (%s); run __graft_entry__.build() or "
                          "python -m paper_2609_39034_amd.build" % _LIB_PATH)
    lib = ctypes.CDLL(_LIB_PATH)
    vp, sp, op = ctypes.c_void_p, ctypes.POINTER(Shape), ctypes.POINTER(Opts)
    lib.swila_version.restype = ctypes.c_int
    lib.swila_version.argtypes = []
    lib.swila_last_error.restype = ctypes.c_char_p
    lib.swila_last_error.argtypes = []
    lib.swila_state_bytes.restype = ctypes.c_size_t
    lib.swila_state_bytes.argtypes = [sp]
    lib.swila_state_init.restype = ctypes.c_int
    lib.swila_state_init.argtypes = [sp, vp, vp, vp]
    lib.swila_forward_workspace_bytes.restype = ctypes.c_size_t
    lib.swila_forward_workspace_bytes.argtypes = [sp, op]
    lib.swila_forward.restype = ctypes.c_int
    lib.swila_forward.argtypes = [sp, op] + [vp] * 6 + [vp, vp, vp, vp, vp, ctypes.c_size_t, vp, vp]
    lib.swila_forward_noalloc.restype = ctypes.c_int
    lib.swila_forward_noalloc.argtypes = [sp, op] + [vp] * 6 + [vp, vp, vp, vp, vp, vp]
    lib.swila_decode_step.restype = ctypes.c_int
    lib.swila_decode_step.argtypes = [sp, op] + [vp] * 6 + [vp, vp, vp, vp]
    tp = ctypes.POINTER(Temporal)
    lib.swila_forward_temporal.restype = ctypes.c_int
    lib.swila_forward_temporal.argtypes = [sp, op] + [vp] * 6 + [tp, vp, vp, vp, vp, vp]
    lib.swila_decode_step_temporal.restype = ctypes.c_int
    lib.swila_decode_step_temporal.argtypes = [sp, op] + [vp] * 6 + [tp, vp, vp, vp, vp]
    gp = ctypes.POINTER(Gated)
    lib.swila_forward_gated.restype = ctypes.c_int
    lib.swila_forward_gated.argtypes = [sp, op] + [vp] * 6 + [gp, tp, vp, vp, vp, vp, vp]
    lib.swila_decode_step_gated.restype = ctypes.c_int
    lib.swila_decode_step_gated.argtypes = [sp, op] + [vp] * 6 + [gp, tp, vp, vp, vp, vp]
    lib.swila_backward_workspace_bytes.restype = ctypes.c_size_t
    lib.swila_backward_workspace_bytes.argtypes = [sp]
    lib.swila_backward.restype = ctypes.c_int
    lib.swila_backward.argtypes = [sp, op] + [vp] * 6 + [vp, vp, vp] + [vp] * 7 + [
        vp, ctypes.c_size_t, vp]
    _lib = lib
    return lib


def _check(rc):
    if rc != OK:
        raise SwilaError(rc, load_library().swila_last_error().decode(errors="replace"))


def version() -> int:
    return load_library().swila_version()


def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError("inputs must be float32 or bfloat16, got %s" % t.dtype)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev_tensor(t, name, dtype=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return t


def _expect_shape(t, shape, name):
    """ValueError unless the tensor ``t`` has ``shape``; None, True and False
    (allocate or discard) pass.  Called before any device check, so a wrong
    size is reported before anything reaches the library."""
    if t is None or t is True or t is False:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))


_IN_NAMES = ("q", "k", "v", "beta_logit", "prior_k_logit", "prior_q_logit")


def _input_shapes(B, H, T, Dk, Dv, J, decode):
    if decode:
        return {"q": (B, H, Dk), "k": (B, H, Dk), "v": (B, H, Dv), "beta_logit": (B, H, J, Dv),
                "prior_k_logit": (B, H, J, Dv), "prior_q_logit": (B, H, J, Dv)}
    return {"q": (B, T, H, Dk), "k": (B, T, H, Dk), "v": (B, T, H, Dv),
            "beta_logit": (B, T, H, J, Dv), "prior_k_logit": (B, T, H, J, Dv),
            "prior_q_logit": (B, T, H, J, Dv)}


def _check_layer(tensors, decode, o=None, state_in=None, state_out=None):
    """Shape checks of one call (inputs, state_in, o, state_out), then device,
    layout and dtype checks of the inputs.  Returns (inputs, dtype code,
    (B, H, T, Dk, Dv, J))."""
    q, v, lb = tensors[0], tensors[2], tensors[3]
    B, H, T, Dk, Dv, J = _layer_shapes(q, v, lb, decode=decode)
    expect = _input_shapes(B, H, T, Dk, Dv, J, decode)
    for t, n in zip(tensors, _IN_NAMES):
        _expect_shape(t, expect[n], n)
    _expect_shape(state_in, (B, H, J, Dk, Dv), "state_in")
    _expect_shape(state_out, (B, H, J, Dk, Dv), "state_out")
    _expect_shape(o, (B, H, Dv) if decode else (B, T, H, Dv), "o")
    ins = [_dev_tensor(t, n) for t, n in zip(tensors, _IN_NAMES)]
    code = _dtype_code(q)
    for t, n in zip(ins, _IN_NAMES):
        if _dtype_code(t) != code:
            raise TypeError("%s has dtype %s but q has %s" % (n, t.dtype, q.dtype))
    return ins, code, (B, H, T, Dk, Dv, J)


def state_bytes(B, H, Dk, Dv, J) -> int:
    return load_library().swila_state_bytes(ctypes.byref(Shape(B, H, 0, Dk, Dv, J)))


def forward_workspace_bytes(B, H, T, Dk, Dv, J, *, in_dtype=BF16, out_dtype=None,
                            algo="auto", chunk=0) -> int:
    """Workspace bytes of swila_forward for this shape and algorithm."""
    opts = Opts(in_dtype, in_dtype if out_dtype is None else out_dtype, _ALGOS[algo], chunk,
                0, 0.0, 0)
    return load_library().swila_forward_workspace_bytes(ctypes.byref(Shape(B, H, T, Dk, Dv, J)),
                                                         ctypes.byref(opts))


def state_init(state, src=None, *, stream=None):
    """state [B,H,J,Dk,Dv] float32 <- copy of src, or zeros when src is None."""
    torch = _torch()
    _dev_tensor(state, "state", torch.float32)
    _dev_tensor(src, "src", torch.float32)
    if state.dim() != 5:
        raise ValueError("state must be [B,H,J,Dk,Dv]")
    if src is not None and src.shape != state.shape:
        raise ValueError("src shape %s != state shape %s" % (tuple(src.shape), tuple(state.shape)))
    B, H, J, Dk, Dv = state.shape
    _check(load_library().swila_state_init(ctypes.byref(Shape(B, H, 0, Dk, Dv, J)), _ptr(state),
                                           _ptr(src), _stream_handle(stream)))
    return state


def _layer_shapes(q, v, lb, decode):
    if decode:
        B, H, Dk = q.shape
        T = 1
        Dv = v.shape[-1]
        J = lb.shape[2]
    else:
        B, T, H, Dk = q.shape
        Dv = v.shape[-1]
        J = lb.shape[3]
    return B, H, T, Dk, Dv, J


def forward(q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in=None, *,
            state_out=True, o=None, out_dtype=None, resp=False, algo="auto", chunk=0,
            workspace=None, max_iters=0, tol=0.0, clamp=True, iters_out=None,
            sync_status=False, unnormalized=False, stream=None):
    """Forward over whole sequences (swila_forward).

    q, k [B,T,H,Dk]; v [B,T,H,Dv]; logits [B,T,H,J,Dv] (one dtype: float32 or
    bfloat16); state_in [B,H,J,Dk,Dv] float32 or None (zeros).
    state_out: True to allocate the final state, False to discard it, or a
    float32 tensor to write (may be state_in itself).  o: optional output
    tensor; out_dtype defaults to the input dtype.  resp=True also returns the
    key-side responsibilities [B,T,H,J,Dv] float32.
    algo: "auto", "recurrent", "chunk" or "newton" (App. D).  For "newton":
    max_iters (0 = 64), tol (0 = 1e-3, < 0 = exactly max_iters sweeps), clamp
    (g clamped to [0, 2/|k|^2]), iters_out (None or a device int32 tensor of 2
    elements: most sweeps of any block, blocks not converged); the workspace
    is allocated here unless given.  sync_status=True (needs iters_out) waits
    for the launch and raises SwilaError with code ENOTCONVERGED when some
    block did not meet tol.  unnormalized=True (algo "newton" only) evaluates
    App. D.2's variant with responsibilities r = pi^k exp(-delta^2/2).
    Returns (o, state_out or None) or (o, state_out, resp).
    """
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), False, o=o, state_in=state_in,
        state_out=state_out)
    _dev_tensor(state_in, "state_in", torch.float32)
    odt = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, T, H, Dv), device=q.device, dtype=odt)
    _dev_tensor(o, "o")
    if state_out is True:
        s_out = torch.empty((B, H, J, Dk, Dv), device=q.device, dtype=torch.float32)
    elif state_out is False or state_out is None:
        s_out = None
    else:
        s_out = _dev_tensor(state_out, "state_out", torch.float32)
    r = None
    if resp:
        r = torch.empty((B, T, H, J, Dv), device=q.device, dtype=torch.float32)
    flags = ((0 if clamp else FLAG_NEWTON_NO_CLAMP) | (FLAG_NEWTON_SYNC if sync_status else 0)
             | (FLAG_UNNORMALIZED if unnormalized else 0))
    opts = Opts(code, _dtype_code(o), _ALGOS[algo], int(chunk), int(max_iters), float(tol),
                flags)
    shape = Shape(B, H, T, Dk, Dv, J)
    lib = load_library()
    if workspace is None:
        need = lib.swila_forward_workspace_bytes(ctypes.byref(shape), ctypes.byref(opts))
        if need:
            workspace = torch.empty(need, device=q.device, dtype=torch.uint8)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        _dev_tensor(workspace, "workspace")
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    if iters_out is not None:
        _dev_tensor(iters_out, "iters_out", torch.int32)
        if iters_out.numel() < 2:
            raise ValueError("iters_out needs 2 int32 elements")
    _check(lib.swila_forward(
        ctypes.byref(shape), ctypes.byref(opts),
        *[_ptr(t) for t in ins], _ptr(state_in), _ptr(s_out), _ptr(o), _ptr(r),
        ws_ptr, ws_bytes, _ptr(iters_out), _stream_handle(stream)))
    return (o, s_out, r) if resp else (o, s_out)


NOALLOC_SCRATCH_BYTES = 64 << 20


def forward_noalloc(q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in, o, *,
                    state_out=None, resp=None, algo="auto", chunk=0, max_iters=0, tol=0.0,
                    clamp=True, iters_out=None, sync_status=False, unnormalized=False,
                    stream=None):
    """swila_forward_noalloc: ``forward`` for callers that cannot allocate.  The
    caller passes every output (o [B,T,H,Dv]; state_out and resp tensors or
    None; iters_out as for ``forward``); nothing is allocated here or in the
    library, whose App. D form uses a scratch array of NOALLOC_SCRATCH_BYTES
    per GPU (larger calls raise with code EUNSUPPORTED).  Calls that overlap on
    one GPU share that array and race.  Returns (o, state_out)."""
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), False, o=o, state_in=state_in,
        state_out=state_out)
    _expect_shape(resp, (B, T, H, J, Dv), "resp")
    _dev_tensor(state_in, "state_in", torch.float32)
    _dev_tensor(o, "o")
    _dev_tensor(state_out, "state_out", torch.float32)
    _dev_tensor(resp, "resp", torch.float32)
    if iters_out is not None:
        _dev_tensor(iters_out, "iters_out", torch.int32)
        if iters_out.numel() < 2:
            raise ValueError("iters_out needs 2 int32 elements")
    flags = ((0 if clamp else FLAG_NEWTON_NO_CLAMP) | (FLAG_NEWTON_SYNC if sync_status else 0)
             | (FLAG_UNNORMALIZED if unnormalized else 0))
    opts = Opts(code, _dtype_code(o), _ALGOS[algo], int(chunk), int(max_iters), float(tol),
                flags)
    _check(load_library().swila_forward_noalloc(
        ctypes.byref(Shape(B, H, T, Dk, Dv, J)), ctypes.byref(opts), *[_ptr(t) for t in ins],
        _ptr(state_in), _ptr(state_out), _ptr(o), _ptr(resp), _ptr(iters_out),
        _stream_handle(stream)))
    return o, state_out


def backward_workspace_bytes(B, H, T, Dk, Dv, J) -> int:
    shape = Shape(B, H, T, Dk, Dv, J)
    return int(load_library().swila_backward_workspace_bytes(ctypes.byref(shape)))


def backward(q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in, grad_o,
             grad_state=None, *, grad_state_in=True, workspace=None, stream=None):
    """Gradients of the plain forward (swila_backward).

    The forward's inputs as for ``forward`` (state_in may be None), grad_o =
    dL/do [B,T,H,Dv] (its dtype is the forward's output dtype), grad_state =
    dL/dW_T float32 or None.  Returns (dq, dk, dv, dbeta_logit, dprior_k_logit,
    dprior_q_logit, dstate_in), every gradient float32 (dstate_in None when
    grad_state_in is False).  The workspace is allocated here unless given.
    """
    torch = _torch()
    B, H, T, Dk, Dv, J = _layer_shapes(q, v, beta_logit, decode=False)
    _expect_shape(grad_state, (B, H, J, Dk, Dv), "grad_state")
    _expect_shape(grad_o, (B, T, H, Dv), "grad_o")
    ins, code, _ = _check_layer((q, k, v, beta_logit, prior_k_logit, prior_q_logit), False,
                                state_in=state_in)
    _dev_tensor(state_in, "state_in", torch.float32)
    _dev_tensor(grad_state, "grad_state", torch.float32)
    _dev_tensor(grad_o, "grad_o")
    f32 = dict(device=q.device, dtype=torch.float32)
    grads = [torch.empty((B, T, H, Dk), **f32), torch.empty((B, T, H, Dk), **f32),
             torch.empty((B, T, H, Dv), **f32)] + [
        torch.empty((B, T, H, J, Dv), **f32) for _ in range(3)]
    ds = torch.empty((B, H, J, Dk, Dv), **f32) if grad_state_in else None
    shape = Shape(B, H, T, Dk, Dv, J)
    opts = Opts(code, _dtype_code(grad_o), _ALGOS["auto"], 0, 0, 0.0, 0)
    lib = load_library()
    if workspace is None:
        workspace = torch.empty(max(1, lib.swila_backward_workspace_bytes(ctypes.byref(shape))),
                                device=q.device, dtype=torch.uint8)
    _dev_tensor(workspace, "workspace")
    _check(lib.swila_backward(
        ctypes.byref(shape), ctypes.byref(opts), *[_ptr(t) for t in ins], _ptr(state_in),
        _ptr(grad_o), _ptr(grad_state), *[_ptr(t) for t in grads], _ptr(ds),
        _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream_handle(stream)))
    return tuple(grads) + (ds,)


def decode_step(q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in, *,
                state_out=None, o=None, out_dtype=None, stream=None):
    """One token per sequence (swila_decode_step).

    q, k [B,H,Dk]; v [B,H,Dv]; logits [B,H,J,Dv]; state_in [B,H,J,Dk,Dv]
    float32 (None = zeros).  state_out defaults to state_in (updated in place;
    with state_in None a new tensor is allocated).  Returns (o, state_out).
    """
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), True, o=o, state_in=state_in,
        state_out=state_out)
    _dev_tensor(state_in, "state_in", torch.float32)
    if state_out is None:
        state_out = state_in if state_in is not None else torch.empty(
            (B, H, J, Dk, Dv), device=q.device, dtype=torch.float32)
    _dev_tensor(state_out, "state_out", torch.float32)
    odt = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, Dv), device=q.device, dtype=odt)
    _dev_tensor(o, "o")
    opts = Opts(code, _dtype_code(o), ALGO_AUTO, 0, 0, 0.0, 0)
    _check(load_library().swila_decode_step(
        ctypes.byref(Shape(B, H, 1, Dk, Dv, J)), ctypes.byref(opts),
        *[_ptr(t) for t in ins], _ptr(state_in), _ptr(state_out), _ptr(o),
        _stream_handle(stream)))
    return o, state_out


def _temporal_args(gate_k_logit, gate_q_logit, prior_in, prior_out, code, gate_shape,
                   prior_shape, device):
    """Checks the temporal tensors; allocates prior_out when it is True."""
    torch = _torch()
    for t, n in ((gate_k_logit, "gate_k_logit"), (gate_q_logit, "gate_q_logit")):
        if t is None:
            raise ValueError("%s is required" % n)
        _expect_shape(t, gate_shape, n)
    _expect_shape(prior_in, prior_shape, "prior_in")
    _expect_shape(prior_out, prior_shape, "prior_out")
    for t, n in ((gate_k_logit, "gate_k_logit"), (gate_q_logit, "gate_q_logit")):
        _dev_tensor(t, n)
        if _dtype_code(t) != code:
            raise TypeError("%s must have the dtype of q" % n)
    _dev_tensor(prior_in, "prior_in", torch.float32)
    if prior_out is True:
        prior_out = torch.empty(prior_shape, device=device, dtype=torch.float32)
    elif prior_out is False or prior_out is None:
        prior_out = None
    else:
        _dev_tensor(prior_out, "prior_out", torch.float32)
    tp = Temporal(gate_k_logit.data_ptr(), gate_q_logit.data_ptr(),
                  None if prior_in is None else prior_in.data_ptr(),
                  None if prior_out is None else prior_out.data_ptr())
    return tp, prior_out


def forward_temporal(q, k, v, beta_logit, prior_k_logit, prior_q_logit, gate_k_logit,
                     gate_q_logit, state_in=None, prior_in=None, *, state_out=True,
                     prior_out=True, o=None, out_dtype=None, resp=False, algo="auto",
                     stream=None):
    """Temporal SwiLA forward (swila_forward_temporal; Sec. 3.3, App. B.3).

    The arguments of ``forward`` plus the gate logits gate_k_logit,
    gate_q_logit [B,T,H,Dv] (the dtype of q) and the prior state prior_in
    [B,H,2,J,Dv] float32 (part 0: r_{t-1}, part 1: rhobar_{t-1}; None = 1/J).
    prior_out: True to allocate, False to discard, or a float32 tensor (may be
    prior_in).  algo: "auto" or "recurrent".
    Returns (o, state_out, prior_out) or (o, state_out, prior_out, resp).
    """
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), False, o=o, state_in=state_in,
        state_out=state_out)
    _dev_tensor(state_in, "state_in", torch.float32)
    tp, p_out = _temporal_args(gate_k_logit, gate_q_logit, prior_in, prior_out, code,
                               (B, T, H, Dv), (B, H, 2, J, Dv), q.device)
    odt = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, T, H, Dv), device=q.device, dtype=odt)
    _dev_tensor(o, "o")
    if state_out is True:
        s_out = torch.empty((B, H, J, Dk, Dv), device=q.device, dtype=torch.float32)
    elif state_out is False or state_out is None:
        s_out = None
    else:
        s_out = _dev_tensor(state_out, "state_out", torch.float32)
    r = None
    if resp:
        r = torch.empty((B, T, H, J, Dv), device=q.device, dtype=torch.float32)
    opts = Opts(code, _dtype_code(o), _ALGOS[algo], 0, 0, 0.0, 0)
    _check(load_library().swila_forward_temporal(
        ctypes.byref(Shape(B, H, T, Dk, Dv, J)), ctypes.byref(opts),
        *[_ptr(t) for t in ins], ctypes.byref(tp), _ptr(state_in), _ptr(s_out), _ptr(o), _ptr(r),
        _stream_handle(stream)))
    return (o, s_out, p_out, r) if resp else (o, s_out, p_out)


def decode_step_temporal(q, k, v, beta_logit, prior_k_logit, prior_q_logit, gate_k_logit,
                         gate_q_logit, state_in, prior_in, *, state_out=None, prior_out=None,
                         o=None, out_dtype=None, stream=None):
    """One Temporal SwiLA token per sequence (swila_decode_step_temporal).

    The arguments of ``decode_step`` plus gate logits [B,H,Dv] and the prior
    state prior_in [B,H,2,J,Dv] float32 (None = 1/J).  state_out and prior_out
    default to the inputs (updated in place), or to new tensors when those are
    None.  Returns (o, state_out, prior_out).
    """
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), True, o=o, state_in=state_in,
        state_out=state_out)
    _dev_tensor(state_in, "state_in", torch.float32)
    if state_out is None:
        state_out = state_in if state_in is not None else torch.empty(
            (B, H, J, Dk, Dv), device=q.device, dtype=torch.float32)
    _dev_tensor(state_out, "state_out", torch.float32)
    if prior_out is None:
        prior_out = prior_in if prior_in is not None else True
    tp, p_out = _temporal_args(gate_k_logit, gate_q_logit, prior_in, prior_out, code,
                               (B, H, Dv), (B, H, 2, J, Dv), q.device)
    odt = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, Dv), device=q.device, dtype=odt)
    _dev_tensor(o, "o")
    opts = Opts(code, _dtype_code(o), ALGO_AUTO, 0, 0, 0.0, 0)
    _check(load_library().swila_decode_step_temporal(
        ctypes.byref(Shape(B, H, 1, Dk, Dv, J)), ctypes.byref(opts),
        *[_ptr(t) for t in ins], ctypes.byref(tp), _ptr(state_in), _ptr(state_out), _ptr(o),
        _stream_handle(stream)))
    return o, state_out, p_out


def _gated_arg(decay_logit, code, shape):
    _expect_shape(decay_logit, shape, "decay_logit")
    _dev_tensor(decay_logit, "decay_logit")
    if _dtype_code(decay_logit) != code:
        raise TypeError("decay_logit must have the dtype of q")
    return Gated(decay_logit.data_ptr())


def forward_gated(q, k, v, beta_logit, prior_k_logit, prior_q_logit, decay_logit,
                  state_in=None, *, gate_k_logit=None, gate_q_logit=None, prior_in=None,
                  prior_out=True, state_out=True, o=None, out_dtype=None, resp=False,
                  algo="auto", stream=None):
    """Gated SwiLA forward (swila_forward_gated; Sec. 3.4, App. B.4, eq. pre-decay).

    The arguments of ``forward`` plus decay_logit [B,T,H,J,Dk] (the dtype of q;
    a = sigmoid, one gate per key dimension and component).  With gate_k_logit
    and gate_q_logit the priors are the temporal ones of ``forward_temporal``
    (Gated Temporal SwiLA), with prior_in / prior_out as there.
    Returns (o, state_out[, prior_out][, resp]).
    """
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), False, o=o, state_in=state_in,
        state_out=state_out)
    _dev_tensor(state_in, "state_in", torch.float32)
    gd = _gated_arg(decay_logit, code, (B, T, H, J, Dk))
    temporal = gate_k_logit is not None or gate_q_logit is not None
    tp, p_out = None, None
    if temporal:
        tp, p_out = _temporal_args(gate_k_logit, gate_q_logit, prior_in, prior_out, code,
                                   (B, T, H, Dv), (B, H, 2, J, Dv), q.device)
    odt = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, T, H, Dv), device=q.device, dtype=odt)
    _dev_tensor(o, "o")
    if state_out is True:
        s_out = torch.empty((B, H, J, Dk, Dv), device=q.device, dtype=torch.float32)
    elif state_out is False or state_out is None:
        s_out = None
    else:
        s_out = _dev_tensor(state_out, "state_out", torch.float32)
    r = torch.empty((B, T, H, J, Dv), device=q.device, dtype=torch.float32) if resp else None
    opts = Opts(code, _dtype_code(o), _ALGOS[algo], 0, 0, 0.0, 0)
    _check(load_library().swila_forward_gated(
        ctypes.byref(Shape(B, H, T, Dk, Dv, J)), ctypes.byref(opts),
        *[_ptr(t) for t in ins], ctypes.byref(gd), ctypes.byref(tp) if tp is not None else None,
        _ptr(state_in), _ptr(s_out), _ptr(o), _ptr(r), _stream_handle(stream)))
    out = (o, s_out)
    if temporal:
        out = out + (p_out,)
    if resp:
        out = out + (r,)
    return out


def decode_step_gated(q, k, v, beta_logit, prior_k_logit, prior_q_logit, decay_logit, state_in,
                      *, gate_k_logit=None, gate_q_logit=None, prior_in=None, prior_out=None,
                      state_out=None, o=None, out_dtype=None, stream=None):
    """One Gated SwiLA token per sequence (swila_decode_step_gated): the arguments
    of ``decode_step`` plus decay_logit [B,H,J,Dk], and optionally the temporal
    gates [B,H,Dv] with the prior state.  state_out and prior_out default to the
    inputs (updated in place).  Returns (o, state_out[, prior_out])."""
    torch = _torch()
    ins, code, (B, H, T, Dk, Dv, J) = _check_layer(
        (q, k, v, beta_logit, prior_k_logit, prior_q_logit), True, o=o, state_in=state_in,
        state_out=state_out)
    _dev_tensor(state_in, "state_in", torch.float32)
    if state_out is None:
        state_out = state_in if state_in is not None else torch.empty(
            (B, H, J, Dk, Dv), device=q.device, dtype=torch.float32)
    _dev_tensor(state_out, "state_out", torch.float32)
    gd = _gated_arg(decay_logit, code, (B, H, J, Dk))
    temporal = gate_k_logit is not None or gate_q_logit is not None
    tp, p_out = None, None
    if temporal:
        if prior_out is None:
            prior_out = prior_in if prior_in is not None else True
        tp, p_out = _temporal_args(gate_k_logit, gate_q_logit, prior_in, prior_out, code,
                                   (B, H, Dv), (B, H, 2, J, Dv), q.device)
    odt = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, Dv), device=q.device, dtype=odt)
    _dev_tensor(o, "o")
    opts = Opts(code, _dtype_code(o), ALGO_AUTO, 0, 0, 0.0, 0)
    _check(load_library().swila_decode_step_gated(
        ctypes.byref(Shape(B, H, 1, Dk, Dv, J)), ctypes.byref(opts),
        *[_ptr(t) for t in ins], ctypes.byref(gd), ctypes.byref(tp) if tp is not None else None,
        _ptr(state_in), _ptr(state_out), _ptr(o), _stream_handle(stream)))
    return (o, state_out, p_out) if temporal else (o, state_out)
