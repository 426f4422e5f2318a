"""Python binding of the C ABI in ``include/ssd.h`` (argument marshalling only).

Every step of the forward runs in the HIP kernels of ``libssd_hip.so``; this
module only turns torch tensors into device pointers and the current HIP stream
into a ``hipStream_t``.  There is no CPU fallback: if the library is missing
or cannot be loaded, every call raises.

Names mirror the ABI: :func:`ssd_workspace_bytes`, :func:`ssd_forward`,
:func:`ssd_forward_block`, :func:`ssd_decode_step`, :func:`ssd_error_string`;
:func:`forward` is the tensor-level convenience wrapper returning
``(y, final_states)`` like the paper's ``ssd(X, A, B, C, block_len,
initial_states)``, :func:`forward_block` the same with the block steps around
the layer, :func:`decode_step` one recurrent step.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libssd_hip.so")

SSD_DTYPE_F32 = 0
SSD_DTYPE_BF16 = 1
SSD_OK = 0
SSD_ERR_NULL_ARG = -1
SSD_ERR_BAD_SHAPE = -2
SSD_ERR_BAD_CHUNK = -3
SSD_ERR_BAD_DTYPE = -4
SSD_ERR_UNSUPPORTED_DIMS = -5
SSD_ERR_SEQIDX_BATCH = -6
SSD_ERR_WORKSPACE = -7
SSD_ERR_LAUNCH = -8
SSD_ERR_TOO_LARGE = -9
SSD_ERR_BAD_OPTION = -10
SSD_ERR_STATE_TIMEOUT = -11
SSD_ERR_SCRATCH_TOO_SMALL = -12
SSD_NOALLOC_SCRATCH_BYTES = 64 << 20

EXPORTED = ("ssd_workspace_bytes", "ssd_forward", "ssd_forward_timed", "ssd_decode_step",
            "ssd_block_workspace_bytes", "ssd_forward_block", "ssd_forward_block_timed",
            "ssd_span_decay", "ssd_span_combine", "ssd_span_correct_workspace_bytes", "ssd_span_correct",
            "ssd_backward_workspace_bytes", "ssd_backward", "ssd_backward_timed",
            "ssd_backward_varlen_workspace_bytes", "ssd_backward_varlen",
            "ssd_forward_varlen_workspace_bytes", "ssd_forward_varlen",
            "ssd_backward_block_workspace_bytes", "ssd_backward_block", "ssd_workspace_status",
            "ssd_set_tuning", "ssd_forward_noalloc", "ssd_error_string")


class SsdProblem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64),
        ("seqlen", ctypes.c_int64),
        ("nheads", ctypes.c_int64),
        ("headdim", ctypes.c_int64),
        ("dstate", ctypes.c_int64),
        ("ngroups", ctypes.c_int64),
        ("chunk_size", ctypes.c_int64),
        ("nseq", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
    ]


class SsdBlockOpts(ctypes.Structure):
    _fields_ = [
        ("dt_bias", ctypes.c_void_p),
        ("dt_softplus", ctypes.c_int32),
        ("dt_min", ctypes.c_float),
        ("dt_max", ctypes.c_float),
        ("z", ctypes.c_void_p),
        ("norm_weight", ctypes.c_void_p),
        ("norm_group_size", ctypes.c_int64),
        ("norm_eps", ctypes.c_float),
    ]


class SsdError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__("%s failed: %s (%d)" % (where, ssd_error_string(code), code))


_lib = None


def load_library(path: str = LIB_PATH):
    """Load ``libssd_hip.so`` (built by ``paper_2405_21060_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            "HIP library %s is missing: build it with `python -m paper_2405_21060_amd.build` "
            "(there is no CPU fallback)" % path)
    lib = ctypes.CDLL(path)
    vp = ctypes.c_void_p
    lib.ssd_workspace_bytes.restype = ctypes.c_int
    lib.ssd_workspace_bytes.argtypes = [ctypes.POINTER(SsdProblem), ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_forward.restype = ctypes.c_int
    lib.ssd_forward.argtypes = [ctypes.POINTER(SsdProblem)] + [vp] * 10 + [vp, ctypes.c_size_t, vp]
    lib.ssd_forward_timed.restype = ctypes.c_int
    lib.ssd_forward_timed.argtypes = lib.ssd_forward.argtypes + [vp, vp]
    lib.ssd_decode_step.restype = ctypes.c_int
    lib.ssd_decode_step.argtypes = [ctypes.POINTER(SsdProblem)] + [vp] * 9
    lib.ssd_block_workspace_bytes.restype = ctypes.c_int
    lib.ssd_block_workspace_bytes.argtypes = [ctypes.POINTER(SsdProblem), ctypes.POINTER(SsdBlockOpts),
                                              ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_forward_block.restype = ctypes.c_int
    lib.ssd_forward_block.argtypes = [ctypes.POINTER(SsdProblem), ctypes.POINTER(SsdBlockOpts)] + [vp] * 10 + [
        vp, ctypes.c_size_t, vp]
    lib.ssd_forward_block_timed.restype = ctypes.c_int
    lib.ssd_forward_block_timed.argtypes = lib.ssd_forward_block.argtypes + [vp, vp]
    pp = ctypes.POINTER(SsdProblem)
    lib.ssd_span_decay.restype = ctypes.c_int
    lib.ssd_span_decay.argtypes = [pp, vp, vp, vp, vp]
    lib.ssd_span_combine.restype = ctypes.c_int
    lib.ssd_span_combine.argtypes = [ctypes.c_int64, pp, vp, vp, vp, vp, vp, vp]
    lib.ssd_span_correct_workspace_bytes.restype = ctypes.c_int
    lib.ssd_span_correct_workspace_bytes.argtypes = [pp, ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_span_correct.restype = ctypes.c_int
    lib.ssd_span_correct.argtypes = [pp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.ssd_error_string.restype = ctypes.c_char_p
    lib.ssd_backward_workspace_bytes.argtypes = [pp, ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_backward_workspace_bytes.restype = ctypes.c_int
    lib.ssd_backward.argtypes = [pp] + [vp] * 16 + [vp, ctypes.c_size_t, vp]
    lib.ssd_backward.restype = ctypes.c_int
    lib.ssd_backward_timed.argtypes = lib.ssd_backward.argtypes + [vp, vp]
    lib.ssd_backward_timed.restype = ctypes.c_int
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.ssd_backward_varlen_workspace_bytes.argtypes = [pp, i64p, ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_backward_varlen_workspace_bytes.restype = ctypes.c_int
    lib.ssd_backward_varlen.argtypes = [pp, i64p] + [vp] * 16 + [vp, ctypes.c_size_t, vp]
    lib.ssd_backward_varlen.restype = ctypes.c_int
    lib.ssd_forward_varlen_workspace_bytes.argtypes = [pp, i64p, ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_forward_varlen_workspace_bytes.restype = ctypes.c_int
    lib.ssd_forward_varlen.argtypes = [pp, i64p] + [vp] * 9 + [vp, ctypes.c_size_t, vp]
    lib.ssd_forward_varlen.restype = ctypes.c_int
    lib.ssd_backward_block_workspace_bytes.argtypes = [pp, ctypes.POINTER(SsdBlockOpts),
                                                       ctypes.POINTER(ctypes.c_size_t)]
    lib.ssd_backward_block_workspace_bytes.restype = ctypes.c_int
    lib.ssd_backward_block.argtypes = [pp, ctypes.POINTER(SsdBlockOpts)] + [vp] * 19 + [vp, ctypes.c_size_t, vp]
    lib.ssd_backward_block.restype = ctypes.c_int
    lib.ssd_error_string.argtypes = [ctypes.c_int]
    lib.ssd_workspace_status.argtypes = [vp, vp]
    lib.ssd_workspace_status.restype = ctypes.c_int
    lib.ssd_set_tuning.argtypes = [ctypes.c_char_p, ctypes.c_int64]
    lib.ssd_set_tuning.restype = ctypes.c_int
    lib.ssd_forward_noalloc.argtypes = [ctypes.POINTER(SsdProblem)] + [vp] * 12
    lib.ssd_forward_noalloc.restype = ctypes.c_int
    _lib = lib
    return lib


def make_problem(batch, seqlen, nheads, headdim, dstate, ngroups, chunk_size, dtype, nseq=0):
    return SsdProblem(batch, seqlen, nheads, headdim, dstate, ngroups, chunk_size, nseq, dtype)


def ssd_workspace_bytes(prob: SsdProblem) -> int:
    out = ctypes.c_size_t(0)
    rc = load_library().ssd_workspace_bytes(ctypes.byref(prob), ctypes.byref(out))
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_workspace_bytes")
    return int(out.value)


def ssd_error_string(code: int) -> str:
    return load_library().ssd_error_string(int(code)).decode()


def ssd_workspace_status(workspace, stream) -> int:
    """Raw ABI call (integer device address and hipStream_t); returns the status."""
    return load_library().ssd_workspace_status(workspace, stream or None)


def ssd_set_tuning(name: str, value: int) -> int:
    """Raw ABI call; returns the status."""
    return load_library().ssd_set_tuning(name.encode(), int(value))


def workspace_status(workspace) -> int:
    """Status word of the last forward that used ``workspace`` (a device
    tensor), read after torch's current stream of its device has finished:
    ``SSD_OK`` or ``SSD_ERR_STATE_TIMEOUT``."""
    import torch

    stream = torch.cuda.current_stream(workspace.device).cuda_stream
    rc = ssd_workspace_status(workspace.data_ptr(), stream)
    if rc not in (SSD_OK, SSD_ERR_STATE_TIMEOUT):
        raise SsdError(rc, "ssd_workspace_status")
    return rc


class tuning:
    """Context manager over :func:`ssd_set_tuning`: ``with tuning(max_workgroups=3):``
    sets the given settings and puts each back to 0 (the library's own
    choice) on exit."""

    def __init__(self, **settings):
        self.settings = settings

    def __enter__(self):
        done = []
        for k, v in self.settings.items():
            rc = ssd_set_tuning(k, v)
            if rc != SSD_OK:
                for d in done:   # nothing stays set when one setting is refused
                    ssd_set_tuning(d, 0)
                raise SsdError(rc, "ssd_set_tuning(%s)" % k)
            done.append(k)
        return self

    def __exit__(self, *exc):
        for k in self.settings:
            ssd_set_tuning(k, 0)
        return False


def ssd_forward(prob: SsdProblem, x, dt, A_log, B, C, D, initial_states, seq_idx, y,
                final_states, workspace, workspace_bytes: int, stream) -> int:
    """Raw ABI call on integer device addresses (0 = NULL); returns the status."""
    return load_library().ssd_forward(
        ctypes.byref(prob), x, dt, A_log, B, C, D or None, initial_states or None,
        seq_idx or None, y, final_states or None, workspace, int(workspace_bytes),
        stream or None)


def ssd_forward_noalloc(prob: SsdProblem, x, dt, A_log, B, C, D, initial_states, seq_idx, y,
                        final_states, status, stream) -> int:
    """Raw ABI call on integer device addresses (0 = NULL): the forward on the
    library's fixed scratch array (no workspace); returns the status."""
    return load_library().ssd_forward_noalloc(
        ctypes.byref(prob), x, dt, A_log, B, C, D or None, initial_states or None,
        seq_idx or None, y, final_states or None, status or None, stream or None)


def ssd_forward_timed(prob: SsdProblem, x, dt, A_log, B, C, D, initial_states, seq_idx, y,
                      final_states, workspace, workspace_bytes: int, stream, event_begin,
                      event_end) -> int:
    """``ssd_forward`` that also records two hipEvent_t handles (integers, 0 =
    none) right before and after the dominant kernel; returns the status."""
    return load_library().ssd_forward_timed(
        ctypes.byref(prob), x, dt, A_log, B, C, D or None, initial_states or None,
        seq_idx or None, y, final_states or None, workspace, int(workspace_bytes),
        stream or None, event_begin or None, event_end or None)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _workspace(workspace, need: int, dev):
    """The caller's workspace (a uint8 device tensor of at least ``need``
    bytes; a smaller one is an error, so that its status word is the one the
    call writes), or a new one."""
    import torch

    if workspace is None:
        return torch.empty(max(int(need), 1), dtype=torch.uint8, device=dev)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError("workspace holds %d bytes, the call needs %d"
                         % (workspace.numel() * workspace.element_size(), need))
    return workspace


def ssd_forward_block(prob: SsdProblem, opts: SsdBlockOpts, x, dt, A_log, B, C, D, initial_states,
                      seq_idx, y, final_states, workspace, workspace_bytes: int, stream) -> int:
    """Raw ABI call on integer device addresses (0 = NULL); returns the status."""
    return load_library().ssd_forward_block(
        ctypes.byref(prob), ctypes.byref(opts), x, dt, A_log, B, C, D or None,
        initial_states or None, seq_idx or None, y, final_states or None, workspace,
        int(workspace_bytes), stream or None)


def ssd_forward_block_timed(prob: SsdProblem, opts: SsdBlockOpts, x, dt, A_log, B, C, D,
                            initial_states, seq_idx, y, final_states, workspace,
                            workspace_bytes: int, stream, event_begin, event_end) -> int:
    """``ssd_forward_block`` with the two events of ``ssd_forward_timed``."""
    return load_library().ssd_forward_block_timed(
        ctypes.byref(prob), ctypes.byref(opts), x, dt, A_log, B, C, D or None,
        initial_states or None, seq_idx or None, y, final_states or None, workspace,
        int(workspace_bytes), stream or None, event_begin or None, event_end or None)


def make_block_opts(dt_bias=None, dt_softplus: bool = True, dt_min: float = 0.0,
                    dt_max: float = float("inf"), z=None, norm_weight=None,
                    norm_group_size: int = 0, norm_eps: float = 1e-5) -> SsdBlockOpts:
    """Block options from tensors (or None) and scalars."""
    return SsdBlockOpts(_ptr(dt_bias), int(bool(dt_softplus)), float(dt_min), float(dt_max),
                        _ptr(z), _ptr(norm_weight), int(norm_group_size), float(norm_eps))


def _call(opts, x, dt, A_log, B, C, D, chunk_size, initial_states, seq_idx, nseq,
          return_final_states, workspace, out, final_out, extra=()):
    import torch

    dev = x.device
    if dev.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    if x.dtype == torch.bfloat16:
        dtype = SSD_DTYPE_BF16
    elif x.dtype == torch.float32:
        dtype = SSD_DTYPE_F32
    else:
        raise TypeError("x must be float32 or bfloat16")
    act = (("dt", dt), ("B", B), ("C", C)) + tuple((n, t) for n, t, f32 in extra if not f32)
    for name, t in act:
        if t is not None and t.dtype != x.dtype:
            raise TypeError("%s must have x's dtype" % name)
    f32s = (("A_log", A_log), ("D", D), ("initial_states", initial_states)) + tuple(
        (n, t) for n, t, f32 in extra if f32)
    for name, t in f32s:
        if t is not None and t.dtype != torch.float32:
            raise TypeError("%s must be float32" % name)
    if seq_idx is not None and seq_idx.dtype != torch.int32:
        raise TypeError("seq_idx must be int32")
    for t in (x, dt, A_log, B, C, D, initial_states, seq_idx) + tuple(t for _, t, _ in extra):
        if t is not None and (t.device != dev or not t.is_contiguous()):
            raise ValueError("all tensors must be contiguous and on x's device")
    b, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    if seq_idx is not None and nseq is None:
        nseq = int(seq_idx[0, -1].item()) + 1
    prob = make_problem(b, T, H, P, N, G, chunk_size, dtype, nseq or 0)
    wsb = ssd_workspace_bytes(prob)
    workspace = _workspace(workspace, wsb, dev)
    y = out if out is not None else torch.empty_like(x)
    units = nseq if seq_idx is not None else b
    fin = None
    if return_final_states:
        fin = final_out if final_out is not None else torch.empty(
            (units, H, P, N), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    args = (_ptr(x), _ptr(dt), _ptr(A_log), _ptr(B), _ptr(C), _ptr(D), _ptr(initial_states),
            _ptr(seq_idx), _ptr(y), _ptr(fin), _ptr(workspace), wsb, stream)
    if opts is None:
        rc, where = ssd_forward(prob, *args), "ssd_forward"
    else:
        rc, where = ssd_forward_block(prob, opts, *args), "ssd_forward_block"
    if rc != SSD_OK:
        raise SsdError(rc, where)
    return y, fin


def forward(x, dt, A_log, B, C, D=None, chunk_size: int = 256, initial_states=None,
            seq_idx=None, nseq: Optional[int] = None, return_final_states: bool = True,
            workspace=None, out=None, final_out=None) -> Tuple[object, object]:
    """SSD forward on device tensors; returns ``(y, final_states or None)``.

    x (b,T,H,P), dt (b,T,H), B/C (b,T,G,N): float32 or bfloat16, all the same
    dtype, contiguous, on one HIP device.  A_log, D (H): float32.
    initial_states (b|nseq,H,P,N) float32.  seq_idx (1,T) int32 with nseq
    sequences.  Launches on torch's current stream of x's device.
    """
    return _call(None, x, dt, A_log, B, C, D, chunk_size, initial_states, seq_idx, nseq,
                 return_final_states, workspace, out, final_out)


def forward_block(x, dt, A_log, B, C, D=None, chunk_size: int = 256, initial_states=None,
                  seq_idx=None, nseq: Optional[int] = None, dt_bias=None, dt_softplus: bool = True,
                  dt_min: float = 0.0, dt_max: float = float("inf"), z=None, norm_weight=None,
                  norm_group_size: int = 0, norm_eps: float = 1e-5,
                  return_final_states: bool = True, workspace=None, out=None,
                  final_out=None) -> Tuple[object, object]:
    """The layer with the block steps around it (``ssd_forward_block``):
    ``dt`` is the raw value (softplus of dt + dt_bias, clamped to
    [dt_min, dt_max]); the output is gated by SiLU(z) when ``z`` is given and
    RMS-normalised over groups of ``norm_group_size`` channels when that is
    positive.  z has x's dtype and shape; dt_bias (H) and norm_weight (H*P)
    are float32."""
    opts = make_block_opts(dt_bias, dt_softplus, dt_min, dt_max, z, norm_weight,
                           norm_group_size, norm_eps)
    return _call(opts, x, dt, A_log, B, C, D, chunk_size, initial_states, seq_idx, nseq,
                 return_final_states, workspace, out, final_out,
                 extra=(("z", z, False), ("dt_bias", dt_bias, True),
                        ("norm_weight", norm_weight, True)))


def ssd_decode_step(prob: SsdProblem, x, dt, A_log, B, C, D, state, y, stream) -> int:
    """Raw ABI call on integer device addresses (0 = NULL); returns the status."""
    return load_library().ssd_decode_step(
        ctypes.byref(prob), x, dt, A_log, B, C, D or None, state, y, stream or None)


def decode_step(x, dt, A_log, B, C, state, D=None, out=None):
    """One decode step on device tensors: updates ``state`` in place, returns y.

    x (b,H,P), dt (b,H), B/C (b,G,N): float32 or bfloat16, the same dtype,
    contiguous, on one HIP device.  A_log, D (H): float32.  state (b,H,P,N)
    float32.  Launches on torch's current stream of x's device.
    """
    import torch

    dev = x.device
    if dev.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    if x.dtype == torch.bfloat16:
        dtype = SSD_DTYPE_BF16
    elif x.dtype == torch.float32:
        dtype = SSD_DTYPE_F32
    else:
        raise TypeError("x must be float32 or bfloat16")
    for name, t in (("dt", dt), ("B", B), ("C", C)):
        if t.dtype != x.dtype:
            raise TypeError("%s must have x's dtype" % name)
    for name, t in (("A_log", A_log), ("D", D), ("state", state)):
        if t is not None and t.dtype != torch.float32:
            raise TypeError("%s must be float32" % name)
    for t in (x, dt, A_log, B, C, D, state):
        if t is not None and (t.device != dev or not t.is_contiguous()):
            raise ValueError("all tensors must be contiguous and on x's device")
    b, H, P = x.shape
    G, N = B.shape[1], B.shape[2]
    prob = make_problem(b, 1, H, P, N, G, 256, dtype, 0)
    y = out if out is not None else torch.empty_like(x)
    rc = ssd_decode_step(prob, _ptr(x), _ptr(dt), _ptr(A_log), _ptr(B), _ptr(C), _ptr(D),
                         _ptr(state), _ptr(y), torch.cuda.current_stream(dev).cuda_stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_decode_step")
    return y


def _span_problem(dt, C, P):
    import torch

    b, T, H = dt.shape
    G, N = C.shape[2], C.shape[3]
    dtype = SSD_DTYPE_BF16 if dt.dtype == torch.bfloat16 else SSD_DTYPE_F32
    return make_problem(b, T, H, P, N, G, 256, dtype, 0)


def span_decay(dt, A_log, P: int = 64, N: int = 16, out=None):
    """Total decay exp(A_h sum_t dt_t) of a span, (batch, nheads) float32.
    P and N only need to be valid layer dimensions (they play no part)."""
    import torch

    b, T, H = dt.shape
    prob = make_problem(b, T, H, P, N, 1, 256, SSD_DTYPE_BF16 if dt.dtype == torch.bfloat16 else SSD_DTYPE_F32, 0)
    out = out if out is not None else torch.empty((b, H), dtype=torch.float32, device=dt.device)
    rc = load_library().ssd_span_decay(ctypes.byref(prob), _ptr(dt), _ptr(A_log), _ptr(out),
                                       torch.cuda.current_stream(dt.device).cuda_stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_span_decay")
    return out


def span_combine(decays, local_finals, initial_states=None):
    """States entering every span and the final state, from per-span (decay,
    zero-state final state) pairs: decays (R, b, H), local_finals (R, b, H, P, N)."""
    import torch

    R, b, H, P, N = local_finals.shape
    prob = make_problem(b, 1, H, P, N, 1, 256, SSD_DTYPE_F32, 0)
    entering = torch.empty_like(local_finals)
    final = torch.empty_like(local_finals[0])
    rc = load_library().ssd_span_combine(R, ctypes.byref(prob), _ptr(decays), _ptr(local_finals),
                                         _ptr(initial_states), _ptr(entering), _ptr(final),
                                         torch.cuda.current_stream(local_finals.device).cuda_stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_span_combine")
    return entering, final


def span_correct(dt, A_log, C, entering, y, workspace=None):
    """y += the output the entering state (b, H, P, N) produces over the span
    (in place); dt (b, T, H), C (b, T, G, N), y (b, T, H, P)."""
    import torch

    prob = _span_problem(dt, C, y.shape[3])
    need = ctypes.c_size_t(0)
    rc = load_library().ssd_span_correct_workspace_bytes(ctypes.byref(prob), ctypes.byref(need))
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_span_correct_workspace_bytes")
    workspace = _workspace(workspace, int(need.value), y.device)
    rc = load_library().ssd_span_correct(ctypes.byref(prob), _ptr(dt), _ptr(A_log), _ptr(C), _ptr(entering),
                                         _ptr(y), _ptr(workspace), int(need.value),
                                         torch.cuda.current_stream(y.device).cuda_stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_span_correct")
    return y


def ssd_backward_workspace_bytes(prob: SsdProblem) -> int:
    out = ctypes.c_size_t(0)
    rc = load_library().ssd_backward_workspace_bytes(ctypes.byref(prob), ctypes.byref(out))
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_backward_workspace_bytes")
    return int(out.value)


def ssd_backward(prob: SsdProblem, x, dt, A_log, B, C, D, initial_states, dy, dfinal_states, dx, ddt,
                 dA_log, dB, dC, dD, dinitial_states, workspace, workspace_bytes: int, stream,
                 event_begin=None, event_end=None) -> int:
    """Raw ABI call on integer device addresses (0 = NULL); with events, the
    timed variant.  Returns the status."""
    lib = load_library()
    args = [ctypes.byref(prob), x, dt, A_log, B, C, D or None, initial_states or None, dy,
            dfinal_states or None, dx, ddt, dA_log, dB, dC, dD or None, dinitial_states or None,
            workspace, int(workspace_bytes), stream or None]
    if event_begin or event_end:
        return lib.ssd_backward_timed(*args, event_begin or None, event_end or None)
    return lib.ssd_backward(*args)


def backward(x, dt, A_log, B, C, dy, D=None, initial_states=None, dfinal_states=None,
             workspace=None, event_begin=None, event_end=None):
    """Gradients of the SSD layer on device tensors, given dy (and optionally
    the gradient of the final states).  Inputs as for ``forward`` (no packed
    rows).  Returns a dict: dx, ddt, dB, dC (x's dtype), dA_log, dD (float32;
    dD None without D), dinit (float32, zeros-shaped like the states)."""
    import torch

    dev = x.device
    if dev.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    if x.dtype == torch.bfloat16:
        dtype = SSD_DTYPE_BF16
    elif x.dtype == torch.float32:
        dtype = SSD_DTYPE_F32
    else:
        raise TypeError("x must be float32 or bfloat16")
    for name, t in (("dt", dt), ("B", B), ("C", C), ("dy", dy)):
        if t.dtype != x.dtype:
            raise TypeError("%s must have x's dtype" % name)
    for name, t in (("A_log", A_log), ("D", D), ("initial_states", initial_states),
                    ("dfinal_states", dfinal_states)):
        if t is not None and t.dtype != torch.float32:
            raise TypeError("%s must be float32" % name)
    for t in (x, dt, A_log, B, C, dy, D, initial_states, dfinal_states):
        if t is not None and (t.device != dev or not t.is_contiguous()):
            raise ValueError("all tensors must be contiguous and on x's device")
    b, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    prob = make_problem(b, T, H, P, N, G, 256, dtype)
    wsb = ssd_backward_workspace_bytes(prob)
    workspace = _workspace(workspace, wsb, dev)
    g = {"dx": torch.empty_like(x), "ddt": torch.empty_like(dt), "dB": torch.empty_like(B),
         "dC": torch.empty_like(C), "dA_log": torch.empty_like(A_log),
         "dD": torch.empty_like(D) if D is not None else None,
         "dinit": torch.empty((b, H, P, N), dtype=torch.float32, device=dev)}
    stream = torch.cuda.current_stream(dev).cuda_stream
    rc = ssd_backward(prob, _ptr(x), _ptr(dt), _ptr(A_log), _ptr(B), _ptr(C), _ptr(D), _ptr(initial_states),
                      _ptr(dy), _ptr(dfinal_states), _ptr(g["dx"]), _ptr(g["ddt"]), _ptr(g["dA_log"]),
                      _ptr(g["dB"]), _ptr(g["dC"]), _ptr(g["dD"]), _ptr(g["dinit"]), _ptr(workspace), wsb,
                      stream, event_begin, event_end)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_backward")
    return g


def ssd_backward_block_workspace_bytes(prob: SsdProblem, opts: SsdBlockOpts) -> int:
    out = ctypes.c_size_t(0)
    rc = load_library().ssd_backward_block_workspace_bytes(ctypes.byref(prob), ctypes.byref(opts),
                                                           ctypes.byref(out))
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_backward_block_workspace_bytes")
    return int(out.value)


def ssd_backward_block(prob: SsdProblem, opts: SsdBlockOpts, x, dt, A_log, B, C, D, initial_states, dout,
                       dfinal_states, dx, ddt, dA_log, dB, dC, dD, dinitial_states, ddt_bias, dz, dnorm_weight,
                       workspace, workspace_bytes: int, stream) -> int:
    """Raw ABI call on integer device addresses (0 = NULL); returns the status."""
    return load_library().ssd_backward_block(
        ctypes.byref(prob), ctypes.byref(opts), x, dt, A_log, B, C, D or None, initial_states or None, dout,
        dfinal_states or None, dx, ddt, dA_log, dB, dC, dD or None, dinitial_states or None, ddt_bias or None,
        dz or None, dnorm_weight or None, workspace, int(workspace_bytes), stream or None)


def backward_block(x, dt, A_log, B, C, dout, D=None, initial_states=None, dfinal_states=None, dt_bias=None,
                   dt_softplus: bool = True, dt_min: float = 0.0, dt_max: float = float("inf"), z=None,
                   norm_weight=None, norm_group_size: int = 0, norm_eps: float = 1e-5, workspace=None):
    """Gradients of ``forward_block`` on device tensors (``dt`` is the raw dt,
    before bias / softplus / clamp).  Returns a dict: dx, ddt, dB, dC, dz (x's
    dtype; dz None without z), dA_log, dD, dinit, ddt_bias, dnorm_weight
    (float32; None where the input is absent)."""
    import torch

    dev = x.device
    if dev.type != "cuda":
        raise ValueError("tensors must live on a HIP device")
    if x.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("x must be float32 or bfloat16")
    for name, t in (("dt", dt), ("B", B), ("C", C), ("dout", dout), ("z", z)):
        if t is not None and t.dtype != x.dtype:
            raise TypeError("%s must have x's dtype" % name)
    for name, t in (("A_log", A_log), ("D", D), ("initial_states", initial_states),
                    ("dfinal_states", dfinal_states), ("dt_bias", dt_bias), ("norm_weight", norm_weight)):
        if t is not None and t.dtype != torch.float32:
            raise TypeError("%s must be float32" % name)
    for t in (x, dt, A_log, B, C, dout, D, initial_states, dfinal_states, dt_bias, z, norm_weight):
        if t is not None and (t.device != dev or not t.is_contiguous()):
            raise ValueError("all tensors must be contiguous and on x's device")
    b, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    prob = make_problem(b, T, H, P, N, G, 256, SSD_DTYPE_BF16 if x.dtype == torch.bfloat16 else SSD_DTYPE_F32)
    opts = make_block_opts(dt_bias, dt_softplus, dt_min, dt_max, z, norm_weight, norm_group_size, norm_eps)
    wsb = ssd_backward_block_workspace_bytes(prob, opts)
    workspace = _workspace(workspace, wsb, dev)
    g = {"dx": torch.empty_like(x), "ddt": torch.empty_like(dt), "dB": torch.empty_like(B),
         "dC": torch.empty_like(C), "dA_log": torch.empty_like(A_log),
         "dD": torch.empty_like(D) if D is not None else None,
         "dinit": torch.empty((b, H, P, N), dtype=torch.float32, device=dev),
         "ddt_bias": torch.empty_like(dt_bias) if dt_bias is not None else None,
         "dz": torch.empty_like(z) if z is not None else None,
         "dnorm_weight": torch.empty_like(norm_weight) if norm_weight is not None and norm_group_size > 0
         else None}
    stream = torch.cuda.current_stream(dev).cuda_stream
    rc = ssd_backward_block(prob, opts, _ptr(x), _ptr(dt), _ptr(A_log), _ptr(B), _ptr(C), _ptr(D),
                            _ptr(initial_states), _ptr(dout), _ptr(dfinal_states), _ptr(g["dx"]), _ptr(g["ddt"]),
                            _ptr(g["dA_log"]), _ptr(g["dB"]), _ptr(g["dC"]), _ptr(g["dD"]), _ptr(g["dinit"]),
                            _ptr(g["ddt_bias"]), _ptr(g["dz"]), _ptr(g["dnorm_weight"]), _ptr(workspace), wsb,
                            stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_backward_block")
    return g


def _starts(seq_starts):
    arr = (ctypes.c_int64 * len(seq_starts))(*[int(v) for v in seq_starts])
    return arr


def ssd_backward_varlen_workspace_bytes(prob: SsdProblem, seq_starts) -> int:
    out = ctypes.c_size_t(0)
    rc = load_library().ssd_backward_varlen_workspace_bytes(ctypes.byref(prob), _starts(seq_starts),
                                                            ctypes.byref(out))
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_backward_varlen_workspace_bytes")
    return int(out.value)


def ssd_backward_varlen(prob: SsdProblem, seq_starts, x, dt, A_log, B, C, D, initial_states, dy, dfinal_states,
                        dx, ddt, dA_log, dB, dC, dD, dinitial_states, workspace, workspace_bytes: int,
                        stream) -> int:
    """Raw ABI call: ``seq_starts`` a host sequence of nseq + 1 offsets,
    integer device addresses (0 = NULL); returns the status."""
    return load_library().ssd_backward_varlen(
        ctypes.byref(prob), _starts(seq_starts), x, dt, A_log, B, C, D or None, initial_states or None, dy,
        dfinal_states or None, dx, ddt, dA_log, dB, dC, dD or None, dinitial_states or None, workspace,
        int(workspace_bytes), stream or None)


def backward_varlen(x, dt, A_log, B, C, dy, seq_starts, D=None, initial_states=None, dfinal_states=None,
                    workspace=None):
    """Gradients of the layer for one packed row (batch 1) of sequences with
    host offsets ``seq_starts`` (nseq + 1).  Returns the dict of ``backward``
    with dinit (nseq, H, P, N)."""
    import torch

    dev = x.device
    if x.shape[0] != 1:
        raise ValueError("packed rows use batch 1")
    for name, t in (("dt", dt), ("B", B), ("C", C), ("dy", dy)):
        if t.dtype != x.dtype:
            raise TypeError("%s must have x's dtype" % name)
    for t in (x, dt, A_log, B, C, dy, D, initial_states, dfinal_states):
        if t is not None and (t.device != dev or not t.is_contiguous()):
            raise ValueError("all tensors must be contiguous and on x's device")
    _, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    nseq = len(seq_starts) - 1
    prob = make_problem(1, T, H, P, N, G, 256, SSD_DTYPE_BF16 if x.dtype == torch.bfloat16 else SSD_DTYPE_F32,
                        nseq)
    wsb = ssd_backward_varlen_workspace_bytes(prob, seq_starts)
    workspace = _workspace(workspace, wsb, dev)
    g = {"dx": torch.empty_like(x), "ddt": torch.empty_like(dt), "dB": torch.empty_like(B),
         "dC": torch.empty_like(C), "dA_log": torch.empty_like(A_log),
         "dD": torch.empty_like(D) if D is not None else None,
         "dinit": torch.empty((nseq, H, P, N), dtype=torch.float32, device=dev)}
    rc = ssd_backward_varlen(prob, seq_starts, _ptr(x), _ptr(dt), _ptr(A_log), _ptr(B), _ptr(C), _ptr(D),
                             _ptr(initial_states), _ptr(dy), _ptr(dfinal_states), _ptr(g["dx"]), _ptr(g["ddt"]),
                             _ptr(g["dA_log"]), _ptr(g["dB"]), _ptr(g["dC"]), _ptr(g["dD"]), _ptr(g["dinit"]),
                             _ptr(workspace), wsb, torch.cuda.current_stream(dev).cuda_stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_backward_varlen")
    return g


def ssd_forward_varlen(prob: SsdProblem, seq_starts, x, dt, A_log, B, C, D, initial_states, y, final_states,
                       workspace, workspace_bytes: int, stream) -> int:
    """Raw ABI call: ``seq_starts`` a host sequence of nseq + 1 offsets,
    integer device addresses (0 = NULL); returns the status."""
    return load_library().ssd_forward_varlen(
        ctypes.byref(prob), _starts(seq_starts), x, dt, A_log, B, C, D or None, initial_states or None, y,
        final_states or None, workspace, int(workspace_bytes), stream or None)


def ssd_forward_varlen_workspace_bytes(prob: SsdProblem, seq_starts) -> int:
    out = ctypes.c_size_t(0)
    rc = load_library().ssd_forward_varlen_workspace_bytes(ctypes.byref(prob), _starts(seq_starts),
                                                           ctypes.byref(out))
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_forward_varlen_workspace_bytes")
    return int(out.value)


def forward_varlen(x, dt, A_log, B, C, seq_starts, D=None, chunk_size: int = 256, initial_states=None,
                   return_final_states: bool = True, workspace=None, out=None):
    """The forward of one packed row (batch 1) with host sequence offsets
    ``seq_starts`` (nseq + 1); returns ``(y, final_states (nseq,H,P,N) or None)``."""
    import torch

    dev = x.device
    if x.shape[0] != 1:
        raise ValueError("packed rows use batch 1")
    _, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    nseq = len(seq_starts) - 1
    prob = make_problem(1, T, H, P, N, G, chunk_size,
                        SSD_DTYPE_BF16 if x.dtype == torch.bfloat16 else SSD_DTYPE_F32, nseq)
    wsb = ssd_forward_varlen_workspace_bytes(prob, seq_starts)
    workspace = _workspace(workspace, wsb, dev)
    y = out if out is not None else torch.empty_like(x)
    fin = torch.empty((nseq, H, P, N), dtype=torch.float32, device=dev) if return_final_states else None
    rc = ssd_forward_varlen(prob, seq_starts, _ptr(x), _ptr(dt), _ptr(A_log), _ptr(B), _ptr(C), _ptr(D),
                            _ptr(initial_states), _ptr(y), _ptr(fin), _ptr(workspace), wsb,
                            torch.cuda.current_stream(dev).cuda_stream)
    if rc != SSD_OK:
        raise SsdError(rc, "ssd_forward_varlen")
    return y, fin
