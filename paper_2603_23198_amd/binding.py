"""ctypes binding of libsfl (include/sfl.h). Argument marshalling only.

Every function here has the name of the C entry point it calls and forwards
device pointers (torch tensors' data_ptr()) and the current HIP stream. All
arithmetic happens in the HIP kernels of libsfl.so; if the library is missing
or fails to load, importing this module raises (there is no fallback path).
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, Structure, c_char_p, c_double, c_int, c_int32, c_int64, c_size_t, c_void_p

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SFL_LIB", os.path.join(_HERE, "libsfl.so"))

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libsfl.so not found at {LIB_PATH}; build it with "
                      "`python -m paper_2603_23198_amd.build` (or __graft_entry__.build())")
_lib = ctypes.CDLL(LIB_PATH)

SFL_F32, SFL_BF16 = 0, 1
SFL_OK, SFL_E_ARG, SFL_E_UNSUPPORTED, SFL_E_WORKSPACE, SFL_E_HIP = 0, -1, -2, -3, -4
BUF_NAMES = ["val", "idx", "cnt", "row_nnz", "row_ovf", "ovf_rows", "n_ovf", "ell_val", "ell_idx", "ovf_dense"]

EXPORTED = ["sfl_status_string", "sfl_version", "sfl_twell_buffer_sizes", "sfl_pack_twell",
            "sfl_workspace_size", "sfl_ffn_forward", "sfl_up_projection", "sfl_ffn_backward",
            "sfl_dense_ffn_baseline", "sfl_transpose", "sfl_pack_down_weights", "sfl_track_active_units",
            "sfl_reinit_dead_units", "sfl_ffn_forward_noalloc", "sfl_bandwidth_probe",
            "sfl_down_projection_rowwise", "sfl_forward_workspace_size", "sfl_backward_workspace_size"]


class SflError(RuntimeError):
    def __init__(self, fn, code):
        msg = _lib.sfl_status_string(code).decode()
        super().__init__(f"{fn} failed: {msg} ({code})")
        self.code = code


class Cfg(Structure):
    _fields_ = [("tile_rows", c_int32), ("tile_cols", c_int32), ("tile_slots", c_int32),
                ("ell_width", c_int32), ("ovf_capacity", c_int32), ("layout", c_int32)]


SFL_TWELL_PLANES, SFL_TWELL_PACKED32 = 0, 1


class Twell(Structure):
    _fields_ = [(n, c_void_p) for n in BUF_NAMES]


class Stats(Structure):
    _fields_ = [("total_nnz", c_int64), ("n_ovf_rows", c_int64), ("n_tile_ovf", c_int64),
                ("l1_sum", c_double), ("capacity_exceeded", c_int32), ("reserved", c_int32)]


class FfnArgs(Structure):
    _fields_ = [("dtype", c_int), ("gated", c_int32), ("T", c_int64), ("d", c_int64), ("f", c_int64),
                ("X", c_void_p), ("W_gate", c_void_p), ("W_up", c_void_p), ("W_down", c_void_p),
                ("W_upT", c_void_p), ("W_gateT", c_void_p), ("W_downT", c_void_p), ("W_down_packed", c_void_p),
                ("W_up_packed", c_void_p),
                ("bias_f", c_void_p), ("shift_t", c_void_p),
                ("cfg", Cfg),
                ("Y", c_void_p), ("twell", Twell), ("stats", c_void_p), ("workspace", c_void_p),
                ("workspace_bytes", c_size_t), ("events", c_void_p), ("n_events", c_int32)]


class BwdArgs(Structure):
    _fields_ = [("dtype", c_int), ("gated", c_int32), ("T", c_int64), ("d", c_int64), ("f", c_int64),
                ("X", c_void_p), ("W_gate", c_void_p), ("W_up", c_void_p), ("W_down", c_void_p),
                ("W_upT", c_void_p), ("W_gateT", c_void_p),
                ("W_down_packed", c_void_p), ("W_up_packed", c_void_p), ("W_gate_packed", c_void_p),
                ("bias_f", c_void_p), ("shift_t", c_void_p),
                ("dY", c_void_p), ("cfg", Cfg), ("saved", Twell), ("lambda_l1", c_double),
                ("dX", c_void_p), ("dW_gate", c_void_p), ("dW_up", c_void_p), ("dW_down", c_void_p),
                ("workspace", c_void_p), ("workspace_bytes", c_size_t), ("events", c_void_p), ("n_events", c_int32)]


_lib.sfl_status_string.restype = c_char_p
_lib.sfl_status_string.argtypes = [c_int]
_lib.sfl_version.restype = c_char_p
_lib.sfl_twell_buffer_sizes.argtypes = [c_int64, c_int64, c_int, POINTER(Cfg), POINTER(c_size_t)]
_lib.sfl_pack_twell.argtypes = [c_void_p, c_int64, c_int64, c_int, POINTER(Cfg), POINTER(Twell), c_void_p, c_void_p]
_lib.sfl_workspace_size.argtypes = [c_void_p, c_int, POINTER(c_size_t)]
_lib.sfl_forward_workspace_size.argtypes = [POINTER(FfnArgs), c_int32, POINTER(c_size_t)]
_lib.sfl_backward_workspace_size.argtypes = [POINTER(BwdArgs), POINTER(c_size_t)]
_lib.sfl_ffn_forward.argtypes = [POINTER(FfnArgs), c_void_p]
_lib.sfl_ffn_forward_noalloc.argtypes = [POINTER(FfnArgs), c_void_p]
_lib.sfl_down_projection_rowwise.argtypes = [POINTER(FfnArgs), c_int32, c_void_p]
_lib.sfl_bandwidth_probe.argtypes = [c_void_p, c_void_p, c_size_t, c_int32, c_void_p, POINTER(c_size_t), c_void_p]
_lib.sfl_up_projection.argtypes = [POINTER(FfnArgs), c_void_p, c_void_p]
_lib.sfl_ffn_backward.argtypes = [POINTER(BwdArgs), c_void_p]
_lib.sfl_dense_ffn_baseline.argtypes = [POINTER(FfnArgs), c_void_p]
_lib.sfl_transpose.argtypes = [c_void_p, c_void_p, c_int64, c_int64, c_int32, c_void_p]
_lib.sfl_pack_down_weights.argtypes = [c_void_p, c_void_p, c_int64, c_int64, c_void_p]
_lib.sfl_track_active_units.argtypes = [POINTER(Twell), c_int64, c_int64, c_int, POINTER(Cfg), c_int64, c_void_p,
                                        c_void_p]
_lib.sfl_reinit_dead_units.argtypes = [c_void_p, c_int, c_int64, c_int64, c_int32, c_void_p, c_int64, ctypes.c_float,
                                       ctypes.c_float, c_void_p, c_void_p]
for _n in EXPORTED[2:]:
    getattr(_lib, _n).restype = c_int


def _check(fn, code):
    if code != SFL_OK:
        raise SflError(fn, code)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def dtype_code(dtype):
    if dtype in ("bf16", torch.bfloat16, SFL_BF16):
        return SFL_BF16
    if dtype in ("f32", torch.float32, SFL_F32):
        return SFL_F32
    raise ValueError(dtype)


def make_cfg(tile_cols=256, tile_slots=32, ell_width=128, ovf_capacity=0, tile_rows=0, layout=0, **_):
    return Cfg(tile_rows, tile_cols, tile_slots, ell_width, ovf_capacity, layout)


def sfl_version():
    return _lib.sfl_version().decode()


def sfl_status_string(code):
    return _lib.sfl_status_string(code).decode()


def sfl_twell_buffer_sizes(T, f, dtype, cfg):
    out = (c_size_t * len(BUF_NAMES))()
    _check("sfl_twell_buffer_sizes", _lib.sfl_twell_buffer_sizes(T, f, dtype_code(dtype), ctypes.byref(cfg), out))
    return list(out)


def alloc_twell(T, f, dtype, cfg, device="cuda", with_ell=True, with_dense=True):
    """Caller-side allocation (torch) of the packed-activation buffers, as dict of tensors."""
    sizes = sfl_twell_buffer_sizes(T, f, dtype, cfg)
    act = torch.bfloat16 if dtype_code(dtype) == SFL_BF16 else torch.float32
    es = 2 if act == torch.bfloat16 else 4
    packed = cfg.layout == SFL_TWELL_PACKED32
    kinds = {"val": torch.int32 if packed else act, "idx": torch.int16, "cnt": torch.int32, "row_nnz": torch.int32,
             "row_ovf": torch.uint8, "ovf_rows": torch.int32, "n_ovf": torch.int32,
             "ell_val": act, "ell_idx": torch.int16, "ovf_dense": act}
    item = {"val": 4 if packed else es, "idx": 2, "cnt": 4, "row_nnz": 4, "row_ovf": 1, "ovf_rows": 4, "n_ovf": 4,
            "ell_val": es, "ell_idx": 2, "ovf_dense": es}
    bufs = {}
    for name, nbytes in zip(BUF_NAMES, sizes):
        if (name in ("ell_val", "ell_idx") and not with_ell) or (name == "ovf_dense" and not with_dense) or \
                (packed and name in ("idx", "cnt")):
            bufs[name] = None
            continue
        n = max(1, nbytes // item[name])
        bufs[name] = torch.empty(n, dtype=kinds[name], device=device)
    return bufs


def _twell_struct(bufs):
    return Twell(*[_ptr(bufs.get(n)) for n in BUF_NAMES])


def sfl_pack_twell(Z, dtype, cfg, bufs, stats=None, stream=None):
    T, f = Z.shape
    tw = _twell_struct(bufs)
    _check("sfl_pack_twell", _lib.sfl_pack_twell(_ptr(Z), T, f, dtype_code(dtype), ctypes.byref(cfg),
                                                 ctypes.byref(tw), _ptr(stats), _stream(stream)))


def alloc_stats(device="cuda"):
    return torch.zeros(ctypes.sizeof(Stats), dtype=torch.uint8, device=device)


def read_stats(stats_tensor):
    raw = bytes(stats_tensor.cpu().numpy().tobytes())
    s = Stats.from_buffer_copy(raw)
    return {n: getattr(s, n) for n, _ in Stats._fields_ if n != "reserved"}


def ffn_args(X, W_up, W_down, cfg, *, Y=None, bufs=None, W_gate=None, W_upT=None, W_gateT=None, W_downT=None,
             W_down_packed=None, W_up_packed=None, bias_f=None, shift_t=None, stats=None, workspace=None,
             events=None):
    T, d = X.shape
    f = W_down.shape[0]
    a = FfnArgs()
    a.dtype = dtype_code(X.dtype)
    a.gated = 1 if W_gate is not None else 0
    a.T, a.d, a.f = T, d, f
    a.X, a.W_gate, a.W_up, a.W_down, a.W_upT = _ptr(X), _ptr(W_gate), _ptr(W_up), _ptr(W_down), _ptr(W_upT)
    a.W_gateT, a.W_downT = _ptr(W_gateT), _ptr(W_downT)
    a.W_down_packed, a.W_up_packed = _ptr(W_down_packed), _ptr(W_up_packed)
    a.bias_f, a.shift_t = _ptr(bias_f), _ptr(shift_t)
    a.cfg = cfg
    a.Y = _ptr(Y)
    if bufs is not None:
        a.twell = _twell_struct(bufs)
    a.stats = _ptr(stats)
    if workspace is not None:
        a.workspace = _ptr(workspace)
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    if events is not None:
        a._events_keepalive = events
        a.events = ctypes.cast(events, c_void_p).value
        a.n_events = len(events)
    return a


def sfl_workspace_size(args, kind=0):
    out = c_size_t(0)
    _check("sfl_workspace_size", _lib.sfl_workspace_size(ctypes.byref(args), kind, ctypes.byref(out)))
    return out.value


def sfl_forward_workspace_size(args, dense=False):
    out = c_size_t(0)
    _check("sfl_forward_workspace_size", _lib.sfl_forward_workspace_size(ctypes.byref(args), 1 if dense else 0,
                                                                          ctypes.byref(out)))
    return out.value


def sfl_backward_workspace_size(args):
    out = c_size_t(0)
    _check("sfl_backward_workspace_size", _lib.sfl_backward_workspace_size(ctypes.byref(args), ctypes.byref(out)))
    return out.value


def sfl_ffn_forward(args, stream=None):
    _check("sfl_ffn_forward", _lib.sfl_ffn_forward(ctypes.byref(args), _stream(stream)))


def sfl_ffn_forward_noalloc(args, stream=None):
    _check("sfl_ffn_forward_noalloc", _lib.sfl_ffn_forward_noalloc(ctypes.byref(args), _stream(stream)))


def sfl_up_projection(args, Z, stream=None):
    _check("sfl_up_projection", _lib.sfl_up_projection(ctypes.byref(args), _ptr(Z), _stream(stream)))


def sfl_dense_ffn_baseline(args, stream=None):
    _check("sfl_dense_ffn_baseline", _lib.sfl_dense_ffn_baseline(ctypes.byref(args), _stream(stream)))


def bwd_args(X, W_up, W_down, dY, cfg, saved_bufs, lambda_l1, dX, dW_up, dW_down, *, W_upT=None, W_down_packed=None,
             W_up_packed=None, W_gate=None, W_gateT=None, W_gate_packed=None, dW_gate=None, bias_f=None,
             shift_t=None, workspace=None, events=None):
    T, d = X.shape
    f = W_down.shape[0]
    a = BwdArgs()
    a.dtype = dtype_code(X.dtype)
    a.T, a.d, a.f = T, d, f
    a.X, a.W_up, a.W_down, a.W_upT, a.dY = _ptr(X), _ptr(W_up), _ptr(W_down), _ptr(W_upT), _ptr(dY)
    a.W_down_packed, a.W_up_packed = _ptr(W_down_packed), _ptr(W_up_packed)
    a.gated = 1 if W_gate is not None else 0
    a.W_gate, a.W_gateT, a.W_gate_packed = _ptr(W_gate), _ptr(W_gateT), _ptr(W_gate_packed)
    a.bias_f, a.shift_t, a.dW_gate = _ptr(bias_f), _ptr(shift_t), _ptr(dW_gate)
    a.cfg = cfg
    a.saved = _twell_struct(saved_bufs)
    a.lambda_l1 = float(lambda_l1)
    a.dX, a.dW_up, a.dW_down = _ptr(dX), _ptr(dW_up), _ptr(dW_down)
    if workspace is not None:
        a.workspace = _ptr(workspace)
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    if events is not None:
        a._events_keepalive = events
        a.events = ctypes.cast(events, c_void_p).value
        a.n_events = len(events)
    return a


def sfl_ffn_backward(args, stream=None):
    _check("sfl_ffn_backward", _lib.sfl_ffn_backward(ctypes.byref(args), _stream(stream)))


def sfl_pack_down_weights(W_down, out, stream=None):
    f, d = W_down.shape
    _check("sfl_pack_down_weights", _lib.sfl_pack_down_weights(_ptr(W_down), _ptr(out), f, d, _stream(stream)))


def sfl_track_active_units(bufs, T, f, dtype, cfg, step, last_active, stream=None):
    tw = _twell_struct(bufs)
    _check("sfl_track_active_units", _lib.sfl_track_active_units(ctypes.byref(tw), T, f, dtype_code(dtype),
                                                                 ctypes.byref(cfg), int(step), _ptr(last_active),
                                                                 _stream(stream)))


def sfl_reinit_dead_units(W, last_active, step, lam, sigma, noise, units_on_rows=False, stream=None):
    rows, cols = W.shape
    _check("sfl_reinit_dead_units", _lib.sfl_reinit_dead_units(_ptr(W), dtype_code(W.dtype), rows, cols,
                                                               1 if units_on_rows else 0, _ptr(last_active),
                                                               int(step), float(lam), float(sigma), _ptr(noise),
                                                               _stream(stream)))


def sfl_down_projection_rowwise(args, split, stream=None):
    _check("sfl_down_projection_rowwise", _lib.sfl_down_projection_rowwise(ctypes.byref(args), split, _stream(stream)))


def sfl_bandwidth_probe(src, dst=None, reps=1, sink=None, nbytes=None, stream=None):
    """Copy (dst given) or L2/HBM read probe (dst None); returns the bytes moved."""
    moved = c_size_t(0)
    n = src.numel() * src.element_size() if nbytes is None else nbytes
    _check("sfl_bandwidth_probe", _lib.sfl_bandwidth_probe(_ptr(src), _ptr(dst), n, reps, _ptr(sink),
                                                           ctypes.byref(moved), _stream(stream)))
    return moved.value


def sfl_transpose(inp, out, stream=None):
    rows, cols = inp.shape
    _check("sfl_transpose", _lib.sfl_transpose(_ptr(inp), _ptr(out), rows, cols, inp.element_size(),
                                               _stream(stream)))


# ---- HIP events through the runtime library torch already loaded (for stage timing) ----
_hip = None


def _hiprt():
    global _hip
    if _hip is None:
        for name in ("libamdhip64.so.7", "libamdhip64.so"):
            try:
                _hip = ctypes.CDLL(name)
                break
            except OSError:
                continue
        if _hip is None:
            raise OSError("libamdhip64 not found")
        _hip.hipEventCreate.argtypes = [POINTER(c_void_p)]
        _hip.hipEventElapsedTime.argtypes = [POINTER(ctypes.c_float), c_void_p, c_void_p]
        _hip.hipEventSynchronize.argtypes = [c_void_p]
        _hip.hipEventDestroy.argtypes = [c_void_p]
    return _hip


def create_events(n):
    """Array of n hipEvent_t handles (ctypes array of c_void_p) for the `events` argument."""
    hip = _hiprt()
    arr = (c_void_p * n)()
    for i in range(n):
        e = c_void_p()
        if hip.hipEventCreate(ctypes.byref(e)) != 0:
            raise RuntimeError("hipEventCreate failed")
        arr[i] = e
    return arr


def event_ms(events, i, j):
    hip = _hiprt()
    hip.hipEventSynchronize(events[j])
    ms = ctypes.c_float()
    if hip.hipEventElapsedTime(ctypes.byref(ms), events[i], events[j]) != 0:
        raise RuntimeError("hipEventElapsedTime failed")
    return ms.value
