"""ctypes binding of libdart.so (C ABI in include/dart.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  PyTorch supplies device memory (tensors) and the stream.  If the
library has not been built, every call raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
import threading
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdart.so")

DART_OK, DART_ERR_INVALID_ARG, DART_ERR_UNSUPPORTED, DART_ERR_HIP = 0, 1, 2, 3
DART_FP32, DART_BF16 = 0, 1
DEFAULT_EPS = 1e-6


class DartError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (_STATUS.get(status, "DART_ERR_%d" % status), msg))
        self.status = status


_STATUS = {0: "DART_OK", 1: "DART_ERR_INVALID_ARG", 2: "DART_ERR_UNSUPPORTED", 3: "DART_ERR_HIP"}


class Dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seqlen", ctypes.c_int64),
                ("nheads", ctypes.c_int32), ("ngroups", ctypes.c_int32),
                ("headdim", ctypes.c_int32), ("dstate", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("mem_capacity", ctypes.c_int64)]


class SmaOpts(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_float), ("q_norm_w", ctypes.c_void_p),
                ("e_norm_w", ctypes.c_void_p), ("normalize", ctypes.c_int32),
                ("z_per_head", ctypes.c_int32)]


EXPORTS = ("dart_scan_workspace_bytes", "dart_ssd_chunk_scan", "dart_sma_workspace_bytes",
           "dart_sma_fwd", "dart_sma_bwd_workspace_bytes", "dart_sma_bwd",
           "dart_ssd_bwd_workspace_bytes", "dart_ssd_bwd",
           "dart_conv1d_silu", "dart_dt_softplus", "dart_gated_rmsnorm",
           "dart_conv1d_silu_bwd_workspace_bytes", "dart_conv1d_silu_bwd",
           "dart_dt_softplus_bwd_workspace_bytes", "dart_dt_softplus_bwd",
           "dart_gated_rmsnorm_bwd_workspace_bytes", "dart_gated_rmsnorm_bwd",
           "dart_decode_workspace_bytes", "dart_decode_step", "dart_decode_step_noalloc",
           "dart_decode_step_ragged", "dart_decode_handoff", "dart_decode_cache_elems", "dart_status_string", "dart_last_error",
           "dart_profile_enable", "dart_profile_filter", "dart_profile_flush", "dart_profile_count",
           "dart_profile_name", "dart_profile_total_ms", "dart_profile_launches",
           "dart_profile_reset")

_lock = threading.Lock()
_lib = None


def load_library(path: str = LIB_PATH):
    """Load libdart.so and declare its signatures.  Raises if it is missing."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(path):
            raise RuntimeError("libdart.so not found at %s: build it with "
                               "`python -m paper_2608_02032_amd.build` (no fallback path exists)"
                               % path)
        lib = ctypes.CDLL(path)
        P, D, O = ctypes.c_void_p, ctypes.POINTER(Dims), ctypes.POINTER(SmaOpts)
        sz, st, i64 = ctypes.c_size_t, ctypes.c_int, ctypes.c_int64
        lib.dart_scan_workspace_bytes.argtypes = [D]
        lib.dart_scan_workspace_bytes.restype = sz
        lib.dart_ssd_chunk_scan.argtypes = [D, P, P, P, P, P, P, P, P, P, P, sz, P]
        lib.dart_ssd_chunk_scan.restype = st
        lib.dart_sma_workspace_bytes.argtypes = [D]
        lib.dart_sma_workspace_bytes.restype = sz
        lib.dart_sma_fwd.argtypes = [D, O, P, P, P, P, P, P, P, P, P, sz, P]
        lib.dart_sma_fwd.restype = st
        lib.dart_sma_bwd_workspace_bytes.argtypes = [D]
        lib.dart_sma_bwd_workspace_bytes.restype = sz
        lib.dart_sma_bwd.argtypes = [D, O, P, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]
        lib.dart_sma_bwd.restype = st
        lib.dart_ssd_bwd_workspace_bytes.argtypes = [D]
        lib.dart_ssd_bwd_workspace_bytes.restype = sz
        lib.dart_ssd_bwd.argtypes = [D] + [P] * 16 + [sz, P]
        lib.dart_ssd_bwd.restype = st
        lib.dart_conv1d_silu.argtypes = [i64, i64, ctypes.c_int32, i64, ctypes.c_int32, P, P, P, P,
                                         P, P, P]
        lib.dart_conv1d_silu.restype = st
        lib.dart_dt_softplus.argtypes = [i64, ctypes.c_int32, i64, ctypes.c_int32, P, P, P, P]
        lib.dart_dt_softplus.restype = st
        lib.dart_gated_rmsnorm.argtypes = [i64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P, P,
                                           i64, P, ctypes.c_float, P, P]
        lib.dart_gated_rmsnorm.restype = st
        lib.dart_conv1d_silu_bwd_workspace_bytes.argtypes = [i64, i64, ctypes.c_int32]
        lib.dart_conv1d_silu_bwd_workspace_bytes.restype = sz
        lib.dart_conv1d_silu_bwd.argtypes = [i64, i64, ctypes.c_int32, i64, ctypes.c_int32, P, P, P,
                                             P, P, P, i64, P, P, P, P, sz, P]
        lib.dart_conv1d_silu_bwd.restype = st
        lib.dart_dt_softplus_bwd_workspace_bytes.argtypes = [i64, ctypes.c_int32]
        lib.dart_dt_softplus_bwd_workspace_bytes.restype = sz
        lib.dart_dt_softplus_bwd.argtypes = [i64, ctypes.c_int32, i64, ctypes.c_int32, P, P, P, P,
                                             i64, P, P, sz, P]
        lib.dart_dt_softplus_bwd.restype = st
        lib.dart_gated_rmsnorm_bwd_workspace_bytes.argtypes = [i64, ctypes.c_int32]
        lib.dart_gated_rmsnorm_bwd_workspace_bytes.restype = sz
        lib.dart_gated_rmsnorm_bwd.argtypes = [i64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               P, P, i64, P, ctypes.c_float, P, P, P, i64, P, P, sz,
                                               P]
        lib.dart_gated_rmsnorm_bwd.restype = st
        lib.dart_decode_workspace_bytes.argtypes = [D]
        lib.dart_decode_workspace_bytes.restype = sz
        lib.dart_decode_step.argtypes = [D, O, i64, P, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]
        lib.dart_decode_step.restype = st
        lib.dart_decode_step_noalloc.argtypes = [D, O, i64] + [P] * 13
        lib.dart_decode_step_noalloc.restype = st
        lib.dart_decode_step_ragged.argtypes = [D, O, P, i64, P, P, P, P, P, P, P, P, P, P, P, P,
                                                P, sz, P]
        lib.dart_decode_step_ragged.restype = st
        lib.dart_decode_handoff.argtypes = [D, P, P, P, P, P, P]
        lib.dart_decode_handoff.restype = st
        lib.dart_decode_cache_elems.argtypes = [D, i64]
        lib.dart_decode_cache_elems.restype = i64
        lib.dart_status_string.argtypes = [st]
        lib.dart_status_string.restype = ctypes.c_char_p
        lib.dart_last_error.argtypes = []
        lib.dart_last_error.restype = ctypes.c_char_p
        lib.dart_profile_enable.argtypes = [ctypes.c_int]
        lib.dart_profile_enable.restype = st
        lib.dart_profile_filter.argtypes = [ctypes.c_char_p]
        lib.dart_profile_filter.restype = st
        lib.dart_profile_flush.argtypes = []
        lib.dart_profile_flush.restype = st
        lib.dart_profile_count.argtypes = []
        lib.dart_profile_count.restype = ctypes.c_int
        lib.dart_profile_name.argtypes = [ctypes.c_int]
        lib.dart_profile_name.restype = ctypes.c_char_p
        lib.dart_profile_total_ms.argtypes = [ctypes.c_int]
        lib.dart_profile_total_ms.restype = ctypes.c_double
        lib.dart_profile_launches.argtypes = [ctypes.c_int]
        lib.dart_profile_launches.restype = i64
        lib.dart_profile_reset.argtypes = []
        lib.dart_profile_reset.restype = None
        _lib = lib
        return lib


def check(status: int):
    if status != DART_OK:
        raise DartError(status, load_library().dart_last_error().decode())


def make_dims(batch, seqlen, nheads, headdim, dstate, chunk, dtype, ngroups=1, mem_capacity=0):
    dt_code = {"fp32": DART_FP32, "bf16": DART_BF16}.get(dtype, dtype)
    return Dims(int(batch), int(seqlen), int(nheads), int(ngroups), int(headdim), int(dstate),
                int(chunk), int(dt_code), int(mem_capacity))


# --------------------------------------------------------------------------- #
# torch-facing helpers (device memory and streams only)
# --------------------------------------------------------------------------- #

def _torch():
    import torch
    return torch


def _dtype_num(t):
    return {"fp32": DART_FP32, "bf16": DART_BF16}[_dtype_code(t)]


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return "bf16"
    if t.dtype == torch.float32:
        return "fp32"
    raise TypeError("storage tensors must be float32 or bfloat16, got %s" % t.dtype)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _ptr_rows(t) -> int:
    """Pointer of a view whose rows are contiguous (innermost stride 1) at a
    common row stride, e.g. a channel slice of a projection output."""
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if t.stride(-1) != 1:
        raise ValueError("tensor rows must be contiguous")
    return t.data_ptr()


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _workspace(nbytes, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _check_f32(t, name):
    torch = _torch()
    if t is not None and t.dtype != torch.float32:
        raise TypeError("%s must be float32" % name)


def ssd_chunk_scan(x, dt, A, Bm, Cm, chunk, h0=None, mem=None, mem_capacity=0, y_ssd=None,
                   h_last=True, workspace=None, stream=None):
    """Chunked SSD scan retaining the chunk state memories (dart_ssd_chunk_scan).

    x [B][L][H][P], dt [B][L][H] f32, A [H] f32, Bm/Cm [B][L][G][N].
    Returns (y_ssd [B][L][H][P], mem [B][Mcap][H][N][P], h_last [B][H][N][P] f32 or None).
    """
    torch = _torch()
    lib = load_library()
    B_, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    dtype = _dtype_code(x)
    for t, nm in ((dt, "dt"), (A, "A"), (h0, "h0")):
        _check_f32(t, nm)
    M = -(-L // chunk)
    if mem is not None:
        mem_capacity = mem.shape[1]
    Mcap = mem_capacity or M
    dims = make_dims(B_, L, H, P, N, chunk, dtype, G, Mcap)
    if y_ssd is None:
        y_ssd = torch.empty_like(x)
    if mem is None:
        mem = torch.empty((B_, Mcap, H, N, P), dtype=x.dtype, device=x.device)
    hl = torch.empty((B_, H, N, P), dtype=torch.float32, device=x.device) if h_last is True else (
        h_last if h_last is not None and h_last is not False else None)
    need = lib.dart_scan_workspace_bytes(ctypes.byref(dims))
    if workspace is None:
        workspace = _workspace(need, x.device)
    check(lib.dart_ssd_chunk_scan(ctypes.byref(dims), _ptr(x), _ptr(dt), _ptr(A), _ptr(Bm),
                                  _ptr(Cm), _ptr(h0), _ptr(y_ssd), _ptr(mem), _ptr(hl),
                                  _ptr(workspace), workspace.numel(), _stream(stream)))
    return y_ssd, mem, hl


def sma_fwd(q, e, Cm, mem, z, y_ssd, chunk, eps=DEFAULT_EPS, normalize=True, q_norm_w=None,
            e_norm_w=None, y=None, lse=True, workspace=None, stream=None):
    """State-memory attention + gated residual (dart_sma_fwd).

    q [B][L][G][N], e [B][L][G][P], Cm [B][L][G][N], mem [B][Mcap][H][N][P],
    z [B][L][H] (one gate per head) or [B][L] (one per token), y_ssd [B][L][H][P].
    Returns (y, lse) with lse [B][L][H] f32 (or None).  y may be y_ssd (in place).
    """
    torch = _torch()
    lib = load_library()
    B_, L, H, P = y_ssd.shape
    G, N = q.shape[2], q.shape[3]
    dtype = _dtype_code(y_ssd)
    _check_f32(q_norm_w, "q_norm_w")
    _check_f32(e_norm_w, "e_norm_w")
    z_per_head = 1 if z.dim() == 3 else 0
    dims = make_dims(B_, L, H, P, N, chunk, dtype, G, mem.shape[1])
    opts = SmaOpts(float(eps), _ptr(q_norm_w), _ptr(e_norm_w), int(bool(normalize)), z_per_head)
    if y is None:
        y = torch.empty_like(y_ssd)
    lse_t = torch.empty((B_, L, H), dtype=torch.float32, device=y_ssd.device) if lse is True else (
        lse if lse is not None and lse is not False else None)
    need = lib.dart_sma_workspace_bytes(ctypes.byref(dims))
    if workspace is None:
        workspace = _workspace(need, y_ssd.device)
    check(lib.dart_sma_fwd(ctypes.byref(dims), ctypes.byref(opts), _ptr(q), _ptr(e), _ptr(Cm),
                           _ptr(mem), _ptr(z), _ptr(y_ssd), _ptr(y), _ptr(lse_t), _ptr(workspace),
                           workspace.numel(), _stream(stream)))
    return y, lse_t


def sma_bwd(q, e, Cm, mem, z, lse, dy, chunk, eps=DEFAULT_EPS, normalize=True, q_norm_w=None,
            e_norm_w=None, out=None, workspace=None, stream=None):
    """Backward of sma_fwd for the loss sum(dy * y) (dart_sma_bwd).

    lse [B][L][H] f32 is the forward's output; dy like y_ssd.  Returns a dict
    of float32 tensors: dq, de, dC ([B][L][G][.], summed over each group's
    heads), dmem (like mem) and dz (like z).  The gradient with respect to
    y_ssd is dy itself.  `out` may hold preallocated tensors under those keys.
    """
    torch = _torch()
    lib = load_library()
    B_, L, H, P = dy.shape
    G, N = q.shape[2], q.shape[3]
    dtype = _dtype_code(dy)
    _check_f32(q_norm_w, "q_norm_w")
    _check_f32(e_norm_w, "e_norm_w")
    _check_f32(lse, "lse")
    z_per_head = 1 if z.dim() == 3 else 0
    dims = make_dims(B_, L, H, P, N, chunk, dtype, G, mem.shape[1])
    opts = SmaOpts(float(eps), _ptr(q_norm_w), _ptr(e_norm_w), int(bool(normalize)), z_per_head)
    f32 = dict(dtype=torch.float32, device=dy.device)
    want = {"dq": q.shape, "de": e.shape, "dC": Cm.shape, "dmem": mem.shape, "dz": z.shape}
    out = dict(out or {})
    for k, shape in want.items():
        if k not in out:
            out[k] = torch.empty(shape, **f32)
        elif tuple(out[k].shape) != tuple(shape) or out[k].dtype != torch.float32 \
                or not out[k].is_contiguous():
            raise ValueError("out[%r] must be a contiguous float32 tensor of shape %s"
                             % (k, tuple(shape)))
    need = lib.dart_sma_bwd_workspace_bytes(ctypes.byref(dims))
    if workspace is None:
        workspace = _workspace(need, dy.device)
    check(lib.dart_sma_bwd(ctypes.byref(dims), ctypes.byref(opts), _ptr(q), _ptr(e), _ptr(Cm),
                           _ptr(mem), _ptr(z), _ptr(lse), _ptr(dy), _ptr(out["dq"]),
                           _ptr(out["de"]), _ptr(out["dC"]), _ptr(out["dmem"]), _ptr(out["dz"]),
                           _ptr(workspace), workspace.numel(), _stream(stream)))
    return out


def ssd_bwd(x, dt, A, Bm, Cm, chunk, dy, dmem=None, dh_last=None, h0=None, out=None,
            workspace=None, stream=None):
    """Backward of ssd_chunk_scan (dart_ssd_bwd) for the loss
    sum(dy * y_ssd) + sum(dmem * mem) + sum(dh_last * h_last).

    dy like x (storage dtype); dmem [B][Mcap][H][N][P] f32 or None; dh_last
    and h0 [B][H][N][P] f32 or None.  Returns a dict of float32 tensors dx,
    ddt, dA, dB, dC (summed over each group's heads) and dh0.  `out` may hold
    preallocated tensors under those keys.
    """
    torch = _torch()
    lib = load_library()
    B_, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    dtype = _dtype_code(x)
    for t, nm in ((dt, "dt"), (A, "A"), (dmem, "dmem"), (dh_last, "dh_last"), (h0, "h0")):
        _check_f32(t, nm)
    mcap = dmem.shape[1] if dmem is not None else 0
    dims = make_dims(B_, L, H, P, N, chunk, dtype, G, mcap)
    f32 = dict(dtype=torch.float32, device=x.device)
    want = {"dx": x.shape, "ddt": dt.shape, "dA": A.shape, "dB": Bm.shape, "dC": Cm.shape,
            "dh0": (B_, H, N, P)}
    out = dict(out or {})
    for k, shape in want.items():
        if k not in out:
            out[k] = torch.empty(shape, **f32)
        elif tuple(out[k].shape) != tuple(shape) or out[k].dtype != torch.float32 \
                or not out[k].is_contiguous():
            raise ValueError("out[%r] must be a contiguous float32 tensor of shape %s"
                             % (k, tuple(shape)))
    need = lib.dart_ssd_bwd_workspace_bytes(ctypes.byref(dims))
    if workspace is None:
        workspace = _workspace(need, x.device)
    check(lib.dart_ssd_bwd(ctypes.byref(dims), _ptr(x), _ptr(dt), _ptr(A), _ptr(Bm), _ptr(Cm),
                           _ptr(h0), _ptr(dy), _ptr(dmem), _ptr(dh_last), _ptr(out["dx"]),
                           _ptr(out["ddt"]), _ptr(out["dA"]), _ptr(out["dB"]), _ptr(out["dC"]),
                           _ptr(out["dh0"]), _ptr(workspace), workspace.numel(), _stream(stream)))
    return out


def conv1d_silu(inp, weight, bias=None, state_in=None, state_out=None, channels=None, out=None,
                stream=None):
    """Causal width-4 depthwise convolution + bias + SiLU (dart_conv1d_silu).

    inp [B][L][R] (channels = the first `channels` of each row, default R;
    pass a view starting at the first x channel), weight [C][4] f32, bias [C]
    f32, state_in/state_out [B][C][3] f32 (state_out=True allocates one).
    Returns (out [B][L][C], state_out or None)."""
    torch = _torch()
    lib = load_library()
    B_, L, R = inp.shape
    C = R if channels is None else int(channels)
    if inp.stride(2) != 1 or inp.stride(0) != L * inp.stride(1):
        raise ValueError("inp rows must be contiguous with a common row stride")
    for t, nm in ((weight, "weight"), (bias, "bias"), (state_in, "state_in")):
        _check_f32(t, nm)
    if state_out is True:
        state_out = torch.empty((B_, C, 3), dtype=torch.float32, device=inp.device)
    if out is None:
        out = torch.empty((B_, L, C), dtype=inp.dtype, device=inp.device)
    check(lib.dart_conv1d_silu(B_, L, C, inp.stride(1), _dtype_num(inp), _ptr_rows(inp), _ptr(weight),
                               _ptr(bias), _ptr(state_in), _ptr(state_out), _ptr(out),
                               _stream(stream)))
    return out, state_out


def dt_softplus(raw, bias=None, nheads=None, out=None, stream=None):
    """dt = softplus(raw + bias) in float (dart_dt_softplus); raw [..][R] with
    the heads the first `nheads` (default R) elements of each row."""
    torch = _torch()
    lib = load_library()
    R = raw.shape[-1]
    H = R if nheads is None else int(nheads)
    rows = raw.numel() // R
    if raw.stride(-1) != 1:
        raise ValueError("raw rows must be contiguous")
    _check_f32(bias, "bias")
    if out is None:
        out = torch.empty(tuple(raw.shape[:-1]) + (H,), dtype=torch.float32, device=raw.device)
    stride = raw.stride(-2) if raw.dim() > 1 else R
    check(lib.dart_dt_softplus(rows, H, stride, _dtype_num(raw), _ptr_rows(raw), _ptr(bias), _ptr(out),
                               _stream(stream)))
    return out


def gated_rmsnorm(y, z, weight=None, group=None, eps=DEFAULT_EPS, out=None, stream=None):
    """u = y * SiLU(z); u / sqrt(mean over each group of u^2 + eps) * weight
    (dart_gated_rmsnorm).  y [..][D] contiguous; z [..][D] rows of a common
    stride (e.g. the gate slice of the projection output)."""
    torch = _torch()
    lib = load_library()
    D = y.shape[-1]
    rows = y.numel() // D
    group = D if group is None else int(group)
    if not y.is_contiguous() or z.stride(-1) != 1:
        raise ValueError("y must be contiguous and z rows contiguous")
    _check_f32(weight, "weight")
    if out is None:
        out = torch.empty_like(y)
    zs = z.stride(-2) if z.dim() > 1 else D
    check(lib.dart_gated_rmsnorm(rows, D, group, _dtype_num(y), _ptr(y), _ptr_rows(z), zs,
                                 _ptr(weight), float(eps), _ptr(out), _stream(stream)))
    return out


def conv1d_silu_bwd(inp, weight, dout, bias=None, state_in=None, channels=None, din=None,
                    want_state=False, stream=None):
    """Backward of conv1d_silu (dart_conv1d_silu_bwd) for output gradient dout
    [B][L][C] (float).  din (optional) may be a float view with a common row
    stride, e.g. the xBC slice of a projection gradient.  Returns
    {"din", "dweight", "dbias" (None without bias), "dstate" (or None)}."""
    torch = _torch()
    lib = load_library()
    B_, L, R = inp.shape
    C = R if channels is None else int(channels)
    if inp.stride(2) != 1 or inp.stride(0) != L * inp.stride(1):
        raise ValueError("inp rows must be contiguous with a common row stride")
    for t, nm in ((weight, "weight"), (bias, "bias"), (state_in, "state_in"), (dout, "dout")):
        _check_f32(t, nm)
    f32 = dict(dtype=torch.float32, device=inp.device)
    if din is None:
        din = torch.empty((B_, L, C), **f32)
    if din.stride(2) != 1 or din.stride(0) != L * din.stride(1):
        raise ValueError("din rows must be contiguous with a common row stride")
    dw = torch.empty((C, 4), **f32)
    db = torch.empty((C,), **f32) if bias is not None else None
    dst = torch.empty((B_, C, 3), **f32) if want_state else None
    ws = _workspace(lib.dart_conv1d_silu_bwd_workspace_bytes(B_, L, C), inp.device)
    check(lib.dart_conv1d_silu_bwd(B_, L, C, inp.stride(1), _dtype_num(inp), _ptr_rows(inp),
                                   _ptr(weight), _ptr(bias), _ptr(state_in), _ptr(dout),
                                   _ptr_rows(din), din.stride(1), _ptr(dw), _ptr(db), _ptr(dst),
                                   _ptr(ws), ws.numel(), _stream(stream)))
    return {"din": din, "dweight": dw, "dbias": db, "dstate": dst}


def dt_softplus_bwd(raw, ddt, bias=None, nheads=None, draw=None, stream=None):
    """Backward of dt_softplus (dart_dt_softplus_bwd): returns (draw, dbias)."""
    torch = _torch()
    lib = load_library()
    R = raw.shape[-1]
    H = R if nheads is None else int(nheads)
    rows = raw.numel() // R
    _check_f32(bias, "bias")
    _check_f32(ddt, "ddt")
    f32 = dict(dtype=torch.float32, device=raw.device)
    if draw is None:
        draw = torch.empty(tuple(raw.shape[:-1]) + (H,), **f32)
    dbias = torch.empty((H,), **f32) if bias is not None else None
    stride = raw.stride(-2) if raw.dim() > 1 else R
    dstride = draw.stride(-2) if draw.dim() > 1 else H
    ws = _workspace(lib.dart_dt_softplus_bwd_workspace_bytes(rows, H), raw.device)
    check(lib.dart_dt_softplus_bwd(rows, H, stride, _dtype_num(raw), _ptr_rows(raw), _ptr(bias),
                                   _ptr(ddt), _ptr_rows(draw), dstride, _ptr(dbias), _ptr(ws),
                                   ws.numel(), _stream(stream)))
    return draw, dbias


def gated_rmsnorm_bwd(y, z, dout, weight=None, group=None, eps=DEFAULT_EPS, dz=None, stream=None):
    """Backward of gated_rmsnorm (dart_gated_rmsnorm_bwd): returns
    {"dy", "dz", "dweight" (None without weight)}; dz (optional) may be a
    float view with a common row stride."""
    torch = _torch()
    lib = load_library()
    D = y.shape[-1]
    rows = y.numel() // D
    group = D if group is None else int(group)
    if not y.is_contiguous() or z.stride(-1) != 1 or not dout.is_contiguous():
        raise ValueError("y and dout must be contiguous and z rows contiguous")
    _check_f32(weight, "weight")
    _check_f32(dout, "dout")
    f32 = dict(dtype=torch.float32, device=y.device)
    dy = torch.empty(y.shape, **f32)
    if dz is None:
        dz = torch.empty(y.shape, **f32)
    dw = torch.empty((D,), **f32) if weight is not None else None
    zs = z.stride(-2) if z.dim() > 1 else D
    dzs = dz.stride(-2) if dz.dim() > 1 else D
    ws = _workspace(lib.dart_gated_rmsnorm_bwd_workspace_bytes(rows, D), y.device)
    check(lib.dart_gated_rmsnorm_bwd(rows, D, group, _dtype_num(y), _ptr(y), _ptr_rows(z), zs,
                                     _ptr(weight), float(eps), _ptr(dout), _ptr(dy), _ptr_rows(dz),
                                     dzs, _ptr(dw), _ptr(ws), ws.numel(), _stream(stream)))
    return {"dy": dy, "dz": dz, "dweight": dw}


def decode_step(pos, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc, mem_cache, chunk,
                eps=DEFAULT_EPS, normalize=True, q_norm_w=None, e_norm_w=None, y=None,
                workspace=None, stream=None):
    """One decode step at position `pos` (dart_decode_step).  Updates h_state,
    chunk_acc and mem_cache in place; returns y [B][H][P]."""
    torch = _torch()
    lib = load_library()
    B_, H, P = x.shape
    G, N = Bm.shape[1], Bm.shape[2]
    dtype = _dtype_code(x)
    for t, nm in ((dt, "dt"), (A, "A"), (h_state, "h_state"), (chunk_acc, "chunk_acc")):
        _check_f32(t, nm)
    z_per_head = 1 if z.dim() == 2 else 0
    dims = make_dims(B_, 0, H, P, N, chunk, dtype, G, mem_cache.shape[1])
    opts = SmaOpts(float(eps), _ptr(q_norm_w), _ptr(e_norm_w), int(bool(normalize)), z_per_head)
    if y is None:
        y = torch.empty_like(x)
    need = lib.dart_decode_workspace_bytes(ctypes.byref(dims))
    if workspace is None:
        workspace = _workspace(need, x.device)
    check(lib.dart_decode_step(ctypes.byref(dims), ctypes.byref(opts), int(pos), _ptr(x), _ptr(dt),
                               _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(q), _ptr(e), _ptr(z),
                               _ptr(h_state), _ptr(chunk_acc), _ptr(mem_cache), _ptr(y),
                               _ptr(workspace), workspace.numel(), _stream(stream)))
    return y


def decode_step_noalloc(pos, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc, mem_cache, chunk,
                        eps=DEFAULT_EPS, normalize=True, q_norm_w=None, e_norm_w=None, y=None,
                        stream=None):
    """dart_decode_step_noalloc: the decode step with the library's fixed
    device scratch instead of a workspace (y is allocated here unless given)."""
    torch = _torch()
    lib = load_library()
    B_, H, P = x.shape
    G, N = Bm.shape[1], Bm.shape[2]
    dtype = _dtype_code(x)
    for t, nm in ((dt, "dt"), (A, "A"), (h_state, "h_state"), (chunk_acc, "chunk_acc")):
        _check_f32(t, nm)
    z_per_head = 1 if z.dim() == 2 else 0
    dims = make_dims(B_, 0, H, P, N, chunk, dtype, G, mem_cache.shape[1])
    opts = SmaOpts(float(eps), _ptr(q_norm_w), _ptr(e_norm_w), int(bool(normalize)), z_per_head)
    if y is None:
        y = torch.empty_like(x)
    check(lib.dart_decode_step_noalloc(ctypes.byref(dims), ctypes.byref(opts), int(pos), _ptr(x),
                                       _ptr(dt), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(q), _ptr(e),
                                       _ptr(z), _ptr(h_state), _ptr(chunk_acc), _ptr(mem_cache),
                                       _ptr(y), _stream(stream)))
    return y


def decode_step_ragged(pos, pos_max, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc, mem_cache,
                       chunk, eps=DEFAULT_EPS, normalize=True, q_norm_w=None, e_norm_w=None,
                       y=None, workspace=None, stream=None):
    """One decode step of a ragged batch (dart_decode_step_ragged): row b at
    position pos[b] (int64 device tensor [B]); pos_max bounds pos (host int).
    Updates h_state, chunk_acc and mem_cache in place; returns y [B][H][P]."""
    torch = _torch()
    lib = load_library()
    B_, H, P = x.shape
    G, N = Bm.shape[1], Bm.shape[2]
    dtype = _dtype_code(x)
    for t, nm in ((dt, "dt"), (A, "A"), (h_state, "h_state"), (chunk_acc, "chunk_acc")):
        _check_f32(t, nm)
    if pos.dtype != torch.int64 or not pos.is_cuda or pos.numel() != B_:
        raise ValueError("pos must be an int64 device tensor of %d entries" % B_)
    z_per_head = 1 if z.dim() == 2 else 0
    dims = make_dims(B_, 0, H, P, N, chunk, dtype, G, mem_cache.shape[1])
    opts = SmaOpts(float(eps), _ptr(q_norm_w), _ptr(e_norm_w), int(bool(normalize)), z_per_head)
    if y is None:
        y = torch.empty_like(x)
    need = lib.dart_decode_workspace_bytes(ctypes.byref(dims))
    if workspace is None:
        workspace = _workspace(need, x.device)
    check(lib.dart_decode_step_ragged(ctypes.byref(dims), ctypes.byref(opts), _ptr(pos), int(pos_max),
                                      _ptr(x), _ptr(dt), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(q),
                                      _ptr(e), _ptr(z), _ptr(h_state), _ptr(chunk_acc),
                                      _ptr(mem_cache), _ptr(y), _ptr(workspace), workspace.numel(),
                                      _stream(stream)))
    return y


def decode_handoff(lengths, mem, h_last, chunk, h_state=None, chunk_acc=None, stream=None):
    """Decode state after a (dt = 0 padded) prefill (dart_decode_handoff):
    returns (h_state, chunk_acc) for the rows' next positions lengths[b]."""
    torch = _torch()
    lib = load_library()
    B_, Mcap, H, N, P = mem.shape
    dtype = _dtype_code(mem)
    _check_f32(h_last, "h_last")
    if lengths.dtype != torch.int64 or not lengths.is_cuda or lengths.numel() != B_:
        raise ValueError("lengths must be an int64 device tensor of %d entries" % B_)
    dims = make_dims(B_, 0, H, P, N, chunk, dtype, 1, Mcap)
    if h_state is None:
        h_state = torch.empty_like(h_last)
    if chunk_acc is None:
        chunk_acc = torch.empty_like(h_last)
    check(lib.dart_decode_handoff(ctypes.byref(dims), _ptr(lengths), _ptr(mem), _ptr(h_last),
                                  _ptr(h_state), _ptr(chunk_acc), _stream(stream)))
    return h_state, chunk_acc


def workspace_bytes(kind: str, dims: Dims) -> int:
    lib = load_library()
    fn = {"scan": lib.dart_scan_workspace_bytes, "sma": lib.dart_sma_workspace_bytes,
          "sma_bwd": lib.dart_sma_bwd_workspace_bytes,
          "ssd_bwd": lib.dart_ssd_bwd_workspace_bytes,
          "decode": lib.dart_decode_workspace_bytes}[kind]
    return int(fn(ctypes.byref(dims)))


def decode_cache_elems(dims: Dims, context: int) -> int:
    return int(load_library().dart_decode_cache_elems(ctypes.byref(dims), int(context)))


# --------------------------------------------------------------------------- #
# optional kernel timing (dart_profile_* in dart.h)
# --------------------------------------------------------------------------- #

def profile_enable(on: bool = True):
    check(load_library().dart_profile_enable(1 if on else 0))


def profile_filter(kernel: Optional[str] = None):
    """Time only the launches of `kernel` (None: every kernel)."""
    check(load_library().dart_profile_filter(kernel.encode() if kernel else None))


def profile_reset():
    load_library().dart_profile_reset()


def profile_read(reset: bool = False):
    """Flush pending kernel events and return {kernel: (total_ms, launches)}."""
    lib = load_library()
    check(lib.dart_profile_flush())
    out = {}
    for i in range(lib.dart_profile_count()):
        out[lib.dart_profile_name(i).decode()] = (float(lib.dart_profile_total_ms(i)),
                                                  int(lib.dart_profile_launches(i)))
    if reset:
        lib.dart_profile_reset()
    return out
