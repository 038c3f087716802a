"""Plain fp64 CPU oracle for DART's hot path (arXiv 2608.02032).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` are the only users.  The product library
(``paper_2608_02032_amd``) never imports this package, and this package never
imports the product.

The arithmetic lives in ``dart_oracle.c`` (literal loops in double precision,
one function per definition of the paper; see its header for the citations).
This module only compiles it with gcc, loads it with ctypes and marshals
numpy arrays.  Every array argument is converted to a C-contiguous float64
array; callers pass values already rounded to the storage precision of the
GPU path (the rounding itself is input preparation, not oracle arithmetic).

parity: see the header of ``dart_oracle.c``; the RMS epsilon, norm weights
and gate granularity are conventions the paper leaves open (parity unpinned
for those conventions beyond the oracle self-tests).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dart_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.c_int64
_INT = ctypes.c_int


def build(force: bool = True) -> str:
    """Compile dart_oracle.c into liboracle.so (plain gcc, OpenMP over rows)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall",
               "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        lib.dart_oracle_ssd_recurrence.argtypes = [_I64, _I64, _INT, _INT, _INT, _INT,
                                                   _D, _D, _D, _D, _D, _D, _D, _D]
        lib.dart_oracle_ssd_recurrence.restype = None
        lib.dart_oracle_ssd_bwd.argtypes = [_I64, _I64, _INT, _INT, _INT, _INT, _INT, _I64,
                                            _D, _D, _D, _D, _D, _D, _D, _D, _D,
                                            _D, _D, _D, _D, _D, _D]
        lib.dart_oracle_ssd_bwd.restype = None
        lib.dart_oracle_conv1d_silu.argtypes = [_I64, _I64, _INT, _I64, _D, _D, _D, _D, _D, _D]
        lib.dart_oracle_conv1d_silu.restype = None
        lib.dart_oracle_dt_softplus.argtypes = [_I64, _INT, _D, _D, _D]
        lib.dart_oracle_dt_softplus.restype = None
        lib.dart_oracle_gated_rmsnorm.argtypes = [_I64, _INT, _INT, ctypes.c_double, _D, _D, _D, _D]
        lib.dart_oracle_gated_rmsnorm.restype = None
        lib.dart_oracle_conv1d_silu_bwd.argtypes = [_I64, _I64, _INT, _I64] + [_D] * 9
        lib.dart_oracle_conv1d_silu_bwd.restype = None
        lib.dart_oracle_dt_softplus_bwd.argtypes = [_I64, _INT] + [_D] * 5
        lib.dart_oracle_dt_softplus_bwd.restype = None
        lib.dart_oracle_gated_rmsnorm_bwd.argtypes = [_I64, _INT, _INT, ctypes.c_double] + [_D] * 7
        lib.dart_oracle_gated_rmsnorm_bwd.restype = None
        lib.dart_oracle_chunk_memories.argtypes = [_I64, _I64, _INT, _INT, _INT, _INT, _INT, _I64,
                                                   _D, _D, _D, _D, _D]
        lib.dart_oracle_chunk_memories.restype = None
        lib.dart_oracle_sma.argtypes = [_I64, _I64, _INT, _INT, _INT, _INT, _INT, _I64,
                                        ctypes.c_double, _INT, _INT,
                                        _D, _D, _D, _D, _D, _D, _D, _D, _D, _D, _D]
        lib.dart_oracle_sma.restype = None
        lib.dart_oracle_sma_rows.argtypes = [_I64, _I64, _INT, _INT, _INT, _INT, _INT, _I64,
                                             ctypes.c_double, _INT, _INT,
                                             _D, _D, _D, _D, _D, _D, _D, _D,
                                             _I64, ctypes.POINTER(ctypes.c_int64), _D, _D]
        lib.dart_oracle_sma_rows.restype = None
        lib.dart_oracle_decode_step.argtypes = [_I64, _INT, _INT, _INT, _INT, _INT, _I64, _I64,
                                                ctypes.c_double, _INT, _INT,
                                                _D, _D, _D, _D, _D, _D, _D, _D, _D, _D,
                                                _D, _D, _D, _D]
        lib.dart_oracle_decode_step.restype = ctypes.c_int
        lib.dart_oracle_sma_bwd.argtypes = [_I64, _I64, _INT, _INT, _INT, _INT, _INT, _I64,
                                            ctypes.c_double, _INT, _INT,
                                            _D, _D, _D, _D, _D, _D, _D, _D,
                                            _D, _D, _D, _D, _D]
        lib.dart_oracle_sma_bwd.restype = None
        _lib = lib
        return lib


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(_D)


def ssd_recurrence(x, dt, A, Bm, Cm, h0=None):
    """Token-level SSD recurrence (Sec. 2).  Shapes as in Table 7.

    x [B][L][H][P], dt [B][L][H], A [H], Bm/Cm [B][L][G][N], h0 [B][H][N][P] or None.
    Returns (y_ssd [B][L][H][P], h_last [B][H][N][P]).
    """
    x, dt, A, Bm, Cm = map(_f64, (x, dt, A, Bm, Cm))
    B_, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    h0 = None if h0 is None else _f64(h0)
    y = np.empty((B_, L, H, P))
    hl = np.empty((B_, H, N, P))
    _load().dart_oracle_ssd_recurrence(B_, L, H, G, P, N, _ptr(x), _ptr(dt), _ptr(A), _ptr(Bm),
                                       _ptr(Cm), _ptr(h0), _ptr(y), _ptr(hl))
    return y, hl


def chunk_memories(x, dt, A, Bm, S, mem_capacity=None):
    """Chunk state memories dH_[c] by the brute-force definition (Sec. 3, App. A).

    Returns mem [B][Mcap][H][N][P]; slots beyond ceil(L/S) are zero.
    """
    x, dt, A, Bm = map(_f64, (x, dt, A, Bm))
    B_, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    M = -(-L // S)
    Mcap = M if mem_capacity is None else int(mem_capacity)
    mem = np.zeros((B_, Mcap, H, N, P))
    _load().dart_oracle_chunk_memories(B_, L, H, G, P, N, int(S), Mcap, _ptr(x), _ptr(dt),
                                       _ptr(A), _ptr(Bm), _ptr(mem))
    return mem


def ssd_bwd(x, dt, A, Bm, Cm, S, dy, dmem=None, dh_last=None, h0=None):
    """Gradients of sum(dy * y_ssd) + sum(dmem * mem) + sum(dh_last * h_last)
    for the recurrence of Sec. 2 and the memories of Sec. 3, by running the
    recurrence backwards.  Shapes as ssd_recurrence / chunk_memories; dmem is
    [B][Mcap][H][N][P] (Mcap >= ceil(L/S)).  Returns {"dx", "ddt", "dA",
    "dB", "dC", "dh0"} (B and C gradients summed over each group's heads)."""
    x, dt, A, Bm, Cm, dy = map(_f64, (x, dt, A, Bm, Cm, dy))
    B_, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    dmem = None if dmem is None else _f64(dmem)
    Mcap = dmem.shape[1] if dmem is not None else -(-L // S)
    assert Mcap >= -(-L // S)
    dhl = None if dh_last is None else _f64(dh_last)
    h0 = None if h0 is None else _f64(h0)
    out = {"dx": np.empty_like(x), "ddt": np.empty_like(dt), "dA": np.empty_like(A),
           "dB": np.empty_like(Bm), "dC": np.empty_like(Cm), "dh0": np.zeros((B_, H, N, P))}
    _load().dart_oracle_ssd_bwd(B_, L, H, G, P, N, int(S), Mcap, _ptr(x), _ptr(dt), _ptr(A),
                                _ptr(Bm), _ptr(Cm), _ptr(h0), _ptr(dy), _ptr(dmem), _ptr(dhl),
                                _ptr(out["dx"]), _ptr(out["ddt"]), _ptr(out["dA"]),
                                _ptr(out["dB"]), _ptr(out["dC"]), _ptr(out["dh0"]))
    return out


def sma(q, e, Cm, mem, z, y_ssd, S, eps=1e-6, normalize=True, q_norm_w=None, e_norm_w=None,
        return_R=False):
    """State-memory attention + gated residual (Sec. 3, App. B.1).

    q [B][L][G][N], e [B][L][G][P], Cm [B][L][G][N], mem [B][Mcap][H][N][P],
    z [B][L][H] (one gate per head) or [B][L] (one gate per token), y_ssd [B][L][H][P].
    Returns (y, lse) or (y, lse, R).
    """
    q, e, Cm, mem, z, y_ssd = map(_f64, (q, e, Cm, mem, z, y_ssd))
    B_, L, H, P = y_ssd.shape
    G, N = q.shape[2], q.shape[3]
    Mcap = mem.shape[1]
    assert Mcap >= -(-L // S)
    z_per_head = 1 if z.ndim == 3 else 0
    qw = None if q_norm_w is None else _f64(q_norm_w)
    ew = None if e_norm_w is None else _f64(e_norm_w)
    y = np.empty((B_, L, H, P))
    lse = np.empty((B_, L, H))
    R = np.empty((B_, L, H, P)) if return_R else None
    _load().dart_oracle_sma(B_, L, H, G, P, N, int(S), Mcap, float(eps), int(bool(normalize)),
                            z_per_head, _ptr(q), _ptr(e), _ptr(Cm), _ptr(qw), _ptr(ew), _ptr(mem),
                            _ptr(z), _ptr(y_ssd), _ptr(y), _ptr(lse), _ptr(R))
    return (y, lse, R) if return_R else (y, lse)


def sma_rows(q, e, Cm, mem, z, y_ssd, S, rows, eps=1e-6, normalize=True, q_norm_w=None,
             e_norm_w=None):
    """The SMA definition evaluated at selected rows only.

    rows: int array [K][3] of (b, t, h).  Returns (y_rows [K][P], lse_rows [K]).
    Arrays may be large; they are converted to float64 once.
    """
    q, e, Cm, mem, z, y_ssd = map(_f64, (q, e, Cm, mem, z, y_ssd))
    B_, L, H, P = y_ssd.shape
    G, N = q.shape[2], q.shape[3]
    Mcap = mem.shape[1]
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1, 3))
    z_per_head = 1 if z.ndim == 3 else 0
    qw = None if q_norm_w is None else _f64(q_norm_w)
    ew = None if e_norm_w is None else _f64(e_norm_w)
    K = rows.shape[0]
    yr = np.empty((K, P))
    lr = np.empty((K,))
    _load().dart_oracle_sma_rows(B_, L, H, G, P, N, int(S), Mcap, float(eps), int(bool(normalize)),
                                 z_per_head, _ptr(q), _ptr(e), _ptr(Cm), _ptr(qw), _ptr(ew),
                                 _ptr(mem), _ptr(z), _ptr(y_ssd), K,
                                 rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                 _ptr(yr), _ptr(lr))
    return yr, lr


def sma_bwd(q, e, Cm, mem, z, dy, S, eps=1e-6, normalize=True, q_norm_w=None, e_norm_w=None):
    """Gradients of the SMA + gate forward for the loss sum(dy * y), by
    recomputing every row (App. C) and the chain rule through Sec. 3 and
    App. B.1 (the norm weights are constants).  Shapes as in sma(); dy like
    y_ssd.  Returns {"dq", "de", "dC", "dmem", "dz", "dy_ssd"}: q, e, C
    gradients summed over the heads of their group, dmem in the cache layout
    (slots never attended are zero), dz like z, dy_ssd = dy."""
    q, e, Cm, mem, z, dy = map(_f64, (q, e, Cm, mem, z, dy))
    B_, L, H, P = dy.shape
    G, N = q.shape[2], q.shape[3]
    Mcap = mem.shape[1]
    assert Mcap >= -(-L // S)
    z_per_head = 1 if z.ndim == 3 else 0
    qw = None if q_norm_w is None else _f64(q_norm_w)
    ew = None if e_norm_w is None else _f64(e_norm_w)
    out = {"dq": np.empty_like(q), "de": np.empty_like(e), "dC": np.empty_like(Cm),
           "dmem": np.empty_like(mem), "dz": np.empty_like(z)}
    _load().dart_oracle_sma_bwd(B_, L, H, G, P, N, int(S), Mcap, float(eps), int(bool(normalize)),
                                z_per_head, _ptr(q), _ptr(e), _ptr(Cm), _ptr(qw), _ptr(ew),
                                _ptr(mem), _ptr(z), _ptr(dy), _ptr(out["dq"]), _ptr(out["de"]),
                                _ptr(out["dC"]), _ptr(out["dmem"]), _ptr(out["dz"]))
    out["dy_ssd"] = dy.copy()
    return out


def forward(x, dt, A, Bm, Cm, q, e, z, S, eps=1e-6, normalize=True, q_norm_w=None,
            e_norm_w=None, h0=None):
    """Whole layer path from scratch: recurrence, brute-force memories, SMA, gate."""
    y_ssd, h_last = ssd_recurrence(x, dt, A, Bm, Cm, h0)
    mem = chunk_memories(x, dt, A, Bm, S)
    y, lse = sma(q, e, Cm, mem, z, y_ssd, S, eps, normalize, q_norm_w, e_norm_w)
    return {"y_ssd": y_ssd, "h_last": h_last, "mem": mem, "y": y, "lse": lse}


def decode_step(pos, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc, mem, S, eps=1e-6,
                normalize=True, q_norm_w=None, e_norm_w=None):
    """One autoregressive token at position ``pos`` for every sequence.

    x [B][H][P], dt [B][H], Bm/Cm/q [B][G][N], e [B][G][P], z [B][H] or [B];
    h_state, chunk_acc [B][H][N][P] and mem [B][Mcap][H][N][P] are updated IN PLACE
    (they must be C-contiguous float64 arrays).  Returns y [B][H][P].
    """
    x, dt, A, Bm, Cm, q, e, z = map(_f64, (x, dt, A, Bm, Cm, q, e, z))
    for arr in (h_state, chunk_acc, mem):
        if not (isinstance(arr, np.ndarray) and arr.dtype == np.float64
                and arr.flags["C_CONTIGUOUS"]):
            raise TypeError("decode state arrays must be C-contiguous float64 ndarrays")
    B_, H, P = x.shape
    G, N = Bm.shape[1], Bm.shape[2]
    Mcap = mem.shape[1]
    z_per_head = 1 if z.ndim == 2 else 0
    qw = None if q_norm_w is None else _f64(q_norm_w)
    ew = None if e_norm_w is None else _f64(e_norm_w)
    y = np.empty((B_, H, P))
    rc = _load().dart_oracle_decode_step(B_, H, G, P, N, int(S), Mcap, int(pos), float(eps),
                                         int(bool(normalize)), z_per_head, _ptr(x), _ptr(dt),
                                         _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(q), _ptr(e), _ptr(qw),
                                         _ptr(ew), _ptr(z), _ptr(h_state), _ptr(chunk_acc),
                                         _ptr(mem), _ptr(y))
    if rc != 0:
        raise ValueError("decode position %d does not fit a cache of %d memories" % (pos, Mcap))
    return y


def conv1d_silu(inp, w, bias=None, state=None, channels=None):
    """Causal width-4 depthwise convolution + bias + SiLU over the token axis.
    inp [B][L][R] (the first `channels` of each row's R elements are the
    channels, default all), w [C][4] (w[c][3] multiplies the current token),
    bias [C], state [B][C][3] (the three inputs before token 0, oldest first)
    or None.  Returns (out [B][L][C], state_out [B][C][3])."""
    inp, w = _f64(inp), _f64(w)
    B_, L, R = inp.shape
    C = R if channels is None else int(channels)
    bias = None if bias is None else _f64(bias)
    state = None if state is None else _f64(state)
    out = np.empty((B_, L, C))
    st = np.empty((B_, C, 3))
    _load().dart_oracle_conv1d_silu(B_, L, C, R, _ptr(inp), _ptr(w), _ptr(bias), _ptr(state),
                                    _ptr(out), _ptr(st))
    return out, st


def dt_softplus(raw, bias=None):
    """dt = softplus(raw + bias[h]); raw [..][H]."""
    raw = _f64(raw)
    H = raw.shape[-1]
    bias = None if bias is None else _f64(bias)
    out = np.empty_like(raw)
    _load().dart_oracle_dt_softplus(raw.size // H, H, _ptr(raw), _ptr(bias), _ptr(out))
    return out


def gated_rmsnorm(y, z, w=None, group=None, eps=1e-6):
    """u = y * SiLU(z); u / sqrt(mean over each group of `group` channels of
    u^2 + eps) * w.  y, z [..][D]; w [D] or None."""
    y, z = _f64(y), _f64(z)
    D = y.shape[-1]
    group = D if group is None else int(group)
    w = None if w is None else _f64(w)
    out = np.empty_like(y)
    _load().dart_oracle_gated_rmsnorm(y.size // D, D, group, float(eps), _ptr(y), _ptr(z), _ptr(w),
                                      _ptr(out))
    return out


def conv1d_silu_bwd(inp, w, dout, bias=None, state=None, channels=None):
    """Gradients of conv1d_silu for a loss with output gradient dout [B][L][C]:
    returns {"din" [B][L][C], "dw" [C][4], "db" [C], "dstate" [B][C][3]}."""
    inp, w, dout = _f64(inp), _f64(w), _f64(dout)
    B_, L, R = inp.shape
    C = R if channels is None else int(channels)
    bias = None if bias is None else _f64(bias)
    state = None if state is None else _f64(state)
    out = {"din": np.empty((B_, L, C)), "dw": np.empty((C, 4)), "db": np.empty((C,)),
           "dstate": np.empty((B_, C, 3))}
    _load().dart_oracle_conv1d_silu_bwd(B_, L, C, R, _ptr(inp), _ptr(w), _ptr(bias), _ptr(state),
                                        _ptr(dout), _ptr(out["din"]), _ptr(out["dw"]),
                                        _ptr(out["db"]), _ptr(out["dstate"]))
    return out


def dt_softplus_bwd(raw, ddt, bias=None):
    """Gradients of dt_softplus: returns (draw like raw, dbias [H])."""
    raw, ddt = _f64(raw), _f64(ddt)
    H = raw.shape[-1]
    bias = None if bias is None else _f64(bias)
    draw = np.empty_like(raw)
    dbias = np.empty((H,))
    _load().dart_oracle_dt_softplus_bwd(raw.size // H, H, _ptr(raw), _ptr(bias), _ptr(ddt),
                                        _ptr(draw), _ptr(dbias))
    return draw, dbias


def gated_rmsnorm_bwd(y, z, dout, w=None, group=None, eps=1e-6):
    """Gradients of gated_rmsnorm: returns {"dy", "dz" like y, "dw" [D]}."""
    y, z, dout = _f64(y), _f64(z), _f64(dout)
    D = y.shape[-1]
    group = D if group is None else int(group)
    w = None if w is None else _f64(w)
    out = {"dy": np.empty_like(y), "dz": np.empty_like(y), "dw": np.empty((D,))}
    _load().dart_oracle_gated_rmsnorm_bwd(y.size // D, D, group, float(eps), _ptr(y), _ptr(z),
                                          _ptr(w), _ptr(dout), _ptr(out["dy"]), _ptr(out["dz"]),
                                          _ptr(out["dw"]))
    return out
