"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects malformed arguments before
launching anything (so these run without a GPU)."""
import ctypes
import json
import os
import re
import subprocess

import pytest

from paper_2608_02032_amd import dart

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dart.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(dart.LIB_PATH):
        pytest.skip("libdart.so not built")
    return dart.load_library()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dart_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_three_entry_points():
    fns = declared_functions()
    for name in ("dart_ssd_chunk_scan", "dart_sma_fwd", "dart_decode_step"):
        assert name in fns
    assert set(fns) == set(dart.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", dart.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (dart_[a-z_0-9]+)\b", out))
    missing = set(declared_functions()) - exported
    assert not missing, missing
    for name in declared_functions():
        assert hasattr(lib, name)


def dims(**kw):
    base = dict(batch=2, seqlen=512, nheads=4, headdim=64, dstate=64, chunk=64, dtype="bf16",
                ngroups=1, mem_capacity=0)
    base.update(kw)
    return dart.make_dims(**base)


def test_status_strings(lib):
    assert lib.dart_status_string(0) == b"DART_OK"
    assert lib.dart_status_string(1) == b"DART_ERR_INVALID_ARG"
    assert lib.dart_status_string(2) == b"DART_ERR_UNSUPPORTED"
    assert lib.dart_status_string(3) == b"DART_ERR_HIP"


def test_workspace_sizes(lib):
    d = dims()
    M = 512 // 64
    ws = lib.dart_scan_workspace_bytes(ctypes.byref(d))
    # chunk log-decays, chunk-entry states (storage dtype) and the per-token
    # record (cumulative log decay, dt, weight); fp32 adds the causal Gram
    # tiles (float; one set per group)
    assert ws >= 4 * 2 * 4 * M + 2 * 2 * M * 4 * 64 * 64 + 4 * 2 * 4 * M * 3 * 64
    pairs = (64 // 32) * (64 // 32 + 1)
    ws32 = lib.dart_scan_workspace_bytes(ctypes.byref(dims(dtype="fp32")))
    assert ws32 >= (4 * 2 * 4 * M + 4 * 2 * M * 4 * 64 * 64 + 4 * 2 * 4 * M * 3 * 64
                    + 4 * 2 * 1 * M * pairs * 512)
    # the SMA forward keeps the key side r (.) dH of every attended memory
    sma = lib.dart_sma_workspace_bytes(ctypes.byref(d))
    assert sma >= 2 * 2 * (M - 1) * 4 * 64 * 64
    d1 = dims(seqlen=64)  # one chunk: no memory is ever attended
    assert lib.dart_sma_workspace_bytes(ctypes.byref(d1)) == 0
    dd = dims(seqlen=0, mem_capacity=40)
    # at least one partial (O[64], m, d) per (b, h) plus the SSM readout y_ssd
    assert lib.dart_decode_workspace_bytes(ctypes.byref(dd)) >= 4 * 2 * 4 * (66 + 64)
    bad = dims(headdim=48)
    assert lib.dart_scan_workspace_bytes(ctypes.byref(bad)) == 0


NULL = None


def call_scan(lib, d, **ptrs):
    p = dict(x=1, dt=1, A=1, Bm=1, Cm=1, h0=NULL, y=1, mem=1, hl=NULL, ws=1)
    p.update(ptrs)
    nbytes = ptrs.get("nbytes", 1 << 40)
    return lib.dart_ssd_chunk_scan(ctypes.byref(d), p["x"], p["dt"], p["A"], p["Bm"], p["Cm"],
                                   p["h0"], p["y"], p["mem"], p["hl"], p["ws"], nbytes, None)


@pytest.mark.parametrize("field,value,status", [
    ("batch", 0, dart.DART_ERR_INVALID_ARG),
    ("seqlen", 0, dart.DART_ERR_INVALID_ARG),
    ("nheads", 3, dart.DART_ERR_INVALID_ARG),      # not a multiple of ngroups = 2 below
    ("dtype", 7, dart.DART_ERR_INVALID_ARG),
    ("headdim", 128, dart.DART_ERR_UNSUPPORTED),
    ("dstate", 48, dart.DART_ERR_UNSUPPORTED),
    ("chunk", 8192, dart.DART_ERR_UNSUPPORTED),
    ("mem_capacity", 3, dart.DART_ERR_INVALID_ARG),  # < ceil(512/64) = 8
])
def test_scan_rejects_bad_dims(lib, field, value, status):
    kw = {"ngroups": 2} if field == "nheads" else {}
    kw[field] = value
    d = dims(**kw)
    assert call_scan(lib, d) == status
    assert lib.dart_last_error()


@pytest.mark.parametrize("name", ["x", "dt", "A", "Bm", "Cm", "y", "mem", "ws"])
def test_scan_rejects_null_required_pointer(lib, name):
    assert call_scan(lib, dims(), **{name: NULL}) == dart.DART_ERR_INVALID_ARG
    assert name.encode() in lib.dart_last_error() or b"NULL" in lib.dart_last_error()


def test_scan_rejects_small_workspace(lib):
    d = dims()
    need = lib.dart_scan_workspace_bytes(ctypes.byref(d))
    assert call_scan(lib, d, nbytes=need - 1) == dart.DART_ERR_INVALID_ARG
    assert b"workspace" in lib.dart_last_error()


def test_sma_rejects_bad_opts_and_partial_alias(lib):
    d = dims()
    o = dart.SmaOpts(0.0, None, None, 1, 1)  # normalize needs eps > 0
    r = lib.dart_sma_fwd(ctypes.byref(d), ctypes.byref(o), 1, 1, 1, 1, 1, 1, 1, None, 1, 1 << 40, None)
    assert r == dart.DART_ERR_INVALID_ARG
    o = dart.SmaOpts(1e-6, None, None, 2, 1)
    r = lib.dart_sma_fwd(ctypes.byref(d), ctypes.byref(o), 1, 1, 1, 1, 1, 1, 1, None, 1, 1 << 40, None)
    assert r == dart.DART_ERR_INVALID_ARG
    o = dart.SmaOpts(1e-6, None, None, 1, 1)
    # y overlapping y_ssd by one element is rejected (exact aliasing is allowed)
    r = lib.dart_sma_fwd(ctypes.byref(d), ctypes.byref(o), 1, 1, 1, 1, 1, 4096, 4098, None, 1,
                         1 << 40, None)
    assert r == dart.DART_ERR_INVALID_ARG
    assert b"overlap" in lib.dart_last_error()


def call_decode(lib, d, pos, nbytes=1 << 40):
    o = dart.SmaOpts(1e-6, None, None, 1, 1)
    return lib.dart_decode_step(ctypes.byref(d), ctypes.byref(o), pos, 1, 1, 1, 1, 1, 1, 1, 1,
                                1, 1, 1, 1, 1, nbytes, None)


def test_decode_rejects_cache_overflow_and_bad_pos(lib):
    d = dims(seqlen=0, chunk=64, mem_capacity=4)
    assert call_decode(lib, d, -1) == dart.DART_ERR_INVALID_ARG
    # pos 255 closes chunk 3 into slot 3 (fits); pos 319 would write slot 4
    assert call_decode(lib, d, 319) == dart.DART_ERR_INVALID_ARG
    assert b"closes chunk" in lib.dart_last_error()
    # pos 320 needs 5 cached memories > 4
    assert call_decode(lib, d, 320) == dart.DART_ERR_INVALID_ARG
    d0 = dims(seqlen=0, mem_capacity=0)
    assert call_decode(lib, d0, 0) == dart.DART_ERR_INVALID_ARG
    dd = dims(seqlen=0, mem_capacity=4)
    need = lib.dart_decode_workspace_bytes(ctypes.byref(dd))
    assert call_decode(lib, dd, 10, nbytes=need - 1) == dart.DART_ERR_INVALID_ARG


def test_ragged_decode_and_handoff_reject_bad_arguments(lib):
    o = dart.SmaOpts(1e-6, None, None, 1, 1)
    d = dims(seqlen=0, chunk=64, mem_capacity=4)

    def ragged(pos_max, pos_ptr=1, nbytes=1 << 40, dd=d):
        return lib.dart_decode_step_ragged(ctypes.byref(dd), ctypes.byref(o), pos_ptr, pos_max, 1, 1,
                                           1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, nbytes, None)
    assert ragged(-1) == dart.DART_ERR_INVALID_ARG
    # positions up to 255 fit four memories; 256 could need slot 4
    assert ragged(256) == dart.DART_ERR_INVALID_ARG
    assert b"pos_max" in lib.dart_last_error()
    assert ragged(10, pos_ptr=None) == dart.DART_ERR_INVALID_ARG
    need = lib.dart_decode_workspace_bytes(ctypes.byref(d))
    assert ragged(10, nbytes=need - 1) == dart.DART_ERR_INVALID_ARG
    assert ragged(10, dd=dims(seqlen=0, mem_capacity=0)) == dart.DART_ERR_INVALID_ARG
    assert lib.dart_decode_handoff(ctypes.byref(d), None, 1, 1, 1, 1, None) == dart.DART_ERR_INVALID_ARG
    assert lib.dart_decode_handoff(ctypes.byref(dims(seqlen=0, mem_capacity=0)), 1, 1, 1, 1, 1,
                                   None) == dart.DART_ERR_INVALID_ARG


def test_cache_ratio_closed_form_matches_paper(lib):
    """Pin C-P12: element count of the length-dependent decode cache over the
    matched KV cache (2 L P per head) is N/(2S); the paper prints 25% at
    S = 256, N = 128 (fixture tests/golden/cache_ratio.json)."""
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "cache_ratio.json")))
    for case in gold["cases"]:
        B, H, P, ctx = 64, 32, 64, 65536
        d = dart.make_dims(B, 0, H, P, case["dstate"], case["chunk"], "bf16")
        ours = lib.dart_decode_cache_elems(ctypes.byref(d), ctx)
        kv = B * H * 2 * ctx * P
        assert ours / kv == pytest.approx(case["ratio"], abs=0)
        assert 1 - ours / kv == pytest.approx(case["saving"], abs=0)
    # other points of the closed form
    for S, N, r in [(64, 128, 1.0), (16, 16, 0.5), (128, 64, 0.25)]:
        d = dart.make_dims(1, 0, 1, 64, N, S, "bf16")
        assert lib.dart_decode_cache_elems(ctypes.byref(d), 4096) / (2 * 4096 * 64) == r


def test_sma_bwd_workspace_and_bad_arguments(lib):
    d = dims()
    M = 512 // 64
    ws = lib.dart_sma_bwd_workspace_bytes(ctypes.byref(d))
    # key side (storage dtype), normalised q (storage) and e (float), two floats
    # per (b, h, attended memory, token), partials per head block, R . dy
    assert ws >= (2 * 2 * (M - 1) * 4 * 64 * 64 + 2 * 2 * 512 * 64 + 4 * 2 * 512 * 64
                  + 2 * 4 * 2 * 4 * (M - 1) * 512 + 4 * 2 * 512 * 4)
    assert lib.dart_sma_bwd_workspace_bytes(ctypes.byref(dims(headdim=48))) == 0
    o = dart.SmaOpts(1e-6, None, None, 1, 1)

    def bwd(ptr_over=None, nbytes=1 << 40, opts=o):
        p = [1] * 13
        if ptr_over is not None:
            p[ptr_over] = None
        return lib.dart_sma_bwd(ctypes.byref(d), ctypes.byref(opts), *p, nbytes, None)
    for k in range(13):
        assert bwd(k) == dart.DART_ERR_INVALID_ARG
        assert b"required pointer" in lib.dart_last_error()
    assert bwd(nbytes=ws - 1) == dart.DART_ERR_INVALID_ARG
    assert b"workspace too small" in lib.dart_last_error()
    assert bwd(opts=dart.SmaOpts(0.0, None, None, 1, 1)) == dart.DART_ERR_INVALID_ARG


def test_ssd_bwd_workspace_and_bad_arguments(lib):
    d = dims()
    ws = lib.dart_ssd_bwd_workspace_bytes(ctypes.byref(d))
    per_chunk = d.batch * (512 // 64) * d.nheads * 64 * 64
    # bf16 (chunked matrix form): the chunk contributions of the state and of
    # the adjoint, the entry states and the chunk adjoints, bf16 per chunk
    assert ws >= 4 * 2 * per_chunk
    # fp32 (token sweeps): the forward scan's workspace plus R and dR, float
    d32 = dims(dtype="fp32")
    ws32 = lib.dart_ssd_bwd_workspace_bytes(ctypes.byref(d32))
    assert ws32 >= lib.dart_scan_workspace_bytes(ctypes.byref(d32)) + 2 * 4 * per_chunk
    assert lib.dart_ssd_bwd_workspace_bytes(ctypes.byref(dims(headdim=48))) == 0
    required = (0, 1, 2, 3, 4, 6, 9, 10, 11, 12, 13, 15)  # h0, dmem, dh_last, dh0 optional

    def bwd(ptr_over=None, nbytes=1 << 40):
        p = [1] * 16
        if ptr_over is not None:
            p[ptr_over] = None
        return lib.dart_ssd_bwd(ctypes.byref(d), *p, nbytes, None)
    for k in required:
        assert bwd(k) == dart.DART_ERR_INVALID_ARG
        assert b"required pointer" in lib.dart_last_error()
    assert bwd(nbytes=ws - 1) == dart.DART_ERR_INVALID_ARG
    assert b"workspace too small" in lib.dart_last_error()


def test_block_entry_points_reject_bad_arguments(lib):
    E = dart.DART_ERR_INVALID_ARG
    # conv: sizes, stride, dtype, pointers, aliasing of the state over a long sequence
    assert lib.dart_conv1d_silu(0, 8, 4, 4, 1, 1, 1, None, None, None, 1, None) == E
    assert lib.dart_conv1d_silu(1, 8, 4, 3, 1, 1, 1, None, None, None, 1, None) == E
    assert lib.dart_conv1d_silu(1, 8, 4, 4, 7, 1, 1, None, None, None, 1, None) == E
    assert lib.dart_conv1d_silu(1, 8, 4, 4, 1, None, 1, None, None, None, 1, None) == E
    assert lib.dart_conv1d_silu(1, 33, 4, 4, 1, 1, 1, None, 8, 8, 1, None) == E
    assert b"alias" in lib.dart_last_error()
    # dt
    assert lib.dart_dt_softplus(4, 3, 2, 1, 1, None, 1, None) == E
    assert lib.dart_dt_softplus(4, 3, 3, 1, None, None, 1, None) == E
    # gated norm: group must divide dim and be a multiple of 8; z stride; alignment; eps
    assert lib.dart_gated_rmsnorm(2, 64, 24, 1, 16, 16, 64, None, 1e-6, 16, None) == E
    assert lib.dart_gated_rmsnorm(2, 64, 12, 1, 16, 16, 64, None, 1e-6, 16, None) == E
    assert lib.dart_gated_rmsnorm(2, 64, 64, 1, 16, 16, 60, None, 1e-6, 16, None) == E
    assert lib.dart_gated_rmsnorm(2, 64, 64, 1, 8, 16, 64, None, 1e-6, 16, None) == E
    assert b"aligned" in lib.dart_last_error()
    assert lib.dart_gated_rmsnorm(2, 64, 64, 1, 16, 16, 64, None, 0.0, 16, None) == E


def test_noalloc_decode_rejects_a_step_beyond_its_scratch(lib):
    """dart_decode_step_noalloc refuses, before any launch, a step whose
    partials would not fit the fixed scratch: B = 4096, H = 64 needs
    4096 * 64 * (66 + 64) * 4 bytes > 16 MiB even for one split."""
    d = dims(batch=4096, nheads=64, seqlen=0, mem_capacity=4)
    opts = dart.SmaOpts(1e-6, None, None, 1, 1)
    buf = ctypes.create_string_buffer(64)
    p = ctypes.cast(buf, ctypes.c_void_p)
    st = lib.dart_decode_step_noalloc(ctypes.byref(d), ctypes.byref(opts), 64, *([p] * 12), None)
    assert st == 2, lib.dart_last_error()
    assert b"scratch" in lib.dart_last_error()
    # a NULL required pointer is still an argument error, found first
    st = lib.dart_decode_step_noalloc(ctypes.byref(d), ctypes.byref(opts), 64, None, *([p] * 11), None)
    assert st == 1


@pytest.mark.parametrize("N,S", [(16, 16), (16, 256), (64, 32), (128, 48), (32, 1)])
def test_generic_shapes_are_accepted_and_sized(lib, N, S):
    """Shapes outside the tuned set (N in {32, 64, 128} with S in {64, 128,
    256}) run the generic kernels: they size workspaces instead of returning
    DART_ERR_UNSUPPORTED."""
    d = dims(dstate=N, chunk=S, seqlen=300)
    M = -(-300 // S)
    assert lib.dart_scan_workspace_bytes(ctypes.byref(d)) >= 2 * 2 * M * 4 * N * 64
    assert lib.dart_sma_bwd_workspace_bytes(ctypes.byref(d)) > 0
    assert lib.dart_ssd_bwd_workspace_bytes(ctypes.byref(d)) > 0
    dd = dims(dstate=N, chunk=S, seqlen=0, mem_capacity=M)
    assert lib.dart_decode_workspace_bytes(ctypes.byref(dd)) > 0
