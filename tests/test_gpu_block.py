"""GPU parity of the block kernels around the path (dart_conv1d_silu,
dart_dt_softplus, dart_gated_rmsnorm) against the oracle's definitions on the
same seeded inputs: max|gpu - ref| / max|ref| per slice -- per (batch row,
channel) for the convolution, per (row, head) for the step sizes, per (row,
group) for the gated norm -- 1e-4 for fp32 storage and 2e-2 for bf16 (outputs
rounded to bf16)."""
import numpy as np
import pytest

import oracle
from paper_2608_02032_amd import dart, synth
from tests.helpers import TOL, assert_close_slices, f32_dev, to_dev, to_np

pytestmark = pytest.mark.gpu


def announce(msg):
    print("\n[gpu-case] " + msg, flush=True)


# C, the row stride and the pointers multiples of 8 take the 8-channel kernel
@pytest.mark.parametrize("dtype,B,L,R,C", [("fp32", 2, 150, 40, 33), ("bf16", 3, 64, 300, 290),
                                           ("bf16", 1, 1000, 2304, 2304), ("fp32", 2, 5, 8, 8),
                                           ("bf16", 2, 200, 2400, 2304), ("fp32", 2, 130, 72, 64)])
def test_conv1d_silu_matches_definition(dtype, B, L, R, C):
    import torch
    announce("conv1d %s B=%d L=%d R=%d C=%d" % (dtype, B, L, R, C))
    rng = np.random.default_rng(L + C)
    x = synth.to_storage(rng.standard_normal((B, L, R)).astype(np.float32), dtype)
    w = (rng.standard_normal((C, 4)) * 0.5).astype(np.float32)
    bias = (rng.standard_normal(C) * 0.1).astype(np.float32)
    st0 = rng.standard_normal((B, C, 3)).astype(np.float32)
    xd = to_dev(x, dtype)
    out, st = dart.conv1d_silu(xd, f32_dev(w), f32_dev(bias), state_in=f32_dev(st0),
                               state_out=True, channels=C)
    torch.cuda.synchronize()
    ref, st_ref = oracle.conv1d_silu(x, w, bias, state=st0, channels=C)
    tol = TOL[dtype]
    assert_close_slices(to_np(out), ref, tol, axes_keep=(0, 2), what="conv out")
    np.testing.assert_array_equal(to_np(st), st_ref)


@pytest.mark.parametrize("dtype,C", [("fp32", 70), ("bf16", 70), ("fp32", 64), ("bf16", 64)])
def test_conv1d_chunked_prefill_then_decode_steps(dtype, C):
    """Prefill in two calls carrying the state, then three single-token decode
    steps updating the state in place: equal to one pass over all tokens."""
    import torch
    B, L = 2, 97
    announce("conv1d chaining %s" % dtype)
    rng = np.random.default_rng(7)
    x = synth.to_storage(rng.standard_normal((B, L + 3, C)).astype(np.float32), dtype)
    w = (rng.standard_normal((C, 4)) * 0.5).astype(np.float32)
    ref, st_ref = oracle.conv1d_silu(x, w)
    xd = to_dev(x, dtype)
    wd = f32_dev(w)
    o1, s1 = dart.conv1d_silu(xd[:, :40].contiguous(), wd, state_out=True)
    o2, s2 = dart.conv1d_silu(xd[:, 40:L].contiguous(), wd, state_in=s1, state_out=True)
    outs = [o1, o2]
    for t in range(L, L + 3):
        o, _ = dart.conv1d_silu(xd[:, t:t + 1].contiguous(), wd, state_in=s2, state_out=s2)
        outs.append(o)
    torch.cuda.synchronize()
    got = np.concatenate([to_np(o) for o in outs], axis=1)
    assert_close_slices(got, ref, TOL[dtype], axes_keep=(0, 2), what="chained conv")
    np.testing.assert_array_equal(to_np(s2), st_ref)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_dt_softplus_matches_definition(dtype):
    import torch
    announce("dt softplus %s" % dtype)
    rng = np.random.default_rng(8)
    rows, H, R = 1000, 24, 40
    raw = synth.to_storage((rng.standard_normal((rows, R)) * 6).astype(np.float32), dtype)
    bias = rng.standard_normal(H).astype(np.float32)
    dt = dart.dt_softplus(to_dev(raw, dtype), f32_dev(bias), nheads=H)
    torch.cuda.synchronize()
    ref = oracle.dt_softplus(raw[:, :H], bias)
    assert_close_slices(to_np(dt), ref, 1e-5, axes_keep=(0, 1), what="dt")
    assert np.all(to_np(dt) > 0)


@pytest.mark.parametrize("dtype,rows,D,group,zs", [("fp32", 37, 128, 64, 200), ("bf16", 300, 2048, 2048, 2048),
                                                   ("bf16", 64, 1536, 768, 3000), ("fp32", 5, 24, 8, 24)])
def test_gated_rmsnorm_matches_definition(dtype, rows, D, group, zs):
    import torch
    announce("gated rmsnorm %s rows=%d D=%d group=%d" % (dtype, rows, D, group))
    rng = np.random.default_rng(D + group)
    y = synth.to_storage(rng.standard_normal((rows, D)).astype(np.float32), dtype)
    zfull = synth.to_storage(rng.standard_normal((rows, zs)).astype(np.float32), dtype)
    w = (1 + 0.1 * rng.standard_normal(D)).astype(np.float32)
    zd = to_dev(zfull, dtype)[:, :D]
    out = dart.gated_rmsnorm(to_dev(y, dtype), zd, f32_dev(w), group=group)
    torch.cuda.synchronize()
    ref = oracle.gated_rmsnorm(y, zfull[:, :D], w, group=group)
    ng = D // group
    assert_close_slices(to_np(out).reshape(rows, ng, group), ref.reshape(rows, ng, group), TOL[dtype],
                        axes_keep=(0, 1), what="gated rmsnorm")


# ---- backward (the block ops of a training step; App. D.1 trains two-layer
# models) against the oracle's chain-rule definitions, pinned by central
# differences ------------------------------------------------------------------

@pytest.mark.parametrize("dtype,B,L,R,C", [("fp32", 2, 70, 40, 33), ("bf16", 2, 200, 300, 290),
                                           ("fp32", 1, 3, 8, 8), ("bf16", 3, 64, 96, 96)])
def test_conv1d_silu_bwd_matches_definition(dtype, B, L, R, C):
    import torch
    announce("conv1d bwd %s B=%d L=%d R=%d C=%d" % (dtype, B, L, R, C))
    rng = np.random.default_rng(L + C + 1)
    x = synth.to_storage(rng.standard_normal((B, L, R)).astype(np.float32), dtype)
    w = (rng.standard_normal((C, 4)) * 0.5).astype(np.float32)
    bias = (rng.standard_normal(C) * 0.1).astype(np.float32)
    st0 = rng.standard_normal((B, C, 3)).astype(np.float32)
    dout = rng.standard_normal((B, L, C)).astype(np.float32)
    # din written into a strided float buffer (a projection gradient's slice)
    dbuf = torch.full((B, L, R + 5), 7.0, dtype=torch.float32, device="cuda")
    g = dart.conv1d_silu_bwd(to_dev(x, dtype), f32_dev(w), f32_dev(dout), bias=f32_dev(bias),
                             state_in=f32_dev(st0), channels=C, din=dbuf[:, :, 2:2 + C],
                             want_state=True)
    torch.cuda.synchronize()
    ref = oracle.conv1d_silu_bwd(x[:, :, :C], w, dout, bias=bias, state=st0)
    tol = TOL["fp32"] * 10 if dtype == "fp32" else 1e-4
    assert_close_slices(to_np(g["din"]), ref["din"], tol, axes_keep=(0, 2), what="din")
    assert_close_slices(to_np(g["dweight"]), ref["dw"], tol, axes_keep=(0,), what="dweight")
    assert_close_slices(to_np(g["dbias"]), ref["db"], tol, axes_keep=(), what="dbias")
    assert_close_slices(to_np(g["dstate"]), ref["dstate"], tol, axes_keep=(0, 1), what="dstate")
    # the buffer outside the slice is untouched
    b = to_np(dbuf)
    assert np.all(b[:, :, :2] == 7.0) and np.all(b[:, :, 2 + C:] == 7.0)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_dt_softplus_bwd_matches_definition(dtype):
    import torch
    announce("dt softplus bwd %s" % dtype)
    rng = np.random.default_rng(9)
    rows, H, R = 700, 6, 20
    raw = synth.to_storage((rng.standard_normal((rows, R)) * 4).astype(np.float32), dtype)
    bias = rng.standard_normal(H).astype(np.float32)
    ddt = rng.standard_normal((rows, H)).astype(np.float32)
    draw, dbias = dart.dt_softplus_bwd(to_dev(raw, dtype), f32_dev(ddt), bias=f32_dev(bias), nheads=H)
    torch.cuda.synchronize()
    rr, rb = oracle.dt_softplus_bwd(raw[:, :H], ddt, bias=bias)
    assert_close_slices(to_np(draw), rr, 1e-5, axes_keep=(0, 1), what="draw")
    assert_close_slices(to_np(dbias), rb, 1e-5, axes_keep=(0,), what="dbias")


@pytest.mark.parametrize("dtype,rows,D,group,zs", [("fp32", 37, 128, 64, 200), ("bf16", 300, 512, 512, 1024),
                                                   ("fp32", 5, 24, 8, 24), ("bf16", 40, 2048, 2048, 2048)])
def test_gated_rmsnorm_bwd_matches_definition(dtype, rows, D, group, zs):
    import torch
    announce("gated rmsnorm bwd %s rows=%d D=%d group=%d" % (dtype, rows, D, group))
    rng = np.random.default_rng(D + group + 1)
    y = synth.to_storage(rng.standard_normal((rows, D)).astype(np.float32), dtype)
    zfull = synth.to_storage(rng.standard_normal((rows, zs)).astype(np.float32), dtype)
    w = (1 + 0.1 * rng.standard_normal(D)).astype(np.float32)
    dout = rng.standard_normal((rows, D)).astype(np.float32)
    g = dart.gated_rmsnorm_bwd(to_dev(y, dtype), to_dev(zfull, dtype)[:, :D], f32_dev(dout),
                               weight=f32_dev(w), group=group)
    torch.cuda.synchronize()
    ref = oracle.gated_rmsnorm_bwd(y, zfull[:, :D], dout, w=w, group=group)
    ng = D // group
    tol = 1e-4
    for k in ("dy", "dz"):
        assert_close_slices(to_np(g[k]).reshape(rows, ng, group), ref[k].reshape(rows, ng, group),
                            tol, axes_keep=(0, 1), what=k)
    assert_close_slices(to_np(g["dweight"]), ref["dw"], tol, axes_keep=(), what="dweight")
