"""GPU parity of the generic kernels: shapes outside the tuned set (N in
{32, 64, 128} with S in {64, 128, 256}) -- the paper's MQAR chunk size S = 16
with N = 16 (App. D.1), its evaluation-time chunk sizes S = 32 and 64
(Sec. 5.2), a chunk size that is not a power of two, S = 1 and N = 16 at a
large S -- through the same C ABI and against the same oracle and metrics as
the tuned shapes (per slice, 1e-4 fp32, 2e-2 bf16; the readout R alone;
per-entry LSE bound)."""
import numpy as np
import pytest

import oracle
from paper_2608_02032_amd import dart, synth
from tests.helpers import TOL, assert_close_slices, assert_lse_close, f32_dev, to_dev, to_np
from tests.test_gpu_parity import check_readout, run_scan, run_sma, sma_case
from tests import test_gpu_scan_bwd as SB
from tests import test_gpu_sma_bwd as MB

pytestmark = pytest.mark.gpu


def announce(msg):
    print("\n[gpu-case] " + msg, flush=True)


SHAPES = [
    # name, B, L, H, N, S, dtype, G
    ("mqar_fp32_L256_N16_S16", 2, 256, 2, 16, 16, "fp32", 1),
    ("mqar_bf16_L250_N16_S16", 2, 250, 4, 16, 16, "bf16", 1),
    ("mqar_bf16_L512_N64_S16", 1, 512, 2, 64, 16, "bf16", 1),
    ("eval_bf16_L1000_N128_S32_G2", 1, 1000, 4, 128, 32, "bf16", 2),
    ("eval_fp32_L333_N64_S32", 2, 333, 3, 64, 32, "fp32", 1),
    ("odd_bf16_L500_N32_S48", 1, 500, 2, 32, 48, "bf16", 1),
    ("s1_fp32_L20_N16_S1", 1, 20, 2, 16, 1, "fp32", 1),
    ("bigS_bf16_L600_N16_S256", 1, 600, 2, 16, 256, "bf16", 1),
    ("S100_fp32_L250_N16", 1, 250, 2, 16, 100, "fp32", 1),
]


def wl(c):
    name, B, L, H, N, S, dtype, G = c
    return synth.Workload(name, B, L, H, 64, N, S, dtype, ngroups=G)


@pytest.mark.parametrize("c", SHAPES, ids=[c[0] for c in SHAPES])
def test_generic_scan_matches_recurrence(c):
    w = wl(c)
    announce("generic scan %s" % (w,))
    d = synth.forward_inputs(w, seed=5)
    y, mem, hl = run_scan(w, d)
    y_ref, hl_ref = oracle.ssd_recurrence(d["x"], d["dt"], d["A"], d["Bm"], d["Cm"])
    mem_ref = oracle.chunk_memories(d["x"], d["dt"], d["A"], d["Bm"], w.chunk)
    tol = TOL[w.dtype]
    assert_close_slices(to_np(y), y_ref, tol, what="y_ssd")
    assert_close_slices(to_np(mem), mem_ref, tol, axes_keep=(0, 1, 2), what="mem")
    assert_close_slices(to_np(hl), hl_ref, tol, axes_keep=(0, 1), what="h_last")


@pytest.mark.parametrize("c", SHAPES, ids=[c[0] for c in SHAPES])
def test_generic_sma_matches_explicit_softmax(c):
    w = wl(c)
    announce("generic sma %s" % (w,))
    d, mem, y_ssd = sma_case(w, seed=8)
    y, lse = run_sma(w, d, mem, y_ssd)
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, w.chunk)
    assert_close_slices(to_np(y), y_ref, TOL[w.dtype], what="y")
    assert_lse_close(to_np(lse), lse_ref, w.dtype)
    S = w.chunk
    np.testing.assert_array_equal(to_np(y)[:, :S], y_ssd[:, :S].astype(np.float64))
    check_readout(w, d, mem)


def test_generic_sma_options():
    w = synth.Workload("opts_bf16_L300_N16_S16", 1, 300, 4, 64, 16, 16, "bf16", z_per_head=False)
    announce("generic sma options %s" % (w,))
    d, mem, y_ssd = sma_case(w, seed=9)
    y, lse = run_sma(w, d, mem, y_ssd, normalize=False)
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, 16, normalize=False)
    assert_close_slices(to_np(y), y_ref, TOL["bf16"], what="y (normalize=0)")
    assert_lse_close(to_np(lse), lse_ref, "bf16")
    rng = np.random.default_rng(2)
    qw = rng.uniform(0.5, 1.5, 16).astype(np.float32)
    ew = rng.uniform(0.5, 1.5, 64).astype(np.float32)
    y, lse = run_sma(w, d, mem, y_ssd, q_norm_w=f32_dev(qw), e_norm_w=f32_dev(ew))
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, 16, q_norm_w=qw,
                                e_norm_w=ew)
    assert_close_slices(to_np(y), y_ref, TOL["bf16"], what="y (weights)")
    assert_lse_close(to_np(lse), lse_ref, "bf16")


BWD_SHAPES = [c for c in SHAPES if c[0] not in ("s1_fp32_L20_N16_S1",)] + [
    ("s1_fp32_L12_N16_S1", 1, 12, 2, 16, 1, "fp32", 1)]


@pytest.mark.parametrize("c", BWD_SHAPES, ids=[c[0] for c in BWD_SHAPES])
def test_generic_sma_bwd_matches_oracle(c):
    w = wl(c)
    announce("generic sma bwd %s" % (w,))
    d, mem, y_ssd, dy = MB.bwd_case(w, seed=13)
    got = MB.run_gpu(w, d, mem, y_ssd, dy)
    MB.check(w, got, d, mem, dy)


def test_generic_sma_bwd_options():
    w = synth.Workload("opts_bf16_L256_N16_S16_G2", 1, 256, 4, 64, 16, 16, "bf16", ngroups=2,
                       z_per_head=False)
    announce("generic sma bwd options %s" % (w,))
    d, mem, y_ssd, dy = MB.bwd_case(w, seed=14)
    rng = np.random.default_rng(3)
    qw = (1.0 + 0.2 * rng.standard_normal(16)).astype(np.float32)
    ew = (1.0 + 0.2 * rng.standard_normal(64)).astype(np.float32)
    got = MB.run_gpu(w, d, mem, y_ssd, dy, q_norm_w=f32_dev(qw), e_norm_w=f32_dev(ew))
    MB.check(w, got, d, mem, dy, " weights", q_norm_w=qw, e_norm_w=ew)
    got = MB.run_gpu(w, d, mem, y_ssd, dy, normalize=False)
    MB.check(w, got, d, mem, dy, " normalize=0", normalize=False)


@pytest.mark.parametrize("c", SHAPES, ids=[c[0] for c in SHAPES])
def test_generic_scan_bwd_matches_oracle(c):
    w = wl(c)
    SB.run_case(w, seed=17)


@pytest.mark.parametrize("dtype,S,N,L", [("fp32", 16, 16, 70), ("bf16", 16, 16, 80),
                                         ("bf16", 32, 64, 100)])
def test_generic_decode_token_by_token_reproduces_forward(dtype, S, N, L):
    import torch
    w = synth.Workload("gdec_%s_S%d_N%d" % (dtype, S, N), 2, L, 2, 64, N, S, dtype)
    announce("generic decode token-by-token %s" % (w,))
    d = synth.forward_inputs(w, seed=23)
    ref = oracle.forward(d["x"], d["dt"], d["A"], d["Bm"], d["Cm"], d["q"], d["e"], d["z"], S)
    B_, H, P = w.batch, w.nheads, w.headdim
    Mcap = -(-L // S)
    dev = {k: to_dev(d[k], dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    dt, A = f32_dev(d["dt"]), f32_dev(d["A"])
    h_state = torch.zeros((B_, H, N, P), dtype=torch.float32, device="cuda")
    chunk_acc = torch.zeros_like(h_state)
    cache = torch.zeros((B_, Mcap, H, N, P), dtype=dev["x"].dtype, device="cuda")
    ys = []
    for t in range(L):
        y = dart.decode_step(t, dev["x"][:, t].contiguous(), dt[:, t].contiguous(), A,
                             dev["Bm"][:, t].contiguous(), dev["Cm"][:, t].contiguous(),
                             dev["q"][:, t].contiguous(), dev["e"][:, t].contiguous(),
                             dev["z"][:, t].contiguous(), h_state, chunk_acc, cache, S)
        ys.append(y)
    torch.cuda.synchronize()
    y_all = np.stack([to_np(y) for y in ys], axis=1)
    tol = TOL[dtype]
    assert_close_slices(y_all, ref["y"], tol, what="decode y")
    full = L // S
    assert_close_slices(to_np(cache)[:, :full], ref["mem"][:, :full], tol, axes_keep=(0, 1, 2),
                        what="cache")
    assert_close_slices(to_np(h_state), ref["h_last"], tol, axes_keep=(0, 1), what="h_state")


@pytest.mark.parametrize("S", [32, 64])
def test_evaluation_time_chunk_sizes_end_to_end(S):
    """One set of layer inputs run at the evaluation-time chunk sizes of the
    paper (S = 32 on the generic kernels, S = 64 on the tuned ones), each
    against the oracle forward at that S: the chunk size is a runtime
    argument of the same library."""
    import torch
    w = synth.Workload("eval_S%d" % S, 2, 2048, 8, 64, 128, S, "bf16")
    announce("evaluation-time chunk size %s" % (w,))
    d = synth.forward_inputs(w, seed=29)
    y_ssd, mem, _ = run_scan(w, d)
    q, e, Cm, z = (to_dev(d[k], w.dtype) for k in ("q", "e", "Cm", "z"))
    y, lse = dart.sma_fwd(q, e, Cm, mem, z, y_ssd, S)
    torch.cuda.synchronize()
    ref = oracle.forward(d["x"][:, :, :2], d["dt"][:, :, :2], d["A"][:2], d["Bm"], d["Cm"],
                         d["q"], d["e"], d["z"][:, :, :2], S)
    assert_close_slices(to_np(y)[:, :, :2], ref["y"], TOL["bf16"], what="y (heads 0-1)")
    assert_lse_close(to_np(lse)[:, :, :2], ref["lse"], "bf16", what="lse (heads 0-1)")
