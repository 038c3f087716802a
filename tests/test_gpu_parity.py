"""GPU parity: the HIP path through the C ABI against the fp64 CPU oracle on
the same seeded inputs.  Tolerance (per (b, h) slice, max|gpu - ref| / max|ref|):
1e-4 for fp32 storage, 2e-2 for bf16 storage with fp32 accumulation.  The SMA
readout R is checked on its own: every SMA case runs a second time with
y_ssd = 0 and one constant gate z = 2, so y = SiLU(2) R and the per-slice
metric sees R alone.  LSE: every finite entry within the per-entry bound of
tests.helpers (|d| <= 1e-4 (1 + |ref|) in fp32, |d| <= 0.1 in bf16) and -inf
exactly where the reference has no history."""
import math

import numpy as np
import pytest

import oracle
from paper_2608_02032_amd import dart, synth
from tests.helpers import (TOL, assert_close_slices, assert_lse_close, f32_dev, to_dev, to_np)

pytestmark = pytest.mark.gpu


def announce(msg):
    print("\n[gpu-case] " + msg, flush=True)


def run_scan(w, d, h0=None, mem_capacity=0):
    import torch
    x, Bm, Cm = (to_dev(d[k], w.dtype) for k in ("x", "Bm", "Cm"))
    dt, A = f32_dev(d["dt"]), f32_dev(d["A"])
    h0_t = None if h0 is None else f32_dev(h0)
    y, mem, hl = dart.ssd_chunk_scan(x, dt, A, Bm, Cm, w.chunk, h0=h0_t, mem_capacity=mem_capacity)
    torch.cuda.synchronize()
    return y, mem, hl


SCAN_CASES = [
    synth.WORKLOADS["tiny_fp32_L512"],
    synth.Workload("ragged_fp32_L200_N64", 2, 200, 3, 64, 64, 64, "fp32"),
    synth.Workload("groups_fp32_L384_N128_S128", 1, 384, 4, 64, 128, 128, "fp32", ngroups=2),
    synth.Workload("bf16_L1024_N128_S256", 2, 1024, 4, 64, 128, 256, "bf16"),
    synth.Workload("bf16_L600_N64_S128", 1, 600, 3, 64, 64, 128, "bf16"),
    synth.Workload("bf16_L320_N32_S64", 2, 320, 2, 64, 32, 64, "bf16"),
    # several heads per output workgroup (two-buffer head loop), full and ragged
    synth.Workload("bf16_L4096_H32_N128_S256", 1, 4096, 32, 64, 128, 256, "bf16"),
    synth.Workload("bf16_L4000_H32_N128_S256", 1, 4000, 32, 64, 128, 256, "bf16"),
    synth.Workload("bf16_L600_H8_G2_N128_S128", 1, 600, 8, 64, 128, 128, "bf16", ngroups=2),
]


@pytest.mark.parametrize("w", SCAN_CASES, ids=lambda w: w.name)
def test_scan_matches_recurrence_and_memories(w):
    announce("scan %s" % (w,))
    d = synth.forward_inputs(w, seed=1)
    y, mem, hl = run_scan(w, d)
    y_ref, hl_ref = oracle.ssd_recurrence(d["x"], d["dt"], d["A"], d["Bm"], d["Cm"])
    mem_ref = oracle.chunk_memories(d["x"], d["dt"], d["A"], d["Bm"], w.chunk)
    tol = TOL[w.dtype]
    assert_close_slices(to_np(y), y_ref, tol, what="y_ssd")
    assert_close_slices(to_np(mem), mem_ref, tol, axes_keep=(0, 1, 2), what="mem")
    assert_close_slices(to_np(hl), hl_ref, tol, axes_keep=(0, 1), what="h_last")


def test_scan_initial_state_and_capacity():
    w = synth.Workload("h0_fp32_L300_N64", 1, 300, 2, 64, 64, 128, "fp32")
    announce("scan with h0 %s" % (w,))
    d = synth.forward_inputs(w, seed=2)
    h0 = np.random.default_rng(5).standard_normal((1, 2, 64, 64)).astype(np.float32) * 0.1
    y, mem, hl = run_scan(w, d, h0=h0, mem_capacity=7)
    assert mem.shape[1] == 7
    y_ref, hl_ref = oracle.ssd_recurrence(d["x"], d["dt"], d["A"], d["Bm"], d["Cm"], h0=h0)
    assert_close_slices(to_np(y), y_ref, 1e-4, what="y_ssd")
    assert_close_slices(to_np(hl), hl_ref, 1e-4, axes_keep=(0, 1), what="h_last")
    mem_ref = oracle.chunk_memories(d["x"], d["dt"], d["A"], d["Bm"], 128)
    assert_close_slices(to_np(mem)[:, :3], mem_ref, 1e-4, axes_keep=(0, 1, 2), what="mem")


def test_scan_single_chunk_memory_is_final_state():
    # S = L: the only memory equals the final state (h0 = 0)
    w = synth.Workload("one_chunk_bf16", 2, 256, 2, 64, 128, 256, "bf16")
    announce("scan one chunk %s" % (w,))
    d = synth.forward_inputs(w, seed=3)
    y, mem, hl = run_scan(w, d)
    assert_close_slices(to_np(mem)[:, 0], to_np(hl), 2e-2, axes_keep=(0, 1), what="mem vs h_last")


def sma_case(w, seed, nmem_extra=0):
    d = synth.forward_inputs(w, seed=seed)
    rng = np.random.default_rng(seed + 100)
    mem = synth.synthetic_memories(rng, w.batch, w.nchunks + nmem_extra, w.nheads, w.dstate,
                                   w.headdim, w.dtype)
    y_ssd = synth.to_storage(rng.standard_normal((w.batch, w.seqlen, w.nheads, w.headdim))
                             .astype(np.float32) * 0.05, w.dtype)
    return d, mem, y_ssd


def run_sma(w, d, mem, y_ssd, z=None, inplace=False, **kw):
    import torch
    q, e, Cm = (to_dev(d[k], w.dtype) for k in ("q", "e", "Cm"))
    zz = to_dev(d["z"] if z is None else z, w.dtype)
    mem_t = to_dev(mem, w.dtype)
    ys = to_dev(y_ssd, w.dtype)
    out = ys if inplace else None
    y, lse = dart.sma_fwd(q, e, Cm, mem_t, zz, ys, w.chunk, y=out, **kw)
    torch.cuda.synchronize()
    return y, lse


SMA_CASES = [
    synth.WORKLOADS["tiny_fp32_L512"],
    synth.Workload("fp32_L700_N64_S128", 1, 700, 2, 64, 64, 128, "fp32"),
    synth.Workload("fp32_L512_N128_S256", 1, 768, 2, 64, 128, 256, "fp32"),
    synth.Workload("bf16_L1280_N128_S256", 2, 1280, 3, 64, 128, 256, "bf16"),
    synth.Workload("bf16_L700_N64_S64", 1, 700, 2, 64, 64, 64, "bf16"),
    synth.Workload("bf16_L1024_N128_S128", 1, 1024, 2, 64, 128, 128, "bf16"),
    synth.Workload("bf16_L1100_N32_S64_G2", 1, 1100, 4, 64, 32, 64, "bf16", ngroups=2),
    # many memories per head, two blocks of four heads per token block
    synth.Workload("bf16_L4096_N128_S256_H8", 1, 4096, 8, 64, 128, 256, "bf16"),
    synth.Workload("bf16_L2304_N64_S64_H4", 1, 2304, 4, 64, 64, 64, "bf16"),
]


@pytest.mark.parametrize("w", SMA_CASES, ids=lambda w: w.name)
def test_sma_matches_explicit_softmax(w):
    announce("sma %s" % (w,))
    d, mem, y_ssd = sma_case(w, seed=7)
    y, lse = run_sma(w, d, mem, y_ssd)
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, w.chunk)
    tol = TOL[w.dtype]
    assert_close_slices(to_np(y), y_ref, tol, what="y")
    assert_lse_close(to_np(lse), lse_ref, w.dtype)
    # first chunk: y == y_ssd bitwise, LSE = -inf
    S = w.chunk
    np.testing.assert_array_equal(to_np(y)[:, :S], y_ssd[:, :S].astype(np.float64))
    check_readout(w, d, mem)


# The small shapes above run with one head per workgroup (the chooser's pick
# for them); these force 2, 4 and 8 heads per workgroup, so the head changes
# inside a workgroup's memory stream and the per-head epilogues are checked
# element by element as well.
FORCED_HPB = [("bf16_L4096_N128_S256_H8", 8), ("bf16_L4096_N128_S256_H8", 4),
              ("bf16_L2304_N64_S64_H4", 4), ("bf16_L2304_N64_S64_H4", 2),
              ("bf16_L1100_N32_S64_G2", 2), ("bf16_L1024_N128_S128", 2), ("fp32_L700_N64_S128", 2)]


@pytest.mark.parametrize("name,hpb", FORCED_HPB, ids=lambda v: str(v))
def test_sma_forced_heads_per_block(name, hpb, monkeypatch):
    w = {c.name: c for c in SMA_CASES}[name]
    announce("sma %s, %d heads per block" % (w, hpb))
    monkeypatch.setenv("DART_SMA_HEADS_PER_BLOCK", str(hpb))
    d, mem, y_ssd = sma_case(w, seed=7)
    y, lse = run_sma(w, d, mem, y_ssd)
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, w.chunk)
    assert_close_slices(to_np(y), y_ref, TOL[w.dtype], what="y")
    assert_lse_close(to_np(lse), lse_ref, w.dtype)
    # the head split changes no arithmetic: bitwise equal to the chosen split
    monkeypatch.delenv("DART_SMA_HEADS_PER_BLOCK")
    y0, lse0 = run_sma(w, d, mem, y_ssd)
    np.testing.assert_array_equal(to_np(y), to_np(y0))
    np.testing.assert_array_equal(to_np(lse), to_np(lse0))


def readout_inputs(w, d):
    """y_ssd = 0 and one gate z = 2 for every token and head: y = SiLU(2) R."""
    z2 = np.full_like(d["z"], 2.0)
    return np.zeros((w.batch, w.seqlen, w.nheads, w.headdim), dtype=np.float32), z2


def check_readout(w, d, mem, **kw):
    """The SMA readout R alone, per (b, h) slice (tokens of the first chunk,
    R = 0, are exact zeros on both sides)."""
    ys0, z2 = readout_inputs(w, d)
    y, _ = run_sma(w, d, mem, ys0, z=z2, **kw)
    okw = {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in kw.items()}
    y_ref, _ = oracle.sma(d["q"], d["e"], d["Cm"], mem, z2, ys0, w.chunk, **okw)
    got = to_np(y)
    assert np.all(got[:, :w.chunk] == 0.0)
    assert_close_slices(got, y_ref, TOL[w.dtype], what="R (y_ssd = 0, z = 2)")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_sma_options(dtype):
    """Alg. 1 literal (normalize = 0), one gate per token, RMSNorm weights, in place."""
    import torch
    w = synth.Workload("opts_%s" % dtype, 1, 640, 2, 64, 64, 64, dtype, z_per_head=False)
    announce("sma options %s" % (w,))
    d, mem, y_ssd = sma_case(w, seed=11)
    tol = TOL[dtype]
    # unnormalised
    y, lse = run_sma(w, d, mem, y_ssd, normalize=False)
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, 64, normalize=False)
    assert_close_slices(to_np(y), y_ref, tol, what="y (normalize=0)")
    assert_lse_close(to_np(lse), lse_ref, dtype)
    check_readout(w, d, mem, normalize=False)
    # norm weights + in place
    rng = np.random.default_rng(3)
    qw = rng.uniform(0.5, 1.5, 64).astype(np.float32)
    ew = rng.uniform(0.5, 1.5, 64).astype(np.float32)
    y, lse = run_sma(w, d, mem, y_ssd, inplace=True, q_norm_w=f32_dev(qw), e_norm_w=f32_dev(ew))
    y_ref, lse_ref = oracle.sma(d["q"], d["e"], d["Cm"], mem, d["z"], y_ssd, 64, q_norm_w=qw,
                                e_norm_w=ew)
    assert_close_slices(to_np(y), y_ref, tol, what="y (weights, in place)")
    assert_lse_close(to_np(lse), lse_ref, dtype)
    check_readout(w, d, mem, q_norm_w=f32_dev(qw), e_norm_w=f32_dev(ew))


def test_sma_gate_zero_returns_ssm_output():
    w = synth.Workload("gate0_bf16", 1, 768, 2, 64, 128, 256, "bf16")
    announce("sma gate zero %s" % (w,))
    d, mem, y_ssd = sma_case(w, seed=12)
    y, _ = run_sma(w, d, mem, y_ssd, z=np.zeros_like(d["z"]))
    np.testing.assert_array_equal(to_np(y), y_ssd.astype(np.float64))


@pytest.mark.parametrize("w", [synth.WORKLOADS["tiny_fp32_L512"],
                               synth.Workload("e2e_bf16", 2, 1024, 4, 64, 128, 256, "bf16")],
                         ids=lambda w: w.name)
def test_forward_end_to_end(w):
    """GPU scan -> GPU SMA + gate, against the oracle run from scratch."""
    import torch
    announce("forward %s" % (w,))
    d = synth.forward_inputs(w, seed=0)
    y_ssd, mem, _ = run_scan(w, d)
    q, e, Cm, z = (to_dev(d[k], w.dtype) for k in ("q", "e", "Cm", "z"))
    y, lse = dart.sma_fwd(q, e, Cm, mem, z, y_ssd, w.chunk)
    torch.cuda.synchronize()
    ref = oracle.forward(d["x"], d["dt"], d["A"], d["Bm"], d["Cm"], d["q"], d["e"], d["z"],
                         w.chunk)
    tol = TOL[w.dtype]
    assert_close_slices(to_np(y), ref["y"], tol, what="y")
    assert_lse_close(to_np(lse), ref["lse"], w.dtype)


def test_scan_and_sma_are_deterministic():
    import torch
    w = synth.Workload("det_bf16", 2, 1024, 4, 64, 128, 256, "bf16")
    announce("determinism %s" % (w,))
    d = synth.forward_inputs(w, seed=4)
    outs = []
    for _ in range(2):
        y_ssd, mem, hl = run_scan(w, d)
        q, e, Cm, z = (to_dev(d[k], w.dtype) for k in ("q", "e", "Cm", "z"))
        y, lse = dart.sma_fwd(q, e, Cm, mem, z, y_ssd, w.chunk)
        torch.cuda.synchronize()
        outs.append([t.cpu() for t in (y_ssd, mem, hl, y, lse)])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_full_size_forward_sampled():
    """The benchmark workload (batch 4, L 8192, 32 heads, N 128, S 256, bf16) in
    the launch configuration the benchmark times: the scan outputs of sampled
    (b, h) slices against the oracle run on those slices, and SMA rows sampled
    across the sequence against the SMA definition on the GPU's own memories."""
    import torch
    w = synth.WORKLOADS["sweep_L8192_S256_N128"]
    announce("full size sampled %s" % (w,))
    d = synth.forward_inputs(w, seed=21)
    y_ssd, mem, hl = run_scan(w, d)
    q, e, Cm, z = (to_dev(d[k], w.dtype) for k in ("q", "e", "Cm", "z"))
    y, lse = dart.sma_fwd(q, e, Cm, mem, z, y_ssd, w.chunk)
    ys0, z2 = readout_inputs(w, d)
    yR, _ = dart.sma_fwd(q, e, Cm, mem, to_dev(z2, w.dtype), to_dev(ys0, w.dtype), w.chunk)
    torch.cuda.synchronize()
    tol = TOL[w.dtype]
    S, L = w.chunk, w.seqlen
    rng = np.random.default_rng(22)
    for b, h in [(0, 0), (1, 13), (3, 31)]:
        xs = d["x"][b:b + 1, :, h:h + 1]
        dts = d["dt"][b:b + 1, :, h:h + 1]
        As = d["A"][h:h + 1]
        Bs, Cs = d["Bm"][b:b + 1], d["Cm"][b:b + 1]
        y_ref, hl_ref = oracle.ssd_recurrence(xs, dts, As, Bs, Cs)
        mem_ref = oracle.chunk_memories(xs, dts, As, Bs, S)
        what = "(b=%d, h=%d)" % (b, h)
        assert_close_slices(to_np(y_ssd[b:b + 1, :, h:h + 1]), y_ref, tol, what="y_ssd " + what)
        assert_close_slices(to_np(mem[b:b + 1, :, h:h + 1]), mem_ref, tol, axes_keep=(0, 1, 2),
                            what="mem " + what)
        assert_close_slices(to_np(hl[b:b + 1, h:h + 1]), hl_ref, tol, axes_keep=(0, 1),
                            what="h_last " + what)
        # SMA rows: first and last token of some chunks and random tokens
        ts = np.unique(np.concatenate([[0, S - 1, S, 2 * S - 1, L - S, L - 1],
                                       rng.integers(0, L, 10)]))
        rows = np.stack([np.zeros_like(ts), ts, np.zeros_like(ts)], axis=1)
        yr, lr = oracle.sma_rows(d["q"][b:b + 1], d["e"][b:b + 1], d["Cm"][b:b + 1],
                                 to_np(mem[b:b + 1, :, h:h + 1]), d["z"][b:b + 1, :, h:h + 1],
                                 to_np(y_ssd[b:b + 1, :, h:h + 1]), S, rows)
        ti = torch.as_tensor(ts, device=y.device)
        got_y = to_np(y[b, :, h][ti])
        got_l = to_np(lse[b, :, h][ti])
        assert_close_slices(got_y[None], yr[None], tol, axes_keep=(0,), what="y rows " + what)
        assert_lse_close(got_l[None], lr[None], w.dtype, what="lse rows " + what)
        # the readout alone on the same rows (y_ssd = 0, z = 2)
        rr, _ = oracle.sma_rows(d["q"][b:b + 1], d["e"][b:b + 1], d["Cm"][b:b + 1],
                                to_np(mem[b:b + 1, :, h:h + 1]), z2[b:b + 1, :, h:h + 1],
                                ys0[b:b + 1, :, h:h + 1], S, rows)
        assert_close_slices(to_np(yR[b, :, h][ti])[None], rr[None], tol, axes_keep=(0,),
                            what="R rows " + what)


# --------------------------------------------------------------------------- #
# decode
# --------------------------------------------------------------------------- #

@pytest.mark.parametrize("dtype,S,N,L,z_per_head", [("fp32", 64, 32, 200, True),
                                                    ("bf16", 64, 64, 160, False)])
def test_decode_token_by_token_reproduces_forward(dtype, S, N, L, z_per_head):
    import torch
    w = synth.Workload("dec_%s" % dtype, 2, L, 2, 64, N, S, dtype, z_per_head=z_per_head)
    announce("decode token-by-token %s" % (w,))
    d = synth.forward_inputs(w, seed=21)
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
        zt = dev["z"][:, t].contiguous()
        y = dart.decode_step(t, dev["x"][:, t].contiguous(), dt[:, t].contiguous(), A,
                             dev["Bm"][:, t].contiguous(), dev["Cm"][:, t].contiguous(),
                             dev["q"][:, t].contiguous(), dev["e"][:, t].contiguous(), zt,
                             h_state, chunk_acc, cache, S)
        ys.append(y)
    torch.cuda.synchronize()
    y_all = np.stack([to_np(y) for y in ys], axis=1)
    tol = TOL[dtype]
    assert_close_slices(y_all, ref["y"], tol, what="decode y")
    full = L // S
    assert_close_slices(to_np(cache)[:, :full], ref["mem"][:, :full], tol, axes_keep=(0, 1, 2),
                        what="cache")
    assert_close_slices(to_np(h_state), ref["h_last"], tol, axes_keep=(0, 1), what="h_state")


@pytest.mark.parametrize("dtype,S,N,z_per_head", [("fp32", 64, 32, True), ("bf16", 64, 64, False)])
def test_decode_state_snapshot_and_restore(dtype, S, N, z_per_head):
    """The decode state (h_state, chunk_acc, the memory cache) copied to host
    memory and back continues exactly as the original: a step sequence that
    crosses a chunk boundary after the snapshot gives bitwise identical outputs
    and final state from the restored copy as from the live one."""
    import torch
    L0, L1 = 100, 60  # snapshot after 100 tokens; the next 60 cross token 128
    w = synth.Workload("snap_%s" % dtype, 2, L0 + L1, 2, 64, N, S, dtype, z_per_head=z_per_head)
    announce("decode snapshot/restore %s" % (w,))
    d = synth.forward_inputs(w, seed=33)
    B_, H, P = w.batch, w.nheads, w.headdim
    Mcap = -(-(L0 + L1) // S)
    dev = {k: to_dev(d[k], dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    dt, A = f32_dev(d["dt"]), f32_dev(d["A"])

    def step(t, hs, ca, cache):
        return dart.decode_step(t, dev["x"][:, t].contiguous(), dt[:, t].contiguous(), A,
                                dev["Bm"][:, t].contiguous(), dev["Cm"][:, t].contiguous(),
                                dev["q"][:, t].contiguous(), dev["e"][:, t].contiguous(),
                                dev["z"][:, t].contiguous(), hs, ca, cache, S)

    h_state = torch.zeros((B_, H, N, P), dtype=torch.float32, device="cuda")
    chunk_acc = torch.zeros_like(h_state)
    cache = torch.zeros((B_, Mcap, H, N, P), dtype=dev["x"].dtype, device="cuda")
    for t in range(L0):
        step(t, h_state, chunk_acc, cache)
    torch.cuda.synchronize()
    snap = [a.cpu() for a in (h_state, chunk_acc, cache)]

    live = [step(t, h_state, chunk_acc, cache).cpu() for t in range(L0, L0 + L1)]
    live_state = [a.cpu() for a in (h_state, chunk_acc, cache)]

    # restore into fresh device buffers that first hold other values
    hs2, ca2, cache2 = (torch.full_like(a, 7.0, device="cuda") for a in snap)
    for dst, src in zip((hs2, ca2, cache2), snap):
        dst.copy_(src.to("cuda"))
    again = [step(t, hs2, ca2, cache2).cpu() for t in range(L0, L0 + L1)]
    torch.cuda.synchronize()
    for t, (a, b) in enumerate(zip(live, again)):
        assert torch.equal(a, b), "y differs at step %d after the restore" % (L0 + t)
    for nm, a, b in zip(("h_state", "chunk_acc", "cache"), live_state, (hs2, ca2, cache2)):
        assert torch.equal(a, b.cpu()), nm + " differs after the restored steps"


@pytest.mark.parametrize("dtype,S,N,lengths,steps", [("fp32", 64, 64, (70, 128, 5), 70),
                                                      ("bf16", 128, 128, (300, 256, 129, 0), 140)])
def test_ragged_prefill_handoff_and_decode(dtype, S, N, lengths, steps):
    """Rows of different prompt lengths: one scan over the batch padded with
    dt = 0, the handoff, then decode steps at each row's own position; every
    row's outputs against the oracle forward over that row's own sequence."""
    import torch
    B_ = len(lengths)
    T = max(lengths) + steps
    w = synth.Workload("ragged_%s" % dtype, B_, T, 2, 64, N, S, dtype)
    announce("ragged prefill/handoff/decode %s lengths %s" % (w, lengths))
    d = synth.forward_inputs(w, seed=31)
    H, P = w.nheads, w.headdim
    Lp = max(lengths)
    Mcap = -(-T // S) + 1
    dt_pad = d["dt"][:, :Lp].copy()
    for b, lb in enumerate(lengths):
        dt_pad[b, lb:] = 0.0
    dev = {k: to_dev(d[k], dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    dt_all, A = f32_dev(d["dt"]), f32_dev(d["A"])
    h_last = None
    if Lp > 0:
        _, mem, h_last = dart.ssd_chunk_scan(dev["x"][:, :Lp].contiguous(), f32_dev(dt_pad), A,
                                             dev["Bm"][:, :Lp].contiguous(),
                                             dev["Cm"][:, :Lp].contiguous(), S, mem_capacity=Mcap)
    lens = torch.tensor(lengths, dtype=torch.int64, device="cuda")
    h_state, chunk_acc = dart.decode_handoff(lens, mem, h_last, S)
    rows = torch.arange(B_, device="cuda")
    ys = []
    for k in range(steps):
        pos = lens + k
        take = lambda t: t[rows, pos].contiguous()
        y = dart.decode_step_ragged(pos, max(lengths) + k, take(dev["x"]), take(dt_all), A,
                                    take(dev["Bm"]), take(dev["Cm"]), take(dev["q"]), take(dev["e"]),
                                    take(dev["z"]), h_state, chunk_acc, mem, S)
        ys.append(to_np(y))
    torch.cuda.synchronize()
    tol = TOL[dtype]
    for b, lb in enumerate(lengths):
        tb = lb + steps
        sl = lambda a: a[b:b + 1, :tb]
        ref = oracle.forward(sl(d["x"]), sl(d["dt"]), d["A"], sl(d["Bm"]), sl(d["Cm"]), sl(d["q"]),
                             sl(d["e"]), sl(d["z"]), S)
        got = np.stack([ys[k][b] for k in range(steps)], axis=0)[None]
        assert_close_slices(got, ref["y"][:, lb:tb], tol, what="decode y row %d (L=%d)" % (b, lb))
        assert_close_slices(to_np(h_state[b:b + 1]), ref["h_last"], tol, axes_keep=(0, 1),
                            what="h_state row %d" % b)
        full = tb // S
        assert_close_slices(to_np(mem[b:b + 1, :full]), ref["mem"][:, :full], tol, axes_keep=(0, 1, 2),
                            what="cache row %d" % b)


@pytest.mark.parametrize("dtype,N,S,m,offset", [("bf16", 128, 256, 40, 17), ("bf16", 128, 256, 19, 255),
                                                ("fp32", 64, 64, 33, 0), ("bf16", 32, 128, 1, 5)])
def test_decode_single_step_on_synthetic_cache(dtype, N, S, m, offset):
    import torch
    B_, H, P = 3, 4, 64
    pos = m * S + offset
    Mcap = m + 2
    announce("decode step dtype=%s N=%d S=%d pos=%d" % (dtype, N, S, pos))
    rng = np.random.default_rng(m)
    mem = np.zeros((B_, Mcap, H, N, P), dtype=np.float32)
    mem[:, :m] = synth.synthetic_memories(rng, B_, m, H, N, P, dtype)
    h_state = (rng.standard_normal((B_, H, N, P)) * 0.01).astype(np.float32)
    chunk_acc = (rng.standard_normal((B_, H, N, P)) * 0.01).astype(np.float32)
    inp = synth.decode_inputs(B_, H, P, N, dtype, seed=m + 1)
    hs_ref, ca_ref, mem_ref = (np.array(a, dtype=np.float64) for a in (h_state, chunk_acc, mem))
    y_ref = oracle.decode_step(pos, inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], inp["q"],
                               inp["e"], inp["z"], hs_ref, ca_ref, mem_ref, S)
    hs, ca = f32_dev(h_state), f32_dev(chunk_acc)
    cache = to_dev(mem, dtype)
    dev = {k: to_dev(inp[k], dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    y = dart.decode_step(pos, dev["x"], f32_dev(inp["dt"]), f32_dev(inp["A"]), dev["Bm"], dev["Cm"],
                         dev["q"], dev["e"], dev["z"], hs, ca, cache, S)
    torch.cuda.synchronize()
    tol = TOL[dtype]
    assert_close_slices(to_np(y), y_ref, tol, axes_keep=(0, 1), what="y")
    assert_close_slices(to_np(hs), hs_ref, 1e-5, axes_keep=(0, 1), what="h_state")
    assert_close_slices(to_np(ca), ca_ref, 1e-5, axes_keep=(0, 1), what="chunk_acc")
    assert_close_slices(to_np(cache), mem_ref, tol, axes_keep=(0, 1, 2), what="cache")
