"""GPU parity at the full sizes of the benchmark configurations, in the launch
configuration bench.py uses, on sampled outputs the oracle computes one by
one: scan outputs of sampled (b, h) slices against the oracle run on those
slices, SMA rows sampled across the sequence against the SMA definition on the
GPU's own memories, and decode rows of the full batch against the oracle's
decode step on those rows (rows are independent).  Metric and tolerances as in
test_gpu_parity.py."""
import numpy as np
import pytest

import oracle
from paper_2608_02032_amd import dart, synth
from tests.helpers import TOL, assert_close_slices, assert_lse_close, f32_dev, to_dev, to_np
from tests.test_gpu_parity import readout_inputs

pytestmark = pytest.mark.gpu


def announce(msg):
    print("\n[gpu-case] " + msg, flush=True)


FORWARD_FULL = [
    # the Mamba-2-130M-shaped layer (B 8, L 4096, 24 heads)
    ("mamba2_130m_L4096", [(0, 0), (5, 11), (7, 23)]),
    # the rest of the chunk/state sweep at L 8192 (S 256, N 128 is in test_gpu_parity.py)
    ("sweep_L8192_S64_N64", [(0, 3), (3, 30)]),
    ("sweep_L8192_S64_N128", [(1, 0), (2, 17)]),
    ("sweep_L8192_S128_N64", [(0, 31), (3, 8)]),
    ("sweep_L8192_S128_N128", [(2, 2), (3, 29)]),
    ("sweep_L8192_S256_N64", [(0, 16), (1, 31)]),
    # the long-context forward (L 65536, 256 memories per head)
    ("long_L65536", [(0, 0), (0, 27)]),
]


@pytest.mark.parametrize("name,slices", FORWARD_FULL, ids=[f[0] for f in FORWARD_FULL])
def test_forward_full_size_sampled(name, slices):
    import torch
    w = synth.WORKLOADS[name]
    announce("forward full size %s" % (w,))
    d = synth.forward_inputs(w, seed=31)
    x, Bm, Cm, q, e, z = (to_dev(d[k], w.dtype) for k in ("x", "Bm", "Cm", "q", "e", "z"))
    y_ssd, mem, hl = dart.ssd_chunk_scan(x, f32_dev(d["dt"]), f32_dev(d["A"]), Bm, Cm, w.chunk)
    y, lse = dart.sma_fwd(q, e, Cm, mem, z, y_ssd, w.chunk)
    # the readout alone: y_ssd = 0 and one gate z = 2 (y = SiLU(2) R)
    ys0, z2 = readout_inputs(w, d)
    yR, _ = dart.sma_fwd(q, e, Cm, mem, to_dev(z2, w.dtype), to_dev(ys0, w.dtype), w.chunk)
    torch.cuda.synchronize()
    tol = TOL[w.dtype]
    S, L = w.chunk, w.seqlen
    rng = np.random.default_rng(32)
    for b, h in slices:
        what = "(b=%d, h=%d)" % (b, h)
        xs = d["x"][b:b + 1, :, h:h + 1]
        dts = d["dt"][b:b + 1, :, h:h + 1]
        As = d["A"][h:h + 1]
        Bs, Cs = d["Bm"][b:b + 1], d["Cm"][b:b + 1]
        y_ref, hl_ref = oracle.ssd_recurrence(xs, dts, As, Bs, Cs)
        mem_ref = oracle.chunk_memories(xs, dts, As, Bs, S)
        assert_close_slices(to_np(y_ssd[b:b + 1, :, h:h + 1]), y_ref, tol, what="y_ssd " + what)
        assert_close_slices(to_np(mem[b:b + 1, :, h:h + 1]), mem_ref, tol, axes_keep=(0, 1, 2),
                            what="mem " + what)
        assert_close_slices(to_np(hl[b:b + 1, h:h + 1]), hl_ref, tol, axes_keep=(0, 1),
                            what="h_last " + what)
        ts = np.unique(np.concatenate([[0, S - 1, S, 2 * S - 1, L - S, L - 1],
                                       rng.integers(0, L, 10)]))
        rows = np.stack([np.zeros_like(ts), ts, np.zeros_like(ts)], axis=1)
        yr, lr = oracle.sma_rows(d["q"][b:b + 1], d["e"][b:b + 1], d["Cm"][b:b + 1],
                                 to_np(mem[b:b + 1, :, h:h + 1]), d["z"][b:b + 1, :, h:h + 1],
                                 to_np(y_ssd[b:b + 1, :, h:h + 1]), S, rows)
        ti = torch.as_tensor(ts, device=y.device)
        assert_close_slices(to_np(y[b, :, h][ti])[None], yr[None], tol, axes_keep=(0,),
                            what="y rows " + what)
        assert_lse_close(to_np(lse[b, :, h][ti])[None], lr[None], w.dtype, what="lse rows " + what)
        rr, _ = oracle.sma_rows(d["q"][b:b + 1], d["e"][b:b + 1], d["Cm"][b:b + 1],
                                to_np(mem[b:b + 1, :, h:h + 1]), z2[b:b + 1, :, h:h + 1],
                                ys0[b:b + 1, :, h:h + 1], S, rows)
        assert_close_slices(to_np(yR[b, :, h][ti])[None], rr[None], tol, axes_keep=(0,),
                            what="R rows " + what)
    del x, Bm, Cm, q, e, z, y_ssd, mem, hl, y, lse, yR
    torch.cuda.empty_cache()


@pytest.mark.parametrize("offset", [0, 255], ids=["pos65536", "pos65791_append"])
def test_decode_full_size_sampled(offset):
    """The decode workload (batch 64, 32 heads, N 128, S 256, 65536 cached
    tokens = 256 memories, bf16 cache): one step for the whole batch at
    position 65536 (first token of chunk 256) or 65791 (last token: appends
    memory 256), checked on sampled rows."""
    import torch
    dw = synth.DECODE_WORKLOADS["decode_B64_ctx65536"]
    B_, H, P, N, S = dw.batch, dw.nheads, dw.headdim, dw.dstate, dw.chunk
    m = dw.context // S
    pos = dw.context + offset
    announce("decode full size %s pos=%d" % (dw.name, pos))
    cache, _ = synth.torch_device_memories(B_, m + 1, m, H, N, P, seed=41)
    g = torch.Generator(device="cuda")
    g.manual_seed(42)
    h_state = torch.randn((B_, H, N, P), generator=g, device="cuda") * 1e-2
    chunk_acc = torch.randn((B_, H, N, P), generator=g, device="cuda") * 1e-2
    inp = synth.decode_inputs(B_, H, P, N, dw.dtype, seed=43)
    rows = [0, 37, 63]
    before = {b: (to_np(cache[b:b + 1]), to_np(h_state[b:b + 1]), to_np(chunk_acc[b:b + 1]))
              for b in rows}
    dev = {k: to_dev(inp[k], dw.dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    y = dart.decode_step(pos, dev["x"], f32_dev(inp["dt"]), f32_dev(inp["A"]), dev["Bm"],
                         dev["Cm"], dev["q"], dev["e"], dev["z"], h_state, chunk_acc, cache, S)
    torch.cuda.synchronize()
    tol = TOL[dw.dtype]
    for b in rows:
        mem_ref, hs_ref, ca_ref = before[b]
        sl = {k: v[b:b + 1] for k, v in inp.items() if k != "A"}
        y_ref = oracle.decode_step(pos, sl["x"], sl["dt"], inp["A"], sl["Bm"], sl["Cm"], sl["q"],
                                   sl["e"], sl["z"], hs_ref, ca_ref, mem_ref, S)
        what = "row %d" % b
        assert_close_slices(to_np(y[b:b + 1]), y_ref, tol, axes_keep=(0, 1), what="y " + what)
        assert_close_slices(to_np(h_state[b:b + 1]), hs_ref, 1e-5, axes_keep=(0, 1),
                            what="h_state " + what)
        assert_close_slices(to_np(chunk_acc[b:b + 1]), ca_ref, 1e-5, axes_keep=(0, 1),
                            what="chunk_acc " + what)
        if offset == S - 1:
            assert_close_slices(to_np(cache[b:b + 1, m:m + 1]), mem_ref[:, m:m + 1], tol,
                                axes_keep=(0, 1, 2), what="appended memory " + what)
        del mem_ref
    del cache, h_state, chunk_acc, y
    torch.cuda.empty_cache()
