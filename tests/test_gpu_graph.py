"""The library under HIP graph capture: the forward (scan, then SMA + gate), the
scan backward, and a ragged decode step (positions on the device, so one
captured graph serves every step) are captured once and replayed several times, with the
program's own eager work and synchronisations between replays (new inputs,
an eager run into separate buffers).  Every replay must equal the eager
result bit for bit (the kernels are deterministic and the library issues no
memsets, allocations or synchronisations of its own)."""
import numpy as np
import pytest

from paper_2608_02032_amd import dart, synth
from tests.helpers import f32_dev, to_dev

pytestmark = pytest.mark.gpu


def announce(msg):
    print("\n[gpu-case] " + msg, flush=True)


def test_forward_replays_in_a_graph():
    import torch
    w = synth.Workload("graph_bf16_L1024_N128_S256", 2, 1024, 4, 64, 128, 256, "bf16")
    announce("graph forward %s" % (w,))
    B, L, H, P, N, S, M = w.batch, w.seqlen, w.nheads, w.headdim, w.dstate, w.chunk, w.nchunks
    bf = torch.bfloat16
    d = synth.forward_inputs(w, seed=61)
    inp = {k: to_dev(d[k], w.dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    inp["dt"], inp["A"] = f32_dev(d["dt"]), f32_dev(d["A"])
    dims = dart.make_dims(B, L, H, P, N, S, w.dtype)
    ws_scan = torch.empty(dart.workspace_bytes("scan", dims), dtype=torch.uint8, device="cuda")
    ws_sma = torch.empty(max(1, dart.workspace_bytes("sma", dims)), dtype=torch.uint8, device="cuda")

    def buffers():
        return {"y_ssd": torch.empty((B, L, H, P), dtype=bf, device="cuda"),
                "mem": torch.empty((B, M, H, N, P), dtype=bf, device="cuda"),
                "hl": torch.empty((B, H, N, P), dtype=torch.float32, device="cuda"),
                "y": torch.empty((B, L, H, P), dtype=bf, device="cuda"),
                "lse": torch.empty((B, L, H), dtype=torch.float32, device="cuda")}

    def fwd(o):
        dart.ssd_chunk_scan(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], S, mem=o["mem"],
                            y_ssd=o["y_ssd"], h_last=o["hl"], workspace=ws_scan)
        dart.sma_fwd(inp["q"], inp["e"], inp["Cm"], o["mem"], inp["z"], o["y_ssd"], S, y=o["y"],
                     lse=o["lse"], workspace=ws_sma)

    out = buffers()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fwd(out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fwd(out)
    for rep in range(3):
        d2 = synth.forward_inputs(w, seed=62 + rep)
        for k in ("x", "Bm", "Cm", "q", "e", "z"):
            inp[k].copy_(to_dev(d2[k], w.dtype))
        inp["dt"].copy_(f32_dev(d2["dt"]))
        inp["A"].copy_(f32_dev(d2["A"]))
        ref = buffers()
        fwd(ref)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in out:
            assert torch.equal(out[k], ref[k]), (rep, k)
        print("  replay %d equals the eager forward" % rep, flush=True)


def test_ragged_decode_step_replays_in_a_graph():
    import torch
    B, H, P, N, S, G = 3, 4, 64, 128, 64, 1
    m_cap = 8
    announce("graph ragged decode B=%d H=%d N=%d S=%d" % (B, H, N, S))
    rng = np.random.default_rng(71)
    mem = synth.synthetic_memories(rng, B, m_cap, H, N, P, "bf16")
    cache = to_dev(mem, "bf16")
    h_state = f32_dev((rng.standard_normal((B, H, N, P)) * 0.01).astype(np.float32))
    chunk_acc = f32_dev((rng.standard_normal((B, H, N, P)) * 0.01).astype(np.float32))
    pos0 = np.array([70, 127, 300], dtype=np.int64)  # the second row appends on its first step
    pos = torch.from_numpy(pos0).to("cuda")
    pos_max = 400
    di = synth.decode_inputs(B, H, P, N, "bf16", seed=72)
    inp = {k: to_dev(di[k], "bf16") for k in ("x", "Bm", "Cm", "q", "e", "z")}
    inp["dt"], inp["A"] = f32_dev(di["dt"]), f32_dev(di["A"])
    ddims = dart.make_dims(B, 0, H, P, N, S, "bf16", G, m_cap)
    ws = torch.empty(dart.workspace_bytes("decode", ddims), dtype=torch.uint8, device="cuda")
    y = torch.empty((B, H, P), dtype=torch.bfloat16, device="cuda")

    def step(hs, ca, cc, yy):
        dart.decode_step_ragged(pos, pos_max, inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"],
                                inp["q"], inp["e"], inp["z"], hs, ca, cc, S, y=yy, workspace=ws)

    # eager twin of the state the graph advances
    hs_e, ca_e, cc_e = h_state.clone(), chunk_acc.clone(), cache.clone()
    y_e = torch.empty_like(y)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        hs_w, ca_w, cc_w = h_state.clone(), chunk_acc.clone(), cache.clone()
        step(hs_w, ca_w, cc_w, torch.empty_like(y))  # warm-up on copies
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(h_state, chunk_acc, cache, y)
    for k in range(4):
        di2 = synth.decode_inputs(B, H, P, N, "bf16", seed=80 + k)
        for name in ("x", "Bm", "Cm", "q", "e", "z"):
            inp[name].copy_(to_dev(di2[name], "bf16"))
        inp["dt"].copy_(f32_dev(di2["dt"]))
        step(hs_e, ca_e, cc_e, y_e)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_e), k
        assert torch.equal(h_state, hs_e) and torch.equal(chunk_acc, ca_e), k
        assert torch.equal(cache, cc_e), k
        pos.add_(1)  # every row moves on one token (device-side, outside the graph)
        print("  replay %d equals the eager step" % k, flush=True)


def test_scan_backward_replays_in_a_graph():
    import torch
    w = synth.Workload("graph_bwd_bf16_L600_N64_S128", 2, 600, 4, 64, 64, 128, "bf16")
    announce("graph scan backward %s" % (w,))
    B, L, H, P, N, S, M = w.batch, w.seqlen, w.nheads, w.headdim, w.dstate, w.chunk, w.nchunks
    d = synth.forward_inputs(w, seed=91)
    inp = {k: to_dev(d[k], w.dtype) for k in ("x", "Bm", "Cm")}
    inp["dt"], inp["A"] = f32_dev(d["dt"]), f32_dev(d["A"])
    rng = np.random.default_rng(92)
    dy = to_dev(synth.to_storage(rng.standard_normal((B, L, H, P)).astype(np.float32), "bf16"), "bf16")
    dmem = f32_dev(rng.standard_normal((B, M, H, N, P)).astype(np.float32))
    dims = dart.make_dims(B, L, H, P, N, S, w.dtype, 1, M)
    ws = torch.empty(dart.workspace_bytes("ssd_bwd", dims), dtype=torch.uint8, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")

    def buffers():
        return {"dx": torch.empty((B, L, H, P), **f32), "ddt": torch.empty((B, L, H), **f32),
                "dA": torch.empty((H,), **f32), "dB": torch.empty((B, L, 1, N), **f32),
                "dC": torch.empty((B, L, 1, N), **f32), "dh0": torch.empty((B, H, N, P), **f32)}

    def bwd(o):
        dart.ssd_bwd(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], S, dy, dmem=dmem, out=o,
                     workspace=ws)

    out = buffers()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        bwd(out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        bwd(out)
    for rep in range(3):
        d2 = synth.forward_inputs(w, seed=93 + rep)
        for k in ("x", "Bm", "Cm"):
            inp[k].copy_(to_dev(d2[k], w.dtype))
        inp["dt"].copy_(f32_dev(d2["dt"]))
        ref = buffers()
        bwd(ref)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in out:
            assert torch.equal(out[k], ref[k]), (rep, k)
        print("  replay %d equals the eager backward" % rep, flush=True)
