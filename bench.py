#!/usr/bin/env python3
"""Benchmark of the DART hot path on one MI355X (gfx950).

One step = the whole hot path over one batch of seeded synthetic inputs that
are already resident in HBM:
  forward   chunked SSD scan (k_chunk_state, k_chunk_gram, k_state_pass, k_chunk_out)
            -> state-memory attention + gated residual (k_sma_prep, k_sma)
            on the L = 8192 workload (batch 4, 32 heads, P = 64, N = 128, S = 256);
  decode    one token (k_decode_partial, k_decode_state_merge) for batch 64, 32 heads,
            N = 128, S = 256 over a 65536-token context (256 cached memories).
`value` is forward tokens/s (batch * L / forward time).  Per-kernel times come
from HIP events the library records around every launch on the launch stream
(dart_profile_*): in the timed steps only around k_sma (the roofline kernel),
then around every launch in a separate pass for the breakdown.

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="sweep_L8192_S256_N128")
    ap.add_argument("--decode-workload", default="decode_B64_ctx65536")
    ap.add_argument("--no-decode", action="store_true", help="time the forward only")
    ap.add_argument("--no-ragged", action="store_true",
                    help="skip the separately timed ragged-batch decode steps")
    ap.add_argument("--no-bwd", action="store_true",
                    help="skip the separately timed backward (SMA and scan) on the same workload")
    ap.add_argument("--no-block", action="store_true",
                    help="skip the separately timed block kernels (conv, dt, gated norm)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-batches", type=int, default=4,
                    help="batches of the workload the CPU oracle is timed on")
    ap.add_argument("--copy-calib-mb", type=int, default=0,
                    help="after the timed steps, run one plain device copy of this many MiB "
                         "(reference kernel for scaling HBM byte counters)")
    ap.add_argument("--extra-out", default=None,
                    help="also write per-kernel detail as JSON to this file")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark line: time the forward (scan and SMA "
                         "separately) on every bf16 forward workload and print one JSON line each")
    ap.add_argument("--sweep-out", default=None,
                    help="with --sweep: also write the results as a markdown table to this file")
    return ap.parse_args()


# --------------------------------------------------------------------------- #
# algorithmic work (what the method must compute or move; see the design notes)
# --------------------------------------------------------------------------- #

def scan_flops(w):
    B, M, G, H, N, P, S = w.batch, w.nchunks, w.ngroups, w.nheads, w.dstate, w.headdim, w.chunk
    return B * M * (G * N * S * (S + 1) + H * (P * S * (S + 1) + 4 * S * N * P + 2 * N * P))


def scan_bytes(w, esize=2):
    B, L, H, G, N, P, M = w.batch, w.seqlen, w.nheads, w.ngroups, w.dstate, w.headdim, w.nchunks
    return (B * L * H * P * esize * 2          # read x, write y_ssd
            + B * L * H * 4                    # read dt
            + 2 * B * L * G * N * esize        # read B, C
            + B * M * H * N * P * esize)       # write the memories


def sma_pairs(w):
    """(token, earlier memory) pairs per (b, h)."""
    L, S = w.seqlen, w.chunk
    return sum(max(0, min(L, (i + 1) * S) - i * S) * i for i in range(w.nchunks))


def sma_flops(w):
    return w.batch * w.nheads * 4 * w.dstate * w.headdim * sma_pairs(w)


def sma_bytes(w, esize=2):
    B, L, H, G, N, P, M = w.batch, w.seqlen, w.nheads, w.ngroups, w.dstate, w.headdim, w.nchunks
    zsz = B * L * H if w.z_per_head else B * L
    return (B * L * G * (2 * N + P) * esize    # read q, C, e
            + B * max(M - 1, 0) * H * N * P * esize  # read the attended memories once
            + zsz * esize                       # read z
            + B * L * H * P * esize * 2         # read y_ssd, write y
            + B * L * H * 4)                    # write lse


def ssd_bwd_bytes(w):
    """Bytes the scan backward must move at the least: x, dy (storage dtype),
    dt, B, C and the memory gradient (float) in; dx, ddt, dB, dC (float) and
    dA out."""
    B, L, H, P, N, G, M = w.batch, w.seqlen, w.nheads, w.headdim, w.dstate, w.ngroups, w.nchunks
    es = 2 if w.dtype == "bf16" else 4
    return (2 * B * L * H * P * es + 4 * B * L * H + 2 * B * L * G * N * es + 4 * B * M * H * N * P
            + 4 * B * L * H * P + 4 * B * L * H + 2 * 4 * B * L * G * N + 4 * H)


def sma_bwd_flops(w):
    """Backward per (token, earlier memory) pair: logits again, dy . V via
    dH dy, dQbar via Kh Ebar (token side) and the two memory-side products."""
    return w.batch * w.nheads * 10 * w.dstate * w.headdim * sma_pairs(w)


def decode_bytes(d, esize=2):
    B, H, N, P, G = d.batch, d.nheads, d.dstate, d.headdim, d.ngroups
    m = d.context // d.chunk
    return (B * H * m * N * P * esize           # stream every cached memory
            + 4 * B * H * N * P * 4             # h_state and chunk_acc read + write
            + B * H * P * esize * 2 + B * G * (3 * N + P) * esize + B * H * 8)


# --------------------------------------------------------------------------- #

def cpu_baseline(w, nbatch):
    """Time the fp64 CPU oracle (as it stands) on `nbatch` batch rows of the
    workload: recurrence + brute-force memories + explicit-softmax SMA + gate."""
    import numpy as np
    import oracle
    from paper_2608_02032_amd import synth
    ws = w.with_(batch=nbatch)
    d = synth.forward_inputs(ws, seed=0)
    f = {k: np.asarray(v, dtype=np.float64) for k, v in d.items()}
    t0 = time.perf_counter()
    oracle.forward(f["x"], f["dt"], f["A"], f["Bm"], f["Cm"], f["q"], f["e"], f["z"], ws.chunk)
    sec = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    threads = min(threads, nbatch * ws.nheads)  # the oracle parallelises over (b, h)
    return {"value": nbatch * ws.seqlen / sec, "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": "%d of %d batch rows of %s (all %d heads, L=%d), fp64, %.1f s wall"
                      % (nbatch, w.batch, w.name, w.nheads, w.seqlen, sec)}


def sweep(args):
    """Scan and SMA time and utilisation on every bf16 forward workload (the
    chunk/state sweep at L = 8192, the Mamba-2-130M-shaped layer and the
    L = 65536 long context)."""
    import torch
    from paper_2608_02032_amd import dart, synth
    dev = torch.device("cuda:0")
    names = [n for n, w in synth.WORKLOADS.items() if w.dtype == "bf16"]
    rows = []
    for name in names:
        w = synth.WORKLOADS[name]
        d = synth.forward_inputs(w, seed=0)
        T = {k: torch.from_numpy(v).to(dev) for k, v in d.items()}
        for k in ("x", "Bm", "Cm", "q", "e", "z"):
            T[k] = T[k].to(torch.bfloat16)
        B, L, H, P, N, S = w.batch, w.seqlen, w.nheads, w.headdim, w.dstate, w.chunk
        y_ssd = torch.empty((B, L, H, P), dtype=torch.bfloat16, device=dev)
        mem = torch.empty((B, w.nchunks, H, N, P), dtype=torch.bfloat16, device=dev)
        h_last = torch.empty((B, H, N, P), dtype=torch.float32, device=dev)
        y = torch.empty_like(y_ssd)
        lse = torch.empty((B, L, H), dtype=torch.float32, device=dev)
        dims = dart.make_dims(B, L, H, P, N, S, w.dtype, w.ngroups)
        ws_scan = torch.empty(dart.workspace_bytes("scan", dims), dtype=torch.uint8, device=dev)
        ws_sma = torch.empty(max(1, dart.workspace_bytes("sma", dims)), dtype=torch.uint8, device=dev)
        stream = torch.cuda.current_stream()

        def forward():
            dart.ssd_chunk_scan(T["x"], T["dt"], T["A"], T["Bm"], T["Cm"], S, mem=mem, y_ssd=y_ssd,
                                h_last=h_last, workspace=ws_scan, stream=stream)
            dart.sma_fwd(T["q"], T["e"], T["Cm"], mem, T["z"], y_ssd, S, y=y, lse=lse,
                         workspace=ws_sma, stream=stream)
        for _ in range(args.warmup):
            forward()
        torch.cuda.synchronize()
        dart.profile_reset()
        dart.profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            forward()
        e1.record(stream)
        torch.cuda.synchronize()
        dart.profile_enable(False)
        kern = dart.profile_read(reset=True)
        avg = {k: v[0] / max(v[1], 1) for k, v in kern.items()}
        fwd_ms = e0.elapsed_time(e1) / args.steps
        scan_ms = sum(avg.get(k, 0.0) for k in ("k_chunk_state", "k_chunk_gram", "k_state_pass",
                                                 "k_chunk_out"))
        sma_ms = sum(avg.get(k, 0.0) for k in ("k_sma_prep", "k_sma_keys", "k_sma"))
        sflops, sbytes, mflops = scan_flops(w), scan_bytes(w), sma_flops(w)
        r = {"workload": name, "batch": B, "seq_len": L, "heads": H, "dstate": N, "chunk": S,
             "fwd_ms": round(fwd_ms, 4), "tokens_per_s": round(B * L / (fwd_ms * 1e-3), 1),
             "scan_us": round(scan_ms * 1e3, 2), "sma_us": round(sma_ms * 1e3, 2),
             "k_sma_us": round(avg.get("k_sma", 0.0) * 1e3, 2),
             "scan_hbm_frac": round(sbytes / (scan_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
             "scan_mfma_util": round(sflops / (scan_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
             "sma_mfma_util": round(mflops / (sma_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
             "k_sma_mfma_util": round(mflops / (avg["k_sma"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
             if avg.get("k_sma") else None}
        rows.append(r)
        print(json.dumps(r), flush=True)
        del T, y_ssd, mem, h_last, y, lse, ws_scan, ws_sma
        torch.cuda.empty_cache()
    if args.sweep_out:
        hdr = ["workload", "fwd_ms", "tokens_per_s", "scan_us", "scan_hbm_frac", "scan_mfma_util",
               "sma_us", "k_sma_us", "sma_mfma_util", "k_sma_mfma_util"]
        lines = ["# Forward sweep (bf16 workloads)", "", "Command:", "", "```",
                 "python3 bench.py --sweep --steps %d --warmup %d --sweep-out <this file>"
                 % (args.steps, args.warmup), "```", "",
                 "Times from the library's HIP events; utilisation against 8 TB/s and "
                 "2.5 PFLOP/s (algorithmic bytes and flops).", "",
                 "| " + " | ".join(hdr) + " |", "|" + "---|" * len(hdr)]
        for r in rows:
            lines.append("| " + " | ".join(str(r[k]) for k in hdr) + " |")
        with open(args.sweep_out, "w") as fh:
            fh.write("\n".join(lines) + "\n")


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(requested --gpus %d, WORLD_SIZE %d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2608_02032_amd import dart, synth
    from paper_2608_02032_amd.profiling import mfma_for, traffic_for

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.sweep:
        sweep(args)
        return
    w = synth.WORKLOADS[args.workload]
    dw = synth.DECODE_WORKLOADS[args.decode_workload]
    bf = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    # ---- resident inputs, outputs and workspaces --------------------------
    d = synth.forward_inputs(w, seed=0)
    T = {k: torch.from_numpy(v).to(dev) for k, v in d.items()}
    for k in ("x", "Bm", "Cm", "q", "e", "z"):
        T[k] = T[k].to(bf)
    B, L, H, P, N, S = w.batch, w.seqlen, w.nheads, w.headdim, w.dstate, w.chunk
    y_ssd = torch.empty((B, L, H, P), dtype=bf, device=dev)
    mem = torch.empty((B, w.nchunks, H, N, P), dtype=bf, device=dev)
    h_last = torch.empty((B, H, N, P), dtype=torch.float32, device=dev)
    y = torch.empty_like(y_ssd)
    lse = torch.empty((B, L, H), dtype=torch.float32, device=dev)
    dims = dart.make_dims(B, L, H, P, N, S, w.dtype, w.ngroups)
    ws_scan = torch.empty(dart.workspace_bytes("scan", dims), dtype=torch.uint8, device=dev)
    ws_sma = torch.empty(max(1, dart.workspace_bytes("sma", dims)), dtype=torch.uint8, device=dev)

    if not args.no_decode:
        m = dw.context // dw.chunk
        cache, _ = synth.torch_device_memories(dw.batch, m + 1, m, dw.nheads, dw.dstate,
                                               dw.headdim, seed=1, device=dev)
        g = torch.Generator(device=dev)
        g.manual_seed(2)
        h_state = torch.randn((dw.batch, dw.nheads, dw.dstate, dw.headdim), generator=g,
                              device=dev) * 1e-2
        chunk_acc = torch.zeros_like(h_state)
        di = synth.decode_inputs(dw.batch, dw.nheads, dw.headdim, dw.dstate, dw.dtype, seed=3)
        D = {k: torch.from_numpy(v).to(dev) for k, v in di.items()}
        for k in ("x", "Bm", "Cm", "q", "e", "z"):
            D[k] = D[k].to(torch.bfloat16)
        y_dec = torch.empty_like(D["x"])
        ddims = dart.make_dims(dw.batch, 0, dw.nheads, dw.headdim, dw.dstate, dw.chunk, dw.dtype,
                               dw.ngroups, m + 1)
        ws_dec = torch.empty(dart.workspace_bytes("decode", ddims), dtype=torch.uint8, device=dev)
        pos = dw.context  # first token after the context: attends all m memories

    stream = torch.cuda.current_stream()

    def forward():
        dart.ssd_chunk_scan(T["x"], T["dt"], T["A"], T["Bm"], T["Cm"], S, mem=mem, y_ssd=y_ssd,
                            h_last=h_last, workspace=ws_scan, stream=stream)
        dart.sma_fwd(T["q"], T["e"], T["Cm"], mem, T["z"], y_ssd, S, y=y, lse=lse,
                     workspace=ws_sma, stream=stream)

    def decode():
        dart.decode_step(pos, D["x"], D["dt"], D["A"], D["Bm"], D["Cm"], D["q"], D["e"], D["z"],
                         h_state, chunk_acc, cache, dw.chunk, y=y_dec, workspace=ws_dec,
                         stream=stream)

    def profiled(fn, reps):
        """Per-kernel times of `reps` further calls, every launch bracketed by
        library events (kept out of the timed calls)."""
        dart.profile_reset()
        dart.profile_enable(True)
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        dart.profile_enable(False)
        return dart.profile_read(reset=True)

    for _ in range(args.warmup):
        forward()
        if not args.no_decode:
            decode()
    torch.cuda.synchronize()

    # ---- timed region --------------------------------------------------------
    # The headline steps run with library events around k_sma only (its
    # average launch time gives the roofline); every other kernel runs back to
    # back with nothing recorded between launches.
    dart.profile_reset()
    dart.profile_filter("k_sma")
    dart.profile_enable(True)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        ev[k][0].record(stream)
        forward()
        ev[k][1].record(stream)
        if not args.no_decode:
            decode()
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    dart.profile_enable(False)
    kmain = dart.profile_read(reset=True)
    fwd_ms = [e[0].elapsed_time(e[1]) for e in ev]
    dec_ms = [e[1].elapsed_time(e[2]) for e in ev]
    step_ms = [e[0].elapsed_time(e[2]) for e in ev]
    fwd_mean = sum(fwd_ms) / len(fwd_ms)
    ms_per_step = sum(step_ms) / len(step_ms)

    # ---- per-kernel breakdown: a separate pass with every launch bracketed --
    nprof = min(args.steps, 20)
    dart.profile_enable(True)
    for _ in range(nprof):
        forward()
        if not args.no_decode:
            decode()
    torch.cuda.synchronize()
    dart.profile_enable(False)
    kernels = dart.profile_read(reset=True)
    avg = {k: v[0] / max(v[1], 1) for k, v in kernels.items()}  # ms per launch

    # ---- rooflines -----------------------------------------------------------
    sflops, sbytes = scan_flops(w), scan_bytes(w)
    mflops, mbytes = sma_flops(w), sma_bytes(w)
    scan_ms = sum(avg.get(k, 0.0) for k in ("k_chunk_state", "k_chunk_gram", "k_state_pass",
                                             "k_chunk_out"))
    sma_ms = sum(avg.get(k, 0.0) for k in ("k_sma_prep", "k_sma_keys", "k_sma"))
    main_ms = kmain["k_sma"][0] / max(kmain["k_sma"][1], 1)
    main_tflops = mflops / (main_ms * 1e-3) / 1e12
    roofline = {"kernel": "k_sma", "bound": "mfma",
                "achieved": round(main_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(main_tflops / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic_for("k_sma"),
                "avg_us": round(main_ms * 1e3, 2),
                "algorithmic_flops_per_launch": mflops,
                "timed": "k_sma launches of the timed steps (library HIP events on its stream)"}
    extra = {
        "mfma_util": {"scan": round(sflops / (scan_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                      "sma": round(mflops / (sma_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)},
        "scan": {"us": round(scan_ms * 1e3, 2), "hbm_gbps": round(sbytes / (scan_ms * 1e-3) / 1e9, 1),
                 "hbm_frac": round(sbytes / (scan_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
                 "algorithmic_bytes": sbytes, "algorithmic_flops": sflops},
        "sma": {"us": round(sma_ms * 1e3, 2), "algorithmic_flops": mflops, "algorithmic_bytes": mbytes},
        "kernels_us": {k: round(v * 1e3, 2) for k, v in sorted(avg.items())},
        "kernels_pass": "%d further steps with library events around every launch" % nprof,
        "mfma_busy": {k: mfma_for(k) for k in ("k_sma", "k_chunk_out_heads", "k_chunk_state_heads",
                                               "k_bwd_scores", "k_bwd_tokens", "k_bwd_mem",
                                               "k_sbwd_group", "k_sbwd_quad")},
    }
    if not args.no_decode:
        dbytes = decode_bytes(dw)
        dec_mean = sum(dec_ms) / len(dec_ms)
        part_ms = avg["k_decode_partial"]
        cache_bytes = dw.batch * dw.nheads * (dw.context // dw.chunk) * dw.dstate * dw.headdim * 2
        extra["decode"] = {
            "workload": dw.name, "us_per_step": round(dec_mean * 1e3, 2),
            "hbm_gbps": round(dbytes / (dec_mean * 1e-3) / 1e9, 1),
            "hbm_frac": round(dbytes / (dec_mean * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "algorithmic_bytes": dbytes,
            "k_decode_partial_gbps": round(cache_bytes / (part_ms * 1e-3) / 1e9, 1),
            "k_decode_partial_traffic": traffic_for("k_decode_partial")}

    if not args.no_decode and not args.no_ragged:
        # ragged batch (row b at its own position, spread evenly over the
        # context), timed on its own after the steps above
        R = 10
        pos_list = [dw.chunk + (b * (dw.context - dw.chunk)) // max(dw.batch - 1, 1)
                    for b in range(dw.batch)]
        pos_r = torch.tensor(pos_list, dtype=torch.int64, device=dev)
        pmax = max(pos_list)

        def decode_ragged():
            dart.decode_step_ragged(pos_r, pmax, D["x"], D["dt"], D["A"], D["Bm"], D["Cm"], D["q"],
                                    D["e"], D["z"], h_state, chunk_acc, cache, dw.chunk, y=y_dec,
                                    workspace=ws_dec, stream=stream)
        for _ in range(3):
            decode_ragged()
        er = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        er[0].record(stream)
        for _ in range(R):
            decode_ragged()
        er[1].record(stream)
        torch.cuda.synchronize()
        rag_ms = er[0].elapsed_time(er[1]) / R
        esz = 2
        rbytes = (sum(p // dw.chunk for p in pos_list) * dw.nheads * dw.dstate * dw.headdim * esz
                  + 4 * dw.batch * dw.nheads * dw.dstate * dw.headdim * 4
                  + dw.batch * dw.nheads * dw.headdim * esz * 2
                  + dw.batch * dw.ngroups * (3 * dw.dstate + dw.headdim) * esz + dw.batch * dw.nheads * 8)
        extra["decode_ragged"] = {
            "positions": "row b at %d + b (%d - %d) / %d" % (dw.chunk, dw.context, dw.chunk, dw.batch - 1),
            "us_per_step": round(rag_ms * 1e3, 2), "algorithmic_bytes": rbytes,
            "hbm_gbps": round(rbytes / (rag_ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(rbytes / (rag_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}

    if not args.no_bwd:
        # SMA backward on the same workload (loss sum dy . y), timed on its own
        # after the steps above, with the forward's LSE and memories
        g = torch.Generator(device=dev)
        g.manual_seed(4)
        dy = torch.randn((B, L, H, P), generator=g, device=dev).to(bf)
        f32 = dict(dtype=torch.float32, device=dev)
        grads = {"dq": torch.empty(T["q"].shape, **f32), "de": torch.empty(T["e"].shape, **f32),
                 "dC": torch.empty(T["Cm"].shape, **f32), "dmem": torch.empty(mem.shape, **f32),
                 "dz": torch.empty(T["z"].shape, **f32)}
        ws_bwd = torch.empty(dart.workspace_bytes("sma_bwd", dims), dtype=torch.uint8, device=dev)

        def backward():
            dart.sma_bwd(T["q"], T["e"], T["Cm"], mem, T["z"], lse, dy, S, out=grads,
                         workspace=ws_bwd, stream=stream)
        for _ in range(3):
            backward()
        R = 10
        eb = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        eb[0].record(stream)
        for _ in range(R):
            backward()
        eb[1].record(stream)
        torch.cuda.synchronize()
        bk = profiled(backward, R)
        bavg = {k: v[0] / max(v[1], 1) for k, v in bk.items()}
        bwd_ms = eb[0].elapsed_time(eb[1]) / R
        bflops = sma_bwd_flops(w)
        extra["sma_bwd"] = {
            "us": round(bwd_ms * 1e3, 2), "algorithmic_flops": bflops,
            "mfma_util": round(bflops / (bwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "tokens_per_s": round(B * L / (bwd_ms * 1e-3), 1),
            "kernels_us": {k: round(v * 1e3, 2) for k, v in sorted(bavg.items())},
            "traffic_bytes": {k: traffic_for(k) for k in ("k_bwd_scores", "k_bwd_tokens", "k_bwd_mem")}}
        del ws_bwd

        # scan backward on the same workload, chained as a layer's backward
        # runs: the y_ssd gradient is dy itself (the residual) and the memory
        # gradient is what the SMA backward just produced
        ws_sb = torch.empty(dart.workspace_bytes("ssd_bwd", dims), dtype=torch.uint8, device=dev)
        sgrads = {"dx": torch.empty((B, L, H, P), **f32), "ddt": torch.empty((B, L, H), **f32),
                  "dA": torch.empty((H,), **f32), "dB": torch.empty(T["Bm"].shape, **f32),
                  "dC": torch.empty(T["Cm"].shape, **f32),
                  "dh0": torch.empty((B, H, w.dstate, P), **f32)}

        def scan_backward():
            dart.ssd_bwd(T["x"], T["dt"], T["A"], T["Bm"], T["Cm"], S, dy, dmem=grads["dmem"],
                         out=sgrads, workspace=ws_sb, stream=stream)
        for _ in range(3):
            scan_backward()
        torch.cuda.synchronize()
        eb[0].record(stream)
        for _ in range(R):
            scan_backward()
        eb[1].record(stream)
        torch.cuda.synchronize()
        sk = profiled(scan_backward, R)
        savg = {k: v[0] / max(v[1], 1) for k, v in sk.items()}
        sb_ms = eb[0].elapsed_time(eb[1]) / R
        sbb = ssd_bwd_bytes(w)
        # measured HBM bytes of one call (the contraction kernel runs twice: the
        # state's and the adjoint's chunk contributions)
        per_call = {k: traffic_for(k) for k in ("k_sbwd_contract", "k_sbwd_pass2", "k_sbwd_group",
                                                "k_sbwd_quad", "k_sbwd_bc")}
        total = (None if any(v is None for v in per_call.values())
                 else 2 * per_call["k_sbwd_contract"] + sum(v for k, v in per_call.items()
                                                            if k != "k_sbwd_contract"))
        extra["ssd_bwd"] = {
            "us": round(sb_ms * 1e3, 2), "tokens_per_s": round(B * L / (sb_ms * 1e-3), 1),
            "algorithmic_bytes": sbb, "hbm_gbps": round(sbb / (sb_ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(sbb / (sb_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "kernels_us": {k: round(v * 1e3, 2) for k, v in sorted(savg.items())},
            "traffic_bytes": per_call,
            "traffic_vs_algorithmic": None if total is None else round(total / sbb, 3)}
        del ws_sb, sgrads, grads

    if not args.no_block:
        # the block around the path at the same shape, timed on its own: the
        # width-4 convolution + SiLU over the x, B, C channels of an input
        # projection row (z, xBC, dt, q, e and gate columns), softplus step
        # sizes, and the gated RMSNorm over the H*P output channels
        G_, N_ = w.ngroups, w.dstate
        D_in = H * P
        C_conv = D_in + 2 * G_ * N_
        row = D_in + C_conv + H + G_ * (N_ + P) + H
        g = torch.Generator(device=dev)
        g.manual_seed(5)
        proj = torch.randn((B, L, row), generator=g, device=dev).to(bf)
        cw = torch.randn((C_conv, 4), generator=g, device=dev) * 0.5
        cb = torch.randn((C_conv,), generator=g, device=dev) * 0.1
        st_c = torch.zeros((B, C_conv, 3), dtype=torch.float32, device=dev)
        conv_out = torch.empty((B, L, C_conv), dtype=bf, device=dev)
        dtb = torch.randn((H,), generator=g, device=dev)
        dt_out = torch.empty((B, L, H), dtype=torch.float32, device=dev)
        ynorm = torch.empty((B, L, D_in), dtype=bf, device=dev)
        nw = torch.ones((D_in,), dtype=torch.float32, device=dev)
        yv = y.view(B, L, D_in) if y.is_contiguous() else y.reshape(B, L, D_in)
        legs = {
            "conv1d_silu": (lambda: dart.conv1d_silu(proj[:, :, D_in:], cw, cb, state_out=st_c,
                                                     channels=C_conv, out=conv_out, stream=stream),
                            2 * B * L * C_conv * 2 + B * C_conv * 12),
            "dt_softplus": (lambda: dart.dt_softplus(proj[:, :, D_in + C_conv:], dtb, nheads=H,
                                                     out=dt_out, stream=stream),
                            B * L * H * (2 + 4)),
            "gated_rmsnorm": (lambda: dart.gated_rmsnorm(yv, proj[:, :, :D_in], nw, out=ynorm,
                                                         stream=stream),
                              3 * B * L * D_in * 2),
        }
        blk = {}
        for name, (fn, nbytes) in legs.items():
            for _ in range(3):
                fn()
            ev2 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            torch.cuda.synchronize()
            ev2[0].record(stream)
            for _ in range(10):
                fn()
            ev2[1].record(stream)
            torch.cuda.synchronize()
            ms = ev2[0].elapsed_time(ev2[1]) / 10
            blk[name] = {"us": round(ms * 1e3, 2), "algorithmic_bytes": nbytes,
                         "hbm_gbps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                         "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}
        extra["block"] = blk
        del proj, conv_out, dt_out, ynorm

    tokens = B * L
    line = {
        "metric": "DART layer fwd tokens/s @L=8192 bf16 + MFMA util %; decode step us & HBM GB/s",
        "value": round(tokens / (fwd_mean * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "seq_len": L, "heads": H, "headdim": P,
                   "dstate": N, "chunk": S, "fwd_ms": round(fwd_mean, 4),
                   "decode_workload": None if args.no_decode else dw.name,
                   "step": "scan+sma+gate forward" + ("" if args.no_decode else " + one decode token")},
        "roofline": roofline,
    }
    line.update(extra)
    if args.copy_calib_mb:
        n = args.copy_calib_mb << 20
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        line["copy_calib_bytes"] = n
        del src, dst
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_batches)
    line["wall_s_timed"] = round(wall, 3)
    if args.extra_out:
        with open(args.extra_out, "w") as fh:
            json.dump({"fwd_ms": fwd_ms, "dec_ms": dec_ms, "kernels": kernels}, fh, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
