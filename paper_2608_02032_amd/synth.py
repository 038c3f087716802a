"""Seeded synthetic inputs for DART's hot path.

This module only draws random numbers and rounds them to the storage
precision; it holds none of the method's arithmetic.  Both the GPU path
(tests, benchmark) and the CPU oracle's checks take their inputs from here,
so the two sides see bit-identical values.

Value distributions (the paper benchmarks its kernels on precomputed synthetic
inputs X, dt, A, B, C, Q, E and memories and gives no distribution; these are
the stated workload recipe):
    x ~ N(0, 1);   B, C ~ N(0, 1/N) (variance 1/N);
    Q, E ~ N(0, 1/sqrt(P)) (variance 1/sqrt(P));   z ~ N(0, 1);
    A_h = -exp(U[ln 1, ln 16]);
    dt = clamp(softplus(eps + b_h), 1e-3, 1e-1), eps ~ N(0, 1),
         b_h = softplus^-1(exp(U[ln 1e-3, ln 1e-1])).
Draw order from numpy.random.default_rng(seed) (PCG64): A, dt-bias,
dt-noise, x, B, C, Q, E, z.  bf16 workloads round every storage-dtype tensor
once, float32 -> bfloat16 round-to-nearest-even; dt and A stay float32.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Dict, Optional

import numpy as np


@dataclass(frozen=True)
class Workload:
    """Shape of one layer invocation (symbols of the paper's App. B.2 Table 7)."""
    name: str
    batch: int
    seqlen: int
    nheads: int
    headdim: int
    dstate: int
    chunk: int
    dtype: str = "bf16"          # storage dtype: "bf16" or "fp32"
    ngroups: int = 1
    z_per_head: bool = True
    mem_capacity: int = 0        # 0 -> ceil(L/S)

    @property
    def nchunks(self) -> int:
        return -(-self.seqlen // self.chunk)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The workloads measured or checked, named by what they are.
WORKLOADS: Dict[str, Workload] = {
    "tiny_fp32_L512": Workload("tiny_fp32_L512", 1, 512, 2, 64, 32, 64, "fp32"),
    "mamba2_130m_L4096": Workload("mamba2_130m_L4096", 8, 4096, 24, 64, 128, 256, "bf16"),
    "long_L65536": Workload("long_L65536", 1, 65536, 32, 64, 128, 256, "bf16"),
}
for _S in (64, 128, 256):
    for _N in (64, 128):
        _nm = "sweep_L8192_S%d_N%d" % (_S, _N)
        WORKLOADS[_nm] = Workload(_nm, 4, 8192, 32, 64, _N, _S, "bf16")


@dataclass(frozen=True)
class DecodeWorkload:
    """One decode step over a cache of `context` tokens (context // S memories)."""
    name: str
    batch: int
    nheads: int
    headdim: int
    dstate: int
    chunk: int
    context: int
    dtype: str = "bf16"
    ngroups: int = 1
    z_per_head: bool = True


DECODE_WORKLOADS: Dict[str, DecodeWorkload] = {
    "decode_B64_ctx65536": DecodeWorkload("decode_B64_ctx65536", 64, 32, 64, 128, 256, 65536),
}


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    nan = np.isnan(a)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    out = u.astype(np.uint32).view(np.float32)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    return round_bf16(a) if dtype == "bf16" else np.ascontiguousarray(a)


def _softplus(v):
    return np.where(v > 20.0, v, np.log1p(np.exp(np.minimum(v, 20.0))))


def _softplus_inv(v):
    return v + np.log(-np.expm1(-v))


def draw_A_dt(rng: np.random.Generator, batch: int, seqlen: int, nheads: int):
    A = -np.exp(rng.uniform(math.log(1.0), math.log(16.0), size=nheads))
    dt_target = np.exp(rng.uniform(math.log(1e-3), math.log(1e-1), size=nheads))
    bias = _softplus_inv(dt_target)
    noise = rng.standard_normal((batch, seqlen, nheads))
    dt = np.clip(_softplus(noise + bias), 1e-3, 1e-1)
    return A.astype(np.float32), dt.astype(np.float32)


def forward_inputs(w: Workload, seed: int = 0) -> Dict[str, np.ndarray]:
    """All inputs of one forward pass as float32 numpy arrays (storage-rounded)."""
    rng = np.random.default_rng(seed)
    B_, L, H, P, N, G = w.batch, w.seqlen, w.nheads, w.headdim, w.dstate, w.ngroups
    A, dt = draw_A_dt(rng, B_, L, H)
    x = rng.standard_normal((B_, L, H, P), dtype=np.float32)
    Bm = rng.standard_normal((B_, L, G, N), dtype=np.float32) * np.float32(1.0 / math.sqrt(N))
    Cm = rng.standard_normal((B_, L, G, N), dtype=np.float32) * np.float32(1.0 / math.sqrt(N))
    qe_std = np.float32(1.0 / math.sqrt(math.sqrt(P)))
    q = rng.standard_normal((B_, L, G, N), dtype=np.float32) * qe_std
    e = rng.standard_normal((B_, L, G, P), dtype=np.float32) * qe_std
    zshape = (B_, L, H) if w.z_per_head else (B_, L)
    z = rng.standard_normal(zshape, dtype=np.float32)
    st = w.dtype
    return {
        "A": A, "dt": dt,
        "x": to_storage(x, st), "Bm": to_storage(Bm, st), "Cm": to_storage(Cm, st),
        "q": to_storage(q, st), "e": to_storage(e, st), "z": to_storage(z, st),
    }


def synthetic_memories(rng: np.random.Generator, batch: int, nmem: int, nheads: int,
                       dstate: int, headdim: int, dtype: str,
                       rms_lo: float = 1.4e-3, rms_hi: float = 1.1e-2) -> np.ndarray:
    """Chunk memories drawn directly: memory c of head h is s * N(0,1) with s
    log-uniform in [rms_lo, rms_hi] (the per-chunk RMS range the scan produces
    under the distributions above)."""
    s = np.exp(rng.uniform(math.log(rms_lo), math.log(rms_hi), size=(batch, nmem, nheads, 1, 1)))
    m = rng.standard_normal((batch, nmem, nheads, dstate, headdim)).astype(np.float32)
    return to_storage((m * s).astype(np.float32), dtype)


def decode_inputs(batch: int, nheads: int, headdim: int, dstate: int, dtype: str, seed: int,
                  ngroups: int = 1, z_per_head: bool = True) -> Dict[str, np.ndarray]:
    """Per-token inputs of one decode step (same distributions as the forward)."""
    rng = np.random.default_rng(seed)
    B_, H, P, N, G = batch, nheads, headdim, dstate, ngroups
    A, dt = draw_A_dt(rng, B_, 1, H)
    dt = dt.reshape(B_, H)
    x = rng.standard_normal((B_, H, P), dtype=np.float32)
    Bm = rng.standard_normal((B_, G, N), dtype=np.float32) * np.float32(1.0 / math.sqrt(N))
    Cm = rng.standard_normal((B_, G, N), dtype=np.float32) * np.float32(1.0 / math.sqrt(N))
    qe_std = np.float32(1.0 / math.sqrt(math.sqrt(P)))
    q = rng.standard_normal((B_, G, N), dtype=np.float32) * qe_std
    e = rng.standard_normal((B_, G, P), dtype=np.float32) * qe_std
    z = rng.standard_normal((B_, H) if z_per_head else (B_,), dtype=np.float32)
    return {
        "A": A, "dt": dt,
        "x": to_storage(x, dtype), "Bm": to_storage(Bm, dtype), "Cm": to_storage(Cm, dtype),
        "q": to_storage(q, dtype), "e": to_storage(e, dtype), "z": to_storage(z, dtype),
    }


def torch_device_memories(batch: int, nmem_cap: int, nmem: int, nheads: int, dstate: int,
                          headdim: int, seed: int, device="cuda", dtype=None,
                          rms_lo: float = 1.4e-3, rms_hi: float = 1.1e-2):
    """A large synthetic memory cache drawn on the device with a seeded torch
    generator (for caches too large to draw on the host).  Slots >= nmem are 0.
    Returns (mem, scales) where mem is [B][Mcap][H][N][P] and scales [B][nmem][H]."""
    import torch
    dtype = dtype or torch.bfloat16
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    mem = torch.zeros((batch, nmem_cap, nheads, dstate, headdim), dtype=dtype, device=device)
    u = torch.rand((batch, nmem, nheads), generator=g, device=device, dtype=torch.float32)
    scales = torch.exp(math.log(rms_lo) + u * (math.log(rms_hi) - math.log(rms_lo)))
    for c in range(nmem):
        blk = torch.randn((batch, nheads, dstate, headdim), generator=g, device=device,
                          dtype=torch.float32)
        blk.mul_(scales[:, c, :, None, None])
        mem[:, c].copy_(blk.to(dtype))
    return mem, scales
