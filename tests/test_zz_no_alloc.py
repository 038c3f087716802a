"""The allocation-free decode step (dart_decode_step_noalloc) against the
decode step with a caller workspace (dart_decode_step): the same kernels, so
every output -- y, h_state, chunk_acc and the cache -- must agree bit for bit.
Two calls in a row share the library's scratch, the second on a smaller
problem than the first."""
import numpy as np
import pytest

from paper_2608_02032_amd import dart, synth
from tests.helpers import f32_dev, to_dev

pytestmark = pytest.mark.gpu


def _step(dtype, B_, H, N, S, m, offset, seed):
    import torch
    P = 64
    pos = m * S + offset
    Mcap = m + 2
    print("\n[gpu-case] decode noalloc vs workspace dtype=%s B=%d H=%d N=%d S=%d pos=%d"
          % (dtype, B_, H, N, S, pos), flush=True)
    rng = np.random.default_rng(seed)
    mem = np.zeros((B_, Mcap, H, N, P), dtype=np.float32)
    mem[:, :m] = synth.synthetic_memories(rng, B_, m, H, N, P, dtype)
    hs0 = (rng.standard_normal((B_, H, N, P)) * 0.01).astype(np.float32)
    ca0 = (rng.standard_normal((B_, H, N, P)) * 0.01).astype(np.float32)
    inp = synth.decode_inputs(B_, H, P, N, dtype, seed=seed + 1)
    dev = {k: to_dev(inp[k], dtype) for k in ("x", "Bm", "Cm", "q", "e", "z")}
    dt, A = f32_dev(inp["dt"]), f32_dev(inp["A"])
    outs = []
    for fn in (dart.decode_step, dart.decode_step_noalloc):
        hs, ca, cache = f32_dev(hs0), f32_dev(ca0), to_dev(mem, dtype)
        y = fn(pos, dev["x"], dt, A, dev["Bm"], dev["Cm"], dev["q"], dev["e"], dev["z"], hs, ca,
               cache, S)
        torch.cuda.synchronize()
        outs.append((y.cpu(), hs.cpu(), ca.cpu(), cache.cpu()))
    for name, a, b in zip(("y", "h_state", "chunk_acc", "cache"), outs[0], outs[1]):
        assert torch.equal(a, b), name
        assert torch.isfinite(a.float()).all(), name


def test_noalloc_decode_equals_workspace_decode_twice_second_smaller():
    # a bf16 step over 40 memories (several splits), then a smaller fp32 step
    # that closes a chunk (append path) in the scratch the first one used
    _step("bf16", 8, 4, 128, 256, 40, 17, seed=3)
    _step("fp32", 2, 2, 64, 64, 5, 63, seed=4)
