"""The parity checks themselves, on the CPU: a planted mistake in the SMA
readout or the log-sum-exp must fail the checks the GPU tests apply.

The mistakes are planted in oracle outputs (never in the HIP path): the
readout check of test_gpu_parity (y_ssd = 0, one gate z = 2, so y = SiLU(2) R,
per (b, h) slice at the bf16 tolerance) must reject R scaled by 1.05, and the
per-entry LSE bound must reject a shift of 0.15 while the forward's own bf16
rounding (about 0.1 at most) stays inside it."""
import numpy as np
import pytest

import oracle
from paper_2608_02032_amd import synth
from tests.helpers import TOL, assert_close_slices, assert_lse_close


def _case():
    w = synth.Workload("planted_bf16_L320_N32_S64", 1, 320, 2, 64, 32, 64, "bf16")
    d = synth.forward_inputs(w, seed=7)
    rng = np.random.default_rng(107)
    mem = synth.synthetic_memories(rng, w.batch, w.nchunks, w.nheads, w.dstate, w.headdim, w.dtype)
    ys0 = np.zeros((w.batch, w.seqlen, w.nheads, w.headdim), dtype=np.float32)
    z2 = np.full_like(d["z"], 2.0)
    y, lse = oracle.sma(d["q"], d["e"], d["Cm"], mem, z2, ys0, w.chunk)
    return w, y, lse


def test_readout_check_rejects_a_five_percent_error_in_R():
    w, y, _ = _case()
    tol = TOL[w.dtype]
    assert_close_slices(y, y, tol, what="R vs itself")
    with pytest.raises(AssertionError):
        assert_close_slices(1.05 * y, y, tol, what="R x 1.05")
    with pytest.raises(AssertionError):
        assert_close_slices(0.95 * y, y, tol, what="R x 0.95")
    # a 5 % error confined to one head still fails (per-slice metric)
    bad = y.copy()
    bad[:, :, 1] *= 1.05
    with pytest.raises(AssertionError):
        assert_close_slices(bad, y, tol, what="R x 1.05 on head 1")


def test_lse_bound_rejects_a_planted_shift():
    w, _, lse = _case()
    assert_lse_close(lse + 0.1, lse, w.dtype, what="lse + 0.1")
    with pytest.raises(AssertionError):
        assert_lse_close(lse + 0.15, lse, w.dtype, what="lse + 0.15")
    bad = lse.copy()
    bad[0, 200, 1] += 0.15          # one entry
    with pytest.raises(AssertionError):
        assert_lse_close(bad, lse, w.dtype, what="one entry + 0.15")
    with pytest.raises(AssertionError):
        assert_lse_close(lse + 2e-3, lse, "fp32", what="fp32 lse + 2e-3")
    # a finite value where the reference has no history
    bad = lse.copy()
    bad[0, 0, 0] = 0.0
    with pytest.raises(AssertionError):
        assert_lse_close(bad, lse, w.dtype, what="first chunk finite")
