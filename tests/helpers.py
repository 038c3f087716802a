"""Shared test helpers: tolerance metric and host/device conversions."""
import numpy as np

# Tolerances: fp32 storage 1e-4, bf16 storage with fp32 accumulation 2e-2.
TOL = {"fp32": 1e-4, "bf16": 2e-2}


def slice_rel_err(got, ref, axes_keep=(0, 2)):
    """max over (b, h) slices of max|got - ref| / max|ref| (NaN/Inf -> inf)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if not np.all(np.isfinite(got)):
        return float("inf")
    diff = np.abs(got - ref)
    red = tuple(i for i in range(got.ndim) if i not in axes_keep)
    num = diff.max(axis=red)
    den = np.abs(ref).max(axis=red)
    den = np.where(den == 0, 1.0, den)
    return float((num / den).max())


def assert_close_slices(got, ref, tol, axes_keep=(0, 2), what=""):
    err = slice_rel_err(got, ref, axes_keep)
    print("  %-28s max slice rel err %.3e (tol %.0e)" % (what, err, tol), flush=True)
    assert err <= tol, "%s: max slice relative error %.3e > %.1e" % (what, err, tol)
    return err


# Per-entry bound on the log-sum-exp.  fp32: |d| <= 1e-4 (1 + |ref|).  bf16:
# a logit passes through three bf16 roundings -- the stored memory, the key
# side r (.) dH and the query operand Qbar log2(e)/sqrt(N) -- each a relative
# error of at most u = 2^-9 per element, independent across the N P terms of
# the logit.  Under the normalisation every operand has unit RMS and the
# 1/sqrt(N) scale cancels the sum over n, so the logit error has a standard
# deviation of about u sqrt(k P / 3) for k roundings: u sqrt(P) = 0.0156 at
# P = 64, k = 3.  The LSE, a weighted mean of its logits, inherits it.  The
# bound is 8 such deviations, |d| <= 8 u sqrt(P) = 0.125 absolute.
LSE_ATOL = {"fp32": 0.0, "bf16": 8.0 * 2.0 ** -9 * 8.0}
LSE_RTOL = {"fp32": 1e-4, "bf16": 0.0}


def assert_lse_close(got, ref, dtype, what="lse"):
    """-inf exactly where the reference has no history; elsewhere every entry
    within |d| <= LSE_ATOL + LSE_RTOL (1 + |ref|)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ninf = np.isneginf(ref)
    assert np.array_equal(np.isneginf(got), ninf), "%s: -inf pattern differs" % what
    fin = ~ninf
    assert np.all(np.isfinite(got[fin])), "%s: non-finite values" % what
    d = np.abs(got[fin] - ref[fin])
    bound = LSE_ATOL[dtype] + LSE_RTOL[dtype] * (1.0 + np.abs(ref[fin]))
    worst = float((d / bound).max()) if d.size else 0.0
    print("  %-28s max |d| %.3e, max |d|/bound %.3f" % (what, float(d.max()) if d.size else 0.0, worst),
          flush=True)
    assert worst <= 1.0, "%s: |d| exceeds the per-entry bound (worst ratio %.3f)" % (what, worst)
    return worst


def to_dev(a, dtype, device="cuda"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32)))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.to(device)


def f32_dev(a, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).to(device)


def to_np(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)
