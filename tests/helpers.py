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


def assert_lse_close(got, ref, tol, what="lse", axes_keep=(0, 2)):
    """-inf exactly where the reference has no history; elsewhere the same
    per-(b, h)-slice metric as the other outputs: max|d| / max|ref| over the
    slice's finite entries."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ninf = np.isneginf(ref)
    assert np.array_equal(np.isneginf(got), ninf), "%s: -inf pattern differs" % what
    fin = ~ninf
    assert np.all(np.isfinite(got[fin])), "%s: non-finite values" % what
    g = np.where(fin, got, 0.0)
    r = np.where(fin, ref, 0.0)
    return assert_close_slices(g, r, tol, axes_keep, what)


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
