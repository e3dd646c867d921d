"""Comparison rule shared by the parity tests.

Per element: |gpu - ref| <= rtol * (|ref| + rms(ref)), where rms is taken over
the whole tensor; integer results must be equal.  The max and normwise errors
are returned for reporting."""
import numpy as np


def compare(gpu, ref, rtol, name=""):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (name, gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{name}: non-finite GPU values"
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    err = np.abs(gpu - ref)
    bound = rtol * (np.abs(ref) + rms)
    bad = err > bound
    worst = float(np.max(err / np.maximum(np.abs(ref) + rms, 1e-300))) if ref.size else 0.0
    normwise = float(np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-300)) if ref.size else 0.0
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{bad.size} elements out of tolerance "
                             f"rtol={rtol}; worst at {i}: gpu={gpu[i]!r} ref={ref[i]!r}; "
                             f"normwise={normwise:.3e}")
    return worst, normwise


def compare_chained(gpu, ref, rtol, name="", frac=1e-3, cap=5.0, exact=None):
    """Rule for results that went through a chain of bfloat16 storage points
    on both sides (a whole forward + backward).  Where a float32 value and its
    float64 counterpart straddle a bf16 rounding boundary the two sides store
    neighbouring bf16 values; downstream sums spread that one-ulp difference,
    so after a few stages the discrepancy settles near one bf16 ulp (2**-8
    relative) in norm, with rare larger elements.  Bar: normwise error <= rtol,
    at most ``frac`` of the elements outside rtol * (|ref| + rms), none
    outside cap * rtol * (|ref| + rms).

    ``exact``, when given, is the oracle's result with no storage rounding
    (exact arithmetic); it measures the spread that bf16 storage alone
    causes.  The GPU is a second bf16-storage pipeline whose rounding errors
    are independent of the oracle's and alike in size: with E exact, R the
    oracle and G the GPU, |G - R| <= |G - E| + |R - E|, so G is more than
    rtol from R only where one of the two is more than rtol/2 from E.  The
    GPU may therefore have up to twice as many elements beyond rtol as the
    oracle has beyond rtol/2 from exact arithmetic, and its worst element
    may be up to twice the oracle's worst distance from exact arithmetic.
    (The strict, per-element check is the teacher-forced one, where both
    sides start every unit from the same stored values.)"""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (name, gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{name}: non-finite GPU values"
    if ref.size == 0:
        return 0.0, 0.0
    rms = float(np.sqrt(np.mean(ref * ref)))
    scale = np.abs(ref) + rms
    ratio = np.abs(gpu - ref) / np.maximum(scale, 1e-300)
    normwise = float(np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-300))
    n_out = int(np.sum(ratio > rtol))
    worst = float(ratio.max())
    assert normwise <= rtol, f"{name}: normwise {normwise:.3e} > {rtol}"
    allowed = frac * ratio.size
    worst_allowed = cap * rtol
    if exact is not None:
        exact = np.asarray(exact, np.float64)
        assert exact.shape == ref.shape, (name, exact.shape, ref.shape)
        spread = np.abs(exact - ref) / np.maximum(scale, 1e-300)
        allowed = max(allowed, 2 * int(np.sum(spread > rtol / 2)))
        worst_allowed = max(worst_allowed, 2 * float(spread.max()))
    i = int(np.argmax(ratio))
    where = f"worst at flat index {i}: gpu={gpu.flat[i]!r} ref={ref.flat[i]!r} scale={scale.flat[i]:.3e}"
    assert n_out <= allowed, f"{name}: {n_out}/{ratio.size} elements beyond {rtol} (allowed {allowed:.0f}); {where}"
    assert worst <= worst_allowed, f"{name}: worst element {worst:.3e} > {worst_allowed:.3e}; {where}"
    return worst, normwise
