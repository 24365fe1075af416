"""Shared comparison helpers for the GPU parity tests (no method arithmetic)."""
import numpy as np

RTOL = 1e-5  # |gpu - oracle| <= RTOL * sum|terms| per output (fp32 sums)


def assert_terms_close(got, ref, mag, rtol=RTOL, what="output", slack=None):
    """Element-wise check of an fp32 result against the fp64 oracle value.

    ``mag`` is the oracle's sum of absolute term values for each output; an
    output with no terms must be exactly zero.  ``slack`` (optional, per
    output) is added to the bound: what the output may differ by when a
    decision inside it (a ReLU's sign) cannot be settled in fp32.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    mag = np.asarray(mag, dtype=np.float64)
    assert got.shape == ref.shape == mag.shape, (got.shape, ref.shape, mag.shape)
    err = np.abs(got - ref)
    bound = rtol * mag
    if slack is not None:
        bound = bound + np.asarray(slack, dtype=np.float64)
    bad = err > bound
    if bad.any():
        k = np.argmax(np.where(bad, err - bound, -np.inf))
        idx = np.unravel_index(k, got.shape)
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {got.size} elements exceed {rtol}*sum|terms|; worst at {idx}: "
            f"got {got[idx]!r} ref {ref[idx]!r} sum|terms| {mag[idx]!r}")
    return float((err / np.where(mag > 0, mag, 1)).max(initial=0.0))
