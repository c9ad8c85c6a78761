"""Shared helpers of the parity tests."""
import numpy as np

# Bound on the scaled error of every float result (embeddings, pooled bags,
# core gradients): |x - r| <= TOL * m, where r is the oracle's value and m the
# oracle's value on the absolute inputs (|G1|, |G2|, |G3|, |dV|).  m bounds
# every partial sum of the exact result, so fp32 accumulation of K terms in
# sequence stays within K * 2^-24 * m in the worst case.  The contractions
# chain at most R = 64 or d-sized terms, but the sums over occurrences and
# rows chain far more: a dE row sums its occurrences 256 at a time and then
# the chunk partials (the hottest row of the 8-table training workload has
# about 76,000 occurrences), dG3 collects every row with its i3, and dG1/dG2
# collect thousands of slice and chunk partials.  For those the worst-case
# bound exceeds TOL; the rounding errors of such sums are not all of one sign
# and m (a sum of magnitudes) is far above |r|, so TOL = 1e-5 holds with a
# margin that is empirical, checked on the hottest rows and slices of the
# full-size training workload, where the chains are longest.
TOL = 1e-5


def scaled_err(x, ref, mag):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    mag = np.asarray(mag, dtype=np.float64)
    err = np.abs(x - ref)
    out = np.zeros_like(err)
    pos = mag > 0
    out[pos] = err[pos] / mag[pos]
    out[~pos] = np.where(err[~pos] == 0, 0.0, np.inf)
    return out


def abs_case(case):
    """The same workload on absolute values: its oracle results bound every partial sum."""
    c = dict(case)
    for k in ("G1", "G2", "G3"):
        c[k] = np.abs(case[k])
    if "dV" in case:
        c["dV"] = np.abs(case["dV"])
    return c


def assert_close(name, x, ref, mag, tol=TOL):
    e = scaled_err(x, ref, mag)
    worst = float(e.max()) if e.size else 0.0
    assert worst <= tol, f"{name}: max scaled error {worst:.3e} > {tol:.1e} at {np.unravel_index(int(e.argmax()), e.shape)}"
    return worst
