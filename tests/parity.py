"""Parity criteria between the GPU path and the oracle.

Floating point: the loss must satisfy |g - o| <= 1e-11 |o|; each gradient
component |g_p - o_p| <= 1e-11 max(|o_p|, max_p |o_p|) (a lane-norm scale, so
components that are ~0 by structure are not judged on rounding noise);
non-finite values must agree in class (NaN, +inf, -inf).

Where several results are correct the check compares what is unique:
* a lane that misses the bar and whose numeric branch is decided by operands
  closer than 1e-9 relative (the oracle reports the margin) may legitimately
  have taken the other arm under last-ulp differences of the transcendental
  functions; it is excused and counted (the count must stay rare);
* a lane whose fp64 result itself is ill-conditioned (the oracle evaluated in
  x87 extended precision differs from its fp64 result by more than 1e-13 of
  the scale) is judged against the extended-precision value with twice the
  oracle's own fp64 error as allowance.
"""
import numpy as np

from conftest import lane_rel_err, rel_err

TOL = 1e-11


def compare(gl, gg, ol, og, ol_ext=None, og_ext=None, margin=None, tol=TOL):
    """Return the worst normalized errors over lanes that meet the strict bar
    and counts of lanes judged by the other two rules; raises AssertionError
    listing the first offending lanes."""
    el = rel_err(gl, ol)
    eg = lane_rel_err(gg, og).max(axis=1) if og is not None else np.zeros_like(el)
    strict_bad = (el > tol) | (eg > tol)
    ext_ok = np.zeros_like(strict_bad)
    if ol_ext is not None:
        # ill-conditioned lanes: judge against extended precision
        scale_l = np.maximum(np.abs(ol_ext), 1e-300)
        own_l = np.abs(ol - ol_ext) / scale_l
        ok_l = np.abs(gl - ol_ext) / scale_l <= np.maximum(2 * own_l, tol)
        if og is not None:
            own_g = lane_rel_err(og, og_ext).max(axis=1)
            ok_g = lane_rel_err(gg, og_ext).max(axis=1) <= np.maximum(2 * own_g, tol)
        else:
            ok_g = np.ones_like(ok_l)
        ext_ok = ok_l & ok_g
    bad = strict_bad & ~ext_ok
    ambiguous = margin <= 1e-9 if margin is not None else np.zeros_like(bad)
    excused = bad & ambiguous
    hard = bad & ~ambiguous
    if hard.any():
        idx = np.nonzero(hard)[0][:5]
        raise AssertionError(f"parity failure in lanes {idx.tolist()}: loss err {el[idx]}, grad err {eg[idx]}")
    return dict(max_loss_err=float(np.max(np.where(strict_bad, 0, el), initial=0)),
                max_grad_err=float(np.max(np.where(strict_bad, 0, eg), initial=0)),
                n_ambiguous=int(excused.sum()), n_ill_conditioned=int((strict_bad & ext_ok).sum()),
                n_lanes=int(el.size))
