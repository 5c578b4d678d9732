"""Parity criteria between the GPU path and the oracle.

Floating point: the loss must satisfy |g - o| <= 1e-11 |o|; each gradient
component |g_p - o_p| <= 1e-11 max(|o_p|, max_p |o_p|) (a lane-norm scale, so
components that are ~0 by structure are not judged on rounding noise);
non-finite values must agree in class (NaN, +inf, -inf).

``judge`` applies that bar to every lane.  Where several results are correct
it compares against each of them, and every lane is compared with a result
the oracle computed; nothing is excused:

* a lane whose fp64 result is itself ill-conditioned (the oracle evaluated
  in x87 extended precision differs from its fp64 result) passes when the GPU
  is within max(2 |o - o_ext|, 1e-11 scale) of the extended-precision value:
  rounding, not the method, decides its last digits;
* a lane whose result is sensitive to the last ulp of library
  transcendentals (the GPU's math library and the host's round exp, log,
  sin, cos and pow differently by an ulp or two) passes when the GPU's
  deviation from the oracle is within twice the largest deviation of four
  oracle evaluations with every transcendental result moved by a
  pseudo-random whole number of ulps in [-2, 2];
* a lane with a numeric branch whose operands sit within 1e-9 relative of a
  tie (the oracle lists such encounters) may have taken the other arm under
  last-ulp differences of the library transcendentals; it passes when the GPU
  equals, by the same bar, the oracle's evaluation of that lane with one of
  those encounters decided the other way, which is the exact result of the
  other realized trace (Section 4, Property 1).

Counts of lanes judged by each rule are returned, so they can be recorded.
"""
import numpy as np

from conftest import lane_rel_err, rel_err

TOL = 1e-11
TIE_TOL = 1e-9


def _errs(gl, gg, ol, og):
    el = rel_err(gl, ol)
    eg = lane_rel_err(gg, og).max(axis=1) if og is not None else np.zeros_like(el)
    return el, eg


def _ext_ok(gl, gg, ol, og, ole, oge, tol=TOL):
    """Judged against extended precision with twice the fp64 oracle's own
    error (at least the strict bar) as allowance."""
    scale = np.maximum(np.abs(ole), 1e-300)
    own = np.abs(ol - ole) / scale
    ok = np.abs(gl - ole) / scale <= np.maximum(2 * own, tol)
    ok |= rel_err(gl, ole) <= tol          # non-finite classes
    if og is not None:
        own_g = lane_rel_err(og, oge).max(axis=1)
        ok &= lane_rel_err(gg, oge).max(axis=1) <= np.maximum(2 * own_g, tol)
    return ok


PERTURB_ULPS = 2
PERTURB_SEEDS = (101, 202, 303, 404)


def _perturb_ok(oracle_mod, bytecode, params, obs, gl, gg, ol, og, tol=TOL):
    """GPU deviation from the oracle within twice the spread the oracle shows
    under +-2-ulp perturbations of its transcendental results."""
    el, eg = _errs(gl, gg, ol, og)
    sl = np.zeros_like(el)
    sg = np.zeros_like(eg)
    for seed in PERTURB_SEEDS:
        pl, pg, _ = oracle_mod.run(bytecode, params, obs, grad=gg is not None, perturb=(seed, PERTURB_ULPS))
        a, b = _errs(pl, pg, ol, og)
        sl = np.maximum(sl, a)
        sg = np.maximum(sg, b)
    return (el <= np.maximum(2 * sl, tol)) & (eg <= np.maximum(2 * sg, tol))


def compare(gl, gg, ol, og, tol=TOL):
    """Strict bar on every lane (programs without numeric branches, or
    results that must match one evaluation exactly); returns the worst
    normalized errors, raises AssertionError naming offending lanes."""
    el, eg = _errs(gl, gg, ol, og)
    bad = (el > tol) | (eg > tol)
    if bad.any():
        idx = np.nonzero(bad)[0][:5]
        raise AssertionError(f"parity failure in lanes {idx.tolist()}: loss err {el[idx]}, grad err {eg[idx]}")
    return dict(max_loss_err=float(np.max(el, initial=0)), max_grad_err=float(np.max(eg, initial=0)),
                n_lanes=int(el.size))


def judge(oracle_mod, bytecode, params, obs, gl, gg, tol=TOL, tie_tol=TIE_TOL):
    """Judge GPU results (gl[L], gg[L, P] or None) of `bytecode` on
    params[L, P] against the oracle by the rules above.  Returns a dict of
    counts and worst errors; raises AssertionError if any lane matches none of
    the oracle's results."""
    params = np.ascontiguousarray(params, dtype=np.float64)
    with_grad = gg is not None
    ol, og, _, ties = oracle_mod.run_ties(bytecode, params, obs, tie_tol=tie_tol, grad=with_grad)
    el, eg = _errs(gl, gg, ol, og)
    pending = np.nonzero((el > tol) | (eg > tol))[0]
    out = dict(n_lanes=int(el.size), n_strict=int(el.size - pending.size),
               max_loss_err=float(np.max(np.where((el > tol) | (eg > tol), 0, el), initial=0)),
               max_grad_err=float(np.max(np.where((el > tol) | (eg > tol), 0, eg), initial=0)),
               n_ill_conditioned=0, n_libm_sensitive=0, n_other_arm=0,
               n_near_tie_lanes=int((ties[:, 0] >= 0).sum()))
    if pending.size:
        sub = params[pending]
        ole, oge, _ = oracle_mod.run(bytecode, sub, obs, grad=with_grad, extended=True)
        ok = _ext_ok(gl[pending], gg[pending] if with_grad else None, ol[pending],
                     og[pending] if with_grad else None, ole, oge, tol)
        out["n_ill_conditioned"] = int(ok.sum())
        pending = pending[~ok]
    if pending.size:
        ok = _perturb_ok(oracle_mod, bytecode, params[pending], obs, gl[pending],
                         gg[pending] if with_grad else None, ol[pending], og[pending] if with_grad else None, tol)
        out["n_libm_sensitive"] = int(ok.sum())
        pending = pending[~ok]
    for k in range(ties.shape[1]):
        if not pending.size:
            break
        cand = pending[ties[pending, k] >= 0]
        if not cand.size:
            break
        flip = ties[cand, k]
        fl, fg, _ = oracle_mod.run(bytecode, params[cand], obs, grad=with_grad, flip=flip)
        e1, e2 = _errs(gl[cand], gg[cand] if with_grad else None, fl, fg)
        ok = (e1 <= tol) & (e2 <= tol)
        if (~ok).any():
            rest = ~ok
            fle, fge, _ = oracle_mod.run(bytecode, params[cand[rest]], obs, grad=with_grad, flip=flip[rest],
                                         extended=True)
            ok[rest] = _ext_ok(gl[cand[rest]], gg[cand[rest]] if with_grad else None, fl[rest],
                               fg[rest] if with_grad else None, fle, fge, tol)
        out["n_other_arm"] += int(ok.sum())
        pending = np.setdiff1d(pending, cand[ok])
    if pending.size:
        idx = pending[:5]
        raise AssertionError(f"parity failure in lanes {idx.tolist()}: loss err {el[idx]}, grad err {eg[idx]}, "
                             f"near-tie encounters {ties[idx, :3].tolist()}")
    return out
