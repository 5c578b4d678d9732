"""Pins for the oracle's two auxiliary modes, against things other than the
oracle itself.

* The x87 extended-precision build (``run(..., extended=True)``), which the
  GPU parity tests use to judge ill-conditioned lanes: every primitive
  against the complex-step derivative of the forward-only evaluator
  (tests/cstep.py), the closed forms of the exponential-decay gradient and of
  RK4 on a linear ODE, the dense Kalman likelihood, random trees; and a
  cancellation that only a wider format resolves, so a build that silently
  evaluates in fp64 (or maps a function to the wrong one) fails.
* The branch-flip option (``flip``) and the near-tie listing (``run_ties``),
  which the parity tests use for lanes whose comparison sits within rounding
  of a tie: encounter counting in walk order (loops count once per trip),
  the closest gaps first, and a flipped lane equal to the closed form of the
  other path.
"""
import math

import numpy as np
import pytest

import cstep
import test_oracle_pins as T
from conftest import lane_rel_err, rel_err
from primitive_programs import primitive_programs
from workloads import bytecode as B
from workloads import configs
from workloads.bytecode import Asm


def _finite_rows(params):
    # rows at exactly the log/sqrt clamp point are pinned apart: there the
    # method's reading (no adjoint at or below 1e-8) is not the analytic one
    return [p for p in params if all(math.isfinite(v) and v != 1e-8 for v in p)]


@pytest.mark.parametrize("k", range(len(primitive_programs())))
def test_extended_every_primitive_vs_cstep(oracle_mod, k):
    bc, params = primitive_programs()[k]
    for theta in _finite_rows(params):
        loss, g, _ = oracle_mod.run(bc, [theta], [], extended=True)
        want_loss = cstep.loss(bc, theta, [])
        want = cstep.gradient(bc, theta, [])
        assert rel_err(loss[0], want_loss.real if isinstance(want_loss, complex) else want_loss) <= 1e-13
        assert lane_rel_err(g, [want]).max() <= 1e-12, (k, theta, g, want)


def test_extended_select_clamp_abs_exact(oracle_mod):
    """Decisions and clamps are the same in either precision."""
    loss, g, m = oracle_mod.run(T._select_prog(), [[1.0, 1.0, 5.0], [float("nan"), 1.0, 5.0],
                                                   [0.5, 1.0, 0.001], [2.0, 1.0, 5.0]],
                                [], margin=True, extended=True)
    assert loss[0] == 10.0 and loss[1] == 10.0 and loss[3] == 10.0
    assert rel_err(loss[2], math.exp(1.0)) <= 1e-15
    assert list(g[0]) == [0.0, 0.0, 2.0] and g[2, 0] == 0.0 and g[2, 1] == 0.0
    for op, f in ((B.LOG, math.log), (B.SQRT, math.sqrt)):
        loss, g, _ = oracle_mod.run(T._log_prog(op), [[1e-9], [-1.0], [1e-8]], [], extended=True)
        assert np.all(loss == f(1e-8)) and np.all(g == 0.0)
    A = Asm(1, 0)
    A.param(0).abs().halt()
    loss, g, _ = oracle_mod.run(A.bytes(), [[0.0], [-2.0], [3.0]], [], extended=True)
    assert list(g[:, 0]) == [0.0, -1.0, 1.0]


def test_extended_resolves_cancellation(oracle_mod):
    """(p0 + p1) - p0 with p0 = 1, p1 = 1e-17: fp64 rounds the sum to 1 and
    returns 0; a 64-bit significand keeps p1 to about 1e-19 absolute.  The
    product p2 * (p0 + p1) * ... checks that the gradient path is wide too."""
    A = Asm(2, 0)
    A.param(0).param(1).add().param(0).sub().halt()
    bc = A.bytes()
    lo, _, _ = oracle_mod.run(bc, [[1.0, 1e-17]], [])
    le, ge, _ = oracle_mod.run(bc, [[1.0, 1e-17]], [], extended=True)
    assert lo[0] == 0.0
    assert abs(le[0] - 1e-17) <= 2e-19
    assert list(ge[0]) == [0.0, 1.0]
    # exp(p0) - exp(p0 + p1): the fp64 result is dominated by rounding
    A = Asm(2, 0)
    A.param(0).exp().param(0).param(1).add().exp().sub().halt()
    le, _, _ = oracle_mod.run(A.bytes(), [[0.5, 1e-15]], [], extended=True)
    want = -math.exp(0.5) * math.expm1(1e-15)
    assert abs(le[0] - want) <= 1e-3 * abs(want)


def test_extended_exp_decay_closed_form(oracle_mod):
    w = configs.exp_decay(L=8)
    n = 64
    t, y = w.obs[:n], w.obs[n:]
    loss, g, _ = oracle_mod.run(w.bytecode, w.params, w.obs, extended=True)
    for l, (a, b, c) in enumerate(w.params):
        e = [math.exp(-b * ti) for ti in t]
        r = [a * ei + c - yi for ei, yi in zip(e, y)]
        want = [2.0 / n * sum(ri * ei for ri, ei in zip(r, e)),
                -2.0 / n * sum(ri * a * ti * ei for ri, ti, ei in zip(r, t, e)),
                2.0 / n * sum(r)]
        assert rel_err(loss[l], sum(ri * ri for ri in r) / n) <= 1e-13
        assert lane_rel_err(g[l], want).max() <= 1e-12


def test_extended_lotka_volterra_decoupled_closed_form(oracle_mod):
    T_, h = 30, 0.02
    al, ga, x0, y0 = 0.9, 1.2, 1.1, 0.7
    obs = np.random.default_rng(5).uniform(0.5, 2.0, 2 * T_)
    loss, g, _ = oracle_mod.run(configs.lotka_volterra_program(T_), [[al, 0.0, ga, 0.0, x0, y0]], obs,
                                extended=True)
    R, dR = T._rk4_R, T._rk4_dR
    zx, zy = al * h, -ga * h
    rx = [x0 * R(zx) ** (k + 1) - obs[2 * k] for k in range(T_)]
    ry = [y0 * R(zy) ** (k + 1) - obs[2 * k + 1] for k in range(T_)]
    want_loss = (sum(r * r for r in rx) + sum(r * r for r in ry)) / (2 * T_)
    d_al = sum(rx[k] * x0 * (k + 1) * R(zx) ** k * dR(zx) * h for k in range(T_)) / T_
    d_x0 = sum(rx[k] * R(zx) ** (k + 1) for k in range(T_)) / T_
    d_ga = sum(ry[k] * y0 * (k + 1) * R(zy) ** k * dR(zy) * (-h) for k in range(T_)) / T_
    d_y0 = sum(ry[k] * R(zy) ** (k + 1) for k in range(T_)) / T_
    assert rel_err(loss[0], want_loss) <= 1e-12
    assert lane_rel_err(g[0, [0, 2, 4, 5]], [d_al, d_ga, d_x0, d_y0]).max() <= 1e-11


@pytest.mark.parametrize("Tk", [1, 3])
def test_extended_kalman_dense_likelihood(oracle_mod, Tk):
    w = configs.kalman(L=2, T=Tk)
    ys = w.obs.reshape(Tk, 2)
    loss, g, _ = oracle_mod.run(w.bytecode, w.params, w.obs, extended=True)
    h = 1e-30
    for l in range(2):
        th = list(w.params[l])
        assert rel_err(loss[l], float(np.real(T._dense_kalman_nll(th, ys)))) <= 1e-11
        grad = []
        for p in range(12):
            tc = [complex(v) for v in th]
            tc[p] = complex(th[p], h)
            grad.append(np.imag(T._dense_kalman_nll(tc, ys)) / h)
        assert lane_rel_err(g[l], grad).max() <= 1e-8


def test_extended_random_trees_vs_cstep(oracle_mod):
    w = configs.random_programs(n_prog=6, L=2, n=3, seed=77)
    for i, bc in enumerate(w.programs):
        P = w.n_params_each[i]
        params = w.params[i][:, :P]
        loss, g, m = oracle_mod.run(bc, params, w.obs, margin=True, extended=True)
        for l in range(2):
            if m[l] < 1e-6:
                continue
            want = cstep.gradient(bc, list(params[l]), list(w.obs))
            assert rel_err(loss[l], cstep.loss(bc, list(params[l]), list(w.obs))) <= 1e-12
            assert lane_rel_err(g[l], want).max() <= 1e-10, (i, l)


def test_extended_agrees_with_fp64_on_well_conditioned_lanes(oracle_mod):
    """On the Lotka-Volterra and Kalman workloads (well conditioned) the two
    builds agree to a few ulp of fp64 accumulated over the trace."""
    for w in (configs.lotka_volterra(L=8, T=200), configs.kalman(L=8, T=50)):
        a = oracle_mod.run(w.bytecode, w.params, w.obs)
        b = oracle_mod.run(w.bytecode, w.params, w.obs, extended=True)
        assert rel_err(a[0], b[0]).max() <= 1e-12
        assert lane_rel_err(a[1], b[1]).max() <= 1e-11


# ------------------------------------------------------------ branch flips
def _branchy(n):
    # the loop counter is structural, so spell out each term instead of
    # indexing a per-trip constant: term k = theta0 < obs_k ? theta1*c_k : theta2^2
    A = Asm(3, n)
    A.push(0.0)
    for k in range(n):
        A.param(0).obs(k).iflt()
        A.param(1).push(float(k + 1)).mul()
        A.else_()
        A.param(2).param(2).mul()
        A.endif()
        A.add()
    return A.halt().bytes()


def test_ties_listing_and_flip_closed_form(oracle_mod):
    n = 5
    bc = _branchy(n)
    th0 = 1.0
    # gaps of theta0 = 1 to obs_k: 1e-12, 0.5, 3e-10, 0 (tie), 2e-9
    obs = np.array([1.0 + 1e-12, 1.5, 1.0 - 3e-10, 1.0, 1.0 + 2e-9])
    theta = [th0, 0.7, -1.3]
    loss, g, m, ties = oracle_mod.run_ties(bc, [theta], obs, tie_tol=1e-9)
    # encounters are numbered in walk order; listed closest first, within 1e-9 only
    assert list(ties[0]) == [3, 0, 2, -1, -1, -1, -1, -1]
    assert m[0] == 0.0

    def closed(decisions):
        l, gr = 0.0, [0.0, 0.0, 0.0]
        for k, take in enumerate(decisions):
            if take:
                l += theta[1] * (k + 1)
                gr[1] += k + 1
            else:
                l += theta[2] * theta[2]
                gr[2] += 2 * theta[2]
        return l, gr

    base = [th0 < o for o in obs]
    l0, g0 = closed(base)
    assert rel_err(loss[0], l0) <= 1e-15 and lane_rel_err(g, [g0]).max() <= 1e-15
    for enc in range(n):
        dec = list(base)
        dec[enc] = not dec[enc]
        lf, gf, _ = oracle_mod.run(bc, [theta], obs, flip=[enc])
        want_l, want_g = closed(dec)
        assert rel_err(lf[0], want_l) <= 1e-15, enc
        assert lane_rel_err(gf, [want_g]).max() <= 1e-15, enc
        lx, gx, _ = oracle_mod.run(bc, [theta], obs, flip=[enc], extended=True)
        assert rel_err(lx[0], want_l) <= 1e-15 and lane_rel_err(gx, [want_g]).max() <= 1e-15
    # -1 flips nothing; encounters are counted per trip of a loop
    lf, _, _ = oracle_mod.run(bc, [theta], obs, flip=[-1])
    assert lf[0] == loss[0]


def test_flip_counts_loop_trips(oracle_mod):
    """An IFLT inside a counted loop is one encounter per trip."""
    A = Asm(2, 4)
    A.push(0.0).storel(0)
    A.loop(4)
    A.loadl(0).param(0).obs(0, 1).iflt().param(1).else_().push(0.0).endif().add().storel(0)
    A.endloop()
    A.loadl(0).halt()
    bc = A.bytes()
    obs = np.array([0.0, 2.0, 0.0, 2.0])         # theta0 = 1: taken on trips 1 and 3
    loss, g, _ = oracle_mod.run(bc, [[1.0, 3.0]], obs)
    assert loss[0] == 6.0 and list(g[0]) == [0.0, 2.0]
    for trip, want in ((0, 9.0), (1, 3.0), (2, 9.0), (3, 3.0)):
        lf, gf, _ = oracle_mod.run(bc, [[1.0, 3.0]], obs, flip=[trip])
        assert lf[0] == want and gf[0, 1] == want / 3.0, trip
    _, _, _, ties = oracle_mod.run_ties(bc, [[2.0, 3.0]], obs, tie_tol=0.0)
    assert list(ties[0][:3]) == [1, 3, -1]      # exact ties on trips 1 and 3, in walk order


# ------------------------------------------------- transcendental perturbation
def test_perturb_zero_ulps_and_no_transcendentals_are_identity(oracle_mod):
    w = configs.random_programs(n_prog=3, L=16, n=8, seed=5)
    for q, bc in enumerate(w.programs):
        P = w.n_params_each[q]
        a = oracle_mod.run(bc, w.params[q][:, :P], w.obs)
        b = oracle_mod.run(bc, w.params[q][:, :P], w.obs, perturb=(7, 0))
        assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()
    lv = configs.lotka_volterra(L=4, T=20)             # no library transcendental at all
    a = oracle_mod.run(lv.bytecode, lv.params, lv.obs)
    b = oracle_mod.run(lv.bytecode, lv.params, lv.obs, perturb=(3, 4))
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()


def _ulp_moves(y, k):
    out = {}
    for d in range(-k, k + 1):
        v = y
        for _ in range(abs(d)):
            v = np.nextafter(v, np.inf if d > 0 else -np.inf)
        out[float(v)] = d
    return out


@pytest.mark.parametrize("op", [B.EXP, B.LOG, B.SIN, B.COS])
def test_perturb_moves_each_result_by_at_most_k_ulps(oracle_mod, op):
    """loss = f(p0) * p1 with p1 = 1: every lane's loss is f(p0) moved by a
    whole number of ulps in [-2, 2]; over many lanes every move occurs; the
    gradient of p1 is that same perturbed value (the rule reads z or a fresh
    evaluation of the derivative, itself perturbed)."""
    A = Asm(2, 0)
    A.param(0).raw(op).param(1).mul().halt()
    L = 400
    params = np.column_stack([np.full(L, 0.7), np.ones(L)])
    loss, g, _ = oracle_mod.run(A.bytes(), params, [], perturb=(11, 2))
    f = {B.EXP: math.exp, B.LOG: math.log, B.SIN: math.sin, B.COS: math.cos}[op]
    moves = _ulp_moves(f(0.7), 2)
    seen = set()
    for l in range(L):
        assert float(loss[l]) in moves, (l, loss[l])
        seen.add(moves[float(loss[l])])
        assert g[l, 1] == loss[l]
    assert seen == {-2, -1, 0, 1, 2}
    # different seeds give different draws; the same seed the same ones
    loss2, _, _ = oracle_mod.run(A.bytes(), params, [], perturb=(12, 2))
    loss3, _, _ = oracle_mod.run(A.bytes(), params, [], perturb=(11, 2))
    assert loss3.tobytes() == loss.tobytes() and loss2.tobytes() != loss.tobytes()


def test_perturb_reaches_adjoint_rule_evaluations(oracle_mod):
    """sin's adjoint evaluates cos(x): with the forward value unused by the
    loss's derivative path (loss = sin(p0)), the gradient moves in ulps of
    cos(p0)."""
    A = Asm(1, 0)
    A.param(0).sin().halt()
    L = 200
    loss, g, _ = oracle_mod.run(A.bytes(), np.full((L, 1), 0.3), [], perturb=(5, 1))
    moves = _ulp_moves(math.cos(0.3), 1)
    assert all(float(v) in moves for v in g[:, 0])
    assert len({float(v) for v in g[:, 0]}) == 3
