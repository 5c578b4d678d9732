"""The parity judge itself (tests/parity.py), on the CPU: results planted from
the oracle's own evaluations must be accepted by the rule that covers them,
and anything else rejected.  No lane may pass without matching some oracle
result."""
import math

import numpy as np
import pytest

from parity import compare, judge
from test_oracle_extended import _branchy
from workloads import configs


def _setup():
    n = 5
    bc = _branchy(n)
    obs = np.array([1.0 + 1e-12, 1.5, 1.0 - 3e-10, 1.0, 1.0 + 2e-9])
    params = np.array([[1.0, 0.7, -1.3], [1.0, 0.2, 0.4], [3.0, 0.7, -1.3], [1.0 + 5e-10, 1.1, 2.0]])
    return bc, params, obs


def test_judge_accepts_oracle_and_flipped_results(oracle_mod):
    bc, params, obs = _setup()
    ol, og, _ = oracle_mod.run(bc, params, obs)
    r = judge(oracle_mod, bc, params, obs, ol.copy(), og.copy())
    assert r["n_strict"] == 4 and r["n_other_arm"] == 0
    # lane 0 took the other arm at its second-closest tie (encounter 0), lane 3 at its
    # third (encounter 2, gap 8e-10; its encounter 4 at 1.5e-9 is no near tie)
    fl, fg, _ = oracle_mod.run(bc, params, obs, flip=np.array([0, -1, -1, 2]))
    r = judge(oracle_mod, bc, params, obs, fl, fg)
    assert r["n_strict"] == 2 and r["n_other_arm"] == 2 and r["n_ill_conditioned"] == 0


def test_judge_rejects_a_flip_of_a_clear_decision(oracle_mod):
    bc, params, obs = _setup()
    # encounter 1 (gap 0.5) is no near tie: the other arm there is not a valid result
    fl, fg, _ = oracle_mod.run(bc, params, obs, flip=np.array([1, -1, -1, -1]))
    with pytest.raises(AssertionError, match="lanes \\[0\\]"):
        judge(oracle_mod, bc, params, obs, fl, fg)


def test_judge_rejects_wrong_gradient_and_wrong_loss(oracle_mod):
    bc, params, obs = _setup()
    ol, og, _ = oracle_mod.run(bc, params, obs)
    g2 = og.copy()
    g2[2, 2] *= 1 + 1e-9
    with pytest.raises(AssertionError):
        judge(oracle_mod, bc, params, obs, ol, g2)
    l2 = ol.copy()
    l2[1] = -l2[1]
    with pytest.raises(AssertionError):
        judge(oracle_mod, bc, params, obs, l2, og)


def test_judge_ill_conditioned_rule(oracle_mod):
    """exp(p0) - exp(p0 + p1) with p1 = 1e-15: the fp64 value is mostly
    rounding.  The extended-precision value passes (it is within twice the
    fp64 oracle's own error of itself); a value off by more than that
    allowance does not."""
    from workloads.bytecode import Asm
    A = Asm(2, 0)
    A.param(0).exp().param(0).param(1).add().exp().sub().halt()
    bc = A.bytes()
    params = np.array([[0.5, 1e-15], [0.25, 3e-15]])
    ol, og, _ = oracle_mod.run(bc, params, [])
    le, ge, _ = oracle_mod.run(bc, params, [], extended=True)
    assert np.any(np.abs(ol - le) > 1e-11 * np.abs(le))        # the case is ill-conditioned
    r = judge(oracle_mod, bc, params, [], le, ge)
    assert r["n_ill_conditioned"] >= 1
    # a value far outside both the extended-precision allowance and the
    # spread under transcendental perturbations (here about 40 %: the
    # result is mostly library rounding) is rejected
    off = -3 * le
    with pytest.raises(AssertionError):
        judge(oracle_mod, bc, params, [], off, ge)


def test_compare_is_strict(oracle_mod):
    w = configs.logistic(L=5, T=20)
    ol, og, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
    assert compare(ol, og, ol, og)["max_grad_err"] == 0.0
    g2 = og.copy()
    g2[4, 0] += 1e-10 * np.abs(og[4]).max()
    with pytest.raises(AssertionError, match="lanes \\[4\\]"):
        compare(ol, g2, ol, og)
    # non-finite classes must agree
    l2 = ol.copy()
    l2[1] = np.nan
    with pytest.raises(AssertionError):
        compare(l2, og, ol, og)


def test_judge_libm_sensitivity_rule(oracle_mod):
    """A lane whose result swings under ulp-level changes of its
    transcendentals: another perturbed evaluation of the oracle (a stand-in
    for a different math library) passes; a result moved well beyond the
    measured spread does not."""
    from workloads.bytecode import Asm
    # (exp(p0) - p1) * p2 with p1 a few ulps from exp(p0): the loss is the
    # last ulps of the library exp
    A = Asm(3, 0)
    A.param(0).exp().param(1).sub().param(2).mul().halt()
    bc = A.bytes()
    rows = []
    for x, d in ((0.3, 3), (1.7, -5), (-0.4, 2)):
        y = math.exp(x)
        for _ in range(abs(d)):
            y = float(np.nextafter(y, np.inf if d > 0 else -np.inf))
        rows.append([x, y, 1.25])
    params = np.array(rows)
    ol, og, _ = oracle_mod.run(bc, params, [])
    pl, pg, _ = oracle_mod.run(bc, params, [], perturb=(999, 2))
    assert np.any(np.abs(pl - ol) > 1e-11 * np.abs(ol)) or \
        np.any(np.abs(pg - og) > 1e-11 * np.abs(og).max(axis=1, keepdims=True))
    r = judge(oracle_mod, bc, params, [], pl, pg)
    assert r["n_libm_sensitive"] + r["n_ill_conditioned"] >= 1
    far = ol + 50 * np.abs(pl - ol) + 1e-9 * np.abs(ol)
    with pytest.raises(AssertionError):
        judge(oracle_mod, bc, params, [], far, og)
