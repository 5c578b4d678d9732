"""Pins for the flattened-data-axis oracle (oracle/flatten.py).

* exponential decay: the flattened loss equals the unflattened program's loss
  bit for bit (same per-point operations, same ascending fold, same final
  multiplication), and the gradient matches the closed form;
* noise-free data at the generating parameters: exact zero gradient;
* random trees: flattened == unflattened oracle within rounding on lanes away
  from branch ties;
* the fold is sequential and ascending: terms chosen so that any other order
  or a pairwise sum gives another value.
"""
import math

import numpy as np

from conftest import lane_rel_err, rel_err
from workloads import configs
from workloads.bytecode import Asm


def test_exp_decay_flattened_equals_unflattened(oracle_mod):
    from oracle import flatten
    w = configs.exp_decay(L=32)
    n = 64
    pts = configs.points_of(w.obs, n)
    lf, gf = flatten.run_points(configs.exp_decay_term_program(), w.params, pts, 1.0 / n)
    lu, gu, _ = oracle_mod.run(w.bytecode, w.params, w.obs)
    assert lf.tobytes() == lu.tobytes()
    assert lane_rel_err(gf, gu).max() <= 1e-13
    t, y = w.obs[:n], w.obs[n:]
    for l, (a, b, c) in enumerate(w.params):
        e = [math.exp(-b * ti) for ti in t]
        r = [a * ei + c - yi for ei, yi in zip(e, y)]
        want = [2.0 / n * sum(ri * ei for ri, ei in zip(r, e)),
                -2.0 / n * sum(ri * a * ti * ei for ri, ti, ei in zip(r, t, e)),
                2.0 / n * sum(r)]
        assert lane_rel_err(gf[l], want).max() <= 1e-12


def test_exp_decay_flattened_zero_gradient_at_truth(oracle_mod):
    from oracle import flatten
    n = 64
    t = np.linspace(0.0, 5.0, n)
    a, b, c = 2.0, 0.7, 0.3
    y = np.array([a * math.exp(-(b * ti)) + c for ti in t])
    pts = np.column_stack([t, y])
    loss, g = flatten.run_points(configs.exp_decay_term_program(), [[a, b, c]], pts, 1.0 / n)
    assert loss[0] == 0.0 and np.all(g == 0.0)


def test_tree_flattened_matches_unflattened(oracle_mod):
    from oracle import flatten
    w = configs.random_programs(n_prog=12, L=6, n=128, seed=4242)
    pts = configs.points_of(w.obs, 128)
    checked = 0
    for q, tree in enumerate(w.meta["trees"]):
        P = w.n_params_each[q]
        pp = w.params[q][:, :P]
        lu, gu, m = oracle_mod.run(w.programs[q], pp, w.obs, margin=True)
        lf, gf = flatten.run_points(configs.tree_term_program(tree, P), pp, pts, 1.0 / 128)
        ok = m > 1e-6
        assert rel_err(lf[ok], lu[ok]).max(initial=0) <= 1e-12, q
        assert lane_rel_err(gf[ok], gu[ok]).max(initial=0) <= 1e-10, q
        checked += int(ok.sum())
    assert checked >= 40


def test_fold_is_sequential_ascending(oracle_mod):
    """term = obs[0] of the point (times p0 = 1): points 1e16, 1, -1e16, 1.
    Ascending left fold: ((1e16 + 1) - 1e16) + 1 = 1 (1e16 + 1 rounds to 1e16);
    a pairwise sum gives 0, a descending fold 1 + ... gives 1e16 - 1e16 + 1 = 1
    only by another route -- so also check a case that separates ascending
    from descending: points 1, 1e16, -1e16: ascending (1 + 1e16) - 1e16 = 0,
    descending (-1e16 + 1e16) + 1 = 1."""
    from oracle import flatten
    A = Asm(1, 1)
    A.obs(0).param(0).mul().halt()
    bc = A.bytes()
    loss, g = flatten.run_points(bc, [[1.0]], [[1e16], [1.0], [-1e16], [1.0]], 1.0)
    assert loss[0] == 1.0 and g[0, 0] == 1.0
    loss, g = flatten.run_points(bc, [[1.0]], [[1.0], [1e16], [-1e16]], 0.5)
    assert loss[0] == 0.0 and g[0, 0] == 0.0
